"""The synthetic workloads have the shapes the paper's model sizes call for.

Byte and leaf totals are recomputed here from the tensor lists; leaf counts
use the oracle's chunk count (Algorithm 1's ceil(|M| / C)).
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle


@pytest.mark.parametrize(
    "k,n_msgs,total,leaves",
    [
        (1, 1, 67_108_864, 64),
        (2, 147, 2_409_762_816, 2_331),
        (3, 32, 13_476_831_232, 3_230),
        (5, 723, 141_107_412_992, 2_153_249),
    ],
)
def test_model_shaped_workloads(k, n_msgs, total, leaves):
    lens = W.workload_lengths(k)
    assert len(lens) == n_msgs
    assert sum(lens) == total == W.workload_bytes(k)
    assert sum(oracle.chunk_count(n, W.CHUNK_BYTES[k]) for n in lens) == leaves


def test_small_message_workload():
    lens = W.small_message_lengths()
    assert len(lens) == 1_000_000
    assert lens.min() >= 4096 and lens.max() <= 65536
    assert not np.any(lens % 64 == 0)
    assert abs(lens.mean() - 34_800) < 200
    offs = W.packed_offsets(lens)
    assert np.all(offs % 64 == 0)
    assert np.all(offs[1:] >= offs[:-1] + lens[:-1])


def test_names_in_bytewise_order_and_shards():
    names = [n for n, _ in W.tensors_70b()]
    assert names == sorted(names, key=lambda s: s.encode())
    assert len(set(names)) == 723
    files = W.shard_files_7b()
    assert [f for f, _ in files] == sorted(f for f, _ in files)
    assert sum(len(t) for _, t in files) == 291
    assert "model.embed_tokens.weight" in files[0][1]
    assert {"lm_head.weight", "model.norm.weight"} <= set(files[31][1])
    kv = dict(W.tensors_70b())["model.layers.0.self_attn.k_proj.weight"]
    assert kv == (1024, 8192)


def test_generators_are_seeded_and_bf16():
    a = W.bf16_weights((64, 33), 5, "cpu")
    b = W.bf16_weights((64, 33), 5, "cpu")
    c = W.bf16_weights((64, 33), 6, "cpu")
    assert a.dtype == torch.bfloat16 and torch.equal(a, b) and not torch.equal(a, c)
    assert 0.01 < a.float().std().item() < 0.03
    r = W.random_bytes(1000, 1, "cpu")
    assert r.dtype == torch.uint8 and torch.equal(r, W.random_bytes(1000, 1, "cpu"))
    ms = W.message_set([("x", a), ("y", r)])
    assert list(ms.lens) == [64 * 33 * 2, 1000]
