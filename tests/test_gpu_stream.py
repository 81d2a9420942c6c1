"""Streaming digests of host-resident messages (Algorithm 1's load / hash /
free loop) equal the resident path's digests and the oracle's, for batches
that split messages at chunk boundaries, whole-message chunks, pinned and
pageable sources."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


def host_messages(lens, seed, pinned):
    out = []
    for i, n in enumerate(lens):
        d = W.random_bytes(int(n), seed + i, DEV).cpu()
        if pinned:
            p = torch.empty(int(n), dtype=torch.uint8, pin_memory=True)
            p.copy_(d)
            d = p
        out.append(d)
    return out


@pytest.mark.parametrize("pinned", [True, False])
@pytest.mark.parametrize("C,batch", [(4096, 64 << 10), (65536, 1 << 20), (64, 8 << 10), (1 << 20, 1 << 20)])
def test_streamed_digests_equal_resident_and_oracle(C, batch, pinned):
    rng = np.random.default_rng(C + batch)
    lens = [0, 1, 63, C, C + 1, 3 * C - 1, batch, batch + 17, 5 * batch + C // 2 + 3] + \
        [int(x) for x in rng.integers(0, 4 * batch, 12)]
    msgs = host_messages(lens, 700, pinned)
    got, seg = hv.hv_hash_host_chunks(msgs, C, batch)
    dev_msgs = [m.to(DEV) for m in msgs]
    resident, seg2 = hv.hv_hash_chunks(dev_msgs, C)
    torch.cuda.synchronize()
    assert np.array_equal(seg, seg2)
    assert torch.equal(got, resident)
    want = oracle.leaf_digests_mt([m.numpy() for m in msgs], C, 8)
    assert np.array_equal(got.cpu().numpy(), want)


def test_whole_message_chunks_streamed():
    lens = [0, 5, 4096, 70000, 65536, 1, 0, 123457]
    msgs = host_messages(lens, 800, True)
    got, _ = hv.hv_hash_host_chunks(msgs, 0, 128 << 10)
    want = oracle.leaf_digests_mt([m.numpy() for m in msgs], 0, 4)
    assert np.array_equal(got.cpu().numpy(), want)


def test_streamed_roots_and_manifest():
    lens = [3 << 20, 17, (1 << 20) + 5, 0, 2 << 20]
    msgs = host_messages(lens, 900, True)
    C = 65536
    leaves, seg = hv.hv_hash_host_chunks(msgs, C, 1 << 20)
    roots = hv.hv_merkle_reduce(leaves, seg)
    top = hv.hv_merkle_reduce(roots, np.array([0, len(lens)], dtype=np.uint64))
    host = [m.numpy() for m in msgs]
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.seg_root(h, C) for h in host]
    assert hv.hv_verify_root(top, oracle.manifest_root(host, C))


def test_stream_argument_errors():
    msgs = host_messages([1 << 20], 1000, False)
    for C, batch in ((4096, 1000), (1 << 20, 1 << 19), (0, 1 << 19)):
        with pytest.raises(hv.HVError) as e:
            hv.hv_hash_host_chunks(msgs, C, batch)
        assert e.value.status == hv.HV_ERR_INVALID_ARG


@pytest.mark.parametrize("C,batch", [(4096, 64 << 10), (128, 8 << 10), (0, 256 << 10)])
def test_streamed_sha384_equal_resident_and_oracle(C, batch):
    rng = np.random.default_rng(C + batch + 384)
    cap = batch if C == 0 else 4 * batch
    lens = [0, 1, 111, 112, 128, max(C, 1) + 1, batch] + [int(x) for x in rng.integers(0, cap, 10)]
    msgs = host_messages(lens, 1100, True)
    got, seg = hv.hv_hash_host_chunks(msgs, C, batch, alg="sha384")
    resident, seg2 = hv.hv_hash_chunks([m.to(DEV) for m in msgs], C, alg="sha384")
    torch.cuda.synchronize()
    assert got.shape[1] == 48 and np.array_equal(seg, seg2)
    assert torch.equal(got, resident)
    want = oracle.leaf_digests_mt([m.numpy() for m in msgs], C, 8, "sha384")
    assert np.array_equal(got.cpu().numpy(), want)


@pytest.mark.parametrize("C", [4096, 0])
def test_stream_empty_sets(C):
    # no messages, and messages that are all empty: the same digests as the
    # resident path (none with C > 0; one SHA-256("") per message with C = 0)
    got, seg = hv.hv_hash_host_chunks((np.zeros(0, np.uint64), np.zeros(0, np.uint64)), C, 1 << 20)
    torch.cuda.synchronize()
    assert got.shape == (0, 32) and list(seg) == [0]
    msgs = [torch.empty(0, dtype=torch.uint8) for _ in range(3)]
    got, seg = hv.hv_hash_host_chunks(msgs, C, 1 << 20)
    resident, seg2 = hv.hv_hash_chunks([m.to(DEV) for m in msgs], C)
    torch.cuda.synchronize()
    assert np.array_equal(seg, seg2) and torch.equal(got, resident)
    assert [bytes(d) for d in got.cpu().numpy()] == ([oracle.digest(b"")] * 3 if C == 0 else [])
