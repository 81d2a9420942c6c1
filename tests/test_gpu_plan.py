"""The prepared path (include/hv_plan.h) against the CPU oracle, and its HIP
graph: a captured pass replayed several times, with eager work and host
synchronisations between the replays, each replay checked against the eager
result.  (The full-size workloads in test_gpu_configs.py run through the same
plan, via ``Pipeline``.)
"""
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle
from test_gpu_parity import host_msgs, place

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


def threads():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_roots(msgs, C, alg, mode):
    leaves = oracle.leaf_digests_mt(msgs, C, threads(), alg)
    if mode == "single":
        return leaves, None, oracle.mth(leaves, alg)
    counts = [oracle.chunk_count(len(m), C, alg) for m in msgs]
    roots = oracle.seg_roots_from_leaves(leaves, counts, alg)
    return leaves, roots, oracle.mth(roots, alg)


@pytest.mark.parametrize("alg,C,mode,align_off", [
    ("sha256", 4096, "manifest", 0), ("sha256", 64, "single", 3), ("sha256", 0, "manifest", 1),
    ("sha384", 1024, "manifest", 0), ("sha384", 128, "single", 15), ("sha384", 0, "single", 0),
])
def test_plan_matches_oracle(alg, C, mode, align_off):
    rng = np.random.default_rng(1100)
    lens = np.concatenate([rng.integers(0, 30000, 300), [0, 1, 64, 128, 600_000]])
    buf, host, ptrs, lens, starts = place(lens, align_off, seed=1101)
    pipe = hv.Pipeline((ptrs, lens), C, mode, DEV, alg=alg)
    root = bytes(pipe.compute().cpu().numpy().reshape(-1))
    want_leaves, want_roots, want = oracle_roots(host_msgs(host, starts, lens), C, alg, mode)
    assert np.array_equal(pipe.leaves.cpu().numpy(), want_leaves)
    if want_roots is not None:
        assert [bytes(r) for r in pipe.roots.cpu().numpy()] == want_roots
    assert root == want
    assert pipe.run(want)
    bad = bytearray(want)
    bad[-1] ^= 1
    assert not pipe.run(bytes(bad))
    assert pipe.run(want)  # the stored expected root is replaced, not accumulated


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_empty_sets(alg):
    e = oracle.digest(b"", alg)
    for mode in ("manifest", "single"):
        pipe = hv.Pipeline((np.zeros(0, np.uint64), np.zeros(0, np.uint64)), 128, mode, DEV, alg=alg)
        assert bytes(pipe.compute().cpu().numpy().reshape(-1)) == oracle.mth([], alg) == e
        assert pipe.run(e)
    pipe = hv.Pipeline((np.zeros(3, np.uint64), np.zeros(3, np.uint64)), 128, "manifest", DEV, alg=alg)
    assert pipe.n_leaves == 0
    assert bytes(pipe.compute().cpu().numpy().reshape(-1)) == oracle.mth([e, e, e], alg)
    # the one-shot calls agree: no messages is the tree over no roots
    v = hv.Verifier(DEV, alg)
    none = (np.zeros(0, np.uint64), np.zeros(0, np.uint64))
    assert bytes(v.manifest_root(none, 128).cpu().numpy().reshape(-1)) == e
    assert bytes(v.single_tree_root(none, 128).cpu().numpy().reshape(-1)) == e
    assert hv.manifest_root({}, 128, alg=alg) == e


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_graph_replays_track_the_weights(alg):
    named = [(f"t{i}", W.bf16_weights(s, 1200 + i, DEV)) for i, s in enumerate([(512, 1024), (3, 5), (4096, 33)])]
    ms = W.message_set(named)
    C = 65536
    host = [v.cpu().numpy() for v in ms.views]
    _, _, want = oracle_roots(host, C, alg, "manifest")
    pipe = hv.Pipeline(ms, C, "manifest", DEV, alg=alg)
    pipe.capture(want)
    side = torch.randn(1024, 1024, device=DEV)
    view = ms.views[0]
    for rep in range(4):
        side = torch.tanh(side @ side)                 # eager work between replays
        torch.cuda.synchronize()
        assert pipe.replay(), f"replay {rep}"
        assert bytes(pipe.root.cpu().numpy().reshape(-1)) == want
        # change one byte eagerly: the next replay must see it and fail
        off = 1000 * rep + 7
        old = int(view[off].item())
        view[off] = old ^ 0x40
        torch.cuda.synchronize()
        assert not pipe.replay(), f"replay {rep} after a change"
        host[0][off] ^= 0x40
        _, _, changed = oracle_roots(host, C, alg, "manifest")
        assert bytes(pipe.root.cpu().numpy().reshape(-1)) == changed
        # the eager path agrees with the replay
        v = hv.Verifier(DEV, alg)
        assert bytes(v.manifest_root(ms.views, C).cpu().numpy().reshape(-1)) == changed
        view[off] = old
        host[0][off] ^= 0x40
        torch.cuda.synchronize()
    assert pipe.replay(want)
    # a new expected root stored between replays is the one compared
    other = bytes(48 if alg == "sha384" else 32)
    assert not pipe.replay(other)
    assert pipe.replay(want)


@pytest.mark.parametrize("alg,C,mode", [("sha256", 4096, "manifest"), ("sha256", 0, "single"),
                                        ("sha384", 1024, "manifest"), ("sha384", 128, "single")])
def test_verify_model_one_call(alg, C, mode):
    rng = np.random.default_rng(1300)
    lens = np.concatenate([rng.integers(0, 9000, 40), [0, 1, 200_000]])
    buf, host, ptrs, lens, starts = place(lens, 1, seed=1301)
    _, _, want = oracle_roots(host_msgs(host, starts, lens), C, alg, mode)
    r = hv.verify_model((ptrs, lens), C, want, alg=alg, mode=mode)
    assert r["root"] == want and r["integrity_verified"] and r["verification_time_ns"] > 0
    bad = bytearray(want)
    bad[0] ^= 0x80
    r = hv.verify_model((ptrs, lens), C, bytes(bad), alg=alg, mode=mode)
    assert r["root"] == want and not r["integrity_verified"]
    r = hv.verify_model((ptrs, lens), C, None, alg=alg, mode=mode)
    assert r["root"] == want and not r["integrity_verified"]


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_verify_model_empty_set(alg):
    # no messages: the root is the empty tree's in both forms, and a wrong
    # expected root is a False verdict, not an error
    e = oracle.mth([], alg)
    none = (np.zeros(0, np.uint64), np.zeros(0, np.uint64))
    for mode in ("manifest", "single"):
        r = hv.verify_model(none, 128, e, alg=alg, mode=mode)
        assert r["integrity_verified"] and r["root"] == e
        bad = bytearray(e)
        bad[0] ^= 1
        assert not hv.verify_model(none, 128, bytes(bad), alg=alg, mode=mode)["integrity_verified"]
