"""SHA-384 path (the *_alg entry points with HV_SHA384) vs the CPU oracle, bit
for bit: leaf digests over every length through several 128-byte blocks and
both padding forms, all alignments, whole-message chunks; RFC 6962 trees with
48-byte nodes; the on-GPU comparisons over 48 bytes; two model-shaped
workloads in full.  Expected values come only from ``oracle``.
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
ALG = "sha384"


def threads():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def check_all(buf, host, ptrs, lens, starts, C, tag=""):
    v = hv.Verifier(DEV, ALG)
    leaves, seg = v.leaf_digests((ptrs, lens), C)
    roots = hv.hv_merkle_reduce(leaves, seg, v.ws_tree, alg=ALG)
    manifest = hv.hv_merkle_reduce(roots, np.array([0, len(lens)], dtype=np.uint64), v.ws_manifest, alg=ALG)
    torch.cuda.synchronize()
    assert leaves.shape[1] == 48
    msgs = host_msgs(host, starts, lens)
    want_leaves = oracle.leaf_digests_mt(msgs, C, threads(), ALG)
    got_leaves = leaves.cpu().numpy()
    if not np.array_equal(got_leaves, want_leaves):
        bad = np.nonzero((got_leaves != want_leaves).any(axis=1))[0]
        owner = np.searchsorted(seg, bad[0], side="right") - 1
        raise AssertionError(f"{tag}: {len(bad)} leaf digests differ; first leaf {bad[0]} "
                             f"(message {owner}, length {int(lens[owner])}, C={C})")
    want_roots = oracle.seg_roots_from_leaves(want_leaves, np.diff(seg), ALG)
    assert [bytes(r) for r in roots.cpu().numpy()] == want_roots, f"{tag}: segment roots differ"
    assert bytes(manifest.cpu().numpy().reshape(-1)) == oracle.mth(want_roots, ALG), f"{tag}: manifest differs"


@pytest.mark.parametrize("align_off", [0, 1, 3, 15])
@pytest.mark.parametrize("C", [128, 1024, 0])
def test_every_length_up_to_2200(C, align_off):
    # 0..17 whole blocks, every tail length, tails of 111 (one final block) and 112 (two)
    lens = np.arange(0, 2201)
    buf, host, ptrs, lens, starts = place(lens, align_off, seed=400 + align_off)
    check_all(buf, host, ptrs, lens, starts, C, f"C={C} off={align_off}")


@pytest.mark.parametrize("C", [128, 65536, 1 << 20, 0])
def test_mixed_batch(C):
    rng = np.random.default_rng(17)
    lens = np.concatenate([
        rng.integers(0, 300, 200), rng.integers(1, 70000, 200), [0, 0, 1, 111, 112, 128, 65536, 65537],
        rng.integers(1 << 20, 3 << 20, 4),
    ])
    rng.shuffle(lens)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=18)
    check_all(buf, host, ptrs, lens, starts, C, f"mixed C={C}")


@pytest.fixture
def leaf_kernel():
    yield hv.set_leaf_kernel
    hv.set_leaf_kernel("auto")


@pytest.mark.parametrize("choice", ["one-wave", "two-wave", "two-wave-compact"])
@pytest.mark.parametrize("align_off", [0, 5])
@pytest.mark.parametrize("C", [128, 4096, 0])
def test_leaf_kernels(C, align_off, choice, leaf_kernel):
    # the one-wave kernel and the two-wave kernel (schedule on a producer wave;
    # one or two pairs per workgroup) forced on the same inputs
    leaf_kernel(choice)
    lens = np.arange(0, 1301)
    buf, host, ptrs, lens, starts = place(lens, align_off, seed=410 + align_off)
    check_all(buf, host, ptrs, lens, starts, C, f"{choice} C={C} off={align_off}")


def place_offsets(lens, offs, seed):
    """Messages each at its own offset from a 16-byte boundary: (buf, host, ptrs, lens, starts)."""
    starts = np.zeros(len(lens), dtype=np.uint64)
    pos = 0
    for i, n in enumerate(lens):
        starts[i] = pos + int(offs[i])
        pos += (int(n) + int(offs[i]) + 16 + 15) // 16 * 16
    buf = W.random_bytes(max(pos, 1), seed, DEV)
    host = buf.cpu().numpy()
    ptrs = np.uint64(buf.data_ptr()) + starts
    ptrs[lens == 0] = 0
    return buf, host, ptrs, lens, starts


@pytest.mark.parametrize("choice", ["auto", "two-wave", "two-wave-compact", "one-wave"])
def test_mixed_alignment_and_two_pairs(choice, leaf_kernel):
    # more than 64 chunks per CU (two pairs per workgroup under the two-wave
    # kernel), random lengths, and 10% of the messages off 16-byte alignment
    leaf_kernel(choice)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 100 * cus
    rng = np.random.default_rng(411)
    lens = rng.integers(0, 1500, n).astype(np.uint64)
    lens[rng.integers(0, n, 30)] = rng.integers(20000, 70000, 30).astype(np.uint64)
    offs = rng.integers(0, 16, n) * (rng.random(n) < 0.1)
    buf, host, ptrs, lens, starts = place_offsets(lens, offs, 412)
    check_all(buf, host, ptrs, lens, starts, 0, f"{choice} n={n}")


@pytest.mark.parametrize("choice", ["one-wave", "two-wave"])
def test_long_chunks(choice, leaf_kernel):
    leaf_kernel(choice)
    lens = [(4 << 20) + 111, (4 << 20) + 112, 3 << 20, 1, 0]
    buf, host, ptrs, lens, starts = place(lens, 0, seed=413)
    check_all(buf, host, ptrs, lens, starts, 0, f"{choice} long")


def test_empty_cases():
    v = hv.Verifier(DEV, ALG)
    leaves, seg = v.leaf_digests((np.zeros(0, np.uint64), np.zeros(0, np.uint64)), 128)
    assert leaves.shape == (0, 48) and list(seg) == [0]
    ptrs, lens = np.zeros(3, np.uint64), np.zeros(3, np.uint64)
    leaves, seg = v.leaf_digests((ptrs, lens), 128)
    assert leaves.shape == (0, 48)
    roots = hv.hv_merkle_reduce(leaves, seg, v.ws_tree, alg=ALG)
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.mth([], ALG)] * 3
    assert oracle.mth([], ALG) == oracle.sha384(b"")
    leaves, seg = v.leaf_digests((ptrs, lens), 0)
    assert [bytes(r) for r in leaves.cpu().numpy()] == [oracle.sha384(b"")] * 3


@pytest.mark.parametrize("sizes", [
    [0], [1], [2], [3], [5], [511, 512, 513], [0, 1, 0, 2, 0], [1023, 1024, 1025, 4097],
    [300_000], [262_145, 3, 0, 70_000],
])
def test_merkle_segments(sizes):
    n = int(sum(sizes))
    entries = W.random_bytes(max(n, 1) * 48, 500 + n, DEV)[: n * 48].view(n, 48)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    roots = hv.hv_merkle_reduce(entries, seg, alg=ALG)
    torch.cuda.synchronize()
    host = entries.cpu().numpy()
    want = [oracle.mth(host[int(seg[s]):int(seg[s + 1])], ALG) for s in range(len(sizes))]
    assert [bytes(r) for r in roots.cpu().numpy()] == want


def test_verify_and_compare_all_48_bytes():
    entries = W.random_bytes(7 * 48, 600, DEV).view(7, 48)
    root = hv.hv_merkle_reduce(entries, np.array([0, 7], dtype=np.uint64), alg=ALG)
    want = oracle.mth(entries.cpu().numpy(), ALG)
    assert hv.hv_verify_root(root, want, alg=ALG)
    for byte in (0, 13, 31, 32, 40, 47):  # bytes past the first 32 count too
        bad = bytearray(want)
        bad[byte] ^= 0x10
        assert not hv.hv_verify_root(root, bytes(bad), alg=ALG)
    a = W.random_bytes(10 * 48, 601, DEV).view(10, 48)
    b = a.clone()
    b[2, 0] ^= 1
    b[5, 33] ^= 4
    b[9, 47] ^= 128
    mism = hv.hv_compare_roots(a, b, alg=ALG).cpu().numpy()
    assert list(np.nonzero(mism)[0]) == [2, 5, 9]


def test_sha256_through_the_alg_entry_point_matches_the_plain_one():
    lens = np.array([0, 1, 64, 1000, 5000, 70001], dtype=np.uint64)
    buf, host, ptrs, lens, starts = place(lens, 3, seed=700)
    plain, seg = hv.hv_hash_chunks((ptrs, lens), 64, DEV)
    arr = hv._msg_array(ptrs, lens)
    out = torch.empty_like(plain)
    ws = hv.Workspace(DEV).get(hv.lib.hv_hash_workspace_bytes(len(arr), plain.shape[0]))
    hv._check(hv.lib.hv_hash_chunks_alg(hv.HV_SHA256, arr.ctypes.data, len(arr), 64, out.data_ptr(),
                                        ws.data_ptr(), ws.numel(), hv._stream(DEV)))
    torch.cuda.synchronize()
    assert torch.equal(out, plain)


def test_bf16_tensors_manifest_and_verify():
    named = [(f"t{i}", W.bf16_weights(s, 60 + i, DEV)) for i, s in enumerate([(3, 7), (1000, 33), (2048,), (64, 1024)])]
    C = 4096
    host = {n: W.as_bytes(t).cpu().numpy().tobytes() for n, t in named}
    order = sorted(host, key=lambda n: n.encode("utf-8"))
    want = oracle.mth([oracle.seg_root_alg(host[n], C, ALG) for n in order], ALG)
    assert hv.manifest_root(dict(named), C, alg=ALG) == want
    hv.verify(dict(named), want, C, alg=ALG)
    with pytest.raises(hv.VerificationError):
        hv.verify(dict(named), bytes(48), C, alg=ALG)
    with pytest.raises(ValueError):
        hv.verify(dict(named), want[:32], C, alg=ALG)  # a SHA-256-sized root is rejected


def test_kernel_timing_covers_the_sha384_kernel():
    lens = np.array([1 << 20] * 8, dtype=np.uint64)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=701)
    hv.set_kernel_timing(True)
    try:
        hv.hv_hash_chunks((ptrs, lens), 1 << 16, DEV, alg=ALG)
        ms = hv.leaf_kernel_ms()
    finally:
        hv.set_kernel_timing(False)
    assert 0 < ms < 1000


@pytest.mark.timeout(600)
@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_workloads_in_full(k):
    # at their full sizes: 64 MiB of random bytes (1 MiB chunks, one root),
    # 1B-shaped weights (per-tensor roots + manifest, 1 MiB chunks), the
    # 7B-shaped shard files (per-file roots + manifest, 4 MiB chunks) and
    # 10^6 small messages (whole-message chunks, one root)
    wl = W.workload(k, DEV)
    pipe = hv.Pipeline(wl.msgs, wl.chunk_bytes, "manifest" if wl.manifest else "single", DEV, alg=ALG)
    root = bytes(pipe.compute().cpu().numpy().reshape(-1))
    torch.cuda.synchronize()
    C = wl.chunk_bytes
    if k == 4:
        hostbuf = wl.msgs.buffer.cpu().numpy()
        want = oracle.leaf_digests_mt_packed(hostbuf, wl.msgs.offsets, wl.msgs.lens, C, threads(), ALG)
    else:
        want = oracle.leaf_digests_mt([v.cpu().numpy() for v in wl.msgs.views], C, threads(), ALG)
    assert np.array_equal(pipe.leaves.cpu().numpy(), want), f"workload {k}: leaf digests differ"
    counts = [oracle.chunk_count(int(n), C) for n in wl.msgs.lens]
    if wl.manifest:
        roots = oracle.seg_roots_from_leaves(want, counts, ALG)
        assert [bytes(r) for r in pipe.roots.cpu().numpy()] == roots
        expected = oracle.mth(roots, ALG)
    else:
        expected = oracle.mth(want, ALG)
    assert root == expected
    assert pipe.run(expected)
    bad = bytearray(expected)
    bad[47] ^= 1
    assert not pipe.run(bytes(bad))
    del wl, pipe
    torch.cuda.empty_cache()
