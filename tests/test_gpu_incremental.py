"""Incremental re-verification: after some chunks change, rehashing only those
chunks and recomputing only the tree branches above them gives exactly the
digests and roots of a full recompute, and the oracle's roots of the new
bytes."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


def leaves_of_range(seg_offsets, chunk_bytes: int, msg: int, lo: int, hi: int) -> np.ndarray:
    """Leaf numbers of the chunks of message ``msg`` that hold any byte in [lo, hi): chunk i of a
    message covers bytes [i*C, (i+1)*C) (Algorithm 1), and C = 0 makes the whole message one leaf."""
    first = int(seg_offsets[msg])
    if hi <= lo:
        return np.zeros(0, dtype=np.uint64)
    if chunk_bytes == 0:
        return np.array([first], dtype=np.uint64)
    return np.arange(first + lo // chunk_bytes, first + (hi - 1) // chunk_bytes + 1, dtype=np.uint64)


@pytest.mark.parametrize("sizes", [[1], [2], [3], [0, 5, 0], [511, 512, 513], [1000, 1, 70000, 2]])
def test_tree_build_roots(sizes):
    n = int(sum(sizes))
    entries = W.random_bytes(max(n, 1) * 32, 400 + n, DEV)[: n * 32].view(n, 32)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    tree = hv.Tree(entries, seg)
    full = hv.hv_merkle_reduce(entries, seg)
    torch.cuda.synchronize()
    assert torch.equal(tree.roots, full)
    host = entries.cpu().numpy()
    assert [bytes(r) for r in tree.roots.cpu().numpy()] == \
        [oracle.mth(host[int(seg[s]):int(seg[s + 1])]) for s in range(len(sizes))]


@pytest.mark.parametrize("C", [4096, 65536, 0])
def test_update_after_partial_change(C):
    rng = np.random.default_rng(C + 3)
    lens = [0, 100, 4096, 5 * 65536 + 7, 300000, 1 << 20, 65536 * 17, 33]
    bufs = [W.random_bytes(n, 500 + i, DEV) for i, n in enumerate(lens)]
    leaves, seg = hv.hv_hash_chunks(bufs, C)
    tree = hv.Tree(leaves, seg)
    torch.cuda.synchronize()
    # change bytes: first byte of a message, its last byte, a run across a chunk boundary, a whole message
    edits = [(2, 0, 1), (3, lens[3] - 1, lens[3]), (5, 65536 - 3, 65536 + 5), (6, 0, lens[6])] + \
        [(4, int(p), int(p) + 1) for p in rng.integers(0, lens[4], 5)]
    dirty = set()
    for m, lo, hi in edits:
        bufs[m][lo:hi] ^= 0x5A
        dirty.update(int(x) for x in leaves_of_range(seg, C, m, lo, hi))
    dirty = np.array(sorted(dirty), dtype=np.uint64)
    hv.hv_rehash_chunks(bufs, C, dirty, leaves)
    roots = tree.update(leaves, dirty)
    full_leaves, _ = hv.hv_hash_chunks(bufs, C)
    full_roots = hv.hv_merkle_reduce(full_leaves, seg)
    torch.cuda.synchronize()
    assert torch.equal(leaves, full_leaves)
    assert torch.equal(roots, full_roots)
    host = [b.cpu().numpy() for b in bufs]
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.seg_root(h, C) for h in host]


def test_update_with_no_change_and_every_leaf():
    bufs = [W.random_bytes(n, 600 + i, DEV) for i, n in enumerate([70000, 3, 200000])]
    leaves, seg = hv.hv_hash_chunks(bufs, 4096)
    tree = hv.Tree(leaves, seg)
    before = tree.roots.clone()
    assert torch.equal(tree.update(leaves, []), before)
    for b in bufs:
        b ^= 0xFF
    allv = np.arange(int(seg[-1]), dtype=np.uint64)
    hv.hv_rehash_chunks(bufs, 4096, allv, leaves)
    roots = tree.update(leaves, allv)
    torch.cuda.synchronize()
    host = [b.cpu().numpy() for b in bufs]
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.seg_root(h, 4096) for h in host]


@pytest.mark.parametrize("sizes", [[1], [3], [0, 5, 0], [511, 512, 513], [1000, 1, 7000, 2]])
def test_tree_build_roots_sha384(sizes):
    n = int(sum(sizes))
    entries = W.random_bytes(max(n, 1) * 48, 450 + n, DEV)[: n * 48].view(n, 48)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    tree = hv.Tree(entries, seg, alg="sha384")
    full = hv.hv_merkle_reduce(entries, seg, alg="sha384")
    torch.cuda.synchronize()
    assert tree.roots.shape[1] == 48 and torch.equal(tree.roots, full)
    host = entries.cpu().numpy()
    assert [bytes(r) for r in tree.roots.cpu().numpy()] == \
        [oracle.mth(host[int(seg[s]):int(seg[s + 1])], "sha384") for s in range(len(sizes))]


@pytest.mark.parametrize("C", [4096, 128, 0])
def test_update_after_partial_change_sha384(C):
    alg = "sha384"
    rng = np.random.default_rng(C + 384)
    lens = [0, 100, 4096, 3 * 65536 + 7, 300000, 33]
    bufs = [W.random_bytes(n, 520 + i, DEV) for i, n in enumerate(lens)]
    leaves, seg = hv.hv_hash_chunks(bufs, C, alg=alg)
    tree = hv.Tree(leaves, seg, alg=alg)
    torch.cuda.synchronize()
    edits = [(2, 0, 1), (3, lens[3] - 1, lens[3]), (3, 4096 - 3, 4096 + 5)] + \
        [(4, int(p), int(p) + 1) for p in rng.integers(0, lens[4], 5)]
    dirty = set()
    for m, lo, hi in edits:
        bufs[m][lo:hi] ^= 0x5A
        dirty.update(int(x) for x in leaves_of_range(seg, C, m, lo, hi))
    dirty = np.array(sorted(dirty), dtype=np.uint64)
    hv.hv_rehash_chunks(bufs, C, dirty, leaves, alg=alg)
    roots = tree.update(leaves, dirty)
    full_leaves, _ = hv.hv_hash_chunks(bufs, C, alg=alg)
    full_roots = hv.hv_merkle_reduce(full_leaves, seg, alg=alg)
    torch.cuda.synchronize()
    assert torch.equal(leaves, full_leaves)
    assert torch.equal(roots, full_roots)
    host = [b.cpu().numpy() for b in bufs]
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.seg_root_alg(h, C, alg) for h in host]


def test_empty_segments_and_empty_lists():
    # segments without leaves keep the empty-tree root; an update with no
    # listed leaves and a rehash of no leaves change nothing
    e = oracle.mth([])
    seg = np.array([0, 0, 0], dtype=np.uint64)
    none = torch.empty((0, 32), dtype=torch.uint8, device=DEV)
    tree = hv.Tree(none, seg)
    torch.cuda.synchronize()
    assert [bytes(r) for r in tree.roots.cpu().numpy()] == [e, e]
    roots = tree.update(none, np.zeros(0, dtype=np.uint64))
    torch.cuda.synchronize()
    assert [bytes(r) for r in roots.cpu().numpy()] == [e, e]

    msgs = [W.random_bytes(5000, 470 + i, DEV) for i in range(2)]
    leaves, seg = hv.hv_hash_chunks(msgs, 4096)
    before = leaves.clone()
    hv.hv_rehash_chunks(msgs, 4096, np.zeros(0, dtype=np.uint64), leaves)
    torch.cuda.synchronize()
    assert torch.equal(leaves, before)
