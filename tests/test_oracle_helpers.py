"""Pins for the oracle's composing helpers: per-message roots from a leaf
array, the per-message root for either hash, the tree over a 2-D digest
array, and the hash dispatcher.

These helpers give the expected per-tensor roots of the GPU parity tests, so
each is checked here against references that share nothing with the oracle:
Python's hashlib for SHA-256 and SHA-384, plain slices of the message for
the chunking rule of Algorithm 1 (ceil(|M| / C) chunks, the last one shorter,
none for an empty message, the whole message when C = 0), and a bottom-up
tree written here (RFC 6962 section 2.1 evaluated level by level: leaf
H(0x00 || d), parent H(0x01 || L || R), an unpaired last node moved up
unchanged, H("") for no entries).
"""
import hashlib

import numpy as np
import pytest

from oracle import oracle

HASHES = {"sha256": (hashlib.sha256, 32), "sha384": (hashlib.sha384, 48)}


def chunk_slices(m: bytes, C: int):
    """Algorithm 1's chunks of one message, as slices."""
    if C == 0:
        return [m]
    return [m[i:i + C] for i in range(0, len(m), C)]


def bottom_up(entries, h):
    if not entries:
        return h(b"").digest()
    level = [h(b"\x00" + d).digest() for d in entries]
    while len(level) > 1:
        nxt = [h(b"\x01" + level[i] + level[i + 1]).digest() for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def messages(seed, lens):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, 256, n, dtype=np.uint8).tobytes() for n in lens]


# empty messages at the start, middle and end, single-chunk and single-block
# messages, exact multiples of C and ragged tails, a message of 2^k + 1 chunks
LENS = [0, 1, 128, 0, 129, 1000, 640, 0, 4096 + 17, 384, 33 * 128, 0]


@pytest.mark.parametrize("alg", sorted(HASHES))
@pytest.mark.parametrize("C", [128, 256, 0])
def test_seg_roots_from_leaves_equals_per_message_trees(alg, C):
    h, D = HASHES[alg]
    msgs = messages(40, LENS)
    per_msg = [[h(s).digest() for s in chunk_slices(m, C)] for m in msgs]
    counts = [len(p) for p in per_msg]
    leaves = np.frombuffer(b"".join(d for p in per_msg for d in p), dtype=np.uint8).reshape(-1, D)
    want = [bottom_up(p, h) for p in per_msg]
    # counts as the tests pass them: a list, and the differences of segment offsets
    assert oracle.seg_roots_from_leaves(leaves, counts, alg) == want
    seg = np.concatenate([[0], np.cumsum(counts)]).astype(np.uint64)
    assert oracle.seg_roots_from_leaves(leaves, np.diff(seg), alg) == want
    # an empty message has no leaves and the root of no entries
    for m, r in zip(msgs, want):
        if not m and C != 0:
            assert r == h(b"").digest()


def test_seg_roots_from_leaves_keeps_message_order():
    h, D = HASHES["sha256"]
    msgs = messages(41, [300, 700])
    per_msg = [[h(s).digest() for s in chunk_slices(m, 256)] for m in msgs]
    leaves = np.frombuffer(b"".join(d for p in per_msg for d in p), dtype=np.uint8).reshape(-1, D)
    counts = [len(p) for p in per_msg]
    roots = oracle.seg_roots_from_leaves(leaves, counts)
    assert roots == [bottom_up(per_msg[0], h), bottom_up(per_msg[1], h)]
    # the same leaves split differently give different roots: the counts decide the segments
    assert oracle.seg_roots_from_leaves(leaves, [counts[0] + 1, counts[1] - 1]) != roots


@pytest.mark.parametrize("alg", sorted(HASHES))
@pytest.mark.parametrize("C", [128, 1024, 0])
def test_seg_root_alg_equals_tree_over_chunk_slices(alg, C):
    h, _ = HASHES[alg]
    for m in messages(42, [0, 1, 127, 128, 129, 1024, 1025, 5 * 1024, 9 * 1024 + 3]):
        assert oracle.seg_root_alg(m, C, alg) == bottom_up([h(s).digest() for s in chunk_slices(m, C)], h), len(m)


def test_seg_root_alg_sha256_is_seg_root():
    for m in messages(43, [0, 64, 65, 4096, 4097]):
        assert oracle.seg_root_alg(m, 64) == oracle.seg_root(m, 64)


@pytest.mark.parametrize("alg", sorted(HASHES))
def test_mth_accepts_2d_arrays_as_its_list_form(alg):
    h, D = HASHES[alg]
    rng = np.random.default_rng(44)
    for n in [0, 1, 2, 3, 7, 8, 9, 100]:
        arr = rng.integers(0, 256, (n, D), dtype=np.uint8)
        as_list = [bytes(r) for r in arr]
        want = bottom_up(as_list, h)
        assert oracle.mth(arr, alg) == want, n
        assert oracle.mth(as_list, alg) == want, n
        # a non-contiguous view (every other row) is read row by row, not by its memory
        if n >= 2:
            wide = rng.integers(0, 256, (2 * n, D), dtype=np.uint8)
            assert oracle.mth(wide[::2], alg) == bottom_up([bytes(r) for r in wide[::2]], h), n


@pytest.mark.parametrize("alg", sorted(HASHES))
def test_digest_dispatches_to_the_named_hash(alg):
    h, _ = HASHES[alg]
    for m in messages(45, [0, 3, 111, 112, 200]):
        assert oracle.digest(m, alg) == h(m).digest()
