"""Pins for the oracle's Merkle tree (RFC 6962 section 2.1) and composition.

The oracle computes MTH recursively.  These tests check it against:
* hand expansions of the definition for n = 0..4 written with hashlib;
* an independent bottom-up construction (pair neighbours, promote an odd last
  node unchanged) written here with hashlib, for every n up to 2000 and
  around powers of two -- the two orders agree only if the split point,
  the prefixes and the operand order are all right;
* invariants: any single-bit flip changes the root, order matters,
  C = 0 behaves as one whole-message chunk, the threaded driver equals the
  single-threaded one, and the closed form for constant bytes equals the
  plain computation.
"""
import hashlib

import numpy as np
import pytest

from oracle import oracle


def S(b: bytes) -> bytes:
    return hashlib.sha256(b).digest()


def bottom_up(entries):
    """Level-by-level tree: leaf = S(0x00||d), parent = S(0x01||L||R), odd last node promoted."""
    if not entries:
        return S(b"")
    level = [S(b"\x00" + d) for d in entries]
    while len(level) > 1:
        nxt = [S(b"\x01" + level[i] + level[i + 1]) for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def rand_entries(n, seed):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, 256, 32, dtype=np.uint8).tobytes() for _ in range(n)]


def test_hand_expansions():
    d = rand_entries(4, 10)
    l = [S(b"\x00" + x) for x in d]
    assert oracle.mth([]) == S(b"")
    assert oracle.mth(d[:1]) == l[0]
    assert oracle.mth(d[:2]) == S(b"\x01" + l[0] + l[1])
    assert oracle.mth(d[:3]) == S(b"\x01" + S(b"\x01" + l[0] + l[1]) + l[2])
    assert oracle.mth(d[:4]) == S(b"\x01" + S(b"\x01" + l[0] + l[1]) + S(b"\x01" + l[2] + l[3]))


def test_five_entries_split_at_four_not_duplicated():
    d = rand_entries(5, 11)
    l = [S(b"\x00" + x) for x in d]
    left = S(b"\x01" + S(b"\x01" + l[0] + l[1]) + S(b"\x01" + l[2] + l[3]))
    assert oracle.mth(d) == S(b"\x01" + left + l[4])
    # duplicating the odd node (another common convention) gives a different root
    dup = S(b"\x01" + left + S(b"\x01" + S(b"\x01" + l[4] + l[4]) + S(b"\x01" + l[4] + l[4])))
    assert oracle.mth(d) != dup


def test_recursive_equals_bottom_up_bruteforce():
    pool = rand_entries(4100, 12)
    sizes = list(range(0, 2001)) + [2047, 2048, 2049, 4095, 4097]
    for n in sizes:
        assert oracle.mth(pool[:n]) == bottom_up(pool[:n]), n


def test_every_single_bit_flip_changes_root():
    rng = np.random.default_rng(13)
    m = bytearray(rng.integers(0, 256, 5 * 64, dtype=np.uint8).tobytes())
    base = oracle.seg_root(bytes(m), 64)
    seen = {base}
    for bit in range(len(m) * 8):
        m[bit // 8] ^= 1 << (bit % 8)
        r = oracle.seg_root(bytes(m), 64)
        m[bit // 8] ^= 1 << (bit % 8)
        assert r != base, bit
        seen.add(r)
    assert len(seen) == 1 + len(m) * 8


def test_chunk_order_matters():
    rng = np.random.default_rng(14)
    m = rng.integers(0, 256, 6 * 128, dtype=np.uint8).tobytes()
    chunks = [m[i:i + 128] for i in range(0, len(m), 128)]
    base = oracle.seg_root(m, 128)
    for i, j in [(0, 1), (0, 5), (2, 3), (4, 5)]:
        sw = list(chunks)
        sw[i], sw[j] = sw[j], sw[i]
        assert oracle.seg_root(b"".join(sw), 128) != base
    # entry order matters for the tree itself too
    d = rand_entries(7, 15)
    assert oracle.mth(d) != oracle.mth(d[::-1])


def test_whole_message_chunking():
    rng = np.random.default_rng(16)
    for n in (1, 64, 1000, 4096):
        m = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        one_leaf = S(b"\x00" + S(m))
        assert oracle.seg_root(m, 0) == one_leaf
        assert oracle.seg_root(m, 4096) == one_leaf  # C >= len: one chunk too
    # empty message: C = 0 still has one leaf, SHA-256(""); C > 0 has none
    assert oracle.seg_root(b"", 0) == S(b"\x00" + S(b""))
    assert oracle.seg_root(b"", 64) == S(b"")


def test_seg_root_is_mth_of_chunk_digests():
    rng = np.random.default_rng(17)
    m = rng.integers(0, 256, 10 * 256 + 17, dtype=np.uint8).tobytes()
    digests = [S(m[i:i + 256]) for i in range(0, len(m), 256)]
    assert oracle.seg_root(m, 256) == bottom_up(digests)


def test_manifest_root_by_hand():
    rng = np.random.default_rng(18)
    msgs = [rng.integers(0, 256, n, dtype=np.uint8).tobytes() for n in (300, 0, 64, 129)]
    roots = [bottom_up([S(m[i:i + 64]) for i in range(0, len(m), 64)]) for m in msgs]
    assert oracle.manifest_root(msgs, 64) == bottom_up(roots)


def test_sharding_split_recombines():
    # a tree split at the largest power of two below n recombines with one node
    d = rand_entries(3000, 19)
    for n in (3, 17, 1000, 2049, 3000):
        k = 1 << ((n - 1).bit_length() - 1)
        assert oracle.mth(d[:n]) == S(b"\x01" + oracle.mth(d[:k]) + oracle.mth(d[k:n]))


@pytest.mark.parametrize("nthreads", [1, 3, 8])
def test_threaded_driver_equals_plain(nthreads):
    rng = np.random.default_rng(20)
    lens = [0, 1, 64, 200, 4096, 4097, 0, 9000, 63]
    msgs = [rng.integers(0, 256, n, dtype=np.uint8).tobytes() for n in lens]
    for C in (64, 4096, 0):
        want = np.concatenate([oracle.chunk_digests(m, C) for m in msgs]) if msgs else None
        got = oracle.leaf_digests_mt(msgs, C, nthreads)
        assert np.array_equal(got, want), C


def test_closed_form_constant_bytes():
    for C in (64, 128, 4096, 0):
        for length in (0, 1, 63, 64, 65, 127, 128, 129, 640, 641, 4096 * 5, 4096 * 5 + 100, 64 * 37 + 3):
            for byte in (0, 0x5A):
                want = oracle.seg_root(bytes([byte]) * length, C)
                assert oracle.const_seg_root(length, C, byte) == want, (C, length, byte)
