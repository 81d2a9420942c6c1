"""Pins for the oracle's SHA-384 (FIPS 180-4 section 6.5) and its 48-byte
RFC 6962 tree, none reusing the oracle's code: published example digests,
the constants re-derived from their definition, hashlib at every length that
takes a different padding path, and a bottom-up tree written here."""
import hashlib

import numpy as np
import pytest

from conftest import golden_message, load_golden
from oracle import oracle
from test_oracle_sha256 import first_primes, iroot


@pytest.mark.parametrize("name,spec,digest", load_golden("fips180_sha384_examples.txt"))
def test_published_examples(name, spec, digest):
    assert oracle.sha384(golden_message(spec)).hex() == digest, name


def test_constants_from_their_definition():
    K, H = oracle.constants512()
    p = first_primes(80)
    assert K == [iroot(q << 192, 3) & ((1 << 64) - 1) for q in p]          # 4.2.3: cube roots, 80 primes
    assert H == [iroot(q << 128, 2) & ((1 << 64) - 1) for q in p[8:16]]    # 5.3.4: square roots, primes 9..16


def test_padding_paths_match_hashlib():
    rng = np.random.default_rng(30)
    data = rng.integers(0, 256, 3 * 128 * 8 + 256, dtype=np.uint8).tobytes()
    lengths = list(range(0, 260)) + [b + r for b in range(0, 3 * 1024, 128) for r in (0, 111, 112, 127)]
    for n in lengths:
        assert oracle.sha384(data[:n]) == hashlib.sha384(data[:n]).digest(), n


def bottom_up384(entries):
    S = lambda b: hashlib.sha384(b).digest()
    if not entries:
        return S(b"")
    level = [S(b"\x00" + d) for d in entries]
    while len(level) > 1:
        nxt = [S(b"\x01" + level[i] + level[i + 1]) for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def test_tree_matches_bottom_up():
    rng = np.random.default_rng(31)
    pool = [rng.integers(0, 256, 48, dtype=np.uint8).tobytes() for _ in range(700)]
    for n in list(range(0, 130)) + [255, 256, 257, 511, 513, 700]:
        assert oracle.mth(pool[:n], "sha384") == bottom_up384(pool[:n]), n


def test_chunks_need_whole_blocks():
    with pytest.raises(ValueError):
        oracle.chunk_count(1000, 64, "sha384")
    assert oracle.chunk_count(1000, 128, "sha384") == 8


@pytest.mark.parametrize("C", [128, 1024, 0])
def test_chunk_digests_are_plain_sha384_of_slices(C):
    rng = np.random.default_rng(32)
    for n in (0, 1, 111, 112, 128, 129, 1024 * 3 + 5):
        m = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        got = [bytes(r) for r in oracle.chunk_digests_alg(m, C, "sha384")]
        want = [hashlib.sha384(m).digest()] if C == 0 else \
            [hashlib.sha384(m[i:i + C]).digest() for i in range(0, n, C)]
        assert got == want, (n, C)


@pytest.mark.parametrize("nthreads", [1, 3, 8])
def test_threaded_drivers_are_hashlib_per_chunk(nthreads):
    # both threaded drivers (separate messages, and messages packed in one
    # buffer at offsets) against hashlib over each chunk slice
    rng = np.random.default_rng(33)
    lens = [0, 1, 111, 112, 128, 300, 4096, 4097, 0, 9000]
    offs, pos = [], 0
    for n in lens:
        offs.append(pos)
        pos += (n + 63) // 64 * 64
    buf = rng.integers(0, 256, max(pos, 1), dtype=np.uint8)
    msgs = [buf[o:o + n].tobytes() for o, n in zip(offs, lens)]
    for C in (128, 1024, 0):
        want = [hashlib.sha384(m).digest() for m in msgs] if C == 0 else \
            [hashlib.sha384(m[i:i + C]).digest() for m in msgs for i in range(0, len(m), C)]
        got = oracle.leaf_digests_mt(msgs, C, nthreads, "sha384")
        assert [bytes(r) for r in got] == want, C
        got = oracle.leaf_digests_mt_packed(buf, offs, lens, C, nthreads, "sha384")
        assert [bytes(r) for r in got] == want, C
