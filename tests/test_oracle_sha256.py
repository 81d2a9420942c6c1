"""Pins for the oracle's SHA-256 (FIPS 180-4), none of which reuse its code.

* published example digests (golden file, FIPS 180-2 Appendix B);
* the round constants and initial value re-derived here from their
  definition (fractional parts of cube / square roots of primes, FIPS 180-4
  sections 4.2.2 and 5.3.3) with exact integer roots;
* an independent library (Python's hashlib) on random data at every length
  that exercises a different padding path.
"""
import hashlib

import numpy as np
import pytest

from conftest import golden_message, load_golden
from oracle import oracle


def first_primes(n):
    ps, k = [], 2
    while len(ps) < n:
        if all(k % p for p in ps if p * p <= k):
            ps.append(k)
        k += 1
    return ps


def iroot(x, r):
    """floor(x ** (1/r)) for a non-negative integer x, exactly."""
    lo, hi = 0, 1 << ((x.bit_length() + r - 1) // r + 1)
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if mid ** r <= x:
            lo = mid
        else:
            hi = mid - 1
    return lo


@pytest.mark.parametrize("name,spec,digest", load_golden("fips180_sha256_examples.txt"))
def test_published_examples(name, spec, digest):
    assert oracle.sha256(golden_message(spec)).hex() == digest, name


def test_constants_from_their_definition():
    K, H0 = oracle.constants()
    primes = first_primes(64)
    # first 32 bits of the fractional part of cbrt(p): floor(cbrt(p) * 2^32) mod 2^32
    K_def = [iroot(p << 96, 3) & 0xFFFFFFFF for p in primes]
    # first 32 bits of the fractional part of sqrt(p) for the first 8 primes
    H_def = [iroot(p << 64, 2) & 0xFFFFFFFF for p in primes[:8]]
    assert K == K_def
    assert H0 == H_def


def test_every_short_length_matches_hashlib():
    rng = np.random.default_rng(1)
    data = rng.integers(0, 256, 400, dtype=np.uint8).tobytes()
    for n in range(0, 301):
        assert oracle.sha256(data[:n]) == hashlib.sha256(data[:n]).digest(), n


def test_padding_boundaries_match_hashlib():
    # lengths = 0, 55, 56, 63 (mod 64): one vs two final blocks, up to 3 * 4096 + 64
    rng = np.random.default_rng(2)
    data = rng.integers(0, 256, 3 * 4096 + 128, dtype=np.uint8).tobytes()
    for base in range(0, 3 * 4096 + 64, 64):
        for r in (0, 55, 56, 63):
            n = base + r
            assert oracle.sha256(data[:n]) == hashlib.sha256(data[:n]).digest(), n


def test_bf16_like_and_constant_bytes_match_hashlib():
    rng = np.random.default_rng(3)
    w = (rng.standard_normal(5000).astype(np.float32) * 0.02).view(np.uint32)
    bf16 = (w >> 16).astype(np.uint16).tobytes()
    for blob in (bf16, bytes(4097), b"\xff" * 70000):
        assert oracle.sha256(blob) == hashlib.sha256(blob).digest()


@pytest.mark.parametrize(
    "length,C,expected",
    [
        (0, 64, 0), (1, 64, 1), (63, 64, 1), (64, 64, 1), (65, 64, 2), (640, 64, 10),
        (1 << 20, 1 << 20, 1), ((1 << 20) + 1, 1 << 20, 2), (0, 0, 1), (12345, 0, 1),
        (5 * 4096 - 1, 4096, 5),
    ],
)
def test_chunk_count(length, C, expected):
    assert oracle.chunk_count(length, C) == expected


@pytest.mark.parametrize("C", [1, 63, 65, 100, 4097])
def test_chunk_size_must_be_multiple_of_64(C):
    with pytest.raises(ValueError):
        oracle.chunk_count(1000, C)


@pytest.mark.parametrize("C", [64, 128, 4096, 0])
def test_chunk_digests_are_plain_sha256_of_slices(C):
    rng = np.random.default_rng(4)
    for n in (0, 1, 63, 64, 65, 4095, 4096, 4097, 3 * 4096 + 55):
        m = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        got = oracle.chunk_digests(m, C)
        if C == 0:
            want = [hashlib.sha256(m).digest()]
        else:
            want = [hashlib.sha256(m[i:i + C]).digest() for i in range(0, n, C)]
        assert [bytes(r) for r in got] == want, (n, C)
