"""Property-based pins (hypothesis) over random shapes, all on the CPU:

* the oracle's chunk digests equal hashlib over each chunk slice, for random
  messages, chunk sizes (multiples of the block, or 0) and both hashes;
* the oracle's recursive RFC 6962 tree equals an independent bottom-up
  construction written here, for random entry lists of either digest size;
* the library's host-side leaf layout (hv_leaf_layout) equals the oracle's
  chunk counts for random message-length lists and chunk sizes.
"""
import hashlib

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import oracle

HASH = {"sha256": hashlib.sha256, "sha384": hashlib.sha384}
BLOCK = {"sha256": 64, "sha384": 128}


@settings(max_examples=60, deadline=None)
@given(alg=st.sampled_from(["sha256", "sha384"]), data=st.binary(min_size=0, max_size=3000),
       blocks=st.integers(min_value=0, max_value=6))
def test_chunk_digests_are_hashlib_of_slices(alg, data, blocks):
    C = blocks * BLOCK[alg]
    got = [bytes(r) for r in oracle.chunk_digests_alg(data, C, alg)]
    if C == 0:
        want = [HASH[alg](data).digest()]
    else:
        want = [HASH[alg](data[i:i + C]).digest() for i in range(0, len(data), C)]
    assert got == want


def bottom_up(entries, alg):
    H = lambda b: HASH[alg](b).digest()
    if not entries:
        return H(b"")
    level = [H(b"\x00" + e) for e in entries]
    while len(level) > 1:
        nxt = [H(b"\x01" + level[i] + level[i + 1]) for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


@settings(max_examples=60, deadline=None)
@given(alg=st.sampled_from(["sha256", "sha384"]), n=st.integers(min_value=0, max_value=300),
       seed=st.integers(min_value=0, max_value=2 ** 32 - 1))
def test_recursive_tree_equals_bottom_up(alg, n, seed):
    D = 32 if alg == "sha256" else 48
    rng = np.random.default_rng(seed)
    entries = [rng.integers(0, 256, D, dtype=np.uint8).tobytes() for _ in range(n)]
    assert oracle.mth(entries, alg) == bottom_up(entries, alg)


from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)


@settings(max_examples=80, deadline=None)
@given(lens=st.lists(st.integers(min_value=0, max_value=1 << 22), min_size=0, max_size=40),
       blocks=st.sampled_from([0, 1, 2, 3, 16, 1024, 16384]))
def test_leaf_layout_equals_oracle_chunk_counts(lens, blocks):
    C = 64 * blocks
    ptrs = np.array([0x10000 + 4096 * i if n else 0 for i, n in enumerate(lens)], dtype=np.uint64)
    seg, n_leaves = hv.hv_leaf_layout(ptrs, np.array(lens, dtype=np.uint64), C)
    counts = [oracle.chunk_count(n, C) for n in lens]
    assert n_leaves == sum(counts)
    assert list(seg) == [0] + list(np.cumsum(counts, dtype=np.int64))
