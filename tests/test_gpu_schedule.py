"""The device-side chunk scheduler: every chunk exactly once, with the
source range and leaf index Algorithm 1's chunking gives it, longest first.

Expected leaf lists are written here from the chunking rule (message m,
chunk i covers [i*C, min((i+1)*C, L)), leaves numbered message-major).
"""
import numpy as np
import pytest
import torch

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu


def expected_leaves(ptrs, lens, C):
    out, leaf = [], 0
    for p, L in zip(ptrs, lens):
        p, L = int(p), int(L)
        if C == 0:
            out.append((p, L, leaf)); leaf += 1
            continue
        for i in range(0, L, C):
            out.append((p + i, min(C, L - i), leaf)); leaf += 1
    return out


def blocks(nbytes):
    return (nbytes + 72) // 64


def sort_class(nblk):
    """Documented order key: exact below 2048 blocks, then 32 classes per octave."""
    if nblk < 2048:
        return nblk
    e = nblk.bit_length() - 1
    return 2048 + (e - 11) * 32 + ((nblk >> (e - 5)) & 31)


@pytest.mark.parametrize("C", [64, 4096, 65536, 0])
def test_schedule_is_a_sorted_permutation(C):
    rng = np.random.default_rng(5)
    lens = np.concatenate([[0, 1, 63, 64, 65, 55, 56, 4096, 65536, 65537, 200000],
                           rng.integers(0, 150000, 300)]).astype(np.uint64)
    buf = torch.empty(int(lens.sum()) + 64 * len(lens), dtype=torch.uint8, device="cuda")
    starts = np.concatenate([[0], np.cumsum(lens + 64)[:-1]]).astype(np.uint64)
    ptrs = np.uint64(buf.data_ptr()) + starts
    table = hv.hv_leaf_schedule((ptrs, lens), C)
    want = expected_leaves(ptrs, lens, C)
    assert table.shape == (len(want), 3)
    got = sorted(tuple(int(x) for x in r) for r in table)
    assert got == sorted(want)
    key = [sort_class(blocks(int(r[1]))) for r in table]
    assert all(a >= b for a, b in zip(key, key[1:])), "not longest-first"


def test_small_message_workload_schedule_is_sorted():
    import workloads as W

    lens = W.small_message_lengths(20000, seed=3)
    offs = W.packed_offsets(lens)
    buf = torch.empty(int(offs[-1] + lens[-1]), dtype=torch.uint8, device="cuda")
    ptrs = np.uint64(buf.data_ptr()) + offs
    table = hv.hv_leaf_schedule((ptrs, lens), 0)
    assert sorted(int(x) for x in table[:, 2]) == list(range(20000))
    assert np.array_equal(table[np.argsort(table[:, 2]), 0], ptrs)
    nblk = (table[:, 1] + 72) // 64
    assert np.all(nblk[:-1] >= nblk[1:])


def test_whole_message_classes_across_octaves():
    # C = 0 with lengths log-uniform from 1 byte to 32 MiB: tails fall in the
    # exact classes and in the quantised classes of many octaves above them
    rng = np.random.default_rng(11)
    lens = np.unique(np.exp(rng.uniform(0, np.log(32 << 20), 80)).astype(np.uint64))
    lens = np.concatenate([lens, [2047 * 64 - 72, 2048 * 64 - 72, 4096 * 64 - 72, 4097 * 64 - 72]]).astype(np.uint64)
    buf = torch.empty(int(lens.sum()) + 64 * len(lens), dtype=torch.uint8, device="cuda")
    starts = np.concatenate([[0], np.cumsum(lens + 64)[:-1]]).astype(np.uint64)
    ptrs = np.uint64(buf.data_ptr()) + starts
    table = hv.hv_leaf_schedule((ptrs, lens), 0)
    assert sorted(tuple(int(x) for x in r) for r in table) == sorted(expected_leaves(ptrs, lens, 0))
    key = [sort_class(blocks(int(r[1]))) for r in table]
    assert all(a >= b for a, b in zip(key, key[1:])), "not longest-first"
    assert len(set(key)) > 40  # many distinct classes exercised
