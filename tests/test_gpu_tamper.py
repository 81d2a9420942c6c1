"""Tampering with resident weights changes the root, and the per-message roots
and leaf digests say where.

* Seeded single-bit flips anywhere in the set (chunk starts, ends and
  middles, first and last message): only the flipped chunk's leaf digest and
  its message's root change, the manifest root changes, and restoring the bit
  restores every value.
* Swapping two distinct chunks of a message swaps their leaf digests and
  changes the message root; swapping two messages changes the manifest.
Both hashes; every tampered result is also checked against the CPU oracle on the same bytes.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")
C = 4096
LENS = [20480, 4096 * 7 + 123, 1, 4096, 65536 + 9, 3 * 4096]


def messages(seed):
    return [W.random_bytes(L, seed + i, DEV) for i, L in enumerate(LENS)]


def state(v, msgs):
    roots, leaves, seg = v.roots(msgs, C)
    top = v.manifest_root(msgs, C)
    torch.cuda.synchronize()
    return leaves.clone(), roots.clone(), bytes(top.cpu().numpy().reshape(-1)), seg


def oracle_state(msgs, alg):
    host = [m.cpu().numpy() for m in msgs]
    leaves = oracle.leaf_digests_mt(host, C, 2, alg)
    counts = [oracle.chunk_count(len(h), C, alg) for h in host]
    roots = oracle.seg_roots_from_leaves(leaves, counts, alg)
    return leaves, roots, oracle.mth(roots, alg)


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_single_bit_flips_are_localised(alg):
    msgs = messages(1600)
    v = hv.Verifier(DEV, alg)
    leaves0, roots0, top0, seg = state(v, msgs)
    rng = np.random.default_rng(1601)
    picks = [(0, 0), (0, 4095), (0, 4096), (1, LENS[1] - 1), (2, 0), (4, 65536), (5, 3 * 4096 - 1)]
    picks += [(int(m), int(rng.integers(0, LENS[m]))) for m in rng.integers(0, len(LENS), 5)]
    for m, pos in picks:
        bit = int(rng.integers(0, 8))
        msgs[m][pos] ^= 1 << bit
        leaves, roots, top, _ = state(v, msgs)
        leaf = int(seg[m]) + pos // C
        tag = f"message {m}, byte {pos}, bit {bit}"
        assert top != top0, tag
        changed_leaves = np.nonzero((leaves != leaves0).any(dim=1).cpu().numpy())[0].tolist()
        assert changed_leaves == [leaf], tag
        mism = hv.hv_compare_roots(roots, roots0, alg=alg).cpu().numpy()
        assert np.nonzero(mism)[0].tolist() == [m], tag
        o_leaves, o_roots, o_top = oracle_state(msgs, alg)
        assert np.array_equal(leaves.cpu().numpy(), o_leaves) and top == o_top, tag
        msgs[m][pos] ^= 1 << bit
        leaves, roots, top, _ = state(v, msgs)
        assert torch.equal(leaves, leaves0) and torch.equal(roots, roots0) and top == top0, tag


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_swapped_chunks_and_messages_change_the_roots(alg):
    msgs = messages(1700)
    v = hv.Verifier(DEV, alg)
    leaves0, roots0, top0, seg = state(v, msgs)
    m, i, j = 1, 1, 5  # two distinct whole chunks of message 1
    a = msgs[m][i * C:(i + 1) * C].clone()
    msgs[m][i * C:(i + 1) * C] = msgs[m][j * C:(j + 1) * C]
    msgs[m][j * C:(j + 1) * C] = a
    leaves, roots, top, _ = state(v, msgs)
    li, lj = int(seg[m]) + i, int(seg[m]) + j
    assert torch.equal(leaves[li], leaves0[lj]) and torch.equal(leaves[lj], leaves0[li])
    assert np.nonzero(hv.hv_compare_roots(roots, roots0, alg=alg).cpu().numpy())[0].tolist() == [m]
    assert top != top0
    o_leaves, o_roots, o_top = oracle_state(msgs, alg)
    assert np.array_equal(leaves.cpu().numpy(), o_leaves) and top == o_top
    # two messages in the other order: same per-message roots, another manifest
    swapped = [msgs[0], msgs[3]] + msgs[2:3] + [msgs[1]] + msgs[4:]
    top_swapped = bytes(v.manifest_root(swapped, C).cpu().numpy().reshape(-1))
    assert top_swapped != top
    assert top_swapped == oracle_state(swapped, alg)[2]
