"""The binding refuses caller tensors the library would overrun or misread.

The C ABI trusts the pointers it is given, so the Python layer checks every
caller-supplied tensor first: a short, host-resident or non-contiguous
buffer raises ValueError before any call reaches the library (no kernel runs
on it).  Valid calls on the same data still give the oracle's values.
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


@pytest.fixture
def data():
    msgs = [W.random_bytes(10000, 1510, DEV), W.random_bytes(5000, 1511, DEV)]  # 3 + 2 chunks
    leaves, seg = hv.hv_hash_chunks(msgs, C)
    torch.cuda.synchronize()
    want = oracle.leaf_digests_mt([m.cpu().numpy() for m in msgs], C, 2)
    assert leaves.shape == (5, 32) and np.array_equal(leaves.cpu().numpy(), want)
    return msgs, leaves, seg


def test_hash_and_merkle_buffers(data):
    msgs, leaves, seg = data
    with pytest.raises(ValueError, match="out holds"):
        hv.hv_hash_chunks(msgs, C, out=torch.empty((4, 32), dtype=torch.uint8, device=DEV))
    with pytest.raises(ValueError, match="device tensor"):
        hv.hv_hash_chunks(msgs, C, out=torch.empty((5, 32), dtype=torch.uint8))
    with pytest.raises(ValueError, match="nodes holds"):
        hv.hv_merkle_reduce(leaves[:4], seg)
    with pytest.raises(ValueError, match="contiguous"):
        hv.hv_merkle_reduce(leaves.t(), seg)
    with pytest.raises(ValueError, match="out holds"):
        hv.hv_merkle_reduce(leaves, seg, out=torch.empty((1, 32), dtype=torch.uint8, device=DEV))
    with pytest.raises(ValueError, match="one segment"):
        hv.hv_merkle_reduce(leaves, np.array([0], dtype=np.uint64))
    with pytest.raises(ValueError, match="root holds"):
        hv.hv_verify_root(leaves[0, :16], bytes(32))
    with pytest.raises(ValueError, match="contiguous"):
        hv.hv_compare_roots(leaves.t().contiguous().t(), leaves)
    # the same calls with whole buffers
    out = torch.empty((5, 32), dtype=torch.uint8, device=DEV)
    got, _ = hv.hv_hash_chunks(msgs, C, out=out)
    roots = hv.hv_merkle_reduce(got, seg)
    torch.cuda.synchronize()
    host = leaves.cpu().numpy()
    assert [bytes(r) for r in roots.cpu().numpy()] == oracle.seg_roots_from_leaves(host, np.diff(seg))


def test_incremental_and_monitor_buffers(data):
    msgs, leaves, seg = data
    with pytest.raises(ValueError, match="leaf_digests holds"):
        hv.hv_rehash_chunks(msgs, C, [0], leaves[:4])
    with pytest.raises(ValueError, match="leaf_digests holds"):
        hv.Tree(leaves[:4], seg)
    with pytest.raises(ValueError, match="roots holds"):
        hv.Tree(leaves, seg, roots=torch.empty((1, 32), dtype=torch.uint8, device=DEV))
    tree = hv.Tree(leaves, seg)
    with pytest.raises(ValueError, match="leaf_digests holds"):
        tree.update(leaves[:2], [0])
    with pytest.raises(ValueError, match="uint8"):
        hv.Monitor(msgs, C, leaves.to(torch.int32), device=DEV)
    mon = hv.Monitor(msgs, C, leaves, slice_leaves=5, device=DEV)
    with pytest.raises(ValueError, match="slice_digests holds"):
        mon.scan(0, 5, torch.empty((4, 32), dtype=torch.uint8, device=DEV))
    out = torch.empty((5, 32), dtype=torch.uint8, device=DEV)
    mon.scan(0, 5, out)
    mon.poll(wait=True)
    assert mon.mismatches == [] and torch.equal(out, leaves)


def test_pipeline_replay_needs_a_capture_and_empty_verify(data):
    msgs, leaves, seg = data
    pipe = hv.Pipeline(msgs, C, "manifest", DEV)
    with pytest.raises(RuntimeError, match="capture"):
        pipe.replay()
    # an empty set has the empty manifest: RFC 6962's hash of no entries
    hv.verify({}, oracle.mth([]), C)
    with pytest.raises(hv.VerificationError):
        hv.verify({}, bytes(32), C)
