"""Continuous runtime monitoring (include/hv_monitor.h) against the CPU oracle.

The reference digests a monitor compares with are the oracle's digests of the
untouched bytes.  A clean scan must report no mismatch and leave digests equal
to the oracle's, bit for bit; after bytes are changed on the device, every
scan's mismatch count and lowest mismatching leaf must equal what the oracle's
digests of the changed bytes say, slice by slice.  At the full 70B shape: a
sweep of the untouched set finds nothing, a one-byte change anywhere is found
at exactly the leaf that holds it, and sampled slices match the oracle.
"""
import ctypes
import gc
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
U64_MAX = (1 << 64) - 1


def threads():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def expected_scan(want, ref, first, count):
    """(mismatch count, lowest mismatching leaf or U64_MAX) of leaves [first, first + count)."""
    bad = np.nonzero((want[first:first + count] != ref[first:first + count]).any(axis=1))[0]
    return (len(bad), first + int(bad[0])) if len(bad) else (0, U64_MAX)


def read(res):
    c, f = (int(v) for v in res.cpu().tolist())
    return c, f & U64_MAX


@pytest.mark.parametrize("alg,C,align_off", [("sha256", 4096, 0), ("sha256", 64, 3), ("sha256", 0, 1),
                                             ("sha384", 4096, 0), ("sha384", 128, 15), ("sha384", 0, 0)])
def test_clean_scans_and_changed_chunks(alg, C, align_off):
    rng = np.random.default_rng(900)
    lens = np.concatenate([rng.integers(0, 20000, 120), [0, 1, 4096, 4097, 65536 + 5]])
    buf, host, ptrs, lens, starts = place(lens, align_off, seed=901)
    msgs = host_msgs(host, starts, lens)
    ref_np = oracle.leaf_digests_mt(msgs, C, threads(), alg)
    ref = torch.from_numpy(ref_np).to(DEV)
    D = ref.shape[1]
    mon = hv.Monitor((ptrs, lens), C, ref, alg=alg, slice_leaves=37, device=DEV)
    n = mon.n_leaves
    assert n == len(ref_np)
    # clean: every slice reports nothing, and its digests are the oracle's
    out = torch.empty((n, D), dtype=torch.uint8, device=DEV)
    for first in range(0, n, 37):
        k = min(37, n - first)
        res = mon.scan(first, k, out[first:first + k])
        torch.cuda.synchronize()
        assert read(res) == (0, U64_MAX)
    assert np.array_equal(out.cpu().numpy(), ref_np)
    # change a few bytes on the device (and in the host copy the oracle reads)
    nz = np.nonzero(lens)[0]
    for m in rng.choice(nz, 5, replace=False):
        off = int(starts[m]) + int(rng.integers(0, int(lens[m])))
        host[off] ^= 0x5A
        buf[off] ^= 0x5A
    torch.cuda.synchronize()  # the changes land before the monitor stream reads them
    want = oracle.leaf_digests_mt(host_msgs(host, starts, lens), C, threads(), alg)
    assert (want != ref_np).any(axis=1).sum() >= 1
    mon.sweep()
    mon.poll(wait=True)
    got = {(s0, k): (cnt, fb) for fb, cnt, s0, k in mon.mismatches}
    for first in range(0, n, mon.slice):
        k = min(mon.slice, n - first)
        e = expected_scan(want, ref_np, first, k)
        assert got.get((first, k), (0, U64_MAX)) == e, (first, k)
    assert sum(c for c, _ in got.values()) == int((want != ref_np).any(axis=1).sum())


def test_empty_and_boundary_slices():
    lens = np.array([5000, 0, 130], dtype=np.uint64)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=902)
    ref_np = oracle.leaf_digests_mt(host_msgs(host, starts, lens), 1024, 1)
    ref = torch.from_numpy(ref_np).to(DEV)
    mon = hv.Monitor((ptrs, lens), 1024, ref, slice_leaves=4, device=DEV)
    assert mon.n_leaves == 6
    res = mon.scan(6, 0)  # empty slice at the end: resets the result
    torch.cuda.synchronize()
    assert read(res) == (0, U64_MAX)
    res = mon.scan(5, 1)  # the last leaf (the 130-byte message)
    torch.cuda.synchronize()
    assert read(res) == (0, U64_MAX)
    bad = ref.clone()
    bad[3, 7] ^= 1
    bad[5, 0] ^= 1
    mon2 = hv.Monitor((ptrs, lens), 1024, bad, slice_leaves=6, device=DEV)
    res = mon2.scan(0, 6)
    torch.cuda.synchronize()
    assert read(res) == (2, 3)
    with pytest.raises(hv.HVError):
        mon.scan(5, 2)
    with pytest.raises(ValueError):
        hv.Monitor((ptrs, lens), 1024, ref[:5], device=DEV)


def test_monitor_stream_runs_beside_other_work():
    # scans queued on the monitor stream while the current stream is busy with
    # matmuls; results arrive through the pinned ring without touching it
    lens = np.full(64, 1 << 16, dtype=np.uint64)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=903)
    ref = torch.from_numpy(oracle.leaf_digests_mt(host_msgs(host, starts, lens), 4096, threads())).to(DEV)
    mon = hv.Monitor((ptrs, lens), 4096, ref, slice_leaves=100, device=DEV, ring=4)
    a = torch.randn(2048, 2048, device=DEV)
    for _ in range(3):
        for _ in range(5):
            a = torch.tanh(a @ a) * 0.5
        for _ in range(3):
            mon.step()
    mon.poll(wait=True)
    torch.cuda.synchronize()
    assert mon.read == mon.issued == 9 and mon.mismatches == []


@pytest.fixture(scope="module")
def w70b_monitor():
    wl = W.workload(5, DEV)
    pipe = hv.Pipeline(wl.msgs, wl.chunk_bytes, "manifest", DEV)
    root = bytes(pipe.compute().cpu().numpy().reshape(-1))
    torch.cuda.synchronize()
    yield wl, pipe, root
    del wl, pipe
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_70b_sweep_finds_nothing_then_exactly_the_changed_chunk(w70b_monitor):
    wl, pipe, root = w70b_monitor
    C = wl.chunk_bytes
    mon = hv.Monitor(wl.msgs, C, pipe.leaves, slice_leaves=16384, device=DEV)
    assert mon.n_leaves == pipe.n_leaves == 2_153_249
    mon.sweep()
    mon.poll(wait=True)
    assert mon.mismatches == [] and mon.read == -(-mon.n_leaves // 16384)
    # sampled slices: fresh digests against the oracle over host copies of those chunks
    rng = np.random.default_rng(W.seed_of(5) + 7)
    seg = pipe.seg
    for first in rng.integers(0, mon.n_leaves - 64, 3):
        first = int(first)
        out = torch.empty((64, 32), dtype=torch.uint8, device=DEV)
        mon.scan(first, 64, out)
        mon.poll(wait=True)
        want = []
        for leaf in range(first, first + 64):
            m = int(np.searchsorted(seg, leaf, side="right")) - 1
            i = leaf - int(seg[m])
            v = wl.msgs.views[m]
            chunk = v[i * C:min((i + 1) * C, v.numel())].cpu().numpy()
            want.append(oracle.sha256(chunk))
        assert [bytes(r) for r in out.cpu().numpy()] == want
    # one changed byte is found at the leaf that holds it, and only there
    total = int(wl.msgs.lens.sum())
    pos = int(rng.integers(0, total))
    ends = np.cumsum(wl.msgs.lens.astype(np.int64))
    m = int(np.searchsorted(ends, pos, side="right"))
    off = pos - (int(ends[m - 1]) if m else 0)
    leaf = int(seg[m]) + off // C
    view = wl.msgs.views[m]
    old = int(view[off].item())
    view[off] = old ^ 0x01
    torch.cuda.synchronize()
    try:
        mon.mismatches.clear()
        mon.sweep()
        mon.poll(wait=True)
        assert [(fb, cnt) for fb, cnt, _, _ in mon.mismatches] == [(leaf, 1)]
    finally:
        view[off] = old
        torch.cuda.synchronize()
    mon.mismatches.clear()
    mon.scan(leaf - leaf % 16384, min(16384, mon.n_leaves - (leaf - leaf % 16384)))
    mon.poll(wait=True)
    assert mon.mismatches == []


def test_cu_masked_raw_stream_scan_then_destroy():
    # a masked stream used only through the C ABI (no torch event ever
    # recorded on it): one scan, then the stream is destroyed, which also
    # frees its hardware queue for the next test
    n_cu = torch.cuda.get_device_properties(DEV).multi_processor_count
    lens = np.full(8, 20_000, dtype=np.uint64)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=905)
    ref_np = oracle.leaf_digests_mt(host_msgs(host, starts, lens), 4096, 1)
    ref = torch.from_numpy(ref_np).to(DEV)
    arr = hv._msg_array(ptrs, lens)
    plan = hv.hv_monitor_plan()
    plan_mem = hv.Workspace(DEV).get(hv.lib.hv_monitor_plan_bytes(len(arr)))
    n = len(ref_np)
    ws = hv.Workspace(DEV).get(hv.lib.hv_monitor_scan_workspace_bytes(0, n))
    out = torch.empty_like(ref)
    result = torch.empty(2, dtype=torch.int64, device=DEV)
    torch.cuda.synchronize()
    words = hv.cu_mask_words(range(0, 8), n_cu)
    handle = ctypes.c_void_p()
    hv._check(hv.lib.hv_stream_create_cu_masked(words.ctypes.data, len(words), ctypes.byref(handle)))
    hv._check(hv.lib.hv_monitor_init(0, arr.ctypes.data, len(arr), 4096, plan_mem.data_ptr(), plan_mem.numel(),
                                     ctypes.byref(plan), handle))
    hv._check(hv.lib.hv_monitor_scan(ctypes.byref(plan), 0, n, ref.data_ptr(), out.data_ptr(), result.data_ptr(),
                                     ws.data_ptr(), ws.numel(), handle))
    hv._check(hv.lib.hv_stream_destroy(handle))  # waits for the scan first
    assert read(result) == (0, U64_MAX)
    assert np.array_equal(out.cpu().numpy(), ref_np)


def test_cu_masked_streams_with_torch():
    n_cu = torch.cuda.get_device_properties(DEV).multi_processor_count
    with pytest.raises(hv.HVError):
        hv.CuMaskedStream([], DEV)  # a mask with no CU is refused before any stream exists
    # each masked stream holds a hardware queue of its own, and a process gets
    # few of those: two at a time here, closed before the next two are made
    mon_s = hv.CuMaskedStream(range(0, 8), DEV)
    rest = hv.CuMaskedStream(range(8, n_cu), DEV)
    assert list(mon_s.mask()) == list(hv.cu_mask_words(range(8), n_cu))
    assert list(rest.mask()) == list(hv.cu_mask_words(range(8, n_cu), n_cu))
    lens = np.full(40, 70_000, dtype=np.uint64)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=904)
    ref_np = oracle.leaf_digests_mt(host_msgs(host, starts, lens), 4096, threads())
    ref = torch.from_numpy(ref_np).to(DEV)
    mon = hv.Monitor((ptrs, lens), 4096, ref, slice_leaves=256, device=DEV, stream=mon_s)
    out = torch.empty_like(ref)
    a = torch.randn(1024, 1024, device=DEV)
    want = a @ a
    torch.cuda.synchronize()
    for first in range(0, mon.n_leaves, 256):
        k = min(256, mon.n_leaves - first)
        mon.scan(first, k, out[first:first + k])
    with torch.cuda.stream(rest.stream):
        got = a @ a
    mon.poll(wait=True)
    rest.stream.synchronize()
    assert mon.mismatches == [] and np.array_equal(out.cpu().numpy(), ref_np)
    assert torch.allclose(got, want, rtol=1e-5, atol=1e-4)
    # ordered teardown: the monitor made on the stream is closed with it
    mon_s.close()
    rest.close()
    mon_s.close()  # idempotent
    assert mon_s.handle is None and rest.handle is None
    with pytest.raises(RuntimeError):
        mon.scan(0, 1)
    # their hardware queues are free again: a second pair is made, used, and closed on leaving the block
    with hv.CuMaskedStream(range(0, 8), DEV) as s2, hv.CuMaskedStream(range(8, n_cu), DEV) as s3:
        mon2 = hv.Monitor((ptrs, lens), 4096, ref, slice_leaves=512, device=DEV, stream=s2)
        mon2.sweep()
        with torch.cuda.stream(s3.stream):
            got2 = a @ a
        mon2.poll(wait=True)
        s3.stream.synchronize()
        assert mon2.mismatches == [] and mon2.read == -(-mon2.n_leaves // 512)
        assert torch.allclose(got2, want, rtol=1e-5, atol=1e-4)
    assert s2.handle is None and s3.handle is None and mon2.events is None
