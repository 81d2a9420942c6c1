"""The C-ABI library loads, exports what include/hv.h declares, and its
host-side planning and argument checks behave as documented.

These run without a GPU: every call here either is host-only (hv_leaf_layout,
the *_workspace_bytes sizers, hv_last_error) or fails validation before the
library issues any HIP call.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)


def declared_functions():
    import glob

    text = "".join(open(f).read() for f in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))))
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hv_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 12
    lib = ctypes.CDLL(hv.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(hv.EXPORTS) == names


def test_kernel_round_constants_match_their_definition():
    # the HIP source's own tables, re-derived from primes (FIPS 180-4 4.2.2, 5.3.3)
    from test_oracle_sha256 import first_primes, iroot

    src = open(os.path.join(ROOT, "paper_2510_23938_amd", "csrc", "sha256_device.h")).read()
    k_body = re.search(r"kRound\[64\]\s*=\s*\{(.*?)\};", src, re.S).group(1)
    h_body = re.search(r"kInit\[8\]\s*=\s*\{(.*?)\};", src, re.S).group(1)
    K = [int(x, 16) for x in re.findall(r"0x([0-9a-fA-F]+)u", k_body)]
    H = [int(x, 16) for x in re.findall(r"0x([0-9a-fA-F]+)u", h_body)]
    p = first_primes(64)
    assert K == [iroot(q << 96, 3) & 0xFFFFFFFF for q in p]
    assert H == [iroot(q << 64, 2) & 0xFFFFFFFF for q in p[:8]]


def _msgs(lens, base=0x10000):
    ptrs = np.array([base + 4096 * i if n else 0 for i, n in enumerate(lens)], dtype=np.uint64)
    return ptrs, np.array(lens, dtype=np.uint64)


@pytest.mark.parametrize("C", [64, 128, 4096, 1 << 20, 0])
def test_leaf_layout_matches_oracle_chunk_count(C):
    lens = [0, 1, 63, 64, 65, 4095, 4096, 4097, 3 * 4096, (1 << 20) + 5, 12345678]
    seg, n = hv.hv_leaf_layout(*_msgs(lens), C)
    counts = [oracle.chunk_count(x, C) for x in lens]
    assert n == sum(counts)
    assert list(seg) == list(np.concatenate([[0], np.cumsum(counts)]))


@pytest.mark.parametrize("C", [1, 32, 100, 65])
def test_bad_chunk_size_rejected(C):
    with pytest.raises(hv.HVError) as e:
        hv.hv_leaf_layout(*_msgs([100]), C)
    assert e.value.status == hv.HV_ERR_INVALID_ARG
    assert "multiple of 64" in str(e.value)


def test_null_data_with_bytes_rejected():
    ptrs = np.array([0x1000, 0], dtype=np.uint64)
    lens = np.array([10, 5], dtype=np.uint64)
    with pytest.raises(hv.HVError) as e:
        hv.hv_leaf_layout(ptrs, lens, 64)
    assert e.value.status == hv.HV_ERR_INVALID_ARG and "message 1" in str(e.value)


def test_chunk_size_limit():
    big = 1 << 37
    ptrs = np.array([0x1000], dtype=np.uint64)
    assert hv.hv_leaf_layout(ptrs, np.array([big], dtype=np.uint64), 0)[1] == 1
    assert hv.hv_leaf_layout(ptrs, np.array([1 << 40], dtype=np.uint64), 1 << 20)[1] == 1 << 20
    assert hv.hv_leaf_layout(ptrs, np.array([1 << 40], dtype=np.uint64), big)[1] == 8
    for lens, C in (([big + 1], 0), ([1 << 39], 1 << 38), ([big + 64], big + 64)):
        with pytest.raises(hv.HVError) as e:
            hv.hv_leaf_layout(ptrs, np.array(lens, dtype=np.uint64), C)
        assert e.value.status == hv.HV_ERR_INVALID_ARG and "limit" in str(e.value)


def test_leaf_count_limit():
    # 2^31 leaves per call at most; every check below fails before any HIP call
    ptrs = np.array([0x1000], dtype=np.uint64)
    arr = hv._msg_array(ptrs, np.array([(1 << 31) * 64 + 64], dtype=np.uint64))
    st = hv.lib.hv_hash_chunks(arr.ctypes.data, 1, 64, 0x1000, 0x100000, 1 << 40, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"limit" in hv.lib.hv_last_error()
    assert hv.lib.hv_plan_bytes(hv.HV_SHA256, arr.ctypes.data, 1, 64, 1) == 0
    seg = np.array([0, (1 << 31) + 1], dtype=np.uint64)
    st = hv.lib.hv_merkle_reduce(0x1000, seg.ctypes.data, 1, 0x1000, 0x100000, 1 << 40, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"limit" in hv.lib.hv_last_error()
    assert hv.lib.hv_tree_bytes(seg.ctypes.data, 1) == 0
    assert hv.lib.hv_hash_workspace_bytes(1, (1 << 31) + 1) == 0 and hv.lib.hv_hash_workspace_bytes(1, 1 << 31) > 0
    assert hv.lib.hv_merkle_workspace_bytes((1 << 31) + 1, 1) == 0
    assert hv.lib.hv_monitor_scan_workspace_bytes(0, 1 << 62) == 0 and b"limit" in hv.lib.hv_last_error()
    seg[1] = 1 << 31
    assert hv.lib.hv_tree_bytes(seg.ctypes.data, 1) > 0


def test_null_n_leaves_and_msgs_rejected():
    assert hv.lib.hv_leaf_layout(None, 3, 64, None, None) == hv.HV_ERR_INVALID_ARG
    n = ctypes.c_uint64(0)
    assert hv.lib.hv_leaf_layout(None, 3, 64, None, ctypes.byref(n)) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_leaf_layout(None, 0, 64, None, ctypes.byref(n)) == hv.HV_OK and n.value == 0


def test_workspace_sizes_grow_and_are_aligned():
    a = hv.lib.hv_hash_workspace_bytes(10, 100)
    b = hv.lib.hv_hash_workspace_bytes(10, 100000)
    assert b > a and a % 256 == 0 and b % 256 == 0
    assert hv.lib.hv_hash_workspace_bytes(1_000_000, 1_000_000) >= 1_000_000 * (16 + 24)
    m1 = hv.lib.hv_merkle_workspace_bytes(1000, 1)
    m2 = hv.lib.hv_merkle_workspace_bytes(10_000_000, 723)
    assert m2 > m1 and m1 % 256 == 0
    assert hv.lib.hv_verify_workspace_bytes() >= 4


def test_hash_rejects_before_launch():
    # every one of these fails validation before any HIP call
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    p = arr.ctypes.data
    st = hv.lib.hv_hash_chunks(p, 2, 100, 0x1000, 0x100000, 1 << 30, None)
    assert st == hv.HV_ERR_INVALID_ARG
    st = hv.lib.hv_hash_chunks(p, 2, 64, None, 0x100000, 1 << 30, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"leaf_digests" in hv.lib.hv_last_error()
    st = hv.lib.hv_hash_chunks(p, 2, 64, 0x1008, 0x100000, 1 << 30, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"aligned" in hv.lib.hv_last_error()
    st = hv.lib.hv_hash_chunks(p, 2, 64, 0x1000, 0x100000, 16, None)
    assert st == hv.HV_ERR_WORKSPACE
    st = hv.lib.hv_hash_chunks(p, 2, 64, 0x1000, None, 1 << 30, None)
    assert st == hv.HV_ERR_WORKSPACE


def test_merkle_rejects_before_launch():
    seg = np.array([0, 5, 3], dtype=np.uint64)  # decreasing
    st = hv.lib.hv_merkle_reduce(0x1000, seg.ctypes.data, 2, 0x2000, 0x100000, 1 << 20, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"decreases" in hv.lib.hv_last_error()
    seg = np.array([1, 5], dtype=np.uint64)
    assert hv.lib.hv_merkle_reduce(0x1000, seg.ctypes.data, 1, 0x2000, 0x100000, 1 << 20, None) == \
        hv.HV_ERR_INVALID_ARG
    seg = np.array([0, 5], dtype=np.uint64)
    assert hv.lib.hv_merkle_reduce(0x1000, seg.ctypes.data, 0, 0x2000, 0x100000, 1 << 20, None) == \
        hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_merkle_reduce(None, seg.ctypes.data, 1, 0x2000, 0x100000, 1 << 20, None) == \
        hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_merkle_reduce(0x1000, seg.ctypes.data, 1, 0x2000, 0x100000, 8, None) == hv.HV_ERR_WORKSPACE


def test_verify_rejects_before_launch():
    exp = (ctypes.c_uint8 * 32)()
    m = ctypes.c_int(0)
    assert hv.lib.hv_verify_root(None, exp, ctypes.byref(m), 0x1000, 256, None) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_verify_root(0x1000, exp, ctypes.byref(m), None, 256, None) == hv.HV_ERR_WORKSPACE
    assert hv.lib.hv_verify_root(0x1000, exp, ctypes.byref(m), 0x1002, 256, None) == hv.HV_ERR_WORKSPACE
    assert b"aligned" in hv.lib.hv_last_error()
    assert hv.lib.hv_compare_roots(None, None, 3, None, None) == hv.HV_ERR_INVALID_ARG


def test_stream_plan_sizes_and_rejections():
    ptrs, lens = _msgs([1 << 20, 100, 0])
    arr = hv._msg_array(ptrs, lens)
    ok = hv.lib.hv_stream_workspace_bytes(arr.ctypes.data, 3, 65536, 1 << 20)
    assert ok >= 2 << 20 and ok % 256 == 0
    assert hv.lib.hv_stream_workspace_bytes(arr.ctypes.data, 3, 65536, 1000) == 0      # not a multiple of 256
    assert b"multiple of 256" in hv.lib.hv_last_error()
    assert hv.lib.hv_stream_workspace_bytes(arr.ctypes.data, 3, 0, 1 << 19) == 0       # whole message > batch
    assert b"does not fit" in hv.lib.hv_last_error()
    assert hv.lib.hv_stream_workspace_bytes(arr.ctypes.data, 3, 100, 1 << 20) == 0     # bad chunk size


def test_incremental_rejects_before_launch():
    seg = np.array([0, 10, 30], dtype=np.uint64)
    assert hv.lib.hv_tree_bytes(seg.ctypes.data, 2) > 0
    assert hv.lib.hv_tree_bytes(np.array([1, 2], dtype=np.uint64).ctypes.data, 1) == 0
    for bad in ([3, 2], [5, 30], [4, 4]):
        d = np.array(bad, dtype=np.uint64)
        st = hv.lib.hv_tree_update(0x1000, seg.ctypes.data, 2, 0x100000, 1 << 20, d.ctypes.data, 2, 0x2000,
                                   0x200000, 1 << 20, None)
        assert st == hv.HV_ERR_INVALID_ARG
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    d = np.array([1, 0], dtype=np.uint64)
    st = hv.lib.hv_rehash_chunks(arr.ctypes.data, 2, 64, d.ctypes.data, 2, 0x2000, 0x200000, 1 << 20, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"increasing" in hv.lib.hv_last_error()


def test_timing_query_without_timed_call():
    with pytest.raises(hv.HVError):
        hv.leaf_kernel_ms()


def test_sha384_kernel_constants_match_their_definition():
    # the SHA-384 tables of the HIP source, re-derived from primes (FIPS 180-4 4.2.3, 5.3.4)
    from test_oracle_sha256 import first_primes, iroot

    src = open(os.path.join(ROOT, "paper_2510_23938_amd", "csrc", "sha384_device.h")).read()
    k_body = re.search(r"kRound512\[80\]\s*=\s*\{(.*?)\};", src, re.S).group(1)
    h_body = re.search(r"kInit384\[8\]\s*=\s*\{(.*?)\};", src, re.S).group(1)
    K = [int(x, 16) for x in re.findall(r"0x([0-9a-fA-F]+)ull", k_body)]
    H = [int(x, 16) for x in re.findall(r"0x([0-9a-fA-F]+)ull", h_body)]
    p = first_primes(80)
    assert K == [iroot(q << 192, 3) & ((1 << 64) - 1) for q in p]
    assert H == [iroot(q << 128, 2) & ((1 << 64) - 1) for q in p[8:16]]


def test_alg_entry_points_reject_before_launch():
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    p = arr.ctypes.data
    for bad in (2, -1):
        assert hv.lib.hv_hash_chunks_alg(bad, p, 2, 64, 0x1000, 0x100000, 1 << 30, None) == hv.HV_ERR_INVALID_ARG
        assert b"unknown algorithm" in hv.lib.hv_last_error()
        assert hv.lib.hv_merkle_workspace_bytes_alg(bad, 100, 1) == 0
        seg = np.array([0, 5], dtype=np.uint64)
        assert hv.lib.hv_merkle_reduce_alg(bad, 0x1000, seg.ctypes.data, 1, 0x2000, 0x100000, 1 << 20, None) == \
            hv.HV_ERR_INVALID_ARG
        exp = (ctypes.c_uint8 * 48)()
        m = ctypes.c_int(0)
        assert hv.lib.hv_verify_root_alg(bad, 0x1000, exp, ctypes.byref(m), 0x1000, 256, None) == \
            hv.HV_ERR_INVALID_ARG
        assert hv.lib.hv_compare_roots_alg(bad, 0x1000, 0x2000, 1, 0x3000, None) == hv.HV_ERR_INVALID_ARG
    # SHA-384 chunks must be whole 128-byte blocks
    for C in (64, 192, 4096 + 64):
        st = hv.lib.hv_hash_chunks_alg(hv.HV_SHA384, p, 2, C, 0x1000, 0x100000, 1 << 30, None)
        assert st == hv.HV_ERR_INVALID_ARG and b"multiple of 128" in hv.lib.hv_last_error()
    # the SHA-256 form of the same call takes C = 64 and fails only at its workspace check
    assert hv.lib.hv_hash_chunks_alg(hv.HV_SHA256, p, 2, 64, 0x1000, 0x100000, 16, None) == hv.HV_ERR_WORKSPACE
    # SHA-384 Merkle workspace covers 48-byte nodes
    assert hv.lib.hv_merkle_workspace_bytes_alg(hv.HV_SHA384, 1 << 20, 3) > \
        hv.lib.hv_merkle_workspace_bytes_alg(hv.HV_SHA256, 1 << 20, 3)
    assert hv.lib.hv_merkle_workspace_bytes_alg(hv.HV_SHA256, 1 << 20, 3) == hv.lib.hv_merkle_workspace_bytes(1 << 20, 3)


def test_binding_checks_root_sizes():
    with pytest.raises(ValueError):
        hv._alg("sha512")
    assert hv.ALGS["sha384"][1] == 48 and hv.ALGS["sha256"][1] == 32


def test_monitor_rejects_before_launch():
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    p = arr.ctypes.data
    plan = hv.hv_monitor_plan()
    need = hv.lib.hv_monitor_plan_bytes(2)
    assert need >= 2 * 16 and need % 256 == 0
    assert hv.lib.hv_monitor_init(5, p, 2, 64, 0x100000, need, ctypes.byref(plan), None) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_monitor_init(0, p, 2, 64, 0x100000, need, None, None) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_monitor_init(0, p, 2, 100, 0x100000, need, ctypes.byref(plan), None) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_monitor_init(1, p, 2, 64, 0x100000, need, ctypes.byref(plan), None) == hv.HV_ERR_INVALID_ARG
    assert b"multiple of 128" in hv.lib.hv_last_error()
    assert hv.lib.hv_monitor_init(0, p, 2, 64, 0x100000, need - 1, ctypes.byref(plan), None) == hv.HV_ERR_WORKSPACE
    assert hv.lib.hv_monitor_init(0, p, 2, 64, 0x100010, need, ctypes.byref(plan), None) == hv.HV_ERR_WORKSPACE
    # scans of a plan filled by hand (never dereferenced: every case fails validation)
    plan = hv.hv_monitor_plan(0x100000, 0, 2, 64, 17)
    ws = hv.lib.hv_monitor_scan_workspace_bytes(0, 17)
    assert ws >= 17 * (24 + 32) and hv.lib.hv_monitor_scan_workspace_bytes(1, 17) > ws
    assert hv.lib.hv_monitor_scan_workspace_bytes(2, 17) == 0 and b"unknown algorithm" in hv.lib.hv_last_error()
    scan = lambda pl, first, n, ref=0x200000, out=None, res=0x300000, w=0x400000, wb=ws: \
        hv.lib.hv_monitor_scan(pl, first, n, ref, out, res, w, wb, None)
    assert scan(None, 0, 1) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(hv.hv_monitor_plan(None, 0, 2, 64, 17)), 0, 1) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(hv.hv_monitor_plan(0x100000, 7, 2, 64, 17)), 0, 1) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 10, 8) == hv.HV_ERR_INVALID_ARG and b"not within" in hv.lib.hv_last_error()
    assert scan(ctypes.byref(plan), 18, 0) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 1, 2 ** 64 - 1) == hv.HV_ERR_INVALID_ARG   # no wrap-around
    assert scan(ctypes.byref(plan), 0, 1, res=None) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 0, 1, res=0x300004) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 0, 1, ref=None) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 0, 1, ref=0x200008) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 0, 1, out=0x500004) == hv.HV_ERR_INVALID_ARG
    assert scan(ctypes.byref(plan), 0, 17, wb=ws - 1) == hv.HV_ERR_WORKSPACE
    assert scan(ctypes.byref(plan), 0, 17, w=0x400040) == hv.HV_ERR_WORKSPACE
    assert scan(ctypes.byref(plan), 0, 17, w=None) == hv.HV_ERR_WORKSPACE


def test_plan_rejects_before_launch():
    ptrs, lens = _msgs([1000, 64, 0])
    arr = hv._msg_array(ptrs, lens)
    p = arr.ctypes.data
    b = hv.lib.hv_plan_bytes(0, p, 3, 64, 1)
    assert b > 0 and b % 256 == 0
    assert hv.lib.hv_plan_bytes(1, p, 3, 128, 1) >= hv.lib.hv_plan_bytes(0, p, 3, 128, 1)  # 48-byte nodes
    assert hv.lib.hv_plan_bytes(0, p, 3, 64, 0) > 0
    assert hv.lib.hv_plan_bytes(0, None, 0, 64, 1) > 0                  # an empty set is a plan too
    assert hv.lib.hv_plan_bytes(3, p, 3, 64, 1) == 0 and b"unknown algorithm" in hv.lib.hv_last_error()
    assert hv.lib.hv_plan_bytes(0, p, 3, 100, 1) == 0
    assert hv.lib.hv_plan_bytes(1, p, 3, 64, 1) == 0 and b"multiple of 128" in hv.lib.hv_last_error()
    plan = hv.hv_verify_plan()
    init = lambda *a: hv.lib.hv_plan_init(*a, None)
    assert init(0, p, 3, 64, 1, 0x100000, b, None) == hv.HV_ERR_INVALID_ARG
    assert init(0, p, 3, 64, 1, 0x100000, b - 1, ctypes.byref(plan)) == hv.HV_ERR_WORKSPACE
    assert init(0, p, 3, 64, 1, 0x100080, b, ctypes.byref(plan)) == hv.HV_ERR_WORKSPACE
    assert init(0, p, 3, 64, 1, None, b, ctypes.byref(plan)) == hv.HV_ERR_WORKSPACE
    # runs of hand-filled plans that fail validation before any launch
    good = dict(device=0x100000, bytes=1 << 20, alg=0, manifest=1, n_msgs=3, n_seg=3, chunk_bytes=64, n_leaves=17)
    run = lambda pl, leaves=0x200000, roots=0x300000, root=0x400000, exp=None, match=None: \
        hv.lib.hv_plan_run(ctypes.byref(pl) if pl is not None else None, leaves, roots, root, exp, match, None)

    def mk(**kw):
        d = dict(good)
        d.update(kw)
        pl = hv.hv_verify_plan()
        for k, v in d.items():
            setattr(pl, k, v)
        pl.launches[0] = pl.launches[1] = 1
        return pl
    assert run(None) == hv.HV_ERR_INVALID_ARG
    assert run(mk(device=None)) == hv.HV_ERR_INVALID_ARG
    assert run(mk(alg=9)) == hv.HV_ERR_INVALID_ARG
    bad = mk()
    bad.launches[0] = 9
    assert run(bad) == hv.HV_ERR_INVALID_ARG and b"corrupt" in hv.lib.hv_last_error()
    assert run(mk(bytes=256)) == hv.HV_ERR_INVALID_ARG and b"corrupt" in hv.lib.hv_last_error()
    assert run(mk(), leaves=None) == hv.HV_ERR_INVALID_ARG
    assert run(mk(), roots=None) == hv.HV_ERR_INVALID_ARG
    assert run(mk(), root=None) == hv.HV_ERR_INVALID_ARG
    assert run(mk(), root=0x400008) == hv.HV_ERR_INVALID_ARG
    assert run(mk(), exp=0x500000) == hv.HV_ERR_INVALID_ARG            # expected without match
    assert run(mk(), match=0x600000) == hv.HV_ERR_INVALID_ARG          # match without expected
    assert run(mk(), exp=0x500000, match=0x600002) == hv.HV_ERR_INVALID_ARG


def test_cu_masked_stream_rejects_before_creating():
    handle = ctypes.c_void_p()
    zero = np.zeros(8, dtype=np.uint32)
    assert hv.lib.hv_stream_create_cu_masked(None, 8, ctypes.byref(handle)) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_stream_create_cu_masked(zero.ctypes.data, 0, ctypes.byref(handle)) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_stream_create_cu_masked(zero.ctypes.data, 8, None) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_stream_cu_mask(None, zero.ctypes.data, 8) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_stream_destroy(None) == hv.HV_ERR_INVALID_ARG
    w = hv.cu_mask_words([0, 31, 32, 255], 256)
    assert list(w) == [0x80000001, 1, 0, 0, 0, 0, 0, 0x80000000]
    with pytest.raises(ValueError):
        hv.cu_mask_words([256], 256)


def test_alg_forms_of_streaming_and_incremental_reject_before_launch():
    seg = np.array([0, 10, 30], dtype=np.uint64)
    assert hv.lib.hv_tree_bytes_alg(7, seg.ctypes.data, 2) == 0
    assert hv.lib.hv_tree_bytes_alg(1, seg.ctypes.data, 2) > hv.lib.hv_tree_bytes_alg(0, seg.ctypes.data, 2)
    assert hv.lib.hv_tree_bytes_alg(0, seg.ctypes.data, 2) == hv.lib.hv_tree_bytes(seg.ctypes.data, 2)
    assert hv.lib.hv_tree_build_alg(7, 0x1000, seg.ctypes.data, 2, 0x100000, 1 << 20, 0x2000, None) == \
        hv.HV_ERR_INVALID_ARG
    d = np.array([1], dtype=np.uint64)
    assert hv.lib.hv_tree_update_alg(7, 0x1000, seg.ctypes.data, 2, 0x100000, 1 << 20, d.ctypes.data, 1, 0x2000,
                                     0x200000, 1 << 20, None) == hv.HV_ERR_INVALID_ARG
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    st = hv.lib.hv_rehash_chunks_alg(1, arr.ctypes.data, 2, 64, d.ctypes.data, 1, 0x2000, 0x200000, 1 << 20, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"multiple of 128" in hv.lib.hv_last_error()
    assert hv.lib.hv_rehash_chunks_alg(7, arr.ctypes.data, 2, 64, d.ctypes.data, 1, 0x2000, 0x200000, 1 << 20,
                                       None) == hv.HV_ERR_INVALID_ARG
    st = hv.lib.hv_hash_host_chunks_alg(1, arr.ctypes.data, 2, 64, 0x2000, 1 << 20, 0x200000, 1 << 30, None, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"multiple of 128" in hv.lib.hv_last_error()


def test_verify_model_rejects_before_launch():
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    p = arr.ctypes.data
    need = hv.lib.hv_verify_model_workspace_bytes(0, p, 2, 64, 1)
    assert need > hv.lib.hv_plan_bytes(0, p, 2, 64, 1) and need % 256 == 0
    assert hv.lib.hv_verify_model_workspace_bytes(5, p, 2, 64, 1) == 0
    assert hv.lib.hv_verify_model_workspace_bytes(1, p, 2, 64, 1) == 0  # SHA-384 needs 128-byte multiples
    res = hv.hv_result()
    call = lambda alg=0, ws=0x100000, wb=need, r=ctypes.byref(res): \
        hv.lib.hv_verify_model(alg, p, 2, 64, 1, None, ws, wb, r, None)
    assert call(r=None) == hv.HV_ERR_INVALID_ARG
    assert call(alg=4) == hv.HV_ERR_INVALID_ARG
    assert call(wb=need - 1) == hv.HV_ERR_WORKSPACE
    assert call(ws=None) == hv.HV_ERR_WORKSPACE
    assert call(ws=0x100010) == hv.HV_ERR_WORKSPACE


def test_headers_compile_as_c_and_the_c_client_links(tmp_path):
    # the C client (tests/c_client) uses only include/*.h and the HIP runtime:
    # compile it as strict C11 with warnings as errors and link it against libhv
    import subprocess

    c_dir = os.path.join(ROOT, "tests", "c_client")
    exe = tmp_path / "verify_example"
    pkg = os.path.join(ROOT, "paper_2510_23938_amd")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", os.path.join(c_dir, "verify_example.c"),
           "-o", str(exe), "-L", pkg, "-lhv", "-L", "/opt/rocm/lib", "-lamdhip64"]
    subprocess.run(cmd, check=True, capture_output=True)
    assert exe.exists()


def test_leaf_kernel_choice_is_validated():
    for bad in (-1, 4):
        assert hv.lib.hv_set_leaf_kernel(bad) == hv.HV_ERR_INVALID_ARG
    for ok in (1, 2, 3, 0):
        assert hv.lib.hv_set_leaf_kernel(ok) == hv.HV_OK
    with pytest.raises(KeyError):
        hv.set_leaf_kernel("fast")
    # forced choices need no device to answer; NULL output is rejected
    for name in ("one-wave", "two-wave-compact"):
        hv.set_leaf_kernel(name)
        assert hv.leaf_kernel_for(100) == name
    hv.set_leaf_kernel("auto")
    assert hv.lib.hv_leaf_kernel_for(10, None) == hv.HV_ERR_INVALID_ARG


def test_merkle_launch_plan_checks_its_arguments():
    seg = np.array([0, 5, 9], dtype=np.uint64)
    n = ctypes.c_int(0)
    kind = (ctypes.c_int * 8)()
    units, one = (ctypes.c_uint64 * 8)(), (ctypes.c_uint64 * 8)()
    f = hv.lib.hv_merkle_launches
    assert f(7, seg.ctypes.data, 2, 256, ctypes.byref(n), kind, units, one) == hv.HV_ERR_INVALID_ARG
    assert f(hv.HV_SHA256, seg.ctypes.data, 0, 256, ctypes.byref(n), kind, units, one) == hv.HV_ERR_INVALID_ARG
    assert f(hv.HV_SHA256, None, 2, 256, ctypes.byref(n), kind, units, one) == hv.HV_ERR_INVALID_ARG
    for i in range(3):
        args = [kind, units, one]
        args[i] = None
        assert f(hv.HV_SHA256, seg.ctypes.data, 2, 256, ctypes.byref(n), *args) == hv.HV_ERR_INVALID_ARG
    assert f(hv.HV_SHA256, seg.ctypes.data, 2, 256, None, kind, units, one) == hv.HV_ERR_INVALID_ARG
    bad = np.array([1, 5, 9], dtype=np.uint64)
    assert f(hv.HV_SHA256, bad.ctypes.data, 2, 256, ctypes.byref(n), kind, units, one) == hv.HV_ERR_INVALID_ARG
    assert b"not 0" in hv.lib.hv_last_error()
    down = np.array([0, 5, 4], dtype=np.uint64)
    assert f(hv.HV_SHA384, down.ctypes.data, 2, 256, ctypes.byref(n), kind, units, one) == hv.HV_ERR_INVALID_ARG
    assert b"decreases" in hv.lib.hv_last_error()
    big = np.array([0, 1 << 40], dtype=np.uint64)
    assert f(hv.HV_SHA256, big.ctypes.data, 1, 256, ctypes.byref(n), kind, units, one) == hv.HV_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        hv.merkle_launches([0])


def _groups(counts, w=8):
    return sum(max(1, -(-int(c) // w)) for c in counts)


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_merkle_launch_plan_on_a_256_cu_device(alg):
    # No device needed with an explicit compute-unit count.  The 70B-shaped
    # set's 723 trees: the first group launch keeps 4 whole rounds of one wave
    # per SIMD (256 groups per CU per round) on one lane and gives its last
    # 7,153 groups four lanes; the second (34,000 groups, under a round) stays
    # on one lane; a tile launch ends the trees.  The manifest takes two tile
    # launches; the single tree of 10^6 entries keeps every group on one lane (its
    # 125,000 groups are under two rounds, where the split would cost more).
    import workloads as W
    leaves = [-(-int(L) // 65536) for L in W.workload_lengths(5)]
    seg = np.concatenate([[0], np.cumsum(leaves)]).astype(np.uint64)
    g1 = _groups(leaves)
    lvl3 = [max(1, -(-c // 8)) for c in leaves]
    g2 = _groups(lvl3)
    assert hv.merkle_launches(seg, alg, cus=256) == [("group", g1, 4 * 65536), ("group", g2, g2), ("tile", 723, 0)]
    assert g1 - 4 * 65536 == 7153
    assert hv.merkle_launches([0, 723], alg, cus=256) == [("tile", 2, 0), ("tile", 1, 0)]
    assert hv.merkle_launches([0, 10 ** 6], alg, cus=256) == [("group", 125000, 125000), ("tile", 245, 0), ("tile", 1, 0)]


def test_merkle_launch_plan_split_rule():
    # the split is taken only where it shortens the busiest SIMD's work:
    # k whole rounds of R = 256 * cus groups plus r more cost (k + 1) * D one
    # lane each, or k * D + ceil(4r / R) * d with four-lane last groups
    # (SHA-256: D = 22, d = 8 block times in leaf mode)
    one = lambda n, cus: hv.merkle_launches([0, 8 * n], "sha256", cus=cus)[0]
    R = 256 * 256
    assert one(R + 1, 256) == ("group", R + 1, R)                  # 22 + 8 < 44: split
    assert one(R + R // 2, 256) == ("group", R + R // 2, R)        # 22 + 16 < 44: split
    assert one(R + R // 2 + 1, 256) == ("group", R + R // 2 + 1, R + R // 2 + 1)  # 22 + 24 >= 44: one lane
    assert one(2 * R, 256) == ("group", 2 * R, 2 * R)              # whole rounds: nothing to split
    assert one(R // 2 + 10000, 256)[2] == R // 2 + 10000           # under one round: one lane
    # the rounds follow the compute-unit count
    assert one(3 * 256 * 100 + 5, 100) == ("group", 3 * 256 * 100 + 5, 3 * 256 * 100)


def test_noalloc_refuses_what_its_static_scratch_cannot_hold():
    # the array's size as the header states it, and the largest single-message set it holds
    hdr = open(os.path.join(ROOT, "include", "hv.h")).read()
    assert re.search(r"HV_NOALLOC_SCRATCH_BYTES\s*=\s*64\s*<<\s*20", hdr)
    assert hv.HV_NOALLOC_SCRATCH_BYTES == 64 << 20
    n_max = 2_794_794
    assert hv.lib.hv_hash_workspace_bytes(1, n_max) == hv.HV_NOALLOC_SCRATCH_BYTES
    assert hv.lib.hv_hash_workspace_bytes(1, n_max + 1) > hv.HV_NOALLOC_SCRATCH_BYTES
    # a 70B-shaped set (723 tensors, 2,153,249 leaves) fits
    assert hv.lib.hv_hash_workspace_bytes(723, 2_153_249) <= hv.HV_NOALLOC_SCRATCH_BYTES
    # checks that fail before the first HIP call (the scratch lookup), so no GPU is needed
    ptrs, lens = _msgs([64 * (n_max + 1)])
    arr = hv._msg_array(ptrs, lens)
    st = hv.lib.hv_hash_chunks_noalloc(hv.HV_SHA256, arr.ctypes.data, 1, 64, 0x1000, None)
    assert st == hv.HV_ERR_INVALID_ARG and b"static scratch" in hv.lib.hv_last_error()
    ptrs, lens = _msgs([1000, 64])
    arr = hv._msg_array(ptrs, lens)
    p = arr.ctypes.data
    assert hv.lib.hv_hash_chunks_noalloc(2, p, 2, 64, 0x1000, None) == hv.HV_ERR_INVALID_ARG
    assert b"unknown algorithm" in hv.lib.hv_last_error()
    assert hv.lib.hv_hash_chunks_noalloc(hv.HV_SHA384, p, 2, 64, 0x1000, None) == hv.HV_ERR_INVALID_ARG
    assert b"multiple of 128" in hv.lib.hv_last_error()
    assert hv.lib.hv_hash_chunks_noalloc(hv.HV_SHA256, p, 2, 96, 0x1000, None) == hv.HV_ERR_INVALID_ARG
    assert hv.lib.hv_hash_chunks_noalloc(hv.HV_SHA256, p, 2, 64, None, None) == hv.HV_ERR_INVALID_ARG
    assert b"leaf_digests is NULL" in hv.lib.hv_last_error()
    assert hv.lib.hv_hash_chunks_noalloc(hv.HV_SHA256, p, 2, 64, 0x1008, None) == hv.HV_ERR_INVALID_ARG
    assert b"16-byte aligned" in hv.lib.hv_last_error()
    assert hv.lib.hv_hash_chunks_noalloc(hv.HV_SHA256, None, 2, 64, 0x1000, None) == hv.HV_ERR_INVALID_ARG


@pytest.mark.parametrize("C", [0, 64, 4096])
def test_large_message_tables_are_laid_out_as_one_pass_would(C):
    # tables of 2^16 messages or more are validated and counted by several host
    # threads: the offsets and counts are those of the plain chunk-count rule
    n = 1_000_003
    lens = np.random.default_rng(41).integers(0, 70000, n).astype(np.uint64)
    ptrs = np.uint64(1 << 40) + np.arange(n, dtype=np.uint64) * np.uint64(1 << 17)
    seg, total = hv.hv_leaf_layout(ptrs, lens, C)
    per = np.ones(n, dtype=np.uint64) if C == 0 else (lens + np.uint64(C - 1)) // np.uint64(C)
    assert total == int(per.sum())
    assert seg[0] == 0 and np.array_equal(seg[1:], np.cumsum(per))
    assert hv.lib.hv_hash_workspace_bytes(n, total) > 0


def test_large_message_tables_report_the_lowest_refused_message():
    n = 300_000
    lens = np.full(n, 1000, dtype=np.uint64)
    ptrs = np.uint64(1 << 40) + np.arange(n, dtype=np.uint64) * np.uint64(4096)
    for bad in ([299_999], [150_000, 7], [7, 150_000], [0], [250_000, 40_000, 260_000]):
        p = ptrs.copy()
        p[bad] = 0  # NULL data with 1000 bytes
        with pytest.raises(hv.HVError) as e:
            hv.hv_leaf_layout(p, lens, 64)
        assert f"message {min(bad)} has NULL data" in str(e.value), bad
    # a chunk over the size limit, and an address range that wraps, in other parts of the table
    l2 = lens.copy()
    l2[200_000] = (1 << 37) + 64
    with pytest.raises(hv.HVError) as e:
        hv.hv_leaf_layout(ptrs, l2, 0)
    assert "message 200000: a chunk of" in str(e.value)
    p = ptrs.copy()
    p[123_456] = np.uint64((1 << 64) - 100)
    with pytest.raises(hv.HVError) as e:
        hv.hv_leaf_layout(p, lens, 64)
    assert "message 123456 wraps" in str(e.value)


def test_descriptor_table_cache_only_for_read_only_arrays():
    cache = hv._TableCache(pinned=False)  # (pinned host memory needs a GPU)
    lens = np.array([0, 100, 5000, 70000], dtype=np.uint64)
    ptrs = np.array([0, 0x10000, 0x20000, 0x40000], dtype=np.uint64)
    assert cache.lookup(ptrs, lens, 4096) is None  # writable: never cached
    ptrs.flags.writeable = False
    lens.flags.writeable = False
    arr, seg, n = cache.lookup(ptrs, lens, 4096)
    assert n == 0 + 1 + 2 + 18 and list(seg) == [0, 0, 1, 3, 21]
    assert list(arr[:, 0]) == list(ptrs) and list(arr[:, 1]) == list(lens)
    assert cache.lookup(ptrs, lens, 4096)[0] is arr  # same set: the same table
    arr2, seg2, n2 = cache.lookup(ptrs, lens, 0)     # another chunk size: rebuilt
    assert n2 == 4 and list(seg2) == [0, 1, 2, 3, 4]
    with pytest.raises(ValueError):
        seg2[0] = 5  # the cached offsets are read-only too
    other = lens.copy()
    other.flags.writeable = False
    assert cache.lookup(ptrs, other, 0)[0] is not arr2  # an equal but different array object: rebuilt


_NO_THREADS = r"""
import sys, resource, ctypes, threading, numpy as np
sys.path.insert(0, sys.argv[1])
from paper_2510_23938_amd import hv
n = 300_000
lens = np.random.default_rng(3).integers(0, 70000, n).astype(np.uint64)
ptrs = np.uint64(1 << 40) + np.arange(n, dtype=np.uint64) * np.uint64(1 << 17)
arr = hv._msg_array(ptrs, lens)
seg = np.zeros(n + 1, dtype=np.uint64)
bad = arr.copy()
bad[200_000, 0] = 0
want = np.concatenate([[0], np.cumsum((lens + np.uint64(4095)) // np.uint64(4096))]).astype(np.uint64)
with open("/proc/self/statm") as f:
    vm = int(f.read().split()[0]) * resource.getpagesize()
resource.setrlimit(resource.RLIMIT_AS, (vm + (6 << 20), resource.RLIM_INFINITY))  # no room for a thread stack
try:
    threading.Thread(target=lambda: None).start()
    sys.exit(3)  # threads still start: the check would prove nothing
except RuntimeError:
    pass
nl = ctypes.c_uint64(0)
assert hv.lib.hv_leaf_layout(arr.ctypes.data, n, 4096, seg.ctypes.data, ctypes.byref(nl)) == hv.HV_OK
assert nl.value == int(want[-1]) and np.array_equal(seg, want)
assert hv.lib.hv_leaf_layout(bad.ctypes.data, n, 4096, None, ctypes.byref(nl)) == hv.HV_ERR_INVALID_ARG
assert b"message 200000 has NULL data" in hv.lib.hv_last_error()
"""


def test_large_tables_fall_back_to_one_pass_when_threads_cannot_start():
    import subprocess
    import sys

    r = subprocess.run([sys.executable, "-c", _NO_THREADS, ROOT], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stderr[-2000:])
