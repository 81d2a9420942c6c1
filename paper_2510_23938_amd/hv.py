"""Python binding of ``include/hv.h``: argument marshalling only.

Every step of the path (chunk scheduling, SHA-256, Merkle levels, root
comparison) runs in the HIP kernels of ``libhv.so``; this module turns torch
device tensors into (pointer, length) descriptors, allocates caller-owned
outputs and workspaces with torch, passes torch's current HIP stream, and
turns error statuses into exceptions.  There is no CPU fallback: if the
library is missing, importing this module fails.

Names follow the C ABI:

* ``hv_leaf_layout(ptrs, lens, C)``        -> (seg_offsets, n_leaves)
* ``hv_hash_chunks(msgs, C)``              -> (leaf digests [n, 32] uint8, seg_offsets)
* ``hv_merkle_reduce(nodes, seg_offsets)`` -> roots [n_seg, 32] uint8
* ``hv_verify_root(root, expected)``       -> bool
* ``hv_compare_roots(roots, expected)``    -> mismatch flags [n] (int32)

Each of the four takes ``alg="sha256"`` (default; 32-byte digests) or
``alg="sha384"`` (48-byte digests, the ``*_alg`` entry points).

plus compositions used by callers: ``manifest_root`` (per-tensor roots, then
one root over them in the given order -- the paper's hierarchical roots) and
``verify`` (raises ``VerificationError`` on a mismatch, as the paper's
loader does when a model fails its check).
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref

import numpy as np
import torch  # loads the HIP runtime libhv.so binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhv.so")

HV_OK, HV_ERR_INVALID_ARG, HV_ERR_WORKSPACE, HV_ERR_HIP = 0, 1, 2, 3
HV_SHA256, HV_SHA384 = 0, 1
HV_NOALLOC_SCRATCH_BYTES = 64 << 20  # the static scratch of hv_hash_chunks_noalloc, per GPU
# hash name -> (hv_alg code, digest bytes)
ALGS = {"sha256": (HV_SHA256, 32), "sha384": (HV_SHA384, 48)}
_STATUS = {1: "HV_ERR_INVALID_ARG", 2: "HV_ERR_WORKSPACE", 3: "HV_ERR_HIP"}

# exported symbols, in the order include/hv.h declares them
EXPORTS = (
    "hv_leaf_layout", "hv_hash_workspace_bytes", "hv_hash_chunks", "hv_merkle_workspace_bytes",
    "hv_merkle_reduce", "hv_verify_workspace_bytes", "hv_verify_root", "hv_compare_roots",
    "hv_hash_chunks_alg", "hv_merkle_workspace_bytes_alg", "hv_merkle_reduce_alg", "hv_verify_root_alg",
    "hv_compare_roots_alg", "hv_hash_chunks_noalloc", "hv_last_error", "hv_set_kernel_timing", "hv_leaf_kernel_ms",
    "hv_leaf_schedule", "hv_set_leaf_kernel", "hv_leaf_kernel_for", "hv_merkle_launches",  # include/hv_inspect.h
    "hv_mb_valu", "hv_mb_sha256", "hv_mb_valu64", "hv_mb_sha384", "hv_mb_op_rate",
    "hv_mb_hbm_read",  # include/hv_microbench.h
    "hv_stream_workspace_bytes", "hv_hash_host_chunks", "hv_hash_host_chunks_alg",  # include/hv_stream.h
    "hv_tree_bytes", "hv_tree_build", "hv_tree_update_workspace_bytes", "hv_tree_update",
    "hv_rehash_workspace_bytes", "hv_rehash_chunks", "hv_tree_bytes_alg", "hv_tree_build_alg",
    "hv_tree_update_alg", "hv_rehash_chunks_alg",  # include/hv_incremental.h
    "hv_monitor_plan_bytes", "hv_monitor_init", "hv_monitor_scan_workspace_bytes",
    "hv_monitor_scan", "hv_stream_create_cu_masked", "hv_stream_cu_mask",
    "hv_stream_destroy",  # include/hv_monitor.h
    "hv_plan_bytes", "hv_plan_init", "hv_plan_run", "hv_verify_model_workspace_bytes",
    "hv_verify_model",  # include/hv_plan.h
)


class HVError(RuntimeError):
    """A non-OK status from libhv; ``status`` holds the code."""

    def __init__(self, status: int, detail: str):
        super().__init__(f"{_STATUS.get(status, status)}: {detail}")
        self.status = status


class VerificationError(Exception):
    """The computed root differs from the expected root."""


class hv_msg(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("nbytes", ctypes.c_uint64)]


HV_PLAN_MAX_LAUNCHES = 8


class hv_verify_plan(ctypes.Structure):
    _fields_ = [("device", ctypes.c_void_p), ("bytes", ctypes.c_size_t), ("alg", ctypes.c_int),
                ("manifest", ctypes.c_int), ("n_msgs", ctypes.c_uint32), ("n_seg", ctypes.c_uint32),
                ("chunk_bytes", ctypes.c_uint64), ("n_leaves", ctypes.c_uint64),
                ("launches", ctypes.c_uint32 * 2), ("tiles", (ctypes.c_uint64 * HV_PLAN_MAX_LAUNCHES) * 2)]


class hv_result(ctypes.Structure):
    _fields_ = [("integrity_verified", ctypes.c_int), ("root_bytes", ctypes.c_uint32),
                ("root", ctypes.c_uint8 * 48), ("verification_time_ns", ctypes.c_uint64)]


class hv_monitor_plan(ctypes.Structure):
    _fields_ = [("device", ctypes.c_void_p), ("alg", ctypes.c_int), ("n_msgs", ctypes.c_uint32),
                ("chunk_bytes", ctypes.c_uint64), ("n_leaves", ctypes.c_uint64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (no CPU fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, u32, u64, sz = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t
    sig = {
        "hv_leaf_layout": ([vp, u32, u64, vp, vp], ctypes.c_int),
        "hv_hash_workspace_bytes": ([u32, u64], sz),
        "hv_hash_chunks": ([vp, u32, u64, vp, vp, sz, vp], ctypes.c_int),
        "hv_merkle_workspace_bytes": ([u64, u32], sz),
        "hv_merkle_reduce": ([vp, vp, u32, vp, vp, sz, vp], ctypes.c_int),
        "hv_verify_workspace_bytes": ([], sz),
        "hv_verify_root": ([vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "hv_compare_roots": ([vp, vp, u32, vp, vp], ctypes.c_int),
        "hv_hash_chunks_alg": ([ctypes.c_int, vp, u32, u64, vp, vp, sz, vp], ctypes.c_int),
        "hv_merkle_workspace_bytes_alg": ([ctypes.c_int, u64, u32], sz),
        "hv_merkle_reduce_alg": ([ctypes.c_int, vp, vp, u32, vp, vp, sz, vp], ctypes.c_int),
        "hv_verify_root_alg": ([ctypes.c_int, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "hv_compare_roots_alg": ([ctypes.c_int, vp, vp, u32, vp, vp], ctypes.c_int),
        "hv_hash_chunks_noalloc": ([ctypes.c_int, vp, u32, u64, vp, vp], ctypes.c_int),
        "hv_last_error": ([], ctypes.c_char_p),
        "hv_set_kernel_timing": ([ctypes.c_int], ctypes.c_int),
        "hv_leaf_kernel_ms": ([vp], ctypes.c_int),
        "hv_leaf_schedule": ([vp, u32, u64, vp, vp, sz, vp], ctypes.c_int),
        "hv_set_leaf_kernel": ([ctypes.c_int], ctypes.c_int),
        "hv_leaf_kernel_for": ([ctypes.c_uint64, ctypes.c_void_p], ctypes.c_int),
        "hv_merkle_launches": ([ctypes.c_int32, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
        "hv_mb_valu": ([vp, u32, u32, vp, vp], ctypes.c_int),
        "hv_mb_hbm_read": ([vp, u64, vp, u32, vp], ctypes.c_int),
        "hv_mb_sha256": ([vp, u32, u32, vp, vp], ctypes.c_int),
        "hv_mb_valu64": ([vp, u32, u32, vp, vp], ctypes.c_int),
        "hv_mb_sha384": ([vp, u32, u32, vp, vp], ctypes.c_int),
        "hv_mb_op_rate": ([u32, vp, u32, u32, vp, vp], ctypes.c_int),
        "hv_stream_workspace_bytes": ([vp, u32, u64, u64], sz),
        "hv_hash_host_chunks": ([vp, u32, u64, vp, u64, vp, sz, vp, vp], ctypes.c_int),
        "hv_tree_bytes": ([vp, u32], sz),
        "hv_tree_build": ([vp, vp, u32, vp, sz, vp, vp], ctypes.c_int),
        "hv_tree_update_workspace_bytes": ([u32], sz),
        "hv_tree_update": ([vp, vp, u32, vp, sz, vp, u32, vp, vp, sz, vp], ctypes.c_int),
        "hv_rehash_workspace_bytes": ([u32, u32], sz),
        "hv_rehash_chunks": ([vp, u32, u64, vp, u32, vp, vp, sz, vp], ctypes.c_int),
        "hv_hash_host_chunks_alg": ([ctypes.c_int, vp, u32, u64, vp, u64, vp, sz, vp, vp], ctypes.c_int),
        "hv_tree_bytes_alg": ([ctypes.c_int, vp, u32], sz),
        "hv_tree_build_alg": ([ctypes.c_int, vp, vp, u32, vp, sz, vp, vp], ctypes.c_int),
        "hv_tree_update_alg": ([ctypes.c_int, vp, vp, u32, vp, sz, vp, u32, vp, vp, sz, vp], ctypes.c_int),
        "hv_rehash_chunks_alg": ([ctypes.c_int, vp, u32, u64, vp, u32, vp, vp, sz, vp], ctypes.c_int),
        "hv_plan_bytes": ([ctypes.c_int, vp, u32, u64, ctypes.c_int], sz),
        "hv_plan_init": ([ctypes.c_int, vp, u32, u64, ctypes.c_int, vp, sz, vp, vp], ctypes.c_int),
        "hv_plan_run": ([vp, vp, vp, vp, vp, vp, vp], ctypes.c_int),
        "hv_verify_model_workspace_bytes": ([ctypes.c_int, vp, u32, u64, ctypes.c_int], sz),
        "hv_verify_model": ([ctypes.c_int, vp, u32, u64, ctypes.c_int, vp, vp, sz, vp, vp], ctypes.c_int),
        "hv_monitor_plan_bytes": ([u32], sz),
        "hv_monitor_init": ([ctypes.c_int, vp, u32, u64, vp, sz, vp, vp], ctypes.c_int),
        "hv_monitor_scan_workspace_bytes": ([ctypes.c_int, u64], sz),
        "hv_monitor_scan": ([vp, u64, u64, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "hv_stream_create_cu_masked": ([vp, u32, vp], ctypes.c_int),
        "hv_stream_cu_mask": ([vp, vp, u32], ctypes.c_int),
        "hv_stream_destroy": ([vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes, f.restype = args, res
    return lib


lib = _load()


def _check(status: int):
    if status != HV_OK:
        raise HVError(status, lib.hv_last_error().decode("utf-8", "replace"))


def _alg(alg: str) -> tuple:
    """(hv_alg code, digest bytes) of a hash name."""
    try:
        return ALGS[alg]
    except KeyError:
        raise ValueError(f"unknown hash {alg!r}; expected one of {sorted(ALGS)}") from None


def _stream(device=None) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dev(device) -> torch.device:
    """``device`` with its index filled in (the current device for a bare "cuda")."""
    d = torch.device(device)
    return d if d.index is not None else torch.device(d.type, torch.cuda.current_device())


def _buffer(t, nbytes: int, what: str, device) -> int:
    """Data pointer of ``t`` once it is known to be a contiguous tensor on ``device``
    holding at least ``nbytes`` bytes.  The library trusts the pointers it is
    given, so a short or misplaced buffer would be overrun on the GPU: it is
    refused here instead."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if _dev(t.device) != _dev(device):
        raise ValueError(f"{what} is on {t.device}, but the call runs on {_dev(device)}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what} holds {have} bytes; the call needs {nbytes}")
    return t.data_ptr()


class Workspace:
    """A growable device byte buffer handed to the library as scratch."""

    def __init__(self, device="cuda"):
        self.device = torch.device(device)
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        nbytes = max(int(nbytes), 256)
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self.buf


class HostBuffer:
    """A growable host byte buffer reused across calls, pinned or pageable.

    For the tables a call hands to the library (the message descriptors) and
    the segment offsets it plans from: the library reads and uploads them
    before it returns, so the next call may overwrite them.  Reuse saves the
    page faults of fresh multi-MB arrays, and a pinned descriptor table
    uploads by DMA; with 10^6 messages that shortens the host work ahead of
    each one-shot pass by about a millisecond."""

    def __init__(self, pinned: bool = True):
        self.pinned = pinned
        self.buf = None

    def get(self, nbytes: int, dtype=np.uint64) -> np.ndarray:
        nbytes = int(nbytes)
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(max(nbytes, 4096), dtype=torch.uint8, pin_memory=self.pinned)
        return self.buf.numpy()[:nbytes].view(dtype)


def _msg_array(ptrs: np.ndarray, lens: np.ndarray, host: HostBuffer | None = None) -> np.ndarray:
    """hv_msg[n] as a (n, 2) uint64 array (data, nbytes), in ``host`` when given."""
    n = len(lens)
    arr = host.get(16 * n).reshape(n, 2) if host is not None else np.empty((n, 2), dtype=np.uint64)
    arr[:, 0] = np.asarray(ptrs, dtype=np.uint64)
    arr[:, 1] = np.asarray(lens, dtype=np.uint64)
    return arr


def messages_of(tensors) -> tuple:
    """(ptrs, lens) of contiguous device tensors' bytes, in the given order."""
    ptrs, lens = [], []
    for t in tensors:
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous: the bytes hashed are the bytes stored")
        ptrs.append(t.data_ptr())
        lens.append(t.numel() * t.element_size())
    return np.array(ptrs, dtype=np.uint64), np.array(lens, dtype=np.uint64)


def _ptr_len(msgs):
    if hasattr(msgs, "ptrs") and hasattr(msgs, "lens"):
        return np.asarray(msgs.ptrs, dtype=np.uint64), np.asarray(msgs.lens, dtype=np.uint64)
    if isinstance(msgs, tuple) and len(msgs) == 2 and isinstance(msgs[0], np.ndarray):
        return msgs
    return messages_of(msgs)


def hv_leaf_layout(ptrs, lens, chunk_bytes: int):
    return _layout_of(_msg_array(ptrs, lens), chunk_bytes)


def _layout_of(arr: np.ndarray, chunk_bytes: int, host: HostBuffer | None = None):
    """(seg_offsets, n_leaves) of an hv_msg array as _msg_array builds it (seg_offsets in ``host`` when given)."""
    n = len(arr)
    seg = host.get(8 * (n + 1)) if host is not None else np.zeros(n + 1, dtype=np.uint64)
    n_leaves = ctypes.c_uint64(0)
    _check(lib.hv_leaf_layout(arr.ctypes.data if n else None, n, chunk_bytes, seg.ctypes.data,
                              ctypes.byref(n_leaves)))
    return seg, int(n_leaves.value)


def _hash_call(alg: str, arr, n, chunk_bytes, out_ptr, ws, stream):
    code, _ = _alg(alg)
    if code == HV_SHA256:
        return lib.hv_hash_chunks(arr, n, chunk_bytes, out_ptr, ws.data_ptr(), ws.numel(), stream)
    return lib.hv_hash_chunks_alg(code, arr, n, chunk_bytes, out_ptr, ws.data_ptr(), ws.numel(), stream)


def _merkle_call(alg: str, nodes_ptr, seg_ptr, n_seg, roots_ptr, ws, stream):
    code, _ = _alg(alg)
    if code == HV_SHA256:
        return lib.hv_merkle_reduce(nodes_ptr, seg_ptr, n_seg, roots_ptr, ws.data_ptr(), ws.numel(), stream)
    return lib.hv_merkle_reduce_alg(code, nodes_ptr, seg_ptr, n_seg, roots_ptr, ws.data_ptr(), ws.numel(), stream)


def _merkle_ws_bytes(alg: str, n_nodes: int, n_seg: int) -> int:
    code, _ = _alg(alg)
    if code == HV_SHA256:
        return lib.hv_merkle_workspace_bytes(n_nodes, n_seg)
    return lib.hv_merkle_workspace_bytes_alg(code, n_nodes, n_seg)


class _TableCache:
    """The descriptor table and leaf layout of the last message set, kept while
    that set's ``ptrs`` and ``lens`` are the same read-only numpy arrays: both are
    pure functions of those arrays and the chunk size, so they are rebuilt only
    when the set changes.  The library still validates and uploads the table on
    every call.  Writable arrays are never cached."""

    def __init__(self, pinned: bool = True):
        self.key = None
        self.pinned = pinned  # pinned tables upload by DMA

    def lookup(self, ptrs, lens, chunk_bytes: int):
        if not (isinstance(ptrs, np.ndarray) and isinstance(lens, np.ndarray)) or \
                ptrs.flags.writeable or lens.flags.writeable:
            return None
        if self.key is not None and self.key[0] is ptrs and self.key[1] is lens and self.key[2] == chunk_bytes:
            return self.table
        host = HostBuffer(pinned=self.pinned)  # owned by this entry
        arr = _msg_array(ptrs, lens, host)
        seg, n_leaves = _layout_of(arr, chunk_bytes)
        seg.flags.writeable = False
        self.key = (ptrs, lens, chunk_bytes)  # the references keep the arrays (and so their ids) alive
        self.host = host
        self.table = (arr, seg, n_leaves)
        return self.table


def hv_hash_chunks(msgs, chunk_bytes: int, device="cuda", workspace: Workspace | None = None, out=None,
                   alg: str = "sha256", host: HostBuffer | None = None, seg_host: HostBuffer | None = None,
                   table=None):
    """Leaf digests of ``msgs`` (tensors, a (ptrs, lens) pair, or an object with
    ``ptrs``/``lens``): ([n_leaves, D] uint8 device tensor, seg_offsets), D the digest size.
    ``host`` holds the descriptor table; with ``seg_host`` the returned seg_offsets
    live in that buffer, valid until its next use.  ``table``: the (descriptor
    table, seg_offsets, n_leaves) of ``msgs`` when the caller already has them."""
    _, D = _alg(alg)
    if table is not None:
        arr, seg, n_leaves = table
    else:
        ptrs, lens = _ptr_len(msgs)
        arr = _msg_array(ptrs, lens, host)
        seg, n_leaves = _layout_of(arr, chunk_bytes, seg_host)
    n = len(arr)
    dev = torch.device(device)
    if out is None:
        out = torch.empty((n_leaves, D), dtype=torch.uint8, device=dev)
    out_ptr = _buffer(out, n_leaves * D, "out", dev)
    ws = (workspace or Workspace(dev)).get(lib.hv_hash_workspace_bytes(n, n_leaves))
    _check(_hash_call(alg, arr.ctypes.data if n else None, n, chunk_bytes, out_ptr if n_leaves else None, ws,
                      _stream(dev)))
    return out, seg


def hv_hash_chunks_noalloc(msgs, chunk_bytes: int, device="cuda", out=None, alg: str = "sha256"):
    """Leaf digests as ``hv_hash_chunks``, with the library's static scratch in place of a
    workspace (the C call allocates nothing; ``out`` is allocated here when not given)."""
    code, D = _alg(alg)
    ptrs, lens = _ptr_len(msgs)
    arr = _msg_array(ptrs, lens)
    seg, n_leaves = _layout_of(arr, chunk_bytes)
    n = len(arr)
    dev = torch.device(device)
    if out is None:
        out = torch.empty((n_leaves, D), dtype=torch.uint8, device=dev)
    out_ptr = _buffer(out, n_leaves * D, "out", dev)
    _check(lib.hv_hash_chunks_noalloc(code, arr.ctypes.data if n else None, n, chunk_bytes,
                                      out_ptr if n_leaves else None, _stream(dev)))
    return out, seg


def host_messages_of(arrays) -> tuple:
    """(ptrs, lens) of host byte buffers: numpy arrays or CPU tensors (pinned ones let copies overlap hashing)."""
    ptrs, lens = [], []
    for a in arrays:
        if isinstance(a, torch.Tensor):
            if a.is_cuda or not a.is_contiguous():
                raise ValueError("host messages must be contiguous CPU tensors")
            ptrs.append(a.data_ptr())
            lens.append(a.numel() * a.element_size())
        else:
            a = np.ascontiguousarray(a)
            ptrs.append(a.ctypes.data if a.nbytes else 0)
            lens.append(a.nbytes)
    return np.array(ptrs, dtype=np.uint64), np.array(lens, dtype=np.uint64)


def hv_hash_host_chunks(host_msgs, chunk_bytes: int, batch_bytes: int = 1 << 30, device="cuda",
                        workspace: Workspace | None = None, copy_stream=None, alg: str = "sha256"):
    """Leaf digests of host-resident messages streamed through GPU memory
    (synchronous): ([n_leaves, D] uint8 device tensor, seg_offsets)."""
    code, D = _alg(alg)
    ptrs, lens = host_messages_of(host_msgs) if not (isinstance(host_msgs, tuple) and len(host_msgs) == 2
                                                     and isinstance(host_msgs[0], np.ndarray)) else host_msgs
    arr = _msg_array(ptrs, lens)
    seg, n_leaves = _layout_of(arr, chunk_bytes)
    n = len(arr)
    dev = torch.device(device)
    need = lib.hv_stream_workspace_bytes(arr.ctypes.data if n else None, n, chunk_bytes, batch_bytes)
    if need == 0:
        raise HVError(HV_ERR_INVALID_ARG, lib.hv_last_error().decode("utf-8", "replace"))
    ws = (workspace or Workspace(dev)).get(need)
    out = torch.empty((n_leaves, D), dtype=torch.uint8, device=dev)
    cs = copy_stream or torch.cuda.Stream(dev)
    _check(lib.hv_hash_host_chunks_alg(code, arr.ctypes.data if n else None, n, chunk_bytes,
                                       out.data_ptr() if n_leaves else None, batch_bytes, ws.data_ptr(), ws.numel(),
                                       cs.cuda_stream, _stream(dev)))
    return out, seg


def hv_merkle_reduce(nodes: torch.Tensor, seg_offsets, workspace: Workspace | None = None, out=None,
                     alg: str = "sha256"):
    """Per-segment RFC 6962 roots of ``nodes`` ([n, D] uint8 device tensor, D the digest size)."""
    _, D = _alg(alg)
    seg = np.ascontiguousarray(seg_offsets, dtype=np.uint64)
    n_seg = len(seg) - 1
    if n_seg < 1:
        raise ValueError("seg_offsets needs at least two entries (one segment)")
    nodes_ptr = _buffer(nodes, int(seg[-1]) * D, "nodes", nodes.device)
    if out is None:
        out = torch.empty((n_seg, D), dtype=torch.uint8, device=nodes.device)
    out_ptr = _buffer(out, n_seg * D, "out", nodes.device)
    ws = (workspace or Workspace(nodes.device)).get(_merkle_ws_bytes(alg, int(seg[-1]), n_seg))
    _check(_merkle_call(alg, nodes_ptr if nodes.numel() else None, seg.ctypes.data, n_seg, out_ptr, ws,
                        _stream(nodes.device)))
    return out


def hv_verify_root(root: torch.Tensor, expected: bytes, workspace: Workspace | None = None,
                   alg: str = "sha256") -> bool:
    """The D device bytes of ``root`` equal ``expected`` (compared on the GPU; D the digest size)."""
    code, D = _alg(alg)
    expected = bytes(expected)
    if len(expected) != D:
        raise ValueError(f"expected root must be {D} bytes for {alg}, got {len(expected)}")
    exp = (ctypes.c_uint8 * D).from_buffer_copy(expected)
    root_ptr = _buffer(root, D, "root", root.device)
    match = ctypes.c_int(-1)
    ws = (workspace or Workspace(root.device)).get(lib.hv_verify_workspace_bytes())
    if code == HV_SHA256:
        st = lib.hv_verify_root(root_ptr, exp, ctypes.byref(match), ws.data_ptr(), ws.numel(),
                                _stream(root.device))
    else:
        st = lib.hv_verify_root_alg(code, root_ptr, exp, ctypes.byref(match), ws.data_ptr(), ws.numel(),
                                    _stream(root.device))
    _check(st)
    return match.value == 1


def hv_compare_roots(roots: torch.Tensor, expected: torch.Tensor, alg: str = "sha256") -> torch.Tensor:
    """int32 [n]: 1 where roots[i] differs from expected[i] (both [n, D] device)."""
    code, D = _alg(alg)
    n = roots.shape[0]
    if roots.shape != (n, D) or expected.shape != (n, D):
        raise ValueError(f"roots and expected must both be [n, {D}] for {alg}")
    _buffer(roots, n * D, "roots", roots.device)
    _buffer(expected, n * D, "expected", roots.device)
    mism = torch.empty(n, dtype=torch.int32, device=roots.device)
    if code == HV_SHA256:
        st = lib.hv_compare_roots(roots.data_ptr(), expected.data_ptr(), n, mism.data_ptr(), _stream(roots.device))
    else:
        st = lib.hv_compare_roots_alg(code, roots.data_ptr(), expected.data_ptr(), n, mism.data_ptr(),
                                      _stream(roots.device))
    _check(st)
    return mism


def hv_leaf_schedule(msgs, chunk_bytes: int, device="cuda") -> np.ndarray:
    """The scheduler's leaf table, in schedule order: uint64 [n_leaves, 3] of
    (source address, byte length, leaf index).  For tests of the scheduler."""
    ptrs, lens = _ptr_len(msgs)
    arr = _msg_array(ptrs, lens)
    _, n_leaves = _layout_of(arr, chunk_bytes)
    n = len(arr)
    table = np.zeros((n_leaves, 3), dtype=np.uint64)
    dev = torch.device(device)
    ws = Workspace(dev).get(lib.hv_hash_workspace_bytes(n, n_leaves))
    _check(lib.hv_leaf_schedule(arr.ctypes.data if n else None, n, chunk_bytes,
                                table.ctypes.data if n_leaves else None, ws.data_ptr(), ws.numel(), _stream(dev)))
    return table


def measure_valu_peak(device="cuda", grid=16384, iters=4096, reps=5, mix: str = "sha256") -> dict:
    """Best rate of a hash's VALU mix over reps launches: "sha256" (alignbit /
    bitop3 / add3) or "sha384" (the same logic on word halves plus 64-bit adds)."""
    fn = {"sha256": lib.hv_mb_valu, "sha384": lib.hv_mb_valu64}[mix]
    dev = torch.device(device)
    sink = torch.empty(grid * 256, dtype=torch.int32, device=dev)
    ops = ctypes.c_uint64(0)
    s = _stream(dev)
    _check(fn(sink.data_ptr(), grid, 64, ctypes.byref(ops), s))  # warm-up
    best = None
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        _check(fn(sink.data_ptr(), grid, iters, ctypes.byref(ops), s))
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    return {"tops": ops.value / (best / 1e3) / 1e12, "ms": best, "ops": ops.value, "grid": grid, "iters": iters}


def measure_sha256_ceiling(device="cuda", grid=8192, blocks=256, reps=5, alg: str = "sha256") -> dict:
    """Best rate of register-only compressions (no memory traffic) of a hash:
    64-byte SHA-256 blocks, or 128-byte SHA-384 blocks with alg="sha384"."""
    fn, block_bytes = {"sha256": (lib.hv_mb_sha256, 64), "sha384": (lib.hv_mb_sha384, 128)}[alg]
    dev = torch.device(device)
    sink = torch.empty(grid * 256, dtype=torch.int32, device=dev)
    n = ctypes.c_uint64(0)
    s = _stream(dev)
    _check(fn(sink.data_ptr(), grid, 8, ctypes.byref(n), s))  # warm-up
    best = None
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        _check(fn(sink.data_ptr(), grid, blocks, ctypes.byref(n), s))
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    return {"blocks_per_s": n.value / (best / 1e3), "GBps_equiv": n.value * block_bytes / (best / 1e3) / 1e9,
            "ms": best, "blocks": n.value}


OP_RATE_NAMES = ("v_alignbit_b32", "v_bitop3_b32", "v_add3_u32", "v_add_u32", "v_xor_b32", "v_lshrrev_b32",
                 "v_perm_b32", "v_lshl_add_u64")


def measure_op_rates(device="cuda", grid=16384, iters=1024, reps=5) -> dict:
    """Best issue rate (T lane-ops/s) of each instruction of OP_RATE_NAMES."""
    dev = torch.device(device)
    sink = torch.empty(grid * 256, dtype=torch.int32, device=dev)
    ops = ctypes.c_uint64(0)
    s = _stream(dev)
    out = {}
    for op, name in enumerate(OP_RATE_NAMES):
        _check(lib.hv_mb_op_rate(op, sink.data_ptr(), grid, 8, ctypes.byref(ops), s))  # warm-up
        best = None
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            _check(lib.hv_mb_op_rate(op, sink.data_ptr(), grid, iters, ctypes.byref(ops), s))
            b.record()
            b.synchronize()
            ms = a.elapsed_time(b)
            best = ms if best is None else min(best, ms)
        out[name] = ops.value / (best / 1e3) / 1e12
    return out


def measure_hbm_read(nbytes=16 << 30, device="cuda", grid=None, reps=5) -> dict:
    """Best streaming-read bandwidth over reps launches on an nbytes buffer."""
    dev = torch.device(device)
    buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    grid = grid or 256 * 64
    sink = torch.empty(grid * 256, dtype=torch.int32, device=dev)
    s = _stream(dev)
    _check(lib.hv_mb_hbm_read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, s))
    best = None
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        _check(lib.hv_mb_hbm_read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, s))
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    del buf
    return {"GBps": nbytes / (best / 1e3) / 1e9, "ms": best, "bytes": nbytes, "grid": grid}


def set_leaf_kernel(choice: str):
    """Leaf kernel (SHA-256 and SHA-384) for this thread: "auto", "one-wave", "two-wave" or
    "two-wave-compact" (two producer/consumer pairs per workgroup); digests do not depend on it."""
    _check(lib.hv_set_leaf_kernel({"auto": 0, "one-wave": 1, "two-wave": 2, "two-wave-compact": 3}[choice]))


def leaf_kernel_for(n_leaves: int) -> str:
    """The leaf kernel a hash call over n_leaves leaves runs on the current device under this thread's
    choice: "one-wave", "two-wave" or "two-wave-compact" (two producer/consumer pairs per workgroup)."""
    k = ctypes.c_int(0)
    _check(lib.hv_leaf_kernel_for(int(n_leaves), ctypes.byref(k)))
    return {1: "one-wave", 2: "two-wave", 3: "two-wave-compact"}[k.value]


def merkle_launches(seg_offsets, alg: str = "sha256", cus: int = 0) -> list:
    """The launches hv_merkle_reduce makes for these segments on a device of ``cus`` compute units
    (0: the current device), as
    (kind, units, one_lane) per launch: kind "group" or "tile", the groups or tiles it reduces,
    and the groups a group launch gives one lane each (its last units - one_lane groups take four)."""
    code, _ = _alg(alg)
    seg = np.ascontiguousarray(seg_offsets, dtype=np.uint64)
    if len(seg) < 2:
        raise ValueError("seg_offsets needs at least two entries (one segment)")
    n = ctypes.c_int(0)
    kind = (ctypes.c_int * 8)()
    units, one = (ctypes.c_uint64 * 8)(), (ctypes.c_uint64 * 8)()
    _check(lib.hv_merkle_launches(code, seg.ctypes.data, len(seg) - 1, int(cus), ctypes.byref(n), kind, units, one))
    return [({1: "group", 2: "tile"}[kind[k]], int(units[k]), int(one[k])) for k in range(n.value)]


def set_kernel_timing(enable: bool):
    _check(lib.hv_set_kernel_timing(1 if enable else 0))


def leaf_kernel_ms() -> float:
    ms = ctypes.c_float(0.0)
    _check(lib.hv_leaf_kernel_ms(ctypes.byref(ms)))
    return float(ms.value)


class Verifier:
    """Reusable workspaces for repeated hash -> per-message roots -> manifest -> verify."""

    def __init__(self, device="cuda", alg: str = "sha256"):
        self.device = torch.device(device)
        self.alg, self.D = alg, _alg(alg)[1]
        self.ws_hash = Workspace(self.device)
        self.ws_tree = Workspace(self.device)
        self.ws_manifest = Workspace(self.device)
        self.ws_verify = Workspace(self.device)
        self.host_msgs = HostBuffer(pinned=True)    # descriptor tables, uploaded by DMA
        self.host_seg = HostBuffer(pinned=False)    # offsets used only inside one call
        self.tables = _TableCache()                 # for message sets given as read-only arrays

    def _leaves(self, msgs, chunk_bytes: int, keep_seg: bool):
        ptrs, lens = _ptr_len(msgs)
        return hv_hash_chunks((ptrs, lens), chunk_bytes, self.device, self.ws_hash, alg=self.alg, host=self.host_msgs,
                              seg_host=None if keep_seg else self.host_seg,
                              table=self.tables.lookup(ptrs, lens, chunk_bytes))

    def leaf_digests(self, msgs, chunk_bytes: int):
        return self._leaves(msgs, chunk_bytes, True)

    def _roots(self, msgs, chunk_bytes: int, keep_seg: bool):
        leaves, seg = self._leaves(msgs, chunk_bytes, keep_seg)
        if len(seg) == 1:  # no messages, no roots (hv_merkle_reduce takes at least one segment)
            return torch.empty((0, self.D), dtype=torch.uint8, device=self.device), leaves, seg
        return hv_merkle_reduce(leaves, seg, self.ws_tree, alg=self.alg), leaves, seg

    def roots(self, msgs, chunk_bytes: int):
        """(per-message roots [n, D], leaf digests, seg_offsets)."""
        return self._roots(msgs, chunk_bytes, True)

    def manifest_root(self, msgs, chunk_bytes: int) -> torch.Tensor:
        """One root over the per-message roots, in message order ([1, D] device)."""
        roots, _, _ = self._roots(msgs, chunk_bytes, False)
        return hv_merkle_reduce(roots, np.array([0, roots.shape[0]], dtype=np.uint64), self.ws_manifest,
                                alg=self.alg)

    def single_tree_root(self, msgs, chunk_bytes: int) -> torch.Tensor:
        """One root over all leaf digests of all messages ([1, D] device)."""
        leaves, _ = self._leaves(msgs, chunk_bytes, False)
        return hv_merkle_reduce(leaves, np.array([0, leaves.shape[0]], dtype=np.uint64), self.ws_tree,
                                alg=self.alg)

    def verify_root(self, root: torch.Tensor, expected: bytes) -> bool:
        return hv_verify_root(root.reshape(-1)[:self.D], expected, self.ws_verify, alg=self.alg)


class Pipeline:
    """One message set, prepared once (include/hv_plan.h), run many times: the whole path.

    mode "manifest": chunk digests -> one root per message -> one root over
    those (hierarchical roots); mode "single": chunk digests -> one root over
    all of them.  ``run(expected)`` ends with the on-GPU root comparison and
    returns its verdict.  The plan, outputs and the expected-root and verdict
    buffers are allocated here, once; a pass only queues kernels, so
    ``capture`` can record it in a HIP graph and ``replay`` re-runs it.
    """

    def __init__(self, msgs, chunk_bytes: int, mode: str = "manifest", device="cuda", alg: str = "sha256"):
        if mode not in ("manifest", "single"):
            raise ValueError(mode)
        code, D = _alg(alg)
        self.alg, self.D = alg, D
        self.device = torch.device(device)
        self.mode, self.C = mode, int(chunk_bytes)
        ptrs, lens = _ptr_len(msgs)
        self.keepalive = msgs
        arr = _msg_array(ptrs, lens)
        self.n_msgs = len(arr)
        self.seg, self.n_leaves = _layout_of(arr, self.C)
        self.total_bytes = int(np.asarray(lens, dtype=np.uint64).sum()) if self.n_msgs else 0
        manifest = 1 if mode == "manifest" else 0
        nbytes = lib.hv_plan_bytes(code, arr.ctypes.data if self.n_msgs else None, self.n_msgs, self.C, manifest)
        if nbytes == 0:
            raise HVError(HV_ERR_INVALID_ARG, lib.hv_last_error().decode("utf-8", "replace"))
        self.plan_mem = Workspace(self.device).get(nbytes)
        self.plan = hv_verify_plan()
        _check(lib.hv_plan_init(code, arr.ctypes.data if self.n_msgs else None, self.n_msgs, self.C, manifest,
                                self.plan_mem.data_ptr(), self.plan_mem.numel(), ctypes.byref(self.plan),
                                _stream(self.device)))
        self.leaves = torch.empty((self.n_leaves, D), dtype=torch.uint8, device=self.device)
        self.roots = torch.empty((max(int(self.plan.n_seg), 1), D), dtype=torch.uint8, device=self.device)
        self.root = torch.empty((1, D), dtype=torch.uint8, device=self.device) if manifest else self.roots[:1]
        self.expected_dev = torch.zeros(D, dtype=torch.uint8, device=self.device)
        self.match_dev = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.match_host = torch.zeros(1, dtype=torch.int32, pin_memory=True)
        self._expected = None
        self.graph = None

    def _run(self, check: bool, stream: int):
        _check(lib.hv_plan_run(ctypes.byref(self.plan), self.leaves.data_ptr() if self.n_leaves else None,
                               self.roots.data_ptr(), self.root.data_ptr(),
                               self.expected_dev.data_ptr() if check else None,
                               self.match_dev.data_ptr() if check else None, stream))

    def compute(self):
        """Queue the digests and roots on the current stream; returns the [1, D] root."""
        self._run(False, _stream(self.device))
        return self.root

    def set_expected(self, expected: bytes):
        """Store the expected root on the device (only when it changed)."""
        expected = bytes(expected)
        if len(expected) != self.D:
            raise ValueError(f"expected root must be {self.D} bytes for {self.alg}")
        if expected != self._expected:
            self.expected_dev.copy_(torch.frombuffer(bytearray(expected), dtype=torch.uint8))
            self._expected = expected

    def _verdict(self) -> bool:
        s = torch.cuda.current_stream(self.device)
        self.match_host.copy_(self.match_dev, non_blocking=True)
        s.synchronize()
        return int(self.match_host[0]) == 1

    def run(self, expected: bytes) -> bool:
        """The whole path: digests, roots, comparison with ``expected`` (synchronous)."""
        self.set_expected(expected)
        self._run(True, _stream(self.device))
        return self._verdict()

    def capture(self, expected: bytes):
        """Record one checked pass in a HIP graph (kernels only) for ``replay``."""
        self.set_expected(expected)
        torch.cuda.synchronize(self.device)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self._run(True, _stream(self.device))
        self.graph = g
        return g

    def replay(self, expected: bytes | None = None) -> bool:
        """Replay the captured pass (against ``expected`` if given, else the captured one); returns the verdict."""
        if self.graph is None:
            raise RuntimeError("nothing captured: call capture() before replay()")
        if expected is not None:
            self.set_expected(expected)
        self.graph.replay()
        return self._verdict()


class Tree:
    """A persistent per-segment Merkle tree on the device (include/hv_incremental.h)."""

    def __init__(self, leaf_digests: torch.Tensor, seg_offsets, roots: torch.Tensor | None = None,
                 alg: str = "sha256"):
        self.code, D = _alg(alg)
        self.alg = alg
        self.seg = np.ascontiguousarray(seg_offsets, dtype=np.uint64)
        self.n_seg = len(self.seg) - 1
        self.device = leaf_digests.device
        nbytes = lib.hv_tree_bytes_alg(self.code, self.seg.ctypes.data, self.n_seg)
        if nbytes == 0:
            raise HVError(HV_ERR_INVALID_ARG, lib.hv_last_error().decode("utf-8", "replace"))
        self.D, self.n = D, int(self.seg[-1])
        leaves_ptr = _buffer(leaf_digests, self.n * D, "leaf_digests", self.device)
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.roots = roots if roots is not None else torch.empty((self.n_seg, D), dtype=torch.uint8,
                                                                 device=self.device)
        _buffer(self.roots, self.n_seg * D, "roots", self.device)
        self.ws = Workspace(self.device)
        _check(lib.hv_tree_build_alg(self.code, leaves_ptr if leaf_digests.numel() else None,
                                     self.seg.ctypes.data, self.n_seg, self.buf.data_ptr(), self.buf.numel(),
                                     self.roots.data_ptr(), _stream(self.device)))

    def update(self, leaf_digests: torch.Tensor, dirty) -> torch.Tensor:
        """Recompute the branches above the listed leaves (sorted unique leaf numbers); returns roots."""
        d = np.ascontiguousarray(dirty, dtype=np.uint64)
        leaves_ptr = _buffer(leaf_digests, self.n * self.D, "leaf_digests", self.device)
        ws = self.ws.get(lib.hv_tree_update_workspace_bytes(len(d)))
        _check(lib.hv_tree_update_alg(self.code, leaves_ptr if leaf_digests.numel() else None,
                                      self.seg.ctypes.data, self.n_seg, self.buf.data_ptr(), self.buf.numel(),
                                      d.ctypes.data if len(d) else None, len(d), self.roots.data_ptr(),
                                      ws.data_ptr(), ws.numel(), _stream(self.device)))
        return self.roots


def hv_rehash_chunks(msgs, chunk_bytes: int, leaves, leaf_digests: torch.Tensor, workspace: Workspace | None = None,
                     alg: str = "sha256"):
    """Recompute leaf_digests[j] for the listed leaf numbers j (sorted, unique) only."""
    code, D = _alg(alg)
    ptrs, lens = _ptr_len(msgs)
    arr = _msg_array(ptrs, lens)
    n = len(arr)
    _, n_leaves = _layout_of(arr, chunk_bytes)
    leaves_ptr = _buffer(leaf_digests, n_leaves * D, "leaf_digests", leaf_digests.device)
    lst = np.ascontiguousarray(leaves, dtype=np.uint64)
    ws = (workspace or Workspace(leaf_digests.device)).get(lib.hv_rehash_workspace_bytes(n, len(lst)))
    _check(lib.hv_rehash_chunks_alg(code, arr.ctypes.data if n else None, n, chunk_bytes,
                                    lst.ctypes.data if len(lst) else None, len(lst),
                                    leaves_ptr if leaf_digests.numel() else None,
                                    ws.data_ptr(), ws.numel(), _stream(leaf_digests.device)))
    return leaf_digests


class Monitor:
    """Continuous runtime monitoring of resident weights (include/hv_monitor.h).

    ``ref_digests`` are the leaf digests recorded when the weights were
    verified against their expected root ([n_leaves, D] device tensor, leaf
    order of ``hv_leaf_layout``).  Each ``scan`` rehashes ``slice_leaves``
    consecutive leaves on the monitor's own stream and compares them with
    their references; consecutive scans sweep the whole set round-robin.
    Each scan's result (mismatch count, lowest mismatching leaf) is copied on
    the monitor stream into a pinned host ring of ``ring`` slots, which
    ``poll`` reads once the scan's event has completed -- the monitor never
    waits on, or makes the host wait for, the work of other streams.
    """

    def __init__(self, msgs, chunk_bytes: int, ref_digests: torch.Tensor, alg: str = "sha256",
                 slice_leaves: int = 4096, device="cuda", stream=None, ring: int = 64):
        code, D = _alg(alg)
        self.device = torch.device(device)
        self.alg, self.D = alg, D
        ptrs, lens = _ptr_len(msgs)
        self.keepalive = msgs
        arr = _msg_array(ptrs, lens)
        n = len(arr)
        self.plan = hv_monitor_plan()
        if isinstance(stream, CuMaskedStream):
            stream._users.add(self)  # closed before the masked stream is destroyed
            stream = stream.stream
        self.stream = stream or torch.cuda.Stream(self.device)
        # the monitor's buffers are allocated on its own stream, which is the
        # only stream that uses them: the allocator then reuses their memory
        # in that stream's order, and the monitor never waits on other work
        with torch.cuda.stream(self.stream):
            self.plan_mem = Workspace(self.device).get(lib.hv_monitor_plan_bytes(n))
        _check(lib.hv_monitor_init(code, arr.ctypes.data if n else None, n, chunk_bytes, self.plan_mem.data_ptr(),
                                   self.plan_mem.numel(), ctypes.byref(self.plan), self.stream.cuda_stream))
        self.n_leaves = int(self.plan.n_leaves)
        if tuple(ref_digests.shape) != (self.n_leaves, D) or ref_digests.dtype != torch.uint8:
            raise ValueError(f"ref_digests must be uint8 [{self.n_leaves}, {D}]")
        _buffer(ref_digests, self.n_leaves * D, "ref_digests", self.device)
        self.ref = ref_digests
        self.slice = max(1, min(int(slice_leaves), max(self.n_leaves, 1)))
        with torch.cuda.stream(self.stream):
            self.ws = Workspace(self.device).get(lib.hv_monitor_scan_workspace_bytes(code, self.slice))
            self.results = torch.empty((ring, 2), dtype=torch.int64, device=self.device)
        self.host = torch.empty((ring, 2), dtype=torch.int64, pin_memory=True)
        self.events = [None] * ring
        self.ranges = [None] * ring
        self.next_leaf = 0
        self.issued = 0
        self.read = 0
        self.mismatches = []  # (first bad leaf, count, slice first, slice length) of each failing scan
        self.stream.wait_stream(torch.cuda.current_stream(self.device))  # ref_digests were made there
        self.stream.synchronize()  # the plan's upload and offsets are ready

    def scan(self, first: int, count: int, slice_digests: torch.Tensor | None = None) -> torch.Tensor:
        """Queue one scan of leaves [first, first + count) on the monitor stream; returns its result slot."""
        if self.events is None:
            raise RuntimeError("the monitor is closed")
        ring = len(self.events)
        slot = self.issued % ring
        while self.read <= self.issued - ring:  # the slot's previous result is still unread
            self.poll(wait=True, limit=1)
        res = self.results[slot]
        out_ptr = _buffer(slice_digests, count * self.D, "slice_digests", self.device) \
            if slice_digests is not None else None
        if count <= self.slice:
            ws = self.ws
        else:  # a one-off larger slice: scratch from the monitor stream's own pool
            with torch.cuda.stream(self.stream):
                ws = Workspace(self.device).get(lib.hv_monitor_scan_workspace_bytes(_alg(self.alg)[0], count))
        _check(lib.hv_monitor_scan(ctypes.byref(self.plan), first, count, self.ref.data_ptr(),
                                   out_ptr,
                                   res.data_ptr(), ws.data_ptr(), ws.numel(), self.stream.cuda_stream))
        with torch.cuda.stream(self.stream):
            self.host[slot].copy_(res, non_blocking=True)
        ev = torch.cuda.Event()
        ev.record(self.stream)
        self.events[slot] = ev
        self.ranges[slot] = (first, count)
        self.issued += 1
        return res

    def step(self) -> tuple:
        """Queue the next slice of the round-robin sweep; returns (first, count)."""
        first = self.next_leaf
        count = min(self.slice, self.n_leaves - first)
        self.scan(first, count)
        self.next_leaf = 0 if first + count >= self.n_leaves else first + count
        return first, count

    def sweep(self):
        """Queue scans covering every leaf once, from leaf 0."""
        self.next_leaf = 0
        for _ in range(-(-self.n_leaves // self.slice)):
            self.step()

    def close(self):
        """Read the results of every queued scan, then release the events, the
        pinned result ring and the device buffers, all of which refer to the
        monitor's stream (idempotent).  A monitor on a CU-masked stream is
        closed by that stream's ``close`` before the stream is destroyed."""
        if self.events is None:
            return
        self.poll(wait=True)
        self.stream.synchronize()
        self.events = self.ranges = None
        self.host = self.results = self.ws = self.plan_mem = None

    def poll(self, wait: bool = False, limit: int | None = None) -> int:
        """Read the results of completed scans, in issue order (waiting for
        each with wait=True), at most ``limit`` of them; returns how many were read."""
        done = 0
        if self.events is None:
            return done
        while self.read < self.issued and (limit is None or done < limit):
            slot = self.read % len(self.events)
            ev = self.events[slot]
            if wait:
                ev.synchronize()
            elif not ev.query():
                break
            cnt, first_bad = (int(v) for v in self.host[slot].tolist())
            if cnt:
                self.mismatches.append((first_bad & 0xFFFFFFFFFFFFFFFF, cnt) + self.ranges[slot])
            self.read += 1
            done += 1
        return done


def cu_mask_words(cus, n_cu: int) -> np.ndarray:
    """The 32-bit mask words selecting compute units ``cus`` of ``n_cu``."""
    words = np.zeros((n_cu + 31) // 32, dtype=np.uint32)
    for cu in cus:
        if not 0 <= cu < n_cu:
            raise ValueError(f"compute unit {cu} is not in 0..{n_cu - 1}")
        words[cu // 32] |= np.uint32(1 << (cu % 32))
    return words


class CuMaskedStream:
    """A stream whose kernels run only on the given compute units
    (include/hv_monitor.h), usable wherever torch takes a stream (``.stream``).

    Each such stream owns a hardware queue of its own, so it is destroyed
    explicitly, in this order, by ``close()`` (or by a context manager's exit):
    the ``Monitor`` objects made on it are closed (their events and pinned
    result rings released), the whole device is synchronized so every event
    torch recorded on the stream has completed, torch's pinned-memory cache
    releases the blocks whose reuse waited on such events, and then the
    stream is destroyed.  Any other object holding events of this stream
    (``torch.cuda.Event``, pinned tensors copied on it) must be dropped before
    ``close()``.  A stream still open when the interpreter exits is closed
    by an ``atexit`` hook, which runs before the HIP runtime's (and any
    profiler's) own exit handlers: the queue is never left to their teardown.
    """

    def __init__(self, cus, device="cuda"):
        self.device = torch.device(device)
        n_cu = torch.cuda.get_device_properties(self.device).multi_processor_count
        self.cus = sorted(set(int(c) for c in cus))
        words = cu_mask_words(self.cus, n_cu)
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(lib.hv_stream_create_cu_masked(words.ctypes.data, len(words), ctypes.byref(handle)))
        self.handle = handle.value
        self.stream = torch.cuda.ExternalStream(self.handle, device=self.device)
        self._users = weakref.WeakSet()
        atexit.register(self.close)

    def close(self):
        """Close the monitors made on this stream, wait for the device, release torch's
        pinned blocks that waited on the stream, and destroy it (idempotent)."""
        if self.handle is None:
            return
        for mon in list(self._users):
            mon.close()
        with torch.cuda.device(self.device):
            torch.cuda.synchronize(self.device)
            torch._C._host_emptyCache()
            _check(lib.hv_stream_destroy(self.handle))
        self.handle = None
        self.stream = None
        atexit.unregister(self.close)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def mask(self) -> np.ndarray:
        if self.handle is None:
            raise RuntimeError("the stream is closed")
        n_cu = torch.cuda.get_device_properties(self.device).multi_processor_count
        words = np.zeros((n_cu + 31) // 32, dtype=np.uint32)
        _check(lib.hv_stream_cu_mask(self.handle, words.ctypes.data, len(words)))
        return words


def verify_model(msgs, chunk_bytes: int, expected: bytes | None = None, alg: str = "sha256",
                 mode: str = "manifest", device="cuda") -> dict:
    """One synchronous verification through ``hv_verify_model``: {"integrity_verified",
    "root" (bytes), "verification_time_ns"}; a mismatch is a False verdict, not an error."""
    code, D = _alg(alg)
    if mode not in ("manifest", "single"):
        raise ValueError(mode)
    manifest = 1 if mode == "manifest" else 0
    if expected is not None and len(bytes(expected)) != D:
        raise ValueError(f"expected root must be {D} bytes for {alg}")
    ptrs, lens = _ptr_len(msgs)
    arr = _msg_array(ptrs, lens)
    n = len(arr)
    dev = torch.device(device)
    need = lib.hv_verify_model_workspace_bytes(code, arr.ctypes.data if n else None, n, chunk_bytes, manifest)
    if need == 0:
        raise HVError(HV_ERR_INVALID_ARG, lib.hv_last_error().decode("utf-8", "replace"))
    ws = Workspace(dev).get(need)
    exp = (ctypes.c_uint8 * D).from_buffer_copy(bytes(expected)) if expected is not None else None
    res = hv_result()
    _check(lib.hv_verify_model(code, arr.ctypes.data if n else None, n, chunk_bytes, manifest, exp, ws.data_ptr(),
                               ws.numel(), ctypes.byref(res), _stream(dev)))
    return {"integrity_verified": bool(res.integrity_verified), "root": bytes(res.root[:res.root_bytes]),
            "verification_time_ns": int(res.verification_time_ns)}


def manifest_root(named_tensors, chunk_bytes: int, alg: str = "sha256") -> bytes:
    """Manifest root of {name: tensor} (byte-wise name order) or [(name, tensor)] (given order)."""
    items = sorted(named_tensors.items(), key=lambda kv: kv[0].encode("utf-8")) \
        if isinstance(named_tensors, dict) else list(named_tensors)
    dev = items[0][1].device if items else torch.device("cuda")
    root = Verifier(dev, alg).manifest_root([t for _, t in items], chunk_bytes)
    return bytes(root.cpu().numpy().reshape(-1))


def verify(named_tensors, expected: bytes, chunk_bytes: int, alg: str = "sha256") -> None:
    """Raise VerificationError unless the manifest root of the tensors equals ``expected``."""
    items = sorted(named_tensors.items(), key=lambda kv: kv[0].encode("utf-8")) \
        if isinstance(named_tensors, dict) else list(named_tensors)
    v = Verifier(items[0][1].device if items else torch.device("cuda"), alg)
    root = v.manifest_root([t for _, t in items], chunk_bytes)
    if not v.verify_root(root, expected):
        raise VerificationError("model root does not match the expected root")
