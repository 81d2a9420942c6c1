"""Python driver for the CPU oracle (``hv_oracle.c``).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module.  It never imports
the HIP package and shares no code with it.

Every function here is either a thin ctypes call into ``hv_oracle.c`` or a
composition of those calls that follows the paper directly:

* ``seg_root``      -- Algorithm 1 (Discussion, "Streaming Model Verification
  for Large Models"): chunk the message, hash each chunk, build the Merkle
  tree over the chunk hashes (RFC 6962, cited in the Introduction).
* ``manifest_root`` -- the hierarchical roots of the Introduction
  ("Hierarchical Integrity Verification"): a tree over per-tensor roots, in
  the order the caller lists the tensors.
* ``const_seg_root`` -- the same MTH for a message whose bytes are all equal,
  evaluated with memoisation (RFC 6962's recursion only ever meets a few
  distinct sub-lists there), so 100 GB-sized shapes can be pinned in
  milliseconds.
"""
from __future__ import annotations

import ctypes
import os
from functools import lru_cache

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

u8p = ctypes.POINTER(ctypes.c_uint8)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from oracle.build import build

        build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_sha256.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    lib.oracle_sha256.restype = None
    lib.oracle_constants.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_constants.restype = None
    lib.oracle_chunk_count.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.oracle_chunk_count.restype = ctypes.c_uint64
    lib.oracle_chunk_digests.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p]
    lib.oracle_chunk_digests.restype = None
    lib.oracle_mth.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    lib.oracle_mth.restype = None
    lib.oracle_seg_root.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p]
    lib.oracle_seg_root.restype = None
    lib.oracle_leaf_digests_mt.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int,
    ]
    lib.oracle_leaf_digests_mt.restype = ctypes.c_uint64
    lib.oracle_leaf_digests_alg_mt.argtypes = [
        ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int,
    ]
    lib.oracle_leaf_digests_alg_mt.restype = ctypes.c_uint64
    lib.oracle_sha384.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    lib.oracle_sha384.restype = None
    lib.oracle_mth384.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    lib.oracle_mth384.restype = None
    lib.oracle_constants512.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_constants512.restype = None
    _lib = lib
    return lib


def _as_u8(data) -> np.ndarray:
    """A C-contiguous uint8 view of bytes / bytearray / numpy data."""
    if isinstance(data, (bytes, bytearray, memoryview)):
        return np.frombuffer(bytes(data), dtype=np.uint8)
    arr = np.ascontiguousarray(data)
    return arr.reshape(-1).view(np.uint8)


def _ptr(arr: np.ndarray):
    return arr.ctypes.data if arr.size else None


UINT64_MAX = (1 << 64) - 1


def constants():
    """(K[0..63], H0[0..7]) exactly as the oracle holds them (FIPS 180-4 4.2.2, 5.3.3)."""
    K = np.zeros(64, dtype=np.uint32)
    H = np.zeros(8, dtype=np.uint32)
    _load().oracle_constants(K.ctypes.data, H.ctypes.data)
    return [int(x) for x in K], [int(x) for x in H]


ALGS = {"sha256": (0, 32, 64), "sha384": (1, 48, 128)}  # id, digest bytes, block bytes


def constants512():
    """(K[0..79], H0[0..7]) of SHA-512 / SHA-384 exactly as the oracle holds them (FIPS 180-4 4.2.3, 5.3.4)."""
    K = np.zeros(80, dtype=np.uint64)
    H = np.zeros(8, dtype=np.uint64)
    _load().oracle_constants512(K.ctypes.data, H.ctypes.data)
    return [int(x) for x in K], [int(x) for x in H]


def sha384(data) -> bytes:
    """FIPS 180-4 SHA-384 of the bytes."""
    a = _as_u8(data)
    out = np.zeros(48, dtype=np.uint8)
    _load().oracle_sha384(_ptr(a), a.size, out.ctypes.data)
    return out.tobytes()


def digest(data, alg: str = "sha256") -> bytes:
    return sha256(data) if alg == "sha256" else sha384(data)


def sha256(data) -> bytes:
    """FIPS 180-4 SHA-256 of the bytes."""
    a = _as_u8(data)
    out = np.zeros(32, dtype=np.uint8)
    _load().oracle_sha256(_ptr(a), a.size, out.ctypes.data)
    return out.tobytes()


def chunk_count(length: int, C: int, alg: str = "sha256") -> int:
    """Algorithm 1's chunk_count = ceil(|M| / C); C = 0: one chunk (the whole message).
    C must be a multiple of the hash's block (64 bytes for SHA-256, 128 for SHA-384)."""
    n = _load().oracle_chunk_count(length, C)
    if n == UINT64_MAX or (C % ALGS[alg][2]):
        raise ValueError(f"chunk size {C} is not a multiple of {ALGS[alg][2]}")
    return int(n)


def chunk_digests(data, C: int) -> np.ndarray:
    """[n, 32] uint8: SHA-256 of each chunk, in chunk order."""
    a = _as_u8(data)
    n = chunk_count(a.size, C)
    out = np.zeros((n, 32), dtype=np.uint8)
    if n:
        _load().oracle_chunk_digests(_ptr(a), a.size, C, out.ctypes.data)
    return out


def mth(entries, alg: str = "sha256") -> bytes:
    """RFC 6962 Merkle Tree Hash over 32-byte (SHA-256) or 48-byte (SHA-384)
    entries ([n, D] uint8 or list of bytes)."""
    D = ALGS[alg][1]
    if isinstance(entries, (list, tuple)):
        e = np.frombuffer(b"".join(entries), dtype=np.uint8) if entries else np.zeros(0, np.uint8)
    else:
        e = np.ascontiguousarray(entries, dtype=np.uint8).reshape(-1)
    assert e.size % D == 0
    out = np.zeros(D, dtype=np.uint8)
    f = _load().oracle_mth if alg == "sha256" else _load().oracle_mth384
    f(_ptr(e), e.size // D, out.ctypes.data)
    return out.tobytes()


def seg_root(data, C: int) -> bytes:
    """Root of one message: MTH over the SHA-256 digests of its chunks."""
    a = _as_u8(data)
    chunk_count(a.size, C)  # validates C
    out = np.zeros(32, dtype=np.uint8)
    _load().oracle_seg_root(_ptr(a), a.size, C, out.ctypes.data)
    return out.tobytes()


def manifest_root(messages, C: int) -> bytes:
    """MTH over the per-message roots, in the order given."""
    return mth([seg_root(m, C) for m in messages])


def leaf_digests_mt(messages, C: int, nthreads: int, alg: str = "sha256") -> np.ndarray:
    """[n_leaves, D]: chunk digests of all messages (message-major), on nthreads threads."""
    arrs = [_as_u8(m) for m in messages]
    ptrs = np.array([a.ctypes.data if a.size else 0 for a in arrs], dtype=np.uint64)
    lens = np.array([a.size for a in arrs], dtype=np.uint64)
    return _leaf_digests_raw(ptrs, lens, C, nthreads, alg)


def leaf_digests_mt_packed(buf: np.ndarray, offsets, lens, C: int, nthreads: int, alg: str = "sha256") -> np.ndarray:
    """As leaf_digests_mt for messages lying in one host buffer at byte offsets."""
    b = _as_u8(buf)
    offsets = np.asarray(offsets, dtype=np.uint64)
    lens = np.asarray(lens, dtype=np.uint64)
    if len(lens) and int((offsets + lens).max()) > b.size:
        raise ValueError("message range outside the buffer")
    ptrs = np.uint64(b.ctypes.data) + offsets
    return _leaf_digests_raw(ptrs, lens, C, nthreads, alg)


def _leaf_digests_raw(ptrs: np.ndarray, lens: np.ndarray, C: int, nthreads: int, alg: str = "sha256") -> np.ndarray:
    n = len(lens)
    alg_id, D, _ = ALGS[alg]
    if C != 0:
        chunk_count(0, C, alg)  # validates C
        total = int(np.sum(lens // np.uint64(C) + (lens % np.uint64(C) != 0))) if n else 0
    else:
        total = n
    out = np.zeros((total, D), dtype=np.uint8)
    got = _load().oracle_leaf_digests_alg_mt(alg_id, ptrs.ctypes.data if n else None, lens.ctypes.data if n else None,
                                             n, C, out.ctypes.data if total else None, nthreads)
    if got != total:
        raise RuntimeError("oracle_leaf_digests_mt failed")
    return out


def seg_roots_from_leaves(leaves: np.ndarray, counts, alg: str = "sha256") -> list:
    """Per-message roots from a message-major leaf array and per-message leaf counts."""
    roots, pos = [], 0
    for c in counts:
        roots.append(mth(leaves[pos:pos + c], alg))
        pos += c
    return roots


def chunk_digests_alg(data, C: int, alg: str = "sha256") -> np.ndarray:
    """[n, D]: digest of each chunk in chunk order, for either hash."""
    return leaf_digests_mt([data], C, 1, alg)


def seg_root_alg(data, C: int, alg: str = "sha256") -> bytes:
    """Root of one message for either hash: MTH over its chunk digests."""
    return mth(chunk_digests_alg(data, C, alg), alg)


def const_seg_root(length: int, C: int, byte: int) -> bytes:
    """seg_root of ``length`` copies of one byte value, without materialising it.

    With every byte equal, all full chunks share one digest D and the tail
    chunk (if any) has digest T, so the entry list is D * f (+ [T]).  RFC 6962's
    recursion splits such a list at a power of two into another list of the
    same form, so memoising on (count, has-tail) leaves O(log^2 n) hashes.
    """
    n = chunk_count(length, C)
    if C == 0:
        return mth([sha256(bytes([byte]) * length)])
    if n == 0:
        return mth([])
    full = length // C
    tail = length - full * C
    D = sha256(bytes([byte]) * C)
    T = sha256(bytes([byte]) * tail) if tail else None
    return _uniform_mth(full, D, T)


def _uniform_mth(full: int, D: bytes, T):
    leaf = _node_leaf

    @lru_cache(maxsize=None)
    def rec(count: int, with_tail: bool) -> bytes:
        n = count + (1 if with_tail else 0)
        if n == 1:
            return leaf(T if with_tail else D)
        k = 1
        while k * 2 < n:
            k *= 2
        # left: the first k entries (all D, since k < n and the tail is last)
        left = rec(k, False)
        right = rec(count - k, with_tail)
        return _node_interior(left, right)

    return rec(full, T is not None)


def _node_leaf(d: bytes) -> bytes:
    return sha256(b"\x00" + d)


def _node_interior(left: bytes, right: bytes) -> bytes:
    return sha256(b"\x01" + left + right)
