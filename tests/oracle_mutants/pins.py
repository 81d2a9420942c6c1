"""Compact forms of the oracle's pins, run against a given build of hv_oracle.c.

Usage: python pins.py <path to a shared library built from hv_oracle.c>
Exit status 0 when every pin holds, 1 (with the first failure on stderr)
otherwise.  The references are independent of the oracle: Python's hashlib
for SHA-256 and SHA-384, slices of the message for the chunking rule, and a
bottom-up tree over hashlib (pairs hashed with the 0x01 prefix, an unpaired
last node moved up unchanged) for RFC 6962's tree.  Used by
test_oracle_mutants.py, which runs it in a child process per build.
"""
import ctypes
import hashlib
import random
import sys


def main(path: str) -> int:
    lib = ctypes.CDLL(path)
    vp, u64, u32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32
    for name in ("oracle_sha256", "oracle_sha384", "oracle_mth", "oracle_mth384"):
        getattr(lib, name).argtypes = [vp, u64, vp]
        getattr(lib, name).restype = None
    lib.oracle_chunk_count.argtypes = [u64, u64]
    lib.oracle_chunk_count.restype = u64
    lib.oracle_chunk_digests.argtypes = [vp, u64, u64, vp]
    lib.oracle_chunk_digests.restype = None
    lib.oracle_leaf_digests_alg_mt.argtypes = [ctypes.c_int, vp, vp, u32, u64, vp, ctypes.c_int]
    lib.oracle_leaf_digests_alg_mt.restype = u64

    rng = random.Random(2510)
    data = bytes(rng.getrandbits(8) for _ in range(10000))  # covers every message below

    def call(fn, msg, size, count=None):
        """fn(bytes, count, out): count is the byte length for a hash, the entry count for a tree."""
        out = ctypes.create_string_buffer(size)
        buf = ctypes.create_string_buffer(msg, len(msg)) if msg else None
        fn(buf, len(msg) if count is None else count, out)
        return out.raw

    def fail(what):
        print(what, file=sys.stderr)
        return 1

    # the hashes at every length 0..300 and across block boundaries up to 3 blocks
    for n in list(range(301)) + [383, 384, 447, 448, 511, 512, 513]:
        m = data[:n]
        if call(lib.oracle_sha256, m, 32) != hashlib.sha256(m).digest():
            return fail(f"SHA-256 differs from hashlib at length {n}")
        if call(lib.oracle_sha384, m, 48) != hashlib.sha384(m).digest():
            return fail(f"SHA-384 differs from hashlib at length {n}")

    # RFC 6962's tree against a bottom-up build, n = 0..40 entries
    for h, D, fn in ((hashlib.sha256, 32, lib.oracle_mth), (hashlib.sha384, 48, lib.oracle_mth384)):
        for n in range(41):
            entries = data[: n * D]
            if n == 0:
                want = h(b"").digest()
            else:
                level = [h(b"\x00" + entries[D * i:D * (i + 1)]).digest() for i in range(n)]
                while len(level) > 1:
                    nxt = [h(b"\x01" + level[i] + level[i + 1]).digest() for i in range(0, len(level) - 1, 2)]
                    if len(level) % 2:
                        nxt.append(level[-1])
                    level = nxt
                want = level[0]
            if call(fn, entries, D, n) != want:
                return fail(f"tree of {n} {D}-byte entries differs from the bottom-up build")

    # chunking: ceil(len / C) chunks, each the plain hash of its slice; C = 0 is the whole message
    for L in (0, 1, 63, 64, 65, 200, 4103):
        for C in (64, 128, 0):
            n = lib.oracle_chunk_count(L, C)
            want_n = 1 if C == 0 else -(-L // C)
            if n != want_n:
                return fail(f"chunk count of {L} bytes with C = {C}: {n}, not {want_n}")
            m = data[:L]
            out = ctypes.create_string_buffer(32 * max(n, 1))
            lib.oracle_chunk_digests(ctypes.create_string_buffer(m, max(L, 1)), L, C, out)
            slices = [m] if C == 0 else [m[i:i + C] for i in range(0, L, C)]
            if out.raw[:32 * n] != b"".join(hashlib.sha256(s).digest() for s in slices):
                return fail(f"chunk digests of {L} bytes with C = {C} differ from hashlib per slice")

    # the threaded driver: both hashes, several messages, three threads
    lens = [0, 1, 130, 4096, 1000, 257]
    msgs = [data[sum(lens[:i]):sum(lens[:i]) + L] for i, L in enumerate(lens)]
    bufs = [ctypes.create_string_buffer(m, max(len(m), 1)) for m in msgs]
    ptrs = (ctypes.c_void_p * len(msgs))(*[ctypes.addressof(b) for b in bufs])
    lens_c = (ctypes.c_uint64 * len(msgs))(*lens)
    for alg, h, D, C in ((0, hashlib.sha256, 32, 128), (1, hashlib.sha384, 48, 128), (0, hashlib.sha256, 32, 0)):
        want = []
        for m in msgs:
            want += [h(m).digest()] if C == 0 else [h(m[i:i + C]).digest() for i in range(0, len(m), C)]
        out = ctypes.create_string_buffer(D * len(want))
        n = lib.oracle_leaf_digests_alg_mt(alg, ptrs, lens_c, len(msgs), C, out, 3)
        if n != len(want) or out.raw != b"".join(want):
            return fail(f"threaded driver (hash {alg}, C = {C}) differs from hashlib per chunk")
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1]))
