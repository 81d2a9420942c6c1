"""Compact pins of the oracle's Python helpers, run against a given copy of
``oracle/oracle.py``.

Usage: python py_pins.py <directory holding the package ``oracle``>
Exit status 0 when every pin holds, 1 (with the first failure on stderr)
otherwise.  References: hashlib, plain slices of each message for Algorithm
1's chunking, and a bottom-up RFC 6962 tree written here.  Used by
test_oracle_mutants.py, which runs it in a child process per copy.
"""
import hashlib
import os
import sys

import numpy as np

HASHES = {"sha256": (hashlib.sha256, 32), "sha384": (hashlib.sha384, 48)}


def slices(m, C):
    return [m] if C == 0 else [m[i:i + C] for i in range(0, len(m), C)]


def tree(entries, h):
    if not entries:
        return h(b"").digest()
    level = [h(b"\x00" + d).digest() for d in entries]
    while len(level) > 1:
        nxt = [h(b"\x01" + level[i] + level[i + 1]).digest() for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def main(pkg_dir: str) -> int:
    sys.path.insert(0, pkg_dir)
    from oracle import oracle

    if not os.path.abspath(oracle.__file__).startswith(os.path.abspath(pkg_dir)):
        print(f"imported {oracle.__file__}, not the copy under {pkg_dir}", file=sys.stderr)
        return 2

    def fail(what):
        print(what, file=sys.stderr)
        return 1

    rng = np.random.default_rng(2510)
    lens = [0, 1, 128, 0, 129, 1000, 640, 4096 + 17, 0]
    msgs = [rng.integers(0, 256, n, dtype=np.uint8).tobytes() for n in lens]
    for alg, (h, D) in HASHES.items():
        for C in (128, 256, 0):
            per = [[h(s).digest() for s in slices(m, C)] for m in msgs]
            leaves = np.frombuffer(b"".join(d for p in per for d in p), dtype=np.uint8).reshape(-1, D)
            counts = np.array([len(p) for p in per], dtype=np.uint64)
            if oracle.seg_roots_from_leaves(leaves, counts, alg) != [tree(p, h) for p in per]:
                return fail(f"per-message roots ({alg}, C = {C}) differ from per-message trees")
            for m, p in zip(msgs, per):
                if oracle.seg_root_alg(m, C, alg) != tree(p, h):
                    return fail(f"seg_root_alg ({alg}, C = {C}, {len(m)} bytes) differs")
        for n in (0, 1, 2, 3, 5, 8, 13):
            arr = rng.integers(0, 256, (2 * n, D), dtype=np.uint8)
            for a in (arr[:n], arr[::2]):
                want = tree([bytes(r) for r in a], h)
                if oracle.mth(a, alg) != want or oracle.mth([bytes(r) for r in a], alg) != want:
                    return fail(f"mth over {n} {D}-byte entries ({alg}) differs from the bottom-up tree")
        for m in msgs[:6]:
            if oracle.digest(m, alg) != h(m).digest():
                return fail(f"digest ({alg}) differs from hashlib")
        # packed messages in one buffer at offsets
        buf = rng.integers(0, 256, 6000, dtype=np.uint8)
        offs, lns = [0, 64, 700, 701, 3000], [10, 600, 0, 1500, 2999]
        want = [h(buf[o:o + n].tobytes()).digest() for o, n in zip(offs, lns)]
        got = oracle.leaf_digests_mt_packed(buf, offs, lns, 0, 2, alg)
        if [bytes(r) for r in got] != want:
            return fail(f"packed driver ({alg}) differs from hashlib per message")
    # the closed form for constant bytes equals the plain root
    for L, C, b in ((0, 64, 7), (64 * 5, 64, 0), (64 * 9 + 3, 64, 255), (1000, 0, 1), (64 * 33 + 1, 128, 9)):
        if oracle.const_seg_root(L, C, b) != oracle.seg_root(bytes([b]) * L, C):
            return fail(f"closed form differs from the plain root ({L} bytes, C = {C})")
    # SHA-384 chunks must be whole 128-byte blocks
    try:
        oracle.chunk_count(1000, 64, "sha384")
        return fail("a 64-byte SHA-384 chunk size was accepted")
    except ValueError:
        pass
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1]))
