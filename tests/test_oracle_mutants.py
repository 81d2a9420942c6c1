"""Planted mistakes in the oracle are caught by its pins.

Each case copies ``oracle/hv_oracle.c`` with one plausible mistake planted (a
wrong rotate or shift amount, a dropped term, a wrong index, prefix or split,
an off-by-one in the padding or the chunking, transposed operands, a wrong
constant), builds the copy with the host compiler and runs compact forms of
the pins against it (``oracle_mutants/pins.py``: hashlib at every length,
an independent bottom-up tree, chunk slices, the threaded driver) in a child
process.  Every mutant must fail them -- a crash of the child counts as
caught -- and the unmodified source must pass.  Mistakes are planted only in
copies, on the CPU; the oracle itself is untouched.

The Python helpers that compose the C primitives (per-message roots from a
leaf array, the per-message root for either hash, the tree over a digest
array, the packed driver, the closed form) get the same treatment: copies of
``oracle/oracle.py`` with one mistake each are imported in a child process
and run against ``oracle_mutants/py_pins.py``.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "hv_oracle.c")
PINS = os.path.join(ROOT, "tests", "oracle_mutants", "pins.py")
PY_SRC = os.path.join(ROOT, "oracle", "oracle.py")
PY_PINS = os.path.join(ROOT, "tests", "oracle_mutants", "py_pins.py")

# (name, text in hv_oracle.c, replacement, which occurrence of the text)
MUTANTS = [
    ("Sigma0 rotate 13 -> 12", "ROTR(x, 2) ^ ROTR(x, 13) ^ ROTR(x, 22)", "ROTR(x, 2) ^ ROTR(x, 12) ^ ROTR(x, 22)", 0),
    ("sigma1 shift 10 -> 9", "ROTR(x, 17) ^ ROTR(x, 19) ^ SHR(x, 10)", "ROTR(x, 17) ^ ROTR(x, 19) ^ SHR(x, 9)", 0),
    ("Ch without the complement", "return (x & y) ^ (~x & z); }", "return (x & y) ^ (x & z); }", 0),
    ("Maj missing a term", "return (x & y) ^ (x & z) ^ (y & z); }", "return (x & y) ^ (x & z); }", 0),
    ("last round constant", "0xc67178f2u", "0xc67178f3u", 0),
    ("schedule index t-7 -> t-6", "+ W[t - 7] +", "+ W[t - 6] +", 0),
    ("e takes c instead of d", "e = d + T1;", "e = c + T1;", 0),
    ("feed-forward of h dropped", "H[7] += h;", "H[7] += 0;", 0),
    ("padding stops at 55", "while (s->used != 56)", "while (s->used != 55)", 0),
    ("length field little-endian", "(uint8_t)(bits >> (56 - 8 * i))", "(uint8_t)(bits >> (8 * i))", 0),
    ("length in bytes, not bits", "uint64_t bits = s->total * 8u;", "uint64_t bits = s->total;", 0),
    ("tree split at the largest power of two <= n", "while (k * 2 < n) k *= 2;", "while (k * 2 <= n) k *= 2;", 0),
    ("leaf prefix 0x01", "sha256_prefixed(0x00, entries, 32, out)", "sha256_prefixed(0x01, entries, 32, out)", 0),
    ("interior prefix dropped", "sha256_prefixed(0x01, lr, 64, out);", "oracle_sha256(lr, 64, out);", 0),
    ("empty tree as a leaf", "if (n == 0) { oracle_sha256(NULL, 0, out); return; }",
     "if (n == 0) { sha256_prefixed(0x00, NULL, 0, out); return; }", 0),
    ("subtrees transposed", "oracle_mth(entries, k, lr);\n    oracle_mth(entries + 32 * k, n - k, lr + 32);",
     "oracle_mth(entries, k, lr + 32);\n    oracle_mth(entries + 32 * k, n - k, lr);", 0),
    ("chunk count rounds up always", "return len / C + (len % C != 0);", "return len / C + 1;", 0),
    ("chunk start off by one", "uint64_t lo = i * C;", "uint64_t lo = i * C + (i > 0);", 0),
    ("SHA-384 Sigma0 rotate 39 -> 38", "ROTR64(x, 28) ^ ROTR64(x, 34) ^ ROTR64(x, 39)",
     "ROTR64(x, 28) ^ ROTR64(x, 34) ^ ROTR64(x, 38)", 0),
    ("SHA-384 sigma0 shift 7 -> 6", "ROTR64(x, 1) ^ ROTR64(x, 8) ^ (x >> 7)", "ROTR64(x, 1) ^ ROTR64(x, 8) ^ (x >> 6)", 0),
    ("SHA-384 initial value", "0xcbbb9d5dc1059ed8ull", "0xcbbb9d5dc1059ed9ull", 0),
    ("SHA-512 feed-forward of h dropped", "H[7] += h;", "H[7] += 0;", 1),
    ("SHA-384 padding stops at 111", "while (s->used != 112)", "while (s->used != 111)", 0),
    ("SHA-384 tree split", "while (k * 2 < n) k *= 2;\n    uint8_t lr[96];", "while (k * 2 <= n) k *= 2;\n    uint8_t lr[96];", 0),
    ("threaded driver writes leaf L to slot L-1",
     "else oracle_sha256(p + lo, hi - lo, j->out + 32 * L);",
     "else oracle_sha256(p + lo, hi - lo, j->out + 32 * (L ? L - 1 : 0));", 0),
]


def build(src_text: str, out_dir) -> str:
    c = os.path.join(out_dir, "hv_oracle.c")
    so = os.path.join(out_dir, "liboracle_mutant.so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O1", "-std=c99", "-fPIC", "-shared", "-pthread", c, "-o", so], check=True,
                   capture_output=True)
    return so


def pins_pass(so: str) -> subprocess.CompletedProcess:
    return subprocess.run([sys.executable, PINS, so], capture_output=True, text=True, timeout=120)


def plant(text: str, old: str, new: str, occurrence: int) -> str:
    at = -1
    for _ in range(occurrence + 1):
        at = text.find(old, at + 1)
        assert at >= 0, f"the mutation target {old!r} is not in the oracle (occurrence {occurrence})"
    return text[:at] + new + text[at + len(old):]


def test_unmodified_oracle_passes_the_pins(tmp_path):
    r = pins_pass(build(open(SRC).read(), tmp_path))
    assert r.returncode == 0, r.stderr


@pytest.mark.parametrize("name,old,new,occurrence", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, old, new, occurrence, tmp_path):
    text = plant(open(SRC).read(), old, new, occurrence)
    r = pins_pass(build(text, tmp_path))
    assert r.returncode != 0, f"the pins did not catch: {name}"


# (name, text in oracle.py, replacement, which occurrence of the text)
PY_MUTANTS = [
    ("per-message roots: position never advances", "        pos += c\n", "", 0),
    ("per-message roots: one leaf too many", "mth(leaves[pos:pos + c], alg)", "mth(leaves[pos:pos + c + 1], alg)", 0),
    ("per-message roots: tree always SHA-256", "roots.append(mth(leaves[pos:pos + c], alg))",
     "roots.append(mth(leaves[pos:pos + c]))", 0),
    ("seg_root_alg: chunk digests always SHA-256", "return mth(chunk_digests_alg(data, C, alg), alg)",
     "return mth(chunk_digests_alg(data, C), alg)", 0),
    ("seg_root_alg: tree always SHA-256", "return mth(chunk_digests_alg(data, C, alg), alg)",
     "return mth(chunk_digests_alg(data, C, alg))", 0),
    ("mth: list entries joined in reverse", 'b"".join(entries)', 'b"".join(entries[::-1])', 0),
    ("mth: array read in memory order, not row order", "e = np.ascontiguousarray(entries, dtype=np.uint8).reshape(-1)",
     "e = np.frombuffer(np.asarray(entries).base.tobytes() if np.asarray(entries).base is not None "
     "else np.asarray(entries).tobytes(), dtype=np.uint8)[:np.asarray(entries).size]", 0),
    ("digest: hashes swapped", 'return sha256(data) if alg == "sha256" else sha384(data)',
     'return sha384(data)[:32] if alg == "sha256" else sha384(data)', 0),
    ("packed driver ignores offsets", "ptrs = np.uint64(b.ctypes.data) + offsets",
     "ptrs = np.uint64(b.ctypes.data) + offsets * np.uint64(0)", 0),
    ("closed form: tail digest of a whole chunk", "T = sha256(bytes([byte]) * tail) if tail else None",
     "T = sha256(bytes([byte]) * C) if tail else None", 0),
    ("closed form: split at the largest power of two <= n", "while k * 2 < n:", "while k * 2 <= n:", 0),
    ("chunk size not checked against the block", "if n == UINT64_MAX or (C % ALGS[alg][2]):",
     "if n == UINT64_MAX:", 0),
]


def py_copy(text: str, out_dir) -> str:
    """A package ``oracle`` under out_dir holding text as oracle.py and the built C oracle."""
    from oracle import oracle as real

    real._load()  # the copy loads the library built from the unmodified C source
    pkg = os.path.join(out_dir, "oracle")
    os.makedirs(pkg)
    open(os.path.join(pkg, "__init__.py"), "w").close()
    with open(os.path.join(pkg, "oracle.py"), "w") as f:
        f.write(text)
    os.symlink(os.path.join(ROOT, "oracle", "liboracle.so"), os.path.join(pkg, "liboracle.so"))
    return str(out_dir)


def py_pins_pass(pkg_dir: str) -> subprocess.CompletedProcess:
    return subprocess.run([sys.executable, PY_PINS, pkg_dir], capture_output=True, text=True, timeout=120,
                          cwd=pkg_dir)


def test_unmodified_python_helpers_pass_the_pins(tmp_path):
    r = py_pins_pass(py_copy(open(PY_SRC).read(), tmp_path))
    assert r.returncode == 0, r.stderr


@pytest.mark.parametrize("name,old,new,occurrence", PY_MUTANTS, ids=[m[0] for m in PY_MUTANTS])
def test_planted_python_mistake_is_caught(name, old, new, occurrence, tmp_path):
    text = plant(open(PY_SRC).read(), old, new, occurrence)
    r = py_pins_pass(py_copy(text, tmp_path))
    assert r.returncode == 1, f"the pins did not catch: {name} (exit {r.returncode}: {r.stderr[-400:]})"
