"""The C client of the ABI (tests/c_client/verify_example.c: hipMalloc'd
buffers, the hv.h calls and hv_verify_model, no Python in the process) gives
the oracle's manifest roots for SHA-256 and SHA-384."""
import os
import subprocess

import numpy as np
import pytest

from conftest import ROOT
from oracle import oracle

pytestmark = pytest.mark.gpu
EXE = os.path.join(ROOT, "tests", "c_client", "verify_example")


def pattern(m: int, n: int) -> bytes:
    # byte i of message m, as the C client writes it
    return ((np.arange(n, dtype=np.uint64) * 131 + 7 * m + 1) & 0xFF).astype(np.uint8).tobytes()


@pytest.mark.parametrize("C,lens", [(4096, [0, 1, 5000, 70000, 4096]), (1024, [3, 300000]), (0, [10, 0, 2048, 99])])
def test_c_client_roots_equal_the_oracle(C, lens):
    if not os.path.exists(EXE):
        raise FileNotFoundError(f"{EXE} is not built; run __graft_entry__.build()")
    out = subprocess.run([EXE, str(C)] + [str(n) for n in lens], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    lines = dict((ln.split()[0], ln.split()[1:]) for ln in out.stdout.strip().splitlines())
    msgs = [pattern(m, n) for m, n in enumerate(lens)]
    for alg in ("sha256", "sha384"):
        roots = [oracle.seg_root_alg(m, C, alg) for m in msgs]
        want = oracle.mth(roots, alg)
        root_hex, verdict = lines[alg]
        assert root_hex == want.hex(), alg
        assert verdict == "1"
