import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def load_golden(name):
    """Rows of a whitespace-separated golden file, comments skipped."""
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def golden_message(spec: str) -> bytes:
    kind, _, rest = spec.partition(":")
    if kind == "ascii":
        return rest.encode("ascii")
    if kind == "repeat":
        ch, _, count = rest.partition(":")
        return ch.encode("ascii") * int(count)
    raise ValueError(spec)
