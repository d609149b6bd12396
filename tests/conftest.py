import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    """Fields of a tests/golden fixture: `key: v1 v2 ...` lines, '#' comments.
    Values are ints where they parse as ints, floats otherwise."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, vals = line.split(":", 1)
            parsed = []
            for v in vals.split():
                try:
                    parsed.append(int(v))
                except ValueError:
                    parsed.append(float(v))
            out[key.strip()] = parsed
    return out
