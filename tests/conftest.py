import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP library)")


def read_golden(name):
    """Parse a tests/golden fixture: 'key: values' lines, '#' comments."""
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, val = line.partition(":")
            out.setdefault(key.strip(), []).append(val.split())
    return out


def cond_err(y, ref, mag):
    """Largest error of y against the fp64 reference, relative to
    max(|ref|, magnitude companion): the rounding error any order of the
    sums can make scales with the companion, so this is the plain relative
    error wherever the sums do not cancel."""
    import numpy as np
    y = np.asarray(y)
    ref = np.asarray(ref)
    den = np.maximum(np.abs(ref), np.asarray(mag))
    den = np.where(den > 0, den, 1.0)
    err = np.abs(y.astype(ref.dtype) - ref) / den
    return float(err.max()) if err.size else 0.0


def announce(msg):
    """Name the case before a GPU step (a fault ends the process)."""
    print("\n[case] " + msg, flush=True)


class forced_fallback:
    """Within the block, every look-back of the return, GAE and TBB kernels
    that finds its predecessor unpublished computes that predecessor's
    summary itself (test-only control of the library)."""

    def __enter__(self):
        from paper_2402_09900_amd import binding
        self._lib = binding
        self._old = binding.memoroid_testing_set_fallback_polls(0)
        return self

    def __exit__(self, *exc):
        self._lib.memoroid_testing_set_fallback_polls(self._old)
        return False
