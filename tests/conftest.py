import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


class Pat:
    """Plain pattern record (kind, H, W, p0, p1) used by the oracle tests."""

    def __init__(self, kind, H, W, p0, p1=0):
        self.kind, self.H, self.W, self.p0, self.p1 = kind, int(H), int(W), int(p0), int(p1)

    @property
    def N(self):
        return self.H * self.W

    @property
    def hilbert(self):
        return self.kind.startswith("hilbert")

    def __repr__(self):
        return f"Pat({self.kind},{self.H}x{self.W},{self.p0},{self.p1})"


def read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            head, _, source = line.partition("  ")
            rows.append((head.split(), source.strip()))
    return rows
