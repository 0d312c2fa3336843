"""The library's exact rounding of Phi0 + delta (compiled for the host) against
exact rational round-half-to-even, including .5 ties and tiny deltas."""
import math
import os
import shutil
import struct
import subprocess
from fractions import Fraction

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _rne(x: Fraction) -> int:
    fl = math.floor(x)
    d = x - fl
    if d != Fraction(1, 2):
        return fl + (1 if d > Fraction(1, 2) else 0)
    return fl if fl % 2 == 0 else fl + 1


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("host") / "grid_round_host")
    src = os.path.join(ROOT, "tests", "host", "grid_round_host.hip")
    cmd = [hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17", "-I", os.path.join(ROOT, "paper_2406_06385_amd", "csrc"),
           src, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def _cases():
    rng = np.random.default_rng(1)
    out = []
    for f in (0, 1, 4, 5, 6):
        codes = list(range(-128, 128)) if f else list(range(-8, 8))
        for code in codes:
            for d in (0.0, 1e-9, -1e-9, 2.0 ** -30, -(2.0 ** -30), 1e-6, -1e-6, 0.03, -0.03, 0.49, -0.51):
                out.append((code, f, np.float32(d)))
        # exact half-integer crossings and random deltas
        for _ in range(3000):
            code = int(rng.integers(-128, 128)) if f else int(rng.integers(-8, 8))
            d = np.float32(rng.normal(0, 0.3) if rng.random() < 0.5 else rng.normal(0, 1e-6))
            out.append((code, f, d))
        for code in (codes[0], codes[-1], 0, 1):
            for k in (-2, -1, 1, 2):
                # delta that lands exactly on a .5 point of u
                v = Fraction(code, 2 ** f)
                target = math.floor(v) + k + Fraction(1, 2)
                d = np.float32(float(target - v))
                if Fraction(float(d)) == target - v:
                    out.append((code, f, d))
    return out


def test_grid_round_matches_exact_rne(driver):
    cases = _cases()
    lines = "".join(f"{c} {f} {struct.unpack('<I', struct.pack('<f', float(d)))[0]:x}\n" for c, f, d in cases)
    r = subprocess.run([driver], input=lines, capture_output=True, text=True)
    assert r.returncode == 0
    got = [tuple(int(t) for t in line.split()) for line in r.stdout.splitlines()]
    assert len(got) == len(cases)
    bad = []
    for (c, f, d), (g32, g64) in zip(cases, got):
        want = _rne(Fraction(c, 2 ** f) + Fraction(float(d)))
        if g32 != want or g64 != want:
            bad.append((c, f, float(d), g32, g64, want))
    assert not bad, bad[:10]
