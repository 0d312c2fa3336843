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


@pytest.fixture(scope="module")
def swar_driver(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("host") / "swar_grid_host")
    src = os.path.join(ROOT, "tests", "host", "swar_grid_host.hip")
    cmd = [hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17", "-I", os.path.join(ROOT, "paper_2406_06385_amd", "csrc"),
           src, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_byte_parallel_grid_matches_exact_rounding(swar_driver):
    """Four Q8 codes per word, delta of a known sign and magnitude below 2^-f:
    each byte's nibble (b <= 4) or whole byte (b >= 5) equals
    round-half-even(code 2^-f + delta) on the grid,
    and exactly the codes that would leave the grid are marked for clipping."""
    rng = np.random.default_rng(7)
    cases = []
    for b in (7, 6, 5, 4, 3, 2):
        f = 8 - b
        for code in range(-128, 128):  # every code, in every byte position, both delta signs
            for pos in range(4):
                for inc in (0, 1):
                    others = rng.integers(0, 256, size=4)
                    others[pos] = code & 0xFF
                    incs = rng.integers(0, 2, size=4)
                    incs[pos] = inc
                    cases.append((others, incs, f, b))
        for _ in range(2000):
            cases.append((rng.integers(0, 256, size=4), rng.integers(0, 2, size=4), f, b))
    lines = []
    for codes, incs, f, b in cases:
        w = sum(int(c) << (8 * j) for j, c in enumerate(codes))
        ib = sum(int(i) << (8 * j) for j, i in enumerate(incs))
        lines.append(f"{w:x} {ib:x} {f} {b}\n")
    r = subprocess.run([swar_driver], input="".join(lines), capture_output=True, text=True)
    assert r.returncode == 0
    out = [tuple(int(t, 16) for t in line.split()) for line in r.stdout.splitlines()]
    assert len(out) == len(cases)
    bad = []
    for (codes, incs, f, b), (q, clip) in zip(cases, out):
        lo, hi = -(1 << (b - 1)), (1 << (b - 1)) - 1
        eps = Fraction(1, 2 ** (f + 3))  # |delta| below 2^-f: only ties depend on its sign
        for j in range(4):
            code = int(codes[j]) - 256 if codes[j] >= 128 else int(codes[j])
            u = Fraction(code, 2 ** f) + (eps if incs[j] else -eps)
            want = _rne(u)
            clipped = want > hi or want < lo
            got_clip = (clip >> (8 * j + 7)) & 1
            if got_clip != int(clipped):
                bad.append(("clip", code, f, int(incs[j]), want, got_clip))
            elif not clipped and ((q >> (8 * j)) & 0xFF) != (want & (0xFF if b > 4 else 15)):
                bad.append(("q", code, f, int(incs[j]), want, (q >> (8 * j)) & 0xFF))
    assert not bad, bad[:10]
