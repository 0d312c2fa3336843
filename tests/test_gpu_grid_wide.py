"""GPU parity of the wide-strip grid pass (marked gpu).

The grid pass takes its wide-strip kernel (256-column strips, four 16 x 64
sub-tiles per wave; rank chunks of 32 accumulated for r = 64, 96, ...) when
r is a multiple of 32, the rows are 16-byte aligned and the layer yields
enough strips x 64-row blocks; smaller layers take the per-wave kernel that
test_gpu_parity's small shapes exercise.  These cases are sized to take the
wide kernel (m = 2050 and k = 4224: ragged in the last 64-row block and in the
last strip) and drive each of its decision paths: rounding flips and clipping
(B std 0.3, large A), exact ties (B = 0 and B of order 1e-20), codes over the
whole int8 range that round off the grid inside the byte-parallel regime, the
rank-chunk accumulation (r = 64, 96), group-wise scales, and int8 q for a
6-bit grid.  Criteria as in test_gpu_parity: the grid (merge bytes) equals the
oracle's outside its .5 window, elements inside it equal the exact rational
round-half-to-even (checked on a sample), and the forward and backward outputs
match the oracle to the float tolerance."""
import math
import sys
from fractions import Fraction

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import lrqat_oracle as O
from test_gpu_parity import Case, check_full, check_merge, check_setup

pytestmark = pytest.mark.gpu

M, K, T = 2050, 4224, 64


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def lr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2406_06385_amd import lrqat
    lrqat.load_library()
    return lrqat


def _rne_exact(x):
    fl = math.floor(x)
    d = x - fl
    if d != Fraction(1, 2):
        return fl + (1 if d > Fraction(1, 2) else 0)
    return fl + (fl & 1)


STRESS = [
    # fmt, bits, r, g
    ("q8", 4, 32, 0),
    ("int_packed2", 4, 32, 0),
    ("q8", 3, 64, 128),
    ("int_packed2", 4, 96, 0),
]


@pytest.mark.parametrize("case", STRESS, ids=[f"{s[0]}b{s[1]}r{s[2]}g{s[3]}" for s in STRESS])
def test_wide_rounding_flips_and_clipping(lr, case):
    fmt, bits, r, g = case
    _log(f"[wide stress {case}]")
    c = Case(lr, M, K, T, r, float(r), bits, fmt, g, 0, "bf16", seed=41 + r, b_std=0.3, a_scale=100.0)
    check_setup(c)
    q_ref, near = check_merge(lr, c, allow_near=True)
    _, Mk, _, _ = O.grid_from_inputs(c.phi0_ref, c.A, c.B, c.L.alpha, c.L.rank, bits, fmt)
    assert (~Mk).sum() > 1000, "the stress case should clip"
    check_full(lr, c)


@pytest.mark.parametrize("fmt,r,b_std", [("q8", 64, 0.0), ("q8", 32, 1e-20), ("int_packed2", 32, 1e-20)])
def test_wide_exact_ties(lr, fmt, r, b_std):
    """B = 0 puts every half-fraction Q-format code on an exact tie (to even); B of order
    1e-20 decides them by the sign of a delta far below float64 resolution at 1/2."""
    _log(f"[wide ties {fmt} r{r} B std {b_std}]")
    c = Case(lr, M, K, T, r, float(r), 4, fmt, 0, 0, "bf16", seed=57, b_std=b_std)
    check_setup(c)
    L = c.L
    q_dev = O.unpack_int4(lr.lrqat_merge_to_int4(c.spec, c.d_phi0, c.d_A, c.d_B).cpu().numpy())
    q_ref, _, near, _ = O.grid_from_inputs(c.phi0_ref, c.A, c.B, L.alpha, L.rank, 4, fmt)
    assert np.array_equal(q_dev[~near], q_ref[~near])
    phi = O.decode_phi0(c.phi0_ref, 4, fmt)
    lo, hi = O.grid_limits(4)
    cc = Fraction(L.alpha) / L.rank
    idx = np.argwhere(near)
    rng = np.random.default_rng(5)
    pick = idx[rng.choice(len(idx), size=min(300, len(idx)), replace=False)] if len(idx) else idx
    for i, j in pick:
        d = sum(Fraction(float(c.A[i, t])) * Fraction(float(c.B[t, j])) for t in range(L.rank))
        want = min(max(_rne_exact(Fraction(float(phi[i, j])) + cc * d), lo), hi)
        assert q_dev[i, j] == want, (i, j, q_dev[i, j], want)
    _log(f"  {len(pick)} of {len(idx)} elements on .5 points checked exactly")
    if b_std == 0.0:
        check_full(lr, c)


@pytest.mark.parametrize("r", [32, 64])
def test_wide_full_code_range(lr, r):
    """Phi0 codes over the whole int8 range: codes n = hi with a fraction above one half
    round up off the grid inside the byte-parallel regime and must be clipped."""
    _log(f"[wide full code range r{r}]")
    rng = np.random.default_rng(61 + r)
    c = Case(lr, M, K, T, r, float(r), 4, "q8", 0, 0, "bf16", seed=63)
    c.phi0_ref = rng.integers(-128, 128, size=c.phi0_ref.shape).astype(np.int8)
    c.d_phi0 = torch.from_numpy(c.phi0_ref).cuda()
    _, Mk, _, _ = O.grid_from_inputs(c.phi0_ref, c.A, c.B, c.L.alpha, c.L.rank, 4, "q8")
    assert (~Mk).sum() > 1000
    check_merge(lr, c)
    check_full(lr, c)


@pytest.mark.parametrize("r", [32, 64])
def test_wide_six_bit_grid_int8_q(lr, r):
    """A 6-bit fixed-point grid writes q as int8 (no merge); checked through the outputs."""
    _log(f"[wide b6 r{r}]")
    c = Case(lr, M, K, T, r, float(r), 6, "q8", 0, 0, "bf16", seed=71, b_std=0.05, a_scale=8.0)
    check_setup(c)
    check_full(lr, c)


@pytest.mark.parametrize("variant", ["copy", "late_rows"])
def test_wide_packed_copy_regime_rounds(lr, variant):
    """Packed INT4 Phi0 with r = 32 at m = 7750, k = 4224: four 16-row rounds per wave, rows past
    m in the last blocks' later rounds, a ragged last strip.  'copy': the adapters' product is
    far below 1/2 everywhere, so every block copies Phi0 (the block-wide Cauchy-Schwarz test);
    'late_rows': rows 64..255 of every 256 (the second to fourth rounds of each block) are
    scaled up, so a block passes the test on its first round's rows and fails it on the
    others, and goes on to the per-sub-tile decisions."""
    m, k = 7750, 4224
    _log(f"[wide packed copy regime {variant}]")
    c = Case(lr, m, k, 64, 32, 32.0, 4, "int_packed2", 0, 0, "bf16", seed=83)
    if variant == "late_rows":
        rows = (np.arange(m) % 256) >= 64
        c.A[rows] *= np.float32(3000.0)
        c.d_A = torch.from_numpy(c.A).cuda()
    check_setup(c)
    q_ref, near = check_merge(lr, c, allow_near=variant == "late_rows")
    phi = O.decode_phi0(c.phi0_ref, 4, "int_packed2")
    moved = int((q_ref != phi).sum())
    if variant == "copy":
        assert moved == 0
    else:
        assert moved > 1000, "the scaled rows should move codes"
    check_full(lr, c)
