"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test ties the oracle to something other than itself: hand-computed values
(tests/golden/), a special case that reduces to a textbook routine, an
invariant, exact-rational brute force on tiny inputs, or finite differences.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import lrqat_oracle as O
from paper_2406_06385_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("|")[0].strip()
            if line and not line.startswith("#"):
                yield line


# ----------------------------------------------------------------------------- generator

def test_splitmix64_published_vectors():
    # splitmix64 seeded with 0: the reference outputs of Steele, Lea & Flood's generator.
    got = [int(v) for v in I.splitmix64(0, 3)]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_normals_moments_and_prefix_stability():
    z = I.normal(123, 200001)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01
    assert np.array_equal(I.normal(123, 1001), z[:1001])
    # chunked generation gives the same stream
    assert np.array_equal(I.normal(123, 5001, chunk=7), z[:5001])


def test_bf16_cast_is_rne():
    x = np.array([1.0, 1.00390625, 1.01171875, 1.0 + 2 ** -8 + 2 ** -20, -3.0, 0.0], np.float32)
    b = I.fp32_to_bf16_bits(x)
    back = I.bf16_bits_to_fp32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> 1 + 2^-6 (even)
    assert back.tolist() == [1.0, 1.0, 1.015625, 1.0078125, -3.0, 0.0]


# ----------------------------------------------------------------------------- formats

@pytest.mark.parametrize("line", list(_rows("phi_encode.txt")))
def test_phi_encode_golden(line):
    fmt, bits, x, want = line.split()
    bits, x, want = int(bits), float(x), int(want)
    W0 = np.array([[x, 0.0]], np.float32)
    s0 = np.array([1.0], np.float32)
    phi = O.encode_phi0(W0, s0, bits, fmt, 0)
    got = int(phi[0, 0]) if fmt == O.FMT_Q8 else int(O.unpack_int4(phi)[0, 0])
    assert got == want


@pytest.mark.parametrize("line", list(_rows("phi_decode.txt")))
def test_phi_decode_golden(line):
    bits, code, val = line.split()
    got = O.decode_phi0(np.array([[int(code)]], np.int8), int(bits), O.FMT_Q8)
    assert got[0, 0] == float(val)


@pytest.mark.parametrize("line", list(_rows("grid.txt")))
def test_grid_golden(line):
    fmt, bits, stored, delta, q_want, m_want = line.split()
    bits, stored, delta = int(bits), int(stored), float(delta)
    if fmt == O.FMT_Q8:
        phi0 = np.array([[stored]], np.int8)
        A = np.array([[delta]], np.float32)
        B = np.array([[1.0]], np.float32)
    else:
        phi0 = O.pack_int4(np.array([[stored, 0]]))
        A = np.array([[delta]], np.float32)
        B = np.array([[1.0, 0.0]], np.float32)
    q, M, near, u = O.grid_from_inputs(phi0, A, B, 1.0, 1, bits, fmt)
    assert int(q[0, 0]) == int(q_want)
    assert bool(M[0, 0]) == bool(int(m_want))


@pytest.mark.parametrize("line", list(_rows("near.txt")))
def test_near_window_golden(line):
    fmt, bits, stored, delta, near_want = line.split()
    bits, stored, delta = int(bits), int(stored), float(delta)
    if fmt == O.FMT_Q8:
        phi0 = np.array([[stored]], np.int8)
        B = np.array([[1.0]], np.float32)
    else:
        phi0 = O.pack_int4(np.array([[stored, 0]]))
        B = np.array([[1.0, 0.0]], np.float32)
    A = np.array([[delta]], np.float32)
    _, _, near, _ = O.grid_from_inputs(phi0, A, B, 1.0, 1, bits, fmt)
    assert bool(near[0, 0]) == bool(int(near_want))


@pytest.mark.parametrize("line", list(_rows("pack_int4.txt")))
def test_pack_golden(line):
    vals, byts = [p.strip() for p in line.split(";")]
    v = np.array([[int(t) for t in vals.split(",")]])
    want = np.array([[int(t, 16) for t in byts.split(",")]], np.uint8)
    assert np.array_equal(O.pack_int4(v), want)
    assert np.array_equal(O.unpack_int4(want), v)


def test_pack_roundtrip_all_nibbles_and_parities():
    v = np.array([[a, b] for a in range(-8, 8) for b in range(-8, 8)]).reshape(1, -1)
    assert np.array_equal(O.unpack_int4(O.pack_int4(v)), v)
    assert np.array_equal(O.unpack_int4(O.pack_int4(v[:, ::-1])), v[:, ::-1])


@pytest.mark.parametrize("line", list(_rows("minmax.txt")))
def test_minmax_encode_golden(line):
    head, row, s_want, phi_want = [p.strip() for p in line.split(";")]
    bits, g, fmt = head.split()
    bits, g = int(bits), int(g)
    W0 = np.array([[float(t) for t in row.split(",")]], np.float32)
    s0 = O.minmax_scale(W0, bits, g)
    assert s0.reshape(-1).tolist() == [float(t) for t in s_want.split(",")]
    phi = O.encode_phi0(W0, s0, bits, fmt, g)
    got = phi.reshape(-1) if fmt == O.FMT_Q8 else O.unpack_int4(phi).reshape(-1)
    assert got.tolist() == [int(t) for t in phi_want.split(",")]


@pytest.mark.parametrize("line", list(_rows("act_quant.txt")))
def test_act_quant_golden(line):
    row, sx_want, n_want = [p.strip() for p in line.split(";")]
    X = np.array([[float(t) for t in row.split(",")]], np.float32)
    xhat, n, sx = O.act_quant(X)
    assert float(sx[0]) == float(sx_want)
    assert n.reshape(-1).tolist() == [int(t) for t in n_want.split(",")]
    assert np.array_equal(xhat, float(sx_want) * n)


def test_act_quant_properties():
    X = I.normal(7, 64 * 300).reshape(64, 300).astype(np.float32) * np.linspace(0.01, 30, 64, dtype=np.float32)[:, None]
    xhat, n, sx = O.act_quant(X)
    assert np.abs(n).max() <= 127
    # the largest-magnitude entry of every row lands on +-127
    assert np.all(np.abs(n[np.arange(64), np.abs(X).argmax(axis=1)]) == 127)
    # round-to-nearest error bound |X - X_hat| <= s_x / 2 (plus float32 slack)
    err = np.abs(X.astype(np.float64) - xhat)
    assert np.all(err <= sx[:, None].astype(np.float64) * (0.5 + 1e-5))


def test_minmax_maps_row_absmax_to_grid_edge():
    W0 = I.gen_w0(37, 256, 11, 12, 0.02, 0.05)
    for fmt in (O.FMT_Q8, O.FMT_PACKED):
        for bits, g in ((4, 0), (3, 0), (4, 128), (2, 64)):
            if fmt == O.FMT_PACKED and bits > 4:
                continue
            s0 = O.minmax_scale(W0, bits, g)
            phi = O.encode_phi0(W0, s0, bits, fmt, g)
            val = O.decode_phi0(phi, bits, fmt)
            lo, hi = O.grid_limits(bits)
            assert val.min() >= lo and val.max() <= hi
            blocks = W0.reshape(37, -1, g) if g else W0.reshape(37, 1, -1)
            vb = val.reshape(37, -1, g) if g else val.reshape(37, 1, -1)
            idx = np.abs(blocks).argmax(axis=2)
            top = np.take_along_axis(vb, idx[..., None], axis=2)[..., 0]
            assert np.all(np.abs(top) == hi)


# ----------------------------------------------------------------------------- special cases

def _rand_layer(seed, m, k, r, bits, fmt, g=0, b_std=1e-3, clip_active=False, a_scale=1.0):
    W0 = I.gen_w0(m, k, seed, seed + 1, 0.02, 0.0)
    s0 = O.minmax_scale(W0, bits, g)
    if clip_active:
        s0 = (s0 * np.float32(0.6)).astype(np.float32)  # some |W0/s0| exceed the grid
    phi0 = O.encode_phi0(W0, s0, bits, fmt, g)
    A = (I.gen_a(m, r, k, seed + 2) * np.float32(a_scale)).astype(np.float32)
    B = I.gen_b(r, k, seed + 3, b_std)
    return W0, s0, phi0, A, B


@pytest.mark.parametrize("bits,g", [(4, 0), (3, 0), (2, 0), (4, 64)])
def test_b_zero_integer_phi_is_rtn_ptq(bits, g):
    """B = 0 with integer Phi0 and s = s0: W_hat = s clip(round(W0/s), lo, hi), the
    round-to-nearest PTQ of Eq. vanilla_qat evaluated on W0 directly."""
    m, k, r = 48, 256, 8
    W0, s0, phi0, A, _ = _rand_layer(5, m, k, r, bits, O.FMT_PACKED, g)
    B = np.zeros((r, k), np.float32)
    q, M, _, _ = O.grid_from_inputs(phi0, A, B, 8.0, r, bits, O.FMT_PACKED)
    W_hat = O.weight_hat(q, s0, g)
    lo, hi = O.grid_limits(bits)
    s_el = np.repeat(s0.reshape(m, -1), k // s0.reshape(m, -1).shape[1], axis=1)
    rtn = s_el.astype(np.float64) * np.clip(np.rint(W0 / s_el), lo, hi)
    assert np.array_equal(W_hat, rtn)
    assert M.all()


def test_grid_bounds_under_clipping_and_large_delta():
    for fmt, bits in ((O.FMT_Q8, 4), (O.FMT_Q8, 3), (O.FMT_Q8, 6), (O.FMT_PACKED, 4), (O.FMT_PACKED, 2)):
        _, _, phi0, A, B = _rand_layer(21, 64, 128, 16, bits, fmt, b_std=0.5, clip_active=True, a_scale=20.0)
        q, M, _, u = O.grid_from_inputs(phi0, A, B, 16.0, 16, bits, fmt)
        lo, hi = O.grid_limits(bits)
        assert q.min() >= lo and q.max() <= hi
        assert (~M).any() and M.any()  # the stress case really clips
        assert np.array_equal(q[M], np.rint(u[M]).astype(np.int64))


# ----------------------------------------------------------------------------- exact brute force

def _rne(x: Fraction) -> int:
    f = math.floor(x)
    d = x - f
    if d > Fraction(1, 2):
        return f + 1
    if d < Fraction(1, 2):
        return f
    return f if f % 2 == 0 else f + 1


def _brute(L, X, phi0_vals, s, A, B, dY):
    """Exact-rational evaluation with explicit loops (decoded Phi0 given as Fractions)."""
    m, k, r = L.m, L.k, L.rank
    T = len(X)
    c = Fraction(L.alpha) / r
    lo, hi = O.grid_limits(L.bits)
    q = [[0] * k for _ in range(m)]
    M = [[0] * k for _ in range(m)]
    for i in range(m):
        for j in range(k):
            u = phi0_vals[i][j] + c * sum(Fraction(float(A[i][p])) * Fraction(float(B[p][j])) for p in range(r))
            t = _rne(u)
            q[i][j] = min(max(t, lo), hi)
            M[i][j] = 1 if lo <= t <= hi else 0
    sc = lambda i, j: Fraction(float(s[i])) if L.group_size == 0 else Fraction(float(s[i][j // L.group_size]))
    W = [[sc(i, j) * q[i][j] for j in range(k)] for i in range(m)]
    Xf = [[Fraction(float(v)) for v in row] for row in X]
    dYf = [[Fraction(float(v)) for v in row] for row in dY]
    Y = [[sum(Xf[t][j] * W[i][j] for j in range(k)) for i in range(m)] for t in range(T)]
    dX = [[sum(dYf[t][i] * W[i][j] for i in range(m)) for j in range(k)] for t in range(T)]
    dW = [[sum(dYf[t][i] * Xf[t][j] for t in range(T)) for j in range(k)] for i in range(m)]
    G = [[sc(i, j) * M[i][j] * dW[i][j] for j in range(k)] for i in range(m)]
    dA = [[c * sum(G[i][j] * Fraction(float(B[p][j])) for j in range(k)) for p in range(r)] for i in range(m)]
    dB = [[c * sum(Fraction(float(A[i][p])) * G[i][j] for i in range(m)) for j in range(k)] for p in range(r)]
    return q, M, Y, dX, dA, dB


def _close(a, b, rtol=1e-12):
    a = np.asarray([[float(v) for v in row] for row in a])
    b = np.asarray(b, dtype=np.float64)
    scale = max(np.abs(a).max(), 1e-300)
    return np.abs(a - b).max() <= rtol * scale


@pytest.mark.parametrize("fmt,bits,g", [(O.FMT_Q8, 4, 0), (O.FMT_Q8, 3, 2), (O.FMT_PACKED, 4, 0), (O.FMT_PACKED, 2, 0)])
def test_exact_rational_brute_force(fmt, bits, g):
    rng = np.random.default_rng(3)
    m, k, r, T = 5, 6, 2, 3
    lo, hi = O.grid_limits(bits)
    f = 8 - bits
    if fmt == O.FMT_Q8:
        codes = rng.integers(-128, 128, size=(m, k))
        codes[0, :] = [(2 * j + 1) << (f - 1) for j in range(-3, 3)]   # exact .5 ties
        phi0 = codes.astype(np.int8)
        vals = [[Fraction(int(codes[i, j]), 1 << f) for j in range(k)] for i in range(m)]
    else:
        ints = rng.integers(lo, hi + 1, size=(m, k))
        phi0 = O.pack_int4(ints)
        vals = [[Fraction(int(ints[i, j])) for j in range(k)] for i in range(m)]
    A = rng.normal(0, 0.4, size=(m, r)).astype(np.float32)
    B = rng.normal(0, 0.4, size=(r, k)).astype(np.float32)
    A[0, :] = 0.0                      # row 0: delta = 0 -> ties go to even
    A[1, :] = [2.0 ** -30, 0.0]        # row 1: tiny positive delta where B[0] > 0
    B[0, :] = np.abs(B[0, :]) + 0.25
    s = (rng.uniform(0.5, 2.0, size=(m,) if g == 0 else (m, k // g))).astype(np.float32)
    X = rng.normal(size=(T, k)).astype(np.float32)
    dY = rng.normal(size=(T, m)).astype(np.float32)
    L = O.Layer(m, k, r, 1.5, bits, fmt, g, 0)
    q_b, M_b, Y_b, dX_b, dA_b, dB_b = _brute(L, X, vals, s, A, B, dY)
    Y, q, M, _ = O.forward(L, X, phi0, s, A, B)
    gr = O.backward(L, X, phi0, s, A, B, dY)
    assert q.tolist() == q_b and M.astype(int).tolist() == M_b
    assert _close(Y_b, Y) and _close(dX_b, gr["dX"]) and _close(dA_b, gr["dA"]) and _close(dB_b, gr["dB"])


def _f32_round(x: Fraction) -> Fraction:
    """Nearest IEEE binary32 value of an exact rational (round half to even),
    for normal magnitudes: 24 significant bits."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp = Fraction(2) ** (e - 23)
    return sign * _rne(a / ulp) * ulp


def _act_quant_exact(X):
    """Per-token symmetric int8 fake quantisation (Section 4 'Quantization',
    Eq. dequant with z = 0 and b = 8) in exact rationals: s_x = fl32(max|X_t| / 127),
    n = clip(round(fl32(X / s_x)), -128, 127), X_hat = s_x n; a zero row gives
    X_hat = 0.  fl32 is the correctly rounded float32 value (the float32 scale and
    quotient of the reading both sides take)."""
    out = []
    for row in X:
        xs = [Fraction(float(v)) for v in row]
        amax = max(abs(v) for v in xs)
        sx = _f32_round(amax / 127)
        if sx == 0:
            out.append([Fraction(0)] * len(xs))
            continue
        out.append([sx * min(max(_rne(_f32_round(v / sx)), -128), 127) for v in xs])
    return out


@pytest.mark.parametrize("fmt,bits,g", [(O.FMT_PACKED, 4, 0), (O.FMT_Q8, 4, 3)])
def test_exact_rational_brute_force_w4a8(fmt, bits, g):
    """The W4A8 composition: the GEMMs see X_hat (not X, not the codes), dX passes
    straight through the activation quantiser, dW = dY^T X_hat.  Token 1 is all
    zeros; token 2 has s_x = 1/8 exactly and entries at exact ties X/s_x = n + 1/2."""
    rng = np.random.default_rng(17)
    m, k, r, T = 4, 6, 2, 4
    lo, hi = O.grid_limits(bits)
    f = 8 - bits
    if fmt == O.FMT_Q8:
        codes = rng.integers(-128, 128, size=(m, k))
        phi0 = codes.astype(np.int8)
        vals = [[Fraction(int(codes[i, j]), 1 << f) for j in range(k)] for i in range(m)]
    else:
        ints = rng.integers(lo, hi + 1, size=(m, k))
        phi0 = O.pack_int4(ints)
        vals = [[Fraction(int(ints[i, j])) for j in range(k)] for i in range(m)]
    A = rng.normal(0, 0.4, size=(m, r)).astype(np.float32)
    B = rng.normal(0, 0.4, size=(r, k)).astype(np.float32)
    s = rng.uniform(0.5, 2.0, size=(m,) if g == 0 else (m, k // g)).astype(np.float32)
    X = rng.normal(0, 3.0, size=(T, k)).astype(np.float32)
    X[1, :] = 0.0
    # 127/8 = 15.875 -> s_x = 0.125; 0.3125 / 0.125 = 2.5 and -0.6875 / 0.125 = -5.5 are ties
    X[2, :] = [15.875, 0.3125, -0.6875, 1.0, -0.1875, 0.0625]
    dY = rng.normal(size=(T, m)).astype(np.float32)
    L = O.Layer(m, k, r, 1.5, bits, fmt, g, 8)
    Xh = _act_quant_exact(X)
    assert Xh[2][1] == Fraction(2, 8) and Xh[2][2] == Fraction(-6, 8) and Xh[2][4] == Fraction(-2, 8)
    assert all(v == 0 for v in Xh[1])
    Xh_f = np.array([[float(v) for v in row] for row in Xh])
    # the brute force of the unquantised layer, fed X_hat, is the W4A8 layer
    q_b, M_b, Y_b, dX_b, dA_b, dB_b = _brute(O.Layer(m, k, r, 1.5, bits, fmt, g, 0), Xh_f, vals, s, A, B, dY)
    assert all(Fraction(float(v)) == w for rowv, roww in zip(Xh_f, Xh) for v, w in zip(rowv, roww))
    Y, q, M, _ = O.forward(L, X, phi0, s, A, B)
    gr = O.backward(L, X, phi0, s, A, B, dY)
    assert q.tolist() == q_b and M.astype(int).tolist() == M_b
    assert _close(Y_b, Y) and _close(dX_b, gr["dX"]) and _close(dA_b, gr["dA"]) and _close(dB_b, gr["dB"])
    # the same layer without activation quantisation differs (the pin can see the quantiser)
    Y0 = O.forward(O.Layer(m, k, r, 1.5, bits, fmt, g, 0), X, phi0, s, A, B)[0]
    assert not np.allclose(Y0, Y, rtol=1e-6, atol=0)


# ----------------------------------------------------------------------------- gradients

def _surrogate_loss(L, X, phi0, s, A, B, dY, q0, M0, u0):
    """<dY, Y> with W_hat replaced by its straight-through surrogate around a base
    point: rounding acts as the identity, clipped elements stay frozen."""
    u = O.decode_phi0(phi0, L.bits, L.fmt) + O.rank_delta(A, B, L.alpha, L.rank)
    W = O.expand_scale(s, L.m, L.k, L.group_size) * (q0 + M0 * (u - u0))
    Y = O.layer_input(X, L.act_bits) @ W.T
    return float(np.sum(np.asarray(dY, np.float64) * Y))


@pytest.mark.parametrize("fmt,bits,g,act", [(O.FMT_Q8, 4, 0, 0), (O.FMT_Q8, 3, 32, 0), (O.FMT_PACKED, 4, 0, 8)])
def test_finite_differences_of_ste_surrogate(fmt, bits, g, act):
    m, k, r, T = 24, 64, 4, 16
    _, s0, phi0, A, B = _rand_layer(31, m, k, r, bits, fmt, g, b_std=0.3, clip_active=True)
    A = A.astype(np.float64) * 20
    B = B.astype(np.float64)
    X = I.normal(41, T * k).reshape(T, k).astype(np.float32)
    dY = I.normal(42, T * m).reshape(T, m)
    L = O.Layer(m, k, r, 2.0, bits, fmt, g, act)
    q0, M0, _, u0 = O.grid_from_inputs(phi0, A, B, L.alpha, r, bits, fmt)
    assert (~M0).any()
    gr = O.backward(L, X, phi0, s0, A, B, dY)
    h = 1e-4
    rng = np.random.default_rng(0)
    for (name, P, grad) in (("A", A, gr["dA"]), ("B", B, gr["dB"])):
        for _ in range(12):
            idx = tuple(rng.integers(0, n) for n in P.shape)
            Pp, Pm = P.copy(), P.copy()
            Pp[idx] += h
            Pm[idx] -= h
            args_p = (A if name == "B" else Pp, Pp if name == "B" else B)
            args_m = (A if name == "B" else Pm, Pm if name == "B" else B)
            fp = _surrogate_loss(L, X, phi0, s0, *args_p, dY, q0, M0, u0)
            fm = _surrogate_loss(L, X, phi0, s0, *args_m, dY, q0, M0, u0)
            fd = (fp - fm) / (2 * h)
            assert abs(fd - grad[idx]) <= 1e-7 * max(1.0, abs(grad[idx])), (name, idx, fd, grad[idx])


def test_finite_differences_of_scale_gradient():
    m, k, r, T = 16, 64, 4, 8
    for g in (0, 16):
        _, s0, phi0, A, B = _rand_layer(51, m, k, r, 4, O.FMT_Q8, g)
        X = I.normal(52, T * k).reshape(T, k).astype(np.float32)
        dY = I.normal(53, T * m).reshape(T, m)
        L = O.Layer(m, k, r, 4.0, 4, O.FMT_Q8, g, 0)
        ds = O.backward(L, X, phi0, s0, A, B, dY)["ds"]
        s = s0.astype(np.float64)
        for idx in [(0,) if g == 0 else (0, 0), (5,) if g == 0 else (3, 2)]:
            h = 1e-6
            sp, sm = s.copy(), s.copy()
            sp[idx] += h
            sm[idx] -= h
            fp = float(np.sum(dY * O.forward(L, X, phi0, sp, A, B)[0]))
            fm = float(np.sum(dY * O.forward(L, X, phi0, sm, A, B)[0]))
            assert abs((fp - fm) / (2 * h) - ds[idx]) < 1e-6 * max(1, abs(ds[idx]))


def test_adjoint_identities():
    """<X, dX> = <Y, dY> (dX is the adjoint of the forward map) and
    <A, dA> = <B, dB> (both equal c <G, A B>)."""
    m, k, r, T = 40, 96, 8, 12
    _, s0, phi0, A, B = _rand_layer(61, m, k, r, 4, O.FMT_Q8, 0, b_std=0.2, clip_active=True, a_scale=20.0)
    X = I.normal(62, T * k).reshape(T, k).astype(np.float32)
    dY = I.normal(63, T * m).reshape(T, m)
    L = O.Layer(m, k, r, 8.0, 4, O.FMT_Q8, 0, 0)
    Y = O.forward(L, X, phi0, s0, A, B)[0]
    gr = O.backward(L, X, phi0, s0, A, B, dY)
    lhs, rhs = np.sum(X * gr["dX"]), np.sum(Y * dY)
    assert abs(lhs - rhs) <= 1e-12 * np.sum(np.abs(X * gr["dX"]))
    a, b = np.sum(A * gr["dA"]), np.sum(B * gr["dB"])
    assert abs(a - b) <= 1e-12 * (np.sum(np.abs(A * gr["dA"])) + np.sum(np.abs(B * gr["dB"])))


def test_zero_adapters_give_zero_gradients():
    m, k, r, T = 16, 32, 4, 8
    _, s0, phi0, A, B = _rand_layer(71, m, k, r, 4, O.FMT_Q8, 0)
    X = I.normal(72, T * k).reshape(T, k).astype(np.float32)
    dY = I.normal(73, T * m).reshape(T, m)
    L = O.Layer(m, k, r, 4.0, 4, O.FMT_Q8, 0, 0)
    assert np.all(O.backward(L, X, phi0, s0, A, np.zeros_like(B), dY)["dA"] == 0)
    assert np.all(O.backward(L, X, phi0, s0, np.zeros_like(A), B, dY)["dB"] == 0)


def test_backward_is_linear_in_dy():
    m, k, r, T = 16, 32, 4, 8
    _, s0, phi0, A, B = _rand_layer(81, m, k, r, 3, O.FMT_Q8, 16, b_std=0.3, clip_active=True, a_scale=20.0)
    X = I.normal(82, T * k).reshape(T, k).astype(np.float32)
    d1 = I.normal(83, T * m).reshape(T, m)
    d2 = I.normal(84, T * m).reshape(T, m)
    L = O.Layer(m, k, r, 4.0, 3, O.FMT_Q8, 16, 0)
    g1 = O.backward(L, X, phi0, s0, A, B, d1)
    g2 = O.backward(L, X, phi0, s0, A, B, d2)
    g3 = O.backward(L, X, phi0, s0, A, B, 2.0 * d1 - 3.0 * d2)
    for key in ("dX", "dA", "dB", "ds"):
        ref = 2.0 * g1[key] - 3.0 * g2[key]
        assert np.allclose(g3[key], ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_group_size_k_equals_per_channel():
    m, k, r, T = 16, 64, 4, 8
    _, s0, phi0, A, B = _rand_layer(91, m, k, r, 4, O.FMT_Q8, 0)
    X = I.normal(92, T * k).reshape(T, k).astype(np.float32)
    dY = I.normal(93, T * m).reshape(T, m)
    Lc = O.Layer(m, k, r, 4.0, 4, O.FMT_Q8, 0, 0)
    Lg = O.Layer(m, k, r, 4.0, 4, O.FMT_Q8, k, 0)
    assert np.array_equal(O.forward(Lc, X, phi0, s0, A, B)[0], O.forward(Lg, X, phi0, s0.reshape(m, 1), A, B)[0])
    gc, gg = O.backward(Lc, X, phi0, s0, A, B, dY), O.backward(Lg, X, phi0, s0.reshape(m, 1), A, B, dY)
    for key in ("dX", "dA", "dB"):
        assert np.array_equal(gc[key], gg[key])
    assert np.array_equal(gc["ds"], gg["ds"].reshape(m))


def test_merge_is_lossless():
    """Section 3: after training W_hat = s * W_Z exactly, so the merged integer
    matrix reproduces the layer's output."""
    m, k, r, T = 32, 64, 8, 10
    for fmt, bits in ((O.FMT_Q8, 4), (O.FMT_Q8, 3), (O.FMT_PACKED, 4)):
        _, s0, phi0, A, B = _rand_layer(101, m, k, r, bits, fmt, b_std=0.3, clip_active=True, a_scale=20.0)
        X = I.normal(102, T * k).reshape(T, k).astype(np.float32)
        L = O.Layer(m, k, r, 8.0, bits, fmt, 0, 0)
        Y, q, _, _ = O.forward(L, X, phi0, s0, A, B)
        Wz = O.unpack_int4(O.merge_to_int4(L, phi0, A, B))
        assert np.array_equal(Wz, q)
        assert np.array_equal(X.astype(np.float64) @ (s0.astype(np.float64)[:, None] * Wz).T, Y)


def test_sampled_outputs_equal_full():
    m, k, r, T = 24, 48, 4, 20
    for act in (0, 8):
        _, s0, phi0, A, B = _rand_layer(111, m, k, r, 4, O.FMT_PACKED, 0, b_std=0.3)
        X = I.normal(112, T * k).reshape(T, k).astype(np.float32)
        dY = I.normal(113, T * m).reshape(T, m)
        L = O.Layer(m, k, r, 4.0, 4, O.FMT_PACKED, 0, act)
        Y = O.forward(L, X, phi0, s0, A, B)[0]
        gr = O.backward(L, X, phi0, s0, A, B, dY)
        tok, rows, cols = np.array([0, 7, 19]), np.array([1, 23]), np.array([0, 5, 47])
        assert np.allclose(O.forward_rows(L, X, phi0, s0, A, B, tok), Y[tok], rtol=1e-13, atol=0)
        assert np.allclose(O.dx_rows(L, phi0, s0, A, B, dY, tok), gr["dX"][tok], rtol=1e-13, atol=0)
        assert np.allclose(O.da_rows(L, X, phi0, s0, A, B, dY, rows), gr["dA"][rows], rtol=1e-12, atol=1e-15)
        assert np.allclose(O.db_cols(L, X, phi0, s0, A, B, dY, cols), gr["dB"][:, cols], rtol=1e-12, atol=1e-15)


def test_adapter_share_of_llama7b_parameters():
    """The paper's footnote on the rank ablation: r = 32 adapters are about 1.2%
    of LLaMA-7B's parameters.  With A [m x r] and B [r x k] on the 7 linears of
    each of the 32 blocks (shapes of the workloads' LLaMA-7B layers)."""
    q = I.WORKLOADS[2].layers[0]
    mlp = I.WORKLOADS[3].layers
    per_block = 4 * (q.m + q.k) * 32 + sum((L.m + L.k) * 32 for L in mlp)
    total_llama7b = 6_738_415_616
    assert round(100 * 32 * per_block / total_llama7b, 1) == 1.2
