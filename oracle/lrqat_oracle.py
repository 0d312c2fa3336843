"""CPU oracle for the LR-QAT linear layer.  TEST INFRASTRUCTURE ONLY.

Only the test-suite (`tests/`), the smoke check of `__graft_entry__` and the
CPU-baseline leg of `bench.py` may import this module.  The library
(`paper_2406_06385_amd`) never imports it and shares no code with it; the two
meet only in the seeded input generator `paper_2406_06385_amd.inputs`, which
holds none of the method's arithmetic.

Everything here is a direct, unblocked evaluation of the paper's definitions
in float64 with numpy; a numpy matmul is the only library primitive used, as
a plain matrix product.  Notation follows the paper (arXiv 2406.06385):

  W0 in R^{m x k}     frozen pretrained weight (nn.Linear: m = out, k = in)
  s0, s               initial (frozen) and trainable quantisation scale
  Phi0 = phi(W0/s0)   downcast frozen weight                (Section 3, Eq. phi)
  A in R^{m x r}, B in R^{r x k}, c = alpha / r             (Section 3, Eq. lr_qat)
  W_hat = s * clip(round(Phi0 + c A B), -2^(b-1), 2^(b-1)-1)  (Eq. lr_qat)
  Y = X W_hat^T with X in R^{T x k} (tokens as rows)

Readings of points the paper leaves open (each listed in the design doc):
  * round() is round-half-to-even (the paper says only "round to nearest").
  * The clip mask of the straight-through estimator is taken on the rounded
    value: M = [lo <= round(u) <= hi], inclusive.
  * Double-packed INT-b: element 2j of a row in the low nibble of byte j,
    element 2j+1 in the high nibble, 4-bit two's complement.
  * Per-token activation quantisation (W4A8): s_x[t] = max_j |X[t, j]| / 127 and
    n = clip(round(X / s_x), -128, 127), evaluated in float32 like the library;
    a zero row gives s_x = 0 and X_hat = 0.  s_x is a constant for the
    gradient and the STE passes dX_hat straight to dX.
  * Range estimation (setup) is min-max: s0 = max|W0 row or group| / (2^(b-1)-1),
    in float32; an all-zero row or group gets s0 = 1.
  * The downcast phi(W0/s0) takes its rounding decision in float32, like the
    library, on the correctly rounded float32 quotient W0/s0.
  * Asymmetric quantisation (Eq. dequant with an integer zero offset z, frozen
    at its range-estimation value z0): the stored Phi0 carries the offset,
    Phi0 = phi(W0/s0 + z0), with z added outside the rounding of the downcast
    (INT-b: clip(round(W0/s0) + z0); fixed point: clip(round(2^f W0/s0) + 2^f z0)),
    so that Phi0 lies on the b-bit grid like a symmetric one; the layer is
    W_hat = s * (clip(round(Phi0 + c A B), lo, hi) - z).  Range estimation for
    it is min-max over [min(W, 0), max(W, 0)]: s0 = (max - min) / (2^b - 1),
    z0 = clip(lo - round(min / s0), lo, hi), in float32.

Pinned by tests/test_oracle_pins.py and tests/test_oracle_pins_next.py
(-m "not gpu"): hand-computed values for the formats and the grid
(tests/golden/), round-to-nearest PTQ as the B = 0 special case (symmetric
and asymmetric), grid bounds, exact-rational brute force on tiny shapes,
finite differences of the straight-through surrogate for dA, dB and ds,
adjoint identities for dX and for dA/dB, the lossless merge, linearity in
dY, closed forms of the AdamW step and its schedule, exhaustive search for
the L^p range, and the Eckart-Young optimum for the LoftQ initialisation.
"""
from __future__ import annotations

import numpy as np

FMT_Q8 = "q8"                 # fixed point Qb.(8-b) stored in int8
FMT_PACKED = "int_packed2"    # two INT-b per byte
NEAR_WINDOW = 1e-5            # |u - (floor(u) + 1/2)| below this is "near a .5 boundary"


def grid_limits(bits: int) -> tuple[int, int]:
    """Signed b-bit integer grid [-2^(b-1), 2^(b-1)-1] (Section 2, Eq. dequant)."""
    return -(1 << (bits - 1)), (1 << (bits - 1)) - 1


def expand_scale(s: np.ndarray, m: int, k: int, group_size: int) -> np.ndarray:
    """Per-element scale [m][k] (float64) from per-channel s[m] or group-wise
    s[m][k/g] (one scale per row and group of g consecutive input columns,
    Section 4 'Quantization': the g128 setting)."""
    s = np.asarray(s, dtype=np.float64)
    if group_size == 0:
        return np.repeat(s.reshape(m, 1), k, axis=1)
    return np.repeat(s.reshape(m, k // group_size), group_size, axis=1)


# ----------------------------------------------------------------------------- setup

def minmax_scale(W0: np.ndarray, bits: int, group_size: int) -> np.ndarray:
    """Initial scale s0 by min-max range estimation (the RTN initialisation of
    Section 4 'Baselines', with the min-max range of Appendix Table A7):
    s0 = max |W0| over a row (or row-group) / (2^(b-1) - 1), in float32."""
    W = np.asarray(W0, dtype=np.float32)
    m, k = W.shape
    _, hi = grid_limits(bits)
    if group_size == 0:
        amax = np.abs(W).max(axis=1)
    else:
        amax = np.abs(W).reshape(m, k // group_size, group_size).max(axis=2)
    s0 = (amax / np.float32(hi)).astype(np.float32)
    s0[amax == 0] = np.float32(1.0)
    return s0


def minmax_scale_zero(W0: np.ndarray, bits: int, group_size: int):
    """Asymmetric min-max range estimation (Eq. dequant with a zero offset; the
    paper's W2 setting, Section 4 'Quantization'): over a row (or row-group),
    the range [min(W, 0), max(W, 0)] maps onto the grid [lo, hi]:
    s0 = (max - min) / (2^b - 1), z0 = clip(lo - round(min / s0), lo, hi),
    float32 arithmetic; a zero range gets s0 = 1, z0 = 0.  Returns
    (s0 float32, z0 int32), each [m] or [m][k/g]."""
    W = np.asarray(W0, dtype=np.float32)
    m, k = W.shape
    lo, hi = grid_limits(bits)
    Wg = W.reshape(m, 1, k) if group_size == 0 else W.reshape(m, k // group_size, group_size)
    wmin = np.minimum(Wg.min(axis=2), np.float32(0))
    wmax = np.maximum(Wg.max(axis=2), np.float32(0))
    rng = (wmax - wmin).astype(np.float32)
    s0 = (rng / np.float32((1 << bits) - 1)).astype(np.float32)
    zero = rng == 0
    s0[zero] = np.float32(1.0)
    z0 = np.clip(lo - np.rint((wmin / s0).astype(np.float32)), lo, hi).astype(np.int32)
    z0[zero] = 0
    if group_size == 0:
        return s0.reshape(m), z0.reshape(m)
    return s0, z0


def pack_int4(v: np.ndarray) -> np.ndarray:
    """Double-pack signed integers in [-8, 7] two per byte (Section 3,
    'Downcasting operator'): byte j of a row holds element 2j in its low
    nibble and element 2j+1 in its high nibble."""
    v = np.asarray(v, dtype=np.int64)
    assert v.shape[-1] % 2 == 0 and v.min(initial=0) >= -8 and v.max(initial=0) <= 7
    nib = (v & 0xF).astype(np.uint8)
    return (nib[..., 0::2] | (nib[..., 1::2] << 4)).astype(np.uint8)


def unpack_int4(p: np.ndarray) -> np.ndarray:
    """Inverse of pack_int4: [..][k/2] bytes -> [..][k] int64 in [-8, 7]."""
    p = np.asarray(p, dtype=np.uint8)
    lo = (p & 0xF).astype(np.int64)
    hi = (p >> 4).astype(np.int64)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int64)
    out[..., 0::2] = lo - 16 * (lo >= 8)
    out[..., 1::2] = hi - 16 * (hi >= 8)
    return out


def encode_phi0(W0: np.ndarray, s0: np.ndarray, bits: int, fmt: str, group_size: int, z0=None) -> np.ndarray:
    """Phi0 = phi(W0 / s0) (Section 3, Eq. phi), or phi(W0 / s0 + z0) with an
    asymmetric zero offset z0 (integer, added outside the rounding as in
    Eq. dequant).

    fmt "q8":  phi(x) = INT8(round(2^(8-b) * clip(x, -2^(b-1), 2^(b-1)-1)))
               (Eq. phi_fixed_point), returned as int8 [m][k].
    fmt "int_packed2": phi(x) = clip(round(x), -2^(b-1), 2^(b-1)-1) (INT-b),
               double-packed, returned as uint8 [m][k/2].
    The quotient and the rounding decision are float32 (see module header)."""
    W = np.asarray(W0, dtype=np.float32)
    m, k = W.shape
    lo, hi = grid_limits(bits)
    s = np.asarray(s0, dtype=np.float32)
    if group_size == 0:
        sx = np.repeat(s.reshape(m, 1), k, axis=1)
    else:
        sx = np.repeat(s.reshape(m, k // group_size), group_size, axis=1)
    x = (W / sx).astype(np.float32)
    if z0 is None:
        zx = np.zeros((m, k), np.int64)
    else:
        zx = np.repeat(np.asarray(z0, np.int64).reshape(m, -1), k // np.asarray(z0).reshape(m, -1).shape[1], axis=1)
    if fmt == FMT_Q8:
        f = 8 - bits
        if z0 is None:
            xc = np.clip(x, np.float32(lo), np.float32(hi))
            return np.rint(xc * np.float32(1 << f)).astype(np.int8)
        # clip(x + z) then scale and round equals clip(round(2^f x) + 2^f z) for integer z
        code = np.rint(x * np.float32(1 << f)).astype(np.int64) + (zx << f)
        return np.clip(code, lo << f, hi << f).astype(np.int8)
    if fmt == FMT_PACKED:
        v = np.clip(np.rint(x).astype(np.int64) + zx, lo, hi)
        return pack_int4(v)
    raise ValueError(fmt)


# ----------------------------------------------------------------------------- forward pieces

def decode_phi0(phi0: np.ndarray, bits: int, fmt: str) -> np.ndarray:
    """phi^-1: stored Phi0 -> its real value (float64, exact).
    q8: code / 2^(8-b) (Eq. phi_fixed_point, upcast); packed: the INT-b value."""
    if fmt == FMT_Q8:
        return np.asarray(phi0, dtype=np.int8).astype(np.float64) * 2.0 ** -(8 - bits)
    if fmt == FMT_PACKED:
        return unpack_int4(phi0).astype(np.float64)
    raise ValueError(fmt)


def rank_delta(A: np.ndarray, B: np.ndarray, alpha: float, rank: int) -> np.ndarray:
    """delta = (alpha / r) * A B, the low-rank term inside the rounding (Eq. lr_qat)."""
    return (float(alpha) / float(rank)) * (np.asarray(A, np.float64) @ np.asarray(B, np.float64))


def reconstruct(phi: np.ndarray, delta: np.ndarray, bits: int):
    """Integer grid of Eq. lr_qat.

    Returns (q, M, near, u): u = Phi0 + delta (the pre-round value),
    q = clip(round(u), lo, hi), the STE clip mask M = [lo <= round(u) <= hi],
    and near = |u - (floor(u) + 1/2)| < 1e-5 (elements whose rounding a
    different but accurate evaluation of u may legitimately decide the
    other way)."""
    lo, hi = grid_limits(bits)
    u = np.asarray(phi, np.float64) + np.asarray(delta, np.float64)
    ut = np.rint(u)
    q = np.clip(ut, lo, hi).astype(np.int64)
    M = (ut >= lo) & (ut <= hi)
    near = np.abs(u - (np.floor(u) + 0.5)) < NEAR_WINDOW
    return q, M, near, u


def grid_from_inputs(phi0, A, B, alpha, rank, bits, fmt):
    """(q, M, near, u) straight from the stored inputs."""
    return reconstruct(decode_phi0(phi0, bits, fmt), rank_delta(A, B, alpha, rank), bits)


def weight_hat(q: np.ndarray, s: np.ndarray, group_size: int, z=None) -> np.ndarray:
    """W_hat = s * q (Eq. lr_qat, the scale outside the clip), or s * (q - z)
    with an asymmetric zero offset (Eq. dequant)."""
    m, k = q.shape
    return expand_scale(s, m, k, group_size) * grid_minus_zero(q, z, group_size)


def grid_minus_zero(q: np.ndarray, z, group_size: int) -> np.ndarray:
    """q - z as float64 (z = None: symmetric, q itself)."""
    if z is None:
        return np.asarray(q, np.float64)
    m, k = q.shape
    return np.asarray(q, np.float64) - expand_scale(np.asarray(z, np.float64), m, k, group_size)


def act_quant(X: np.ndarray):
    """Per-token dynamic symmetric int8 fake quantisation of the layer input
    (Section 4 'Quantization', per-token activation quantisation; Eq. dequant
    with z = 0, b = 8 and s = s_x[t]).  X is float32 (a bfloat16 input widened
    exactly).  Returns (X_hat float64 [T][k], n int64 [T][k], s_x float32 [T])."""
    X = np.asarray(X, dtype=np.float32)
    amax = np.abs(X).max(axis=1)
    sx = (amax / np.float32(127.0)).astype(np.float32)
    safe = np.where(sx > 0, sx, np.float32(1.0)).astype(np.float32)
    n = np.clip(np.rint(X / safe[:, None]), -128, 127).astype(np.int64)
    n[sx == 0] = 0
    xhat = sx.astype(np.float64)[:, None] * n
    return xhat, n, sx


def layer_input(X: np.ndarray, act_bits: int) -> np.ndarray:
    """The matrix the GEMMs see: X itself, or X_hat under W4A8."""
    if act_bits == 0:
        return np.asarray(X, dtype=np.float64)
    if act_bits == 8:
        return act_quant(X)[0]
    raise ValueError(act_bits)


# ----------------------------------------------------------------------------- the layer

class Layer:
    """Hyper-parameters of one LR-QAT linear (Eq. lr_qat's alpha, r, b, the
    storage format of Phi0 and the scale granularity)."""

    def __init__(self, m, k, rank, alpha, bits, fmt, group_size=0, act_bits=0):
        self.m, self.k, self.rank, self.alpha = int(m), int(k), int(rank), float(alpha)
        self.bits, self.fmt, self.group_size, self.act_bits = int(bits), fmt, int(group_size), int(act_bits)

    @property
    def c(self) -> float:
        return self.alpha / self.rank


def forward(L: Layer, X, phi0, s, A, B, z=None):
    """Y = X_hat W_hat^T (Eq. lr_qat applied to a linear layer).  Returns
    (Y float64 [T][m], q, M, near)."""
    q, M, near, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    W = weight_hat(q, s, L.group_size, z)
    return layer_input(X, L.act_bits) @ W.T, q, M, near


def backward(L: Layer, X, phi0, s, A, B, dY, z=None):
    """Straight-through-estimator gradients of the layer (Section 3: STE for
    the rounding, d round(t)/dt = 1; the scale s sits outside the clip):

      dX  = dY W_hat                       (through X_hat unchanged under W4A8)
      dW  = dY^T X_hat                     gradient w.r.t. W_hat
      G   = s * M * dW                     gradient w.r.t. Phi0 + c A B
      dA  = c G B^T,   dB = c A^T G
      ds  = sum over a row (or row-group) of dW * (q - z)   (dW_hat/ds = q - z)

    W_hat is recomputed from (Phi0, A, B, s), never taken from the forward,
    as under the paper's checkpointing of W_hat.  Returns a dict of float64."""
    q, M, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    W = weight_hat(q, s, L.group_size, z)
    dY = np.asarray(dY, dtype=np.float64)
    Xh = layer_input(X, L.act_bits)
    dX = dY @ W
    dW = dY.T @ Xh
    G = expand_scale(s, L.m, L.k, L.group_size) * M * dW
    dA = L.c * (G @ np.asarray(B, np.float64).T)
    dB = L.c * (np.asarray(A, np.float64).T @ G)
    dWq = dW * grid_minus_zero(q, z, L.group_size)
    if L.group_size == 0:
        ds = dWq.sum(axis=1)
    else:
        ds = dWq.reshape(L.m, L.k // L.group_size, L.group_size).sum(axis=2)
    return {"dX": dX, "dA": dA, "dB": dB, "ds": ds}


def merge_to_int4(L: Layer, phi0, A, B) -> np.ndarray:
    """W_Z = clip(round(Phi0 + c A B)) as packed int4 (Section 3: after training
    the adapters merge into one b-bit integer matrix, W_hat = s * W_Z)."""
    assert L.bits <= 4
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    return pack_int4(q)


# ----------------------------------------------------------------------------- sampled outputs
# The same definitions restricted to a subset of output rows / columns, for
# parity checks at sizes where the full products would take too long.

def forward_rows(L: Layer, X, phi0, s, A, B, tok, z=None):
    """Rows `tok` of Y."""
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    W = weight_hat(q, s, L.group_size, z)
    return layer_input(np.asarray(X)[tok], L.act_bits) @ W.T


def dx_rows(L: Layer, phi0, s, A, B, dY, tok, z=None):
    """Rows `tok` of dX = dY W_hat."""
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    W = weight_hat(q, s, L.group_size, z)
    return np.asarray(dY, np.float64)[tok] @ W


def da_rows(L: Layer, X, phi0, s, A, B, dY, rows):
    """Rows `rows` of dA = c (s * M * dY^T X_hat) B^T."""
    q, M, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    Xh = layer_input(X, L.act_bits)
    dW = np.asarray(dY, np.float64)[:, rows].T @ Xh
    G = expand_scale(s, L.m, L.k, L.group_size)[rows] * M[rows] * dW
    return L.c * (G @ np.asarray(B, np.float64).T)


def db_cols(L: Layer, X, phi0, s, A, B, dY, cols):
    """Columns `cols` of dB = c A^T (s * M * dY^T X_hat)."""
    q, M, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    Xh = layer_input(X, L.act_bits)
    dW = np.asarray(dY, np.float64).T @ Xh[:, cols]
    G = expand_scale(s, L.m, L.k, L.group_size)[:, cols] * M[:, cols] * dW
    return L.c * (np.asarray(A, np.float64).T @ G)


def ds_rows(L: Layer, X, phi0, s, A, B, dY, rows, z=None):
    """Rows `rows` of ds = sum over a row (or row-group) of dW * (q - z)."""
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    Xh = layer_input(X, L.act_bits)
    dW = np.asarray(dY, np.float64)[:, rows].T @ Xh
    qz = grid_minus_zero(q, z, L.group_size)[rows]
    if L.group_size == 0:
        return (dW * qz).sum(axis=1)
    return (dW * qz).reshape(len(rows), L.k // L.group_size, L.group_size).sum(axis=2)


# ----------------------------------------------------------------------------- inference on merged weights

def infer_forward(L: Layer, X, W_Z, s, z=None):
    """Inference after the merge (Section 3: W_hat = s * W_Z without extra
    overhead; with a zero offset, s * (W_Z - z) as in Eq. dequant):
    Y = X_hat (s * (unpack(W_Z) - z))^T, X_hat the layer's (possibly int8
    fake-quantised) input."""
    q = unpack_int4(W_Z)
    return layer_input(X, L.act_bits) @ weight_hat(q, s, L.group_size, z).T


# ----------------------------------------------------------------------------- optimizer step

def clip_coefficient(grads, max_norm: float, eps: float = 1e-6) -> float:
    """Global L2-norm gradient clipping (Appendix B, Table B1: maximum norm 1.0):
    every gradient is multiplied by min(1, max_norm / (||g||_2 + eps)), with the
    norm over all trainable tensors together.  The eps keeps the division finite
    for a zero gradient (reading: the clip of the training library the paper
    names)."""
    total = float(np.sqrt(sum(float(np.sum(np.asarray(g, np.float64) ** 2)) for g in grads)))
    return min(1.0, max_norm / (total + eps)), total


def lr_at(step: int, lr_max: float, total_steps: int, warmup_steps: int) -> float:
    """Learning rate of optimizer step `step` (1-based) under the paper's
    schedule (Appendix B): linear warm-up over the first warm-up steps, then
    linear decay to zero at the end of training.  With t = step - 1 steps
    already taken: lr_max t / W while t < W, else lr_max (N - t) / (N - W),
    never below zero (reading: the linear schedule of the training library
    the paper names, whose first step runs at t = 0)."""
    t = step - 1
    if t < warmup_steps:
        return lr_max * t / max(1, warmup_steps)
    return lr_max * max(0.0, (total_steps - t) / max(1, total_steps - warmup_steps))


def adamw_step(p, g, m, v, step: int, lr: float, beta1: float, beta2: float, eps: float, weight_decay: float,
               clip: float = 1.0):
    """One AdamW update (Loshchilov & Hutter, decoupled weight decay; the
    optimizer of Appendix B with (beta1, beta2) = (0.9, 0.95)) of one tensor,
    on its gradient g times the global clip coefficient `clip`:
        p <- p (1 - lr wd)
        m <- beta1 m + (1 - beta1) g,   v <- beta2 v + (1 - beta2) g^2
        p <- p - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
    Returns (p, m, v) as new float64 arrays."""
    g = np.asarray(g, np.float64) * clip
    p = np.asarray(p, np.float64) * (1.0 - lr * weight_decay)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    return p - lr * mhat / (np.sqrt(vhat) + eps), m, v


# ----------------------------------------------------------------------------- setup-side initialisation

def lp_scale_search(W0: np.ndarray, bits: int, group_size: int, p: float, n_grid: int = 100):
    """L^p-norm range estimation (Section 4 'Baselines', Appendix B 'PTQ
    initialization': the range minimising the L^p norm between quantized and
    unquantized weights, p in {2, 2.4, 3, 3.5, 4, 5}).  Candidates are the
    clipping ratios j / n_grid, j = 1..n_grid, of the min-max range: for each
    row (or row-group) s_j = (j / n_grid) max|W| / (2^(b-1) - 1) and the error
    E_j = sum |W - s_j clip(round(W / s_j), lo, hi)|^p; the smallest j of the
    minimal E_j is taken (reading: the grid of candidates is not given).
    s_j and the quotient W / s_j are float32; E_j is float64.  Returns
    (s0 float32, j int32, E float64 [.., n_grid])."""
    W = np.asarray(W0, dtype=np.float32)
    m, k = W.shape
    lo, hi = grid_limits(bits)
    Wg = W.reshape(m, 1, k) if group_size == 0 else W.reshape(m, k // group_size, group_size)
    S = lp_candidate_scales(W0, bits, group_size, n_grid).reshape(Wg.shape[:2] + (n_grid,))
    E = np.empty(S.shape, np.float64)
    for j in range(1, n_grid + 1):
        sj = S[..., j - 1]
        qv = np.clip(np.rint((Wg / sj[..., None]).astype(np.float32)), lo, hi)
        err = np.abs(Wg.astype(np.float64) - sj[..., None].astype(np.float64) * qv)
        E[..., j - 1] = np.sum(err ** p, axis=2)
    jbest = np.argmin(E, axis=-1)
    s0 = np.take_along_axis(S, jbest[..., None], axis=-1)[..., 0]
    if group_size == 0:
        return s0.reshape(m), (jbest + 1).reshape(m).astype(np.int32), E.reshape(m, n_grid)
    return s0, (jbest + 1).astype(np.int32), E


def lp_candidate_scales(W0: np.ndarray, bits: int, group_size: int, n_grid: int = 100) -> np.ndarray:
    """The candidate scales s_j = fl32(fl32(j / n_grid) max|W| / (2^(b-1) - 1)),
    j = 1..n_grid, of every row (or row-group): float32 [m][n_grid] or
    [m][k/g][n_grid] (an all-zero row or group gets 1)."""
    W = np.asarray(W0, dtype=np.float32)
    m, k = W.shape
    _, hi = grid_limits(bits)
    Wg = W.reshape(m, 1, k) if group_size == 0 else W.reshape(m, k // group_size, group_size)
    amax = np.abs(Wg).max(axis=2)
    S = np.empty(amax.shape + (n_grid,), np.float32)
    for j in range(1, n_grid + 1):
        sj = ((np.float32(j) / np.float32(n_grid)) * amax / np.float32(hi)).astype(np.float32)
        S[..., j - 1] = np.where(amax > 0, sj, np.float32(1.0)).astype(np.float32)
    return S.reshape(m, n_grid) if group_size == 0 else S


def loftq_init(W0: np.ndarray, s0: np.ndarray, bits: int, group_size: int, rank: int, alpha: float):
    """LoftQ initialisation with T = 1 alternating step (Section 3 'Downcasting
    operator' and the ablation of Section 4.2), in the units of Eq. lr_qat:
    x = W0 / s0, Phi0 = INT-b(x) = clip(round(x)), the residual R = x - Phi0 (the
    fractional part the integer downcast loses), and the best rank-r
    approximation of R from its SVD, R_r = U_r Sigma_r V_r^T (Eckart-Young),
    split evenly so that (alpha / r) A B = R_r:
        A = U_r Sigma_r^(1/2) / sqrt(alpha / r),  B = Sigma_r^(1/2) V_r^T / sqrt(alpha / r).
    The quotient and the rounding are float32 like encode_phi0; the SVD is
    float64.  Returns (Phi0 packed uint8, A, B float64, R, singular values)."""
    W = np.asarray(W0, dtype=np.float32)
    m, k = W.shape
    lo, hi = grid_limits(bits)
    x = (W / expand_scale(s0, m, k, group_size).astype(np.float32)).astype(np.float32)
    n = np.clip(np.rint(x), lo, hi)
    R = x.astype(np.float64) - n
    U, S, Vt = np.linalg.svd(R, full_matrices=False)
    c = float(alpha) / float(rank)
    root = np.sqrt(S[:rank]) / np.sqrt(c)
    A = U[:, :rank] * root[None, :]
    B = root[:, None] * Vt[:rank]
    return pack_int4(n.astype(np.int64)), A, B, R, S


# ----------------------------------------------------------------------------- error scales
# Magnitudes of the terms of the layer's contractions: |X_hat| |W_hat|^T for Y,
# |dY| |W_hat| for dX, c |G| |B|^T for dA and c |A|^T |G| for dB (|.|
# elementwise).  A contraction whose operands carry a relative rounding error e
# is accurate to about e times these, whatever the cancellation inside the
# sums; the parity tests use them as the scale of the bound for output lines
# whose own norm is small against them.

def forward_rows_abs(L: Layer, X, phi0, s, A, B, tok, z=None):
    """Rows `tok` of |X_hat| |W_hat|^T."""
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    W = np.abs(weight_hat(q, s, L.group_size, z))
    return np.abs(layer_input(np.asarray(X)[tok], L.act_bits)) @ W.T


def dx_rows_abs(L: Layer, phi0, s, A, B, dY, tok, z=None):
    """Rows `tok` of |dY| |W_hat|."""
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    W = np.abs(weight_hat(q, s, L.group_size, z))
    return np.abs(np.asarray(dY, np.float64)[tok]) @ W


def _abs_g(L: Layer, X, phi0, s, A, B, dY, rows=None, cols=None):
    q, M, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    Xh = layer_input(X, L.act_bits)
    dY = np.asarray(dY, np.float64)
    S = expand_scale(s, L.m, L.k, L.group_size)
    if rows is not None:
        return np.abs(S[rows] * M[rows] * (dY[:, rows].T @ Xh))
    return np.abs(S[:, cols] * M[:, cols] * (dY.T @ Xh[:, cols]))


def da_rows_abs(L: Layer, X, phi0, s, A, B, dY, rows):
    """Rows `rows` of |c| |G| |B|^T."""
    return abs(L.c) * (_abs_g(L, X, phi0, s, A, B, dY, rows=rows) @ np.abs(np.asarray(B, np.float64)).T)


def db_cols_abs(L: Layer, X, phi0, s, A, B, dY, cols):
    """Columns `cols` of |c| |A|^T |G|."""
    return abs(L.c) * (np.abs(np.asarray(A, np.float64)).T @ _abs_g(L, X, phi0, s, A, B, dY, cols=cols))


def ds_rows_abs(L: Layer, X, phi0, s, A, B, dY, rows, z=None):
    """Rows `rows` of the magnitude of ds's terms: sum over a row (or row-group)
    of |dW| |q - z|."""
    q, _, _, _ = grid_from_inputs(phi0, A, B, L.alpha, L.rank, L.bits, L.fmt)
    Xh = layer_input(X, L.act_bits)
    dW = np.abs(np.asarray(dY, np.float64)[:, rows].T @ Xh)
    qz = np.abs(grid_minus_zero(q, z, L.group_size)[rows])
    if L.group_size == 0:
        return (dW * qz).sum(axis=1)
    return (dW * qz).reshape(len(rows), L.k // L.group_size, L.group_size).sum(axis=2)
