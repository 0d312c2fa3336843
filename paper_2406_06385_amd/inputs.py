"""Seeded synthetic inputs for the LR-QAT linear layer.

This module is shared by the HIP path's harness (tests, benchmark) and by the
CPU oracle's tests.  It holds no arithmetic of the method itself: it only draws
random numbers and casts them to the storage dtypes.  Range estimation, the
downcast of W0/s0 into Phi0, rounding and clipping all live on each side
separately (the library and the oracle each implement them).

Generator: splitmix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014) used as a counter-based stream: element i of
a stream with seed S is mix(S + (i + 1) * 0x9E3779B97F4A7C15).  Uniforms take
the top 53 bits; normals use the Box-Muller transform on consecutive pairs.

Workloads follow the layer shapes of LLaMA-1-7B, LLaMA-2-13B and LLaMA-3-8B
(the models of the paper's experiments section) with the value distributions
of a freshly initialised LR-QAT layer (LoRA-style init, the paper's ablation on
A, B initialisation): W0 ~ N(0, 0.02^2), A ~ U(+-1/sqrt(k)), B ~ N(0, 1e-3^2),
X ~ N(0, 1), dY ~ N(0, 1e-2^2).  The pretrained weights, SlimPajama token
activations and gradients the paper trains on are not available; these seeded
tensors stand in for them.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
SEED_BASE = 2406063850

# tensor ids inside one layer's seed block
T_W0, T_OUTLIER, T_A, T_B, T_X, T_DY = range(6)


def splitmix64(seed: int, n: int, offset: int = 0) -> np.ndarray:
    """n consecutive outputs (uint64) of the counter-based splitmix64 stream."""
    with np.errstate(over="ignore"):
        i = np.arange(offset + 1, offset + n + 1, dtype=np.uint64)
        z = np.uint64(seed % (1 << 64)) + i * _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return z


def uniform01(seed: int, n: int, offset: int = 0) -> np.ndarray:
    """n uniforms in [0, 1) with 53 random bits each (float64)."""
    return (splitmix64(seed, n, offset) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def normal(seed: int, n: int, std: float = 1.0, chunk: int = 1 << 24) -> np.ndarray:
    """n standard normals * std (float64), Box-Muller on consecutive uniform pairs."""
    out = np.empty(n, dtype=np.float64)
    npairs = (n + 1) // 2
    for p0 in range(0, npairs, chunk):
        p1 = min(npairs, p0 + chunk)
        u = uniform01(seed, 2 * (p1 - p0), offset=2 * p0)
        u1 = 1.0 - u[0::2]          # (0, 1]: log is finite
        u2 = u[1::2]
        rad = np.sqrt(-2.0 * np.log(u1))
        ang = 2.0 * math.pi * u2
        z = np.empty(2 * (p1 - p0), dtype=np.float64)
        z[0::2] = rad * np.cos(ang)
        z[1::2] = rad * np.sin(ang)
        lo, hi = 2 * p0, min(n, 2 * p1)
        out[lo:hi] = z[: hi - lo]
    if std != 1.0:
        out *= std
    return out


def fp32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even cast float32 -> bfloat16, returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    with np.errstate(over="ignore"):
        r = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = (r >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_fp32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------- workloads

@dataclasses.dataclass(frozen=True)
class LayerSpec:
    name: str
    m: int              # out features
    k: int              # in features


@dataclasses.dataclass(frozen=True)
class Workload:
    """One benchmark/parity workload: a list of LR-QAT linears sharing hyper-parameters."""
    cfg: int
    name: str
    layers: tuple
    tokens: int
    rank: int
    alpha: float
    bits: int
    phi_format: str          # "q8" (fixed point Qb.(8-b) in int8) or "int_packed2"
    group_size: int          # 0 = per output channel
    act_bits: int            # 0 or 8 (per-token dynamic symmetric)
    act_dtype: str           # "fp32" or "bf16"
    outlier_frac: float = 0.0   # fraction of input columns scaled x20 in W0
    w_std: float = 0.02
    b_std: float = 1e-3
    dy_std: float = 1e-2

    def flops_fwd_bwd(self, tokens: int | None = None) -> float:
        """Algorithmic flops of one forward+backward: 6*T*m*k GEMM terms plus
        8*m*k*r for the rank-r product (forward, backward recompute) and the
        two rank-r gradient contractions."""
        t = self.tokens if tokens is None else tokens
        return float(sum(6 * t * L.m * L.k + 8 * L.m * L.k * self.rank for L in self.layers))


WORKLOADS = {
    1: Workload(1, "single-linear-512x256-fp32", (LayerSpec("linear", 512, 256),),
                tokens=128, rank=8, alpha=8.0, bits=4, phi_format="q8", group_size=0,
                act_bits=0, act_dtype="fp32"),
    2: Workload(2, "llama7b-q_proj-4096x4096", (LayerSpec("q_proj", 4096, 4096),),
                tokens=8192, rank=32, alpha=32.0, bits=4, phi_format="q8", group_size=0,
                act_bits=0, act_dtype="bf16", outlier_frac=0.01),
    3: Workload(3, "llama7b-mlp", (LayerSpec("gate_proj", 11008, 4096),
                                   LayerSpec("up_proj", 11008, 4096),
                                   LayerSpec("down_proj", 4096, 11008)),
                tokens=8192, rank=32, alpha=32.0, bits=4, phi_format="int_packed2", group_size=0,
                act_bits=0, act_dtype="bf16"),
    4: Workload(4, "llama2-13b-mlp-w3g128", (LayerSpec("up_proj", 13824, 5120),
                                             LayerSpec("down_proj", 5120, 13824)),
                tokens=8192, rank=64, alpha=64.0, bits=3, phi_format="q8", group_size=128,
                act_bits=0, act_dtype="bf16"),
    5: Workload(5, "llama3-8b-block-w4a8", (LayerSpec("q_proj", 4096, 4096),
                                            LayerSpec("k_proj", 1024, 4096),
                                            LayerSpec("v_proj", 1024, 4096),
                                            LayerSpec("o_proj", 4096, 4096),
                                            LayerSpec("gate_proj", 14336, 4096),
                                            LayerSpec("up_proj", 14336, 4096),
                                            LayerSpec("down_proj", 4096, 14336)),
                tokens=8192, rank=32, alpha=32.0, bits=4, phi_format="int_packed2", group_size=0,
                act_bits=8, act_dtype="bf16"),
}


def layer_seed(cfg: int, layer: int, tensor: int) -> int:
    return SEED_BASE + 100 * cfg + 10 * layer + tensor


def gen_w0(m: int, k: int, seed_w: int, seed_perm: int, std: float = 0.02,
           outlier_frac: float = 0.0) -> np.ndarray:
    """W0 [m][k] float32 ~ N(0, std^2); round(outlier_frac*k) input columns,
    chosen by a seeded permutation, are multiplied by 20."""
    w = normal(seed_w, m * k, std).reshape(m, k)
    n_out = int(round(outlier_frac * k))
    if n_out:
        perm = np.argsort(splitmix64(seed_perm, k), kind="stable")
        w[:, perm[:n_out]] *= 20.0
    return w.astype(np.float32)


def gen_a(m: int, r: int, k: int, seed: int) -> np.ndarray:
    """A [m][r] float32 ~ U(-1/sqrt(k), 1/sqrt(k))."""
    bound = 1.0 / math.sqrt(k)
    return ((uniform01(seed, m * r) * 2.0 - 1.0) * bound).reshape(m, r).astype(np.float32)


def gen_b(r: int, k: int, seed: int, std: float = 1e-3) -> np.ndarray:
    """B [r][k] float32 ~ N(0, std^2)."""
    return normal(seed, r * k, std).reshape(r, k).astype(np.float32)


def gen_act(rows: int, cols: int, seed: int, std: float, dtype: str) -> np.ndarray:
    """Activation-like tensor [rows][cols] ~ N(0, std^2): float32 array for
    dtype "fp32", uint16 bfloat16 bit patterns (RNE cast) for "bf16"."""
    x = normal(seed, rows * cols, std).astype(np.float32).reshape(rows, cols)
    if dtype == "fp32":
        return x
    if dtype == "bf16":
        return fp32_to_bf16_bits(x)
    raise ValueError(dtype)


@dataclasses.dataclass
class LayerInputs:
    spec: LayerSpec
    W0: np.ndarray      # [m][k] float32
    A: np.ndarray       # [m][r] float32
    B: np.ndarray       # [r][k] float32
    X: np.ndarray       # [T][k] float32 or uint16 (bf16 bits)
    dY: np.ndarray      # [T][m] float32 or uint16 (bf16 bits)


def make_layer_inputs(wl: Workload, layer: int = 0, tokens: int | None = None,
                      with_acts: bool = True) -> LayerInputs:
    """Seeded inputs of one layer of a workload.  `tokens` overrides T (the
    first `tokens` rows of the full-size streams are the same numbers)."""
    spec = wl.layers[layer]
    t = wl.tokens if tokens is None else tokens
    c = wl.cfg
    w0 = gen_w0(spec.m, spec.k, layer_seed(c, layer, T_W0), layer_seed(c, layer, T_OUTLIER),
                wl.w_std, wl.outlier_frac)
    a = gen_a(spec.m, wl.rank, spec.k, layer_seed(c, layer, T_A))
    b = gen_b(wl.rank, spec.k, layer_seed(c, layer, T_B), wl.b_std)
    if with_acts:
        x = gen_act(t, spec.k, layer_seed(c, layer, T_X), 1.0, wl.act_dtype)
        dy = gen_act(t, spec.m, layer_seed(c, layer, T_DY), wl.dy_std, wl.act_dtype)
    else:
        x = dy = None
    return LayerInputs(spec, w0, a, b, x, dy)
