// Dispatch of the bf16 MFMA GEMM variants (one translation unit per variant
// family, see gemm_impl.h) and the deterministic reduction of the rank-r
// partial products.
#include "kernels.h"

namespace lrqat {

// Deterministic sum of partial buffers: out = (accumulate ? out : 0) + c * sum_p part[p].
__global__ __launch_bounds__(256) void k_reduce(const float* __restrict__ part, int64_t nparts, int64_t n,
                                                float* __restrict__ out, float c, int accumulate) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  float s = 0.f;
  for (int64_t q = 0; q < nparts; ++q) s += part[q * n + idx];
  out[idx] = (accumulate ? out[idx] : 0.f) + c * s;
}

// Both rank-r gradients in one launch: out = (accumulate ? out : 0) + c * sum_p part[p] for
// dA (side 0) and dB (side 1).  Four consecutive elements per thread; the partial buffers
// are summed in a fixed order (two interleaved running sums), so results are deterministic.
__global__ __launch_bounds__(256) void k_reduce2(Reduce2Args ra) {
  const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t nt0 = (ra.n[0] + 3) / 4;
  const int side = t < nt0 ? 0 : 1;
  const int64_t idx = 4 * (side ? t - nt0 : t);
  const int64_t n = ra.n[side], np = ra.nparts[side];
  if (idx >= n) return;
  const float* part = ra.part[side] + idx;
  float* out = ra.out[side] + idx;
  if (ra.vec[side] && idx + 4 <= n) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
    int64_t q = 0;
    for (; q + 2 <= np; q += 2) {
      s0 += *reinterpret_cast<const f32x4*>(part + q * n);
      s1 += *reinterpret_cast<const f32x4*>(part + (q + 1) * n);
    }
    if (q < np) s0 += *reinterpret_cast<const f32x4*>(part + q * n);
    const f32x4 prev = ra.accumulate ? *reinterpret_cast<const f32x4*>(out) : f32x4{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4*>(out) = prev + ra.c * (s0 + s1);
  } else {
    for (int64_t e = 0; e < 4 && idx + e < n; ++e) {
      float s0 = 0.f, s1 = 0.f;
      int64_t q = 0;
      for (; q + 2 <= np; q += 2) {
        s0 += part[q * n + e];
        s1 += part[(q + 1) * n + e];
      }
      if (q < np) s0 += part[q * n + e];
      out[e] = (ra.accumulate ? out[e] : 0.f) + ra.c * (s0 + s1);
    }
  }
}

hipError_t launch_reduce2(const Reduce2Args& ra, hipStream_t st) {
  const int64_t nt = (ra.n[0] + 3) / 4 + (ra.n[1] + 3) / 4;
  k_reduce2<<<unsigned((nt + 255) / 256), 256, 0, st>>>(ra);
  return hipGetLastError();
}

hipError_t launch_gemm(GemmVariant v, bool act, bool grouped, int opt, const GemmArgs& p, hipStream_t st) {
  const bool zp = (opt & kOptZ) != 0, i8 = (opt & kOptQ8) != 0;
  switch (v) {
    case kFwd:
      if (act) return i8 ? launch_fwd_act_i8(grouped, zp, p, st) : launch_fwd_act_i4(grouped, zp, p, st);
      return i8 ? launch_fwd_i8(grouped, zp, p, st) : launch_fwd_i4(grouped, zp, p, st);
    case kDx:
      return i8 ? launch_dx_i8(grouped, zp, p, st) : launch_dx_i4(grouped, zp, p, st);
    case kDw:  // W4A8 runs the dW GEMM on X_hat in bfloat16
      if (act) return hipErrorInvalidValue;
      return grouped ? launch_dw_grp(p, st) : launch_dw_pc(p, st);
  }
  return hipErrorInvalidValue;
}

// ds[row][grp] = (accumulate ? ds : 0) + the partials of the group's 32-column chunks, summed in
// chunk order (deterministic).  One thread per (row, group).
__global__ __launch_bounds__(256) void k_reduce_ds(const float* __restrict__ part, int64_t m, int64_t ldpart,
                                                   int64_t nchunks, int64_t cpg, int64_t ngroups,
                                                   float* __restrict__ ds, int accumulate) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= m * ngroups) return;
  const int64_t row = idx / ngroups, grp = idx % ngroups;
  const int64_t c0 = grp * cpg, c1 = min(nchunks, c0 + cpg);
  const float* src = part + row * ldpart;
  float s0 = 0.f, s1 = 0.f;
  int64_t c = c0;
  for (; c + 2 <= c1; c += 2) {
    s0 += src[c];
    s1 += src[c + 1];
  }
  if (c < c1) s0 += src[c];
  ds[idx] = (accumulate ? ds[idx] : 0.f) + (s0 + s1);
}

hipError_t launch_reduce_ds(const float* part, int64_t m, int64_t ldpart, int64_t nchunks, int64_t chunks_per_group,
                            int64_t ngroups, float* ds, int accumulate, hipStream_t st) {
  const int64_t n = m * ngroups;
  if (n == 0) return hipSuccess;
  k_reduce_ds<<<unsigned((n + 255) / 256), 256, 0, st>>>(part, m, ldpart, nchunks, chunks_per_group, ngroups, ds,
                                                         accumulate);
  return hipGetLastError();
}

// dst[row][0 .. ldd) = src[row][0 .. w) followed by zeros; one thread per destination byte.
__global__ __launch_bounds__(256) void k_repack_rows(const uint8_t* __restrict__ src, int64_t m, int64_t w,
                                                     uint8_t* __restrict__ dst, int64_t ldd) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= m * ldd) return;
  const int64_t row = idx / ldd, col = idx % ldd;
  dst[idx] = col < w ? src[row * w + col] : uint8_t(0);
}

hipError_t launch_repack_rows(const uint8_t* src, int64_t m, int64_t w, uint8_t* dst, int64_t ldd, hipStream_t st) {
  const int64_t n = m * ldd;
  if (n == 0) return hipSuccess;
  k_repack_rows<<<unsigned((n + 255) / 256), 256, 0, st>>>(src, m, w, dst, ldd);
  return hipGetLastError();
}

hipError_t launch_reduce(const float* part, int64_t nparts, int64_t n, float* out, float c, int accumulate,
                         hipStream_t st) {
  k_reduce<<<unsigned((n + 255) / 256), 256, 0, st>>>(part, nparts, n, out, c, accumulate);
  return hipGetLastError();
}

}  // namespace lrqat
