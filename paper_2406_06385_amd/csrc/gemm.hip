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

hipError_t launch_gemm(GemmVariant v, bool act, bool grouped, const GemmArgs& p, hipStream_t st) {
  switch (v) {
    case kFwd:
      if (act) return grouped ? launch_fwd_act_grp(p, st) : launch_fwd_act(p, st);
      return grouped ? launch_fwd_grp(p, st) : launch_fwd(p, st);
    case kDx:
      return grouped ? launch_dx_grp(p, st) : launch_dx(p, st);
    case kDw:
      if (act) return grouped ? launch_dw_act_grp(p, st) : launch_dw_act(p, st);
      return grouped ? launch_dw_grp(p, st) : launch_dw(p, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_reduce(const float* part, int64_t nparts, int64_t n, float* out, float c, int accumulate,
                         hipStream_t st) {
  k_reduce<<<unsigned((n + 255) / 256), 256, 0, st>>>(part, nparts, n, out, c, accumulate);
  return hipGetLastError();
}

}  // namespace lrqat
