// Launchers of the setup-side initialisation kernels (init.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lrqat {

constexpr int64_t kLpMaxGroup = 16384;  // weights of one row or group the L^p search holds in LDS
constexpr int kLoftqMaxRank = 48;        // the subspace (rank + 16) and its Gram matrix fit one block
constexpr int kLoftqOversample = 16;

// s0[row][grp] by L^p range search over n_grid clipping ratios; jbest (nullable) the chosen ratio index.
hipError_t launch_lp_search(const float* W0, int64_t m, int64_t k, int64_t gsize, int bits, float p, int n_grid,
                            float* s0, int32_t* jbest, hipStream_t st);
size_t loftq_workspace(int64_t m, int64_t k, int l);
hipError_t launch_loftq(const float* W0, const float* s0, int64_t m, int64_t k, int64_t gsize, int bits, int r,
                        int l, double c, int n_iter, uint8_t* phi0, float* A, float* B, float* sigma, void* ws,
                        hipStream_t st);

}  // namespace lrqat
