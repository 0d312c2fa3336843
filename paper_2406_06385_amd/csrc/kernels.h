// Kernel argument blocks and host-side launchers of the LR-QAT library.
#pragma once

#include "common.h"

namespace lrqat {

// Integer grid pass (reconstruction / merge).
struct GridArgs {
  const uint8_t* phi0;   // Phi0: int8 [m][ld_phi] (fixed point) or uint8 [m][ld_phi] packed
  int64_t ld_phi;        // bytes per row of phi0
  const float* A;        // [m][r]
  const float* B;        // [r][k]
  int64_t m, k;
  int r;
  float c;               // alpha / r
  double c64;            // alpha / r in float64 (for the exact re-decision)
  int bits;
  int packed;            // 1: Phi0 is double-packed INT-b
  uint8_t* qout;         // packed q [m][ldq]
  int64_t ldq;           // bytes per row of qout
  int64_t kq;            // columns written per row of qout (>= k; columns >= k are 0)
  uint16_t* mout;        // clip-mask bits: bit (row % 16) of word [row / 16][col] (nullable)
  int64_t ldm;           // words per 16-row block of mout (>= kq)
  float tau_coef;        // set by launch_grid: error-bound coefficient of the float32 delta
  int nit;               // set by launch_grid: 16-row rounds per wave
};

// bf16 MFMA GEMM family.  C[M][N] = sum_K a(M, K) b(K, N) with the operand
// sources and epilogue chosen by the kernel variant.
enum GemmVariant { kFwd = 0, kDx = 1, kDw = 2 };

struct GemmArgs {
  int64_t M, N, K;
  const void* a;          // kFwd: X bf16 [T][k] or n int8 [T][lda]; kDx: dY [T][m]; kDw: dY [T][m]
  int64_t lda;
  const void* b;          // kFwd/kDx: packed q [m][ldb]; kDw: X bf16 [T][k] or n int8 [T][ldb]
  int64_t ldb;
  const float* s;         // weight scale [m] or [m][ngroups]
  int64_t gsize, ngroups;
  const float* sx;        // per-token activation scale [T] (W4A8) or null
  void* out;              // kFwd: Y [T][m]; kDx: dX [T][k]
  int64_t ldo;
  const uint16_t* mask;   // kDw: clip-mask bits, bit (row % 16) of word [row / 16][col]
  int64_t ldm;            // words per 16-row block
  const float* Am;        // kDw: A [m][r]
  const float* Bm;        // kDw: B [r][k]
  int r;
  float* dA_part;         // kDw: [ceil(N/256)][M][r]
  float* dB_part;         // kDw: [ceil(M/256)][r][N]
};

constexpr int GEMM_BM = 256, GEMM_BN = 256, GEMM_BK = 64;

hipError_t launch_minmax_scale(const float* W0, int64_t m, int64_t k, int64_t gsize, int bits, float* s0,
                               hipStream_t st);
hipError_t launch_encode(const float* W0, const float* s0, int64_t m, int64_t k, int64_t gsize, int bits,
                         int packed, void* phi0, hipStream_t st);
hipError_t launch_grid(const GridArgs& a, hipStream_t st);
hipError_t launch_act_quant(const uint16_t* X, int64_t T, int64_t k, int8_t* n, int64_t ldn, float* sx,
                            hipStream_t st);
hipError_t launch_gemm(GemmVariant v, bool act, bool grouped, const GemmArgs& p, hipStream_t st);
// per-variant launchers (gemm_fwd.hip, gemm_fwd_act.hip, gemm_dx.hip, gemm_dw.hip, gemm_dw_act.hip)
hipError_t launch_fwd(const GemmArgs& p, hipStream_t st);
hipError_t launch_fwd_grp(const GemmArgs& p, hipStream_t st);
hipError_t launch_fwd_act(const GemmArgs& p, hipStream_t st);
hipError_t launch_fwd_act_grp(const GemmArgs& p, hipStream_t st);
hipError_t launch_dx(const GemmArgs& p, hipStream_t st);
hipError_t launch_dx_grp(const GemmArgs& p, hipStream_t st);
hipError_t launch_dw(const GemmArgs& p, hipStream_t st);
hipError_t launch_dw_grp(const GemmArgs& p, hipStream_t st);
hipError_t launch_dw_act(const GemmArgs& p, hipStream_t st);
hipError_t launch_dw_act_grp(const GemmArgs& p, hipStream_t st);
hipError_t launch_reduce(const float* part, int64_t nparts, int64_t n, float* out, float c, int accumulate,
                         hipStream_t st);
struct Reduce2Args {        // side 0: dA, side 1: dB
  const float* part[2];     // [nparts][n] partial sums
  int64_t nparts[2], n[2];
  float* out[2];
  int vec[2];               // 16-byte aligned rows and n % 4 == 0
  float c;
  int accumulate;
};
hipError_t launch_reduce2(const Reduce2Args& ra, hipStream_t st);

// float32 activation path (simple tiled FMA kernels).
struct F32Args {
  int64_t T, m, k;
  int r;
  float c;
  const float* X;
  const float* dY;
  const uint8_t* q;       // packed q [m][ldq]
  int64_t ldq;
  const uint16_t* mask;   // clip-mask bits, bit (row % 16) of word [row / 16][col]
  int64_t ldm;            // words per 16-row block
  const float* s;
  int64_t gsize, ngroups;
  const float* A;
  const float* B;
  float* G;               // workspace [m][k]
};
hipError_t launch_f32_forward(const F32Args& a, float* Y, hipStream_t st);
hipError_t launch_f32_dx(const F32Args& a, float* dX, hipStream_t st);
hipError_t launch_f32_dw(const F32Args& a, float* dA, float* dB, int accumulate, hipStream_t st);

}  // namespace lrqat
