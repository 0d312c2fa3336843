// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): Forward GEMM, int8 grid (5..7 bits).
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_fwd_i8(bool grouped, bool zp, const GemmArgs& p, hipStream_t st) { return launch_zg<kFwd, false, kOptQ8>(grouped, zp, p, st); }

}  // namespace lrqat
