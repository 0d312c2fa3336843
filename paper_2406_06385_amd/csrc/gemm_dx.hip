// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): dX GEMM, packed int4 grid.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_dx_i4(bool grouped, bool zp, const GemmArgs& p, hipStream_t st) { return launch_zg<kDx, false, 0>(grouped, zp, p, st); }

}  // namespace lrqat
