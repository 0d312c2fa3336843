// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): Forward GEMM, packed int4 grid.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_fwd_i4(bool grouped, bool zp, const GemmArgs& p, hipStream_t st) { return launch_zg<kFwd, false, 0>(grouped, zp, p, st); }

}  // namespace lrqat
