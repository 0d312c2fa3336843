// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): Forward GEMM on int8 activation codes (W4A8), packed int4 grid.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_fwd_act_i4(bool grouped, bool zp, const GemmArgs& p, hipStream_t st) { return launch_zg<kFwd, true, 0>(grouped, zp, p, st); }

}  // namespace lrqat
