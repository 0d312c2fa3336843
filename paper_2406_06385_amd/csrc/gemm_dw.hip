// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): launch_dw, launch_dw_grp.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_dw(const GemmArgs& p, hipStream_t st) { return launch_variant<kDw, false, false>(p, st); }
hipError_t launch_dw_grp(const GemmArgs& p, hipStream_t st) { return launch_variant<kDw, false, true>(p, st); }

}  // namespace lrqat
