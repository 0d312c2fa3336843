// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): launch_dw_act, launch_dw_act_grp.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_dw_act(const GemmArgs& p, hipStream_t st) { return launch_variant<kDw, true, false>(p, st); }
hipError_t launch_dw_act_grp(const GemmArgs& p, hipStream_t st) { return launch_variant<kDw, true, true>(p, st); }

}  // namespace lrqat
