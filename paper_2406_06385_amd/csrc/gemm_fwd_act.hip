// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): launch_fwd_act, launch_fwd_act_grp.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_fwd_act(const GemmArgs& p, hipStream_t st) { return launch_variant<kFwd, true, false>(p, st); }
hipError_t launch_fwd_act_grp(const GemmArgs& p, hipStream_t st) { return launch_variant<kFwd, true, true>(p, st); }

}  // namespace lrqat
