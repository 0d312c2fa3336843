// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): launch_fwd, launch_fwd_grp.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_fwd(const GemmArgs& p, hipStream_t st) { return launch_variant<kFwd, false, false>(p, st); }
hipError_t launch_fwd_grp(const GemmArgs& p, hipStream_t st) { return launch_variant<kFwd, false, true>(p, st); }

}  // namespace lrqat
