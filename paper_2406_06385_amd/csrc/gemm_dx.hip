// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): launch_dx, launch_dx_grp.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_dx(const GemmArgs& p, hipStream_t st) { return launch_variant<kDx, false, false>(p, st); }
hipError_t launch_dx_grp(const GemmArgs& p, hipStream_t st) { return launch_variant<kDx, false, true>(p, st); }

}  // namespace lrqat
