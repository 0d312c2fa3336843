// Instantiations of the bf16 MFMA GEMM (gemm_impl.h): dW GEMM with the G epilogue, group-wise scales.
#include "gemm_impl.h"

namespace lrqat {

hipError_t launch_dw_grp(const GemmArgs& p, hipStream_t st) { return launch_variant<kDw, false, true, 0>(p, st); }

}  // namespace lrqat
