// Prefill GEMM instantiation: LdsSquareSuper, bf16 output (see gemm_lds.h).
#include "gemm_lds.h"

namespace nvfp4 {

hipError_t launch_lds_super_bf16(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                 hipStream_t stream) {
  return launch_lds_as<LdsSquareSuper, false>(o, p, n_begin, n_end, stream);
}

}  // namespace nvfp4
