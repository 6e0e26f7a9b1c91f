// Prefill GEMM instantiation: LdsSquare (see gemm_lds.h).
#include "gemm_lds.h"

namespace nvfp4 {

hipError_t launch_lds_square(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end, bool out_f32,
                            hipStream_t stream) {
  return launch_lds<LdsSquare>(o, p, n_begin, n_end, out_f32, stream);
}

}  // namespace nvfp4
