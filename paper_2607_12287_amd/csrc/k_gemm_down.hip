// Instances of the per-layer GEMM for the MLP down projection with its
// residual and cache write in the epilogue (unsplit K).
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_down(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_DOWN>(cols, a, s); }

}  // namespace incvit
