// Instances of the per-layer GEMM that write split-K partial sums (the MLP
// down projection, whose K = F is long).
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_part(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_PART>(cols, a, s); }

}  // namespace incvit
