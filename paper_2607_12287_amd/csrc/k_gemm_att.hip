// Instances of the per-layer GEMM that write the attention branch into the
// cache (output projection of the all-rows MLP reading).
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_att(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_ATT>(cols, a, s); }

}  // namespace incvit
