// Instances of the per-layer GEMM with the FC1 epilogue.
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_fc1(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_FC1>(cols, a, s); }

}  // namespace incvit
