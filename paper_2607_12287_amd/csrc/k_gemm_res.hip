// Instances of the per-layer GEMM with the residual epilogue (the output
// projection: H and the block statistics of LN2).
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_res(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_RES>(cols, a, s); }

}  // namespace incvit
