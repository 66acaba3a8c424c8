// Instances of the per-layer GEMM with the OPROJ epilogue.
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_oproj(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_OPROJ>(cols, a, s); }

}  // namespace incvit
