// Instances of the per-layer GEMM with the QKV epilogue.
#include "gemm.hpp"

namespace incvit {

hipError_t launch_gemm_qkv(int cols, const GemmArgs& a, hipStream_t s) { return launch_gemm_epi<EPI_QKV>(cols, a, s); }

}  // namespace incvit
