// Dispatch of the per-layer GEMMs; each epilogue's instances are compiled in a
// file of their own (k_gemm_*.hip) so the builds run in parallel.
#include "common.hpp"

namespace incvit {

hipError_t launch_gemm_qkv(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_fc1(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_part(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_res(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_att(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_down(int cols, const GemmArgs& a, hipStream_t s);

hipError_t launch_gemm(int epi, int cols, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_gemm_qkv(cols, a, s);
    case EPI_FC1: return launch_gemm_fc1(cols, a, s);
    case EPI_RES: return launch_gemm_res(cols, a, s);
    case EPI_ATT: return launch_gemm_att(cols, a, s);
    case EPI_DOWN: return launch_gemm_down(cols, a, s);
    default: return launch_gemm_part(cols, a, s);
  }
}

}  // namespace incvit
