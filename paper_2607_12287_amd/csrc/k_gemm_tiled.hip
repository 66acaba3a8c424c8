// Instances of the large-row GEMM (gemm_tiled.hpp) for every epilogue.
#include "gemm_tiled.hpp"

namespace incvit {

hipError_t launch_gemm_tiled(int epi, const GemmArgs& a, int rows, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_tiled_epi<EPI_QKV>(a, rows, s);
    case EPI_FC1: return launch_tiled_epi<EPI_FC1>(a, rows, s);
    case EPI_RES: return launch_tiled_epi<EPI_RES>(a, rows, s);
    case EPI_ATT: return launch_tiled_epi<EPI_ATT>(a, rows, s);
    case EPI_DOWN: return launch_tiled_epi<EPI_DOWN>(a, rows, s);
    default: return launch_tiled_epi<EPI_PART>(a, rows, s);
  }
}

}  // namespace incvit
