// Dispatch of the per-layer GEMMs (each epilogue's instances are compiled in a
// file of their own, k_gemm_*.hip, so the builds run in parallel) and the row
// kernel that finishes a split-K MLP down projection.
#include "common.hpp"

namespace incvit {

hipError_t launch_gemm_qkv(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_oproj(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_fc1(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_fc2(int cols, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_part(int cols, const GemmArgs& a, hipStream_t s);

hipError_t launch_gemm(int epi, int cols, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_gemm_qkv(cols, a, s);
    case EPI_OPROJ: return launch_gemm_oproj(cols, a, s);
    case EPI_FC1: return launch_gemm_fc1(cols, a, s);
    case EPI_FC2: return launch_gemm_fc2(cols, a, s);
    default: return launch_gemm_part(cols, a, s);
  }
}

__device__ __forceinline__ void put4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void put4(uint16_t* p, float4 v) {
  const uint32_t lo = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  const uint32_t hi = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  *reinterpret_cast<uint2*>(p) = make_uint2(lo, hi);
}
__device__ __forceinline__ float4 rnd4(float4 v, float) { return v; }
__device__ __forceinline__ float4 rnd4(float4 v, uint16_t) {
  return make_float4(bf2f(f2bf(v.x)), bf2f(f2bf(v.y)), bf2f(f2bf(v.z)), bf2f(f2bf(v.w)));
}

// One wave per compact row r: Z_{l+1}[r] = S(H[r] + ((P_0[r] + P_1[r]) + ...) + b_2),
// written compact and into X^{l+1} of the row's stream.  Every load is issued
// before M is known (the buffers are padded past every launched row).
template <class T, int S>
__global__ __launch_bounds__(256) void fix_kernel(FixArgs a) {
  constexpr int kPer = kMaxDim / 256;  // float4 per lane
  const int lane = threadIdx.x & 63, r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int M = a.meta->m;
  const int D = a.sh.D, D4 = D / 4;
  const RowInfo ri = a.rows[r];
  const float4* h = reinterpret_cast<const float4*>(a.h + (size_t)r * D);
  const float4* bias = reinterpret_cast<const float4*>(a.bias);
  float4 p[S][kPer], hv[kPer], bv[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int q = min(lane + 64 * j, D4 - 1);
#pragma unroll
    for (int s = 0; s < S; ++s)
      p[s][j] = reinterpret_cast<const float4*>(a.part + ((size_t)s * a.mpad + r) * D)[q];
    hv[j] = h[q];
    bv[j] = bias[q];
  }
  if (r >= M) return;
  T* z = static_cast<T*>(a.z) + (size_t)r * D;
  T* x = x_row<T>(ri.cache, a.cl, a.sh, a.layer + 1, ri.tok);
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int q = lane + 64 * j;
    if (q < D4) {
      float4 t = p[0][j];
#pragma unroll
      for (int s = 1; s < S; ++s) {
        t.x += p[s][j].x; t.y += p[s][j].y; t.z += p[s][j].z; t.w += p[s][j].w;
      }
      t.x += bv[j].x; t.y += bv[j].y; t.z += bv[j].z; t.w += bv[j].w;
      const float4 o = rnd4(make_float4(hv[j].x + t.x, hv[j].y + t.y, hv[j].z + t.z, hv[j].w + t.w), T());
      put4(z + 4 * q, o);
      put4(x + 4 * q, o);
    }
  }
}

hipError_t launch_fix(const FixArgs& a, int mmax, hipStream_t s) {
  const dim3 grid(max(1, (mmax + 3) / 4));
  switch (a.ksplit * 2 + a.sh.dtype) {
    case 4: return launch_k(fix_kernel<float, 2>, grid, dim3(256), 0, s, a);
    case 5: return launch_k(fix_kernel<uint16_t, 2>, grid, dim3(256), 0, s, a);
    case 6: return launch_k(fix_kernel<float, 3>, grid, dim3(256), 0, s, a);
    case 7: return launch_k(fix_kernel<uint16_t, 3>, grid, dim3(256), 0, s, a);
    case 8: return launch_k(fix_kernel<float, 4>, grid, dim3(256), 0, s, a);
    case 9: return launch_k(fix_kernel<uint16_t, 4>, grid, dim3(256), 0, s, a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace incvit
