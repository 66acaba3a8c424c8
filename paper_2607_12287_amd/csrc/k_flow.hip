// The compressed 2-step flow update of the action expert (paper §III-C): the
// Euler sum of the solver's step velocities, modelled with two anchor
// velocities, collapses to x_T = x_0 + alpha v_0 + beta v_7 + b per sample.
// Elementwise fp32, evaluated as fma(beta, v7, fma(alpha, v0, x0)) + b; HBM /
// launch bound: 16-byte loads where the sample length allows, grid-stride.
#include "common.hpp"

namespace incvit {

template <bool VEC>
__global__ __launch_bounds__(256) void flow_kernel(FlowArgs a) {
  const long per = VEC ? a.n / 4 : a.n;  // units per sample
  const long total = (long)a.S * per;
  for (long u = (long)blockIdx.x * blockDim.x + threadIdx.x; u < total; u += (long)gridDim.x * blockDim.x) {
    const int s = (int)(u / per);
    const float al = a.alpha[s], be = a.beta[s];
    if constexpr (VEC) {
      const float4 x = reinterpret_cast<const float4*>(a.x0)[u];
      const float4 p = reinterpret_cast<const float4*>(a.v0)[u];
      const float4 q = reinterpret_cast<const float4*>(a.v7)[u];
      const float4 r = reinterpret_cast<const float4*>(a.b)[u];
      float4 o;
      o.x = __fadd_rn(__fmaf_rn(be, q.x, __fmaf_rn(al, p.x, x.x)), r.x);
      o.y = __fadd_rn(__fmaf_rn(be, q.y, __fmaf_rn(al, p.y, x.y)), r.y);
      o.z = __fadd_rn(__fmaf_rn(be, q.z, __fmaf_rn(al, p.z, x.z)), r.z);
      o.w = __fadd_rn(__fmaf_rn(be, q.w, __fmaf_rn(al, p.w, x.w)), r.w);
      reinterpret_cast<float4*>(a.xT)[u] = o;
    } else {
      a.xT[u] = __fadd_rn(__fmaf_rn(be, a.v7[u], __fmaf_rn(al, a.v0[u], a.x0[u])), a.b[u]);
    }
  }
}

hipError_t launch_flow(const FlowArgs& a, hipStream_t s) {
  const bool vec = a.n % 4 == 0 && ((uintptr_t)a.x0 | (uintptr_t)a.v0 | (uintptr_t)a.v7 | (uintptr_t)a.b |
                                    (uintptr_t)a.xT) % 16 == 0;
  const long units = (long)a.S * (vec ? a.n / 4 : a.n);
  const dim3 grid((unsigned)std::min<long>((units + 255) / 256, 2048));
  if (vec) return launch_k(flow_kernel<true>, grid, dim3(256), 0, s, a);
  return launch_k(flow_kernel<false>, grid, dim3(256), 0, s, a);
}

}  // namespace incvit
