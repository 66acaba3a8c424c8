// Patch embedding + position, and the per-token cosine similarity against the
// cached reference (paper §III-B, eq. 3).
//
// Selection must be bit-reproducible, so both are computed in a fixed fp32
// order with explicitly rounded operations (no contraction):
//   T[i][d] = fma-chain over k = 0..P-1 of x_i[k] * W_pe[k][d], started at
//             b_pe[d], then one fp32 add of Pos[i][d];
//   cos: lane j of a wave sums the terms d = j, j+64, ... with fma, the 64
//        lane partials are combined by the halving tree (offsets 32..1), then
//        dot / max(sqrt(|a|^2) * sqrt(|b|^2), 1e-8).
// This is fp32 vector-ALU work (P*D fma per token).
#include "common.hpp"

namespace incvit {

// Workgroup: 16 tokens x 64 columns; wave w computes tokens 4w..4w+3 of the
// tile, lane = column.  k is staged through LDS in tiles of 64; the next
// tile's global loads are issued before the current tile is computed.
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  __shared__ __align__(16) float sx[64][16];  // [k][token]
  __shared__ __align__(16) float sw[64][64];  // [k][column]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int v = blockIdx.z, tok0 = blockIdx.x * 16, c0 = blockIdx.y * 64;
  const int N = a.N, P = a.P, D = a.D;

  if (blockIdx.x == 0 && blockIdx.y == 0) {
    for (int i = tid; i < a.nzero && v == 0; i += 256) a.zero[i] = 0;
    if (a.ident_idx) {
      for (int i = tid; i < N; i += 256) a.ident_idx[v * N + i] = i;
      if (tid == 0) a.ident_count[v] = N;
    }
  }

  const int d = c0 + lane;
  const float* xp = a.patches + (size_t)v * N * P;
  // this thread's share of a tile: 4 patch values and 16 weights
  float rx[4], rw[16];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j, t = e >> 6, k = kt + (e & 63), tok = tok0 + t;
      rx[j] = (tok < N && k < P) ? xp[(size_t)tok * P + k] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int e = tid + 256 * j, k = kt + (e >> 6), col = c0 + (e & 63);
      float wv = 0.0f;
      if (k < P && col < D) {
        const size_t i = (size_t)k * D + col;
        wv = a.dtype ? bf2f(static_cast<const uint16_t*>(a.w_pe)[i]) : static_cast<const float*>(a.w_pe)[i];
      }
      rw[j] = wv;
    }
  };
  float acc[4];
  const float bias = d < D ? a.b_pe[d] : 0.0f;
  float posv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    acc[r] = bias;
    const int tok = tok0 + 4 * w + r;
    posv[r] = (tok < N && d < D) ? a.pos[(size_t)tok * D + d] : 0.0f;
  }
  fetch(0);
  for (int kt = 0; kt < P; kt += 64) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j;
      sx[e & 63][e >> 6] = rx[j];
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int e = tid + 256 * j;
      sw[e >> 6][e & 63] = rw[j];
    }
    __syncthreads();
    if (kt + 64 < P) fetch(kt + 64);  // in flight while this tile computes
    const int kmax = min(64, P - kt);
#pragma unroll 8
    for (int kk = 0; kk < kmax; ++kk) {
      const float wv = sw[kk][lane];
      const float4 xv = *reinterpret_cast<const float4*>(&sx[kk][4 * w]);
      acc[0] = __fmaf_rn(xv.x, wv, acc[0]);
      acc[1] = __fmaf_rn(xv.y, wv, acc[1]);
      acc[2] = __fmaf_rn(xv.z, wv, acc[2]);
      acc[3] = __fmaf_rn(xv.w, wv, acc[3]);
    }
    __syncthreads();
  }
  if (d < D) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = tok0 + 4 * w + r;
      if (tok < N) a.t0[((size_t)v * N + tok) * D + d] = __fadd_rn(acc[r], posv[r]);
    }
  }
}

// One wave per token: cos(T0[v][i], ref[v][i]); the wave's loads go out in one batch.
__global__ __launch_bounds__(256) void sim_kernel(SimArgs a) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gt = blockIdx.x * 4 + w;
  if (gt >= a.B * a.N) return;
  const int v = gt / a.N, tok = gt - v * a.N;
  const float* x = a.t0 + (size_t)gt * a.D;
  const float* y = reinterpret_cast<const float*>(a.caches.p[v] + a.ref_off) + (size_t)tok * a.D;
  constexpr int kPer = kMaxDim / 64;
  float xv[kPer], yv[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int d = lane + 64 * j;
    xv[j] = d < a.D ? x[d] : 0.0f;
    yv[j] = d < a.D ? y[d] : 0.0f;
  }
  float pd = 0.0f, pa = 0.0f, pb = 0.0f;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {  // d = lane + 64 j in increasing d; zero pads add nothing
    if (lane + 64 * j < a.D) {
      pd = __fmaf_rn(xv[j], yv[j], pd);
      pa = __fmaf_rn(xv[j], xv[j], pa);
      pb = __fmaf_rn(yv[j], yv[j], pb);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    pd = __fadd_rn(pd, __shfl_down(pd, off, 64));
    pa = __fadd_rn(pa, __shfl_down(pa, off, 64));
    pb = __fadd_rn(pb, __shfl_down(pb, off, 64));
  }
  if (lane == 0) {
    const float denom = __fmul_rn(__fsqrt_rn(pa), __fsqrt_rn(pb));
    a.sim[gt] = __fdiv_rn(pd, fmaxf(denom, 1e-8f));
  }
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  dim3 grid((a.N + 15) / 16, (a.D + 63) / 64, a.B);
  (void)launch_k(embed_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sim(const SimArgs& a, hipStream_t s) {
  dim3 grid((a.B * a.N + 3) / 4);
  (void)launch_k(sim_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace incvit
