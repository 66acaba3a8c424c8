// Patch embedding + position, the first-layer key score, and the per-token
// cosine similarity against the cached reference (paper §III-B, eq. 3).
//
// Selection must be bit-reproducible, so all three are computed in a fixed
// fp32 order with explicitly rounded operations (no contraction):
//   T[i][d] = fma-chain over k = 0..P-1 of x_i[k] * W_pe[k][d], started at
//             b_pe[d], then one fp32 add of Pos[i][d];
//   key score: x = S(T[i]); mean and variance of x from 64 lane partials
//        (lane j takes d = j, j+64, ... in increasing d: adds for the sum, fma
//        of (x - mean)^2 for the variance) and the halving tree, each / D;
//        rstd = 1 / sqrt(var + eps); n_d = fma((x_d - mean) * rstd, g_d, b_d);
//        key[e] = fma-chain over d of n_d * W_K[d][e] started at b_K[e];
//   cos: lane j of a wave sums the terms d = j, j+64, ... with fma, the 64
//        lane partials are combined by the halving tree (offsets 32..1), then
//        dot / max(sqrt(|a|^2) * sqrt(|b|^2), 1e-8).
// This is fp32 vector-ALU work (P*D fma per token, D*D more for the key).
#include "common.hpp"

namespace incvit {

// 16 consecutive bytes of weights and their values as floats
__device__ __forceinline__ void load16(V8<uint16_t>& v, const uint16_t* p) { v.load(p); }
__device__ __forceinline__ void load16(V8<float>& v, const float* p) {
  v.a = __builtin_bit_cast(float4, *(const INCVIT_GLOBAL f32x4_t*)p);
}
__device__ __forceinline__ void unpack16(float* f, const V8<uint16_t>& v) {
  const uint32_t q[4] = {v.v.x, v.v.y, v.v.z, v.v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = __uint_as_float(q[e] << 16);
    f[2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack16(float* f, const V8<float>& v) {
  f[0] = v.a.x; f[1] = v.a.y; f[2] = v.a.z; f[3] = v.a.w;
}

// Workgroup: 16 tokens x 64 columns; wave w computes tokens 4w..4w+3 of the
// tile, lane = column.  k is staged through LDS in tiles of 64.  Every global
// load is unconditional (clamped addresses; values past P are loaded but never
// used because the k loop stops at P) and issued two tiles ahead, so a tile's
// data arrives while the two before it are computed.
template <class T>
__device__ __forceinline__ void embed_body(const EmbedArgs& a) {
  constexpr int WV = 16 / sizeof(T);  // weights per 16-byte load
  constexpr int WL = 64 * 64 / (256 * WV);  // weight loads per thread per tile
  __shared__ __align__(16) float sx[64][16];  // [k][token]
  __shared__ __align__(16) float sw[64][64];  // [k][column]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // Workgroups are dealt to the 8 XCDs round robin by linear launch index, and
  // each XCD has its own L2.  Renumber them XCD-major (a bijection) and take
  // (stream, column block, token group) from the new number, so that the
  // workgroups of one column block sit on one XCD (at most two): its weights
  // come from HBM once rather than once per XCD.
  const int ntg = gridDim.x, ncb = gridDim.y;
  const int total = ntg * ncb * gridDim.z;
  const int i = blockIdx.x + ntg * (blockIdx.y + ncb * blockIdx.z);
  const int x = i % 8, q = total / 8, rem = total % 8;
  const int pos = x * q + min(x, rem) + i / 8;
  const int v = pos / (ncb * ntg), cb = (pos / ntg) % ncb, tg = pos % ntg;
  const int tok0 = tg * 16, c0 = cb * 64;
  const int N = a.N, P = a.P, D = a.D;

  if (tg == 0 && cb == 0) {
    for (int k = tid; k < a.nzero && v == 0; k += 256) a.zero[k] = 0;
    if (a.ident_idx) {
      for (int k = tid; k < N; k += 256) a.ident_idx[v * N + k] = k;
      if (tid == 0) a.ident_count[v] = N;
    }
  }

  const int d = c0 + lane;
  const float* xp = a.patches + (size_t)v * N * P;
  const T* wp = static_cast<const T*>(a.w_pe);
  // this thread's share of a tile: 4 patch values (token e/64, k e%64) and WL
  // 16-byte runs of weights (row k, WV consecutive columns)
  struct Tile {
    float x[4];
    V8<T> wv[WL > 0 ? WL : 1];
  };
  auto fetch = [&](Tile& t, int kt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j;
      const int tok = min(tok0 + (e >> 6), N - 1), k = min(kt + (e & 63), P - 1);
      t.x[j] = xp[(size_t)tok * P + k];
    }
#pragma unroll
    for (int j = 0; j < WL; ++j) {
      const int e = tid + 256 * j;                 // run index in the tile
      const int k = min(kt + e / (64 / WV), P - 1);
      const int col = min(c0 + (e % (64 / WV)) * WV, D - WV);
      load16(t.wv[j], wp + (size_t)k * D + col);
    }
  };
  auto stage = [&](const Tile& t) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j;
      sx[e & 63][e >> 6] = t.x[j];
    }
#pragma unroll
    for (int j = 0; j < WL; ++j) {
      const int e = tid + 256 * j;
      float f[WV];
      unpack16(f, t.wv[j]);
#pragma unroll
      for (int q = 0; q < WV; ++q) sw[e / (64 / WV)][(e % (64 / WV)) * WV + q] = f[q];
    }
  };

  float acc[4];
  const float bias = a.b_pe[min(d, D - 1)];
  float posv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    acc[r] = bias;
    const int tok = min(tok0 + 4 * w + r, N - 1);
    if (a.pos) posv[r] = a.pos[(size_t)tok * D + min(d, D - 1)];
  }
  Tile t0, t1;
  fetch(t0, 0);
  fetch(t1, 64);
  for (int kt = 0; kt < P; kt += 64) {
    stage(t0);
    __syncthreads();
    t0 = t1;
    fetch(t1, kt + 128);  // two tiles ahead (clamped past the end)
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
      if (tok < N) a.t0[((size_t)v * N + tok) * D + d] = a.pos ? __fadd_rn(acc[r], posv[r]) : acc[r];
    }
  }
}

template <class T>
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  embed_body<T>(a);
}

// The key projection of the key score: the same fixed-order product with
// x = LayerNorm rows, K = D, W = W_K of layer 0, no position term.
template <class T>
__global__ __launch_bounds__(256) void keyproj_kernel(EmbedArgs a) {
  embed_body<T>(a);
}

// Correctly rounded fp32 square root.  HIP's __fsqrt_rn is the bare hardware
// square root (about 1 ulp) unless OCML's rounded operations are enabled;
// __builtin_sqrtf compiles to the hardware estimate plus the fma correction
// that rounds it correctly (the fp32 divide is correctly rounded by default).
__device__ __forceinline__ float sqrt_rn(float x) { return __builtin_sqrtf(x); }

// Sum of the 64 lane values by the halving tree; lane 0's value is the
// result, broadcast to the wave.
__device__ __forceinline__ float tree64(float p) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) p = __fadd_rn(p, __shfl_down(p, off, 64));
  return __shfl(p, 0, 64);
}

// One wave per token: n = LayerNorm 1 of layer 0 on S(T0[token]), fixed order.
template <class T>
__global__ __launch_bounds__(256) void keyln_kernel(KeyLnArgs a) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int row = blockIdx.x * 4 + w;
  if (row >= a.rows) return;
  const int D = a.D;
  const float* x = a.t0 + (size_t)row * D;
  constexpr int kPer = kMaxDim / 64;
  float xv[kPer], g[kPer], b[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int d = lane + 64 * j;
    xv[j] = d < D ? Elem<T>::rnd(x[d]) : 0.0f;
    g[j] = d < D ? a.ln_g[d] : 0.0f;
    b[j] = d < D ? a.ln_b[d] : 0.0f;
  }
  float p = 0.0f;
#pragma unroll
  for (int j = 0; j < kPer; ++j)
    if (lane + 64 * j < D) p = __fadd_rn(p, xv[j]);
  const float mean = __fdiv_rn(tree64(p), (float)D);
  float q = 0.0f;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    xv[j] = __fsub_rn(xv[j], mean);
    if (lane + 64 * j < D) q = __fmaf_rn(xv[j], xv[j], q);
  }
  const float var = __fdiv_rn(tree64(q), (float)D);
  const float rstd = __fdiv_rn(1.0f, sqrt_rn(__fadd_rn(var, a.eps)));
  float* out = a.out + (size_t)row * D;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int d = lane + 64 * j;
    if (d < D) out[d] = __fmaf_rn(__fmul_rn(xv[j], rstd), g[j], b[j]);
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
    const float denom = __fmul_rn(sqrt_rn(pa), sqrt_rn(pb));
    a.sim[gt] = __fdiv_rn(pd, fmaxf(denom, 1e-8f));
  }
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  dim3 grid((a.N + 15) / 16, (a.D + 63) / 64, a.B);
  if (a.dtype) return launch_k(embed_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  return launch_k(embed_kernel<float>, grid, dim3(256), 0, s, a);
}

hipError_t launch_keyproj(const EmbedArgs& a, hipStream_t s) {
  dim3 grid((a.N + 15) / 16, (a.D + 63) / 64, a.B);
  if (a.dtype) return launch_k(keyproj_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  return launch_k(keyproj_kernel<float>, grid, dim3(256), 0, s, a);
}

hipError_t launch_keyln(const KeyLnArgs& a, hipStream_t s) {
  dim3 grid((a.rows + 3) / 4);
  if (a.dtype) return launch_k(keyln_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  return launch_k(keyln_kernel<float>, grid, dim3(256), 0, s, a);
}

hipError_t launch_sim(const SimArgs& a, hipStream_t s) {
  dim3 grid((a.B * a.N + 3) / 4);
  (void)launch_k(sim_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace incvit
