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
// the same 16 bytes through a buffer resource (lane offset voff, uniform soff)
__device__ __forceinline__ void bload16(V8<uint16_t>& v, Rsrc r, uint32_t voff, uint32_t soff) { v.bload(r, voff, soff); }
__device__ __forceinline__ void bload16(V8<float>& v, Rsrc r, uint32_t voff, uint32_t soff) {
  v.a = bload16f(r, voff, soff);
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
// tile, lane = column.  k is staged through LDS in tiles of 64, double
// buffered, with one barrier per tile.  A tile's global loads go out two
// tiles of compute ahead into one of three register slots (the loop body is unrolled over
// the slots, so no register copy waits on a load in flight); every load is
// unconditional (clamped addresses; values past P are loaded but never used
// because the k loop stops at P).
template <class T, int NT>
__device__ __forceinline__ void embed_body(const EmbedArgs& a) {
  constexpr int WV = 16 / sizeof(T);  // weights per 16-byte load
  constexpr int WL = 64 * 64 / (256 * WV);  // weight loads per thread per tile
  __shared__ __align__(16) float sx[2][64][16];  // [buffer][k][token]
  __shared__ __align__(16) float sw[2][64][64];  // [buffer][k][column]
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
  // Operands through buffer loads: every lane offset below is fixed for the
  // whole kernel and the tile's k position is a wave-uniform offset, so a
  // fetch needs no address registers.  Reads past the buffer return zero; reads
  // past a row's end (k >= P) are never used because the k loop stops at P.
  const Rsrc rx = make_rsrc(a.patches + (size_t)v * N * P, (uint32_t)((size_t)N * P * 4));
  const Rsrc rw = make_rsrc(a.w_pe, (uint32_t)((size_t)P * D * sizeof(T)));
  uint32_t xoff[4], woff[WL > 0 ? WL : 1];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = tid + 256 * j;
    xoff[j] = (uint32_t)((min(tok0 + (e & 15), N - 1) * P + (e >> 4)) * 4);
  }
#pragma unroll
  for (int j = 0; j < WL; ++j) {
    const int e = tid + 256 * j;
    woff[j] = (uint32_t)(((e / (64 / WV)) * D + min(c0 + (e % (64 / WV)) * WV, D - WV)) * sizeof(T));
  }
  // this thread's share of a tile: 4 patch values (token e%16, k e/16) and WL
  // 16-byte runs of weights (row k, WV consecutive columns)
  struct Tile {
    float x[4];
    V8<T> wv[WL > 0 ? WL : 1];
  };
  auto fetch = [&](Tile& t, int kt) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      t.x[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rx, xoff[j], (uint32_t)kt * 4, 0));
#pragma unroll
    for (int j = 0; j < WL; ++j) bload16(t.wv[j], rw, woff[j], (uint32_t)(kt * D * sizeof(T)));
  };
  auto stage = [&](const Tile& t, int b) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j;
      sx[b][e >> 4][e & 15] = t.x[j];
    }
#pragma unroll
    for (int j = 0; j < WL; ++j) {
      const int e = tid + 256 * j;
      float f[WV];
      unpack16(f, t.wv[j]);
#pragma unroll
      for (int q = 0; q < WV; ++q) sw[b][e / (64 / WV)][(e % (64 / WV)) * WV + q] = f[q];
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
  auto compute = [&](int b, int kmax) {
#pragma unroll 8
    for (int kk = 0; kk < kmax; ++kk) {
      const float wv = sw[b][kk][lane];
      const float4 xv = *reinterpret_cast<const float4*>(&sx[b][kk][4 * w]);
      acc[0] = __fmaf_rn(xv.x, wv, acc[0]);
      acc[1] = __fmaf_rn(xv.y, wv, acc[1]);
      acc[2] = __fmaf_rn(xv.z, wv, acc[2]);
      acc[3] = __fmaf_rn(xv.w, wv, acc[3]);
    }
  };
  Tile tl[3];
  fetch(tl[0], 0);
  fetch(tl[1], 64);
  fetch(tl[2], 128);
  stage(tl[0], 0);
  __syncthreads();
  if constexpr (NT > 0) {
    // NT = ceil(P / 64) tiles, unrolled: every slot and buffer index is a
    // constant, so each wait covers exactly the loads of the tile it stages
#pragma unroll
    for (int it = 0; it < NT; ++it) {
      if (it + 1 < NT) {
#pragma unroll
        for (int kk = 0; kk < 64; ++kk) {  // a full tile
          const float wv = sw[it & 1][kk][lane];
          const float4 xv = *reinterpret_cast<const float4*>(&sx[it & 1][kk][4 * w]);
          acc[0] = __fmaf_rn(xv.x, wv, acc[0]);
          acc[1] = __fmaf_rn(xv.y, wv, acc[1]);
          acc[2] = __fmaf_rn(xv.z, wv, acc[2]);
          acc[3] = __fmaf_rn(xv.w, wv, acc[3]);
        }
        stage(tl[(it + 1) % 3], (it + 1) & 1);
        if (it + 3 < NT) fetch(tl[it % 3], 64 * (it + 3));
        __syncthreads();
      } else {
        compute(it & 1, P - 64 * it);
      }
    }
  } else {
    const int nt = (P + 63) / 64;
    for (int i0 = 0; i0 < nt; i0 += 3) {
#pragma unroll
      for (int s3 = 0; s3 < 3; ++s3) {
        const int it = i0 + s3;
        if (it < nt) {  // uniform
          // tile it is in LDS buffer it & 1; tile it + 1 waits in slot (s3 + 1) % 3
          // and is staged after the compute; slot s3 (tile it, already staged)
          // then takes tile it + 3, whose loads have two tiles of compute to land
          const int b = it & 1;
          compute(b, min(64, P - 64 * it));
          if (it + 1 < nt) stage(tl[(s3 + 1) % 3], b ^ 1);
          fetch(tl[s3], 64 * (it + 3));
          __syncthreads();
        }
      }
    }
  }
  if (d < D) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = tok0 + 4 * w + r;
      if (tok < N) a.t0[((size_t)v * N + tok) * D + d] = a.pos ? __fadd_rn(acc[r], posv[r]) : acc[r];
    }
  }
}

template <class T, int NT>
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  embed_body<T, NT>(a);
}

// The key projection of the key score: the same fixed-order product with
// x = LayerNorm rows, K = D, W = W_K of layer 0, no position term.
template <class T, int NT>
__global__ __launch_bounds__(256) void keyproj_kernel(EmbedArgs a) {
  embed_body<T, NT>(a);
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
  // unconditional loads (clamped index), all issued before any is used; the
  // values past D are never used
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int d = min(lane + 64 * j, D - 1);
    xv[j] = x[d];
    g[j] = a.ln_g[d];
    b[j] = a.ln_b[d];
  }
#pragma unroll
  for (int j = 0; j < kPer; ++j) xv[j] = Elem<T>::rnd(xv[j]);
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
  // unconditional loads (clamped index), all issued before any is used; the
  // values past D are never used
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int d = min(lane + 64 * j, a.D - 1);
    xv[j] = x[d];
    yv[j] = y[d];
  }
  float pd = 0.0f, pa = 0.0f, pb = 0.0f;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {  // d = lane + 64 j in increasing d; entries past D are skipped
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

// Tile counts of the shapes in use are compiled unrolled (patch 14 and 16 with
// 3 channels: P = 588, 768; D = 192, 1024, 1152); other lengths run the loop.
template <class T, template <class, int> class Launch>
hipError_t launch_nt(const EmbedArgs& a, dim3 grid, hipStream_t s) {
  switch ((a.P + 63) / 64) {
    case 3: return Launch<T, 3>::go(a, grid, s);
    case 10: return Launch<T, 10>::go(a, grid, s);
    case 12: return Launch<T, 12>::go(a, grid, s);
    case 16: return Launch<T, 16>::go(a, grid, s);
    case 18: return Launch<T, 18>::go(a, grid, s);
    default: return Launch<T, 0>::go(a, grid, s);
  }
}
template <class T, int NT>
struct EmbedLaunch {
  static hipError_t go(const EmbedArgs& a, dim3 g, hipStream_t s) { return launch_k(embed_kernel<T, NT>, g, dim3(256), 0, s, a); }
};
template <class T, int NT>
struct KeyLaunch {
  static hipError_t go(const EmbedArgs& a, dim3 g, hipStream_t s) { return launch_k(keyproj_kernel<T, NT>, g, dim3(256), 0, s, a); }
};

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  dim3 grid((a.N + 15) / 16, (a.D + 63) / 64, a.B);
  return a.dtype ? launch_nt<uint16_t, EmbedLaunch>(a, grid, s) : launch_nt<float, EmbedLaunch>(a, grid, s);
}

hipError_t launch_keyproj(const EmbedArgs& a, hipStream_t s) {
  dim3 grid((a.N + 15) / 16, (a.D + 63) / 64, a.B);
  return a.dtype ? launch_nt<uint16_t, KeyLaunch>(a, grid, s) : launch_nt<float, KeyLaunch>(a, grid, s);
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
