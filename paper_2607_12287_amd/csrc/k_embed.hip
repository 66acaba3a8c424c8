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

// Workgroup: 4*TM tokens x 64*TN columns; wave w computes tokens
// TM*w..TM*w+TM-1 of the tile and lane l one column (TN = 1: column l) or two
// adjacent ones (TN = 2, bf16 weights: columns 2l, 2l+1, kept in LDS as one
// packed pair), so a k step reads TM + 1 values from LDS for TM*TN fma.  k is
// staged through LDS in tiles of 64, double buffered, with one barrier per
// tile.  A tile's global loads go out two tiles of compute ahead into one of
// three register slots (the loop body is unrolled over the slots, so no
// register copy waits on a load in flight); every load is unconditional
// (clamped addresses; values past P are loaded but never used because the k
// loop stops at P).  The patch tiles sit first in LDS and every buffer stays
// below 64 KB, so each LDS read is a base register plus an immediate offset.
template <class T, int NT, int TM, int TN>
__device__ __forceinline__ void embed_body(const EmbedArgs& a) {
  static_assert(TN == 1 || (TN == 2 && sizeof(T) == 2), "two columns per lane need bf16 weights");
  constexpr int TT = 4 * TM, TC = 64 * TN;  // tile tokens, tile columns
  constexpr int WV = 16 / sizeof(T);  // weights per 16-byte load
  constexpr int WL = 64 * TC / (256 * WV);  // weight loads per thread per tile
  constexpr int XL = 64 * TT / 256;  // patch loads per thread per tile (= TM)
  constexpr int XB = 64 * TT;  // floats per patch buffer
  constexpr int WB = 64 * 64;  // 32-bit words per weight buffer (one per lane and k)
  __shared__ __align__(16) float smem[2 * XB + 2 * WB];
  float* const sx = smem;                                            // [buffer][k][token]
  float* const swf = smem + 2 * XB;                                  // TN = 1: [buffer][k][column]
  uint32_t* const swp = reinterpret_cast<uint32_t*>(smem + 2 * XB);  // TN = 2: [buffer][k][lane] pairs
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
  const int tok0 = tg * TT, c0 = cb * TC;
  const int N = a.N, P = a.P, D = a.D;

  if (tg == 0 && cb == 0) {
    for (int k = tid; k < a.nzero && v == 0; k += 256) a.zero[k] = 0;
    if (a.ident_idx) {
      for (int k = tid; k < N; k += 256) a.ident_idx[v * N + k] = k;
      if (tid == 0) a.ident_count[v] = N;
    }
  }

  // Operands through buffer loads: every lane offset below is fixed for the
  // whole kernel and the tile's k position is a wave-uniform offset, so a
  // fetch needs no address registers.  Reads past the buffer return zero; reads
  // past a row's end (k >= P) are never used because the k loop stops at P.
  const Rsrc rx = make_rsrc(a.patches + (size_t)v * N * P, (uint32_t)((size_t)N * P * 4));
  const Rsrc rw = make_rsrc(a.w_pe, (uint32_t)((size_t)P * D * sizeof(T)));
  uint32_t xoff[XL], woff[WL];
  // patch element e of a tile: token e / 64, k e % 64 (a wave reads 64
  // consecutive k of one token's row)
#pragma unroll
  for (int j = 0; j < XL; ++j) {
    const int e = tid + 256 * j;
    xoff[j] = (uint32_t)((min(tok0 + (e >> 6), N - 1) * P + (e & 63)) * 4);
  }
  // weight run e of a tile: row k = e / (TC / WV), WV columns from (e % (TC / WV)) * WV
#pragma unroll
  for (int j = 0; j < WL; ++j) {
    const int e = tid + 256 * j;
    woff[j] = (uint32_t)(((e / (TC / WV)) * D + min(c0 + (e % (TC / WV)) * WV, D - WV)) * sizeof(T));
  }
  struct Tile {
    float x[XL];
    V8<T> wv[WL];
  };
  auto fetch = [&](Tile& t, int kt) {
#pragma unroll
    for (int j = 0; j < XL; ++j)
      t.x[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rx, xoff[j], (uint32_t)kt * 4, 0));
#pragma unroll
    for (int j = 0; j < WL; ++j) bload16(t.wv[j], rw, woff[j], (uint32_t)(kt * D * sizeof(T)));
  };
  auto stage = [&](const Tile& t, int b) {
#pragma unroll
    for (int j = 0; j < XL; ++j) {
      const int e = tid + 256 * j;
      sx[b * XB + (e & 63) * TT + (e >> 6)] = t.x[j];
    }
#pragma unroll
    for (int j = 0; j < WL; ++j) {
      const int e = tid + 256 * j;
      const int k = e / (TC / WV), c = (e % (TC / WV)) * WV;
      if constexpr (TN == 2) {
        // 8 bf16 columns = 4 packed pairs, stored as they came
        *reinterpret_cast<uint4*>(&swp[b * WB + k * 64 + c / 2]) = __builtin_bit_cast(uint4, t.wv[j]);
      } else {
        float f[WV];
        unpack16(f, t.wv[j]);
#pragma unroll
        for (int q = 0; q < WV; ++q) swf[b * WB + k * 64 + c + q] = f[q];
      }
    }
  };

  // the lane's columns: TN = 1: c0 + lane; TN = 2: c0 + 2 lane and the next
  const int dl = c0 + (TN == 2 ? 2 * lane : lane);
  float acc[TM][TN], posv[TM][TN];
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    const int d = min(dl + n, D - 1);
    const float bias = a.b_pe[d];
#pragma unroll
    for (int r = 0; r < TM; ++r) {
      acc[r][n] = bias;
      const int tok = min(tok0 + TM * w + r, N - 1);
      posv[r][n] = a.pos ? a.pos[(size_t)tok * D + d] : 0.0f;
    }
  }
  // one k step: TM patch values (the same for the whole wave) and TN weights
  // (TN = 2: one packed bf16 pair), read from LDS, then the TM * TN fma
  struct Ops {
    float x[TM];
    uint32_t w;
  };
  auto read_ops = [&](Ops& o, int b, int kk) {
    if constexpr (TN == 2) o.w = swp[b * WB + kk * 64 + lane];
    else o.w = __float_as_uint(swf[b * WB + kk * 64 + lane]);
    if constexpr (TM == 4) {
      const float4 x4 = *reinterpret_cast<const float4*>(&sx[b * XB + kk * TT + 4 * w]);
      o.x[0] = x4.x; o.x[1] = x4.y; o.x[2] = x4.z; o.x[3] = x4.w;
    } else {
#pragma unroll
      for (int r = 0; r < TM; ++r) o.x[r] = sx[b * XB + kk * TT + TM * w + r];
    }
  };
  auto fma_ops = [&](const Ops& o) {
    float wv[TN];
    if constexpr (TN == 2) {
      wv[0] = __uint_as_float(o.w << 16);
      wv[1] = __uint_as_float(o.w & 0xffff0000u);
    } else {
      wv[0] = __uint_as_float(o.w);
    }
#pragma unroll
    for (int r = 0; r < TM; ++r)
#pragma unroll
      for (int n = 0; n < TN; ++n) acc[r][n] = __fmaf_rn(o.x[r], wv[n], acc[r][n]);
  };
  auto kstep = [&](int b, int kk) {
    Ops o;
    read_ops(o, b, kk);
    fma_ops(o);
  };
  // A full tile of 64 k steps with each step's LDS reads issued PD steps
  // ahead of its fma: with one wave per SIMD nothing else hides the LDS
  // latency (the fma order is unchanged).
  constexpr int PD = 4;
  auto full_tile = [&](int b) {
    Ops o[PD];
#pragma unroll
    for (int p = 0; p < PD; ++p) read_ops(o[p], b, p);
#pragma unroll
    for (int kk = 0; kk < 64; ++kk) {
      const Ops cur = o[kk % PD];
      if (kk + PD < 64) read_ops(o[kk % PD], b, kk + PD);
      fma_ops(cur);
    }
  };
  auto compute = [&](int b, int kmax) {
    if (kmax == 64) {  // uniform
      full_tile(b);
      return;
    }
#pragma unroll 8
    for (int kk = 0; kk < kmax; ++kk) kstep(b, kk);
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
        full_tile(it & 1);
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
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    const int d = dl + n;
    if (d < D) {
#pragma unroll
      for (int r = 0; r < TM; ++r) {
        const int tok = tok0 + TM * w + r;
        if (tok < N) a.t0[((size_t)v * N + tok) * D + d] = a.pos ? __fadd_rn(acc[r][n], posv[r][n]) : acc[r][n];
      }
    }
  }
}

template <class T, int NT, int TM, int TN>
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  embed_body<T, NT, TM, TN>(a);
}

// The key projection of the key score: the same fixed-order product with
// x = LayerNorm rows, K = D, W = W_K of layer 0, no position term.
template <class T, int NT, int TM, int TN>
__global__ __launch_bounds__(256) void keyproj_kernel(EmbedArgs a) {
  embed_body<T, NT, TM, TN>(a);
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
template <class T, int TM, int TN, template <class, int, int, int> class Launch>
hipError_t launch_nt(const EmbedArgs& a, dim3 grid, hipStream_t s) {
  switch ((a.P + 63) / 64) {
    case 3: return Launch<T, 3, TM, TN>::go(a, grid, s);
    case 10: return Launch<T, 10, TM, TN>::go(a, grid, s);
    case 12: return Launch<T, 12, TM, TN>::go(a, grid, s);
    case 16: return Launch<T, 16, TM, TN>::go(a, grid, s);
    case 18: return Launch<T, 18, TM, TN>::go(a, grid, s);
    default: return Launch<T, 0, TM, TN>::go(a, grid, s);
  }
}
template <class T, int NT, int TM, int TN>
struct EmbedLaunch {
  static hipError_t go(const EmbedArgs& a, dim3 g, hipStream_t s) {
    return launch_k(embed_kernel<T, NT, TM, TN>, g, dim3(256), 0, s, a);
  }
};
template <class T, int NT, int TM, int TN>
struct KeyLaunch {
  static hipError_t go(const EmbedArgs& a, dim3 g, hipStream_t s) {
    return launch_k(keyproj_kernel<T, NT, TM, TN>, g, dim3(256), 0, s, a);
  }
};

// Register tile of the fixed-order product, TM tokens x TN columns per lane,
// chosen per shape.  Per k step a CU's LDS returns 4 waves x 64 lanes x
// (TM + 1) words at 128 bytes per clock, 8 (TM + 1) clocks, while each SIMD
// spends 4 clocks per wave64 instruction on TM TN fma (and two more to unpack a
// bf16 pair); the workgroups run in ceil(count / 256) rounds of one per CU.
// The tile with the fewest estimated clocks wins (the first listed on a tie).
struct Tiling {
  int tm, tn;
};
constexpr Tiling kTilings[] = {{4, 1}, {3, 2}, {4, 2}};

// fp32 weights take one column per lane only
inline int pick_tiling(const EmbedArgs& a) {
  int best = 0;
  long best_cost = -1;
  for (int t = 0; t < (a.dtype ? (int)(sizeof(kTilings) / sizeof(kTilings[0])) : 1); ++t) {
    const int tm = kTilings[t].tm, tn = kTilings[t].tn;
    const long wgs = (long)((a.N + 4 * tm - 1) / (4 * tm)) * ((a.D + 64 * tn - 1) / (64 * tn)) * a.B;
    const long step = std::max(8 * (tm + 1), 4 * (tm * tn + (tn == 2 ? 2 : 0)));
    const long cost = (wgs + 255) / 256 * step;
    if (best_cost < 0 || cost < best_cost) {
      best = t;
      best_cost = cost;
    }
  }
  return best;
}

template <class T, template <class, int, int, int> class Launch>
hipError_t launch_tiled(const EmbedArgs& a, hipStream_t s) {
  const int t = pick_tiling(a);
  const int tm = kTilings[t].tm, tn = kTilings[t].tn;
  const dim3 grid((a.N + 4 * tm - 1) / (4 * tm), (a.D + 64 * tn - 1) / (64 * tn), a.B);
  // two columns per lane: the patch lengths in use (10 and 12 tiles) run
  // unrolled, longer rows the tile loop (unrolled over 16 or more tiles the
  // compiler's hoisting exceeds the register file and spills)
  if constexpr (sizeof(T) == 2) {
    const int nt = (a.P + 63) / 64;
    if (t == 1) {
      if (nt == 10) return Launch<T, 10, 3, 2>::go(a, grid, s);
      if (nt == 12) return Launch<T, 12, 3, 2>::go(a, grid, s);
      return Launch<T, 0, 3, 2>::go(a, grid, s);
    }
    if (t == 2) {
      if (nt == 10) return Launch<T, 10, 4, 2>::go(a, grid, s);
      if (nt == 12) return Launch<T, 12, 4, 2>::go(a, grid, s);
      return Launch<T, 0, 4, 2>::go(a, grid, s);
    }
  }
  return launch_nt<T, 4, 1, Launch>(a, grid, s);
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  return a.dtype ? launch_tiled<uint16_t, EmbedLaunch>(a, s) : launch_tiled<float, EmbedLaunch>(a, s);
}

hipError_t launch_keyproj(const EmbedArgs& a, hipStream_t s) {
  return a.dtype ? launch_tiled<uint16_t, KeyLaunch>(a, s) : launch_tiled<float, KeyLaunch>(a, s);
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
