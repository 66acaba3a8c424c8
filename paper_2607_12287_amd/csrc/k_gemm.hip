// The four per-layer GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and
// the residual + MLP that follows the attention):
//   QKV : [Q K V] = S(S(LN1(X^l[U])) W_qkv + b); Q -> workspace, K and V rows
//         scattered into the cached K^l, V^l of each stream (eq. 5);
//   OPROJ: H = X^l[U] + (O W_o + b_o)            (fp32)
//   FC1 : G = S(GELU(S(LN2(H)) W_1 + b_1))
//   FC2 : X^{l+1}[U] = S(H + (G W_2 + b_2))      scattered into the cache.
//
// Only the rows of U (M rows over all streams) are computed.  With M small
// the time is set by memory latency and by the traffic through each CU's load
// path, not by HBM bandwidth, so:
//   * the loads whose addresses are known first (M, the row map and the
//     per-row LayerNorm partials of the first 64 rows) go out before anything
//     else; the A rows and residuals follow; the bulk weight stream last;
//   * weights come straight into MFMA operand registers: the packed layout
//     makes one 32-deep chunk of a 16-column block one vector load per lane;
//   * the number of 16-row tiles of a block is a template parameter chosen at
//     run time, so a lane issues exactly the loads it needs, unconditionally
//     (addresses clamped), and the wait before an MFMA covers only its own
//     operands;
//   * wide outputs give a workgroup two column blocks, so each A row is read
//     once for 32 columns;
//   * the LayerNorm of the A operand is applied in registers from per-row
//     (sum, sum of squares) partials that the producing kernel wrote in its
//     epilogue.
// The waves' partial tiles are summed in a fixed order through LDS; nothing is
// summed with atomics, so results are deterministic.
#include "common.hpp"

namespace incvit {

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanhf(u));
}

// A-operand element type: H is fp32, everything else is the storage dtype.
template <class T, int EPI> struct AType { using type = T; };
template <class T> struct AType<T, EPI_FC1> { using type = float; };

// Normalise 8 A values (one lane's share of a 32-deep chunk) to the storage type.
__device__ __forceinline__ void ln8(V8<uint16_t>& out, const float* x, float mean, float rstd,
                                    const float* g, const float* b) {
  uint32_t q[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float y0 = (x[2 * e] - mean) * rstd * g[2 * e] + b[2 * e];
    const float y1 = (x[2 * e + 1] - mean) * rstd * g[2 * e + 1] + b[2 * e + 1];
    q[e] = (uint32_t)f2bf(y0) | ((uint32_t)f2bf(y1) << 16);
  }
  out.v = make_uint4(q[0], q[1], q[2], q[3]);
}
__device__ __forceinline__ void ln8(V8<float>& out, const float* x, float mean, float rstd,
                                    const float* g, const float* b) {
  float y[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = (x[e] - mean) * rstd * g[e] + b[e];
  out.a = make_float4(y[0], y[1], y[2], y[3]);
  out.b = make_float4(y[4], y[5], y[6], y[7]);
}

__device__ __forceinline__ void unpack8(float* x, const V8<uint16_t>& v) {
  const uint32_t q[4] = {v.v.x, v.v.y, v.v.z, v.v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(q[e] << 16);
    x[2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack8(float* x, const V8<float>& v) {
  x[0] = v.a.x; x[1] = v.a.y; x[2] = v.a.z; x[3] = v.a.w;
  x[4] = v.b.x; x[5] = v.b.y; x[6] = v.b.z; x[7] = v.b.w;
}

// Residual element type: the cached X row (storage type) for the output
// projection, H (fp32) for the MLP down projection.
template <class T, int EPI> struct ResType { using type = float; };
template <class T> struct ResType<T, EPI_OPROJ> { using type = T; };

struct GemmShared {
  RowInfo rows[kGemmRows];
  float mean[kGemmRows], rstd[kGemmRows];
  int m;
};

// One block of up to 64 rows (RT 16-row tiles) against this workgroup's NB
// column blocks.  part: this thread's share of the LayerNorm partial sums of
// row (tid / NW), already loaded.
template <class T, int EPI, int NW, int NB, int RT>
__device__ __forceinline__ void gemm_rows(const GemmArgs& a, GemmShared& sh, char* smem, int m0, int mrows,
                                          float2 part) {
  constexpr bool kLN = (EPI == EPI_QKV || EPI == EPI_FC1);
  using TA = typename AType<T, EPI>::type;
  constexpr int PF = (sizeof(TA) == 4 || RT >= 3) ? 2 : 4;  // chunks in flight per wave
  // w is read into a scalar register so every guard that depends on it is a
  // scalar branch: an MFMA must never sit under a lane mask (it would still
  // accumulate with the mask empty).
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, n = lane & 15;
  const int D = a.sh.D;
  const int cb0 = blockIdx.x * NB;
  const int nw = max(0, (a.kchunks - w + NW - 1) / NW);
  const int kclamp = a.kchunks - 1;
  auto chunk = [&](int i) { return min(w + NW * i, kclamp); };
  const float* s_g = reinterpret_cast<const float*>(smem + NW * 4 * NB * 64 * 16);
  const float* s_b = s_g + D;

  // ---- A rows (and residuals): latency-critical, issued first
  const TA* ap[RT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    const int rl = min(16 * r + n, mrows - 1);
    if constexpr (EPI == EPI_QKV) {
      const RowInfo ri = sh.rows[rl];
      ap[r] = x_row<T>(ri.cache, a.cl, a.sh, a.layer, ri.tok) + 8 * g;
    } else {
      ap[r] = static_cast<const TA*>(a.A) + (size_t)(m0 + rl) * a.lda + 8 * g;
    }
  }
  V8<TA> ab[PF][RT];
#pragma unroll
  for (int s = 0; s < PF; ++s)
#pragma unroll
    for (int r = 0; r < RT; ++r) ab[s][r].load(ap[r] + chunk(s) * 32);
  const int rt = w;  // the row tile this wave finishes (if rt < RT)
  // epilogue residuals of this lane's 4 rows, kept raw until the epilogue;
  // loaded by every wave (clamped) so no branch waits on them
  typename ResType<T, EPI>::type rres[NB][4];
  if constexpr (EPI == EPI_FC2 || EPI == EPI_OPROJ) {
    const int rtl = min(rt, RT - 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rl = min(16 * rtl + 4 * g + i, mrows - 1);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int col = (cb0 + b) * 16 + n;
        if constexpr (EPI == EPI_FC2) {
          rres[b][i] = a.hres[(size_t)(m0 + rl) * D + col];
        } else {
          const RowInfo ri = sh.rows[rl];
          rres[b][i] = gbl(x_row<T>(ri.cache, a.cl, a.sh, a.layer, ri.tok))[col];
        }
      }
    }
  }
  // ---- the weight stream
  const T* wbase[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    wbase[b] = static_cast<const T*>(a.W) + (size_t)(cb0 + b) * a.kchunks * kChunkElems + lane * 8;
  V8<T> wb[PF][NB];
#pragma unroll
  for (int s = 0; s < PF; ++s)
#pragma unroll
    for (int b = 0; b < NB; ++b) wb[s][b].load(wbase[b] + (size_t)chunk(s) * kChunkElems);

  // ---- LayerNorm statistics of the block's rows (fixed-order reduction)
  if constexpr (kLN) {
#pragma unroll
    for (int off = NW / 2; off >= 1; off >>= 1) {
      part.x += __shfl_xor(part.x, off, NW);
      part.y += __shfl_xor(part.y, off, NW);
    }
    const int srow = tid / NW;
    if (tid % NW == 0 && srow < mrows) {
      const float mean = part.x / (float)D;
      const float var = fmaxf(part.y / (float)D - mean * mean, 0.0f);
      sh.mean[srow] = mean;
      sh.rstd[srow] = 1.0f / sqrtf(var + a.sh.eps);
    }
    __syncthreads();
  }
  float rmean[RT], rrstd[RT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    const int rl = min(16 * r + n, mrows - 1);
    rmean[r] = kLN ? sh.mean[rl] : 0.0f;
    rrstd[r] = kLN ? sh.rstd[rl] : 0.0f;
  }

  // ---- MFMA over this wave's chunks
  f32x4_t acc[RT][NB];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  for (int i0 = 0; i0 < nw; i0 += PF) {
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      const int i = i0 + s;
      if (i < nw) {  // uniform; no memory operation inside
        const int kc = w + NW * i;
        float gg[8], bb[8];
        if constexpr (kLN) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            gg[e] = s_g[kc * 32 + 8 * g + e];
            bb[e] = s_b[kc * 32 + 8 * g + e];
          }
        }
#pragma unroll
        for (int r = 0; r < RT; ++r) {
          if constexpr (kLN) {
            float x[8];
            unpack8(x, ab[s][r]);
            V8<T> av;
            ln8(av, x, rmean[r], rrstd[r], gg, bb);
#pragma unroll
            for (int b = 0; b < NB; ++b) mma(acc[r][b], av, wb[s][b]);
          } else {
#pragma unroll
            for (int b = 0; b < NB; ++b) mma(acc[r][b], ab[s][r], wb[s][b]);
          }
        }
      }
      const int kn = chunk(i + PF);
#pragma unroll
      for (int r = 0; r < RT; ++r) ab[s][r].load(ap[r] + kn * 32);
#pragma unroll
      for (int b = 0; b < NB; ++b) wb[s][b].load(wbase[b] + (size_t)kn * kChunkElems);
    }
  }

  // ---- sum the waves' partial tiles in wave order; wave w finishes row tile w
  f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) red[((w * RT + r) * NB + b) * 64 + lane] = acc[r][b];
  __syncthreads();
  if (rt < RT) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int cb = cb0 + b;
      const int col = cb * 16 + n;
      f32x4_t val = red[((0 * RT + rt) * NB + b) * 64 + lane];
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) val += red[((ww * RT + rt) * NB + b) * 64 + lane];
      const float bias = a.bias[col];

      // ---- epilogue: stores
      float y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = 16 * rt + 4 * g + i;
        const float x = val[i] + bias;
        const RowInfo ri = sh.rows[min(rl, mrows - 1)];
        const bool ok = rl < mrows;
        y[i] = 0.0f;
        if constexpr (EPI == EPI_QKV) {
          const int which = col / D, c = col - which * D;
          const T o = Elem<T>::cv(x);
          if (ok) {
            if (which == 0) {
              static_cast<T*>(a.out)[(size_t)(m0 + rl) * a.ldo + c] = o;
            } else {
              const int hh = c / a.sh.dh, d = c - hh * a.sh.dh;
              char* base = ri.cache + (which == 1 ? a.cl.k : a.cl.v) + (size_t)a.layer * a.cl.kv_layer;
              const size_t e = which == 1 ? ((size_t)hh * a.sh.Npad + ri.tok) * a.sh.dh + d
                                          : ((size_t)hh * a.sh.dh + d) * a.sh.Npad + ri.tok;
              gbl(reinterpret_cast<T*>(base))[e] = o;
            }
          }
        } else if constexpr (EPI == EPI_OPROJ) {
          y[i] = Elem<T>::f(rres[b][i]) + x;
          if (ok) static_cast<float*>(a.out)[(size_t)(m0 + rl) * a.ldo + col] = y[i];
        } else if constexpr (EPI == EPI_FC1) {
          if (ok) static_cast<T*>(a.out)[(size_t)(m0 + rl) * a.ldo + col] = Elem<T>::cv(gelu_tanh(x));
        } else {
          const T o = Elem<T>::cv(rres[b][i] + x);
          y[i] = Elem<T>::f(o);
          if (ok) gbl(x_row<T>(ri.cache, a.cl, a.sh, a.layer + 1, ri.tok))[col] = o;
        }
      }
      if constexpr (EPI == EPI_OPROJ || EPI == EPI_FC2) {
        // per-row (sum, sum of squares) over this block's 16 columns: the
        // LayerNorm statistics of the next GEMM, combined there in block order
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float s1 = y[i], s2 = y[i] * y[i];
#pragma unroll
          for (int off = 8; off >= 1; off >>= 1) {
            s1 += __shfl_xor(s1, off, 16);
            s2 += __shfl_xor(s2, off, 16);
          }
          const int rl = 16 * rt + 4 * g + i;
          if (n == 0 && rl < mrows) a.stats_out[(size_t)(m0 + rl) * a.stat_stride + cb] = make_float2(s1, s2);
        }
      }
    }
  }
}

// LayerNorm partials of row (m0 + tid / NW): this thread sums the partials
// j = tid % NW, + NW, ... in order.
template <int NW>
__device__ __forceinline__ float2 load_partials(const GemmArgs& a, int m0, int rows_bound) {
  constexpr int kJ = (kMaxStat + NW - 1) / NW;
  const int srow = min((int)threadIdx.x / NW, rows_bound - 1), sq = threadIdx.x % NW;
  const float2* sp = a.stats_in + (size_t)(m0 + srow) * a.stat_stride;
  float2 pv[kJ];
#pragma unroll
  for (int jj = 0; jj < kJ; ++jj) pv[jj] = sp[min(sq + NW * jj, a.nstat - 1)];
  float2 part = make_float2(0.0f, 0.0f);
#pragma unroll
  for (int jj = 0; jj < kJ; ++jj) {
    if (sq + NW * jj < a.nstat) {
      part.x += pv[jj].x;
      part.y += pv[jj].y;
    }
  }
  return part;
}

template <class T, int EPI, int NW, int NB>
__global__ __launch_bounds__(NW * 64) void gemm_kernel(GemmArgs a) {
  constexpr bool kLN = (EPI == EPI_QKV || EPI == EPI_FC1);
  constexpr int NT = NW * 64;
  constexpr int kGB = (kMaxDim + NT - 1) / NT;
  extern __shared__ __align__(16) char smem[];
  __shared__ GemmShared sh;
  const int tid = threadIdx.x;
  const int D = a.sh.D;

  // ---- first: M, the row map and LayerNorm partials of the first 64 rows
  // (rows past M are read but never used), and the LayerNorm parameters
  if (tid == 0) sh.m = a.meta->m;
  if (tid < kGemmRows) sh.rows[tid] = a.rows[tid];
  float2 part = make_float2(0.0f, 0.0f);
  if constexpr (kLN) part = load_partials<NW>(a, 0, kGemmRows);
  float* s_g = reinterpret_cast<float*>(smem + NW * 4 * NB * 64 * 16);
  float* s_b = s_g + D;
  if constexpr (kLN) {
    float gv[kGB], bv[kGB];
#pragma unroll
    for (int j = 0; j < kGB; ++j) {
      const int k = min(tid + NT * j, D - 1);
      gv[j] = a.ln_g[k];
      bv[j] = a.ln_b[k];
    }
#pragma unroll
    for (int j = 0; j < kGB; ++j) {
      const int k = tid + NT * j;
      if (k < D) {
        s_g[k] = gv[j];
        s_b[k] = bv[j];
      }
    }
  }
  __syncthreads();
  const int M = sh.m;
  for (int m0 = 0; m0 < M; m0 += kGemmRows) {
    const int mrows = min(kGemmRows, M - m0);
    if (m0 > 0) {  // later blocks: row map and partials of this block
      __syncthreads();
      if (tid < kGemmRows) sh.rows[tid] = a.rows[m0 + min(tid, mrows - 1)];
      if constexpr (kLN) part = load_partials<NW>(a, m0, mrows);
      __syncthreads();
    }
    switch ((mrows + 15) >> 4) {
      case 1: gemm_rows<T, EPI, NW, NB, 1>(a, sh, smem, m0, mrows, part); break;
      case 2: gemm_rows<T, EPI, NW, NB, 2>(a, sh, smem, m0, mrows, part); break;
      case 3: gemm_rows<T, EPI, NW, NB, 3>(a, sh, smem, m0, mrows, part); break;
      default: gemm_rows<T, EPI, NW, NB, 4>(a, sh, smem, m0, mrows, part); break;
    }
  }
}

template <int NW, int NB>
static size_t gemm_lds(const GemmArgs& a) {
  return (size_t)NW * 4 * NB * 64 * 16 + (size_t)2 * a.sh.D * sizeof(float);
}

// Allow each instantiation the largest dynamic LDS any shape needs, once.
template <class T, int EPI, int NW, int NB>
static hipError_t allow_lds() {
  static hipError_t done = hipErrorNotReady;
  if (done != hipSuccess) {
    const int most = NW * 4 * NB * 64 * 16 + 2 * kMaxDim * (int)sizeof(float);
    done = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, EPI, NW, NB>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, most);
  }
  return done;
}

template <int EPI, int NW, int NB>
static hipError_t launch_cfg(const GemmArgs& a, hipStream_t s) {
  const dim3 grid(a.Nout / 16 / NB);
  const size_t lds = gemm_lds<NW, NB>(a);
  hipError_t e;
  if (a.sh.dtype) {
    if ((e = allow_lds<uint16_t, EPI, NW, NB>()) != hipSuccess) return e;
    (void)launch_k((gemm_kernel<uint16_t, EPI, NW, NB>), grid, dim3(NW * 64), lds, s, a);
  } else {
    if ((e = allow_lds<float, EPI, NW, NB>()) != hipSuccess) return e;
    (void)launch_k((gemm_kernel<float, EPI, NW, NB>), grid, dim3(NW * 64), lds, s, a);
  }
  return hipGetLastError();
}

// cols: column blocks per workgroup (1 or 2; 2 needs an even block count).
template <int EPI>
static hipError_t launch_epi(int waves, int cols, const GemmArgs& a, hipStream_t s) {
  const bool two = cols == 2 && (a.Nout / 16) % 2 == 0;
  if (waves >= 8) return two ? launch_cfg<EPI, 8, 2>(a, s) : launch_cfg<EPI, 8, 1>(a, s);
  return two ? launch_cfg<EPI, 4, 2>(a, s) : launch_cfg<EPI, 4, 1>(a, s);
}

hipError_t launch_gemm(int epi, int waves, int cols, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(waves, cols, a, s);
    case EPI_OPROJ: return launch_epi<EPI_OPROJ>(waves, cols, a, s);
    case EPI_FC1: return launch_epi<EPI_FC1>(waves, cols, a, s);
    default: return launch_epi<EPI_FC2>(waves, cols, a, s);
  }
}

}  // namespace incvit
