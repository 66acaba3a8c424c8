// The four per-layer GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and
// the residual + MLP that follows the attention):
//   QKV : [Q K V] = S(S(LN1(X^l[U])) W_qkv + b); Q -> workspace, K and V rows
//         scattered into the cached K^l, V^l of each stream (eq. 5);
//   OPROJ: H = X^l[U] + (O W_o + b_o)            (fp32)
//   FC1 : G = S(GELU(S(LN2(H)) W_1 + b_1))
//   FC2 : X^{l+1}[U] = S(H + (G W_2 + b_2))      scattered into the cache.
//
// Only the rows of U (M rows over all streams) are computed.  With M small
// the time is set by memory latency, not bandwidth, so the kernel is laid out
// as a fixed number of dependent load batches:
//   1. the first weight chunks (straight into MFMA operand registers: the
//      packed layout makes a 32-deep chunk one vector load per lane), M, and
//      the LayerNorm parameters;
//   2. the row map, the per-row LayerNorm partials (sum, sum of squares) that
//      the producing kernel wrote in its epilogue, the compact A rows, and the
//      compact residual of FC2;
//   3. the rows gathered from the caches (QKV's A, OPROJ's residual);
// then the MFMA loop with a prefetch ring, a fixed-order reduction of the
// waves' partial tiles through LDS, and the stores.  Nothing is summed with
// atomics, so results are deterministic.
//
// Grid: one workgroup per 16-column block of the output; it loops over the M
// rows in blocks of 64; its NW waves take every NW-th 32-deep K chunk.
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

template <class T, int EPI, int NW>
__global__ __launch_bounds__(NW * 64) void gemm_kernel(GemmArgs a) {
  constexpr bool kLN = (EPI == EPI_QKV || EPI == EPI_FC1);
  using TA = typename AType<T, EPI>::type;
  constexpr int PF = (sizeof(TA) == 4 || NW >= 16) ? 2 : 4;  // chunks in flight per wave
  constexpr int RT = 4;                                       // 16-row tiles per row block
  constexpr int NT = NW * 64;
  constexpr int kGB = (kMaxDim + NT - 1) / NT;                // LN parameters per thread
  constexpr int kJ = (kMaxStat + NW - 1) / NW;                // LN partials per thread
  extern __shared__ __align__(16) char smem[];
  __shared__ RowInfo s_rows[kGemmRows];
  __shared__ float s_mean[kGemmRows], s_rstd[kGemmRows];
  __shared__ int s_m;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int cb = blockIdx.x;
  const int D = a.sh.D;
  const int col = cb * 16 + n;
  const int nw = max(0, (a.kchunks - w + NW - 1) / NW);
  const T* wbase = static_cast<const T*>(a.W) + (size_t)cb * a.kchunks * kChunkElems + lane * 8;
  float* s_g = reinterpret_cast<float*>(smem + NW * RT * 64 * 16);
  float* s_b = s_g + D;

  // ---- batch 1: weights, M, LayerNorm parameters
  // Every load below is issued unconditionally (addresses clamped into range),
  // so each loop iteration issues a fixed number of loads and the wait before
  // an MFMA covers only the loads it needs, not the prefetches behind them.
  const int kclamp = a.kchunks - 1;
  auto chunk = [&](int i) { return min(w + NW * i, kclamp); };
  V8<T> wb[PF];
#pragma unroll
  for (int s = 0; s < PF; ++s) wb[s].load(wbase + (size_t)chunk(s) * kChunkElems);
  if (tid == 0) s_m = a.meta->m;
  if constexpr (kLN) {
    float gv[kGB], bv[kGB];
#pragma unroll
    for (int j = 0; j < kGB; ++j) {
      const int k = tid + NT * j;
      gv[j] = k < D ? a.ln_g[k] : 0.0f;
      bv[j] = k < D ? a.ln_b[k] : 0.0f;
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
  const float bias = a.bias[col];
  __syncthreads();
  const int M = s_m;

  V8<TA> ab[PF][RT];
  const TA* ap[RT];
  for (int m0 = 0; m0 < M; m0 += kGemmRows) {
    const int mrows = min(kGemmRows, M - m0);
    const int nrt = (mrows + 15) >> 4;
    const int rt = w;  // the row tile this wave finishes
    // ---- batch 2: row map, LayerNorm partials, compact rows
    if (tid < kGemmRows) s_rows[tid] = a.rows[m0 + min(tid, mrows - 1)];
    if (m0 > 0) {
#pragma unroll
      for (int s = 0; s < PF; ++s) wb[s].load(wbase + (size_t)chunk(s) * kChunkElems);
    }
    float2 part = make_float2(0.0f, 0.0f);
    const int srow = tid / NW, sq = tid % NW;  // NW threads (adjacent lanes) per row
    if constexpr (kLN) {
      float2 pv[kJ];
      const float2* sp = a.stats_in + (size_t)(m0 + min(srow, mrows - 1)) * a.stat_stride;
#pragma unroll
      for (int jj = 0; jj < kJ; ++jj) pv[jj] = sp[min(sq + NW * jj, a.nstat - 1)];
#pragma unroll
      for (int jj = 0; jj < kJ; ++jj) {
        if (sq + NW * jj < a.nstat) {
          part.x += pv[jj].x;
          part.y += pv[jj].y;
        }
      }
    }
    if constexpr (EPI != EPI_QKV) {
#pragma unroll
      for (int r = 0; r < RT; ++r)
        ap[r] = static_cast<const TA*>(a.A) + (size_t)(m0 + min(16 * r + n, mrows - 1)) * a.lda + 8 * g;
#pragma unroll
      for (int s = 0; s < PF; ++s)
#pragma unroll
        for (int r = 0; r < RT; ++r) ab[s][r].load(ap[r] + chunk(s) * 32);
    }
    float res[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // epilogue residual of this lane's 4 rows
    if constexpr (EPI == EPI_FC2) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        res[i] = a.hres[(size_t)(m0 + min(16 * min(rt, RT - 1) + 4 * g + i, mrows - 1)) * D + col];
    }
    __syncthreads();  // s_rows
    // ---- batch 3: rows gathered from the caches
    if constexpr (EPI == EPI_QKV) {
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        const RowInfo ri = s_rows[min(16 * r + n, mrows - 1)];
        ap[r] = x_row<T>(ri.cache, a.cl, a.sh, a.layer, ri.tok) + 8 * g;
      }
#pragma unroll
      for (int s = 0; s < PF; ++s)
#pragma unroll
        for (int r = 0; r < RT; ++r) ab[s][r].load(ap[r] + chunk(s) * 32);
    }
    if constexpr (EPI == EPI_OPROJ) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const RowInfo ri = s_rows[min(16 * min(rt, RT - 1) + 4 * g + i, mrows - 1)];
        res[i] = Elem<T>::f(gbl(x_row<T>(ri.cache, a.cl, a.sh, a.layer, ri.tok))[col]);
      }
    }
    // ---- LayerNorm statistics of the block's rows (fixed-order reduction)
    if constexpr (kLN) {
#pragma unroll
      for (int off = NW / 2; off >= 1; off >>= 1) {
        part.x += __shfl_xor(part.x, off, NW);
        part.y += __shfl_xor(part.y, off, NW);
      }
      if (sq == 0 && srow < mrows) {
        const float mean = part.x / (float)D;
        const float var = fmaxf(part.y / (float)D - mean * mean, 0.0f);
        s_mean[srow] = mean;
        s_rstd[srow] = 1.0f / sqrtf(var + a.sh.eps);
      }
      __syncthreads();
    }
    float rmean[RT], rrstd[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const int rl = min(16 * r + n, mrows - 1);
      rmean[r] = kLN ? s_mean[rl] : 0.0f;
      rrstd[r] = kLN ? s_rstd[rl] : 0.0f;
    }

    // ---- MFMA over this wave's chunks
    f32x4_t acc[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) acc[r] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
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
            if (r < nrt) {
              if constexpr (kLN) {
                float x[8];
                unpack8(x, ab[s][r]);
                V8<T> av;
                ln8(av, x, rmean[r], rrstd[r], gg, bb);
                mma(acc[r], av, wb[s]);
              } else {
                mma(acc[r], ab[s][r], wb[s]);
              }
            }
          }
        }
        const int kn = chunk(i + PF);
        wb[s].load(wbase + (size_t)kn * kChunkElems);
#pragma unroll
        for (int r = 0; r < RT; ++r) ab[s][r].load(ap[r] + kn * 32);
      }
    }

    // ---- sum the waves' partial tiles in wave order; wave w finishes row tile w
    f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);
#pragma unroll
    for (int r = 0; r < RT; ++r)
      if (r < nrt) red[(w * RT + r) * 64 + lane] = acc[r];
    __syncthreads();
    if (rt < nrt) {
      f32x4_t val = red[rt * 64 + lane];
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) val += red[(ww * RT + rt) * 64 + lane];

      // ---- epilogue: stores only
      float y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = 16 * rt + 4 * g + i;
        const float x = val[i] + bias;
        const RowInfo ri = s_rows[min(rl, mrows - 1)];
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
          y[i] = res[i] + x;
          if (ok) static_cast<float*>(a.out)[(size_t)(m0 + rl) * a.ldo + col] = y[i];
        } else if constexpr (EPI == EPI_FC1) {
          if (ok) static_cast<T*>(a.out)[(size_t)(m0 + rl) * a.ldo + col] = Elem<T>::cv(gelu_tanh(x));
        } else {
          const T o = Elem<T>::cv(res[i] + x);
          y[i] = Elem<T>::ld(&o, 0);
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
    __syncthreads();  // shared state reused by the next row block
  }
}

template <int NW>
static size_t gemm_lds(const GemmArgs& a) {
  return (size_t)NW * 4 * 64 * 16 + (size_t)2 * a.sh.D * sizeof(float);
}

// Allow each instantiation the largest dynamic LDS any shape needs, once.
template <class T, int EPI, int NW>
static hipError_t allow_lds() {
  static hipError_t done = hipErrorNotReady;
  if (done != hipSuccess) {
    const int most = NW * 4 * 64 * 16 + 2 * kMaxDim * (int)sizeof(float);
    done = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, EPI, NW>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, most);
  }
  return done;
}

template <int EPI, int NW>
static hipError_t launch_nw(const GemmArgs& a, hipStream_t s) {
  const dim3 grid(a.Nout / 16);
  const size_t lds = gemm_lds<NW>(a);
  hipError_t e;
  if (a.sh.dtype) {
    if ((e = allow_lds<uint16_t, EPI, NW>()) != hipSuccess) return e;
    hipLaunchKernelGGL((gemm_kernel<uint16_t, EPI, NW>), grid, dim3(NW * 64), lds, s, a);
  } else {
    if ((e = allow_lds<float, EPI, NW>()) != hipSuccess) return e;
    hipLaunchKernelGGL((gemm_kernel<float, EPI, NW>), grid, dim3(NW * 64), lds, s, a);
  }
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_epi(int waves, const GemmArgs& a, hipStream_t s) {
  if (waves >= 16) return launch_nw<EPI, 16>(a, s);
  if (waves >= 8) return launch_nw<EPI, 8>(a, s);
  return launch_nw<EPI, 4>(a, s);
}

hipError_t launch_gemm(int epi, int waves, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(waves, a, s);
    case EPI_OPROJ: return launch_epi<EPI_OPROJ>(waves, a, s);
    case EPI_FC1: return launch_epi<EPI_FC1>(waves, a, s);
    default: return launch_epi<EPI_FC2>(waves, a, s);
  }
}

}  // namespace incvit
