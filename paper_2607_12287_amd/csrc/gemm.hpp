// The four per-layer GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and
// the residual + MLP that follows the attention):
//   QKV  : [Q K V] = S(S(LN1(Z_l)) W_qkv + b); Q -> workspace, K and V rows
//          scattered into the cached K^l, V^l of each stream (eq. 5);
//   OPROJ: H = Z_l + (O W_o + b_o)                (fp32)
//   FC1  : G = S(GELU(S(LN2(H)) W_1 + b_1))
//   FC2  : Z_{l+1} = S(H + (G W_2 + b_2)), written compact and scattered into
//          X^{l+1} of each stream's cache.
// Z_l, O, H and G are compact [row][column] workspace buffers over the M
// refreshed rows of the call (rows padded to a multiple of 64).
//
// With M a few dozen rows these are weight-streaming problems whose time is set
// by memory latency, so a workgroup issues every load it will need for its
// first 32 rows at once, before it knows M: the A fragments of rows 0..31 (the
// padded workspace makes that in bounds), all of its wave's weight chunks, and
// the epilogue operands.  Weights go straight into MFMA operand registers (the
// packed layout makes one 32-deep chunk of a 16-column block one 16-byte load
// per lane) and stay there for later row blocks.  LayerNorm statistics are
// computed in two passes from the A fragments already in registers (each
// workgroup sees whole rows, because it reduces over all of K).
//
// Workgroup: 8 waves, NB 16-column blocks; wave w owns a contiguous run of CPW
// chunks of K (rounds of 8*CPW chunks when K is longer).  The waves' partial
// tiles are summed in wave order through LDS, and the epilogue is spread over
// all waves.  No atomics anywhere: results are bit-deterministic.
#pragma once
#include "common.hpp"

namespace incvit {

constexpr int kGemmWaves = 8;
constexpr int kGemmRB = 32;  // rows per block: two 16-row MFMA tiles

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanhf(u));
}

// A-operand element type: H is fp32, everything else is the storage dtype.
template <class T, int EPI> struct AType { using type = T; };
template <class T> struct AType<T, EPI_FC1> { using type = float; };
// Residual element type: Z_l (storage type) for the output projection, H
// (fp32) for the MLP down projection.
template <class T, int EPI> struct ResType { using type = float; };
template <class T> struct ResType<T, EPI_OPROJ> { using type = T; };

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

// LayerNorm of 8 A values (one lane's share of a chunk), rounded to the
// storage type of the MFMA operand.
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

// Sum over the four lanes of a row (n, n+16, n+32, n+48), fixed order.
__device__ __forceinline__ float row_sum4(float s) {
  s += __shfl_xor(s, 16, 64);
  s += __shfl_xor(s, 32, 64);
  return s;
}

template <int NB>
__host__ __device__ constexpr int gemm_red_bytes() {
  return kGemmWaves * 2 * NB * 64 * 16;
}

template <class T, int EPI, int NB, int CPW>
__global__ __launch_bounds__(kGemmWaves * 64) void gemm_kernel(GemmArgs a) {
  constexpr bool kLN = (EPI == EPI_QKV || EPI == EPI_FC1);
  constexpr int NW = kGemmWaves;
  using TA = typename AType<T, EPI>::type;
  using TR = typename ResType<T, EPI>::type;
  extern __shared__ __align__(16) char smem[];
  f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);                       // [NW][2][NB][64]
  float* s_g = reinterpret_cast<float*>(smem + gemm_red_bytes<NB>());    // [D]
  float* s_b = s_g + a.sh.D;                                              // [D]
  float* s_st = s_b + a.sh.D;                                             // [2][NW][32]

  const int tid = threadIdx.x, lane = tid & 63;
  // w lives in a scalar register, so every guard that depends on it is a
  // scalar branch: an MFMA must never run under a partial or empty lane mask
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, n = lane & 15;
  const int D = a.sh.D;
  const int M = a.meta->m;
  const int cb0 = blockIdx.x * NB;
  // this workgroup's share of K: chunks [kb, kb + kn) (all of K unless split)
  const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
  const int kb = blockIdx.y * kper, kn = min(kper, a.kchunks - kb);
  const int kc_last = kn - 1;
  const int rounds = (kn + NW * CPW - 1) / (NW * CPW);
  const TA* A = static_cast<const TA*>(a.A);
  const T* W = static_cast<const T*>(a.W);

  // ---- LayerNorm parameters (small; issued first so the LDS copy does not
  // wait for anything else)
  float4 gq = make_float4(0, 0, 0, 0), bq = gq;
  if constexpr (kLN) {
    const int q = min(tid, D / 4 - 1);
    gq = reinterpret_cast<const float4*>(a.ln_g)[q];
    bq = reinterpret_cast<const float4*>(a.ln_b)[q];
  }

  auto kc_of = [&](int round, int c) { return kb + min((round * NW + w) * CPW + c, kc_last); };
  V8<TA> ab[CPW][2];
  V8<T> wb[CPW][NB];
  auto load_a = [&](int m0, int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int r = 0; r < 2; ++r)
        ab[c][r].load(A + (size_t)(m0 + 16 * r + n) * a.lda + kc_of(round, c) * 32 + 8 * g);
  };
  auto load_w = [&](int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int b = 0; b < NB; ++b)
        wb[c][b].load(W + ((size_t)(cb0 + b) * a.kchunks + kc_of(round, c)) * kChunkElems + lane * 8);
  };
  // epilogue item of this wave: row tile w/4, row 4g + (w%4) of the tile
  const int re = w >> 2, ie = w & 3;
  RowInfo rinfo = RowInfo{nullptr, 0, 0};
  TR resv[NB];
  float biasv[NB];
  auto load_epi = [&](int m0) {
    const int row = m0 + 16 * re + 4 * g + ie;
    if constexpr (EPI == EPI_QKV || EPI == EPI_FC2) rinfo = a.rows[row];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if constexpr (EPI == EPI_OPROJ || EPI == EPI_FC2)
        resv[b] = static_cast<const TR*>(a.res)[(size_t)row * D + (cb0 + b) * 16 + n];
      else
        resv[b] = TR(0);
    }
  };

  load_a(0, 0);
  load_w(0);
#pragma unroll
  for (int b = 0; b < NB; ++b) biasv[b] = EPI == EPI_PART ? 0.0f : a.bias[(cb0 + b) * 16 + n];
  load_epi(0);
  if constexpr (kLN) {
    // after every load above is issued (the scheduling barrier keeps the
    // compiler from hoisting the wait for these two loads above them), and
    // unconditional (threads past D/4 rewrite the last slot with the same
    // value), so the loads are not sunk behind the others either
    __builtin_amdgcn_sched_barrier(0);
    const int q = min(tid, D / 4 - 1);
    reinterpret_cast<float4*>(s_g)[q] = gq;
    reinterpret_cast<float4*>(s_b)[q] = bq;
  }

  // The first row block runs whatever M is (with M = 0 it stores nothing), so
  // the loads above are never held back behind the read of M.
  int m0 = 0;
  do {
    if (m0 > 0) {
      load_a(m0, 0);
      if (rounds > 1) load_w(0);
      load_epi(m0);
    }
    f32x4_t acc[2][NB];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[r][b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    for (int round = 0; round < rounds; ++round) {
      if (round > 0) {
        load_a(m0, round);
        load_w(round);
      }
      // chunks this wave owns in this round (uniform)
      const int nv = max(0, min(CPW, kn - (round * NW + w) * CPW));

      float mean[2] = {0.0f, 0.0f}, rstd[2] = {0.0f, 0.0f};
      if constexpr (kLN) {  // K = D fits one round for the LayerNorm GEMMs
        float s[2] = {0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          if (c < nv) {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
              float x[8];
              unpack8(x, ab[c][r]);
#pragma unroll
              for (int j = 0; j < 8; ++j) s[r] += x[j];
            }
          }
        }
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          s[r] = row_sum4(s[r]);
          if (g == 0) s_st[w * 32 + 16 * r + n] = s[r];
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          float t = 0.0f;
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) t += s_st[ww * 32 + 16 * r + n];
          mean[r] = t / (float)D;
        }
        float q[2] = {0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          if (c < nv) {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
              float x[8];
              unpack8(x, ab[c][r]);
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const float d = x[j] - mean[r];
                q[r] += d * d;
              }
            }
          }
        }
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          q[r] = row_sum4(q[r]);
          if (g == 0) s_st[(NW + w) * 32 + 16 * r + n] = q[r];
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          float t = 0.0f;
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) t += s_st[(NW + ww) * 32 + 16 * r + n];
          rstd[r] = 1.0f / sqrtf(t / (float)D + a.sh.eps);
        }
      }

#pragma unroll
      for (int c = 0; c < CPW; ++c) {
        if (c < nv) {  // uniform: a scalar branch
          if constexpr (kLN) {
            const int k0 = (kb + (round * NW + w) * CPW + c) * 32 + 8 * g;
            float gg[8], bb[8];
            const float4 g0 = reinterpret_cast<const float4*>(s_g + k0)[0];
            const float4 g1 = reinterpret_cast<const float4*>(s_g + k0)[1];
            const float4 b0 = reinterpret_cast<const float4*>(s_b + k0)[0];
            const float4 b1 = reinterpret_cast<const float4*>(s_b + k0)[1];
            gg[0] = g0.x; gg[1] = g0.y; gg[2] = g0.z; gg[3] = g0.w;
            gg[4] = g1.x; gg[5] = g1.y; gg[6] = g1.z; gg[7] = g1.w;
            bb[0] = b0.x; bb[1] = b0.y; bb[2] = b0.z; bb[3] = b0.w;
            bb[4] = b1.x; bb[5] = b1.y; bb[6] = b1.z; bb[7] = b1.w;
#pragma unroll
            for (int r = 0; r < 2; ++r) {
              float x[8];
              unpack8(x, ab[c][r]);
              V8<T> av;
              ln8(av, x, mean[r], rstd[r], gg, bb);
#pragma unroll
              for (int b = 0; b < NB; ++b) mma(acc[r][b], av, wb[c][b]);
            }
          } else {
#pragma unroll
            for (int r = 0; r < 2; ++r)
#pragma unroll
              for (int b = 0; b < NB; ++b) mma(acc[r][b], ab[c][r], wb[c][b]);
          }
        }
      }
    }

    // ---- sum the waves' partial tiles in wave order
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int b = 0; b < NB; ++b) red[((w * 2 + r) * NB + b) * 64 + lane] = acc[r][b];
    __syncthreads();

    // ---- epilogue: wave w finishes row 4g + (w%4) of row tile w/4
    const float* redf = reinterpret_cast<const float*>(red);
    const int row = m0 + 16 * re + 4 * g + ie;
    const bool ok = row < M;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int col = (cb0 + b) * 16 + n;
      float x = 0.0f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) x += redf[(((ww * 2 + re) * NB + b) * 64 + lane) * 4 + ie];
      if constexpr (EPI == EPI_PART) {  // raw partial sum; bias and residual come with the fix-up
        if (ok) static_cast<float*>(a.out)[((size_t)blockIdx.y * a.mpad + row) * a.ldo + col] = x;
        continue;
      }
      x += biasv[b];
      if constexpr (EPI == EPI_QKV) {
        const int which = col / D, c = col - which * D;
        const T o = Elem<T>::cv(x);
        if (ok) {
          if (which == 0) {
            static_cast<T*>(a.out)[(size_t)row * a.ldo + c] = o;
          } else {
            const int hh = c / a.sh.dh, d = c - hh * a.sh.dh;
            char* base = rinfo.cache + (which == 1 ? a.cl.k : a.cl.v) + (size_t)a.layer * a.cl.kv_layer;
            const size_t e = which == 1 ? ((size_t)hh * a.sh.Npad + rinfo.tok) * a.sh.dh + d
                                        : ((size_t)hh * a.sh.dh + d) * a.sh.Npad + rinfo.tok;
            gbl(reinterpret_cast<T*>(base))[e] = o;
          }
        }
      } else if constexpr (EPI == EPI_OPROJ) {
        if (ok) static_cast<float*>(a.out)[(size_t)row * a.ldo + col] = Elem<T>::f(resv[b]) + x;
      } else if constexpr (EPI == EPI_FC1) {
        if (ok) static_cast<T*>(a.out)[(size_t)row * a.ldo + col] = Elem<T>::cv(gelu_tanh(x));
      } else {
        const T o = Elem<T>::cv(resv[b] + x);
        if (ok) {
          static_cast<T*>(a.out)[(size_t)row * a.ldo + col] = o;
          gbl(x_row<T>(rinfo.cache, a.cl, a.sh, a.layer + 1, rinfo.tok))[col] = o;
        }
      }
    }
    __syncthreads();  // red and the statistics are reused by the next row block
    m0 += kGemmRB;
  } while (m0 < M);
}

template <int NB>
inline size_t gemm_lds(const GemmArgs& a) {
  return (size_t)gemm_red_bytes<NB>() + (size_t)2 * a.sh.D * sizeof(float) + 2 * kGemmWaves * 32 * sizeof(float);
}

template <class T, int EPI, int NB, int CPW>
hipError_t launch_gemm_cfg(const GemmArgs& a, hipStream_t s) {
  static hipError_t attr = hipErrorNotReady;
  if (attr != hipSuccess) {
    const int most = gemm_red_bytes<NB>() + 2 * kMaxDim * (int)sizeof(float) + 2 * kGemmWaves * 32 * (int)sizeof(float);
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, EPI, NB, CPW>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, most);
    if (attr != hipSuccess) return attr;
  }
  return launch_k(gemm_kernel<T, EPI, NB, CPW>, dim3(a.Nout / 16 / NB, a.ksplit), dim3(kGemmWaves * 64),
                  gemm_lds<NB>(a), s, a);
}

// Chunks per wave: the smallest instantiated count that covers K in one round
// (the last wave may own fewer); longer K runs in rounds of the largest.
template <class T, int EPI, int NB>
hipError_t launch_gemm_nb(int cpw, const GemmArgs& a, hipStream_t s) {
  constexpr bool kWideA = sizeof(typename AType<T, EPI>::type) == 4;
  if (cpw <= 1) return launch_gemm_cfg<T, EPI, NB, 1>(a, s);
  if (cpw <= 2) return launch_gemm_cfg<T, EPI, NB, 2>(a, s);
  if (cpw <= 3) return launch_gemm_cfg<T, EPI, NB, 3>(a, s);
  if (cpw <= 4) return launch_gemm_cfg<T, EPI, NB, 4>(a, s);
  if (cpw <= 5) return launch_gemm_cfg<T, EPI, NB, 5>(a, s);
  if (cpw <= 6) return launch_gemm_cfg<T, EPI, NB, 6>(a, s);
  if constexpr (kWideA) {
    return launch_gemm_cfg<T, EPI, NB, 8>(a, s);
  } else {
    if (cpw <= 8) return launch_gemm_cfg<T, EPI, NB, 8>(a, s);
    if (cpw <= 12) return launch_gemm_cfg<T, EPI, NB, 12>(a, s);
    return launch_gemm_cfg<T, EPI, NB, 17>(a, s);
  }
}

// Largest chunks-per-wave instance for an A operand of this element size.
inline int gemm_max_cpw(bool wide_a) { return wide_a ? 8 : 17; }

template <int EPI>
hipError_t launch_gemm_epi(int cols, const GemmArgs& a, hipStream_t s) {
  const bool two = cols == 2 && (a.Nout / 16) % 2 == 0;
  const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
  const int need = (kper + kGemmWaves - 1) / kGemmWaves;
  if (a.sh.dtype) {
    const int cpw = std::min(need, gemm_max_cpw(EPI == EPI_FC1));
    return two ? launch_gemm_nb<uint16_t, EPI, 2>(cpw, a, s) : launch_gemm_nb<uint16_t, EPI, 1>(cpw, a, s);
  }
  const int cpw = std::min(need, gemm_max_cpw(true));
  return two ? launch_gemm_nb<float, EPI, 2>(cpw, a, s) : launch_gemm_nb<float, EPI, 1>(cpw, a, s);
}

}  // namespace incvit
