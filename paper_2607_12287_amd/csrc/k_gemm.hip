// The four per-layer GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and
// the residual + MLP that follows the attention):
//   QKV : [Q K V] = S(S(LN1(X^l[U])) W_qkv + b); Q -> workspace, K and V rows
//         scattered into the cached K^l, V^l of each stream (eq. 5);
//   OPROJ: H = X^l[U] + (O W_o + b_o)            (fp32)
//   FC1 : G = S(GELU(S(LN2(H)) W_1 + b_1))
//   FC2 : X^{l+1}[U] = S(H + (G W_2 + b_2))      scattered into the cache.
// Only the rows of U (M rows over all streams) are computed: with M small the
// work is streaming the weights from HBM, so each workgroup reads its weight
// columns exactly once, straight into MFMA operand registers (the packed
// layout makes every 32-deep chunk one vector load per lane), while the M
// activation rows sit in LDS.  K is split over the 4 waves and, when asked,
// over workgroups; partial sums are combined in a fixed order (no float
// atomics), so results are deterministic.
#include "common.hpp"

namespace incvit {

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanhf(u));
}

template <class T, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  constexpr bool kLN = (EPI == EPI_QKV || EPI == EPI_FC1);
  constexpr int PF = sizeof(T) == 2 ? 8 : 4;  // weight chunks in flight per wave
  constexpr int EB = sizeof(T);
  extern __shared__ __align__(16) char smem[];
  __shared__ int s_off[kMaxViews + 1];
  __shared__ int s_view[kGemmRows], s_tok[kGemmRows];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int cb = blockIdx.x, m0 = blockIdx.y * kGemmRows, z = blockIdx.z;
  const int M = row_offsets(a.rm, s_off);
  if (m0 >= M) return;
  const int mrows = min(kGemmRows, M - m0);
  const int nrt = (mrows + 15) >> 4;
  if (tid < kGemmRows) {
    int v = 0, tok = 0;
    if (tid < mrows) row_token(a.rm, s_off, m0 + tid, v, tok);
    s_view[tid] = v;
    s_tok[tid] = tok;
  }

  // K chunks of this workgroup, and every 4th of them for this wave.
  const int kc0 = (int)((long)z * a.kchunks / a.ksplit);
  const int kc1 = (int)((long)(z + 1) * a.kchunks / a.ksplit);
  const int nw = max(0, (kc1 - kc0 - w + kGemmWaves - 1) / kGemmWaves);
  const T* wbase = static_cast<const T*>(a.W) + (size_t)cb * a.kchunks * kChunkElems + lane * 8;

  V8<T> wb[PF];
#pragma unroll
  for (int s = 0; s < PF; ++s)
    if (s < nw) wb[s].load(wbase + (size_t)(kc0 + w + kGemmWaves * s) * kChunkElems);
  __syncthreads();

  // Stage this workgroup's A block (mrows x [klo, klo+kwid)) in LDS.
  const int D = a.sh.D;
  const int klo = kc0 * 32, kwid = (kc1 - kc0) * 32;
  const int ldsb = kwid * EB + 16;  // row stride in bytes (+16: no bank conflicts)
  if constexpr (kLN) {
    constexpr int kG = kMaxDim / 512;  // 8-element groups per lane
    for (int rl = w; rl < mrows; rl += kGemmWaves) {
      float x[kG][8];
#pragma unroll
      for (int j = 0; j < kG; ++j) {
        const int d = 8 * lane + 512 * j;
#pragma unroll
        for (int e = 0; e < 8; ++e) x[j][e] = 0.0f;
        if (d < D) {
          if constexpr (EPI == EPI_QKV) {
            const T* src = x_row<T>(a.caches, a.cl, a.sh, s_view[rl], a.layer, s_tok[rl]) + d;
            V8<T> t;
            t.load(src);
            if constexpr (sizeof(T) == 2) {
              const uint32_t q[4] = {t.v.x, t.v.y, t.v.z, t.v.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                x[j][2 * e] = __uint_as_float(q[e] << 16);
                x[j][2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
              }
            } else {
              x[j][0] = t.a.x; x[j][1] = t.a.y; x[j][2] = t.a.z; x[j][3] = t.a.w;
              x[j][4] = t.b.x; x[j][5] = t.b.y; x[j][6] = t.b.z; x[j][7] = t.b.w;
            }
          } else {
            const float4* src = reinterpret_cast<const float4*>(
                static_cast<const float*>(a.A) + (size_t)(m0 + rl) * a.lda + d);
            const float4 p0 = src[0], p1 = src[1];
            x[j][0] = p0.x; x[j][1] = p0.y; x[j][2] = p0.z; x[j][3] = p0.w;
            x[j][4] = p1.x; x[j][5] = p1.y; x[j][6] = p1.z; x[j][7] = p1.w;
          }
        }
      }
      float s = 0.0f;
#pragma unroll
      for (int j = 0; j < kG; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) s += x[j][e];
      const float mean = wave_sum(s) / (float)D;
      float q = 0.0f;
#pragma unroll
      for (int j = 0; j < kG; ++j) {
        if (8 * lane + 512 * j < D) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float c = x[j][e] - mean;
            q += c * c;
          }
        }
      }
      const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + a.sh.eps);
      char* row = smem + rl * ldsb;
#pragma unroll
      for (int j = 0; j < kG; ++j) {
        const int d = 8 * lane + 512 * j;
        if (d < D && d >= klo && d < klo + kwid) {
          T* dst = reinterpret_cast<T*>(row + (d - klo) * EB);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            dst[e] = Elem<T>::cv((x[j][e] - mean) * rstd * a.ln_g[d + e] + a.ln_b[d + e]);
        }
      }
    }
  } else {
    // plain copy of the compact rows, 8 elements (one MFMA operand) at a time
    const int groups = kwid / 8;
    for (int rl = w; rl < mrows; rl += kGemmWaves) {
      const T* src = static_cast<const T*>(a.A) + (size_t)(m0 + rl) * a.lda + klo;
      char* row = smem + rl * ldsb;
      for (int e = lane; e < groups; e += 64) {
        V8<T> t;
        t.load(src + 8 * e);
        *reinterpret_cast<V8<T>*>(row + 8 * e * EB) = t;
      }
    }
  }
  __syncthreads();

  f32x4_t acc[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) acc[rt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  for (int i0 = 0; i0 < nw; i0 += PF) {
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      const int i = i0 + s;
      if (i < nw) {
        const int kc = kc0 + w + kGemmWaves * i;
        const char* abase = smem + n * ldsb + ((kc - kc0) * 32 + 8 * g) * EB;
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
          if (rt < nrt) {
            V8<T> av = *reinterpret_cast<const V8<T>*>(abase + 16 * rt * ldsb);
            mma(acc[rt], av, wb[s]);
          }
        }
        if (i + PF < nw) wb[s].load(wbase + (size_t)(kc + kGemmWaves * PF) * kChunkElems);
      }
    }
  }

  // Sum the 4 waves' partial tiles in wave order; wave w finishes row tile w.
  __syncthreads();
  f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
    if (rt < nrt) red[(w * 4 + rt) * 64 + lane] = acc[rt];
  __syncthreads();
  const int rt = w;
  f32x4_t val = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  if (rt < nrt) {
    val = red[(0 * 4 + rt) * 64 + lane];
#pragma unroll
    for (int ww = 1; ww < kGemmWaves; ++ww) val += red[(ww * 4 + rt) * 64 + lane];
  }
  const int col = cb * 16 + n;

  if (a.ksplit > 1) {
    // Partial tile to global; the last workgroup of this tile adds all splits
    // in split order and runs the epilogue; it then re-arms the counter.
    if (rt < nrt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + 16 * rt + 4 * g + i;
        a.partial[((size_t)z * a.Mpad + row) * a.Nout + col] = val[i];
      }
    }
    __threadfence();
    __syncthreads();
    int* ctr = a.counters + blockIdx.y * gridDim.x + cb;
    if (tid == 0) {
      const int prev = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == a.ksplit - 1);
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (rt < nrt) {
      val = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      for (int zz = 0; zz < a.ksplit; ++zz) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + 16 * rt + 4 * g + i;
          val[i] += __hip_atomic_load(a.partial + ((size_t)zz * a.Mpad + row) * a.Nout + col,
                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
    if (tid == 0) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (rt >= nrt) return;

  const float bias = a.bias[col];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rl = 16 * rt + 4 * g + i;
    if (rl >= mrows) continue;
    const float x = val[i] + bias;
    const int v = s_view[rl], tok = s_tok[rl];
    if constexpr (EPI == EPI_QKV) {
      const int which = col / D, c = col - which * D;
      const T o = Elem<T>::cv(x);
      if (which == 0) {
        static_cast<T*>(a.out)[(size_t)(m0 + rl) * a.ldo + c] = o;
      } else {
        const int hh = c / a.sh.dh, d = c - hh * a.sh.dh;
        char* base = a.caches.p[v] + (which == 1 ? a.cl.k : a.cl.v) + (size_t)a.layer * a.cl.kv_layer;
        const size_t e = which == 1 ? ((size_t)hh * a.sh.Npad + tok) * a.sh.dh + d
                                    : ((size_t)hh * a.sh.dh + d) * a.sh.Npad + tok;
        reinterpret_cast<T*>(base)[e] = o;
      }
    } else if constexpr (EPI == EPI_OPROJ) {
      const float xin = Elem<T>::ld(x_row<T>(a.caches, a.cl, a.sh, v, a.layer, tok), col);
      static_cast<float*>(a.out)[(size_t)(m0 + rl) * a.ldo + col] = xin + x;
    } else if constexpr (EPI == EPI_FC1) {
      static_cast<T*>(a.out)[(size_t)(m0 + rl) * a.ldo + col] = Elem<T>::cv(gelu_tanh(x));
    } else {
      const float hv = a.hres[(size_t)(m0 + rl) * D + col];
      x_row<T>(a.caches, a.cl, a.sh, v, a.layer + 1, tok)[col] = Elem<T>::cv(hv + x);
    }
  }
}

template <int EPI>
static hipError_t launch_one(const GemmArgs& a, dim3 grid, size_t lds, hipStream_t s) {
  if (a.sh.dtype) hipLaunchKernelGGL((gemm_kernel<uint16_t, EPI>), grid, dim3(256), lds, s, a);
  else hipLaunchKernelGGL((gemm_kernel<float, EPI>), grid, dim3(256), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, const GemmArgs& a, int mmax, size_t lds, hipStream_t s) {
  dim3 grid(a.Nout / 16, (mmax + kGemmRows - 1) / kGemmRows, a.ksplit);
  switch (epi) {
    case EPI_QKV: return launch_one<EPI_QKV>(a, grid, lds, s);
    case EPI_OPROJ: return launch_one<EPI_OPROJ>(a, grid, lds, s);
    case EPI_FC1: return launch_one<EPI_FC1>(a, grid, lds, s);
    default: return launch_one<EPI_FC2>(a, grid, lds, s);
  }
}

template <int EPI>
static hipError_t set_lds(size_t bytes) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<uint16_t, EPI>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<float, EPI>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

hipError_t gemm_set_lds_limits(size_t bytes) {
  hipError_t e;
  if ((e = set_lds<EPI_QKV>(bytes)) != hipSuccess) return e;
  if ((e = set_lds<EPI_OPROJ>(bytes)) != hipSuccess) return e;
  if ((e = set_lds<EPI_FC1>(bytes)) != hipSuccess) return e;
  return set_lds<EPI_FC2>(bytes);
}

}  // namespace incvit
