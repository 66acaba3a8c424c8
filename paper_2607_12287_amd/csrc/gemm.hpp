// The GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and the residual +
// MLP that follows the attention), on compact workspace buffers over the M
// refreshed rows of the call (rows padded to a multiple of 64):
//   QKV : [Q K V] = S(A1 W_qkv + b), A1 = S(LN1(Z_l)) already normalised by the
//         row kernel that produced Z_l; Q -> workspace, K and V rows scattered
//         into the cached K^l, V^l of each stream (eq. 5);
//   RES : the output projection with its residual, H = S(Z_l + (O W_o + b_o)),
//         plus LayerNorm partial statistics of H over each 16-column block
//         (mean and sum of squared deviations);
//   FC1 : G = S(GELU(A2 W_1 + b_1)) with A2 = S(LN2(H)) formed while the
//         operand is loaded: the block statistics of H are merged in a fixed
//         order into the row mean and variance first;
//   PART: raw partial sums of A W over one share of K (the MLP down
//         projection); a row kernel adds the bias, the residual and the next
//         LayerNorm.
// A1, O, G and H are kept in MFMA operand order (frag_off).
//
// With M a few dozen rows these are weight-streaming problems whose time is set
// by memory latency, so a workgroup issues every load it needs for its first
// 32 rows at once, before it knows M: the A fragments of rows 0..31 (the padded
// workspace keeps that in bounds), all of its waves' weight chunks and the
// epilogue operands.  Weights go straight into MFMA operand registers (the
// packed layout makes one 32-deep chunk of a 16-column block one 16-byte load
// per lane) and stay there for later row blocks.
//
// Workgroup: NW waves (8; 12 for FC1, whose operand conversion needs the
// registers), NB 16-column blocks; wave w owns a contiguous run of CPW chunks
// of this workgroup's share of K (rounds of NW*CPW chunks when longer).  The
// waves' partial tiles are summed in wave order through LDS and the epilogue
// is spread over the first 8 waves.  No atomics: results are deterministic.
#pragma once
#include <type_traits>

#include "common.hpp"

namespace incvit {

constexpr int kGemmWaves = 8;                     // waves of every GEMM but FC1
constexpr int kFc1Waves = 12;
constexpr int kGemmRB = 32;                       // rows per block: two 16-row MFMA tiles
constexpr int kStatParts = 16;                    // lanes that merge one row's block statistics
constexpr int kStatMax = kMaxDim / 16 / kStatParts;  // blocks per lane

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanhf(u));
}

template <int EPI>
__host__ __device__ constexpr int gemm_waves() {
  return EPI == EPI_FC1 ? kFc1Waves : kGemmWaves;
}
template <int NB, int NW>
__host__ __device__ constexpr int gemm_red_bytes() {
  return NW * 2 * NB * 64 * 16;
}
// LDS: the wave partial tiles, then (mean, rstd) of the block's rows, then
// (FC1) the LN2 gamma and beta
template <int NB, int NW>
__host__ __device__ constexpr int gemm_lds_bytes() {
  return gemm_red_bytes<NB, NW>() + kGemmRB * 8;
}
// FC1 stages gamma and beta through LDS: every thread stores kGbPer float4 of
// each (unconditionally, past D into padding), gamma first
template <int NW>
__host__ __device__ constexpr int gb_per() {
  return (kMaxDim / 4 + NW * 64 - 1) / (NW * 64);
}
template <int NW>
__host__ __device__ constexpr int gb_bytes() {
  return 2 * gb_per<NW>() * NW * 64 * 16;
}
template <int EPI, int NB>
inline size_t gemm_lds_bytes(int D) {
  (void)D;
  return (size_t)gemm_lds_bytes<NB, gemm_waves<EPI>()>() + (EPI == EPI_FC1 ? gb_bytes<gemm_waves<EPI>()>() : 0);
}

// LDS-only barrier: waits for this wave's LDS traffic, not for its global
// loads (a full __syncthreads also waits for every outstanding global load)
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0); vmcnt, expcnt unconstrained
  __builtin_amdgcn_s_barrier();
}

// Row statistics from the 16-column block statistics (block mean m_b, sum of
// squared deviations q_b; every block has 16 columns): mean = sum_b m_b / nblk,
// M2 = sum_b (q_b + 16 (m_b - mean)^2).  Lane `part` of a row's 16 lanes sums
// blocks part, part + 16, ... in order, then the lanes are combined by a fixed
// butterfly.
__device__ __forceinline__ float sum16(float x) {
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// A2 operand from 8 values of H: S(((h - mean) * rstd) * gamma + beta),
// evaluated as fma(fma(h, rstd, -mean * rstd), gamma, beta) (nm = -mean * rstd)
__device__ __forceinline__ void ln_operand(V8<uint16_t>& out, const V8<uint16_t>& h, float rstd, float nm,
                                           const V8<float>& gm, const V8<float>& bt) {
  const uint32_t hq[4] = {h.v.x, h.v.y, h.v.z, h.v.w};
  float x[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(hq[e] << 16);
    x[2 * e + 1] = __uint_as_float(hq[e] & 0xffff0000u);
  }
  const float g8[8] = {gm.a.x, gm.a.y, gm.a.z, gm.a.w, gm.b.x, gm.b.y, gm.b.z, gm.b.w};
  const float b8[8] = {bt.a.x, bt.a.y, bt.a.z, bt.a.w, bt.b.x, bt.b.y, bt.b.z, bt.b.w};
  uint32_t q[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    q[e] = f2bf2(fmaf(fmaf(x[2 * e], rstd, nm), g8[2 * e], b8[2 * e]),
                 fmaf(fmaf(x[2 * e + 1], rstd, nm), g8[2 * e + 1], b8[2 * e + 1]));
  out.v = make_uint4(q[0], q[1], q[2], q[3]);
}
__device__ __forceinline__ float ln1(float x, float rstd, float nm, float g, float b) {
  return fmaf(fmaf(x, rstd, nm), g, b);
}
__device__ __forceinline__ void ln_operand(V8<float>& out, const V8<float>& h, float rstd, float nm,
                                           const V8<float>& gm, const V8<float>& bt) {
  out.a = make_float4(ln1(h.a.x, rstd, nm, gm.a.x, bt.a.x), ln1(h.a.y, rstd, nm, gm.a.y, bt.a.y),
                      ln1(h.a.z, rstd, nm, gm.a.z, bt.a.z), ln1(h.a.w, rstd, nm, gm.a.w, bt.a.w));
  out.b = make_float4(ln1(h.b.x, rstd, nm, gm.b.x, bt.b.x), ln1(h.b.y, rstd, nm, gm.b.y, bt.b.y),
                      ln1(h.b.z, rstd, nm, gm.b.z, bt.b.z), ln1(h.b.w, rstd, nm, gm.b.w, bt.b.w));
}

template <class T, int EPI, int NB, int CPW>
__global__ __launch_bounds__(gemm_waves<EPI>() * 64) void gemm_kernel(GemmArgs a) {
  constexpr int NW = gemm_waves<EPI>();
  extern __shared__ __align__(16) char smem[];
  f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);                          // [NW][2][NB][64]
  float2* s_st = reinterpret_cast<float2*>(smem + gemm_red_bytes<NB, NW>());  // [32] (mean, rstd)
  float* s_gb = reinterpret_cast<float*>(smem + gemm_lds_bytes<NB, NW>());     // FC1: gamma, beta (padded)
  constexpr int kGbFloats = gb_per<NW>() * NW * 64 * 4;                        // floats of gamma's region

  const int tid = threadIdx.x, lane = tid & 63;
  // w lives in a scalar register, so every guard that depends on it is a
  // scalar branch: an MFMA must never run under a partial or empty lane mask
  // (it would still accumulate)
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, n = lane & 15;
  const int D = a.sh.D;
  const int M = a.meta->m;
  const int cb0 = blockIdx.x * NB;
  // this workgroup's share of K: chunks [kb, kb + kn)
  const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
  const int kb = blockIdx.y * kper, kn = min(kper, a.kchunks - kb);
  const int kc_last = kn - 1;
  const int rounds = (kn + NW * CPW - 1) / (NW * CPW);
  const T* W = static_cast<const T*>(a.W);

  auto kc_of = [&](int round, int c) { return kb + min((round * NW + w) * CPW + c, kc_last); };
  V8<T> ab[CPW][2];
  V8<T> wb[CPW][NB];
  // operand loads are buffer loads: one lane offset for all of them, the
  // chunk's position as a wave-uniform offset.  A is stored in operand order
  // (frag_off): row tile t, chunk kc is the kilobyte (t * akc + kc) (bf16;
  // two kilobytes for fp32).  FC1 reads H, normalised below with gamma/beta
  // staged in LDS.
  const int akc = a.lda / 32;
  constexpr uint32_t kAeb = sizeof(T);
  const Rsrc rA = make_rsrc(a.A, (uint32_t)a.mpad * a.lda * kAeb);
  const Rsrc rW = make_rsrc(a.W, (uint32_t)(a.Nout / 16) * a.kchunks * kChunkElems * sizeof(T));
  const uint32_t voffA = lane * 8 * kAeb, voffW = lane * 8 * sizeof(T);
  V8<T> hf[EPI == EPI_FC1 ? CPW : 1][2];
  auto load_a = [&](int m0, int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      const int kc = kc_of(round, c);
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const uint32_t soff = (uint32_t)(((m0 >> 4) + r) * akc + kc) * kChunkElems * kAeb;
        if constexpr (EPI == EPI_FC1) hf[c][r].bload(rA, voffA, soff);
        else ab[c][r].bload(rA, voffA, soff);
      }
    }
  };
  auto load_w = [&](int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int b = 0; b < NB; ++b)
        wb[c][b].bload(rW, voffW, (uint32_t)((cb0 + b) * a.kchunks + kc_of(round, c)) * kChunkElems * sizeof(T));
  };
  // FC1: block statistics of the rows of this block ([row][block]); thread
  // t < 512 merges blocks part, part + 16, ... of row t / 16 (blocks past the
  // last are not merged; those past the buffer read zero)
  const int st_row = (tid >> 4) & (kGemmRB - 1), st_part = tid & (kStatParts - 1);
  const int nblk = D / 16;
  float2 sv[EPI == EPI_FC1 ? kStatMax : 1];
  const Rsrc rS = make_rsrc(a.stats, (uint32_t)nblk * a.mpad * 8);
  auto load_stats = [&](int m0) {
#pragma unroll
    for (int i = 0; i < kStatMax; ++i) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(rS, (uint32_t)(st_row * nblk + st_part) * 8,
                                                          (uint32_t)(m0 * nblk + kStatParts * i) * 8, 0);
      sv[i] = make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
    }
  };
  // epilogue item of this wave: row tile w/4, row 4g + (w%4) of the tile
  const int re = w >> 2, ie = w & 3;
  RowInfo rinfo = RowInfo{nullptr, 0, 0};
  float biasv[NB], resv[NB];
  auto load_res = [&](int m0) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
      resv[b] = Elem<T>::f(static_cast<const T*>(a.resid)[(size_t)(m0 + 16 * re + 4 * g + ie) * D + (cb0 + b) * 16 + n]);
  };

  if constexpr (EPI == EPI_FC1) {
    // gamma and beta into LDS (made visible by the barrier of the statistics);
    // every load is issued before the first wait
    constexpr int kPer = gb_per<NW>();
    float4 gv[kPer], bv[kPer];
    const Rsrc rg = make_rsrc(a.ln_g, D * 4), rb = make_rsrc(a.ln_b, D * 4);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {  // past D these read zero
      gv[i] = bload16f(rg, tid * 16, i * NW * 64 * 16);
      bv[i] = bload16f(rb, tid * 16, i * NW * 64 * 16);
    }
    load_stats(0);
    __builtin_amdgcn_sched_barrier(0);  // the small loads go out first
    load_a(0, 0);
    load_w(0);
#pragma unroll
    for (int b = 0; b < NB; ++b) biasv[b] = a.bias[(cb0 + b) * 16 + n];
    __builtin_amdgcn_sched_barrier(0);  // every load is out before the first wait
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = tid + i * NW * 64;
      reinterpret_cast<float4*>(s_gb)[q] = gv[i];
      reinterpret_cast<float4*>(s_gb + kGbFloats)[q] = bv[i];
    }
  } else {
    load_a(0, 0);
    load_w(0);
#pragma unroll
    for (int b = 0; b < NB; ++b) biasv[b] = EPI == EPI_PART ? 0.0f : a.bias[(cb0 + b) * 16 + n];
  }
  if constexpr (EPI == EPI_QKV) rinfo = a.rows[16 * re + 4 * g + ie];
  if constexpr (EPI == EPI_RES) load_res(0);

  // One 32-row block.  The first block is a copy of its own (FIRST), which
  // runs whatever M is (with M = 0 it stores nothing), so the loads above are
  // never held back behind the read of M, and its waits count exactly the
  // loads issued above instead of the fewer a later block reloads.
  auto row_block = [&](const int m0, auto first) {
    if constexpr (!decltype(first)::value) {
      if constexpr (EPI == EPI_FC1) load_stats(m0);
      load_a(m0, 0);
      if (rounds > 1) load_w(0);
      if constexpr (EPI == EPI_QKV) rinfo = a.rows[m0 + 16 * re + 4 * g + ie];
      if constexpr (EPI == EPI_RES) load_res(m0);
    }
    float nmr[2] = {0.0f, 0.0f}, rstd[2] = {0.0f, 0.0f};  // -mean * rstd, rstd of the lane's rows
    if constexpr (EPI == EPI_FC1) {
      // row statistics: a fixed merge order over the 16-column blocks (the
      // first 8 waves; a scalar branch)
      if (w < kGemmRB * kStatParts / 64) {
        float s1 = 0.0f;
#pragma unroll
        for (int i = 0; i < kStatMax; ++i)
          if (st_part + kStatParts * i < nblk) s1 += sv[i].x;
        const float mean = sum16(s1) / (float)nblk;
        float s2 = 0.0f;
#pragma unroll
        for (int i = 0; i < kStatMax; ++i) {
          const float d = sv[i].x - mean;
          if (st_part + kStatParts * i < nblk) s2 += sv[i].y + 16.0f * (d * d);
        }
        const float m2 = sum16(s2);
        if (st_part == 0) s_st[st_row] = make_float2(mean, 1.0f / sqrtf(m2 / (float)D + a.sh.eps));
      }
      lds_barrier();
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const float2 s = s_st[16 * r + n];
        rstd[r] = s.y;
        nmr[r] = -s.x * s.y;
      }
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
      const int nv = max(0, min(CPW, kn - (round * NW + w) * CPW));  // chunks owned (uniform)
#pragma unroll
      for (int c = 0; c < CPW; ++c) {
        if constexpr (EPI == EPI_FC1) {  // A2 = S(LN2(H)) of this chunk, just before its products
          V8<float> gm, bt;
          const int k0 = kc_of(round, c) * 32 + 8 * g;
          gm.a = reinterpret_cast<const float4*>(s_gb + k0)[0];
          gm.b = reinterpret_cast<const float4*>(s_gb + k0)[1];
          bt.a = reinterpret_cast<const float4*>(s_gb + kGbFloats + k0)[0];
          bt.b = reinterpret_cast<const float4*>(s_gb + kGbFloats + k0)[1];
#pragma unroll
          for (int r = 0; r < 2; ++r) ln_operand(ab[c][r], hf[c][r], rstd[r], nmr[r], gm, bt);
        }
        if (c < nv) {  // a scalar branch
#pragma unroll
          for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int b = 0; b < NB; ++b) mma(acc[r][b], ab[c][r], wb[c][b]);
        }
      }
    }

    // ---- sum the waves' partial tiles in wave order
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int b = 0; b < NB; ++b) red[((w * 2 + r) * NB + b) * 64 + lane] = acc[r][b];
    __syncthreads();

    // ---- epilogue: wave w < 8 finishes row 4g + (w%4) of row tile w/4
    const float* redf = reinterpret_cast<const float*>(red);
    const int row = m0 + 16 * re + 4 * g + ie;
    const bool ok = row < M;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (w >= kGemmWaves) break;  // a scalar branch
      const int col = (cb0 + b) * 16 + n;
      float x = 0.0f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) x += redf[(((ww * 2 + re) * NB + b) * 64 + lane) * 4 + ie];
      if constexpr (EPI == EPI_PART) {
        if (ok) static_cast<float*>(a.out)[((size_t)blockIdx.y * a.mpad + row) * a.ldo + col] = x;
      } else if constexpr (EPI == EPI_RES) {
        // H = S(Z + (O W_o + b_o)), and the moments of this row's 16 columns
        const float hv = Elem<T>::rnd(resv[b] + (x + biasv[b]));
        float s = hv;
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) s += __shfl_xor(s, off, 64);
        const float bm = s * (1.0f / 16.0f);
        float q = (hv - bm) * (hv - bm);
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) q += __shfl_xor(q, off, 64);
        if (ok) {
          static_cast<T*>(a.out)[frag_off(row, col, a.ldo / 32)] = Elem<T>::cv(hv);
          if (n == 0) a.stats[(size_t)row * (D / 16) + cb0 + b] = make_float2(bm, q);
        }
      } else if constexpr (EPI == EPI_QKV) {
        x += biasv[b];
        const int which = col / D, c = col - which * D;
        const T o = Elem<T>::cv(x);
        if (ok) {
          if (which == 0) {
            static_cast<T*>(a.out)[(size_t)row * a.ldo + c] = o;
          } else {
            const int hh = c / a.sh.dh, d = c - hh * a.sh.dh;
            char* base = rinfo.cache + (which == 1 ? a.cl.k : a.cl.v) + (size_t)a.layer * a.cl.kv_layer;
            const size_t e = which == 1 ? k_elem(a.sh, hh, rinfo.tok, d) : v_elem(a.sh, hh, rinfo.tok, d);
            gbl(reinterpret_cast<T*>(base))[e] = o;
          }
        }
      } else {  // EPI_FC1
        x += biasv[b];
        if (ok) static_cast<T*>(a.out)[frag_off(row, col, a.ldo / 32)] = Elem<T>::cv(gelu_tanh(x));
      }
    }
    __syncthreads();  // red and the row statistics are reused by the next row block
  };
  row_block(0, std::true_type{});
  for (int m0 = kGemmRB; m0 < M; m0 += kGemmRB) row_block(m0, std::false_type{});
}

template <class T, int EPI, int NB, int CPW>
hipError_t launch_gemm_cfg(const GemmArgs& a, hipStream_t s) {
  return launch_k(gemm_kernel<T, EPI, NB, CPW>, dim3(a.Nout / 16 / NB, a.ksplit), dim3(gemm_waves<EPI>() * 64),
                  gemm_lds_bytes<EPI, NB>(a.sh.D), s, a);
}

// Chunks per wave: the smallest instantiated count that covers this
// workgroup's share of K in one round (the last wave may own fewer); longer
// shares run in rounds of the largest.
template <class T, int EPI, int NB>
hipError_t launch_gemm_nb(int cpw, const GemmArgs& a, hipStream_t s) {
  if (cpw <= 1) return launch_gemm_cfg<T, EPI, NB, 1>(a, s);
  if (cpw <= 2) return launch_gemm_cfg<T, EPI, NB, 2>(a, s);
  if (cpw <= 3) return launch_gemm_cfg<T, EPI, NB, 3>(a, s);
  if (cpw <= 4) return launch_gemm_cfg<T, EPI, NB, 4>(a, s);
  if (cpw <= 5) return launch_gemm_cfg<T, EPI, NB, 5>(a, s);
  if (cpw <= 6) return launch_gemm_cfg<T, EPI, NB, 6>(a, s);
  return launch_gemm_cfg<T, EPI, NB, 8>(a, s);
}

template <int EPI>
hipError_t launch_gemm_epi(int cols, const GemmArgs& a, hipStream_t s) {
  const bool two = cols == 2 && (a.Nout / 16) % 2 == 0;
  const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
  const int cpw = std::min((kper + gemm_waves<EPI>() - 1) / gemm_waves<EPI>(), 8);
  if (a.sh.dtype) return two ? launch_gemm_nb<uint16_t, EPI, 2>(cpw, a, s) : launch_gemm_nb<uint16_t, EPI, 1>(cpw, a, s);
  return two ? launch_gemm_nb<float, EPI, 2>(cpw, a, s) : launch_gemm_nb<float, EPI, 1>(cpw, a, s);
}

}  // namespace incvit
