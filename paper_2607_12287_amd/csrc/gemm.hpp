// The GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and the residual +
// MLP that follows the attention), on compact [row][column] workspace buffers
// over the M refreshed rows of the call (rows padded to a multiple of 64):
//   QKV : [Q K V] = S(A1 W_qkv + b), A1 = S(LN1(Z_l)) already normalised by the
//         row kernel that produced Z_l; Q -> workspace, K and V rows scattered
//         into the cached K^l, V^l of each stream (eq. 5);
//   FC1 : G = S(GELU(A2 W_1 + b_1)), A2 = S(LN2(H)) from the row kernel;
// (A1, A2, O and G are kept in MFMA operand order, frag_off)
//   PART: raw partial sums of A W over one share of K (the output projection
//         and the MLP down projection); a row kernel adds the bias, the
//         residual and the next LayerNorm.
//
// With M a few dozen rows these are weight-streaming problems whose time is set
// by memory latency, so a workgroup issues every load it needs for its first
// 32 rows at once, before it knows M: the A fragments of rows 0..31 (the padded
// workspace keeps that in bounds), all of its waves' weight chunks and the
// epilogue operands.  Weights go straight into MFMA operand registers (the
// packed layout makes one 32-deep chunk of a 16-column block one 16-byte load
// per lane) and stay there for later row blocks.
//
// Workgroup: 8 waves, NB 16-column blocks; wave w owns a contiguous run of CPW
// chunks of this workgroup's share of K (rounds of 8*CPW chunks when longer).
// The waves' partial tiles are summed in wave order through LDS and the
// epilogue is spread over all waves.  No atomics: results are deterministic.
#pragma once
#include "common.hpp"

namespace incvit {

constexpr int kGemmWaves = 8;
constexpr int kGemmRB = 32;  // rows per block: two 16-row MFMA tiles

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanhf(u));
}

template <int NB>
__host__ __device__ constexpr int gemm_red_bytes() {
  return kGemmWaves * 2 * NB * 64 * 16;
}

template <class T, int EPI, int NB, int CPW>
__global__ __launch_bounds__(kGemmWaves * 64) void gemm_kernel(GemmArgs a) {
  constexpr int NW = kGemmWaves;
  extern __shared__ __align__(16) char smem[];
  f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);  // [NW][2][NB][64]

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
  const T* A = static_cast<const T*>(a.A);
  const T* W = static_cast<const T*>(a.W);

  auto kc_of = [&](int round, int c) { return kb + min((round * NW + w) * CPW + c, kc_last); };
  V8<T> ab[CPW][2];
  V8<T> wb[CPW][NB];
  const int akc = a.lda / 32;  // A is stored in operand order (frag_off)
  auto load_a = [&](int m0, int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int r = 0; r < 2; ++r)
        ab[c][r].load(A + (((size_t)((m0 >> 4) + r) * akc + kc_of(round, c)) * 64 + lane) * 8);
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
  float biasv[NB];

  load_a(0, 0);
  load_w(0);
#pragma unroll
  for (int b = 0; b < NB; ++b) biasv[b] = EPI == EPI_PART ? 0.0f : a.bias[(cb0 + b) * 16 + n];
  if constexpr (EPI == EPI_QKV) rinfo = a.rows[16 * re + 4 * g + ie];

  // The first row block runs whatever M is (with M = 0 it stores nothing), so
  // the loads above are never held back behind the read of M.
  int m0 = 0;
  do {
    if (m0 > 0) {
      load_a(m0, 0);
      if (rounds > 1) load_w(0);
      if constexpr (EPI == EPI_QKV) rinfo = a.rows[m0 + 16 * re + 4 * g + ie];
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
      if constexpr (EPI == EPI_PART) {
        if (ok) static_cast<float*>(a.out)[((size_t)blockIdx.y * a.mpad + row) * a.ldo + col] = x;
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
    __syncthreads();  // red is reused by the next row block
    m0 += kGemmRB;
  } while (m0 < M);
}

template <class T, int EPI, int NB, int CPW>
hipError_t launch_gemm_cfg(const GemmArgs& a, hipStream_t s) {
  return launch_k(gemm_kernel<T, EPI, NB, CPW>, dim3(a.Nout / 16 / NB, a.ksplit), dim3(kGemmWaves * 64),
                  (size_t)gemm_red_bytes<NB>(), s, a);
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
  const int cpw = std::min((kper + kGemmWaves - 1) / kGemmWaves, 8);
  if (a.sh.dtype) return two ? launch_gemm_nb<uint16_t, EPI, 2>(cpw, a, s) : launch_gemm_nb<uint16_t, EPI, 1>(cpw, a, s);
  return two ? launch_gemm_nb<float, EPI, 2>(cpw, a, s) : launch_gemm_nb<float, EPI, 1>(cpw, a, s);
}

}  // namespace incvit
