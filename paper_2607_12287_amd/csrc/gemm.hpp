// The GEMMs of the refreshed rows (paper §III-B, eqs. 4-5 and the residual +
// MLP that follows the attention), on compact workspace buffers over the M
// refreshed rows of the call (rows padded to a multiple of 64):
//   QKV : [Q K V] = S(LN1(Z_l) W_qkv + b); Q -> workspace, K and V rows
//         scattered into the cached K^l, V^l of each stream (eq. 5);
//   RES : the output projection with its residual, H = S(Z_l + S(O W_o + b_o));
//   FC1 : G = S(GELU(S(LN2(H) W_1 + b_1)));
//   PART: raw partial sums of A W over one share of K (the MLP down
//         projection); a row kernel adds the bias, the residual and the
//         next LayerNorm;
//   ATT : the attention branch S(O W_o + b_o) alone, scattered into the
//         cache's A^l rows (the all-rows MLP reading, whose residual is
//         formed for every row by a row kernel);
//   DOWN: the MLP down projection over the whole K with its residual,
//         Z_{l+1} = S(H + S(G W_2 + b_2)) into the compact Z and the cache's
//         X^{l+1} (one kernel instead of split-K partials and a row kernel).
// Every operation's result is rounded to the storage type once, as a
// half-precision pipeline stores it: the linear output with its bias, then the
// residual sum, and the MLP's up projection before its GELU.
// Z, O, H and G are kept in MFMA operand order (frag_off).
//
// LayerNorm folded into the GEMM (QKV, FC1): the weights are packed as
// W' = S(gamma W) with c1 = column sums of W' and c2b = beta^T W + b, so that
// LN(x) W + b = rstd (x W') - rstd mean c1 + c2b.  The GEMM runs on the raw
// rows x; a workgroup holds the whole K range of its 32 rows, split over its
// waves, and forms the row statistics on the matrix cores alongside the
// product: x * ones gives the row sums and x * x^T (the A fragment is also a
// valid B fragment of x^T) the sums of squares on its diagonal.  The waves'
// partial sums meet in LDS with the partial tiles and are combined in wave
// order in the epilogue (mean = sum / D, var = sumsq / D - mean^2).  This
// one-pass variance loses about (mean / spread)^2 * 2^-24 of its relative
// precision, harmless against bf16 storage (1e-3 at a mean 130 times the
// spread); fp32 models, whose results are held to fp32 precision, take the
// sums of the shifted values x - x_0 (x_0: the row's first element, so the
// differences are exact) on the vector units instead, which leaves no
// cancellation when the row's mean is large against its spread.
//
// With M a few dozen rows these are weight-streaming problems whose time is set
// by memory latency, so a workgroup of the first row group issues every load
// it needs at once, before it knows M: the A fragments of rows 0..31 (the
// padded workspace keeps that in bounds), all of its waves' weight chunks and
// the epilogue operands.  Weights go straight into MFMA operand registers (the
// packed layout makes one 32-deep chunk of a 16-column block one 16-byte load
// per lane).  Operands are read with buffer loads: one lane offset shared by
// all of them and the chunk's position as a wave-uniform offset.
//
// Grid: (column groups) x (K splits) x (row groups: up to 8, enough for the
// call's largest M).  Row group z owns the 32-row blocks z, z + nz, ...; row
// groups past M leave after reading M.  Workgroups are renumbered XCD-major (the hardware deals
// them to the 8 XCDs round robin), with the row group fastest, so the row
// groups of one column block share an XCD and its L2 holds their weights.
//
// Workgroup: NW = 8 waves, NB 16-column blocks; wave w owns a
// contiguous run of CPW chunks of this workgroup's share of K (rounds of
// NW*CPW chunks when longer).  The waves'
// partial tiles are summed in wave order through LDS and the epilogue is
// spread over the waves.  No atomics: results are deterministic.
#pragma once
#include <type_traits>

#include "common.hpp"

namespace incvit {

constexpr int kGemmWaves = 8;
constexpr int kGemmRB = 32;                       // rows per block: two 16-row MFMA tiles

// GELU, tanh form, with tanh(u) = 1 - 2 / (1 + e^(2u)) on the hardware
// exponential (error a few fp32 ulps, far below the bf16 rounding that
// follows; the limits u -> +-inf give +-1).
__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  const float t = 1.0f - __fdividef(2.0f, 1.0f + __expf(2.0f * u));
  return 0.5f * x * (1.0f + t);
}

template <int EPI>
__host__ __device__ constexpr bool has_resid() {
  return EPI == EPI_RES || EPI == EPI_DOWN;
}
template <int EPI>
__host__ __device__ constexpr bool has_rows() {
  return EPI == EPI_QKV || EPI == EPI_ATT || EPI == EPI_DOWN;
}
template <int EPI>
__host__ __device__ constexpr bool ln_on_load() {
  return EPI == EPI_QKV || EPI == EPI_FC1;
}
template <int EPI>
__host__ __device__ constexpr int gemm_waves() {
  return kGemmWaves;
}
template <int NB, int NW>
__host__ __device__ constexpr int gemm_red_bytes() {
  return NW * 2 * NB * 64 * 16;
}
// LDS: the wave partial tiles; with LayerNorm folding, then the waves' row
// partials [NW][32] (sum, sum of squares) and the rows' shifts [32]
template <int EPI, int NB>
__host__ __device__ constexpr int gemm_lds_bytes() {
  constexpr int NW = gemm_waves<EPI>();
  return gemm_red_bytes<NB, NW>() + (ln_on_load<EPI>() ? NW * kGemmRB * 8 + kGemmRB * 4 : 0);
}

// an operand fragment of all ones (B of the row-sum product)
__device__ __forceinline__ void ones(V8<uint16_t>& v) { v.v = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u); }
__device__ __forceinline__ void ones(V8<float>& v) { v.a = make_float4(1.0f, 1.0f, 1.0f, 1.0f); v.b = v.a; }

__device__ __forceinline__ float elem4(const f32x4_t& v, int i) {
  return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}

// One output element of a GEMM, x = the fp32 product over the whole K (or,
// for PART, over this workgroup's share of K) at (row, col) with row < M:
// bias, the folded LayerNorm (rstd, nmr = -mean * rstd of the row; QKV, FC1),
// the residual element (RES, DOWN), the row's map entry (QKV, ATT, DOWN), and
// the K split (PART).  Every operation's result is rounded to the storage type
// once, as a half-precision pipeline stores it.
template <class T, int EPI>
__device__ __forceinline__ void epilogue_store(const GemmArgs& a, int row, int col, float x, float bias, float c1,
                                               float resid, float rstd, float nmr, const RowInfo& rinfo, int ks) {
  const int D = a.sh.D;
  if constexpr (EPI == EPI_PART) {
    static_cast<float*>(a.out)[((size_t)ks * a.mpad + row) * a.ldo + col] = x;
  } else if constexpr (EPI == EPI_RES) {  // H = S(Z + S(O W_o + b_o))
    static_cast<T*>(a.out)[frag_off(row, col, a.ldo / 32)] = Elem<T>::cv(resid + Elem<T>::rnd(x + bias));
  } else if constexpr (EPI == EPI_DOWN) {  // Z_{l+1} = S(H + S(G W_2 + b_2))
    const T z = Elem<T>::cv(resid + Elem<T>::rnd(x + bias));
    static_cast<T*>(a.out)[frag_off(row, col, a.ldo / 32)] = z;
    gbl(x_row<T>(rinfo.cache, a.cl, a.sh, a.layer + 1, rinfo.tok))[col] = z;
  } else if constexpr (EPI == EPI_ATT) {  // A^l[tok] = S(O W_o + b_o)
    T* arow = reinterpret_cast<T*>(rinfo.cache + a.cl.a + (size_t)a.layer * a.cl.x_layer);
    gbl(arow)[(size_t)rinfo.tok * D + col] = Elem<T>::cv(x + bias);
  } else if constexpr (EPI == EPI_QKV) {  // [Q K V] = S(LN1(Z) W_qkv + b), K and V into the cache
    const T o = Elem<T>::cv(fmaf(rstd, x, fmaf(nmr, c1, bias)));
    const int which = col / D, c = col - which * D;
    if (which == 0) {
      static_cast<T*>(a.out)[(size_t)row * a.ldo + c] = o;
    } else {
      const int hh = c / a.sh.dh, d = c - hh * a.sh.dh;
      char* base = rinfo.cache + (which == 1 ? a.cl.k : a.cl.v) + (size_t)a.layer * a.cl.kv_layer;
      const size_t e = which == 1 ? k_elem(a.sh, hh, rinfo.tok, d) : v_elem(a.sh, hh, rinfo.tok, d);
      gbl(reinterpret_cast<T*>(base))[e] = o;
    }
  } else {  // EPI_FC1: G = S(GELU(S(LN2(H) W_1 + b_1)))
    const float f = fmaf(rstd, x, fmaf(nmr, c1, bias));
    static_cast<T*>(a.out)[frag_off(row, col, a.ldo / 32)] = Elem<T>::cv(gelu_tanh(Elem<T>::rnd(f)));
  }
}

template <class T, int EPI, int NB, int CPW>
__global__ __launch_bounds__(gemm_waves<EPI>() * 64) void gemm_kernel(GemmArgs a) {
  constexpr int NW = gemm_waves<EPI>();
  constexpr bool LNA = ln_on_load<EPI>();
  extern __shared__ __align__(16) char smem[];
  f32x4_t* red = reinterpret_cast<f32x4_t*>(smem);                          // [NW][2][NB][64]
  float2* s_ps = reinterpret_cast<float2*>(smem + gemm_red_bytes<NB, NW>());  // [NW][32] (sum, sumsq)
  float* s_shift = reinterpret_cast<float*>(s_ps + NW * kGemmRB);              // [32] (fp32 models)
  constexpr bool SHIFT = LNA && std::is_same<T, float>::value;  // shifted row statistics

  const int tid = threadIdx.x, lane = tid & 63;
  // w lives in a scalar register, so every guard that depends on it is a
  // scalar branch: an MFMA must never run under a partial or empty lane mask
  // (it would still accumulate)
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, n = lane & 15;
  const int D = a.sh.D;
  // (column group, K split, row group) of this workgroup, XCD-major; the
  // grid's shape comes from the arguments (no load of the dispatch packet)
  const int nz = a.rgroups, ny = a.ksplit, nx = a.Nout / 16 / NB;
  int zg = 0, ks = blockIdx.y, cg = blockIdx.x;  // one row group, one K range: launch order
  if (nz > 1 || ny > 1) {                         // uniform
    const int total = nx * ny * nz;
    const int lin = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
    const int xcd = lin % 8, per = total / 8, rem = total % 8;
    const int pos = xcd * per + min(xcd, rem) + lin / 8;
    if (nz > 1) {  // the row groups of a column block together: its weights once per XCD
      zg = pos % nz;
      ks = (pos / nz) % ny;
      cg = pos / (nz * ny);
    } else {  // K ranges apart: an XCD reads about one range of A (nothing else is shared)
      ks = pos / nx;
      cg = pos % nx;
    }
  }
  if (zg > 0) {  // a later row group reads M first and leaves when it has no rows (uniform)
    if (zg * kGemmRB >= *static_cast<const volatile int*>(&a.meta->m)) return;
  }
  const int M = a.meta->m;
  const int cb0 = cg * NB;
  // this workgroup's share of K: chunks [kb, kb + kn)
  const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
  const int kb = ks * kper, kn = min(kper, a.kchunks - kb);
  const int kc_last = kn - 1;
  const int rounds = (kn + NW * CPW - 1) / (NW * CPW);

  auto kc_of = [&](int round, int c) { return kb + min((round * NW + w) * CPW + c, kc_last); };
  V8<T> ab[CPW][2];
  V8<T> wb[CPW][NB];
  // A is stored in operand order (frag_off): row tile t, chunk kc is the
  // kilobyte (t * akc + kc) (bf16; two kilobytes for fp32)
  const int akc = a.lda / 32;
  const Rsrc rA = make_rsrc(a.A, (uint32_t)a.mpad * a.lda * sizeof(T));
  const Rsrc rW = make_rsrc(a.W, (uint32_t)(a.Nout / 16) * a.kchunks * kChunkElems * sizeof(T));
  const uint32_t voff = lane * 8 * sizeof(T);
  float shv[2] = {0.0f, 0.0f};  // SHIFT: the first element of row 16 r + n of the block
  auto load_a = [&](int m0, int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int r = 0; r < 2; ++r)
        ab[c][r].bload(rA, voff, (uint32_t)(((m0 >> 4) + r) * akc + kc_of(round, c)) * kChunkElems * sizeof(T));
    if constexpr (SHIFT) {
      if (round == 0) {
#pragma unroll
        for (int r = 0; r < 2; ++r) shv[r] = static_cast<const float*>(a.A)[frag_off(m0 + 16 * r + n, 0, akc)];
      }
    }
  };
  auto load_w = [&](int round) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int b = 0; b < NB; ++b)
        wb[c][b].bload(rW, voff, (uint32_t)((cb0 + b) * a.kchunks + kc_of(round, c)) * kChunkElems * sizeof(T));
  };
  // epilogue item of this wave: row tile w/4, row 4g + (w%4) of the tile
  const int re = w >> 2, ie = w & 3;
  RowInfo rinfo = RowInfo{nullptr, 0, 0};
  float biasv[NB], resv[NB], c1v[NB];
  auto load_res = [&](int m0) {  // the residual Z rows (operand order)
#pragma unroll
    for (int b = 0; b < NB; ++b)
      resv[b] = Elem<T>::f(
          static_cast<const T*>(a.resid)[frag_off(m0 + 16 * re + 4 * g + ie, (cb0 + b) * 16 + n, D / 32)]);
  };

  // the first row group runs whatever M is (with M = 0 it stores nothing),
  // so its loads are never held back behind the read of M
  const int mfirst = zg * kGemmRB, mstep = nz * kGemmRB;
  load_a(mfirst, 0);
  load_w(0);
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    biasv[b] = EPI == EPI_PART ? 0.0f : a.bias[(cb0 + b) * 16 + n];  // DOWN: b_2
    c1v[b] = LNA ? a.c1[(cb0 + b) * 16 + n] : 0.0f;
  }
  if constexpr (has_rows<EPI>()) rinfo = a.rows[mfirst + 16 * re + 4 * g + ie];
  if constexpr (has_resid<EPI>()) load_res(mfirst);

  // One 32-row block.  The group's first block is a copy of its own (FIRST),
  // so its waits count exactly the loads issued above instead of the fewer a
  // later block reloads (the weights stay in registers).
  auto row_block = [&](const int m0, auto first) {
    if constexpr (!decltype(first)::value) {
      if (rounds > 1) {  // with one round the A fragments were loaded ahead (below)
        load_a(m0, 0);
        load_w(0);
      }
      if constexpr (has_rows<EPI>()) rinfo = a.rows[m0 + 16 * re + 4 * g + ie];
      if constexpr (has_resid<EPI>()) load_res(m0);
    }
    f32x4_t acc[2][NB], accs[2], accq[2];  // accs, accq: row sums and sums of squares (LNA)
    float vsu[2] = {0.0f, 0.0f}, vsq[2] = {0.0f, 0.0f};  // SHIFT: this lane's sums of x - x_0
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      accs[r] = accq[r] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[r][b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    }
    V8<T> one;
    ones(one);

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
          for (int r = 0; r < 2; ++r) {
#pragma unroll
            for (int b = 0; b < NB; ++b) mma(acc[r][b], ab[c][r], wb[c][b]);
            if constexpr (SHIFT) {  // lane (g, n): row n, k = 8g..8g+7 of the chunk, in k order
              const float xv[8] = {ab[c][r].a.x, ab[c][r].a.y, ab[c][r].a.z, ab[c][r].a.w,
                                   ab[c][r].b.x, ab[c][r].b.y, ab[c][r].b.z, ab[c][r].b.w};
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const float d = xv[j] - shv[r];
                vsu[r] += d;
                vsq[r] = fmaf(d, d, vsq[r]);
              }
            } else if constexpr (LNA) {
              mma(accs[r], ab[c][r], one);
              mma(accq[r], ab[c][r], ab[c][r]);
            }
          }
        }
      }
    }
    // One round: the weights stay in registers and the A fragments are free
    // once the products are issued, so the group's next row block loads its A
    // now, behind this block's reduction and epilogue (uniform branch).  The
    // shifts of this block are kept first (the preload replaces them).
    const float shcur[2] = {shv[0], shv[1]};
    if (rounds == 1 && m0 + mstep < M) load_a(m0 + mstep, 0);

    // ---- sum the waves' partial tiles in wave order
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int b = 0; b < NB; ++b) red[((w * 2 + r) * NB + b) * 64 + lane] = acc[r][b];
    if constexpr (SHIFT) {
      // the four lanes of row n (g = 0..3) combined in a fixed order
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        vsu[r] += __shfl_xor(vsu[r], 16, 64);
        vsq[r] += __shfl_xor(vsq[r], 16, 64);
        vsu[r] += __shfl_xor(vsu[r], 32, 64);
        vsq[r] += __shfl_xor(vsq[r], 32, 64);
        if (g == 0) {
          s_ps[w * kGemmRB + 16 * r + n] = make_float2(vsu[r], vsq[r]);
          if (w == 0) s_shift[16 * r + n] = shcur[r];
        }
      }
    } else if constexpr (LNA) {
      // lane (g, n) holds rows 4g..4g+3 of column n: row n's sum (any column)
      // and its sum of squares (the diagonal) sit in element n - 4g
      const int i = n - 4 * g;
      if (i >= 0 && i < 4) {
#pragma unroll
        for (int r = 0; r < 2; ++r) s_ps[w * kGemmRB + 16 * r + n] = make_float2(elem4(accs[r], i), elem4(accq[r], i));
      }
    }
    __syncthreads();

    // ---- epilogue: wave w < 8 finishes row 4g + (w%4) of row tile w/4
    const float* redf = reinterpret_cast<const float*>(red);
    const int row = m0 + 16 * re + 4 * g + ie;
    const bool ok = row < M;
    float rstd = 0.0f, nmr = 0.0f;  // LNA: rstd and -mean * rstd of the row
    if constexpr (LNA) {
      float su = 0.0f, sq = 0.0f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) {
        const float2 p = s_ps[ww * kGemmRB + 16 * re + 4 * g + ie];
        su += p.x;
        sq += p.y;
      }
      float mean = su / (float)D;
      const float var = fmaxf(sq / (float)D - mean * mean, 0.0f);
      if constexpr (SHIFT) mean += s_shift[16 * re + 4 * g + ie];  // the sums were of x - x_0
      rstd = 1.0f / sqrtf(var + a.sh.eps);
      nmr = -mean * rstd;
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (w >= kGemmWaves) break;  // a scalar branch
      const int col = (cb0 + b) * 16 + n;
      float x = 0.0f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) x += redf[(((ww * 2 + re) * NB + b) * 64 + lane) * 4 + ie];
      if (ok) epilogue_store<T, EPI>(a, row, col, x, biasv[b], c1v[b], resv[b], rstd, nmr, rinfo, ks);
    }
    __syncthreads();  // red and the row partials are reused by the next row block
  };
  row_block(mfirst, std::true_type{});
  for (int m0 = mfirst + mstep; m0 < M; m0 += mstep) row_block(m0, std::false_type{});
}

template <class T, int EPI, int NB, int CPW>
hipError_t launch_gemm_cfg(const GemmArgs& a, hipStream_t s) {
  constexpr int lds = gemm_lds_bytes<EPI, NB>();
  if constexpr (lds > 65536) {  // four column blocks: the partial tiles exceed the default 64 KB
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, EPI, NB, CPW>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (attr != hipSuccess) return attr;
  }
  return launch_k(gemm_kernel<T, EPI, NB, CPW>, dim3(a.Nout / 16 / NB, a.ksplit, a.rgroups),
                  dim3(gemm_waves<EPI>() * 64), (size_t)lds, s, a);
}

// Chunks per wave: the smallest instantiated count that covers this
// workgroup's share of K in one round (the last wave may own fewer); longer
// shares run in rounds of the largest (8, or 6 for four column blocks).
template <class T, int EPI, int NB>
hipError_t launch_gemm_nb(int cpw, const GemmArgs& a, hipStream_t s) {
  if (cpw <= 1) return launch_gemm_cfg<T, EPI, NB, 1>(a, s);
  if (cpw <= 2) return launch_gemm_cfg<T, EPI, NB, 2>(a, s);
  if (cpw <= 3) return launch_gemm_cfg<T, EPI, NB, 3>(a, s);
  if (cpw <= 4) return launch_gemm_cfg<T, EPI, NB, 4>(a, s);
  if (cpw <= 5) return launch_gemm_cfg<T, EPI, NB, 5>(a, s);
  // four column blocks hold at most 6 chunks per wave in registers (8 spill)
  if (cpw <= 6 || NB == 4) return launch_gemm_cfg<T, EPI, NB, 6>(a, s);
  if constexpr (NB != 4) return launch_gemm_cfg<T, EPI, NB, 8>(a, s);
  return hipErrorInvalidValue;
}

// cols: 16-column blocks per workgroup, 1, 2 or 4 (4: bf16 only, fp32 takes
// 2: its operands would not fit the registers); a count that does not divide
// the output's blocks falls back to fewer.
template <int EPI>
hipError_t launch_gemm_epi(int cols, const GemmArgs& a, hipStream_t s) {
  const int nb = a.Nout / 16;
  int c = cols >= 4 && nb % 4 == 0 ? 4 : cols >= 2 && nb % 2 == 0 ? 2 : 1;
  if (c == 4 && !a.sh.dtype) c = nb % 2 == 0 ? 2 : 1;
  const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
  const int cpw = std::min((kper + gemm_waves<EPI>() - 1) / gemm_waves<EPI>(), 8);
  // the folded LayerNorm needs the whole K range in one workgroup
  if (ln_on_load<EPI>() && a.ksplit != 1) return hipErrorInvalidValue;
  if (a.sh.dtype) {
    if (c == 4) return launch_gemm_nb<uint16_t, EPI, 4>(cpw, a, s);
    return c == 2 ? launch_gemm_nb<uint16_t, EPI, 2>(cpw, a, s) : launch_gemm_nb<uint16_t, EPI, 1>(cpw, a, s);
  }
  return c == 2 ? launch_gemm_nb<float, EPI, 2>(cpw, a, s) : launch_gemm_nb<float, EPI, 1>(cpw, a, s);
}

}  // namespace incvit
