// Large-M GEMM of the encoder layers (paper §III-B: the QKV, output
// projection and MLP products, eqs. 4-5), for calls whose row count M is known
// on the host and large: full encodes, top-k steps of several hundred rows and
// the all-rows MLP.  The small-M kernel (gemm.hpp) streams the weights once
// and re-reads the few A rows per 16-64 columns; here each workgroup stages a
// tile of A rows and of W columns through LDS once per K chunk and all its
// waves multiply from there (the staging, at 13-26 bytes per clock per CU
// from L2, sets the pace):
//
//   * output tile BM x 128 per workgroup, 4 waves in a WR x WC grid, each
//     wave owning (BM / WR) x (128 / WC) outputs as 16x16 MFMA accumulators
//     (v_mfma_f32_16x16x32_bf16, fp32 accumulation);
//   * the K loop runs over 32-deep chunks.  A chunk's operands are BM / 16 A
//     fragments and 8 W fragments, each a contiguous kilobyte in HBM (the
//     compact rows and the packed weights are stored in MFMA operand order),
//     so one wave instruction (global_load_lds_dwordx4: 16 bytes per lane
//     straight into LDS, no registers) stages one fragment.  A ring of NS
//     chunk slots keeps NS - 1 chunks in flight while one is multiplied; one
//     barrier per chunk;
//   * the folded LayerNorm (QKV, MLP up) takes its row statistics on the
//     matrix cores from the staged A fragments (x * ones and the diagonal of
//     x * x^T), each wave for a quarter of the row tiles, combined in a fixed
//     order;
//   * the epilogue applies the small-M kernel's operations (bias, the
//     LayerNorm fold, residual, GELU, rounding points and scatters), with
//     every address split into a row part and a column part formed once;
//   * each XCD takes a compact block of about sqrt(tiles / 8) row tiles by as
//     many column tiles, so its workgroups share their A and W tiles in its
//     L2 (the hardware deals workgroups to the XCDs round robin);
//   * partial sums (the MLP down projection while its tiles are fewer than
//     the CUs) may split K over the grid's third dimension: split z takes a
//     contiguous range of chunks and writes its fp32 partial sums, which the
//     row kernel adds in split order.
//
// bf16 models only (fp32 models use the small-M kernel).  Results do not
// depend on the tile shape beyond the fp32 order of the MFMA accumulation,
// which is fixed (k ascending); no atomics.
#pragma once
#include "gemm.hpp"

namespace incvit {

constexpr int kTiledBN = 128;   // output columns per workgroup (8 blocks of 16)

// LDS: the ring of NS chunk slots, reused after the K loop for the
// epilogue's fp32 tiles (4 waves x rows x (columns + 4)), then the row
// statistics [BM] x 2 float2.
template <int BM, int NS>
__host__ __device__ constexpr int tiled_stage_bytes() {
  constexpr int ring = NS * (BM / 16 + kTiledBN / 16) * 1024;
  constexpr int WR = BM == 128 ? 2 : 1;
  constexpr int tile = 4 * (BM / WR) * (kTiledBN / (4 / WR) + 4) * 4;
  return ring > tile ? ring : tile;
}
template <int BM, int NS>
__host__ __device__ constexpr int tiled_lds_bytes() {
  return tiled_stage_bytes<BM, NS>() + BM * 16;
}

template <int EPI, int BM, int NS>
__global__ __launch_bounds__(256) void gemm_tiled_kernel(GemmArgs a) {
  using T = uint16_t;
  constexpr int TRB = BM / 16, CBB = kTiledBN / 16;  // row tiles, column blocks per workgroup
  constexpr int FPC = TRB + CBB;                     // fragments per chunk
  static_assert(FPC % 4 == 0, "fragments of a chunk split evenly over the waves");
  constexpr int LPW = FPC / 4;                       // fragment loads per wave per chunk
  constexpr int WR = BM == 128 ? 2 : 1, WC = 4 / WR;
  constexpr int TR = TRB / WR, TC = CBB / WC;        // per wave
  constexpr bool LNA = ln_on_load<EPI>();
  constexpr int SR = TRB / 4;                        // statistics row tiles per wave (LNA)
  static_assert(!LNA || TRB % 4 == 0, "statistics row tiles split evenly over the waves");
  extern __shared__ __align__(16) char smem[];
  char* ring = smem;  // [NS][FPC][1 KB]; after the K loop the epilogue's tiles
  float2* s_ps = reinterpret_cast<float2*>(smem + tiled_stage_bytes<BM, NS>());  // [BM] (sum, sum of squares)
  float2* s_ln = s_ps + BM;                                                       // [BM] (rstd, -mean * rstd)

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, n = lane & 15;
  const int wr = w / WC, wc = w % WC;
  const int D = a.sh.D;
  // tile of this workgroup.  The hardware deals workgroups to the 8 XCDs
  // round robin; each XCD is given a contiguous range of positions in a
  // grouped order (groups of GM row tiles, column-major inside a group), so
  // that its tiles form a compact GM x (range / GM) block whose A row tiles
  // and W column tiles fit its L2 together (the host picks GM).
  const int mt = gridDim.x, nt = gridDim.y;
  const int total = mt * nt;
  const int lin = blockIdx.x + mt * blockIdx.y;
  const int xcd = lin % 8, per = total / 8, rem = total % 8;
  const int pos = xcd * per + min(xcd, rem) + lin / 8;
  const int GM = a.rgroups;
  const int grp = pos / (GM * nt), inside = pos - grp * GM * nt;
  const int gm = min(GM, mt - grp * GM);
  const int m0 = (grp * GM + inside % gm) * BM, cb0 = (inside / gm) * CBB;
  const int M = a.meta->m;
  if (m0 >= M) return;  // uniform: no rows in this tile
  const int nblocks = a.Nout / 16, kchunks = a.kchunks, akc = a.lda / 32;
  // K split (partial sums only): split ks takes chunks kbeg .. kbeg + nk - 1
  const int ks = blockIdx.z;
  const int kper = (kchunks + (int)gridDim.z - 1) / (int)gridDim.z;
  const int kbeg = ks * kper, nk = min(kchunks - kbeg, kper);

  // operand fragments of chunk kc: A row tile t is kilobyte (m0/16 + t) * akc + kc
  // of the compact rows, W column block b is kilobyte (cb0 + b) * kchunks + kc
  // of the packed weights; fragment f of a chunk goes to slot offset f KB.
  // Wave w stages fragments w, w + 4, ...: with TRB a multiple of 4 the first
  // TRB / 4 of them are A fragments.  Every wave issues exactly LPW loads per
  // chunk (the wait counts rely on it): a fragment past its operand's end
  // loads the weights' first kilobyte instead, whose products only reach
  // outputs that are never stored.
  const char* gA = static_cast<const char*>(a.A);
  const char* gW = static_cast<const char*>(a.W);
  const uint32_t a_frags = (uint32_t)(a.mpad / 16) * akc;  // kilobytes of A
  auto issue = [&](int i) {  // chunk kbeg + i into ring slot i % NS
    const int kc = kbeg + i;
    char* slot = ring + (i % NS) * FPC * 1024;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int f = w + 4 * j;  // uniform
      const char* src;
      if (j < TRB / 4) {
        const uint32_t fr = (uint32_t)(m0 / 16 + f) * akc + kc;
        src = fr < a_frags ? gA + (size_t)fr * 1024 : gW;
      } else {
        const int cb = cb0 + f - TRB;
        src = cb < nblocks ? gW + ((size_t)cb * kchunks + kc) * 1024 : gW;
      }
      __builtin_amdgcn_global_load_lds((const INCVIT_GLOBAL void*)(src + lane * 16),
                                       (__attribute__((address_space(3))) void*)(slot + f * 1024), 16, 0, 0);
    }
  };

  f32x4_t acc[TR][TC], accs[SR > 0 ? SR : 1], accq[SR > 0 ? SR : 1];
#pragma unroll
  for (int t = 0; t < TR; ++t)
#pragma unroll
    for (int b = 0; b < TC; ++b) acc[t][b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int t = 0; t < (SR > 0 ? SR : 1); ++t) accs[t] = accq[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  V8<T> one;
  ones(one);
  // LDS byte addresses of this lane's 16 bytes in the fragments it multiplies
  const uint32_t ring_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)ring;
  const uint32_t offA = (uint32_t)(wr * TR) * 1024 + lane * 16;
  const uint32_t offB = (uint32_t)(TRB + wc * TC) * 1024 + lane * 16;
  const uint32_t offS = (uint32_t)w * 1024 + lane * 16;  // statistics row tiles w, w + 4

  // One chunk's products: the fragments of the chunk in ring slot sb (LDS
  // byte address) are read with explicit LDS reads and an explicit wait (the
  // compiler would otherwise wait for every outstanding LDS-bound load, as it
  // cannot tell the slots apart, and empty the pipeline).
  auto compute = [&](uint32_t sb) {
    u32x4_t af[TR], bf[TC], sf[SR > 0 ? SR : 1];
#pragma unroll
    for (int t = 0; t < TR; ++t) lds_read16(af[t], sb + offA, t * 1024);
#pragma unroll
    for (int b = 0; b < TC; ++b) lds_read16(bf[b], sb + offB, b * 1024);
    if constexpr (LNA) {
#pragma unroll
      for (int t = 0; t < SR; ++t) lds_read16(sf[t], sb + offS, 4 * t * 1024);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int t = 0; t < TR; ++t) asm volatile("" : "+v"(af[t]));
#pragma unroll
    for (int b = 0; b < TC; ++b) asm volatile("" : "+v"(bf[b]));
#pragma unroll
    for (int t = 0; t < TR; ++t) {
      V8<T> x;
      x.v = __builtin_bit_cast(uint4, af[t]);
#pragma unroll
      for (int b = 0; b < TC; ++b) {
        V8<T> y;
        y.v = __builtin_bit_cast(uint4, bf[b]);
        mma(acc[t][b], x, y);
      }
    }
    if constexpr (LNA) {
#pragma unroll
      for (int t = 0; t < SR; ++t) {
        asm volatile("" : "+v"(sf[t]));
        V8<T> x;
        x.v = __builtin_bit_cast(uint4, sf[t]);
        mma(accs[t], x, one);
        mma(accq[t], x, x);
      }
    }
  };

  // The K loop over the split's chunks (kc counts from kbeg): chunk kc sits
  // in ring slot kc % NS; NS - 1 chunks are in
  // flight while one is multiplied, one barrier per chunk (two chunks per
  // barrier with NS - 2 in flight measured slower: the loads' latency, not
  // the barriers, sets the pace).
#pragma unroll
  for (int c = 0; c < NS - 1; ++c)
    if (c < nk) issue(c);
  for (int kc = 0; kc < nk; ++kc) {
    // chunk kc has landed once at most the loads of the chunks issued after
    // it are outstanding (loads complete in issue order)
    if (kc + NS - 2 < nk) __builtin_amdgcn_s_waitcnt(vmcnt_imm(LPW * (NS - 2)));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    // every wave's fragments of chunk kc are in LDS; every wave is done with
    // chunk kc - 1, whose slot the next issue refills
    __builtin_amdgcn_s_barrier();
    if (kc + NS - 1 < nk) issue(kc + NS - 1);
    compute(ring_lds + (uint32_t)(kc % NS) * FPC * 1024);
  }
  __syncthreads();

  // ---- LayerNorm statistics of the block's rows (row tile w + 4t is this wave's)
  if constexpr (LNA) {
    const int i = n - 4 * g;
    if (i >= 0 && i < 4) {
#pragma unroll
      for (int t = 0; t < SR; ++t) s_ps[16 * (w + 4 * t) + n] = make_float2(elem4(accs[t], i), elem4(accq[t], i));
    }
    __syncthreads();
    if (tid < BM) {
      const float2 p = s_ps[tid];
      const float mean = p.x / (float)D;
      const float var = fmaxf(p.y / (float)D - mean * mean, 0.0f);
      const float rstd = 1.0f / sqrtf(var + a.sh.eps);
      s_ln[tid] = make_float2(rstd, -mean * rstd);
    }
    __syncthreads();
  }

  // ---- epilogue.  Each wave stages its (16 TR) x (16 TC) fp32 outputs
  // through LDS (row-major, rows padded by 4 floats against bank conflicts),
  // so that lane l then finishes 8 consecutive columns (column group l % CG)
  // of rows l / CG, l / CG + 64 / CG, ...: 16-byte residual loads and 16-byte
  // stores (the operand-order and row-major outputs keep 8 consecutive
  // columns of a row contiguous), the column parts of every address formed
  // once.  Operations and rounding points are the small-M kernel's
  // (epilogue_store).
  constexpr int RW = 16 * TR, CW = 16 * TC, CG = CW / 8, RPL = RW * CG / 64;  // rows per lane
  constexpr int LDT = CW + 4;                                                  // floats per staged row
  float* stile = reinterpret_cast<float*>(smem) + w * RW * LDT;
#pragma unroll
  for (int t = 0; t < TR; ++t)
#pragma unroll
    for (int b = 0; b < TC; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) stile[(16 * t + 4 * g + i) * LDT + 16 * b + n] = elem4(acc[t][b], i);
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");

  const int cgi = lane % CG;
  const int col0 = (cb0 + wc * TC) * 16 + 8 * cgi;  // first of this lane's 8 columns
  const bool colok = col0 < a.Nout;                // 8-column groups never straddle the end (Nout % 16 == 0)
  const int ldk = a.ldo / 32;
  float biasv[8], c1v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int col = colok ? col0 + j : 0;
    biasv[j] = EPI == EPI_PART ? 0.0f : a.bias[col];
    c1v[j] = LNA ? a.c1[col] : 0.0f;
  }
  size_t cpart = 0;
  int which = 0;
  if constexpr (EPI == EPI_QKV) {
    const int c = col0 - (col0 / D) * D;
    const int hh = c / a.sh.dh, d = c - hh * a.sh.dh;  // d % 8 == 0: the 8 columns stay in one head
    which = col0 / D;
    cpart = which == 0 ? (size_t)c : which == 1 ? k_col(a.sh, hh, d) : v_col(a.sh, hh, d);
  } else if constexpr (EPI == EPI_RES || EPI == EPI_DOWN || EPI == EPI_FC1) {
    cpart = frag_col(col0);
  } else {
    cpart = (size_t)col0;
  }
  if (colok) {
#pragma unroll
    for (int q = 0; q < RPL; ++q) {
      const int rw = lane / CG + q * (64 / CG);  // row within the wave's tile
      const int rl = wr * RW + rw;               // row within the workgroup's tile
      const int row = m0 + rl;
      if (row >= M) continue;
      float x[8];
      const float4 lo = *reinterpret_cast<const float4*>(stile + rw * LDT + 8 * cgi);
      const float4 hi = *reinterpret_cast<const float4*>(stile + rw * LDT + 8 * cgi + 4);
      x[0] = lo.x; x[1] = lo.y; x[2] = lo.z; x[3] = lo.w;
      x[4] = hi.x; x[5] = hi.y; x[6] = hi.z; x[7] = hi.w;
      RowInfo rinfo = RowInfo{nullptr, 0, 0};
      if constexpr (has_rows<EPI>()) rinfo = a.rows[row];
      const size_t rpart = frag_row(row, ldk);
      float o[8];
      if constexpr (EPI == EPI_PART) {
        float4* dst =
            reinterpret_cast<float4*>(static_cast<float*>(a.out) + ((size_t)ks * a.mpad + row) * a.ldo + cpart);
        dst[0] = lo;
        dst[1] = hi;
        continue;
      } else if constexpr (EPI == EPI_RES || EPI == EPI_DOWN) {  // S(resid + S(x + b))
        const uint4 rv = *reinterpret_cast<const uint4*>(static_cast<const T*>(a.resid) + rpart + cpart);
        const uint32_t rw4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float res = __uint_as_float(j & 1 ? rw4[j >> 1] & 0xffff0000u : rw4[j >> 1] << 16);
          o[j] = res + Elem<T>::rnd(x[j] + biasv[j]);
        }
      } else if constexpr (EPI == EPI_ATT) {
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = x[j] + biasv[j];
      } else if constexpr (EPI == EPI_QKV) {
        float rstd = 0.0f, nmr = 0.0f;
        const float2 st = s_ln[rl];
        rstd = st.x;
        nmr = st.y;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = fmaf(rstd, x[j], fmaf(nmr, c1v[j], biasv[j]));
      } else {  // EPI_FC1
        const float2 st = s_ln[rl];
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = gelu_tanh(Elem<T>::rnd(fmaf(st.x, x[j], fmaf(st.y, c1v[j], biasv[j]))));
      }
      const uint4 ov = make_uint4(f2bf2(o[0], o[1]), f2bf2(o[2], o[3]), f2bf2(o[4], o[5]), f2bf2(o[6], o[7]));
      const u32x4_t ovv = __builtin_bit_cast(u32x4_t, ov);
      if constexpr (EPI == EPI_RES || EPI == EPI_DOWN || EPI == EPI_FC1) {
        *reinterpret_cast<uint4*>(static_cast<T*>(a.out) + rpart + cpart) = ov;
        if constexpr (EPI == EPI_DOWN)
          *gbl(reinterpret_cast<u32x4_t*>(x_row<T>(rinfo.cache, a.cl, a.sh, a.layer + 1, rinfo.tok) + col0)) = ovv;
      } else if constexpr (EPI == EPI_ATT) {
        T* arow = reinterpret_cast<T*>(rinfo.cache + a.cl.a + (size_t)a.layer * a.cl.x_layer) + (size_t)rinfo.tok * D;
        *gbl(reinterpret_cast<u32x4_t*>(arow + cpart)) = ovv;
      } else if constexpr (EPI == EPI_QKV) {
        if (which == 0) {
          *reinterpret_cast<uint4*>(static_cast<T*>(a.out) + (size_t)row * a.ldo + cpart) = ov;
        } else if (which == 1) {  // K: 8 consecutive dims are 8 contiguous elements
          T* kb = reinterpret_cast<T*>(rinfo.cache + a.cl.k + (size_t)a.layer * a.cl.kv_layer);
          *gbl(reinterpret_cast<u32x4_t*>(kb + k_tok(a.sh, rinfo.tok) + cpart)) = ovv;
        } else {  // V (transposed): consecutive dims are 8 elements apart
          T* vb = reinterpret_cast<T*>(rinfo.cache + a.cl.v + (size_t)a.layer * a.cl.kv_layer) + v_tok(a.sh, rinfo.tok) + cpart;
#pragma unroll
          for (int j = 0; j < 8; ++j) gbl(vb)[8 * j] = f2bf(o[j]);
        }
      }
    }
  }
}

template <int EPI, int BM, int NS>
hipError_t launch_tiled_cfg(const GemmArgs& a, int rows, hipStream_t s) {
  constexpr int lds = tiled_lds_bytes<BM, NS>();
  if constexpr (lds > 65536) {
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_tiled_kernel<EPI, BM, NS>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (attr != hipSuccess) return attr;
  }
  const int mt = (rows + BM - 1) / BM, nt = (a.Nout / 16 + kTiledBN / 16 - 1) / (kTiledBN / 16);
  // row tiles per group: about the square root of one XCD's share of tiles
  // (A and W tiles of a workgroup are the same size), at most mt
  GemmArgs b = a;
  const int per_xcd = (mt * nt + 7) / 8;
  int gm = 1;
  while ((gm + 1) * (gm + 1) <= per_xcd) ++gm;
  b.rgroups = std::max(1, std::min(gm, mt));
  return launch_k(gemm_tiled_kernel<EPI, BM, NS>, dim3(mt, nt, a.ksplit), dim3(256), (size_t)lds, s, b);
}

// rows: the call's row count M (known on the host); bf16 only.  The K split
// (a.ksplit > 1) only for partial sums, each split at least one chunk.
// 128-row tiles once they give a workgroup per CU or more, 64-row tiles below.
template <int EPI>
hipError_t launch_tiled_epi(const GemmArgs& a, int rows, hipStream_t s) {
  if (!a.sh.dtype || a.ksplit < 1 || a.sh.dh % 8) return hipErrorInvalidValue;
  if (a.ksplit > 1) {
    const int kper = (a.kchunks + a.ksplit - 1) / a.ksplit;
    if (EPI != EPI_PART || kper * (a.ksplit - 1) >= a.kchunks) return hipErrorInvalidValue;
  }
  const int ntile = (a.Nout / 16 + kTiledBN / 16 - 1) / (kTiledBN / 16);
  if ((rows + 127) / 128 * ntile * a.ksplit >= 256) return launch_tiled_cfg<EPI, 128, 4>(a, rows, s);
  return launch_tiled_cfg<EPI, 64, 6>(a, rows, s);
}

}  // namespace incvit
