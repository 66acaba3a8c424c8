// Attention of the refreshed queries over all N cached keys of their stream
// (paper §III-B: attention is computed only for the updated tokens; the keys
// and values are the scattered full K/V -- new rows for U, cached rows for R).
//
// Per block of 32 keys and tile of 16 queries a wave forms S^T = K Q^T with
// MFMA (so each lane keeps a single query and its softmax state), updates the
// online softmax in fp32 (exp2 with the 1/sqrt(d_h) scale folded in), and
// accumulates O^T = V^T P^T with MFMA.  K and V are cached in operand order
// (transposed V), with a key order that makes the P^T operand need no lane
// exchange.
#include "common.hpp"

namespace incvit {

__device__ __forceinline__ void pack_p(V8<uint16_t>& out, const float* p) {
  out.v = make_uint4(f2bf2(p[0], p[1]), f2bf2(p[2], p[3]), f2bf2(p[4], p[5]), f2bf2(p[6], p[7]));
}
__device__ __forceinline__ void pack_p(V8<float>& out, const float* p) {
  out.a = make_float4(p[0], p[1], p[2], p[3]);
  out.b = make_float4(p[4], p[5], p[6], p[7]);
}

template <class T>
__device__ __forceinline__ void store4(T* dst, const float* v);
template <>
__device__ __forceinline__ void store4<uint16_t>(uint16_t* dst, const float* v) {
  *reinterpret_cast<uint2*>(dst) = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
}
template <>
__device__ __forceinline__ void store4<float>(float* dst, const float* v) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
}

constexpr int kMaxDT = kMaxHeadDim / 16;  // 16-wide d tiles

// K/V operands of one 32-key block come straight from the cache, which stores
// them in operand order (k_elem / v_elem): every load is one contiguous
// kilobyte.  Dims past d_h are zeroed in the K operand (the matching Q values
// are in-bounds data of the same row); the lanes that hold them read the
// position of lane group 0 instead (lines the wave fetches anyway), so a
// padded chunk moves only the bytes of its real dims (a quarter of the chunk
// at d_h = 72).  Keys past N are masked in the
// scores and zeroed in the V operand (their cache entries are never written).
template <class T, int NDC>
__device__ __forceinline__ void load_kblock(V8<T> (&kop)[2][NDC], const T* kbase, int kb, int dh, int g, int lane) {
  const T* blk = kbase + (size_t)kb * 2 * NDC * kChunkElems;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int c = 0; c < NDC; ++c) {
      const bool pad = 32 * c + 8 * g >= dh;
      kop[t][c].load(blk + (t * NDC + c) * kChunkElems + (pad ? lane & 15 : lane) * 8);
      if (pad) kop[t][c].zero();
    }
}

// V: the block stores NDT 16-dim tiles; only the first NDTU (those holding
// dims below d_h) are loaded and multiplied
template <class T, int NDT, int NDTU>
__device__ __forceinline__ void load_vblock(V8<T> (&vop)[NDTU], const T* vbase, int kb, int lane) {
  const T* blk = vbase + (size_t)kb * NDT * kChunkElems + lane * 8;
#pragma unroll
  for (int t = 0; t < NDTU; ++t) vop[t].load(blk + t * kChunkElems);
}

// zero the V operand entries of keys >= N (lane group g holds keys 8g..8g+7)
__device__ __forceinline__ void mask_v(V8<uint16_t>& v, int first_key, int N) {
  uint32_t q[4] = {v.v.x, v.v.y, v.v.z, v.v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int k0 = first_key + 2 * e;
    if (k0 >= N) q[e] = 0;
    else if (k0 + 1 >= N) q[e] &= 0x0000ffffu;
  }
  v.v = make_uint4(q[0], q[1], q[2], q[3]);
}
__device__ __forceinline__ void mask_v(V8<float>& v, int first_key, int N) {
  float f[8] = {v.a.x, v.a.y, v.a.z, v.a.w, v.b.x, v.b.y, v.b.z, v.b.w};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (first_key + e >= N) f[e] = 0.0f;
  v.a = make_float4(f[0], f[1], f[2], f[3]);
  v.b = make_float4(f[4], f[5], f[6], f[7]);
}

// One workgroup: QT query tiles (16 queries each) of one head of one stream.
// Its KW waves split the stream's key blocks into contiguous runs (about two
// 32-key blocks per wave: 4 waves at N = 256, 8 at N = 1024), so the K/V of a
// head are pulled through the CU by several waves at once and each wave's
// chain of dependent MFMA and softmax steps stays short, while the exchange
// of the waves' partial results stays small; every wave processes all QT
// query tiles against its keys.  Key/value loads do not depend on the row offsets, so the first
// `a.nspec` query groups issue their first key blocks before the offsets are
// read; the first stream's rows always start at 0, so its query loads are
// issued early too.  The waves' (max, sum, O) are exchanged through LDS once
// and combined in wave order, each wave finishing a share of the output
// tiles.
template <class T, int NDC, int NDT, int NDTU, int GB, int QT, int KW>
__global__ __launch_bounds__(KW * 64) void attn_kernel(AttnArgs a) {
  extern __shared__ __align__(16) char attn_smem[];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, n = lane & 15;
  // launch order: heads, then streams, then query groups, so the query
  // groups that are likely to have rows (the first of every head and stream)
  // are dispatched before all groups that will find none; the query groups of
  // one head and stream are H * B launch positions apart, which keeps them on
  // one XCD whenever H * B is a multiple of 8
  const int h = blockIdx.x, v = blockIdx.y, qg = blockIdx.z;
  const int N = a.sh.N, dh = a.sh.dh, D = a.sh.D;
  const int nkb = (N + 31) / 32;  // = Npad / 32
  const T* kbase = reinterpret_cast<const T*>(a.caches.p[v] + a.cl.k + (size_t)a.layer * a.cl.kv_layer) +
                   (size_t)h * nkb * 2 * NDC * kChunkElems;
  const T* vbase = reinterpret_cast<const T*>(a.caches.p[v] + a.cl.v + (size_t)a.layer * a.cl.kv_layer) +
                   (size_t)h * nkb * NDT * kChunkElems;
  const T* Q = static_cast<const T*>(a.q);

  // the stream's row offsets: scalar loads, issued first, waited for last
  const int off_v = a.meta->off[v], off_next = a.meta->off[v + 1];
  const int kb0 = w * nkb / KW, kb1 = (w + 1) * nkb / KW;  // this wave's key blocks (may be none)
  V8<T> kop[GB][2][NDC], vop[GB][NDTU];
  auto load_group = [&](int kb) {
#pragma unroll
    for (int b = 0; b < GB; ++b) {
      const int k = min(kb + b, nkb - 1);
      load_kblock<T, NDC>(kop[b], kbase, k, dh, g, lane);
      load_vblock<T, NDT, NDTU>(vop[b], vbase, k, lane);
    }
  };
  // The first query groups of a stream are the likely active ones: they load
  // before reading the offsets.  The other groups read them first and leave
  // without loading when they have no rows.
  const bool spec = qg < a.nspec;
  if (spec && kb0 < kb1) load_group(kb0);

  const int q0 = qg * QT * 16;
  // Q fragments: dims past d_h read in-bounds data of the same row and are
  // not zeroed, because the K fragments are zero there (no select on Q, so no
  // wait right after its loads)
  V8<T> qop[QT][NDC];
  auto load_q = [&](int rowbase, int kv) {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const int qr = min(rowbase + min(q0 + 16 * qt + n, max(kv - 1, 0)), a.qmax);
#pragma unroll
      for (int c = 0; c < NDC; ++c) {
        const int dd = 32 * c + 8 * g;
        qop[qt][c].load(Q + (size_t)qr * D + h * dh + (dd < dh ? dd : 0));
      }
    }
  };
  // the first stream's rows start at 0: its queries are loaded before the
  // offsets arrive (rows past the stream's count are clamped and never stored)
  if (spec && v == 0) load_q(0, a.qmax + 1);
  const int rowbase = off_v;
  const int kv = off_next - off_v;
  if (q0 >= kv) return;  // uniform per workgroup
  if (!spec && kb0 < kb1) load_group(kb0);
  if (!spec || v != 0) load_q(rowbase, kv);

  float m_run[QT], l_run[QT];
  f32x4_t o[QT][NDTU];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_run[qt] = -INFINITY;
    l_run[qt] = 0.0f;
#pragma unroll
    for (int t = 0; t < NDTU; ++t) o[qt][t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  }

  for (int kb = kb0; kb < kb1; kb += GB) {
    if (kb > kb0) load_group(kb);
#pragma unroll
    for (int b = 0; b < GB; ++b) {
      if (kb + b < kb1) {  // uniform
        const int key0 = (kb + b) * 32;
        if (key0 + 32 > N) {  // the stream's last, partial block (uniform)
#pragma unroll
          for (int t = 0; t < NDTU; ++t) mask_v(vop[b][t], key0 + 8 * g, N);
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          f32x4_t st[2];
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            st[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int c = 0; c < NDC; ++c) mma(st[t], kop[b][t][c], qop[qt][c]);
          }
          // st[t][i] = score of key key0 + 8g + 4t + i for query n of tile qt
          // (the cache's key order within a block), so slot 4t + i of this
          // lane is key 8g + 4t + i: the P operand order of the V product
          float sc[8];
          float mloc = -INFINITY;
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int key = key0 + 8 * g + 4 * t + i;
              const float x = key < N ? st[t][i] * a.scale_log2 : -INFINITY;
              sc[4 * t + i] = x;
              mloc = fmaxf(mloc, x);
            }
          mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
          mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
          const float m_new = fmaxf(m_run[qt], mloc);
          const bool none = (m_new == -INFINITY);
          const float alpha = none ? 1.0f : exp2f(m_run[qt] - m_new);
          float p[8], psum = 0.0f;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            p[j] = none ? 0.0f : exp2f(sc[j] - m_new);
            psum += p[j];
          }
          l_run[qt] = l_run[qt] * alpha + psum;
          V8<T> pop;
          pack_p(pop, p);
#pragma unroll
          for (int t = 0; t < NDTU; ++t) {
            o[qt][t] *= alpha;
            mma(o[qt][t], vop[b][t], pop);
          }
          m_run[qt] = m_new;
        }
      }
    }
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    l_run[qt] += __shfl_xor(l_run[qt], 16, 64);
    l_run[qt] += __shfl_xor(l_run[qt], 32, 64);
  }

  // merge: every wave publishes (max, sum, O) of its keys (a wave without keys
  // publishes max = -inf, sum = 0, O = 0); then each wave combines the KW
  // partials, in wave order, for its share of the output tiles and stores them
  float* s_m = reinterpret_cast<float*>(attn_smem);               // [KW][QT][16]
  float* s_l = s_m + KW * QT * 16;                                 // [KW][QT][16]
  f32x4_t* s_o = reinterpret_cast<f32x4_t*>(s_l + KW * QT * 16);   // [KW][QT][NDTU][64]
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    if (g == 0) {
      s_m[(w * QT + qt) * 16 + n] = m_run[qt];
      s_l[(w * QT + qt) * 16 + n] = l_run[qt];
    }
#pragma unroll
    for (int t = 0; t < NDTU; ++t) s_o[((w * QT + qt) * NDTU + t) * 64 + lane] = o[qt][t];
  }
  __syncthreads();
  for (int it = w; it < QT * NDTU; it += KW) {
    const int qt = it / NDTU, t = it % NDTU;
    const int qrow = q0 + 16 * qt + n;
    const int d0 = 16 * t + 4 * g;
    float mm = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < KW; ++ww) mm = fmaxf(mm, s_m[(ww * QT + qt) * 16 + n]);
    float lsum = 0.0f;
    f32x4_t acc = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ww = 0; ww < KW; ++ww) {
      const float mw = s_m[(ww * QT + qt) * 16 + n];
      const float f = mw == -INFINITY ? 0.0f : exp2f(mw - mm);
      lsum += f * s_l[(ww * QT + qt) * 16 + n];
      acc += s_o[((ww * QT + qt) * NDTU + t) * 64 + lane] * f;
    }
    if (qrow < kv && d0 < dh) {
      const float inv = 1.0f / lsum;
      float r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = acc[i] * inv;
      store4<T>(static_cast<T*>(a.o) + frag_off(rowbase + qrow, h * dh + d0, D / 32), r);
    }
  }
}

template <int NDT, int QT, int KW>
constexpr int attn_lds_bytes() {
  return KW * QT * 16 * 4 * 2 + KW * QT * NDT * 64 * 16;  // m and l, then O
}

template <class T, int NDC, int NDT, int NDTU, int GB, int QT, int KW>
static void launch_g(const AttnArgs& a, dim3 grid, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<T, NDC, NDT, NDTU, GB, QT, KW>),
                               hipFuncAttributeMaxDynamicSharedMemorySize,
                               attn_lds_bytes<NDTU, QT, KW>()) == hipSuccess;
  }
  (void)launch_k((attn_kernel<T, NDC, NDT, NDTU, GB, QT, KW>), grid, dim3(KW * 64),
                 (size_t)attn_lds_bytes<NDTU, QT, KW>(), s, a);
}

template <class T, int NDC, int NDT, int NDTU, int QT>
static void launch_t(const AttnArgs& a, int kw, dim3 grid, hipStream_t s) {
  // two key blocks in flight per wave where the registers allow
  constexpr int kGB = NDT <= (sizeof(T) == 2 ? 6 : 4) ? 2 : 1;
  if (kw == 2) launch_g<T, NDC, NDT, NDTU, kGB, QT, 2>(a, grid, s);
  else if (kw == 4) launch_g<T, NDC, NDT, NDTU, kGB, QT, 4>(a, grid, s);
  else launch_g<T, NDC, NDT, NDTU, kGB, QT, 8>(a, grid, s);
}

// head dims in 32-wide K chunks (NDC) and 16-wide V tiles (NDT stored, NDTU
// used: d_h = 72 stores 96 dims and uses 80)
template <class T, int QT>
static void launch_dh(const AttnArgs& a, int kw, dim3 grid, hipStream_t s) {
  const int dh = a.sh.dh;
  if (dh <= 32) launch_t<T, 1, 2, 2, QT>(a, kw, grid, s);
  else if (dh <= 64) launch_t<T, 2, 4, 4, QT>(a, kw, grid, s);
  else if (dh <= 80) launch_t<T, 3, 6, 5, QT>(a, kw, grid, s);
  else if (dh <= 96) launch_t<T, 3, 6, 6, QT>(a, kw, grid, s);
  else launch_t<T, 4, 8, 8, QT>(a, kw, grid, s);
}

// qtiles: 16-query tiles per workgroup (1 or 2).  One tile per workgroup
// doubles the workgroups (and the K/V reads) for short per-stream row counts;
// two halve the K/V traffic when there are many rows.  waves: 2, 4 or 8 per
// workgroup; 0 = about two key blocks per wave.
hipError_t launch_attn(const AttnArgs& a0, int max_rows_per_view, int qtiles, int waves, hipStream_t s) {
  AttnArgs a = a0;
  if (!a.sh.dtype) qtiles = 1;
  const int qrows = 16 * qtiles;
  dim3 grid(a.sh.H, a.B, (max_rows_per_view + qrows - 1) / qrows);
  if (grid.z == 0) return hipSuccess;
  a.nspec = qtiles == 1 ? 2 : 1;
  const int nkb = a.sh.Npad / 32;
  const int kw = waves > 0 ? waves : nkb >= 16 ? 8 : 4;
  if (!a.sh.dtype) launch_dh<float, 1>(a, kw, grid, s);  // fp32 operands: one tile (registers)
  else if (qtiles == 1) launch_dh<uint16_t, 1>(a, kw, grid, s);
  else launch_dh<uint16_t, 2>(a, kw, grid, s);
  return hipGetLastError();
}

}  // namespace incvit
