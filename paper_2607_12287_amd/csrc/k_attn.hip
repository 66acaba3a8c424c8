// Attention of the refreshed queries over all N cached keys of their stream
// (paper §III-B: attention is computed only for the updated tokens; the keys
// and values are the scattered full K/V -- new rows for U, cached rows for R).
//
// One wave owns 16 queries of one head.  Per block of 32 keys it forms
// S^T = K Q^T with MFMA (so each lane keeps a single query and its softmax
// state), updates the online softmax in fp32 (exp2 with the 1/sqrt(d_h)
// scale folded in), and accumulates O^T = V^T P^T with MFMA.  V is cached
// transposed per head ([d_h][Npad]) so that the P^T operand needs no lane
// exchange.  For few queries (an incremental step) the 4 waves of a workgroup
// split the keys and their partial results are merged in a fixed order.
#include "common.hpp"

namespace incvit {

template <class T> struct Half4;
template <> struct Half4<uint16_t> {  // 4 bf16 = 8 bytes
  __device__ static uint2 load(const uint16_t* p, int valid) {
    uint2 r = *reinterpret_cast<const uint2*>(p);
    if (valid < 4) {
      if (valid <= 3) r.y &= 0x0000ffffu;
      if (valid <= 2) r.y = 0;
      if (valid <= 1) r.x &= 0x0000ffffu;
      if (valid <= 0) r.x = 0;
    }
    return r;
  }
};

template <class T>
__device__ __forceinline__ void load_v(V8<T>& out, const T* row, int k0, int N);

template <>
__device__ __forceinline__ void load_v<uint16_t>(V8<uint16_t>& out, const uint16_t* row, int k0, int N) {
  // slots 0..3: keys k0..k0+3, slots 4..7: keys k0+16..k0+19
  const uint2 lo = Half4<uint16_t>::load(row + k0, N - k0);
  const uint2 hi = Half4<uint16_t>::load(row + k0 + 16, N - k0 - 16);
  out.v = make_uint4(lo.x, lo.y, hi.x, hi.y);
}

template <>
__device__ __forceinline__ void load_v<float>(V8<float>& out, const float* row, int k0, int N) {
  float4 lo = *reinterpret_cast<const float4*>(row + k0);
  float4 hi = *reinterpret_cast<const float4*>(row + k0 + 16);
  const int a = N - k0, b = N - k0 - 16;
  if (a < 4) { if (a <= 3) lo.w = 0; if (a <= 2) lo.z = 0; if (a <= 1) lo.y = 0; if (a <= 0) lo.x = 0; }
  if (b < 4) { if (b <= 3) hi.w = 0; if (b <= 2) hi.z = 0; if (b <= 1) hi.y = 0; if (b <= 0) hi.x = 0; }
  out.a = lo;
  out.b = hi;
}

__device__ __forceinline__ void pack_p(V8<uint16_t>& out, const float* p) {
  out.v = make_uint4((uint32_t)f2bf(p[0]) | ((uint32_t)f2bf(p[1]) << 16),
                     (uint32_t)f2bf(p[2]) | ((uint32_t)f2bf(p[3]) << 16),
                     (uint32_t)f2bf(p[4]) | ((uint32_t)f2bf(p[5]) << 16),
                     (uint32_t)f2bf(p[6]) | ((uint32_t)f2bf(p[7]) << 16));
}
__device__ __forceinline__ void pack_p(V8<float>& out, const float* p) {
  out.a = make_float4(p[0], p[1], p[2], p[3]);
  out.b = make_float4(p[4], p[5], p[6], p[7]);
}

template <class T>
__device__ __forceinline__ void store4(T* dst, const float* v);
template <>
__device__ __forceinline__ void store4<uint16_t>(uint16_t* dst, const float* v) {
  *reinterpret_cast<uint2*>(dst) = make_uint2((uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                                              (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
}
template <>
__device__ __forceinline__ void store4<float>(float* dst, const float* v) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
}

constexpr int kMaxDT = kMaxHeadDim / 16;  // 16-wide d tiles

// Loads below are unconditional with clamped addresses (out-of-range values
// are zeroed by selects afterwards), so the wait before each MFMA covers only
// the loads it needs.

// K operands of one 32-key block: tile t holds keys kb*32 + 16t + (lane%16).
template <class T, int NDC>
__device__ __forceinline__ void load_kblock(V8<T> (&kop)[2][NDC], const T* kbase, int kb, int N, int dh,
                                            int g, int n) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int key = kb * 32 + 16 * t + n;
    const int kc = min(key, N - 1);
#pragma unroll
    for (int c = 0; c < NDC; ++c) {
      const int dd = 32 * c + 8 * g;
      kop[t][c].load(kbase + (size_t)kc * dh + (dd < dh ? dd : 0));
      if (key >= N || dd >= dh) kop[t][c].zero();
    }
  }
}

// V^T operands of one 32-key block: d tile t, row d = 16t + (lane%16).
template <class T, int NDT>
__device__ __forceinline__ void load_vblock(V8<T> (&vop)[NDT], const T* vbase, int kb, int N, int dh, int Npad,
                                            int g, int n) {
#pragma unroll
  for (int t = 0; t < NDT; ++t) {
    const int d = 16 * t + n;
    load_v<T>(vop[t], vbase + (size_t)min(d, dh - 1) * Npad, kb * 32 + 4 * g, N);
    if (d >= dh) vop[t].zero();
  }
}

template <class T, int NDC, int NDT>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  __shared__ float s_m[4][16], s_l[4][16];
  __shared__ f32x4_t s_o[4][NDT][64];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int h = blockIdx.y, v = blockIdx.z;
  const int rowbase = a.meta->off[v];
  const int kv = a.meta->off[v + 1] - rowbase;
  const int qt = a.split == 4 ? (int)blockIdx.x : (int)blockIdx.x * 4 + w;
  const int q0 = qt * 16;
  if (a.split == 4 && q0 >= kv) return;
  const bool active = q0 < kv;
  const int N = a.sh.N, Npad = a.sh.Npad, dh = a.sh.dh, D = a.sh.D;
  const T* kbase = reinterpret_cast<const T*>(a.caches.p[v] + a.cl.k + (size_t)a.layer * a.cl.kv_layer) +
                   (size_t)h * Npad * dh;
  const T* vbase = reinterpret_cast<const T*>(a.caches.p[v] + a.cl.v + (size_t)a.layer * a.cl.kv_layer) +
                   (size_t)h * dh * Npad;
  const T* Q = static_cast<const T*>(a.q);

  const int nkb = (N + 31) / 32;
  int kb0 = 0, kb1 = nkb;
  if (a.split == 4) {
    kb0 = w * nkb / 4;
    kb1 = (w + 1) * nkb / 4;
  }
  if (!active) kb1 = kb0;

  // one batch: Q, and K/V of the first key block
  const int qrow = q0 + n;
  const bool qok = active && qrow < kv;
  const int qr = min(max(rowbase + min(qrow, kv - 1), 0), a.qmax);
  V8<T> qop[NDC];
#pragma unroll
  for (int c = 0; c < NDC; ++c) {
    const int dd = 32 * c + 8 * g;
    qop[c].load(Q + (size_t)qr * D + h * dh + (dd < dh ? dd : 0));
    if (!qok || dd >= dh) qop[c].zero();
  }
  V8<T> kop[2][NDC], vop[NDT];
  load_kblock<T, NDC>(kop, kbase, min(kb0, nkb - 1), N, dh, g, n);
  load_vblock<T, NDT>(vop, vbase, min(kb0, nkb - 1), N, dh, Npad, g, n);

  float m_run = -INFINITY, l_run = 0.0f;
  f32x4_t o[NDT];
#pragma unroll
  for (int t = 0; t < NDT; ++t) o[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  for (int kb = kb0; kb < kb1; ++kb) {
    V8<T> kn[2][NDC], vn[NDT];
    // next block in flight while this one computes (past the end: a repeat)
    load_kblock<T, NDC>(kn, kbase, min(kb + 1, nkb - 1), N, dh, g, n);
    load_vblock<T, NDT>(vn, vbase, min(kb + 1, nkb - 1), N, dh, Npad, g, n);
    const int kbase0 = kb * 32;
    f32x4_t st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c = 0; c < NDC; ++c) mma(st[t], kop[t][c], qop[c]);
    }
    // st[t][i] = score of key kbase0 + 16t + 4g + i for query n
    float s[8];
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kbase0 + 16 * t + 4 * g + i;
        const float x = key < N ? st[t][i] * a.scale_log2 : -INFINITY;
        s[4 * t + i] = x;
        mloc = fmaxf(mloc, x);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_run, mloc);
    const bool none = (m_new == -INFINITY);
    const float alpha = none ? 1.0f : exp2f(m_run - m_new);
    float p[8], psum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      p[j] = none ? 0.0f : exp2f(s[j] - m_new);
      psum += p[j];
    }
    l_run = l_run * alpha + psum;
    V8<T> pop;
    pack_p(pop, p);
#pragma unroll
    for (int t = 0; t < NDT; ++t) {
      o[t] *= alpha;
      mma(o[t], vop[t], pop);
    }
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int c = 0; c < NDC; ++c) kop[t][c] = kn[t][c];
#pragma unroll
    for (int t = 0; t < NDT; ++t) vop[t] = vn[t];
  }

  float l_tot = l_run + __shfl_xor(l_run, 16, 64);
  l_tot = l_tot + __shfl_xor(l_tot, 32, 64);

  if (a.split == 4) {
    if (g == 0) {
      s_m[w][n] = m_run;
      s_l[w][n] = l_tot;
    }
#pragma unroll
    for (int t = 0; t < NDT; ++t) s_o[w][t][lane] = o[t];
    __syncthreads();
    if (w != 0) return;
    float mm = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) mm = fmaxf(mm, s_m[ww][n]);
    float f[4];
    l_tot = 0.0f;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) {
      f[ww] = s_m[ww][n] == -INFINITY ? 0.0f : exp2f(s_m[ww][n] - mm);
      l_tot += f[ww] * s_l[ww][n];
    }
#pragma unroll
    for (int t = 0; t < NDT; ++t) {
      f32x4_t acc = s_o[0][t][lane] * f[0];
#pragma unroll
      for (int ww = 1; ww < 4; ++ww) acc += s_o[ww][t][lane] * f[ww];
      o[t] = acc;
    }
  }

  if (!active || qrow >= kv) return;
  const float inv = 1.0f / l_tot;
  T* out = static_cast<T*>(a.o) + (size_t)(rowbase + qrow) * D + h * dh;
#pragma unroll
  for (int t = 0; t < NDT; ++t) {
    const int d0 = 16 * t + 4 * g;
    if (d0 < dh) {
      float r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = o[t][i] * inv;
      store4<T>(out + d0, r);
    }
  }
}

template <class T, int NDC, int NDT>
static void launch_t(const AttnArgs& a, dim3 grid, hipStream_t s) {
  (void)launch_k((attn_kernel<T, NDC, NDT>), grid, dim3(256), 0, s, a);
}

template <class T>
static void launch_dh(const AttnArgs& a, dim3 grid, hipStream_t s) {
  const int dh = a.sh.dh;
  if (dh <= 32) launch_t<T, 1, 2>(a, grid, s);
  else if (dh <= 64) launch_t<T, 2, 4>(a, grid, s);
  else if (dh <= 96) launch_t<T, 3, 6>(a, grid, s);
  else launch_t<T, 4, 8>(a, grid, s);
}

hipError_t launch_attn(const AttnArgs& a, int max_rows_per_view, hipStream_t s) {
  const int qtiles = (max_rows_per_view + 15) / 16;
  dim3 grid(a.split == 4 ? qtiles : (qtiles + 3) / 4, a.sh.H, a.B);
  if (grid.x == 0) return hipSuccess;
  if (a.sh.dtype) launch_dh<uint16_t>(a, grid, s);
  else launch_dh<float>(a, grid, s);
  return hipGetLastError();
}

}  // namespace incvit
