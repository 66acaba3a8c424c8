// Row kernel that finishes the split-K MLP down projection of a layer (paper
// §III-B: the residual addition after the MLP), one workgroup per compact row:
//
//   Z' = S(H + S((P_0 + P_1 + ...) + b_2))  (X^{l+1} rows, and the next
//                                           layer's input in operand order)
//   after the last layer also Y = S(LN_f(Z')) into the cache and the caller's
//   `refreshed` rows.
//
// The partial sums are added in split order, then the bias; the MLP output is
// rounded to the storage type before the residual add, whose sum is rounded
// again (each operation stores its result, as in a half-precision pipeline).  LayerNorm: two passes
// (mean, then mean squared deviation) over the row in fp32, thread partials
// summed in index order and combined across the workgroup in a fixed order.
// Every load is issued before M is known (the compact buffers are padded past
// every launched row); rows at or past M return before storing anything.
#include "common.hpp"

namespace incvit {

namespace {

__device__ __forceinline__ float4 ld4(const float* p, int q) { return reinterpret_cast<const float4*>(p)[q]; }

// 4 consecutive storage elements as floats
__device__ __forceinline__ float4 ld4s(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4s(const uint16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}

__device__ __forceinline__ void st4(float* p, int q, float4 v) { reinterpret_cast<float4*>(p)[q] = v; }
__device__ __forceinline__ void st4(uint16_t* p, int q, float4 v) {
  const uint32_t lo = f2bf2(v.x, v.y);
  const uint32_t hi = f2bf2(v.z, v.w);
  reinterpret_cast<uint2*>(p)[q] = make_uint2(lo, hi);
}

__device__ __forceinline__ float4 rnd4(float4 v, float*) { return v; }
__device__ __forceinline__ float4 rnd4(float4 v, uint16_t*) {
  return make_float4(bf2f(f2bf(v.x)), bf2f(f2bf(v.y)), bf2f(f2bf(v.z)), bf2f(f2bf(v.w)));
}

__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }

}  // namespace

// Sum over the 4 waves of a 256-thread workgroup in a fixed order (lanes by
// butterfly, then waves 0..3); every thread gets the total.
__device__ __forceinline__ float block_sum4(float x, float* s) {
  x = wave_sum(x);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) s[w] = x;
  __syncthreads();
  const float t = (s[0] + s[1]) + (s[2] + s[3]);
  __syncthreads();
  return t;
}

// One 256-thread workgroup per compact row r; thread t owns the float4 slots
// q = t + 256 j, j < KP (D <= 1024 * KP).  S: K splits.
template <class T, int S, int KP>
__global__ __launch_bounds__(256) void res_kernel(ResArgs a) {
  __shared__ float s_red[4];
  const int tid = threadIdx.x, r = blockIdx.x;
  const int M = a.meta->m;
  // the first 32 rows load before M is known; later rows (rarely used) check first
  if (r >= 32 && r >= M) return;
  const int D = a.sh.D, D4 = D / 4;
  const RowInfo ri = a.rows[r];

  float4 p[S][KP], res[KP], bias[KP], gam[KP], bet[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = min(tid + 256 * j, D4 - 1);
#pragma unroll
    for (int s = 0; s < S; ++s) p[s][j] = ld4(a.part + ((size_t)s * a.mpad + r) * D, q);
    res[j] = ld4s(static_cast<const T*>(a.res) + frag_off(r, 4 * q, D / 32));  // H is in operand order
    bias[j] = ld4(a.bias, q);
    gam[j] = bet[j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (a.last) {  // uniform: the final LayerNorm's parameters
      gam[j] = ld4(a.ln_g, q);
      bet[j] = ld4(a.ln_b, q);
    }
  }
  if (r >= M) return;  // uniform per workgroup

  // the new row Z' and, after the last layer, its LayerNorm statistics
  float4 v[KP];
  float sum = 0.0f;
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    float4 x = p[0][j];
#pragma unroll
    for (int s = 1; s < S; ++s) x = add4(x, p[s][j]);
    x = rnd4(add4(x, bias[j]), static_cast<T*>(nullptr));
    v[j] = rnd4(add4(res[j], x), static_cast<T*>(nullptr));
    if (tid + 256 * j < D4) sum += (v[j].x + v[j].y) + (v[j].z + v[j].w);
  }
  // compact position of the next layer's input row: r itself, or with the
  // all-rows map the row's place among the refreshed rows (-1: not one)
  const int zr = a.zpos ? a.zpos[r] : r;
  if (!ri.cache) return;  // uniform: a stream whose step does not run
  T* xrow = x_row<T>(ri.cache, a.cl, a.sh, a.layer + 1, ri.tok);
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = tid + 256 * j;
    if (q < D4) {
      if (zr >= 0) st4(static_cast<T*>(a.z_out) + frag_off(zr, 4 * q, D / 32), 0, v[j]);
      st4(xrow, q, v[j]);
    }
  }
  if (!a.last) return;  // uniform

  const float mean = block_sum4(sum, s_red) / (float)D;
  float sq = 0.0f;
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    if (tid + 256 * j < D4) {
      const float dx = v[j].x - mean, dy = v[j].y - mean, dz = v[j].z - mean, dw = v[j].w - mean;
      sq += (dx * dx + dy * dy) + (dz * dz + dw * dw);
    }
  }
  const float rstd = 1.0f / sqrtf(block_sum4(sq, s_red) / (float)D + a.sh.eps);
  T* yrow = reinterpret_cast<T*>(ri.cache + a.cl.y) + (size_t)ri.tok * D;
  T* outrow = nullptr;
  if (a.refreshed && zr >= 0) {
    const int j = a.zpos ? zr - a.umeta->off[ri.view] : r - a.meta->off[ri.view];
    outrow = static_cast<T*>(a.refreshed) + ((size_t)ri.view * a.N + j) * D;
  }
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = tid + 256 * j;
    if (q < D4) {
      const float4 n4 = make_float4((v[j].x - mean) * rstd * gam[j].x + bet[j].x,
                                    (v[j].y - mean) * rstd * gam[j].y + bet[j].y,
                                    (v[j].z - mean) * rstd * gam[j].z + bet[j].z,
                                    (v[j].w - mean) * rstd * gam[j].w + bet[j].w);
      st4(yrow, q, n4);
      if (outrow) st4(outrow, q, n4);
    }
  }
}

// mlp_all: one 256-thread workgroup per row r of the all-rows map:
// H[r] = S(X^l[tok] + A^l[tok]) into the compact H buffer (operand order).
template <class T, int KP>
__global__ __launch_bounds__(256) void hsum_kernel(HsumArgs a) {
  const int tid = threadIdx.x, r = blockIdx.x;
  const int D = a.sh.D, D4 = D / 4;
  const RowInfo ri = a.rows[r];
  T* h = static_cast<T*>(a.h);
  if (!ri.cache) {  // uniform
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      const int q = tid + 256 * j;
      if (q < D4) st4(h + frag_off(r, 4 * q, D / 32), 0, make_float4(0.0f, 0.0f, 0.0f, 0.0f));
    }
    return;
  }
  const T* x = x_row<T>(ri.cache, a.cl, a.sh, a.layer, ri.tok);
  const T* at = reinterpret_cast<const T*>(ri.cache + a.cl.a + (size_t)a.layer * a.cl.x_layer) + (size_t)ri.tok * D;
  float4 xv[KP], av[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = min(tid + 256 * j, D4 - 1);
    xv[j] = ld4s(x + 4 * q);
    av[j] = ld4s(at + 4 * q);
  }
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = tid + 256 * j;
    if (q < D4) st4(h + frag_off(r, 4 * q, D / 32), 0, add4(xv[j], av[j]));
  }
}

namespace {

template <class T, int S>
hipError_t launch_s(const ResArgs& a, dim3 grid, hipStream_t s) {
  if (a.sh.D <= 1024) return launch_k(res_kernel<T, S, 1>, grid, dim3(256), 0, s, a);
  return launch_k(res_kernel<T, S, 2>, grid, dim3(256), 0, s, a);
}

template <class T>
hipError_t launch_t(const ResArgs& a, dim3 grid, hipStream_t s) {
  switch (a.ksplit) {
    case 1: return launch_s<T, 1>(a, grid, s);
    case 2: return launch_s<T, 2>(a, grid, s);
    case 3: return launch_s<T, 3>(a, grid, s);
    case 4: return launch_s<T, 4>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_res(const ResArgs& a, int mmax, hipStream_t s) {
  const dim3 grid(max(1, mmax));
  return a.sh.dtype ? launch_t<uint16_t>(a, grid, s) : launch_t<float>(a, grid, s);
}

hipError_t launch_hsum(const HsumArgs& a, hipStream_t s) {
  const dim3 grid(max(1, a.rows_n));
  if (a.sh.dtype)
    return a.sh.D <= 1024 ? launch_k(hsum_kernel<uint16_t, 1>, grid, dim3(256), 0, s, a)
                          : launch_k(hsum_kernel<uint16_t, 2>, grid, dim3(256), 0, s, a);
  return a.sh.D <= 1024 ? launch_k(hsum_kernel<float, 1>, grid, dim3(256), 0, s, a)
                        : launch_k(hsum_kernel<float, 2>, grid, dim3(256), 0, s, a);
}

}  // namespace incvit
