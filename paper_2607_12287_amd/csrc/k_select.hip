// Token selection (paper §III-B: the least similar tokens are updated, chosen
// once before the first layer) and the per-row kernels around the layers.
//
// select: U = {i : sim_i < tau} (strict); if |U| > cap keep the cap lowest
// similarities, equal similarities going to the lower index; write U ascending.
// The cap-th smallest key is found by an exact 4-pass radix select over the
// order-preserving integer image of the fp32 similarity, so the result is a
// pure function of the similarities.
#include "common.hpp"

namespace incvit {


__device__ __forceinline__ uint32_t order_key(float s) {
  if (s == 0.0f) s = 0.0f;  // -0 and +0 compare equal
  const uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive scan of one int per thread over the workgroup (in thread order).
__device__ int block_exclusive_scan(int x, int* s_wave, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) s_wave[w] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < nw; ++i) {
      const int t = s_wave[i];
      s_wave[i] = acc;
      acc += t;
    }
    s_wave[nw] = acc;
  }
  __syncthreads();
  const int res = s_wave[w] + incl - x;
  total = s_wave[nw];
  __syncthreads();
  return res;
}

// TH threads: one wave for up to 256 tokens (its barriers and scans are the
// cheapest: 7.2 -> 6.9 us per step at 256 tokens), 16 waves beyond (4 waves
// made the radix passes of 1024 tokens slower: 11.2 -> 11.8 us); every thread
// owns a contiguous segment of at most kPer tokens.
template <int TH>
__global__ __launch_bounds__(TH) void select_kernel(SelectArgs a) {
  __shared__ uint32_t skey[kMaxTokens];
  __shared__ int s_hist[256];
  __shared__ int s_wave[TH / 64 + 1];
  __shared__ int s_misc[4];
  const int v = blockIdx.x, tid = threadIdx.x, N = a.N;
  CacheHeader* hdr = reinterpret_cast<CacheHeader*>(a.caches.p[v]);
  if (tid == 0) {
    const CacheHeader h = *hdr;
    s_misc[0] = (h.magic == kCacheMagic && h.hash == a.hash && h.status == 0) ? 1 : 0;
    s_misc[1] = 0;  // non-finite seen
    s_misc[2] = 0;  // candidates
  }
  // contiguous token segment per thread (keeps scans in index order); the
  // segment's similarities are loaded in one batch
  constexpr int kPer = 4;  // N <= 4 TH by the launch rule (256 = 4 * 64; kMaxTokens = 4 * 1024)
  const int per = (N + TH - 1) / TH;
  const int i0 = min(N, tid * per), i1 = min(N, i0 + per);
  float sv[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) sv[j] = (i0 + j < i1) ? a.sim[(size_t)v * N + i0 + j] : 0.0f;
  int cand = 0, bad = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    if (i0 + j < i1) {
      const float sj = sv[j];
      bad |= (sj != sj);
      const bool f = sj < a.tau;
      skey[i0 + j] = f ? order_key(sj) : 0xffffffffu;
      cand += f;
    }
  }
  __syncthreads();
  if (!s_misc[0]) {  // never encoded, or another model: this stream is a no-op
    if (tid == 0) {
      a.count[v] = 0;
      if (a.valid) a.valid[v] = 0;
    }
    return;
  }
  if (bad) atomicOr(&s_misc[1], 1);
  atomicAdd(&s_misc[2], cand);
  __syncthreads();
  if (s_misc[1]) {
    if (tid == 0) {
      hdr->status = kStatusNonFinite;
      a.count[v] = 0;
      if (a.valid) a.valid[v] = 0;
    }
    return;
  }
  if (tid == 0 && a.valid) a.valid[v] = 1;
  const int total = s_misc[2];
  const int cap = min(max(a.cap[v], 0), N);

  uint32_t thr = 0xffffffffu;  // keys < thr are taken, keys == thr by index
  int need_eq = 0;
  if (total > cap) {
    if (cap == 0) {
      thr = 0;
      need_eq = 0;
    } else {
      uint32_t prefix = 0;
      int kth = cap;  // 1-based rank of the wanted key among the remaining
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int b = tid; b < 256; b += TH) s_hist[b] = 0;
        __syncthreads();
        for (int i = i0; i < i1; ++i) {
          const uint32_t k = skey[i];
          if (k == 0xffffffffu) continue;
          if (pass > 0 && (k >> (shift + 8)) != (prefix >> (shift + 8))) continue;
          atomicAdd(&s_hist[(k >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid < 64) {  // wave 0 finds the digit holding the kth key
          const int lane = tid;
          int loc[4], sum = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            loc[j] = s_hist[4 * lane + j];
            sum += loc[j];
          }
          int incl = sum;
#pragma unroll
          for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off, 64);
            if (lane >= off) incl += y;
          }
          int before = incl - sum;
          for (int j = 0; j < 4; ++j) {
            if (before < kth && kth <= before + loc[j]) {
              s_misc[3] = 4 * lane + j;
              s_wave[0] = before;  // reuse as scratch; consumed below
            }
            before += loc[j];
          }
        }
        __syncthreads();
        const int digit = s_misc[3];
        kth -= s_wave[0];
        prefix |= (uint32_t)digit << shift;
        __syncthreads();
      }
      thr = prefix;
      need_eq = kth;
    }
  }

  // Ties at thr are taken in index order: a tie is taken iff the number of
  // ties before it is < need_eq.  Both scans run over contiguous segments, so
  // thread order is index order.
  const bool has_thr = thr != 0xffffffffu;
  int eq = 0;
  for (int i = i0; i < i1; ++i) eq += (has_thr && skey[i] == thr);
  int eq_total;
  const int eq_before = block_exclusive_scan(eq, s_wave, eq_total);
  int sel = 0;
  {
    int e = eq_before;
    for (int i = i0; i < i1; ++i) {
      const uint32_t k = skey[i];
      if (k == 0xffffffffu) continue;
      if (k < thr) ++sel;
      else if (k == thr) sel += (e++ < need_eq);
    }
  }
  int total_sel;
  int pos = block_exclusive_scan(sel, s_wave, total_sel);
  {
    int e = eq_before;
    for (int i = i0; i < i1; ++i) {
      const uint32_t k = skey[i];
      if (k == 0xffffffffu) continue;
      bool take = k < thr;
      if (k == thr) take = (e++ < need_eq);
      if (take) a.idx[(size_t)v * N + pos++] = i;
    }
  }
  if (tid == 0) a.count[v] = total_sel;
}

// 4 consecutive elements (already representable in T) to storage
__device__ __forceinline__ void store4v(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void store4v(uint16_t* p, float4 v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(f2bf2(v.x, v.y), f2bf2(v.z, v.w));
}

// Row r = v * N + tok of the all-rows map (mlp_all): X0[tok] = S(T0[tok]) for
// every token, the map entry (cache null if the stream's step does not run),
// and zpos[r] = compact position of the token among the refreshed rows or -1
// (binary search of the ascending index list).
template <class T, int KP>
__device__ void commit_all_row(const RowsArgs& a, int r, const int* s_off) {
  const int N = a.rm.N, D = a.sh.D, D4 = D / 4;
  const int v = r / N, tok = r - v * N;
  const bool ok = a.init_header || !a.valid || a.valid[v];
  char* cache = a.caches.p[v];
  if (threadIdx.x == 0) {
    a.rows_all[r] = RowInfo{ok ? cache : nullptr, tok, v};
    int lo = 0, hi = a.rm.count[v];  // idx[v][lo..hi) ascending
    const int* ix = a.rm.idx + (size_t)v * N;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (ix[mid] < tok) lo = mid + 1; else hi = mid;
    }
    a.zpos[r] = (lo < a.rm.count[v] && ix[lo] == tok) ? s_off[v] + lo : -1;
  }
  if (!ok) return;
  const float4* src = reinterpret_cast<const float4*>(a.t0 + ((size_t)v * N + tok) * D);
  T* x0 = x_row<T>(cache, a.cl, a.sh, 0, tok);
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = threadIdx.x + 256 * j;
    if (q < D4) {
      const float4 t = src[q];
      store4v(x0 + 4 * q, make_float4(Elem<T>::rnd(t.x), Elem<T>::rnd(t.y), Elem<T>::rnd(t.z), Elem<T>::rnd(t.w)));
    }
  }
}

// One workgroup per compact row r: ref[tok] = score[tok] (fp32: the embedded
// token or its first-layer key), X0[tok] = S(T0[tok]),
// the compact Z0 row (operand order, the layer-0 input), and the row's entry in
// the row map.  Block 0 also publishes M and the per-stream row offsets.
// Thread t owns float4 slots t + 256 j of the row (D <= 1024 * KP).
template <class T, int KP>
__global__ __launch_bounds__(256) void commit_kernel(RowsArgs a) {
  __shared__ int s_cnt[kMaxViews];
  __shared__ int s_off[kMaxViews + 1];
  const int tid = threadIdx.x;
  const int B = a.rm.B, N = a.rm.N, D = a.sh.D, D4 = D / 4;
  if (tid < B) s_cnt[tid] = a.rm.count[tid];
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int v = 0; v < B; ++v) {
      s_off[v] = acc;
      acc += s_cnt[v];
    }
    s_off[B] = acc;
  }
  __syncthreads();
  const int M = s_off[B];
  if (blockIdx.x == 0) {
    if (tid <= B) a.meta->off[tid] = s_off[tid];
    if (tid == 0) a.meta->m = M;
    if (a.init_header && tid < B) {
      CacheHeader* hdr = reinterpret_cast<CacheHeader*>(a.caches.p[tid]);
      hdr->magic = kCacheMagic;
      hdr->hash = a.hash;
      hdr->status = 0;
      hdr->frames = 0;
    }
  }
  const int r = blockIdx.x;
  if (a.all_rows) {  // uniform: this workgroup's row of the all-rows map
    if (blockIdx.x == 0) {
      if (tid == 0) a.meta_all->m = B * N;
      if (tid <= B) a.meta_all->off[tid] = tid * N;
    }
    if (r < B * N) commit_all_row<T, KP>(a, r, s_off);
  }
  if (r >= M) return;  // uniform per workgroup
  int v = 0;
  while (v + 1 < B && s_off[v + 1] <= r) ++v;
  const int tok = a.rm.idx[v * N + (r - s_off[v])];
  char* cache = a.caches.p[v];
  const float4* src = reinterpret_cast<const float4*>(a.t0 + ((size_t)v * N + tok) * D);
  const float4* sc = reinterpret_cast<const float4*>(a.score + ((size_t)v * N + tok) * D);
  float4* ref = reinterpret_cast<float4*>(cache + a.cl.ref + (size_t)tok * D * 4);
  T* x0 = x_row<T>(cache, a.cl, a.sh, 0, tok);
  T* z0 = static_cast<T*>(a.z);  // operand order (frag_off)
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const int q = tid + 256 * j;
    if (q < D4) {
      const float4 t = src[q];
      const float4 zr = make_float4(Elem<T>::rnd(t.x), Elem<T>::rnd(t.y), Elem<T>::rnd(t.z), Elem<T>::rnd(t.w));
      ref[q] = sc[q];
      store4v(x0 + 4 * q, zr);
      store4v(z0 + frag_off(r, 4 * q, D / 32), zr);
    }
  }
  if (tid == 0) a.rows[r] = RowInfo{cache, tok, v};
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  static_assert(kMaxTokens <= 4 * 1024, "at most 4 tokens per thread");
  if (a.N <= 256) (void)launch_k(select_kernel<64>, dim3(a.B), dim3(64), 0, s, a);
  else (void)launch_k(select_kernel<1024>, dim3(a.B), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_commit(const RowsArgs& a, int mmax, hipStream_t s) {
  const dim3 grid(max(1, a.all_rows ? max(mmax, a.rm.B * a.rm.N) : mmax));
  const bool wide = a.sh.D > 1024;
  if (a.sh.dtype)
    return wide ? launch_k(commit_kernel<uint16_t, 2>, grid, dim3(256), 0, s, a)
                : launch_k(commit_kernel<uint16_t, 1>, grid, dim3(256), 0, s, a);
  return wide ? launch_k(commit_kernel<float, 2>, grid, dim3(256), 0, s, a)
              : launch_k(commit_kernel<float, 1>, grid, dim3(256), 0, s, a);
}



}  // namespace incvit
