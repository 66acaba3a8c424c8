// Weight packing and cache export/import.
#include "common.hpp"

namespace incvit {

// canonical [K][Ncols] -> packed [nblocks][kchunks][64 lanes][8]: lane l of
// chunk (nb, kc) holds W[32kc + 8(l/16) + j][16nb + l%16], j = 0..7, zero
// outside the matrix (K and column padding).
template <class T>
__global__ void pack_kernel(PackArgs a) {
  const T* src = static_cast<const T*>(a.src);
  T* dst = static_cast<T*>(a.dst);
  const size_t total = (size_t)a.nblocks * a.kchunks * kChunkElems;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (size_t)gridDim.x * blockDim.x) {
    const int j = (int)(e & 7), lane = (int)((e >> 3) & 63);
    const size_t ch = e >> 9;
    const int kc = (int)(ch % a.kchunks), nb = (int)(ch / a.kchunks);
    const int k = kc * 32 + 8 * (lane >> 4) + j, col = nb * 16 + (lane & 15);
    T val = T(0);
    if (k < a.K && col < a.Ncols) val = src[(size_t)k * a.Ncols + col];
    dst[e] = val;
  }
}

// One thread per packed column: the folded weights of the column (rounded to
// the storage type), their sum, and beta^T W + b, both accumulated in fp64.
template <class T>
__global__ void fold_kernel(FoldArgs a) {
  const int col = blockIdx.x * blockDim.x + threadIdx.x;
  if (col >= a.nblocks * 16) return;
  const T* src = static_cast<const T*>(a.src);
  const T* gm = static_cast<const T*>(a.gamma);
  const T* bt = static_cast<const T*>(a.beta);
  T* dst = static_cast<T*>(a.dst);
  double c1 = 0.0, c2 = 0.0;
  if (col < a.Ncols) {
    const int nb = col / 16, cl = col % 16;
    for (int k = 0; k < a.K; ++k) {
      const float w = Elem<T>::f(src[(size_t)k * a.Ncols + col]);
      const float wf = Elem<T>::rnd(Elem<T>::f(gm[k]) * w);
      const int kc = k / 32, kk = k % 32;
      dst[(((size_t)nb * a.kchunks + kc) * 64 + 16 * (kk / 8) + cl) * 8 + kk % 8] = Elem<T>::cv(wf);
      c1 += (double)wf;
      c2 += (double)Elem<T>::f(bt[k]) * (double)w;
    }
    c2 += (double)Elem<T>::f(static_cast<const T*>(a.bias)[col]);
  }
  a.c1[col] = (float)c1;
  a.c2b[col] = (float)c2;
}

__global__ void conv_kernel(ConvArgs a) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < a.npad; i += (long)gridDim.x * blockDim.x) {
    float x = 0.0f;
    if (i < a.n) x = a.dtype ? bf2f(static_cast<const uint16_t*>(a.src)[i]) : static_cast<const float*>(a.src)[i];
    a.dst[i] = x;
  }
}

// Canonical layout of one cache: ref [N][D] f32 | X [L+1][N][D] | K [L][N][D]
// | V [L][N][D] | Y [N][D] | with mlp_all A [L][N][D] (storage dtype).  Device
// layout differs for K and V (attention operand order, k_elem / v_elem).
template <class T>
__global__ void export_kernel(ExportArgs a) {
  const Shape& sh = a.sh;
  const size_t nd = (size_t)sh.N * sh.D;
  const size_t n_ref = nd, n_x = (size_t)(sh.L + 1) * nd, n_kv = (size_t)sh.L * nd;
  const size_t n_a = sh.mlp_all ? (size_t)sh.L * nd : 0;
  const size_t total = n_ref + n_x + 2 * n_kv + nd + n_a;
  char* cache = const_cast<char*>(a.cache);
  const float* cref = reinterpret_cast<const float*>(a.canon);
  const T* cT = reinterpret_cast<const T*>(a.canon + n_ref * sizeof(float));
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (size_t)gridDim.x * blockDim.x) {
    if (e < n_ref) {
      float* dev = reinterpret_cast<float*>(cache + a.cl.ref) + e;
      float* can = const_cast<float*>(cref) + e;
      if (a.to_canonical) *can = *dev; else *dev = *can;
      continue;
    }
    const size_t f = e - n_ref;  // index into the storage-dtype part
    T* can = const_cast<T*>(cT) + f;
    T* dev;
    if (f < n_x) {
      dev = reinterpret_cast<T*>(cache + a.cl.x) + f;
    } else if (f < n_x + 2 * n_kv) {
      const bool isv = f >= n_x + n_kv;
      const size_t r = f - n_x - (isv ? n_kv : 0);
      const int l = (int)(r / nd);
      const size_t rem = r - (size_t)l * nd;
      const int tok = (int)(rem / sh.D), c = (int)(rem % sh.D);
      const int hh = c / sh.dh, d = c % sh.dh;
      T* base = reinterpret_cast<T*>(cache + (isv ? a.cl.v : a.cl.k) + (size_t)l * a.cl.kv_layer);
      dev = base + (isv ? v_elem(sh, hh, tok, d) : k_elem(sh, hh, tok, d));
    } else if (f < n_x + 2 * n_kv + nd) {
      dev = reinterpret_cast<T*>(cache + a.cl.y) + (f - n_x - 2 * n_kv);
    } else {
      dev = reinterpret_cast<T*>(cache + a.cl.a) + (f - n_x - 2 * n_kv - nd);
    }
    if (a.to_canonical) *can = *dev; else *dev = *can;
  }
  if (!a.to_canonical && blockIdx.x == 0 && threadIdx.x == 0) {
    CacheHeader* hdr = reinterpret_cast<CacheHeader*>(cache);
    hdr->magic = kCacheMagic;
    hdr->hash = a.hash;
    hdr->status = 0;
    hdr->frames = 0;
  }
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  if (a.dtype) (void)launch_k(pack_kernel<uint16_t>, dim3(1024), dim3(256), 0, s, a);
  else (void)launch_k(pack_kernel<float>, dim3(1024), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fold(const FoldArgs& a, hipStream_t s) {
  const dim3 grid((a.nblocks * 16 + 63) / 64);
  if (a.dtype) (void)launch_k(fold_kernel<uint16_t>, grid, dim3(64), 0, s, a);
  else (void)launch_k(fold_kernel<float>, grid, dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_conv(const ConvArgs& a, hipStream_t s) {
  (void)launch_k(conv_kernel, dim3(256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_export(const ExportArgs& a, hipStream_t s) {
  if (a.sh.dtype) (void)launch_k(export_kernel<uint16_t>, dim3(1024), dim3(256), 0, s, a);
  else (void)launch_k(export_kernel<float>, dim3(1024), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace incvit
