// Shared definitions of the incvit HIP library: device layouts, kernel argument
// structs, launchers and small device helpers.  gfx950 (CDNA4) only.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace incvit {

constexpr int kMaxViews = 64;
constexpr int kMaxTokens = 4096;
constexpr int kMaxDim = 2048;
constexpr int kMaxHeadDim = 128;
constexpr uint32_t kCacheMagic = 0x31435649u;  // "IVC1"
constexpr int kStatusNonFinite = -1;           // a step saw a NaN similarity

// Compact row buffers (row map, Z, Q, O, H, G) are padded to a multiple of
// kGemmRows rows, so a GEMM may read rows past M of its current 32-row block
// before it knows M.  Weights are packed so that one 32-deep chunk of a
// 16-column block is one 16-byte (bf16) or 32-byte (fp32) load per lane,
// already in MFMA operand order.
constexpr int kGemmRows = 64;
// Calls of bf16 models with at least this many rows known on the host run
// the large-row GEMM (gemm_tiled.hpp) instead of the weight-streaming one.
constexpr int kTiledMinRows = 512;
constexpr int kChunkElems = 512;  // 64 lanes x 8 elements

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

struct Shape {
  int N, P, D, L, H, dh, F, Fpad, Npad;
  int ndc;    // 32-wide chunks per head dim: ceil(d_h / 32)
  int dtype;  // 0 = fp32, 1 = bf16
  int eb;     // element bytes of the storage dtype
  float eps;
  int score;  // 0: the cosine compares embedded tokens; 1: first-layer keys
  int mlp_all;  // 1: every row through the MLP each frame (cached attention branch)
};

// Byte offsets inside one stream's cache.
struct CacheLayout {
  size_t ref, x, k, v, y, total;
  size_t a;         // attention-branch outputs [L][N][D] (mlp_all only, else 0)
  size_t x_layer;   // N*D*eb
  size_t kv_layer;  // H*Npad*dh*eb
};

struct CacheHeader {
  uint32_t magic;
  uint32_t hash;
  int32_t status;
  uint32_t frames;
  uint32_t pad[60];
};
static_assert(sizeof(CacheHeader) == 256, "header is 256 bytes");

struct Views {
  char* p[kMaxViews];
};

// Rows of a call: row r of the compact M rows is token `tok` of the stream
// whose cache starts at `cache`.  Written once per call (by the commit
// kernel) so that later kernels find a row with a single load.
struct RowInfo {
  char* cache;
  int tok;
  int view;
};

// Per-call bookkeeping in the workspace.
struct Meta {
  int m;                     // M: rows of the call
  int off[kMaxViews + 1];    // first compact row of each stream
};

// Rows of a call as the selection left them: count[v] rows of stream v are
// tokens idx[v*N + 0 .. count[v]).  Read only by the commit kernel.
struct RowMap {
  const int* count;
  const int* idx;
  int B, N;
};

struct LayerW {
  const float* ln1_g;
  const float* ln1_b;
  const void* w_qkv;
  const float* b_qkv;
  const void* w_o;
  const float* b_o;
  const float* ln2_g;
  const float* ln2_b;
  const void* w_1;
  const float* b_1;
  const void* w_2;
  const float* b_2;
};

// ---------------------------------------------------------------- kernels --

// Fixed-order fp32 product of token rows with a storage-type matrix: the patch
// embedding (x = patches, K = P, W = W_pe, + Pos) and the key projection of
// the key score (x = LayerNorm rows, K = D, W = W_K, pos = null).
struct EmbedArgs {
  const float* patches;  // [B][N][P] (P = K, the row length of x)
  const void* w_pe;      // [P][D] storage dtype
  const float* b_pe;     // [D]
  const float* pos;      // [N][D], or null: nothing added after the chain
  float* t0;             // [B][N][D]
  int B, N, P, D, dtype;
  int* zero;             // counters to clear (may be null)
  int nzero;
  int* ident_idx;        // if set: idx[v][i] = i, count[v] = N
  int* ident_count;
};

// Key score, first part: LayerNorm 1 of layer 0 of every token's stored
// layer-0 input, fixed order (one wave per token).
struct KeyLnArgs {
  const float* t0;     // [rows][D] embedded tokens
  const float* ln_g;   // [D] layer-0 LayerNorm 1
  const float* ln_b;
  float* out;          // [rows][D]
  int rows, D, dtype;
  float eps;
};

struct SimArgs {
  const float* t0;
  Views caches;
  size_t ref_off;
  float* sim;  // [B][N]
  int B, N, D;
};

struct SelectArgs {
  const float* sim;
  Views caches;
  int B, N;
  float tau;
  uint32_t hash;
  int cap[kMaxViews];
  int* idx;    // [B][N]
  int* count;  // [B]
  int* valid;  // [B] (may be null): 1 if the stream's step runs, else 0
};

struct RowsArgs {  // commit: ref/X0/Z0 of the refreshed rows, row map
  RowMap rm;
  RowInfo* rows;     // commit writes
  Meta* meta;        // commit writes
  Views caches;
  CacheLayout cl;
  Shape sh;
  const float* t0;
  const float* score;  // [B][N][D] score vectors: the new references of the rows
  int init_header;   // commit of a full encode: write header
  uint32_t hash;
  void* z;           // compact Z_0 [Mpad][D] (operand order)
  // mlp_all: every row of every stream, r = v * N + tok.  X0 of all rows,
  // the all-rows map (cache null for a stream whose step does not run), and
  // zpos[r] = the row's compact position among the refreshed rows, or -1
  int all_rows;
  const int* valid;  // [B] from the selection; null: every stream runs
  RowInfo* rows_all;
  Meta* meta_all;
  int* zpos;
};

enum Epi { EPI_QKV = 0, EPI_FC1 = 1, EPI_PART = 2, EPI_RES = 3, EPI_ATT = 4, EPI_DOWN = 5 };

// Fields in the order the kernel's prologue needs them, so that its argument
// loads go out together.
struct GemmArgs {
  const void* A;      // compact A rows in operand order: QKV Z_l, RES O, FC1 H, PART G
  const void* W;      // packed [Nout/16][kchunks][512]
  const float* bias;  // [Nout] (not used by PART)
  const float* c1;    // QKV, FC1: column sums of the LayerNorm-folded weights; `bias`
                      // then holds beta^T W + b (see FoldArgs)
  const RowInfo* rows;  // row map (cache, token, stream) of each compact row
  const Meta* meta;
  const void* resid;  // RES: Z_l rows, DOWN: H rows (operand order)
  void* out;          // QKV Q [Mpad][D]; RES H (operand order); FC1 G; PART f32 [ksplit][mpad][ldo];
                      // ATT: unused (rows go to the cache's A^l); DOWN: Z_{l+1} (operand
                      // order), also written to the cache's X^{l+1}
  int lda, kchunks, Nout, ldo;
  int ksplit;         // K is split over ksplit workgroups (PART)
  int rgroups;        // 32-row groups launched: enough for the largest M of the call
  int mpad;           // padded rows (partial slices)
  int layer;
  Shape sh;
  CacheLayout cl;
};

// Row kernel that finishes the split-K MLP down projection, one workgroup per
// compact row: Z_{l+1} = S(H + (partials + b_2)) -> compact Z (operand order)
// and X^{l+1} of the cache; after the last layer also Y = S(LN_f(Z_L)) into
// the cache and the refreshed output.
struct ResArgs {
  const Meta* meta;
  const RowInfo* rows;
  CacheLayout cl;
  Shape sh;
  int layer;
  int last;           // after the last layer: final LayerNorm
  const float* part;  // [ksplit][mpad][D]
  int ksplit, mpad;
  const void* res;    // H (storage type, operand order)
  const float* bias;
  const float* ln_g;  // the final LayerNorm (last layer)
  const float* ln_b;
  void* z_out;        // Z_{l+1} (operand order)
  void* refreshed;    // final: optional [B][N][D]
  int N;
  // mlp_all (rows = all rows of the call): Z_{l+1} goes to compact row zpos[r]
  // (skipped when -1), `refreshed` row = zpos[r] - umeta->off[view]; rows
  // whose cache is null are skipped
  const int* zpos;
  const Meta* umeta;
};

// mlp_all: H = S(X^l + A^l) of every row of the call (cache rows), into the
// compact H buffer in operand order; rows of a stream whose step does not run
// (cache null) get zeros.
struct HsumArgs {
  const RowInfo* rows;  // all-rows map
  CacheLayout cl;
  Shape sh;
  int layer;
  int rows_n;           // B * N
  void* h;
};

struct AttnArgs {
  const Meta* meta;
  int B;
  Views caches;
  CacheLayout cl;
  Shape sh;
  int layer;
  const void* q;  // [Mpad][D]
  void* o;        // [Mpad][D]
  int qmax;       // Mpad - 1: last row a clamped load may touch
  float scale_log2;
  int nspec;      // query groups that load keys before reading the row offsets
};

struct PackArgs {
  const void* src;  // canonical [K][Ncols] storage dtype
  void* dst;        // packed
  int K, Ncols, kchunks, nblocks, dtype;
};

// Folding a LayerNorm (gamma, beta) into the packed weights W that follow it:
// W' = S(gamma_k W[k][n]) in the packed layout, c1[n] = sum_k W'[k][n] and
// c2b[n] = sum_k beta_k W[k][n] + b[n] (fp32, columns up to nblocks * 16).
struct FoldArgs {
  const void* src;    // canonical W [K][Ncols] storage dtype
  const void* gamma;  // canonical [K] storage dtype
  const void* beta;
  const void* bias;   // canonical [Ncols] storage dtype
  void* dst;          // packed W (written by pack_kernel first)
  float* c1;
  float* c2b;
  int K, Ncols, kchunks, nblocks, dtype;
};

struct ConvArgs {  // storage dtype vector -> fp32 (with zero padding)
  const void* src;
  float* dst;
  long n, npad;
  int dtype;
};

// The two-anchor flow update: x_T[s] = x_0[s] + alpha[s] v_0[s] + beta[s] v_7[s] + b[s].
struct FlowArgs {
  const float* x0;
  const float* v0;
  const float* v7;
  const float* alpha;  // [S]
  const float* beta;   // [S]
  const float* b;
  float* xT;           // [S][n]; may alias x0
  int S;
  long n;
};

struct ExportArgs {
  const char* cache;
  char* canon;
  CacheLayout cl;
  Shape sh;
  int to_canonical;  // 1 export, 0 import
  uint32_t hash;
};

// Start/stop events that the next kernel launch on this host thread records
// with its own dispatch (per-kernel timing that adds no stream operations);
// both null outside profiled calls.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();

// Every kernel here takes one argument struct by value.
template <class A>
hipError_t launch_k(void (*kernel)(A), dim3 grid, dim3 block, size_t lds, hipStream_t s, A arg) {
  void* argv[] = {&arg};
  const LaunchEvents& ev = launch_events();
  if (ev.start)
    return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, lds, s, ev.start, ev.stop, 0);
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, lds, s);
}

// launchers (return the launch error)
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);
hipError_t launch_keyproj(const EmbedArgs& a, hipStream_t s);
hipError_t launch_keyln(const KeyLnArgs& a, hipStream_t s);
hipError_t launch_sim(const SimArgs& a, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
hipError_t launch_commit(const RowsArgs& a, int mmax, hipStream_t s);
hipError_t launch_gemm(int epi, int cols, const GemmArgs& a, hipStream_t s);
// the large-row GEMM (gemm_tiled.hpp): bf16, whole K, rows = the call's M
hipError_t launch_gemm_tiled(int epi, const GemmArgs& a, int rows, hipStream_t s);
hipError_t launch_res(const ResArgs& a, int mmax, hipStream_t s);
hipError_t launch_hsum(const HsumArgs& a, hipStream_t s);
hipError_t launch_attn(const AttnArgs& a, int max_rows_per_view, int qtiles, int waves, hipStream_t s);
hipError_t launch_pack(const PackArgs& a, hipStream_t s);
hipError_t launch_fold(const FoldArgs& a, hipStream_t s);
hipError_t launch_conv(const ConvArgs& a, hipStream_t s);
hipError_t launch_export(const ExportArgs& a, hipStream_t s);
hipError_t launch_flow(const FlowArgs& a, hipStream_t s);

}  // namespace incvit

// ------------------------------------------------------------ device side --
#if defined(__HIPCC__)
namespace incvit {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

// Pointers read from memory (the row map) are generic to the compiler, which
// then emits flat accesses; flat accesses count against both the vector-memory
// and the LDS counters and defeat load pipelining.  Every such pointer here
// points to device global memory, so it is cast to the global address space.
#define INCVIT_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ INCVIT_GLOBAL T* gbl(T* p) {
  return (INCVIT_GLOBAL T*)p;
}
template <class T>
__device__ __forceinline__ const INCVIT_GLOBAL T* gbl(const T* p) {
  return (const INCVIT_GLOBAL T*)p;
}

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16 bits, round to nearest even: gfx950's v_cvt_pk_bf16_f32 (two
// conversions per instruction; NaN stays NaN).
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// two values packed, the first in the low half
__device__ __forceinline__ uint32_t f2bf2(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

template <class T> struct Elem;
template <> struct Elem<uint16_t> {
  __device__ static float f(uint16_t x) { return bf2f(x); }
  __device__ static float ld(const uint16_t* p, long i) { return bf2f(p[i]); }
  __device__ static uint16_t cv(float f) { return f2bf(f); }
  __device__ static float rnd(float f) { return bf2f(f2bf(f)); }
};
template <> struct Elem<float> {
  __device__ static float f(float x) { return x; }
  __device__ static float ld(const float* p, long i) { return p[i]; }
  __device__ static float cv(float f) { return f; }
  __device__ static float rnd(float f) { return f; }
};

// Buffer resources: a wave-uniform base and byte size in SGPRs, so that a
// load needs one 32-bit lane offset (shared by every load of a wave) plus a
// wave-uniform offset instead of a 64-bit address per load; reads past the
// size return zero.
typedef __amdgpu_buffer_rsrc_t Rsrc;
__device__ __forceinline__ Rsrc make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 bload16(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ float4 bload16f(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// 8 consecutive elements of one lane: one MFMA operand for a 32-deep chunk.
template <class T> struct V8;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <> struct V8<uint16_t> {
  uint4 v;
  __device__ void load(const uint16_t* p) { v = __builtin_bit_cast(uint4, *(const INCVIT_GLOBAL u32x4_t*)p); }
  // lane offset voff (16 bytes per lane), wave-uniform offset soff, in bytes
  __device__ void bload(Rsrc r, uint32_t voff, uint32_t soff) { v = bload16(r, voff, soff); }
  __device__ void zero() { v = make_uint4(0, 0, 0, 0); }
};
template <> struct V8<float> {
  float4 a, b;
  __device__ void load(const float* p) {
    a = __builtin_bit_cast(float4, ((const INCVIT_GLOBAL f32x4_t*)p)[0]);
    b = __builtin_bit_cast(float4, ((const INCVIT_GLOBAL f32x4_t*)p)[1]);
  }
  // lane offset voff (32 bytes per lane), wave-uniform offset soff, in bytes
  __device__ void bload(Rsrc r, uint32_t voff, uint32_t soff) {
    a = bload16f(r, voff, soff);
    b = bload16f(r, voff + 16, soff);
  }
  __device__ void zero() { a = make_float4(0, 0, 0, 0); b = a; }
};

// acc(16x16) += A(16x32) * B(32x16) where lane l holds A[l%16][8*(l/16)+j] and
// B[8*(l/16)+j][l%16], j = 0..7.  Output lane l holds rows 4*(l/16)+i, col l%16.
__device__ __forceinline__ void mma(f32x4_t& acc, const V8<uint16_t>& a, const V8<uint16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                __builtin_bit_cast(bf16x8_t, b.v), acc, 0, 0, 0);
}
// fp32: eight 16x16x4 products; product j pairs element j of every lane, so
// the chunk's k = 8*(l/16)+j assignment is the same as for bf16.
__device__ __forceinline__ void mma(f32x4_t& acc, const V8<float>& a, const V8<float>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.x, b.a.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.y, b.a.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.z, b.a.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.w, b.a.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.x, b.b.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.y, b.b.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.z, b.b.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.w, b.b.w, acc, 0, 0, 0);
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

template <class T>
__device__ __forceinline__ T* x_row(char* cache, const CacheLayout& cl, const Shape& sh, int layer, int tok) {
  return reinterpret_cast<T*>(cache + cl.x + (size_t)layer * cl.x_layer) + (size_t)tok * sh.D;
}

// Compact GEMM inputs (A1/A2, O, G) are stored as MFMA A operands: for row r
// and column k of a [rows][32 kc] matrix, 16-row tile r/16 and 32-deep chunk
// k/32 form one kilobyte (bf16) in which lane 16*((k%32)/8) + r%16 holds 8
// consecutive k; so a GEMM loads each operand fragment as one contiguous
// block, and a row's 4-aligned runs of 4 columns stay contiguous for writers.
__host__ __device__ __forceinline__ size_t frag_off(int r, int k, int kc) {
  return (((size_t)(r >> 4) * kc + (k >> 5)) * 64 + (((k & 31) >> 3) << 4) + (r & 15)) * 8 + (k & 7);
}

// Cached K and V of one layer are stored as the attention's MFMA operands, so
// that each operand load is one contiguous kilobyte.  Per head, per block of
// 32 keys (kb), head dims padded to 32 * ndc:
//   K: [kb][tile t (2)][dim chunk c (ndc)][lane (64)][8]; lane 16g + n of
//      tile t holds key 8(n/4) + 4t + n%4 of the block, dims 32c + 8g .. +7.
//      The key order makes the score tile give each lane 8 consecutive keys.
//   V: [kb][dim tile (2 ndc)][lane (64)][8]; lane 16g + n holds dim 16 tile + n,
//      keys 8g .. 8g + 7 of the block (the transposed operand).
// Entries for padded dims or keys past N are never written; readers mask them.
__host__ __device__ __forceinline__ size_t k_elem(const Shape& sh, int h, int tok, int d) {
  const int kb = tok >> 5, r = tok & 31;
  const int t = (r & 7) >> 2, n = 4 * (r >> 3) + (r & 3);
  const int c = d >> 5, g = (d >> 3) & 3, j = d & 7;
  return (((((size_t)h * (sh.Npad >> 5) + kb) * 2 + t) * sh.ndc + c) * 64 + (16 * g + n)) * 8 + j;
}
__host__ __device__ __forceinline__ size_t v_elem(const Shape& sh, int h, int tok, int d) {
  const int kb = tok >> 5, r = tok & 31;
  const int g = r >> 3, j = r & 7, dt = d >> 4, n = d & 15;
  return ((((size_t)h * (sh.Npad >> 5) + kb) * (2 * sh.ndc) + dt) * 64 + (16 * g + n)) * 8 + j;
}

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (gfx9 encoding: vmcnt split over bits 3:0 and
// 15:14; expcnt and lgkmcnt left at their no-wait maxima).
__host__ __device__ constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// 16 bytes of LDS at byte address addr + off (off a compile-time constant)
// into a register quad, without a wait: the caller waits for lgkmcnt.
__device__ __forceinline__ void lds_read16(u32x4_t& out, uint32_t addr, int off) {
  switch (off) {  // the offset is an immediate of the instruction
#define INCVIT_DSR(o) \
    case o: asm volatile("ds_read_b128 %0, %1 offset:" #o : "=v"(out) : "v"(addr)); break;
    INCVIT_DSR(0) INCVIT_DSR(1024) INCVIT_DSR(2048) INCVIT_DSR(3072) INCVIT_DSR(4096) INCVIT_DSR(5120)
    INCVIT_DSR(6144) INCVIT_DSR(7168) INCVIT_DSR(8192) INCVIT_DSR(9216) INCVIT_DSR(10240) INCVIT_DSR(11264)
    INCVIT_DSR(12288) INCVIT_DSR(13312) INCVIT_DSR(14336) INCVIT_DSR(15360)
#undef INCVIT_DSR
    default: asm volatile("ds_read_b128 %0, %1" : "=v"(out) : "v"(addr + off)); break;
  }
}

// The offsets above separate into a row (token) part and a column (dim) part,
// so an epilogue that writes many rows of the same columns forms each part
// once: frag_off = frag_row + frag_col, k_elem = k_tok + k_col, v_elem =
// v_tok + v_col.
__host__ __device__ __forceinline__ size_t frag_row(int r, int kc) { return ((size_t)(r >> 4) * kc * 64 + (r & 15)) * 8; }
__host__ __device__ __forceinline__ size_t frag_col(int k) {
  return ((size_t)(k >> 5) * 64 + (((k & 31) >> 3) << 4)) * 8 + (k & 7);
}
__host__ __device__ __forceinline__ size_t k_tok(const Shape& sh, int tok) {
  const int r = tok & 31;
  return (size_t)(tok >> 5) * 2 * sh.ndc * 512 + ((r & 7) >> 2) * sh.ndc * 512 + 8 * (4 * (r >> 3) + (r & 3));
}
__host__ __device__ __forceinline__ size_t k_col(const Shape& sh, int h, int d) {
  return (size_t)h * (sh.Npad >> 5) * 2 * sh.ndc * 512 + (d >> 5) * 512 + 128 * ((d >> 3) & 3) + (d & 7);
}
__host__ __device__ __forceinline__ size_t v_tok(const Shape& sh, int tok) {
  const int r = tok & 31;
  return (size_t)(tok >> 5) * 2 * sh.ndc * 512 + 128 * (r >> 3) + (r & 7);
}
__host__ __device__ __forceinline__ size_t v_col(const Shape& sh, int h, int d) {
  return (size_t)h * (sh.Npad >> 5) * 2 * sh.ndc * 512 + (d >> 4) * 512 + 8 * (d & 15);
}

}  // namespace incvit
#endif
