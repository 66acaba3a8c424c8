// C ABI of the incremental ViT encoder: validation, buffer layouts and the
// launch sequence of one encode call.  The host only enqueues; it never waits
// for the device inside incvit_full_encode / incvit_step.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"
#include "incvit.h"

using namespace incvit;

namespace {

constexpr size_t kAlign = 256;
constexpr int kMaxSplit = 8;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

thread_local std::string g_error;

struct PackedLayer {
  size_t ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o, ln2_g, ln2_b, w_1, b_1, w_2, b_2;
  // LN1 folded into W_qkv and LN2 into W_1 (packed only): column sums of the
  // folded weights and beta^T W + b
  size_t qkv_c1, qkv_c2b, fc1_c1, fc1_c2b;
};

struct PackedLayout {
  size_t w_pe, b_pe, pos, lnf_g, lnf_b, total;
  size_t w_key;  // W_K of layer 0, [D][D] storage dtype (key score)
  std::vector<PackedLayer> layers;
};

struct CanonLayout {  // element offsets into the canonical buffer
  size_t w_pe, b_pe, pos, lnf_g, lnf_b, total;
  std::vector<PackedLayer> layers;
};

struct WsLayout {
  size_t meta, rows, count, idx, sim, t0, kn, key, z, q, o, h, g, part, total;
  size_t valid, zpos, rows_all, meta_all;  // all-rows MLP reading
  int Mpad;
};

enum GemmKind { G_QKV = 0, G_OPROJ = 1, G_FC1 = 2, G_FC2 = 3 };

bool make_shape(const incvit_config* c, Shape& sh, incvit_status& st, std::string& err) {
  char buf[256];
  st = INCVIT_ERR_SHAPE;
  if (!c) { st = INCVIT_ERR_ARG; err = "null config"; return false; }
  if (c->img_h <= 0 || c->img_w <= 0 || c->channels <= 0 || c->patch <= 0 || c->dim <= 0 ||
      c->depth <= 0 || c->heads <= 0 || c->mlp_dim <= 0) {
    err = "config sizes must be positive";
    return false;
  }
  if (c->img_h % c->patch || c->img_w % c->patch) { err = "image size is not a multiple of the patch size"; return false; }
  if (c->dim % c->heads) { err = "dim is not a multiple of heads"; return false; }
  if (!(c->ln_eps > 0.0f) || !std::isfinite(c->ln_eps)) { err = "ln_eps must be positive and finite"; return false; }
  if (c->dtype != INCVIT_F32 && c->dtype != INCVIT_BF16) { st = INCVIT_ERR_UNSUPPORTED; err = "dtype must be INCVIT_F32 or INCVIT_BF16"; return false; }
  if (c->score != INCVIT_SCORE_EMBED && c->score != INCVIT_SCORE_KEY) { st = INCVIT_ERR_ARG; err = "score must be INCVIT_SCORE_EMBED or INCVIT_SCORE_KEY"; return false; }
  if (c->mlp_all != 0 && c->mlp_all != 1) { st = INCVIT_ERR_ARG; err = "mlp_all must be 0 or 1"; return false; }
  sh.N = (c->img_h / c->patch) * (c->img_w / c->patch);
  sh.P = c->channels * c->patch * c->patch;
  sh.D = c->dim;
  sh.L = c->depth;
  sh.H = c->heads;
  sh.dh = c->dim / c->heads;
  sh.F = c->mlp_dim;
  sh.Fpad = round_up(c->mlp_dim, 32);
  sh.Npad = round_up(sh.N, 32);
  sh.ndc = (sh.dh + 31) / 32;
  sh.dtype = c->dtype;
  sh.eb = c->dtype == INCVIT_BF16 ? 2 : 4;
  sh.eps = c->ln_eps;
  sh.score = c->score;
  sh.mlp_all = c->mlp_all;
  st = INCVIT_ERR_UNSUPPORTED;
  if (sh.D % 32) { err = "dim must be a multiple of 32"; return false; }
  if (sh.D > kMaxDim) { snprintf(buf, sizeof buf, "dim must be <= %d", kMaxDim); err = buf; return false; }
  if (sh.dh % 8 || sh.dh > kMaxHeadDim) { err = "head dim must be a multiple of 8 and <= 128"; return false; }
  if (sh.N > kMaxTokens) { snprintf(buf, sizeof buf, "at most %d tokens", kMaxTokens); err = buf; return false; }
  if (c->max_streams < 1 || c->max_streams > kMaxViews) { snprintf(buf, sizeof buf, "max_streams must be in [1, %d]", kMaxViews); err = buf; return false; }
  // Kernels address each buffer through 32-bit offsets (buffer resources and
  // 32-bit index products), so the largest buffer one launch can touch must
  // stay below 4 GiB: a stream's patches, W_pe, a packed GEMM matrix, and the
  // compact GEMM operands of the largest call (every token of max_streams
  // streams, the MLP hidden rows being the widest).
  {
    const size_t lim = 0xffffffffu;
    const size_t mpad = (size_t)round_up(c->max_streams * sh.N, kGemmRows);
    const size_t kmax = (size_t)std::max(sh.D, sh.Fpad);
    const size_t wide = (size_t)round_up(std::max(3 * sh.D, sh.Fpad), 32);
    const size_t sizes[] = {(size_t)sh.N * sh.P * 4, (size_t)sh.P * sh.D * sh.eb, mpad * kmax * sh.eb,
                            wide * kmax * sh.eb};
    for (size_t b : sizes)
      if (b > lim) { err = "a buffer that one kernel addresses would exceed 4 GiB (fewer streams, tokens, channels or a smaller MLP)"; return false; }
  }
  st = INCVIT_OK;
  return true;
}

size_t packed_gemm_bytes(int K, int Ncols, int eb) {
  return (size_t)(round_up(Ncols, 16) / 16) * (size_t)(round_up(K, 32) / 32) * kChunkElems * eb;
}

PackedLayout packed_layout(const Shape& sh) {
  PackedLayout p;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  const int D = sh.D, eb = sh.eb;
  p.w_pe = take((size_t)sh.P * D * eb);
  p.b_pe = take((size_t)D * 4);
  p.pos = take((size_t)sh.N * D * 4);
  for (int l = 0; l < sh.L; ++l) {
    PackedLayer L;
    L.ln1_g = take(D * 4);
    L.ln1_b = take(D * 4);
    L.w_qkv = take(packed_gemm_bytes(D, 3 * D, eb));
    L.b_qkv = take(3 * D * 4);
    L.w_o = take(packed_gemm_bytes(D, D, eb));
    L.b_o = take(D * 4);
    L.ln2_g = take(D * 4);
    L.ln2_b = take(D * 4);
    L.w_1 = take(packed_gemm_bytes(D, sh.Fpad, eb));
    L.b_1 = take((size_t)sh.Fpad * 4);
    L.w_2 = take(packed_gemm_bytes(sh.Fpad, D, eb));
    L.b_2 = take(D * 4);
    L.qkv_c1 = take(3 * D * 4);
    L.qkv_c2b = take(3 * D * 4);
    L.fc1_c1 = take((size_t)sh.Fpad * 4);
    L.fc1_c2b = take((size_t)sh.Fpad * 4);
    p.layers.push_back(L);
  }
  p.lnf_g = take(D * 4);
  p.lnf_b = take(D * 4);
  p.w_key = take((size_t)D * D * eb);
  p.total = off;
  return p;
}

CanonLayout canon_layout(const Shape& sh) {
  CanonLayout c;
  size_t off = 0;
  auto take = [&](size_t n) { size_t o = off; off += n; return o; };
  const size_t D = sh.D, F = sh.F;
  c.w_pe = take((size_t)sh.P * D);
  c.b_pe = take(D);
  c.pos = take((size_t)sh.N * D);
  for (int l = 0; l < sh.L; ++l) {
    PackedLayer L;
    L.ln1_g = take(D);
    L.ln1_b = take(D);
    L.w_qkv = take(D * 3 * D);
    L.b_qkv = take(3 * D);
    L.w_o = take(D * D);
    L.b_o = take(D);
    L.ln2_g = take(D);
    L.ln2_b = take(D);
    L.w_1 = take(D * F);
    L.b_1 = take(F);
    L.w_2 = take(F * D);
    L.b_2 = take(D);
    c.layers.push_back(L);
  }
  c.lnf_g = take(D);
  c.lnf_b = take(D);
  c.total = off;
  return c;
}

CacheLayout cache_layout(const Shape& sh) {
  CacheLayout cl;
  size_t off = kAlign;  // header
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  cl.x_layer = (size_t)sh.N * sh.D * sh.eb;
  cl.kv_layer = (size_t)sh.H * (sh.Npad / 32) * sh.ndc * 1024 * sh.eb;  // see k_elem / v_elem
  cl.ref = take((size_t)sh.N * sh.D * 4);
  cl.x = take(cl.x_layer * (sh.L + 1));
  cl.k = take(cl.kv_layer * sh.L);
  cl.v = take(cl.kv_layer * sh.L);
  cl.y = take(cl.x_layer);
  cl.a = sh.mlp_all ? take(cl.x_layer * sh.L) : 0;
  cl.total = off;
  return cl;
}

uint32_t config_hash(const incvit_config& c) {
  const int32_t f[11] = {c.img_h, c.img_w, c.channels, c.patch, c.dim, c.depth, c.heads, c.mlp_dim, c.dtype, c.score,
                         c.mlp_all};
  uint32_t h = 2166136261u;
  auto mix = [&](uint32_t x) {
    for (int i = 0; i < 4; ++i) {
      h ^= (x >> (8 * i)) & 0xffu;
      h *= 16777619u;
    }
  };
  for (int i = 0; i < 11; ++i) mix((uint32_t)f[i]);
  uint32_t e;
  memcpy(&e, &c.ln_eps, 4);
  mix(e);
  return h == 0 ? 1u : h;
}

struct GemmGeom {
  int K, kchunks, Nout, nblocks, ksplit;
};

GemmGeom gemm_geom(const Shape& sh, int kind) {
  GemmGeom g;
  switch (kind) {
    case G_QKV: g.K = sh.D; g.Nout = 3 * sh.D; break;
    case G_OPROJ: g.K = sh.D; g.Nout = sh.D; break;
    case G_FC1: g.K = sh.D; g.Nout = sh.Fpad; break;
    default: g.K = sh.Fpad; g.Nout = sh.D; break;
  }
  g.kchunks = round_up(g.K, 32) / 32;
  g.nblocks = g.Nout / 16;
  // The MLP down projection has D/16 column blocks over a long K = F: its K is
  // split over up to 4 workgroups (at least 8 chunks each), and a row kernel
  // adds the partial sums, the bias, the residual and the next LayerNorm.  The
  // output projection (K = D) is not split: its epilogue adds the residual
  // itself and leaves the LN2 block statistics for fc1.
  g.ksplit = 1;
  if (kind == G_FC2)
    g.ksplit = std::max(1, std::min(std::min(4, 256 / std::max(g.nblocks, 1)), g.kchunks / 8));
  return g;
}

// Column blocks per workgroup.  With one row group (threshold steps, M not
// known on the host) parallelism over columns wins: one block per workgroup,
// two only for outputs with more blocks than CUs (each A row is then read
// once for 32 columns).  With several row groups (M known: full encodes,
// top-k steps) there are workgroups enough, and two blocks per workgroup for
// the output projection and the MLP down projection (and the MLP up
// projection from 1536 rows) halve the A reads: measured on MI355X, e.g. the
// 8-stream full encode 5.75 -> 4.70 ms, the 448x448 top-k step 1.58 -> 1.47 ms.
int cols_of(const int* tuned, const GemmGeom& g, int kind, int rgroups, int rows, bool exact) {
  const int t = tuned ? tuned[kind] : 0;
  if (t > 0) return t;
  if (rgroups > 1) {
    // four blocks (bf16; fewer where they do not divide) for QKV and for the
    // unsplit MLP down projection: 448x448 top-k at 102 / 256 / 1024 rows,
    // QKV 11.2 -> 8.9, 17.3 -> 15.3, 41.9 -> 33.1 us; down projection at 256
    // and 1024 rows 18.5 -> 15.7, 65.1 -> 45.5 us; the output projection, fc1
    // and the K-split down projection were slower with four.  Not beyond 1024
    // known rows, where each row group loops over many row blocks and a
    // quarter of the workgroups leaves CUs idle (8 streams' full encode
    // 4.7 -> 5.2 ms), and for QKV only while the workgroups still cover the
    // CUs (448x448 top-k at 51 rows, 2 row groups, 108 workgroups: the step
    // 1.21 -> 1.26 ms).
    const bool few = !exact || rows <= 1024;
    if (kind == G_QKV && few && g.nblocks / 4 * rgroups >= 192) return 4;
    if (kind == G_FC2 && g.ksplit == 1 && few) return 4;
    if (kind == G_OPROJ || kind == G_FC2) return g.nblocks % 2 == 0 ? 2 : 1;
    if (kind == G_FC1) return rows >= 1536 || g.nblocks > 256 * rgroups ? 2 : 1;
    return 1;
  }
  return g.nblocks > 256 ? 2 : 1;
}

// Row groups of one GEMM launch, from the call's row groups R (rows known on
// the host, or the caller's expected count).  While R is small (at most 6
// blocks of 32 rows, as in the steps; full encodes of 256 or more rows have
// 8, and keep them) each GEMM keeps only as many
// groups as its workgroups fill the chip once; the groups then loop over the
// remaining row blocks with their weights still in registers:
//   QKV with four-block workgroups: at most one workgroup per CU (more put two
//     on a few CUs, which then finish last), as long as the four-block form
//     still applies (>= 192 workgroups);
//   MLP up projection (one block per workgroup): at most two per CU;
//   K-split MLP down projection (two blocks per workgroup): one per CU;
//   the output projection keeps R (its few workgroups gain from every group).
// Measured on MI355X, 8 ViT-L streams at 172 rows (R = 6): QKV 13.3 -> 11.8,
// fc1 10.9 -> 10.0, fc2 9.3 -> 8.2 us; 3 So400m streams at 101 rows (R = 4):
// fc1 12.7 -> 12.1, fc2 8.1 -> 7.4 us.
int gemm_rgroups(const Shape& sh, const GemmGeom& g, int kind, int R) {
  if (R <= 1 || R > 6) return R;
  int cap = R;
  if (kind == G_QKV && sh.dtype && g.nblocks % 4 == 0) {
    const int cg = g.nblocks / 4;
    if (cg * R > 256 && cg * (256 / cg) >= 192) cap = 256 / cg;
  } else if (kind == G_FC1) {
    cap = 512 / g.nblocks;
  } else if (kind == G_FC2 && g.ksplit > 1) {
    cap = 256 / ((g.nblocks % 2 == 0 ? g.nblocks / 2 : g.nblocks) * g.ksplit);
  }
  return std::max(1, std::min(R, cap));
}

// Query tiles per attention workgroup: one tile per workgroup while two-tile
// workgroups would leave most CUs idle (few streams and heads), otherwise
// two, which halves the K/V reads when a stream has many refreshed rows.
// With the rows known on the host and long streams (N >= 512) every query
// tile's workgroup reads the head's whole K/V (295 KB at N = 1024, d_h = 72),
// so two tiles per workgroup as soon as their workgroups still cover the CUs:
// the 448x448 full encode, 1024 rows, 26.9 -> 21.3 us per launch.
int attn_qtiles_of(int tuned, int B, int H, int N, int max_rows_per_view, bool exact) {
  if (tuned > 0) return tuned;
  const int groups2 = (max_rows_per_view + 31) / 32;
  if (exact && N >= 512 && groups2 * B * H >= 256) return 2;
  return std::min(groups2, 2) * B * H < 128 ? 1 : 2;
}

WsLayout ws_layout(const Shape& sh, int B) {
  WsLayout w;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  const int M = B * sh.N;
  w.Mpad = round_up(std::max(M, 1), kGemmRows);
  w.meta = take(sizeof(Meta));
  w.rows = take((size_t)w.Mpad * sizeof(RowInfo));
  w.count = take(kMaxViews * 4);
  w.idx = take((size_t)M * 4);
  w.sim = take((size_t)M * 4);
  w.t0 = take((size_t)M * sh.D * 4);
  // key score: LayerNorm rows and keys of every token (key mode only)
  w.kn = take(sh.score ? (size_t)M * sh.D * 4 : 0);
  w.key = take(sh.score ? (size_t)M * sh.D * 4 : 0);
  w.z = take((size_t)w.Mpad * sh.D * sh.eb);
  w.q = take((size_t)w.Mpad * sh.D * sh.eb);
  w.o = take((size_t)w.Mpad * sh.D * sh.eb);
  w.h = take((size_t)w.Mpad * sh.D * sh.eb);
  w.g = take((size_t)w.Mpad * sh.Fpad * sh.eb);
  w.part = take((size_t)gemm_geom(sh, G_FC2).ksplit * w.Mpad * sh.D * 4);
  w.valid = take(kMaxViews * 4);
  w.zpos = take(sh.mlp_all ? (size_t)M * 4 : 0);
  w.rows_all = take(sh.mlp_all ? (size_t)w.Mpad * sizeof(RowInfo) : 0);
  w.meta_all = take(sh.mlp_all ? sizeof(Meta) : 0);
  w.total = off;
  return w;
}

}  // namespace

struct incvit_handle {
  incvit_config cfg;
  Shape sh;
  CacheLayout cl;
  uint32_t hash;
  const char* packed;
  PackedLayout pl;
  std::string err;
  bool prof = false;
  struct Rec {
    int kind;
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  double prof_ms[INCVIT_K_COUNT] = {};
  int64_t prof_n[INCVIT_K_COUNT] = {};
  int cols[4] = {0, 0, 0, 0};  // 0 = automatic
  int attn_qtiles = 0;         // 0 = automatic
  int attn_waves = 0;          // 0 = automatic
  int fc2_mode = 0;            // 1: split-K + row kernel, 2: unsplit with the residual in the epilogue, 0: by M
  int row_groups = 1;          // GEMM row groups of threshold steps
  int tiled = 0;               // 0: the large-row GEMM where it applies, 1: never
};

struct incvit_graph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

LaunchEvents& incvit::launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}

namespace {

incvit_status fail(incvit_handle* h, incvit_status st, const std::string& msg) {
  if (h) h->err = msg;
  else g_error = msg;
  return st;
}

hipEvent_t take_event(incvit_handle* h) {
  if (!h->pool.empty()) {
    hipEvent_t e = h->pool.back();
    h->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// One kernel launch; with profiling on, the launch itself records a start and
// a stop event (timestamps of its own dispatch, as a kernel trace sees it).
template <class F>
incvit_status run(incvit_handle* h, int kind, hipStream_t s, F&& launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (h->prof) {
    e0 = take_event(h);
    e1 = take_event(h);
  }
  if (e0 && e1) launch_events() = {e0, e1};
  const hipError_t err = launch();
  launch_events() = {};
  if (e0 && e1) {
    h->recs.push_back({kind, e0, e1});
  } else {
    if (e0) h->pool.push_back(e0);
    if (e1) h->pool.push_back(e1);
  }
  if (err != hipSuccess) {
    char buf[256];
    snprintf(buf, sizeof buf, "kernel launch failed (kind %d): %s", kind, hipGetErrorString(err));
    return fail(h, INCVIT_ERR_HIP, buf);
  }
  return INCVIT_OK;
}

const float* fptr(const incvit_handle* h, size_t off) { return reinterpret_cast<const float*>(h->packed + off); }

// Launch the per-layer kernels for the rows of the call (row map in ws).
// refreshed: optional output of the last layer's final LayerNorm rows.
// With mlp_all the output projection writes the attention branch of the
// refreshed rows into the cache, and the residual and the MLP run over every
// row of the call (the all-rows map in ws).
incvit_status run_layers(incvit_handle* h, const Views& views, int B, const WsLayout& wl, char* ws,
                         int max_rows_per_view, int mmax, bool exact_m, void* refreshed, hipStream_t s) {
  // GEMM row groups: when the call's row count M is known on the host (a full
  // encode, or a pure top-k step where M is the sum of the caps), one 32-row
  // block per workgroup (up to 8 groups); otherwise one group, which loops over
  // the row blocks (idle groups cost about a microsecond each per launch)
  auto groups_for = [&](int rows, bool known) {
    const int need = std::max(1, (rows + 31) / 32);
    return std::min(known ? need : std::max(1, std::min(need, h->row_groups)), 8);
  };
  const Shape& sh = h->sh;
  const bool all = sh.mlp_all != 0;
  const int mall = B * sh.N;
  const int rgroups = groups_for(mmax, exact_m);
  const RowInfo* rows = reinterpret_cast<const RowInfo*>(ws + wl.rows);
  const Meta* meta = reinterpret_cast<const Meta*>(ws + wl.meta);
  // the rows of the MLP: the refreshed rows, or with mlp_all every row
  const RowInfo* mrows = all ? reinterpret_cast<const RowInfo*>(ws + wl.rows_all) : rows;
  const Meta* mmeta = all ? reinterpret_cast<const Meta*>(ws + wl.meta_all) : meta;
  const int mlp_rows = all ? mall : mmax;
  const int mgroups = all ? groups_for(mall, true) : rgroups;
  // the large-row GEMM: bf16 models, the rows of the call known on the host
  // and at least kTiledMinRows (full encodes, pure top-k steps, the all-rows
  // MLP); the output projection only once its tiles fill the chip, and the
  // MLP down projection split over K while they do not (below)
  const bool tiled_att = h->tiled == 0 && sh.dtype && exact_m && mmax >= kTiledMinRows;
  const bool tiled_mlp = h->tiled == 0 && sh.dtype && (exact_m || all) && mlp_rows >= kTiledMinRows;
  // the large-row MLP down projection runs over K = F: its workgroup's chunks
  // follow one another, so while its tiles give fewer than one workgroup per
  // CU it is split over K like the small-M form (partial sums added by the
  // row kernel): So400m at 768 and 1024 rows, 36-37 us for the whole K in
  // one workgroup
  int fc2_split = 1;
  if (tiled_mlp) {
    const GemmGeom g2 = gemm_geom(sh, G_FC2);
    const int tiles = (mlp_rows + 63) / 64 * ((g2.nblocks + 7) / 8);
    if (h->fc2_mode == 1 || (h->fc2_mode == 0 && tiles < 256)) fc2_split = g2.ksplit;
  }
  for (int l = 0; l < sh.L; ++l) {
    const PackedLayer& P = h->pl.layers[l];
    // the MLP down projection of every layer but the last (whose row kernel
    // also applies the final LayerNorm) can run unsplit with the residual and
    // the cache write in its epilogue instead of split-K partials + row kernel:
    // slower for a few dozen rows (the whole K of 16 columns per workgroup
    // against a third of it), faster once M is in the hundreds (the partial
    // sums of every row no longer go through memory), so by default only when
    // M is known on the host and at least 192; the large-row form whenever it
    // is not split over K (above)
    const bool down = !all && l + 1 < sh.L &&
                      (tiled_mlp ? fc2_split == 1
                                 : h->fc2_mode == 2 || (h->fc2_mode == 0 && exact_m && mmax >= 192));
    auto gemm = [&](int kind, int kernel_kind) -> incvit_status {
      GemmGeom g = gemm_geom(sh, kind);
      const bool mlp = kind == G_FC1 || kind == G_FC2;
      // the output projection (N = D) takes the large-row form only once its
      // 64-row tiles fill the chip: with fewer its workgroups each run the
      // whole K while most CUs idle (So400m at 512 / 768 / 1024 rows: 13.6 /
      // 14.0 / 13.5 us against 8.3 / 10.9 / 12.7 us for the small-M form; 8
      // ViT-L streams, 2048 rows and 256 tiles: 13.0 against 14.1 us)
      const bool tiled = mlp ? tiled_mlp
                             : tiled_att && (kind != G_OPROJ || (mmax + 63) / 64 * ((g.nblocks + 7) / 8) >= 256);
      if (kind == G_FC2 && down) g.ksplit = 1;
      else if (kind == G_FC2 && tiled) g.ksplit = fc2_split;
      GemmArgs a;
      memset(&a, 0, sizeof a);
      a.rows = mlp ? mrows : rows;
      a.meta = mlp ? mmeta : meta;
      a.cl = h->cl;
      a.sh = sh;
      a.layer = l;
      a.kchunks = g.kchunks;
      a.Nout = g.Nout;
      a.ksplit = g.ksplit;
      a.rgroups = mlp ? mgroups : rgroups;
      if (!all && !down) a.rgroups = gemm_rgroups(sh, g, kind, a.rgroups);
      a.mpad = wl.Mpad;
      int epi = EPI_PART;
      switch (kind) {
        case G_QKV:
          epi = EPI_QKV;
          a.A = ws + wl.z; a.lda = sh.D;
          a.W = h->packed + P.w_qkv; a.bias = fptr(h, P.qkv_c2b); a.c1 = fptr(h, P.qkv_c1);
          a.out = ws + wl.q; a.ldo = sh.D;
          break;
        case G_OPROJ:
          epi = all ? EPI_ATT : EPI_RES;
          a.A = ws + wl.o; a.lda = sh.D;
          a.W = h->packed + P.w_o; a.bias = fptr(h, P.b_o);
          a.resid = ws + wl.z;
          a.out = ws + wl.h; a.ldo = sh.D;
          break;
        case G_FC1:
          epi = EPI_FC1;
          a.A = ws + wl.h; a.lda = sh.D;
          a.W = h->packed + P.w_1; a.bias = fptr(h, P.fc1_c2b); a.c1 = fptr(h, P.fc1_c1);
          a.out = ws + wl.g; a.ldo = sh.Fpad;
          break;
        default:
          a.A = ws + wl.g; a.lda = sh.Fpad;
          a.W = h->packed + P.w_2;
          a.out = ws + wl.part; a.ldo = sh.D;
          if (down) {
            epi = EPI_DOWN;
            a.bias = fptr(h, P.b_2);
            a.resid = ws + wl.h;
            a.out = ws + wl.z;
          }
          break;
      }
      if (tiled)
        return run(h, kernel_kind, s, [&] { return launch_gemm_tiled(epi, a, mlp ? mlp_rows : mmax, s); });
      const int cols = cols_of(h->cols, g, kind, a.rgroups, mlp ? mlp_rows : mmax, exact_m || (mlp && all));
      return run(h, kernel_kind, s, [&] { return launch_gemm(epi, cols, a, s); });
    };
    auto rowk = [&](int kernel_kind) -> incvit_status {
      const GemmGeom g = gemm_geom(sh, G_FC2);
      ResArgs r;
      memset(&r, 0, sizeof r);
      r.meta = mmeta;
      r.rows = mrows;
      r.cl = h->cl;
      r.sh = sh;
      r.layer = l;
      r.part = reinterpret_cast<const float*>(ws + wl.part);
      r.ksplit = tiled_mlp ? fc2_split : g.ksplit;
      r.mpad = wl.Mpad;
      r.N = sh.N;
      r.res = ws + wl.h;
      r.bias = fptr(h, P.b_2);
      r.z_out = ws + wl.z;
      r.last = l + 1 == sh.L;
      if (all) {
        r.zpos = reinterpret_cast<const int*>(ws + wl.zpos);
        r.umeta = meta;
      }
      if (r.last) {
        r.ln_g = fptr(h, h->pl.lnf_g);
        r.ln_b = fptr(h, h->pl.lnf_b);
        r.refreshed = refreshed;
      }
      return run(h, kernel_kind, s, [&] { return launch_res(r, mlp_rows, s); });
    };

    incvit_status st;
    if (mmax > 0) {  // attention part: the refreshed rows only
      if ((st = gemm(G_QKV, INCVIT_K_QKV)) != INCVIT_OK) return st;
      AttnArgs aa;
      memset(&aa, 0, sizeof aa);
      aa.meta = meta;
      aa.B = B;
      aa.caches = views;
      aa.cl = h->cl;
      aa.sh = sh;
      aa.layer = l;
      aa.q = ws + wl.q;
      aa.o = ws + wl.o;
      aa.qmax = wl.Mpad - 1;
      aa.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)sh.dh));
      const int qtiles = attn_qtiles_of(h->attn_qtiles, B, sh.H, sh.N, max_rows_per_view, exact_m);
      if ((st = run(h, INCVIT_K_ATTN, s, [&] { return launch_attn(aa, max_rows_per_view, qtiles, h->attn_waves, s); })) != INCVIT_OK)
        return st;
      if ((st = gemm(G_OPROJ, INCVIT_K_OPROJ)) != INCVIT_OK) return st;
    }
    if (all) {
      HsumArgs ha{mrows, h->cl, sh, l, mall, ws + wl.h};
      if ((st = run(h, INCVIT_K_HSUM, s, [&] { return launch_hsum(ha, s); })) != INCVIT_OK) return st;
    }
    if ((st = gemm(G_FC1, INCVIT_K_FC1)) != INCVIT_OK) return st;
    if ((st = gemm(G_FC2, INCVIT_K_FC2)) != INCVIT_OK) return st;
    if (!down && (st = rowk(INCVIT_K_RES_LN1)) != INCVIT_OK) return st;
  }
  return INCVIT_OK;
}

incvit_status check_views(incvit_handle* h, int32_t B, void* const* caches, Views& views) {
  if (!caches) return fail(h, INCVIT_ERR_ARG, "caches is null");
  memset(&views, 0, sizeof views);
  for (int v = 0; v < B; ++v) {
    if (!caches[v]) return fail(h, INCVIT_ERR_ARG, "a cache pointer is null");
    if (reinterpret_cast<uintptr_t>(caches[v]) % kAlign) return fail(h, INCVIT_ERR_ARG, "cache pointers must be 256-byte aligned");
    views.p[v] = static_cast<char*>(caches[v]);
  }
  // each stream's step writes its whole cache: two streams sharing bytes would race
  uintptr_t base[kMaxViews];
  for (int v = 0; v < B; ++v) base[v] = reinterpret_cast<uintptr_t>(caches[v]);
  std::sort(base, base + B);
  for (int v = 1; v < B; ++v)
    if (base[v] - base[v - 1] < h->cl.total) return fail(h, INCVIT_ERR_ARG, "caches of one call must not overlap");
  return INCVIT_OK;
}

incvit_status check_common(incvit_handle* h, int32_t B, const float* patches, void* ws) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  if (B < 1 || B > h->cfg.max_streams) return fail(h, INCVIT_ERR_ARG, "B must be in [1, max_streams]");
  if (!patches) return fail(h, INCVIT_ERR_ARG, "patches is null");
  if (reinterpret_cast<uintptr_t>(patches) % 16) return fail(h, INCVIT_ERR_ARG, "patches must be 16-byte aligned");
  if (!ws) return fail(h, INCVIT_ERR_ARG, "workspace is null");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(h, INCVIT_ERR_ARG, "workspace must be 256-byte aligned");
  return INCVIT_OK;
}

// mlp_all: the commit also writes X0 of every row, the all-rows map and the
// rows' compact positions among the refreshed rows.
void set_all_rows(RowsArgs& ra, const Shape& sh, char* ws, const WsLayout& wl, const int* valid) {
  if (!sh.mlp_all) return;
  ra.all_rows = 1;
  ra.valid = valid;
  ra.rows_all = reinterpret_cast<RowInfo*>(ws + wl.rows_all);
  ra.meta_all = reinterpret_cast<Meta*>(ws + wl.meta_all);
  ra.zpos = reinterpret_cast<int*>(ws + wl.zpos);
}

// The score vectors of every token of the call: the embedded tokens t0, or in
// key mode their first-layer keys (LayerNorm 1 of layer 0, then W_K), both in
// the fixed fp32 order.  Returns the buffer the cosine and the commit read.
incvit_status score_pass(incvit_handle* h, int B, char* ws, const WsLayout& wl, const float** out, hipStream_t s) {
  const Shape& sh = h->sh;
  const float* t0 = reinterpret_cast<const float*>(ws + wl.t0);
  *out = t0;
  if (!sh.score) return INCVIT_OK;
  float* kn = reinterpret_cast<float*>(ws + wl.kn);
  float* key = reinterpret_cast<float*>(ws + wl.key);
  const PackedLayer& L0 = h->pl.layers[0];
  KeyLnArgs ka{t0, fptr(h, L0.ln1_g), fptr(h, L0.ln1_b), kn, B * sh.N, sh.D, sh.dtype, sh.eps};
  incvit_status st = run(h, INCVIT_K_KEY_LN, s, [&] { return launch_keyln(ka, s); });
  if (st != INCVIT_OK) return st;
  EmbedArgs pa{kn, h->packed + h->pl.w_key, fptr(h, L0.b_qkv) + sh.D, nullptr, key,
               B, sh.N, sh.D, sh.D, sh.dtype, nullptr, 0, nullptr, nullptr};
  st = run(h, INCVIT_K_KEY_PROJ, s, [&] { return launch_keyproj(pa, s); });
  if (st != INCVIT_OK) return st;
  *out = key;
  return INCVIT_OK;
}

// Full forward of B frames.  idx/count (device) receive the identity row map
// (every token refreshed) when given, else the workspace's own copy does;
// refreshed (optional) receives Y of every token.
incvit_status full_impl(incvit_handle* h, int32_t B, const float* patches, void* const* caches, int32_t* out_idx,
                        int32_t* out_count, void* refreshed, void* workspace, void* stream) {
  incvit_status st = check_common(h, B, patches, workspace);
  if (st != INCVIT_OK) return st;
  if (reinterpret_cast<uintptr_t>(refreshed) % 16) return fail(h, INCVIT_ERR_ARG, "refreshed must be 16-byte aligned");
  Views views;
  if ((st = check_views(h, B, caches, views)) != INCVIT_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Shape& sh = h->sh;
  char* ws = static_cast<char*>(workspace);
  const WsLayout wl = ws_layout(sh, B);
  int* count = out_count ? out_count : reinterpret_cast<int*>(ws + wl.count);
  int* idx = out_idx ? out_idx : reinterpret_cast<int*>(ws + wl.idx);
  float* t0 = reinterpret_cast<float*>(ws + wl.t0);

  EmbedArgs ea{patches, h->packed + h->pl.w_pe, fptr(h, h->pl.b_pe), fptr(h, h->pl.pos), t0,
               B, sh.N, sh.P, sh.D, sh.dtype, nullptr, 0, idx, count};
  if ((st = run(h, INCVIT_K_EMBED, s, [&] { return launch_embed(ea, s); })) != INCVIT_OK) return st;
  const float* score = nullptr;
  if ((st = score_pass(h, B, ws, wl, &score, s)) != INCVIT_OK) return st;
  const int mmax = B * sh.N;
  RowsArgs ra;
  memset(&ra, 0, sizeof ra);
  ra.rm = RowMap{count, idx, B, sh.N};
  ra.rows = reinterpret_cast<RowInfo*>(ws + wl.rows);
  ra.meta = reinterpret_cast<Meta*>(ws + wl.meta);
  ra.caches = views;
  ra.cl = h->cl;
  ra.sh = sh;
  ra.t0 = t0;
  ra.score = score;
  ra.init_header = 1;
  ra.hash = h->hash;
  ra.z = ws + wl.z;
  set_all_rows(ra, sh, ws, wl, nullptr);
  if ((st = run(h, INCVIT_K_COMMIT, s, [&] { return launch_commit(ra, mmax, s); })) != INCVIT_OK) return st;
  return run_layers(h, views, B, wl, ws, sh.N, mmax, true, refreshed, s);
}

}  // namespace

extern "C" {

size_t incvit_canonical_weights_bytes(const incvit_config* cfg) {
  Shape sh;
  incvit_status st;
  std::string err;
  if (!make_shape(cfg, sh, st, err)) { g_error = err; return 0; }
  return canon_layout(sh).total * sh.eb;
}

size_t incvit_packed_weights_bytes(const incvit_config* cfg) {
  Shape sh;
  incvit_status st;
  std::string err;
  if (!make_shape(cfg, sh, st, err)) { g_error = err; return 0; }
  return packed_layout(sh).total;
}

incvit_status incvit_pack_weights(const incvit_config* cfg, const void* canonical, void* packed, void* stream) {
  Shape sh;
  incvit_status st;
  std::string err;
  if (!make_shape(cfg, sh, st, err)) return fail(nullptr, st, err);
  if (!canonical || !packed) return fail(nullptr, INCVIT_ERR_ARG, "null weight buffer");
  if (reinterpret_cast<uintptr_t>(packed) % kAlign || reinterpret_cast<uintptr_t>(canonical) % 16)
    return fail(nullptr, INCVIT_ERR_ARG, "packed must be 256-byte and canonical 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const PackedLayout pl = packed_layout(sh);
  const CanonLayout cn = canon_layout(sh);
  const char* src = static_cast<const char*>(canonical);
  char* dst = static_cast<char*>(packed);
  const size_t eb = sh.eb;
  hipError_t e = hipSuccess;
  auto conv = [&](size_t coff, size_t poff, long n, long npad) {
    if (e != hipSuccess) return;
    ConvArgs a{src + coff * eb, reinterpret_cast<float*>(dst + poff), n, npad, sh.dtype};
    e = launch_conv(a, s);
  };
  auto pack = [&](size_t coff, size_t poff, int K, int Ncols, int Kpad, int Npadc) {
    if (e != hipSuccess) return;
    PackArgs a{src + coff * eb, dst + poff, K, Ncols, round_up(Kpad, 32) / 32, round_up(Npadc, 16) / 16, sh.dtype};
    e = launch_pack(a, s);
  };
  // the LayerNorm (gamma, beta) before a GEMM folded into its packed weights
  auto fold = [&](size_t coff, size_t poff, size_t g, size_t b, size_t bias, size_t c1, size_t c2b, int K, int Ncols,
                  int Npadc) {
    if (e != hipSuccess) return;
    FoldArgs a{src + coff * eb, src + g * eb, src + b * eb, src + bias * eb, dst + poff,
               reinterpret_cast<float*>(dst + c1), reinterpret_cast<float*>(dst + c2b),
               K, Ncols, round_up(K, 32) / 32, round_up(Npadc, 16) / 16, sh.dtype};
    e = launch_fold(a, s);
  };
  const int D = sh.D;
  e = hipMemcpyAsync(dst + pl.w_pe, src + cn.w_pe * eb, (size_t)sh.P * D * eb, hipMemcpyDeviceToDevice, s);
  conv(cn.b_pe, pl.b_pe, D, D);
  conv(cn.pos, pl.pos, (long)sh.N * D, (long)sh.N * D);
  for (int l = 0; l < sh.L; ++l) {
    const PackedLayer& C = cn.layers[l];
    const PackedLayer& P = pl.layers[l];
    conv(C.ln1_g, P.ln1_g, D, D);
    conv(C.ln1_b, P.ln1_b, D, D);
    pack(C.w_qkv, P.w_qkv, D, 3 * D, D, 3 * D);
    fold(C.w_qkv, P.w_qkv, C.ln1_g, C.ln1_b, C.b_qkv, P.qkv_c1, P.qkv_c2b, D, 3 * D, 3 * D);
    conv(C.b_qkv, P.b_qkv, 3 * D, 3 * D);
    pack(C.w_o, P.w_o, D, D, D, D);
    conv(C.b_o, P.b_o, D, D);
    conv(C.ln2_g, P.ln2_g, D, D);
    conv(C.ln2_b, P.ln2_b, D, D);
    pack(C.w_1, P.w_1, D, sh.F, D, sh.Fpad);
    fold(C.w_1, P.w_1, C.ln2_g, C.ln2_b, C.b_1, P.fc1_c1, P.fc1_c2b, D, sh.F, sh.Fpad);
    conv(C.b_1, P.b_1, sh.F, sh.Fpad);
    pack(C.w_2, P.w_2, sh.F, D, sh.Fpad, D);
    conv(C.b_2, P.b_2, D, D);
  }
  conv(cn.lnf_g, pl.lnf_g, D, D);
  conv(cn.lnf_b, pl.lnf_b, D, D);
  // W_K of layer 0 as its own [D][D] matrix (columns D..2D-1 of W_qkv) for the key score
  if (e == hipSuccess)
    e = hipMemcpy2DAsync(dst + pl.w_key, (size_t)D * eb, src + (cn.layers[0].w_qkv + D) * eb, (size_t)3 * D * eb,
                         (size_t)D * eb, D, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return fail(nullptr, INCVIT_ERR_HIP, std::string("pack: ") + hipGetErrorString(e));
  return INCVIT_OK;
}

incvit_status incvit_create(const incvit_config* cfg, const void* packed_weights, incvit_handle** out) {
  if (!out) return fail(nullptr, INCVIT_ERR_ARG, "out is null");
  *out = nullptr;
  Shape sh;
  incvit_status st;
  std::string err;
  if (!make_shape(cfg, sh, st, err)) return fail(nullptr, st, err);
  if (!packed_weights || reinterpret_cast<uintptr_t>(packed_weights) % kAlign)
    return fail(nullptr, INCVIT_ERR_ARG, "packed weights must be non-null and 256-byte aligned");
  incvit_handle* h = new incvit_handle();
  h->cfg = *cfg;
  h->sh = sh;
  h->cl = cache_layout(sh);
  h->hash = config_hash(*cfg);
  h->packed = static_cast<const char*>(packed_weights);
  h->pl = packed_layout(sh);
  *out = h;
  return INCVIT_OK;
}

void incvit_destroy(incvit_handle* h) {
  if (!h) return;
  for (auto& r : h->recs) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
  }
  for (auto e : h->pool) hipEventDestroy(e);
  delete h;
}

size_t incvit_cache_bytes(const incvit_handle* h) { return h ? h->cl.total : 0; }

size_t incvit_cache_canonical_bytes(const incvit_handle* h) {
  if (!h) return 0;
  const Shape& sh = h->sh;
  const size_t nd = (size_t)sh.N * sh.D;
  return nd * 4 + ((size_t)(sh.L + 1) * nd + 2 * (size_t)sh.L * nd + nd + (sh.mlp_all ? (size_t)sh.L * nd : 0)) * sh.eb;
}

size_t incvit_workspace_bytes(const incvit_handle* h, int32_t B) {
  if (!h || B < 1 || B > h->cfg.max_streams) return 0;
  return ws_layout(h->sh, B).total;
}

incvit_status incvit_full_encode(incvit_handle* h, int32_t B, const float* patches, void* const* caches,
                                 void* workspace, void* stream) {
  return full_impl(h, B, patches, caches, nullptr, nullptr, nullptr, workspace, stream);
}

incvit_status incvit_step(incvit_handle* h, int32_t B, const float* patches, void* const* caches, float tau,
                          const int32_t* cap, int32_t* idx, int32_t* count, void* refreshed, void* workspace,
                          void* stream) {
  incvit_status st = check_common(h, B, patches, workspace);
  if (st != INCVIT_OK) return st;
  if (std::isnan(tau)) return fail(h, INCVIT_ERR_ARG, "tau is NaN");
  if (!cap) return fail(h, INCVIT_ERR_ARG, "cap is null");
  if (!idx || !count) return fail(h, INCVIT_ERR_ARG, "idx and count must be non-null");
  if (reinterpret_cast<uintptr_t>(refreshed) % 16) return fail(h, INCVIT_ERR_ARG, "refreshed must be 16-byte aligned");
  Views views;
  if ((st = check_views(h, B, caches, views)) != INCVIT_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Shape& sh = h->sh;
  char* ws = static_cast<char*>(workspace);
  const WsLayout wl = ws_layout(sh, B);
  float* t0 = reinterpret_cast<float*>(ws + wl.t0);
  float* sim = reinterpret_cast<float*>(ws + wl.sim);

  SelectArgs sa;
  memset(&sa, 0, sizeof sa);
  int mmax = 0, max_rows = 0;
  for (int v = 0; v < B; ++v) {
    const int c = std::min(std::max(cap[v], 0), sh.N);
    sa.cap[v] = c;
    mmax += c;
    max_rows = std::max(max_rows, c);
  }
  EmbedArgs ea{patches, h->packed + h->pl.w_pe, fptr(h, h->pl.b_pe), fptr(h, h->pl.pos), t0,
               B, sh.N, sh.P, sh.D, sh.dtype, nullptr, 0, nullptr, nullptr};
  if ((st = run(h, INCVIT_K_EMBED, s, [&] { return launch_embed(ea, s); })) != INCVIT_OK) return st;
  const float* score = nullptr;
  if ((st = score_pass(h, B, ws, wl, &score, s)) != INCVIT_OK) return st;
  SimArgs si{score, views, h->cl.ref, sim, B, sh.N, sh.D};
  if ((st = run(h, INCVIT_K_SIM, s, [&] { return launch_sim(si, s); })) != INCVIT_OK) return st;
  sa.sim = sim;
  sa.caches = views;
  sa.B = B;
  sa.N = sh.N;
  sa.tau = tau;
  sa.hash = h->hash;
  sa.idx = idx;
  sa.count = count;
  sa.valid = reinterpret_cast<int*>(ws + wl.valid);
  if ((st = run(h, INCVIT_K_SELECT, s, [&] { return launch_select(sa, s); })) != INCVIT_OK) return st;
  // nothing can be selected: done (with mlp_all every row still follows the frame)
  if (mmax == 0 && !sh.mlp_all) return INCVIT_OK;

  RowsArgs ra;
  memset(&ra, 0, sizeof ra);
  ra.rm = RowMap{count, idx, B, sh.N};
  ra.rows = reinterpret_cast<RowInfo*>(ws + wl.rows);
  ra.meta = reinterpret_cast<Meta*>(ws + wl.meta);
  ra.caches = views;
  ra.cl = h->cl;
  ra.sh = sh;
  ra.t0 = t0;
  ra.score = score;
  ra.z = ws + wl.z;
  set_all_rows(ra, sh, ws, wl, sa.valid);
  if ((st = run(h, INCVIT_K_COMMIT, s, [&] { return launch_commit(ra, mmax, s); })) != INCVIT_OK) return st;
  // with the threshold disabled every stream refreshes exactly its cap
  return run_layers(h, views, B, wl, ws, max_rows, mmax, std::isinf(tau) && tau > 0, refreshed, s);
}

incvit_status incvit_encode_frame(incvit_handle* h, int32_t B, const float* patches, void* const* caches,
                                  int64_t frame_index, int32_t period, float tau, const int32_t* cap, int32_t* idx,
                                  int32_t* count, void* refreshed, void* workspace, void* stream) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  if (period < 1) return fail(h, INCVIT_ERR_ARG, "period must be >= 1");
  if (frame_index < 0) return fail(h, INCVIT_ERR_ARG, "frame_index must be >= 0");
  if (frame_index % period == 0) {
    if (!idx || !count) return fail(h, INCVIT_ERR_ARG, "idx and count must be non-null");
    return full_impl(h, B, patches, caches, idx, count, refreshed, workspace, stream);
  }
  return incvit_step(h, B, patches, caches, tau, cap, idx, count, refreshed, workspace, stream);
}

}  // extern "C"

// Workspace of incvit_step_noalloc: one file-scope device array.  Each GPU the
// library runs on holds its own copy (at its own address) until the process
// ends.  Host code never uses the array's name as an address: its device
// address is resolved once per device with hipGetSymbolAddress and kept.
static __device__ __align__(256) char scratch[INCVIT_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The current device's copy of `scratch`, resolved on its first use.
incvit_status scratch_of_current_device(incvit_handle* h, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(h, INCVIT_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(h, INCVIT_ERR_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(h, INCVIT_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return INCVIT_OK;
}
}  // namespace

extern "C" {

incvit_status incvit_step_noalloc(incvit_handle* h, int32_t B, const float* patches, void* const* caches, float tau,
                                  const int32_t* cap, int32_t* idx, int32_t* count, void* refreshed, void* stream) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  if (B < 1 || B > h->cfg.max_streams) return fail(h, INCVIT_ERR_ARG, "B must be in [1, max_streams]");
  const size_t need = ws_layout(h->sh, B).total;
  if (need > (size_t)INCVIT_NOALLOC_SCRATCH_BYTES) {
    char buf[256];
    snprintf(buf, sizeof buf,
             "a step of %d stream(s) needs %zu bytes of workspace, beyond the %d-byte static scratch of "
             "incvit_step_noalloc: call incvit_step with a workspace",
             B, need, INCVIT_NOALLOC_SCRATCH_BYTES);
    return fail(h, INCVIT_ERR_ARG, buf);
  }
  void* ws = nullptr;
  incvit_status st = scratch_of_current_device(h, &ws);
  if (st != INCVIT_OK) return st;
  // no per-kernel profiling events here: creating one may allocate
  const bool prof = h->prof;
  h->prof = false;
  st = incvit_step(h, B, patches, caches, tau, cap, idx, count, refreshed, ws, stream);
  h->prof = prof;
  return st;
}

incvit_status incvit_flow_two_anchor(int32_t S, int64_t n, const float* x0, const float* v0, const float* v7,
                                     const float* alpha, const float* beta, const float* b, float* xT, void* stream) {
  if (S < 1 || n < 1) return fail(nullptr, INCVIT_ERR_ARG, "S and n must be >= 1");
  if (!x0 || !v0 || !v7 || !alpha || !beta || !b || !xT) return fail(nullptr, INCVIT_ERR_ARG, "null buffer");
  FlowArgs a{x0, v0, v7, alpha, beta, b, xT, S, (long)n};
  const hipError_t e = launch_flow(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(nullptr, INCVIT_ERR_HIP, std::string("flow: ") + hipGetErrorString(e));
  return INCVIT_OK;
}

incvit_status incvit_cache_export(const incvit_handle* h, const void* cache, void* canonical_dst, void* stream) {
  if (!h || !cache || !canonical_dst) return fail(const_cast<incvit_handle*>(h), INCVIT_ERR_ARG, "null argument");
  ExportArgs a{static_cast<const char*>(cache), static_cast<char*>(canonical_dst), h->cl, h->sh, 1, h->hash};
  const hipError_t e = launch_export(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(const_cast<incvit_handle*>(h), INCVIT_ERR_HIP, hipGetErrorString(e));
  return INCVIT_OK;
}

incvit_status incvit_cache_import(const incvit_handle* h, const void* canonical_src, void* cache, void* stream) {
  if (!h || !cache || !canonical_src) return fail(const_cast<incvit_handle*>(h), INCVIT_ERR_ARG, "null argument");
  ExportArgs a{static_cast<char*>(cache), static_cast<char*>(const_cast<void*>(canonical_src)), h->cl, h->sh, 0, h->hash};
  const hipError_t e = launch_export(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(const_cast<incvit_handle*>(h), INCVIT_ERR_HIP, hipGetErrorString(e));
  return INCVIT_OK;
}

incvit_status incvit_cache_status(const incvit_handle* h, const void* cache, void* stream) {
  if (!h || !cache) return fail(const_cast<incvit_handle*>(h), INCVIT_ERR_ARG, "null argument");
  CacheHeader hdr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(&hdr, cache, sizeof hdr, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(const_cast<incvit_handle*>(h), INCVIT_ERR_HIP, hipGetErrorString(e));
  if (hdr.magic != kCacheMagic || hdr.hash != h->hash) return INCVIT_ERR_STATE;
  if (hdr.status == kStatusNonFinite) return INCVIT_ERR_ARG;
  return hdr.status == 0 ? INCVIT_OK : INCVIT_ERR_STATE;
}

const char* incvit_last_error(const incvit_handle* h) { return h ? h->err.c_str() : g_error.c_str(); }

incvit_status incvit_profile_enable(incvit_handle* h, int32_t enable) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  h->prof = enable != 0;
  return INCVIT_OK;
}

incvit_status incvit_profile_read(incvit_handle* h, double* total_ms, int64_t* launches, int32_t reset) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  for (auto& r : h->recs) {
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return fail(h, INCVIT_ERR_HIP, hipGetErrorString(e));
    h->prof_ms[r.kind] += ms;
    h->prof_n[r.kind] += 1;
    h->pool.push_back(r.a);
    h->pool.push_back(r.b);
  }
  h->recs.clear();
  for (int k = 0; k < INCVIT_K_COUNT; ++k) {
    if (total_ms) total_ms[k] = h->prof_ms[k];
    if (launches) launches[k] = h->prof_n[k];
    if (reset) {
      h->prof_ms[k] = 0.0;
      h->prof_n[k] = 0;
    }
  }
  return INCVIT_OK;
}

incvit_status incvit_set_tuning(incvit_handle* h, const incvit_tuning* t) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  for (int k = 0; k < 4; ++k) {
    const int c = t ? t->cols[k] : 0;
    if (c < 0 || c > 4 || c == 3) return fail(h, INCVIT_ERR_ARG, "cols must be 0, 1, 2 or 4");
  }
  const int q = t ? t->attn_qtiles : 0;
  if (q < 0 || q > 2) return fail(h, INCVIT_ERR_ARG, "attn_qtiles must be 0, 1 or 2");
  const int rg = t ? t->row_groups : 0;
  if (rg < 0 || rg > 8) return fail(h, INCVIT_ERR_ARG, "row_groups must be in [0, 8]");
  const int aw = t ? t->attn_waves : 0;
  if (aw != 0 && aw != 2 && aw != 4 && aw != 8) return fail(h, INCVIT_ERR_ARG, "attn_waves must be 0, 2, 4 or 8");
  const int fm = t ? t->fc2_mode : 0;
  if (fm < 0 || fm > 2) return fail(h, INCVIT_ERR_ARG, "fc2_mode must be 0, 1 or 2");
  const int tl = t ? t->tiled : 0;
  if (tl < 0 || tl > 1) return fail(h, INCVIT_ERR_ARG, "tiled must be 0 or 1");
  for (int k = 0; k < 4; ++k) h->cols[k] = t ? t->cols[k] : 0;
  h->attn_qtiles = q;
  h->row_groups = rg > 0 ? rg : 1;
  h->attn_waves = aw;
  h->fc2_mode = fm;
  h->tiled = tl;
  return INCVIT_OK;
}

}  // extern "C"

namespace {
template <class F>
incvit_status capture(incvit_handle* h, incvit_graph** out, F&& body) {
  if (!out) return fail(h, INCVIT_ERR_ARG, "out is null");
  *out = nullptr;
  hipStream_t cs = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
  if (e != hipSuccess) return fail(h, INCVIT_ERR_HIP, std::string("hipStreamCreate: ") + hipGetErrorString(e));
  const bool prof = h->prof;
  h->prof = false;
  incvit_graph* g = new incvit_graph();
  incvit_status st = INCVIT_OK;
  e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
  if (e == hipSuccess) {
    st = body(cs);
    const hipError_t e2 = hipStreamEndCapture(cs, &g->graph);
    if (st == INCVIT_OK && e2 != hipSuccess) e = e2;
  }
  if (st == INCVIT_OK && e == hipSuccess) e = hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0);
  h->prof = prof;
  hipStreamDestroy(cs);
  if (st != INCVIT_OK || e != hipSuccess) {
    if (g->exec) hipGraphExecDestroy(g->exec);
    if (g->graph) hipGraphDestroy(g->graph);
    delete g;
    if (st != INCVIT_OK) return st;
    return fail(h, INCVIT_ERR_HIP, std::string("graph capture: ") + hipGetErrorString(e));
  }
  *out = g;
  return INCVIT_OK;
}
}  // namespace

extern "C" {

incvit_status incvit_step_graph_create(incvit_handle* h, int32_t B, const float* patches, void* const* caches,
                                       float tau, const int32_t* cap, int32_t* idx, int32_t* count,
                                       void* refreshed, void* workspace, incvit_graph** out) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  return capture(h, out, [&](hipStream_t cs) {
    return incvit_step(h, B, patches, caches, tau, cap, idx, count, refreshed, workspace, cs);
  });
}

incvit_status incvit_full_graph_create(incvit_handle* h, int32_t B, const float* patches, void* const* caches,
                                       void* workspace, incvit_graph** out) {
  if (!h) return fail(nullptr, INCVIT_ERR_ARG, "null handle");
  return capture(h, out, [&](hipStream_t cs) { return incvit_full_encode(h, B, patches, caches, workspace, cs); });
}

incvit_status incvit_graph_launch(incvit_graph* g, void* stream) {
  if (!g || !g->exec) return fail(nullptr, INCVIT_ERR_ARG, "null graph");
  const hipError_t e = hipGraphLaunch(g->exec, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(nullptr, INCVIT_ERR_HIP, std::string("hipGraphLaunch: ") + hipGetErrorString(e));
  return INCVIT_OK;
}

void incvit_graph_destroy(incvit_graph* g) {
  if (!g) return;
  if (g->exec) hipGraphExecDestroy(g->exec);
  if (g->graph) hipGraphDestroy(g->graph);
  delete g;
}

}  // extern "C"
