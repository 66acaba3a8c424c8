/*
 * incvit: incremental ViT encoding of streaming camera frames on MI355X (gfx950).
 *
 * The method (paper §III-B, "Temporal Token Reuse"): for each new frame every
 * token is scored by the cosine similarity of its current and cached
 * representation (eq. 3); the least similar tokens form the updated set U and
 * are recomputed through every layer -- Q, K, V only for U (eq. 4), the new K/V
 * rows scattered into the cached full K/V (eq. 5), attention only for the
 * updated queries over all N keys, then the residual and the MLP -- while the
 * other tokens reuse their cached outputs.  The index set is chosen once,
 * before the first layer, and reused by every layer.
 *
 * Readings taken where the paper is silent (each is an argument of this API or
 * fixed here):
 *   - the score is the cosine of a per-token vector against that token's
 *     vector at its last refresh, computed in a fixed fp32 order so that
 *     selection is reproducible bit for bit.  The vector is, per config
 *     (incvit_score), either the layer-1 input token (patch embedding +
 *     position) or the first layer's key of that token, as eq. 3 states it;
 *   - the paper's odd/even chunks (a full pass on odd chunks whose keys become
 *     the reference, incremental encoding on even chunks) are
 *     incvit_encode_frame with period 2; between full passes every refreshed
 *     token's vector becomes its new reference;
 *   - the statement that every token goes through the MLP is read exactly by default
 *     (a reused row's MLP input is its cached state, so only U is computed);
 *     cfg.mlp_all = 1 selects the non-exact reading: every frame, every row
 *     starts from this frame's embedded token, reused rows add their cached
 *     attention-branch output S(O W_o + b_o) of each layer to their current
 *     residual stream, and the MLP runs over all rows (their K and V stay
 *     cached; their outputs follow the new frame);
 *   - the rule of refreshing the rho*N least similar tokens is generalised to: U = {i : sim_i < tau}
 *     (strict), and if |U| > cap only the cap lowest similarities are kept,
 *     equal similarities going to the lower token index.  tau = +INFINITY with
 *     cap = round(rho*N) is the paper's top-rho*N rule;
 *   - the encoder is a pre-LN ViT without CLS token: learned positions added
 *     after the patch embedding, biased linear layers, LayerNorm with biased
 *     variance, tanh GELU, attention scaled by 1/sqrt(d_h), final LayerNorm.
 *
 * Conventions for every entry point:
 *   - every buffer argument is DEVICE memory owned by the caller, except
 *     `cap` of incvit_step and the config / handle structs, which are host;
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream); work
 *     is enqueued asynchronously on it and results are valid after the caller
 *     synchronises it; no entry point below synchronises unless it says so;
 *   - argument and shape errors are returned before anything is enqueued;
 *     HIP launch errors return INCVIT_ERR_HIP; incvit_last_error() gives text;
 *   - a handle is not thread-safe; handles are independent of each other;
 *   - the library allocates no device memory: weights, caches, workspace,
 *     inputs and outputs are all passed in.
 */
#ifndef INCVIT_H_
#define INCVIT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  INCVIT_OK = 0,
  INCVIT_ERR_ARG = -1,         /* null pointer, bad count, NaN tau, ...          */
  INCVIT_ERR_SHAPE = -2,       /* inconsistent model shape                        */
  INCVIT_ERR_UNSUPPORTED = -3, /* shape valid but outside what the kernels cover  */
  INCVIT_ERR_STATE = -4,       /* cache not initialised or from another model     */
  INCVIT_ERR_HIP = -5          /* a HIP call failed                               */
} incvit_status;

typedef enum { INCVIT_F32 = 0, INCVIT_BF16 = 1 } incvit_dtype;

/* What the cosine of eq. 3 compares, per token (both in fp32, fixed order):
 *   INCVIT_SCORE_EMBED: T[i] = patch embedding + position (the layer-1 input);
 *   INCVIT_SCORE_KEY:   the first layer's key, LN1(S(T[i])) W_K + b_K with
 *     layer 0's LayerNorm and key columns, S = rounding to the storage type:
 *     mean and variance from 64 lane partials (lane j takes d = j, j+64, ...
 *     in increasing d; the sum with adds, the squares of x - mean with fma)
 *     combined by the halving tree 32,16,..,1, each divided by D;
 *     rstd = 1 / sqrt(var + eps); n_d = fma((x_d - mean) * rstd, gamma_d, beta_d);
 *     key_e = fma chain over d = 0..D-1 of n_d * W_K[d][e] started at b_K[e].
 *     Costs D*D fma per token more than the embedding score. */
typedef enum { INCVIT_SCORE_EMBED = 0, INCVIT_SCORE_KEY = 1 } incvit_score;

/* Model and limits.  N = (img_h/patch)*(img_w/patch) tokens, P = channels*patch^2
 * patch features, D = dim, L = depth, h = heads, d_h = D/h, F = mlp_dim.
 * Supported: img_h, img_w multiples of patch; D % 32 == 0; D % h == 0;
 * d_h % 8 == 0 and d_h <= 128; N <= 4096; D <= 2048; F >= 1;
 * 1 <= max_streams <= 64; and every buffer one kernel addresses below 4 GiB:
 * N*P*4 bytes (one stream's patches), P*D*e (W_pe), max(3D, F)*max(D, F)*e (a
 * packed GEMM matrix) and max_streams*N*max(D, F)*e (the widest compact GEMM
 * operand), e = 2 (bf16) or 4 (f32); otherwise INCVIT_ERR_UNSUPPORTED.
 * dtype is the storage type of weights, caches and activations (GEMMs
 * accumulate in fp32; LayerNorm, softmax, GELU in fp32). */
typedef struct {
  int32_t img_h, img_w, channels, patch;
  int32_t dim, depth, heads, mlp_dim;
  int32_t dtype;       /* incvit_dtype */
  float ln_eps;        /* e.g. 1e-6 */
  int32_t max_streams; /* largest B accepted by a call */
  int32_t score;       /* incvit_score; part of the cache identity */
  int32_t mlp_all;     /* 0: exact reuse (default); 1: every row through the MLP
                          each frame (see above); part of the cache identity */
} incvit_config;

typedef struct incvit_handle incvit_handle;

/* ---------------------------------------------------------------- weights -- */

/* Bytes of the canonical weight buffer: the parameters below, in this order,
 * each row-major, each element of the storage dtype:
 *   W_pe [P][D] (row (c*p + dy)*p + dx), b_pe [D], Pos [N][D],
 *   per layer l = 0..L-1: ln1_g [D], ln1_b [D], W_qkv [D][3D] (columns
 *     [0,D) Q, [D,2D) K, [2D,3D) V; head j owns columns [j*d_h,(j+1)*d_h) of
 *     each block), b_qkv [3D], W_o [D][D], b_o [D], ln2_g [D], ln2_b [D],
 *     W_1 [D][F], b_1 [F], W_2 [F][D], b_2 [D],
 *   lnf_g [D], lnf_b [D].
 * Every linear layer computes y = x W + b.  Returns 0 for an invalid config. */
size_t incvit_canonical_weights_bytes(const incvit_config* cfg);

/* Bytes of the packed (device-layout) weight buffer.  0 for an invalid config. */
size_t incvit_packed_weights_bytes(const incvit_config* cfg);

/* Repack canonical weights (device) into the kernels' layout (device):
 * GEMM weights in 16-column x 32-row MFMA operand chunks, vectors in fp32.
 * The LayerNorm before the QKV and MLP-up projections is folded into their
 * packed weights: W' = S(gamma * W) row by row, with the column sums of W' and
 * beta^T W + b stored beside them (the encoder then computes
 * LN(x) W + b = rstd (x W') - rstd mean colsum(W') + beta^T W + b).
 * The two buffers must not overlap.  Asynchronous on `stream`. */
incvit_status incvit_pack_weights(const incvit_config* cfg, const void* canonical,
                                  void* packed, void* stream);

/* ----------------------------------------------------------------- handle -- */

/* Validate cfg and bind the packed weights (which must outlive the handle and
 * not change while it is used).  No device allocation.  On failure *out is
 * NULL and incvit_last_error(NULL) describes the problem. */
incvit_status incvit_create(const incvit_config* cfg, const void* packed_weights,
                            incvit_handle** out);

void incvit_destroy(incvit_handle* h);

/* Bytes of one stream's cache (device layout, 256-byte aligned parts): a header
 * (magic, config hash, status word), ref [N][D] fp32 (each token's score
 * vector -- embedding or first-layer key, per cfg.score -- at its last
 * refresh), X [L+1][N][D] (layer inputs), K and V of every layer, Y [N][D]
 * (final output), and with mlp_all A [L][N][D] (attention-branch outputs).
 * Base addresses must be 256-byte aligned. */
size_t incvit_cache_bytes(const incvit_handle* h);

/* Bytes of one stream's cache in the canonical (export) layout:
 * ref [N][D] fp32, then in the storage dtype X [L+1][N][D], K [L][N][D],
 * V [L][N][D], Y [N][D], and with mlp_all A [L][N][D]. */
size_t incvit_cache_canonical_bytes(const incvit_handle* h);

/* Bytes of workspace a call with B streams needs (256-byte aligned base). */
size_t incvit_workspace_bytes(const incvit_handle* h, int32_t B);

/* ----------------------------------------------------------------- encode -- */

/* Full forward of B frames (the paper's full pass on odd chunks, §III-B):
 * patches [B][N][P] fp32 (frame pixels, token-major, features (c, dy, dx));
 * caches: host array of B device pointers, one cache per stream (B distinct
 * buffers that do not overlap, else INCVIT_ERR_ARG); every cache row is
 * (re)written and the cache header is initialised for this model.
 * workspace: incvit_workspace_bytes(h, B) bytes, device. */
incvit_status incvit_full_encode(incvit_handle* h, int32_t B, const float* patches,
                                 void* const* caches, void* workspace, void* stream);

/* Incremental encode of B frames (§III-B, eqs. 3-5).  For each stream v:
 * U_v is selected from this frame's patches against the cache (tau, cap[v]),
 * rows U_v are recomputed through every layer and written into the cache
 * (ref, X, K, V, Y); all other rows are left untouched.  With mlp_all the
 * rows U_v get new ref, K, V and A rows, and every row of X and Y is
 * recomputed (also when U_v is empty); `refreshed` still receives Y[U_v].
 *   tau: threshold (not NaN; +INFINITY disables it);
 *   cap: HOST int32[B], each clamped to [0, N];
 *   idx: device int32 [B][N]; idx[v][0..count[v]) = U_v ascending;
 *   count: device int32 [B];
 *   refreshed: device [B][N][D] storage dtype; rows 0..count[v] of stream v
 *     receive Y[U_v] (the new outputs of the refreshed tokens); may be NULL.
 * No host synchronisation inside.  A cache that was never full-encoded, or was
 * encoded by a different model, or a frame whose similarity is NaN, makes that
 * stream's step a no-op (count = 0) and sets the cache's status word; read it
 * with incvit_cache_status. */
incvit_status incvit_step(incvit_handle* h, int32_t B, const float* patches,
                          void* const* caches, float tau, const int32_t* cap,
                          int32_t* idx, int32_t* count, void* refreshed,
                          void* workspace, void* stream);

/* One frame of a stream under a refresh period (§III-B, odd/even chunks for
 * period 2): if frame_index % period == 0 the frame is encoded in full (every
 * cache row and reference replaced) and reported as a step that refreshed
 * every token: idx[v][i] = i, count[v] = N, refreshed rows = Y; otherwise it
 * is incvit_step with the same arguments.  period >= 1, frame_index >= 0
 * (host values).  Same buffers, errors and asynchrony as incvit_step. */
incvit_status incvit_encode_frame(incvit_handle* h, int32_t B, const float* patches,
                                  void* const* caches, int64_t frame_index, int32_t period,
                                  float tau, const int32_t* cap, int32_t* idx, int32_t* count,
                                  void* refreshed, void* workspace, void* stream);

/* Incremental encode without any allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): incvit_step with the workspace taken from
 * a static device array of INCVIT_NOALLOC_SCRATCH_BYTES (64 MiB) that the
 * library holds on each GPU it runs on until the process ends (its address is
 * resolved on the first call on a device).  Arguments, results, errors and
 * kernels are those of incvit_step; the caller still passes inputs, caches and
 * outputs.  A call whose workspace (incvit_workspace_bytes(h, B)) exceeds the
 * array returns INCVIT_ERR_ARG before anything is enqueued (64 MiB holds up to
 * seven streams of a So400m-shaped model at 224x224, 8.9 MiB each, one at
 * 448x448, 35.5 MiB, or four ViT-L streams at 224x224, 36 MiB).
 * No part of the array needs to start at zero: every call writes what it
 * reads.  Every call on one GPU shares that GPU's array: calls that overlap in
 * time on one GPU (other host threads, other streams) race and must be
 * serialised by the caller.  Per-kernel profiling is not recorded. */
#define INCVIT_NOALLOC_SCRATCH_BYTES (64 << 20)
incvit_status incvit_step_noalloc(incvit_handle* h, int32_t B, const float* patches,
                                  void* const* caches, float tau, const int32_t* cap,
                                  int32_t* idx, int32_t* count, void* refreshed,
                                  void* stream);

/* ----------------------------------------------------------- cache state -- */

/* Copy a cache into the canonical layout (incvit_cache_canonical_bytes). */
incvit_status incvit_cache_export(const incvit_handle* h, const void* cache,
                                  void* canonical_dst, void* stream);

/* Fill a cache from the canonical layout and mark it valid for this model. */
incvit_status incvit_cache_import(const incvit_handle* h, const void* canonical_src,
                                  void* cache, void* stream);

/* Synchronises `stream`, then returns the cache's status: INCVIT_OK,
 * INCVIT_ERR_STATE (never encoded / other model) or INCVIT_ERR_ARG (a step saw
 * a non-finite similarity). */
incvit_status incvit_cache_status(const incvit_handle* h, const void* cache, void* stream);

/* Text of the last error on h (or of the last failed create/size query when
 * h is NULL).  Valid until the next call on h. */
const char* incvit_last_error(const incvit_handle* h);

/* ----------------------------------------------------------- action side -- */

/* The compressed 2-step flow update of the action expert (§III-C): with the
 * solver's step velocities modelled by two anchors (the first, v_0, and a
 * mid-trajectory one, v_7), the Euler sum reduces to, for each of S samples,
 *   x_T[s] = x_0[s] + alpha[s] v_0[s] + beta[s] v_7[s] + b[s],
 * elementwise over the n values of a sample (an action chunk: horizon x action
 * dimensions).  The coefficients come from the caller (the paper predicts them
 * with a trained adaptor from v_0).  All device fp32: x0, v0, v7, b, xT [S][n];
 * alpha, beta [S]; xT may alias x0, no other overlap.  Evaluated as
 * fma(beta, v7, fma(alpha, v0, x0)) + b.  S >= 1, n >= 1, pointers non-null,
 * else INCVIT_ERR_ARG before anything is enqueued (text: incvit_last_error(NULL)).
 * Asynchronous on `stream`. */
incvit_status incvit_flow_two_anchor(int32_t S, int64_t n, const float* x0, const float* v0,
                                     const float* v7, const float* alpha, const float* beta,
                                     const float* b, float* xT, void* stream);

/* ------------------------------------------------------------ HIP graphs -- */

typedef struct incvit_graph incvit_graph;

/* Capture one incvit_step (same arguments, no stream) into a HIP graph, for
 * callers that encode frame after frame with fixed buffers: write the next
 * frame into `patches` (on the stream you launch on), then incvit_graph_launch.
 * The buffers, caches, tau and caps are baked in and must stay valid.  The
 * graph holds no memory operations other than kernels, so it is safe to
 * replay any number of times; one graph must not run concurrently with
 * itself or with other work on the same caches or workspace. */
incvit_status incvit_step_graph_create(incvit_handle* h, int32_t B, const float* patches,
                                       void* const* caches, float tau, const int32_t* cap,
                                       int32_t* idx, int32_t* count, void* refreshed,
                                       void* workspace, incvit_graph** out);

/* Same for incvit_full_encode. */
incvit_status incvit_full_graph_create(incvit_handle* h, int32_t B, const float* patches,
                                       void* const* caches, void* workspace, incvit_graph** out);

/* Enqueue a captured graph on `stream`. */
incvit_status incvit_graph_launch(incvit_graph* g, void* stream);

void incvit_graph_destroy(incvit_graph* g);

/* ---------------------------------------------------------------- tuning -- */

/* Performance knobs; every setting gives a deterministic result, and the
 * settings differ only in the order of fp32 partial sums.
 * cols[k]: 16-column blocks per workgroup of GEMM k (0 = QKV, 1 = output
 * projection, 2 = MLP up, 3 = MLP down): 1, 2 or 4 (a count takes effect only
 * when it divides the output's block count; 4 only for bf16 models, fp32 ones
 * take 2); 0 = automatic: with one row group (threshold steps without
 * row_groups) one block, two for outputs of more than 256 blocks; with
 * several (full encodes, pure top-k steps, or row_groups > 1) four for QKV and
 * for the MLP down projection when it runs unsplit (fc2_mode), unless the call
 * has more than 1024 rows known on the host, two for the
 * output projection and the K-split down projection, and for the MLP up
 * projection from 1536 rows.
 * attn_qtiles: 16-query tiles per attention workgroup: 1 or 2; 0 = automatic
 * (two when many streams and heads would still fill the CUs, or when the rows
 * are known on the host, the stream has 512 tokens or more and two-tile
 * workgroups still number 256 or more).
 * attn_waves: waves per attention workgroup, splitting the stream's keys: 2, 4
 * or 8; 0 = automatic (about two 32-key blocks per wave).
 * fc2_mode: the MLP down projection of every layer but the last: 1 = K split
 * over workgroups, partial sums finished by a row kernel; 2 = whole K per
 * workgroup with the residual and the cache write in its epilogue; 0 = 2 when
 * the call's row count is known on the host (full encodes, pure top-k steps)
 * and at least 192, else 1.
 * row_groups: 32-row groups per GEMM launch in steps with a finite threshold
 * (1..8; 0 = 1): a caller that expects about R refreshed rows per call can set
 * ceil(R / 32).  Full encodes and pure top-k steps (tau = +inf), whose row
 * count is known, choose it themselves.  With at most 6 groups each GEMM keeps
 * only as many as its workgroups fill the chip once (QKV in four-block
 * workgroups: one per CU; MLP up projection: two per CU; K-split MLP down
 * projection: one per CU; output projection: all), the rest looping over the
 * row blocks.
 * tiled: the large-row GEMM of bf16 models (output tiles of 64 or 128 rows
 * by 128 columns, K staged through LDS), used where the call's row count is
 * known on the host and at least 512 (full encodes of several streams or of
 * 448x448 frames, pure top-k steps of that many rows, the all-rows MLP):
 * 0 = automatic (used there; the output projection only once its 64-row
 * tiles number 256 or more), 1 = never (the weight-streaming GEMM above).
 * The cols and row_groups fields do not apply to its launches; its MLP down
 * projection follows fc2_mode (1: split over K with the row kernel, 2:
 * unsplit; 0: split while its 64-row tiles give fewer than 256 workgroups).
 * A NULL pointer restores the defaults. */
typedef struct {
  int32_t cols[4];
  int32_t attn_qtiles;
  int32_t row_groups;
  int32_t attn_waves;
  int32_t fc2_mode;
  int32_t tiled;
} incvit_tuning;

incvit_status incvit_set_tuning(incvit_handle* h, const incvit_tuning* t);

/* ------------------------------------------------------------- profiling -- */

/* Kernel kinds for the per-kernel timers. */
typedef enum {
  INCVIT_K_EMBED = 0, /* patch embedding + position, all tokens            */
  INCVIT_K_SIM,       /* cosine against the cached reference              */
  INCVIT_K_SELECT,    /* threshold / top-k selection and compaction      */
  INCVIT_K_COMMIT,    /* ref, X0 of the selected rows; LN1 of layer 0     */
  INCVIT_K_QKV,       /* LN1 + QKV projection, K/V scattered into cache   */
  INCVIT_K_ATTN,      /* attention of the selected queries                */
  INCVIT_K_OPROJ,     /* output projection + residual -> H                */
  INCVIT_K_FC1,       /* LN2 + MLP up projection + GELU                   */
  INCVIT_K_FC2,       /* MLP down projection (split-K partial sums)       */
  INCVIT_K_RES_LN1,   /* + bias + residual -> X^{l+1}; final LN (last)    */
  INCVIT_K_KEY_LN,    /* key score: LayerNorm 1 of layer 0, all tokens    */
  INCVIT_K_KEY_PROJ,  /* key score: key projection, all tokens            */
  INCVIT_K_HSUM,      /* mlp_all: H = X + cached attention branch, all rows */
  INCVIT_K_COUNT
} incvit_kernel_kind;

/* When enabled, every kernel launch of the encode calls records a start and a
 * stop event with its own dispatch on the call's stream (no extra stream
 * operations); incvit_profile_read synchronises those events and returns, per
 * kind, the summed duration (ms) and the number of launches since the last
 * reset. */
incvit_status incvit_profile_enable(incvit_handle* h, int32_t enable);
incvit_status incvit_profile_read(incvit_handle* h, double* total_ms /* [INCVIT_K_COUNT] */,
                                  int64_t* launches /* [INCVIT_K_COUNT] */, int32_t reset);

#ifdef __cplusplus
}
#endif
#endif /* INCVIT_H_ */
