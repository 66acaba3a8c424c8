/*
 * CPU oracle, fp32 part: patch embedding and the per-token cosine similarity
 * that decides which tokens are refreshed.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link or call this
 * file; only the tests, the smoke check and the benchmark's CPU baseline do.
 *
 * The paper scores each token by the cosine of its current and cached
 * representation (§III-B, eq. 3) and refreshes the least similar ones.  Token
 * selection must come out identical on the GPU and here, so this part is
 * computed in a fixed fp32 order, written out step by step:
 *
 *   T[i][d] = (b_pe[d] (+) x_i[0]*W[0][d] (+) ... (+) x_i[P-1]*W[P-1][d]) + Pos[i][d]
 *
 * where each (+) is one fused multiply-add (fmaf, one rounding) taken in
 * increasing k, and the final + Pos is one fp32 addition.
 *
 *   dot, |a|^2, |b|^2: 64 partial sums; partial j accumulates the terms
 *   d = j, j+64, j+128, ... (increasing d) with fmaf, starting from 0.  The 64
 *   partials are then combined by the tree: for off = 32,16,8,4,2,1:
 *   s[j] = s[j] + s[j+off] for j < off; the result is s[0].
 *   cos = dot / max(sqrt(|a|^2) * sqrt(|b|^2), 1e-8), each operation one
 *   correctly rounded fp32 operation.
 *
 * The paper's own score (eq. 3) compares first-layer keys rather than the
 * embedded tokens; that score is computed here in a fixed order too:
 *
 *   x_d  = S(T[i][d])                 (the layer-0 input as stored: bf16 with
 *                                      ties to even for a bf16 model)
 *   mean = tree64(partials of x) / D  (partial j adds x_j, x_{j+64}, ... to 0)
 *   c_d  = x_d - mean
 *   var  = tree64(partials of c*c) / D (partial j: fmaf(c_d, c_d, .) in increasing d)
 *   rstd = 1 / sqrt(var + eps)
 *   n_d  = fmaf(c_d * rstd, gamma_d, beta_d)           (LayerNorm 1 of layer 0)
 *   key_e = (b_k[e] (+) n_0*Wk[0][e] (+) ... (+) n_{D-1}*Wk[D-1][e])  (fmaf chain)
 *
 * Build: gcc -O3 -mavx2 -mfma -ffp-contract=off -fopenmp -fPIC -shared.
 * Contraction stays off so that no other product or sum is fused; OpenMP only
 * splits independent tokens across threads.
 */
#include <math.h>
#include <stdint.h>

/* T0[n][D] for n tokens; patches [n][P] fp32, w_pe [P][D], b_pe [D], pos [n][D].
 * Every output follows its own fmaf chain in increasing k; the loops only
 * interleave independent chains (k outer, d inner) so W_pe is read row-wise. */
void oracle_embed_f32(const float* patches, const float* w_pe, const float* b_pe,
                      const float* pos, int32_t n, int32_t P, int32_t D, float* t0) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < n; ++i) {
    const float* x = patches + (int64_t)i * P;
    float* acc = t0 + (int64_t)i * D;
    for (int32_t d = 0; d < D; ++d) acc[d] = b_pe[d];
    for (int32_t k = 0; k < P; ++k) {
      const float xk = x[k];
      const float* wk = w_pe + (int64_t)k * D;
      for (int32_t d = 0; d < D; ++d) acc[d] = fmaf(xk, wk[d], acc[d]);
    }
    for (int32_t d = 0; d < D; ++d) acc[d] = acc[d] + pos[(int64_t)i * D + d];
  }
}

static float tree64(float* s) {
  for (int off = 32; off >= 1; off >>= 1)
    for (int j = 0; j < off; ++j) s[j] = s[j] + s[j + off];
  return s[0];
}

/* sim[n] = cos(a_i, b_i) in the fixed order above; a, b are [n][D]. */
void oracle_cosine_f32(const float* a, const float* b, int32_t n, int32_t D, float* sim) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < n; ++i) {
    const float* x = a + (int64_t)i * D;
    const float* y = b + (int64_t)i * D;
    float sd[64], sa[64], sb[64];
    for (int j = 0; j < 64; ++j) {
      float pd = 0.0f, pa = 0.0f, pb = 0.0f;
      for (int32_t d = j; d < D; d += 64) {
        pd = fmaf(x[d], y[d], pd);
        pa = fmaf(x[d], x[d], pa);
        pb = fmaf(y[d], y[d], pb);
      }
      sd[j] = pd;
      sa[j] = pa;
      sb[j] = pb;
    }
    float dot = tree64(sd), na = tree64(sa), nb = tree64(sb);
    float denom = sqrtf(na) * sqrtf(nb);
    sim[i] = dot / fmaxf(denom, 1e-8f);
  }
}

/* fp32 value rounded to the nearest bf16 value, ties to even (NaN kept). */
static float round_bf16_f32(float f) {
  if (isnan(f)) return f;
  union { float f; uint32_t u; } v = {f};
  v.u = (v.u + 0x7fffu + ((v.u >> 16) & 1u)) & 0xffff0000u;
  return v.f;
}

/* key[n][D]: the first layer's key of each token in the fixed order above.
 * t0 [n][D] fp32 embedded tokens; ln_g, ln_b [D], wk [D][D] (input row, key
 * column), bk [D]: layer-0 LayerNorm and key projection, values as stored;
 * bf16 != 0 rounds the input to bf16 first. */
void oracle_key_score_f32(const float* t0, const float* ln_g, const float* ln_b, const float* wk,
                          const float* bk, int32_t n, int32_t D, float eps, int32_t bf16, float* key) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < n; ++i) {
    float x[4096], c[4096], nv[4096], s[64];
    const float* t = t0 + (int64_t)i * D;
    for (int32_t d = 0; d < D; ++d) x[d] = bf16 ? round_bf16_f32(t[d]) : t[d];
    for (int j = 0; j < 64; ++j) {
      float p = 0.0f;
      for (int32_t d = j; d < D; d += 64) p = p + x[d];
      s[j] = p;
    }
    const float mean = tree64(s) / (float)D;
    for (int32_t d = 0; d < D; ++d) c[d] = x[d] - mean;
    for (int j = 0; j < 64; ++j) {
      float p = 0.0f;
      for (int32_t d = j; d < D; d += 64) p = fmaf(c[d], c[d], p);
      s[j] = p;
    }
    const float var = tree64(s) / (float)D;
    const float rstd = 1.0f / sqrtf(var + eps);
    for (int32_t d = 0; d < D; ++d) nv[d] = fmaf(c[d] * rstd, ln_g[d], ln_b[d]);
    float* out = key + (int64_t)i * D;
    for (int32_t e = 0; e < D; ++e) out[e] = bk[e];
    for (int32_t d = 0; d < D; ++d) {
      const float nd = nv[d];
      const float* w = wk + (int64_t)d * D;
      for (int32_t e = 0; e < D; ++e) out[e] = fmaf(nd, w[e], out[e]);
    }
  }
}
