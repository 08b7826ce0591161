/*
 * AnchorKV oracle: a plain, slow CPU reference of what the compression pass and
 * the decode attention compute, written from the paper (arXiv 2608.02901,
 * "AnchorKV: Anchor-Residual KV Cache Compression").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the package's smoke check and the CPU
 * baseline leg of the benchmark do.  It shares no code with the HIP path.
 *
 * Arithmetic conventions (the canonical forms both implementations follow so
 * that every integer output -- anchor sets, anchor indices, coefficient bits,
 * residual codes -- is unique):
 *   - fp64 everywhere the paper gives a formula, except where a stored value
 *     has a narrower type (coefficients, residuals, rotated residuals, codes).
 *   - dot64(x, y): the fp64 products x_j*y_j (exact for fp32 and bf16 data)
 *     summed sequentially for j = 0..D-1.  Built with -ffp-contract=off, so no
 *     fused multiply-add ever merges a product into the running sum.
 *   - fp32 steps are single IEEE roundings in the order written.
 *   - bf16 conversion is round-to-nearest-even of the fp32 value.
 *
 * Parity status of each function (pins live in tests/test_oracle_*.py):
 *   pinned   : splitmix64 (published first output), Hadamard (dense Sylvester
 *              product, orthogonality), codec levels (Lloyd's iteration for a
 *              unit Gaussian), byte budget (the worked example of App. A.1),
 *              assignment (exhaustive search, closed-form special cases,
 *              projection orthogonality), decode attention (all-anchor case
 *              equals dense attention; output-error theorem of App. A.4),
 *              selector (brute force on tiny inputs; the raw score against
 *              column means of scipy's causal softmax and the pool against a
 *              centred zero-padded numpy convolution at kappa = 1..9),
 *              utilities (numpy brute force over m = 6 observation rows, each
 *              with its own causal softmax and y_w; finite-difference test of
 *              the two-channel expansion, Eq. channels), positional rotation
 *              (the rotary table against numpy's cos and sin, the rotation as
 *              a complex product, worked unit vectors, relative-position
 *              invariance; the rotated pass's selector, utilities and
 *              attention against numpy over explicitly rotated keys; zero
 *              frequencies reduce it to the unrotated pass bit for bit).
 *              Planted mistakes in a copy of this file (off-centre or
 *              renormalised pool, one-row sums, offset-major rows, alpha for
 *              alpha^2, reversed rotation, unrotated observation keys or key
 *              residuals, mirrored positions) fail these pins.
 *   parity unpinned beyond self-consistency: the absmax scale readings of the
 *              codec (Sec. 3.1 / App. A.1 leave the scale rule ambiguous).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Primitives                                                                 */
/* ------------------------------------------------------------------------ */

/* SplitMix64 (Steele, Lea & Flood 2014): the first output of a generator
 * whose state is x.  Used as a counter-based hash for the uniform anchor share
 * (Sec. 3.2, anchor selection) and for the Hadamard sign pattern (App. A.1). */
uint64_t akvref_splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* Seeds derived from the user seed: one stream for anchor sampling, one for
 * the sign pattern s of the randomized Hadamard rotation. */
static uint64_t anchor_seed(uint64_t seed) { return akvref_splitmix64(seed ^ 1ULL); }
static uint64_t sign_seed(uint64_t seed) { return akvref_splitmix64(seed ^ 2ULL); }

static float bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u = u + 0x7FFFu + ((u >> 16) & 1u);
  u &= 0xFFFF0000u;
  memcpy(&f, &u, 4);
  return f;
}

/* Sequential fp64 dot product (canonical order). */
static double dot64(const double* x, const double* y, int D) {
  double s = 0.0;
  for (int j = 0; j < D; ++j) s += x[j] * y[j];
  return s;
}

/* Sign pattern s in {+1,-1}^D of the rotation U = H_D diag(s)/sqrt(D)
 * (App. A.1, Eq. hadamard): s_j = -1 when the top bit of the hash of j is set. */
void akvref_hadamard_signs(uint64_t seed, int D, float* s) {
  uint64_t ss = sign_seed(seed);
  for (int j = 0; j < D; ++j) s[j] = (akvref_splitmix64(ss ^ (uint64_t)j) >> 63) ? -1.0f : 1.0f;
}

/* Unnormalized fast Walsh-Hadamard transform in fp32, Sylvester ordering:
 * stages h = 1, 2, 4, ..., D/2; in stage h every pair (i, i+h) with i & h == 0
 * becomes (z_i + z_{i+h}, z_i - z_{i+h}).  Applying it twice multiplies by D. */
void akvref_fwht(float* z, int D) {
  for (int h = 1; h < D; h <<= 1)
    for (int i = 0; i < D; ++i)
      if ((i & h) == 0) {
        float a = z[i], b = z[i + h];
        z[i] = a + b;
        z[i + h] = a - b;
      }
}

/* ------------------------------------------------------------------------ */
/* Rotary position embedding (Sec. 3.2: keys are projected before the        */
/* rotation, anchors are scored with rotated keys, and the stored keys are   */
/* rotated at decoding; App. E "Implementation").                            */
/* ------------------------------------------------------------------------ */

/* Cosines and sines of the rotation R_t of positions t = 0 .. npos-1 in the
 * rotate-half pairing of Llama-family models: coordinate pair (f, f + D/2),
 * f < D/2, turns by the angle t * inv_freq[f].  Both are fp32, the roundings
 * of the fp64 cos and sin of the fp64 angle (t exact, inv_freq[f] an fp32
 * value), as a model's rotary table holds them: cs[t][f][0] = cos,
 * cs[t][f][1] = sin. */
void akvref_rope_table(const float* inv_freq, int D, int npos, float* cs) {
  int F = D / 2;
  for (int t = 0; t < npos; ++t)
    for (int f = 0; f < F; ++f) {
      double ang = (double)t * (double)inv_freq[f];
      cs[((size_t)t * F + f) * 2] = (float)cos(ang);
      cs[((size_t)t * F + f) * 2 + 1] = (float)sin(ang);
    }
}

/* out = R_t x in fp64 from position t's fp32 cosines and sines (cs_t, D
 * values): (x_f, x_{f+D/2}) -> (c x_f - s x_{f+D/2}, s x_f + c x_{f+D/2}).
 * A product of an fp32 factor and an fp32 or bf16 coordinate is exact in
 * fp64, so each output coordinate is rounded once. */
void akvref_rope_rotate(const float* cs_t, const double* x, int D, double* out) {
  int F = D / 2;
  for (int f = 0; f < F; ++f) {
    double c = cs_t[2 * f], s = cs_t[2 * f + 1];
    double a = x[f], b = x[f + F];
    out[f] = c * a - s * b;
    out[f + F] = s * a + c * b;
  }
}

/* Rotated keys of one head as attention sees them: R_t K_t for every
 * position, rounded to fp32 and, for a bf16 cache, on to bf16 (the dtype of a
 * model's rotated keys).  They feed the observation pass -- anchor scores,
 * attention weights and the outputs y_w -- while assignment, projection and
 * storage use the unrotated keys. */
void akvref_rope_keys(const double* K, int S, int D, const float* cs, int bf16, double* Kpost) {
  double* tmp = (double*)malloc(sizeof(double) * D);
  for (int t = 0; t < S; ++t) {
    akvref_rope_rotate(cs + (size_t)t * D, K + (size_t)t * D, D, tmp);
    for (int j = 0; j < D; ++j) {
      float v = (float)tmp[j];
      if (bf16) v = bf16_rne(v);
      Kpost[(size_t)t * D + j] = v;
    }
  }
  free(tmp);
}

/* ------------------------------------------------------------------------ */
/* Residual codec (Sec. 3.1 "Residual quantization"; App. A.1 rotation and    */
/* codebook).                                                                 */
/* ------------------------------------------------------------------------ */

/* Four-level Lloyd-Max quantizer for a unit Gaussian source (Lloyd 1957,
 * Max 1960): reconstruction levels +-L0, +-L1 and decision threshold T. */
#define AKV_LM_L0 0.4527800f
#define AKV_LM_L1 1.5104176f
#define AKV_LM_T 0.9815988f

enum { SCALE_ABSMAX_OUTER = 0, SCALE_ABSMAX_LITERAL = 1, SCALE_RMS = 2, SCALE_NAIVE = 3 };

/* Scale of one group of rotated coordinates: the Gaussian standard deviation
 * the codebook is applied at.  The paper names a per-token absmax scale; the
 * three readings of how the absmax enters are:
 *   OUTER   : sigma = A / L1, so the largest coordinate lands on the outer level;
 *   LITERAL : sigma = A (coordinates divided by the absmax, then quantized);
 *   RMS     : sigma = sqrt(sum z^2 / G) (the marginal the rotation produces). */
static float group_scale(const float* z, int G, int mode) {
  if (mode == SCALE_RMS) {
    float acc = 0.0f;
    for (int j = 0; j < G; ++j) {
      float sq = z[j] * z[j];
      acc = acc + sq;
    }
    float ms = acc / (float)G;
    return sqrtf(ms);
  }
  float A = 0.0f;
  for (int j = 0; j < G; ++j) {
    float m = fabsf(z[j]);
    if (m > A) A = m;
  }
  if (mode == SCALE_ABSMAX_LITERAL) return A;
  return A / AKV_LM_L1;
}

/* Encode one residual r[D] (fp32): z = FWHT(s * r); per group of G
 * coordinates a scale sigma; code in {0,1,2,3} for levels {-L1,-L0,+L0,+L1};
 * four codes per byte, coordinate j in byte j/4 at bits 2*(j%4)..2*(j%4)+1.
 *
 * SCALE_NAIVE is the ablation of Sec. 4.3 "Component Removal" (iv): 2-bit
 * quantization without the Hadamard rotation and without the Lloyd-Max
 * codebook, i.e. z = r and the uniform four-level quantizer of [-A, A]
 * (A = group absmax): cells of width A/2, levels +-A/4, +-3A/4, so
 * sigma = A/4 with levels {-3,-1,+1,+3} sigma and threshold 2 sigma. */
void akvref_codec_encode(const float* r, int D, int G, int mode, uint64_t seed,
                         uint8_t* codes, float* scales) {
  float* s = (float*)malloc(sizeof(float) * D);
  float* z = (float*)malloc(sizeof(float) * D);
  akvref_hadamard_signs(seed, D, s);
  if (mode == SCALE_NAIVE) {
    for (int j = 0; j < D; ++j) z[j] = r[j];
  } else {
    for (int j = 0; j < D; ++j) z[j] = s[j] * r[j];
    akvref_fwht(z, D);
  }
  memset(codes, 0, (size_t)D / 4);
  for (int g0 = 0; g0 < D; g0 += G) {
    float sigma, T;
    if (mode == SCALE_NAIVE) {
      float A = 0.0f;
      for (int j = g0; j < g0 + G; ++j) {
        float m = fabsf(z[j]);
        if (m > A) A = m;
      }
      sigma = A * 0.25f;
      T = sigma * 2.0f;
    } else {
      sigma = group_scale(z + g0, G, mode);
      T = sigma * AKV_LM_T;
    }
    scales[g0 / G] = sigma;
    for (int j = g0; j < g0 + G; ++j) {
      int outer = fabsf(z[j]) > T;
      int c = (z[j] < 0.0f) ? (outer ? 0 : 1) : (outer ? 3 : 2);
      codes[j / 4] |= (uint8_t)(c << (2 * (j % 4)));
    }
  }
  free(s);
  free(z);
}

/* Decode: zhat_j = sigma * level(code_j); r~ = s * FWHT(zhat) / D, i.e.
 * U^T applied to the dequantized rotated coordinates (App. A.1, Eq. arc-tuple).
 * SCALE_NAIVE: levels {-3,-1,+1,+3} and no rotation, r~ = zhat. */
void akvref_codec_decode(const uint8_t* codes, const float* scales, int D, int G,
                         uint64_t seed, int mode, float* rt) {
  static const float lev[4] = {-AKV_LM_L1, -AKV_LM_L0, AKV_LM_L0, AKV_LM_L1};
  static const float ulev[4] = {-3.0f, -1.0f, 1.0f, 3.0f};
  if (mode == SCALE_NAIVE) {
    for (int j = 0; j < D; ++j) {
      int c = (codes[j / 4] >> (2 * (j % 4))) & 3;
      rt[j] = scales[j / G] * ulev[c];
    }
    return;
  }
  float* s = (float*)malloc(sizeof(float) * D);
  akvref_hadamard_signs(seed, D, s);
  for (int j = 0; j < D; ++j) {
    int c = (codes[j / 4] >> (2 * (j % 4))) & 3;
    rt[j] = scales[j / G] * lev[c];
  }
  akvref_fwht(rt, D);
  float invD = 1.0f / (float)D;
  for (int j = 0; j < D; ++j) rt[j] = (rt[j] * invD) * s[j];
  free(s);
}

/* ------------------------------------------------------------------------ */
/* Byte budget (Sec. 3.4, Eq. byte-budget; App. A.1, Eq. mfixed and Table of  */
/* the layout).                                                              */
/* ------------------------------------------------------------------------ */

/* M_base of one layer: anchors (K and V, elem_bytes each), int64 anchor
 * positions of the non-window anchors, per-side index (b_a = 2) and
 * coefficient (b_gamma) for the P = S - W non-window positions, residual
 * mask words and int32 prefix counts per side, head offsets, int32 position
 * ids. */
double akvref_base_bytes(int S, int H, int D, int W, int k, int elem_bytes, int b_gamma) {
  double P = (double)(S - W);
  double words = ceil(P / 64.0);
  return (double)H * (2.0 * elem_bytes * k * D + 8.0 * (k - W) + 2.0 * P * (2.0 + b_gamma)) +
         24.0 * H * words + 8.0 * (H + 1) + 4.0 * P;
}

/* N = max{0, floor((theta*M_full - M_base) / b_res)} with b_res the mean of
 * the key residual cost c_K = D/4 + 4*(D/G) and the value residual cost
 * c_V = c_K + 1 (one-byte chunk-local position). */
int64_t akvref_theta_budget(int S, int H, int D, int W, int k, int G, int elem_bytes,
                            int b_gamma, double theta) {
  double Mfull = 2.0 * elem_bytes * (double)S * H * D;
  double Mbase = akvref_base_bytes(S, H, D, W, k, elem_bytes, b_gamma);
  double cK = D / 4.0 + 4.0 * (D / G);
  double cV = cK + 1.0;
  double bres = 0.5 * (cK + cV);
  double n = floor((theta * Mfull - Mbase) / bres);
  return n > 0 ? (int64_t)n : 0;
}

/* ------------------------------------------------------------------------ */
/* Observation window and anchor selection (Sec. 3.2; App. A.2 Eq.           */
/* selector-score).                                                           */
/* ------------------------------------------------------------------------ */

/* Exact attention of the m = W*g observation rows of one KV head.  Row
 * w = jj*W + i is query head jj of the group at window offset i, position
 * S-W+i; it attends causally to t <= S-W+i.  Outputs the row max M_w of the
 * logits l = q.k/sqrt(D), Z_w = sum_t exp(l - M_w), and y_w = sum_t alpha_wt v_t.
 * Qg is [g][W][D]. */
void akvref_obs_head(const double* Kh, const double* Vh, const double* Qg, int S, int D,
                     int W, int g, double* M, double* Z, double* Y) {
  int m = W * g;
  double isd = 1.0 / sqrt((double)D);
#pragma omp parallel for schedule(dynamic, 1)
  for (int w = 0; w < m; ++w) {
    int i = w % W;
    int last = S - W + i;
    const double* q = Qg + (size_t)w * D;
    double* l = (double*)malloc(sizeof(double) * (size_t)(last + 1));
    double mx = -INFINITY;
    for (int t = 0; t <= last; ++t) {
      l[t] = dot64(q, Kh + (size_t)t * D, D) * isd;
      if (l[t] > mx) mx = l[t];
    }
    double z = 0.0;
    for (int t = 0; t <= last; ++t) z += exp(l[t] - mx);
    double* y = Y + (size_t)w * D;
    for (int j = 0; j < D; ++j) y[j] = 0.0;
    for (int t = 0; t <= last; ++t) {
      double a = exp(l[t] - mx) / z;
      const double* v = Vh + (size_t)t * D;
      for (int j = 0; j < D; ++j) y[j] += a * v[j];
    }
    M[w] = mx;
    Z[w] = z;
    free(l);
  }
}

/* Attention weight alpha_{w,t} of observation row w on position t. */
static double obs_alpha(const double* Kh, const double* Qg, const double* M, const double* Z,
                        int S, int D, int W, int w, int t) {
  int i = w % W;
  if (t > S - W + i) return 0.0;
  double l = dot64(Qg + (size_t)w * D, Kh + (size_t)t * D, D) / sqrt((double)D);
  return exp(l - M[w]) / Z[w];
}

/* SnapKV-style score of every non-window position t in [0, P):
 * sc(t) = (1/m) sum_w alpha_{w,t}, then average pooling of width kappa
 * (odd), centred, zero padding outside [0, P), divided by kappa. */
void akvref_selector_scores(const double* Kh, const double* Qg, const double* M,
                            const double* Z, int S, int D, int W, int g, int kappa,
                            double* sc, double* pooled) {
  int m = W * g, P = S - W;
#pragma omp parallel for schedule(static)
  for (int t = 0; t < P; ++t) {
    double s = 0.0;
    for (int w = 0; w < m; ++w) s += obs_alpha(Kh, Qg, M, Z, S, D, W, w, t);
    sc[t] = s / m;
  }
  int half = kappa / 2;
  for (int t = 0; t < P; ++t) {
    double s = 0.0;
    for (int d = -half; d <= half; ++d) {
      int u = t + d;
      if (u >= 0 && u < P) s += sc[u];
    }
    pooled[t] = s / kappa;
  }
}

typedef struct { double v; int t; } score_pos;
static int by_score_desc(const void* a, const void* b) {
  const score_pos* x = (const score_pos*)a;
  const score_pos* y = (const score_pos*)b;
  if (x->v > y->v) return -1;
  if (x->v < y->v) return 1;
  return (x->t > y->t) - (x->t < y->t);
}
typedef struct { uint64_t key; int t; } key_pos;
static int by_key_asc(const void* a, const void* b) {
  const key_pos* x = (const key_pos*)a;
  const key_pos* y = (const key_pos*)b;
  if (x->key < y->key) return -1;
  if (x->key > y->key) return 1;
  return (x->t > y->t) - (x->t < y->t);
}
static int int_asc(const void* a, const void* b) {
  int x = *(const int*)a, y = *(const int*)b;
  return (x > y) - (x < y);
}

/* Number of attention-scored anchors: floor(rho * (k - W)) in fp64. */
int akvref_n_top(int k, int W, float rho) { return (int)floor((double)rho * (double)(k - W)); }

/* Anchor set of one head (Algorithm 1, first step): the last W positions,
 * the n_top best pooled scores among [0, P) (ties to the lower position),
 * and the remaining k - W - n_top sampled uniformly without replacement from
 * the rest of [0, P): the positions with the smallest hash
 * splitmix64(anchor_seed ^ (h << 40) ^ t).  Output sorted ascending; the
 * anchor index of a position is its rank in this list. */
void akvref_select_anchors(const double* pooled, int S, int W, int k, float rho, uint64_t seed,
                           int h, int* anchors) {
  int P = S - W;
  int n_top = akvref_n_top(k, W, rho);
  int n_rand = k - W - n_top;
  score_pos* sp = (score_pos*)malloc(sizeof(score_pos) * (size_t)(P > 0 ? P : 1));
  for (int t = 0; t < P; ++t) { sp[t].v = pooled[t]; sp[t].t = t; }
  qsort(sp, (size_t)P, sizeof(score_pos), by_score_desc);
  char* taken = (char*)calloc((size_t)(P > 0 ? P : 1), 1);
  int n = 0;
  for (int i = 0; i < n_top; ++i) { taken[sp[i].t] = 1; anchors[n++] = sp[i].t; }
  key_pos* kp = (key_pos*)malloc(sizeof(key_pos) * (size_t)(P > 0 ? P : 1));
  int nk = 0;
  uint64_t as = anchor_seed(seed);
  for (int t = 0; t < P; ++t)
    if (!taken[t]) {
      kp[nk].key = akvref_splitmix64(as ^ ((uint64_t)h << 40) ^ (uint64_t)t);
      kp[nk].t = t;
      ++nk;
    }
  qsort(kp, (size_t)nk, sizeof(key_pos), by_key_asc);
  for (int i = 0; i < n_rand; ++i) anchors[n++] = kp[i].t;
  for (int t = P; t < S; ++t) anchors[n++] = t;
  qsort(anchors, (size_t)k, sizeof(int), int_asc);
  free(sp);
  free(taken);
  free(kp);
}

/* ------------------------------------------------------------------------ */
/* Anchor-residual representation (Sec. 3.1, Eqs. nearest-anchor, projection, */
/* reconstruction).                                                           */
/* ------------------------------------------------------------------------ */

/* Nearest anchor of one vector x among the k anchor vectors A[k][D] with
 * squared norms nrm[k]: maximize c_a = d_a*d_a / n_a (d_a = dot64(x, A_a);
 * c_a = -1 for a zero anchor), ties to the lowest index.  For fixed x this
 * orders anchors like |cos(x, A_a)|.  Then gamma = d/n in fp64, rounded to
 * fp32 and, for a bf16 cache, to bf16 (the stored coefficient). */
static void nearest_anchor(const double* x, const double* A, const double* nrm, int k, int D,
                           int bf16, int* a_out, double* g_out) {
  int best = 0;
  double bc = -INFINITY, bd = 0.0;
  for (int a = 0; a < k; ++a) {
    double d = dot64(x, A + (size_t)a * D, D);
    double c = nrm[a] > 0.0 ? (d * d) / nrm[a] : -1.0;
    if (c > bc) { bc = c; best = a; bd = d; }
  }
  double g64 = nrm[best] > 0.0 ? bd / nrm[best] : 0.0;
  float g32 = (float)g64;
  if (bf16) g32 = bf16_rne(g32);
  *a_out = best;
  *g_out = (double)g32;
}

/* Residual against the stored coefficient and anchor, in fp32:
 * r_j = x_j - fp32(gamma * a_j). */
static void residual(const double* x, const double* anc, double gamma, int D, float* r) {
  float g = (float)gamma;
  for (int j = 0; j < D; ++j) {
    float p = g * (float)anc[j];
    r[j] = (float)x[j] - p;
  }
}

/* Assignment of an explicit list of tokens of one head against anchors at
 * positions anchors[k] of X[S][D].  Anchor tokens keep their own index with
 * gamma = 1 and a zero residual (the layout stores gamma = 1 on anchors). */
void akvref_assign_tokens(const double* X, int S, int D, const int* anchors, int k, int bf16,
                          const int* toks, int ntok, int* a_out, double* g_out, float* r_out) {
  double* A = (double*)malloc(sizeof(double) * (size_t)k * D);
  double* nrm = (double*)malloc(sizeof(double) * (size_t)k);
  int* rank = (int*)malloc(sizeof(int) * (size_t)S);
  for (int t = 0; t < S; ++t) rank[t] = -1;
  for (int a = 0; a < k; ++a) {
    memcpy(A + (size_t)a * D, X + (size_t)anchors[a] * D, sizeof(double) * D);
    nrm[a] = dot64(A + (size_t)a * D, A + (size_t)a * D, D);
    rank[anchors[a]] = a;
  }
#pragma omp parallel for schedule(dynamic, 16)
  for (int i = 0; i < ntok; ++i) {
    int t = toks[i];
    float* r = r_out ? r_out + (size_t)i * D : NULL;
    if (rank[t] >= 0) {
      a_out[i] = rank[t];
      g_out[i] = 1.0;
      if (r) for (int j = 0; j < D; ++j) r[j] = 0.0f;
      continue;
    }
    nearest_anchor(X + (size_t)t * D, A, nrm, k, D, bf16, &a_out[i], &g_out[i]);
    if (r) residual(X + (size_t)t * D, A + (size_t)a_out[i] * D, g_out[i], D, r);
  }
  free(A);
  free(nrm);
  free(rank);
}

/* Nearest anchor of free vectors (appended tokens) against explicit anchor
 * vectors A[k][D]. */
void akvref_assign_vectors(const double* xs, int n, const double* A, int k, int D, int bf16,
                           int* a_out, double* g_out) {
  double* nrm = (double*)malloc(sizeof(double) * (size_t)k);
  for (int a = 0; a < k; ++a) nrm[a] = dot64(A + (size_t)a * D, A + (size_t)a * D, D);
  for (int i = 0; i < n; ++i) nearest_anchor(xs + (size_t)i * D, A, nrm, k, D, bf16, &a_out[i], &g_out[i]);
  free(nrm);
}

/* ------------------------------------------------------------------------ */
/* Attention-output-aware utilities (Sec. 3.3, Eq. utilities; App. A.3).      */
/* ------------------------------------------------------------------------ */

/* Utilities of listed non-anchor tokens of one head.  rK, rV are the fp32
 * residuals of those tokens; Kh holds the keys the observation rows attend to
 * (rotated when positions are encoded), cs the rotation table or NULL.
 *   uK_t = (1/m) sum_w alpha_wt^2 (q_w . R_t rK_t)^2 / D * ||v_t - y_w||^2
 *   uV_t = (1/m) sum_w alpha_wt^2 ||rV_t||^2
 * R_t r is formed in fp64 (akvref_rope_rotate); without a table R_t = I. */
static void utilities_impl(const double* Kh, const double* Vh, const double* Qg, const double* M,
                           const double* Z, const double* Y, int S, int D, int W, int g,
                           const int* toks, int ntok, const float* rK, const float* rV, const float* cs,
                           double* uK, double* uV) {
  int m = W * g;
#pragma omp parallel for schedule(dynamic, 16)
  for (int i = 0; i < ntok; ++i) {
    int t = toks[i];
    double* rk = (double*)malloc(sizeof(double) * D);
    double* rv = (double*)malloc(sizeof(double) * D);
    double* dv = (double*)malloc(sizeof(double) * D);
    for (int j = 0; j < D; ++j) {
      rk[j] = rK[(size_t)i * D + j];
      rv[j] = rV[(size_t)i * D + j];
    }
    if (cs) {
      akvref_rope_rotate(cs + (size_t)t * D, rk, D, dv);
      memcpy(rk, dv, sizeof(double) * D);
    }
    double rvn = dot64(rv, rv, D);
    double sk = 0.0, sv = 0.0;
    for (int w = 0; w < m; ++w) {
      double a = obs_alpha(Kh, Qg, M, Z, S, D, W, w, t);
      double a2 = a * a;
      double qr = dot64(Qg + (size_t)w * D, rk, D);
      for (int j = 0; j < D; ++j) dv[j] = Vh[(size_t)t * D + j] - Y[(size_t)w * D + j];
      double vy = dot64(dv, dv, D);
      sk += a2 * (qr * qr / D) * vy;
      sv += a2 * rvn;
    }
    uK[i] = sk / m;
    uV[i] = sv / m;
    free(rk);
    free(rv);
    free(dv);
  }
}

void akvref_utilities(const double* Kh, const double* Vh, const double* Qg, const double* M,
                      const double* Z, const double* Y, int S, int D, int W, int g,
                      const int* toks, int ntok, const float* rK, const float* rV, double* uK,
                      double* uV) {
  utilities_impl(Kh, Vh, Qg, M, Z, Y, S, D, W, g, toks, ntok, rK, rV, NULL, uK, uV);
}

/* The same with positions encoded: Kh_rot the rotated keys of the head
 * (akvref_rope_keys), cs the rotation table of its S positions. */
void akvref_utilities_rope(const double* Kh_rot, const double* Vh, const double* Qg, const double* M,
                           const double* Z, const double* Y, int S, int D, int W, int g,
                           const int* toks, int ntok, const float* rK, const float* rV, const float* cs,
                           double* uK, double* uV) {
  utilities_impl(Kh_rot, Vh, Qg, M, Z, Y, S, D, W, g, toks, ntok, rK, rV, cs, uK, uV);
}

/* ------------------------------------------------------------------------ */
/* Head-pooled residual budget (Sec. 3.4; Algorithm 1).                      */
/* ------------------------------------------------------------------------ */

typedef struct { double u; int h, t; } cand;
static int cand_cmp(const void* a, const void* b) {
  const cand* x = (const cand*)a;
  const cand* y = (const cand*)b;
  if (x->u > y->u) return -1;
  if (x->u < y->u) return 1;
  if (x->h != y->h) return x->h < y->h ? -1 : 1;
  return (x->t > y->t) - (x->t < y->t);
}

/* Marks sel[h*S+t] = 1 for the N candidates of highest utility across all
 * heads (candidates are entries with u >= 0; anchors carry u = -1), ties to
 * the lower head, then the lower position.  Returns the number selected. */
int64_t akvref_budget_select(const double* u, int H, int S, int64_t N, uint8_t* sel) {
  cand* c = (cand*)malloc(sizeof(cand) * (size_t)H * S);
  int64_t nc = 0;
  for (int h = 0; h < H; ++h)
    for (int t = 0; t < S; ++t) {
      sel[(size_t)h * S + t] = 0;
      double v = u[(size_t)h * S + t];
      if (v >= 0.0) { c[nc].u = v; c[nc].h = h; c[nc].t = t; ++nc; }
    }
  qsort(c, (size_t)nc, sizeof(cand), cand_cmp);
  int64_t n = N < nc ? N : nc;
  for (int64_t i = 0; i < n; ++i) sel[(size_t)c[i].h * S + c[i].t] = 1;
  free(c);
  return n;
}

/* Equal per-head budgets (Sec. 4.3 "Component Removal" (ii), the pooling
 * across heads dropped): every head selects its own floor(N / H) candidates
 * of highest key, ties to the lower position.  Returns the number selected. */
int64_t akvref_budget_select_per_head(const double* u, int H, int S, int64_t N, uint8_t* sel) {
  int64_t tot = 0;
  for (int h = 0; h < H; ++h) tot += akvref_budget_select(u + (size_t)h * S, 1, S, N / H, sel + (size_t)h * S);
  return tot;
}

/* ------------------------------------------------------------------------ */
/* Residual ranking (Sec. 3.3 utilities and the alternatives of Sec. 4.3     */
/* "Residual Ranking").                                                       */
/* ------------------------------------------------------------------------ */

enum { RANK_UTILITY = 0, RANK_COSINE = 1, RANK_RESNORM = 2, RANK_ATTENTION = 3, RANK_RANDOM = 4 };

/* Ranking key of non-anchor token t of head h on one side (larger = earlier
 * residual), for the alternatives to the utility:
 *   COSINE    : 1 - |cos(x_t, abar_a(t))|, the least aligned first (cos from
 *               sequential fp64 dots; a zero vector counts as orthogonal);
 *   RESNORM   : ||r_t||^2 of the fp32 residual (sequential fp64 sum);
 *   ATTENTION : the raw selector score sc(t) (mean attention of the
 *               observation rows, App. A.2), the same on both sides;
 *   RANDOM    : a uniform variate in [0, 1) from the counter-based hash
 *               splitmix64(seed_r ^ (side + 1) << 60 ^ h << 40 ^ t), 53 bits. */
double akvref_rank_key(int mode, int side, int h, int t, const double* x, const double* abar, int D,
                       const float* r, double sc_t, uint64_t seed) {
  if (mode == RANK_COSINE) {
    double d = dot64(x, abar, D), xx = dot64(x, x, D), nn = dot64(abar, abar, D);
    double den = sqrt(xx * nn);
    return den > 0.0 ? 1.0 - fabs(d) / den : 1.0;
  }
  if (mode == RANK_RESNORM) {
    double s = 0.0;
    for (int j = 0; j < D; ++j) s += (double)r[j] * (double)r[j];
    return s;
  }
  if (mode == RANK_ATTENTION) return sc_t;
  uint64_t rs = akvref_splitmix64(seed ^ 3ULL);
  uint64_t key = akvref_splitmix64(rs ^ ((uint64_t)(side + 1) << 60) ^ ((uint64_t)h << 40) ^ (uint64_t)t);
  return (double)(key >> 11) * 0x1p-53;
}

/* ------------------------------------------------------------------------ */
/* Whole compression pass of one request (Algorithm 1).                      */
/* ------------------------------------------------------------------------ */

enum { BUDGET_FRACTION = 0, BUDGET_THETA = 1, BUDGET_COUNT = 2 };

/* K, V: [H][S][D]; Qobs: [Hq][W][D] (values exactly representable in the
 * cache dtype).  anchor_override: [H][k] sorted positions or NULL.
 * rank_mode: RANK_* (the utility is the method; the rest are the ablations
 * of Sec. 4.3); head_budget: 0 pools the budget over heads (the method), 1
 * gives every head floor(N / H).
 * Outputs, all per head in position order:
 *   anchors[H][k]; aK, aV [H][S] anchor index; gK, gV [H][S] stored gamma;
 *   uK, uV [H][S] utilities (-1 on anchors); selK, selV [H][S] residual flags;
 *   codesK, codesV [H][S][D/4]; scalesK, scalesV [H][S][D/G] (zero where the
 *   position stores no residual); pooled [H][S-W] selector scores (may be NULL).
 * nsel[2] receives the residual counts per side. */
static int encode_impl(int H, int Hq, int D, int S, int W, int k, float rho, int kappa, int bf16,
                       uint64_t seed, int budget_mode, double budget, int64_t budget_count, int G,
                       int scale_mode, int rank_mode, int head_budget, const double* K, const double* V,
                       const double* Qobs, const int* anchor_override, const float* inv_freq, int* anchors,
                       int* aK, double* gK, int* aV, double* gV, double* uK, double* uV, uint8_t* selK,
                       uint8_t* selV, uint8_t* codesK, float* scalesK, uint8_t* codesV, float* scalesV,
                       double* pooled, int64_t* nsel) {
  if (H <= 0 || Hq % H != 0 || D < 4 || (D & (D - 1)) || W < 0 || k < W || k > S ||
      G <= 0 || D % G || G % 4 || kappa <= 0 || (kappa & 1) == 0 || rank_mode < 0 || rank_mode > 4)
    return 1;
  int g = Hq / H, m = W * g, P = S - W;
  size_t SD = (size_t)S * D;
  float* rK = (float*)calloc((size_t)H * SD, sizeof(float));
  float* rV = (float*)calloc((size_t)H * SD, sizeof(float));
  int* all = (int*)malloc(sizeof(int) * (size_t)S);
  for (int t = 0; t < S; ++t) all[t] = t;
  double* M = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1));
  double* Zs = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1));
  double* Y = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1) * D);
  double* sc = (double*)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
  double* pl = (double*)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
  /* With positions encoded, the observation pass runs on the rotated keys
   * (Sec. 3.2: anchor scoring uses post-rotation keys). */
  float* cs = NULL;
  double* Krot = NULL;
  if (inv_freq) {
    cs = (float*)malloc(sizeof(float) * (size_t)S * D);
    Krot = (double*)malloc(sizeof(double) * SD);
    akvref_rope_table(inv_freq, D, S, cs);
  }
  for (int h = 0; h < H; ++h) {
    const double* Kh = K + (size_t)h * SD;
    const double* Vh = V + (size_t)h * SD;
    const double* Qg = Qobs + (size_t)h * g * W * D;
    int* anc = anchors + (size_t)h * k;
    const double* Ko = Kh;
    if (inv_freq) {
      akvref_rope_keys(Kh, S, D, cs, bf16, Krot);
      Ko = Krot;
    }
    akvref_obs_head(Ko, Vh, Qg, S, D, W, g, M, Zs, Y);
    if (anchor_override) {
      memcpy(anc, anchor_override + (size_t)h * k, sizeof(int) * k);
      if (rank_mode == RANK_ATTENTION) akvref_selector_scores(Ko, Qg, M, Zs, S, D, W, g, kappa, sc, pl);
    } else {
      akvref_selector_scores(Ko, Qg, M, Zs, S, D, W, g, kappa, sc, pl);
      if (pooled) memcpy(pooled + (size_t)h * P, pl, sizeof(double) * P);
      akvref_select_anchors(pl, S, W, k, rho, seed, h, anc);
    }
    float* rKh = rK + (size_t)h * SD;
    float* rVh = rV + (size_t)h * SD;
    akvref_assign_tokens(Kh, S, D, anc, k, bf16, all, S, aK + (size_t)h * S, gK + (size_t)h * S, rKh);
    akvref_assign_tokens(Vh, S, D, anc, k, bf16, all, S, aV + (size_t)h * S, gV + (size_t)h * S, rVh);
    char* isanc = (char*)calloc((size_t)S, 1);
    for (int a = 0; a < k; ++a) isanc[anc[a]] = 1;
    int* cand_t = (int*)malloc(sizeof(int) * (size_t)S);
    int nc = 0;
    for (int t = 0; t < S; ++t)
      if (!isanc[t]) cand_t[nc++] = t;
    float* crk = (float*)malloc(sizeof(float) * (size_t)(nc > 0 ? nc : 1) * D);
    float* crv = (float*)malloc(sizeof(float) * (size_t)(nc > 0 ? nc : 1) * D);
    double* cuk = (double*)malloc(sizeof(double) * (size_t)(nc > 0 ? nc : 1));
    double* cuv = (double*)malloc(sizeof(double) * (size_t)(nc > 0 ? nc : 1));
    for (int i = 0; i < nc; ++i) {
      memcpy(crk + (size_t)i * D, rKh + (size_t)cand_t[i] * D, sizeof(float) * D);
      memcpy(crv + (size_t)i * D, rVh + (size_t)cand_t[i] * D, sizeof(float) * D);
    }
    utilities_impl(Ko, Vh, Qg, M, Zs, Y, S, D, W, g, cand_t, nc, crk, crv, cs, cuk, cuv);
    for (int t = 0; t < S; ++t) { uK[(size_t)h * S + t] = -1.0; uV[(size_t)h * S + t] = -1.0; }
    for (int i = 0; i < nc; ++i) {
      uK[(size_t)h * S + cand_t[i]] = cuk[i];
      uV[(size_t)h * S + cand_t[i]] = cuv[i];
    }
    if (rank_mode != RANK_UTILITY) {
      double* ak = (double*)malloc(sizeof(double) * D);
      double* av = (double*)malloc(sizeof(double) * D);
      for (int i = 0; i < nc; ++i) {
        int t = cand_t[i];
        size_t e = (size_t)h * S + t;
        memcpy(ak, Kh + (size_t)anc[aK[e]] * D, sizeof(double) * D);
        memcpy(av, Vh + (size_t)anc[aV[e]] * D, sizeof(double) * D);
        double sct = t < P ? sc[t] : 0.0;
        uK[e] = akvref_rank_key(rank_mode, 0, h, t, Kh + (size_t)t * D, ak, D, crk + (size_t)i * D, sct, seed);
        uV[e] = akvref_rank_key(rank_mode, 1, h, t, Vh + (size_t)t * D, av, D, crv + (size_t)i * D, sct, seed);
      }
      free(ak);
      free(av);
    }
    free(isanc); free(cand_t); free(crk); free(crv); free(cuk); free(cuv);
  }
  int64_t NK, NV;
  if (budget_mode == BUDGET_THETA) {
    int eb = bf16 ? 2 : 4;
    int64_t N = akvref_theta_budget(S, H, D, W, k, G, eb, eb, budget);
    NK = N / 2;
    NV = N - NK;
  } else if (budget_mode == BUDGET_COUNT) {
    NK = NV = budget_count;
  } else {
    NK = NV = (int64_t)floor((double)(float)budget * (double)H * (double)S);
  }
  if (head_budget) {
    nsel[0] = akvref_budget_select_per_head(uK, H, S, NK, selK);
    nsel[1] = akvref_budget_select_per_head(uV, H, S, NV, selV);
  } else {
    nsel[0] = akvref_budget_select(uK, H, S, NK, selK);
    nsel[1] = akvref_budget_select(uV, H, S, NV, selV);
  }
  int nb = D / 4, ns = D / G;
  memset(codesK, 0, (size_t)H * S * nb);
  memset(codesV, 0, (size_t)H * S * nb);
  memset(scalesK, 0, sizeof(float) * (size_t)H * S * ns);
  memset(scalesV, 0, sizeof(float) * (size_t)H * S * ns);
  for (int h = 0; h < H; ++h)
    for (int t = 0; t < S; ++t) {
      size_t e = (size_t)h * S + t;
      if (selK[e]) akvref_codec_encode(rK + e * D, D, G, scale_mode, seed, codesK + e * nb, scalesK + e * ns);
      if (selV[e]) akvref_codec_encode(rV + e * D, D, G, scale_mode, seed, codesV + e * nb, scalesV + e * ns);
    }
  free(rK); free(rV); free(all); free(M); free(Zs); free(Y); free(sc); free(pl);
  free(cs); free(Krot);
  return 0;
}

int akvref_encode(int H, int Hq, int D, int S, int W, int k, float rho, int kappa, int bf16,
                  uint64_t seed, int budget_mode, double budget, int64_t budget_count, int G,
                  int scale_mode, int rank_mode, int head_budget, const double* K, const double* V,
                  const double* Qobs, const int* anchor_override, int* anchors, int* aK, double* gK, int* aV,
                  double* gV, double* uK, double* uV, uint8_t* selK, uint8_t* selV,
                  uint8_t* codesK, float* scalesK, uint8_t* codesV, float* scalesV,
                  double* pooled, int64_t* nsel) {
  return encode_impl(H, Hq, D, S, W, k, rho, kappa, bf16, seed, budget_mode, budget, budget_count, G, scale_mode,
                     rank_mode, head_budget, K, V, Qobs, anchor_override, NULL, anchors, aK, gK, aV, gV, uK, uV,
                     selK, selV, codesK, scalesK, codesV, scalesV, pooled, nsel);
}

/* The compression pass with positions encoded (Sec. 3.2 "RoPE"): K holds the
 * keys before the rotation (position t of request's prompt is t) and
 * inv_freq[D/2] the rotation's frequencies.  Anchor selection, the attention
 * weights and y_w use the rotated keys, u^K uses R_t r^K_t (Eq. utilities);
 * assignment, coefficients, residuals and codes are those of the unrotated
 * keys, which is what the cache stores.  Same outputs as akvref_encode. */
int akvref_encode_rope(int H, int Hq, int D, int S, int W, int k, float rho, int kappa, int bf16,
                       uint64_t seed, int budget_mode, double budget, int64_t budget_count, int G,
                       int scale_mode, int rank_mode, int head_budget, const double* K, const double* V,
                       const double* Qobs, const int* anchor_override, const float* inv_freq, int* anchors,
                       int* aK, double* gK, int* aV, double* gV, double* uK, double* uV, uint8_t* selK,
                       uint8_t* selV, uint8_t* codesK, float* scalesK, uint8_t* codesV, float* scalesV,
                       double* pooled, int64_t* nsel) {
  if (!inv_freq) return 1;
  return encode_impl(H, Hq, D, S, W, k, rho, kappa, bf16, seed, budget_mode, budget, budget_count, G, scale_mode,
                     rank_mode, head_budget, K, V, Qobs, anchor_override, inv_freq, anchors, aK, gK, aV, gV, uK,
                     uV, selK, selV, codesK, scalesK, codesV, scalesV, pooled, nsel);
}

/* ------------------------------------------------------------------------ */
/* Reconstruction (Eq. reconstruction) and decode attention (Eq.             */
/* exact-attention over the reconstructed cache).                             */
/* ------------------------------------------------------------------------ */

/* Dense reconstruction of one side of one head, fp32:
 *   anchor positions: the stored anchor vector;
 *   others: p_j = fp32(gamma * abar_j); with a residual, x^_j = fp32(p_j + r~_j). */
void akvref_reconstruct(const double* X, int S, int D, int G, uint64_t seed, int scale_mode, const int* anchors,
                        int k, const int* a, const double* gm, const uint8_t* sel,
                        const uint8_t* codes, const float* scales, float* out) {
  int* rank = (int*)malloc(sizeof(int) * (size_t)S);
  for (int t = 0; t < S; ++t) rank[t] = -1;
  for (int i = 0; i < k; ++i) rank[anchors[i]] = i;
  float* rt = (float*)malloc(sizeof(float) * D);
  for (int t = 0; t < S; ++t) {
    float* o = out + (size_t)t * D;
    if (rank[t] >= 0) {
      for (int j = 0; j < D; ++j) o[j] = (float)X[(size_t)t * D + j];
      continue;
    }
    const double* an = X + (size_t)anchors[a[t]] * D;
    float g = (float)gm[t];
    for (int j = 0; j < D; ++j) o[j] = g * (float)an[j];
    if (sel[t]) {
      akvref_codec_decode(codes + (size_t)t * (D / 4), scales + (size_t)t * (D / G), D, G, seed, scale_mode, rt);
      for (int j = 0; j < D; ++j) o[j] = o[j] + rt[j];
    }
  }
  free(rank);
  free(rt);
}

/* Softmax attention of Hq query heads over T entries per KV head (query head
 * j reads KV head j / (Hq/H)): Kt, Vt are [H][T][D] fp32, q is [Hq][D];
 * logits dot64(q, k)*scale, softmax in fp64, output [Hq][D] fp64. */
void akvref_attention(const float* Kt, const float* Vt, int H, int T, int D, const double* q,
                      int Hq, double scale, double* out) {
  int g = Hq / H;
#pragma omp parallel for schedule(static)
  for (int j = 0; j < Hq; ++j) {
    int h = j / g;
    double* l = (double*)malloc(sizeof(double) * (size_t)T);
    double* kk = (double*)malloc(sizeof(double) * D);
    double mx = -INFINITY;
    for (int t = 0; t < T; ++t) {
      const float* kr = Kt + ((size_t)h * T + t) * D;
      for (int c = 0; c < D; ++c) kk[c] = kr[c];
      l[t] = dot64(q + (size_t)j * D, kk, D) * scale;
      if (l[t] > mx) mx = l[t];
    }
    double z = 0.0;
    for (int t = 0; t < T; ++t) z += exp(l[t] - mx);
    double* o = out + (size_t)j * D;
    for (int c = 0; c < D; ++c) o[c] = 0.0;
    for (int t = 0; t < T; ++t) {
      double p = exp(l[t] - mx) / z;
      const float* vr = Vt + ((size_t)h * T + t) * D;
      for (int c = 0; c < D; ++c) o[c] += p * vr[c];
    }
    free(l);
    free(kk);
  }
}

/* Attention with positions encoded: entry t of every head sits at position
 * t (prompt positions, then appended tokens) and its key enters the logit
 * rotated, dot64(q, R_t k_t) * scale with R_t k_t in fp64 from the table cs
 * of T positions; values are not rotated.  Otherwise as akvref_attention. */
void akvref_attention_rope(const float* Kt, const float* Vt, int H, int T, int D, const double* q,
                           int Hq, double scale, const float* cs, double* out) {
  int g = Hq / H;
#pragma omp parallel for schedule(static)
  for (int j = 0; j < Hq; ++j) {
    int h = j / g;
    double* l = (double*)malloc(sizeof(double) * (size_t)T);
    double* kk = (double*)malloc(sizeof(double) * D);
    double* kr = (double*)malloc(sizeof(double) * D);
    double mx = -INFINITY;
    for (int t = 0; t < T; ++t) {
      const float* k0 = Kt + ((size_t)h * T + t) * D;
      for (int c = 0; c < D; ++c) kk[c] = k0[c];
      akvref_rope_rotate(cs + (size_t)t * D, kk, D, kr);
      l[t] = dot64(q + (size_t)j * D, kr, D) * scale;
      if (l[t] > mx) mx = l[t];
    }
    double z = 0.0;
    for (int t = 0; t < T; ++t) z += exp(l[t] - mx);
    double* o = out + (size_t)j * D;
    for (int c = 0; c < D; ++c) o[c] = 0.0;
    for (int t = 0; t < T; ++t) {
      double p = exp(l[t] - mx) / z;
      const float* vr = Vt + ((size_t)h * T + t) * D;
      for (int c = 0; c < D; ++c) o[c] += p * vr[c];
    }
    free(l);
    free(kk);
    free(kr);
  }
}

int akvref_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the parallel loops from now on (timing only; results do not
 * depend on it). */
void akvref_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
