/*
 * anchorkv.h -- C ABI of the AnchorKV hot path for AMD MI355X (gfx950).
 *
 * AnchorKV (arXiv 2608.02901) compresses one attention layer's per-KV-head key
 * and value caches at the end of prefill (Sec. 3.2, Algorithm 1): k anchor
 * tokens per head are kept exactly, every other token is stored as the index
 * of its nearest anchor plus one projection coefficient gamma (Sec. 3.1, Eqs.
 * nearest-anchor and projection), and a head-pooled budget of tokens also
 * stores a 2-bit Hadamard-rotated residual (Sec. 3.1 "Residual quantization",
 * Sec. 3.3 utilities, Sec. 3.4 budget).  Decode attention then reads that
 * compressed cache directly; no token leaves the softmax (Sec. 3.4 "Storage
 * and Decoding"; App. E.1).
 *
 * Conventions for every entry point:
 *   - Device pointers are HIP device memory owned by the caller.  The library
 *     never allocates or frees device memory and never synchronizes the stream.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     work is enqueued on it in order; results are valid once it completes.
 *   - Host pointers are read (or written) only during the call.
 *   - Every buffer comes with its size in bytes.  A size below what the plan
 *     needs returns ANCHORKV_ERR_BUFFER_TOO_SMALL (larger buffers are fine);
 *     the library never reads or writes past the size the plan needs.
 *   - Every argument is validated before anything is enqueued.  On an error
 *     nothing is enqueued, the status says why and anchorkv_last_error()
 *     returns a detail string for the calling thread.  A HIP launch failure
 *     returns ANCHORKV_ERR_HIP; the stream state is then undefined for the
 *     work of that call.  No entry point throws or aborts.
 *   - Fault injection (tests of the error path): when the environment
 *     variable ANCHORKV_FAULT_INJECT names a kernel (e.g. "k_assign"), a call
 *     that reaches that kernel enqueues nothing from it on, and returns
 *     ANCHORKV_ERR_HIP with a message naming the kernel.
 *   - Query head j reads KV head j / (num_q_heads / num_kv_heads) (GQA).
 */
#ifndef ANCHORKV_H
#define ANCHORKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ANCHORKV_OK = 0,
  ANCHORKV_ERR_INVALID_ARG = 1,   /* null pointer, bad size, inconsistent config */
  ANCHORKV_ERR_UNSUPPORTED = 2,   /* valid for the method, outside this build's limits */
  ANCHORKV_ERR_CAPACITY = 3,      /* append beyond the capacity reserved at plan time */
  ANCHORKV_ERR_CORRUPT_CACHE = 4, /* export of a blob whose header does not match the plan */
  ANCHORKV_ERR_HIP = 5,           /* a HIP runtime call failed (or a fault was injected) */
  ANCHORKV_ERR_BUFFER_TOO_SMALL = 6 /* a buffer's size is below what the plan needs */
} anchorkv_status;

typedef enum { ANCHORKV_F32 = 0, ANCHORKV_BF16 = 1 } anchorkv_dtype;

/* Scale of the 2-bit residual codec (Sec. 3.1; App. A.1 "Codebook").  The
 * paper quantizes each rotated coordinate with the four-level Lloyd-Max
 * codebook of a unit Gaussian after normalizing by a per-token absmax; how
 * the absmax enters is not fixed by the text, so the scale sigma (the Gaussian
 * standard deviation the codebook is applied at) has three readings:
 *   OUTER   : sigma = absmax / L1 -- the largest coordinate lands on the outer level;
 *   LITERAL : sigma = absmax;
 *   RMS     : sigma = root mean square of the group's rotated coordinates.
 * NAIVE is the ablation of Sec. 4.3 ("Component Removal" (iv)): no Hadamard
 * rotation and no Lloyd-Max codebook, the uniform four-level quantizer of
 * [-A, A] (A = group absmax, levels +-A/4, +-3A/4) on the raw residual. */
typedef enum {
  ANCHORKV_SCALE_ABSMAX_OUTER = 0,
  ANCHORKV_SCALE_ABSMAX_LITERAL = 1,
  ANCHORKV_SCALE_RMS = 2,
  ANCHORKV_SCALE_NAIVE = 3
} anchorkv_scale_mode;

/* What ranks the candidates for a residual (Sec. 3.3 utilities; the
 * alternatives are the ablations of Sec. 4.3 "Residual Ranking"):
 *   UTILITY   : the attention-output-aware utilities of Eq. utilities (the method);
 *   COSINE    : 1 - |cos(x_t, anchor)|, the least aligned first;
 *   RESNORM   : the residual's squared norm;
 *   ATTENTION : the mean attention of the observation rows on the token;
 *   RANDOM    : a uniform draw (seeded).
 * Every mode ranks exactly (fp64 keys, ties to the lower head, then position). */
typedef enum {
  ANCHORKV_RANK_UTILITY = 0,
  ANCHORKV_RANK_COSINE = 1,
  ANCHORKV_RANK_RESNORM = 2,
  ANCHORKV_RANK_ATTENTION = 3,
  ANCHORKV_RANK_RANDOM = 4
} anchorkv_rank_mode;

/* Residual budget per side (Sec. 3.4).
 *   FRACTION : N_side = floor(budget * H * S) per request and side;
 *   THETA    : N = max{0, floor((theta*M_full - M_base)/b_res)} (Eq. byte-budget,
 *              with M_base from Eq. mfixed and b_res the mean key/value residual
 *              cost), keys get floor(N/2), values the rest;
 *   COUNT    : N_side = budget_count.
 * N_side is capped at the number of non-anchor tokens, H * (S - k). */
typedef enum {
  ANCHORKV_BUDGET_FRACTION = 0,
  ANCHORKV_BUDGET_THETA = 1,
  ANCHORKV_BUDGET_COUNT = 2
} anchorkv_budget_mode;

/* What an appended (generated) token stores (App. E "Generated Tokens"):
 *   ENCODED : its nearest anchor and coefficient on both sides, no residual
 *             (8 bytes per KV head at bf16), assigned against the current anchors;
 *   DENSE   : its key and value exactly, in the cache dtype (the paper's choice:
 *             generated tokens join the exact window and are never compressed). */
typedef enum { ANCHORKV_APPEND_ENCODED = 0, ANCHORKV_APPEND_DENSE = 1 } anchorkv_append_mode;

typedef struct anchorkv_config {
  int32_t num_kv_heads;   /* H */
  int32_t num_q_heads;    /* Hq, a multiple of H */
  int32_t head_dim;       /* D; this build supports D = 128 */
  int32_t window;         /* W: the last W positions are anchors and give the observation queries */
  int32_t anchor_count;   /* k per head when > 0 (window included) ... */
  float anchor_frac;      /* ... else k = max(W, floor(anchor_frac * S)), capped at S */
  float rho;              /* share of the k - W free anchors taken by score (paper: 0.7) */
  int32_t kappa;          /* odd average-pooling width of the selector score, <= 255 (paper: 7) */
  int32_t budget_mode;    /* anchorkv_budget_mode */
  float budget;           /* FRACTION: residual fraction; THETA: retained fraction theta */
  int64_t budget_count;   /* COUNT: residuals per side */
  int32_t quant_group;    /* G: coordinates per residual scale, G | D, 4 | G; 0 -> G = D */
  int32_t scale_mode;     /* anchorkv_scale_mode */
  int32_t dtype;          /* anchorkv_dtype of K, V, queries, anchors and coefficients */
  int32_t max_append;     /* capacity for tokens appended after the compression pass */
  int32_t rank_mode;      /* an anchorkv_rank_mode; 0 is the method's utilities */
  int32_t head_budget;    /* 0: the budget is pooled over heads (the method); 1: every head gets
                             floor(N_side / H) (Sec. 4.3 ablation; needs batch * H <= 64) */
  int32_t append_mode;    /* an anchorkv_append_mode */
  uint64_t seed;          /* seeds the uniform anchor share, the Hadamard signs and the random ranking */
  /* Rotary position encoding (Sec. 3.2 "RoPE"; App. E "Implementation").
   * 0: the keys are used as given (no rotation).  1: K (encode) and k_new
   * (append) hold keys BEFORE the rotation; the token at prompt position t
   * (appended token n: position S + n) enters attention as R_t k, where R_t
   * turns each rotate-half coordinate pair (f, f + D/2) by the angle
   * t * rope_inv_freq[f] (the Llama convention: x cos + rotate_half(x) sin).
   * The compression pass scores anchors and computes the attention weights
   * and y_w with the rotated keys, projects and stores the unrotated keys,
   * and ranks key residuals by q . R_t r (Eq. utilities); decode attention
   * rotates every stored key at its position.  Q_obs and q are the rotated
   * queries, as the model produces them.  The encode-side rotation uses the
   * fp32 roundings of the fp64 cos and sin of the fp64 angle; decode
   * evaluates them in fp32 within about 1e-6. */
  int32_t rope;
  float rope_inv_freq[64]; /* the D/2 frequencies (radians per position); unused entries ignored */
} anchorkv_config;

/* Derived per-request sizes (host memory). */
typedef struct anchorkv_request_info {
  int32_t seq_len;        /* S */
  int32_t anchors;        /* k */
  int32_t n_top;          /* floor(rho * (k - W)), anchors chosen by selector score */
  int32_t n_rand;         /* k - W - n_top, anchors sampled uniformly */
  int64_t residuals_k;    /* N_K: key residuals stored */
  int64_t residuals_v;    /* N_V: value residuals stored */
} anchorkv_request_info;

/* Opaque host-side plan: the config, the batch's sequence lengths and the
 * byte layout of the cache blob, all computed on the host. */
typedef struct anchorkv_plan anchorkv_plan;

/* Validates `cfg` for `batch` requests with host lengths seq_lens[batch] and
 * builds a plan.  batch in [1, 64], every S >= max(W, 1) + 1, k <= 16384.
 * On success *out owns host memory released by anchorkv_plan_destroy. */
anchorkv_status anchorkv_plan_create(const anchorkv_config* cfg, int32_t batch, const int32_t* seq_lens,
                                     anchorkv_plan** out);
void anchorkv_plan_destroy(anchorkv_plan* plan);

/* Byte sizes of the caller-provided device buffers. */
size_t anchorkv_cache_bytes(const anchorkv_plan* plan);
size_t anchorkv_encode_workspace_bytes(const anchorkv_plan* plan);
size_t anchorkv_decode_workspace_bytes(const anchorkv_plan* plan);
anchorkv_status anchorkv_plan_request(const anchorkv_plan* plan, int32_t request, anchorkv_request_info* info);

/* The compression pass (Algorithm 1) for all requests of the plan.
 *   K, V    : device, dtype; request b is a contiguous [H][S_b][D] block, the
 *             blocks packed back to back in request order.  kv_bytes: the size
 *             of each (>= sum_b H S_b D element bytes).
 *   Q_obs   : device, dtype; request b is [Hq][W][D] (the queries of the last W
 *             positions, the observation window of Sec. 3.2), packed likewise;
 *             q_obs_bytes >= batch Hq W D element bytes.
 *   anchor_pos_override : NULL, or device int32 [sum_b H*k_b]: per request and
 *             head the k_b anchor positions, strictly increasing, containing the
 *             last W positions; replaces the selection step.  An override that
 *             breaks these rules marks the cache invalid (anchorkv_export then
 *             returns ANCHORKV_ERR_CORRUPT_CACHE).  override_bytes >= 4 sum_b H k_b
 *             when it is given.
 *   cache   : device, cache_bytes >= anchorkv_cache_bytes(plan); receives the
 *             compressed layer.
 *   workspace : device, workspace_bytes >= anchorkv_encode_workspace_bytes(plan);
 *             scratch, contents undefined afterwards.  cache and workspace must
 *             not overlap the inputs. */
anchorkv_status anchorkv_encode(const anchorkv_plan* plan, const void* K, const void* V, size_t kv_bytes,
                                const void* Q_obs, size_t q_obs_bytes, const int32_t* anchor_pos_override,
                                size_t override_bytes, void* cache, size_t cache_bytes, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Appends one generated token per request and KV head (config max_append
 * slots).  ENCODED append mode: the token is encoded against the request's
 * existing anchors (its nearest anchor and coefficient, Eqs. nearest-anchor
 * and projection, with the same certified argmax and canonical coefficient as
 * the compression pass) and stores no residual.  DENSE append mode: the key
 * and value are stored exactly (App. E "Generated Tokens").  n_appended: tokens already appended to this cache
 * (host-tracked), must be < max_append, else ANCHORKV_ERR_CAPACITY.
 * k_new, v_new: device [batch][H][D], dtype, new_bytes the size of each.
 * workspace: device, workspace_bytes >= anchorkv_decode_workspace_bytes(plan),
 * contents undefined afterwards. */
anchorkv_status anchorkv_append(const anchorkv_plan* plan, void* cache, size_t cache_bytes, int32_t n_appended,
                                const void* k_new, const void* v_new, size_t new_bytes, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Decode attention over the compressed cache (Eq. exact-attention with the
 * reconstructed keys and values of Eq. reconstruction), never materializing
 * them: q.k^_t = gamma_t (q.k_a(t)) + q.r~_t and the values accumulate as
 * per-anchor weights plus a rotated residual sum (App. E.1).
 *   n_appended : appended tokens included (the first n_appended tail slots).
 *   q          : device [batch][Hq][D], dtype (q_bytes its size); query head j
 *                reads KV head j / g.
 *   out        : device [batch][Hq][D], out_dtype (anchorkv_dtype), out_bytes
 *                its size.
 *   softmax_scale : <= 0 selects 1/sqrt(D).
 *   workspace  : device, workspace_bytes >= anchorkv_decode_workspace_bytes(plan);
 *                contents undefined afterwards.  Two calls that share a
 *                workspace must not run concurrently. */
anchorkv_status anchorkv_decode_attn(const anchorkv_plan* plan, const void* cache, size_t cache_bytes,
                                     int32_t n_appended, const void* q, size_t q_bytes, void* out, size_t out_bytes,
                                     int32_t out_dtype, float softmax_scale, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* One generation step: anchorkv_append of (k_new, v_new) as tail slot
 * n_appended, then anchorkv_decode_attn over the cache including it
 * (n_appended + 1 tail tokens).  The result equals the two calls in sequence;
 * the append's anchor scan shares the attention's passes over the anchors, so
 * it adds no pass over HBM.  Arguments as in those two calls. */
anchorkv_status anchorkv_decode_step(const anchorkv_plan* plan, void* cache, size_t cache_bytes, int32_t n_appended,
                                     const void* k_new, const void* v_new, size_t new_bytes, const void* q,
                                     size_t q_bytes, void* out, size_t out_bytes, int32_t out_dtype,
                                     float softmax_scale, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * anchorkv_decode_step without the workspace argument.  Its scratch is a
 * library-owned static device array of ANCHORKV_NOALLOC_SCRATCH_BYTES per GPU,
 * held until the process ends; a plan whose decode workspace is larger
 * returns ANCHORKV_ERR_BUFFER_TOO_SMALL.  The call allocates nothing.  The
 * stream must belong to the current device.  Every call on one GPU shares
 * that GPU's array: calls that overlap on it (other streams, other threads)
 * race, so the caller serializes them.  Nothing in the array has to start at
 * zero: each call writes all the scratch it reads.  Other arguments and the
 * result as in anchorkv_decode_step. */
#define ANCHORKV_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
anchorkv_status anchorkv_decode_step_noalloc(const anchorkv_plan* plan, void* cache, size_t cache_bytes,
                                             int32_t n_appended, const void* k_new, const void* v_new,
                                             size_t new_bytes, const void* q, size_t q_bytes, void* out,
                                             size_t out_bytes, int32_t out_dtype, float softmax_scale, void* stream);

/* Dense reconstruction (Eq. reconstruction) of one side (0 = keys, 1 = values)
 * of one request: out is device fp32 [H][S_b + n_appended][D], position order,
 * out_bytes its size. */
anchorkv_status anchorkv_reconstruct(const anchorkv_plan* plan, const void* cache, size_t cache_bytes,
                                     int32_t n_appended, int32_t request, int32_t side, float* out, size_t out_bytes,
                                     void* stream);

/* Logical content of one request, in position order, from a HOST copy of the
 * cache blob (pure host code).  Every pointer is caller-allocated host memory,
 * any may be NULL to skip it.  Shapes (S = S_b, k = k_b, per side X in {K, V}):
 *   anchors [H][k] int32; a_X [H][S] int32 anchor index; gamma_X [H][S] fp32
 *   stored coefficient; sel_X [H][S] uint8 residual flag; codes_X [H][S][D/4];
 *   scales_X [H][S][D/G] (zero where no residual); tail_a_X, tail_gamma_X
 *   [H][n_appended] (-1 and 0 in DENSE append mode); stats[6]: tokens resolved by the exact fp64 path of the
 *   certified argmax, keys then values, then N_K, N_V, then the candidates
 *   whose utility bounds straddled the residual budget's cut and were re-scored
 *   in fp64, keys then values. */
typedef struct anchorkv_export_arrays {
  int32_t* anchors;
  int32_t* a_k;
  float* gamma_k;
  uint8_t* sel_k;
  uint8_t* codes_k;
  float* scales_k;
  int32_t* a_v;
  float* gamma_v;
  uint8_t* sel_v;
  uint8_t* codes_v;
  float* scales_v;
  int32_t* tail_a_k;
  float* tail_gamma_k;
  int32_t* tail_a_v;
  float* tail_gamma_v;
  int64_t* stats;
} anchorkv_export_arrays;

/* Decodes request `request` of a host copy of cache_bytes bytes (>= the
 * plan's cache size) with n_appended tail tokens.  The export is a host-side
 * reading of the layout the compression pass writes (App. A.1 "Layout"). */
anchorkv_status anchorkv_export(const anchorkv_plan* plan, const void* cache_host, size_t cache_bytes, int32_t request,
                                int32_t n_appended, anchorkv_export_arrays* out);

/* Kernel timing for benchmarks and tracing.  While enabled, every launch of
 * a kernel named in the comma-separated list `kernels` (e.g.
 * "k_dec_stream,k_assign") carries a pair of HIP events that the launch on
 * its own stream stamps with the kernel's begin and end (hipExtLaunchKernel),
 * up to max_launches pairs per kernel (events are created here, host side,
 * no device memory).  anchorkv_profile_read waits
 * for the recorded events of one kernel and returns their summed elapsed
 * milliseconds and the number of timed launches; disable releases the events.
 * Process-wide; calls are serialized by a lock. */
anchorkv_status anchorkv_profile_enable(const char* kernels, int32_t max_launches);
anchorkv_status anchorkv_profile_read(const char* kernel, float* total_ms, int32_t* launches);
anchorkv_status anchorkv_profile_disable(void);

const char* anchorkv_status_string(anchorkv_status status);
const char* anchorkv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ANCHORKV_H */
