// Host layer of the AnchorKV library: configuration checks, the byte layout
// of the cache blob and of the workspaces (a pure function of the config and
// the batch's sequence lengths), launch sequencing on the caller's stream,
// error mapping, and the host-side export of a cache blob.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "akv_common.h"
#include "anchorkv.h"

namespace akv {
hipError_t launch_init(const Geo& g, const Cache& c, const Ws& w, hipStream_t st);
hipError_t launch_obs(const Geo& g, const Ws& w, const void* K, const void* Q, hipStream_t st);
hipError_t launch_obs64(const Geo& g, const Ws& w, const void* K, const void* V, const void* Q, hipStream_t st);
hipError_t launch_rope(const Geo& g, const Ws& w, const void* K, hipStream_t st);
hipError_t launch_select(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs, const void* V,
                         const void* Q, const int32_t* ovr, hipStream_t st);
hipError_t launch_assign(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, hipStream_t st);
hipError_t launch_epilogue(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs, const void* V,
                           const void* Q, hipStream_t st);
hipError_t launch_budget(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs, const void* V,
                         hipStream_t st);
hipError_t launch_layout(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, hipStream_t st);
hipError_t launch_decode(const Geo& g, const Cache& c, const DecWs& dw, const void* q, const void* kn,
                         const void* vn, void* out, int out_dtype, float scale, int n_app, hipStream_t st);
hipError_t launch_reconstruct(const Geo& g, const Cache& c, int b, int side, int n_app, float* out,
                              hipStream_t st);
}  // namespace akv

using akv::Geo;

static const uint32_t kMagic = 0x314B5641u;  // "AVK1" little endian
static const uint32_t kVersion = 1;
static const int kBudgetChunk = 4096;

static thread_local std::string g_last_error;

static anchorkv_status fail(anchorkv_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

// ------------------------------------------------------------------ fault injection
// ANCHORKV_FAULT_INJECT=<kernel>: a device entry point that reaches that
// kernel launches nothing from it on and returns ANCHORKV_ERR_HIP.  The state
// is per thread and per call (FaultScope).
namespace {
thread_local std::string g_fi_target, g_fi_kernel;
thread_local bool g_fi_tripped = false;
struct FaultScope {
  FaultScope() {
    const char* e = getenv("ANCHORKV_FAULT_INJECT");
    g_fi_target = e ? e : "";
    g_fi_tripped = false;
  }
  ~FaultScope() { g_fi_target.clear(); }
  anchorkv_status finish(anchorkv_status s) const {
    if (s == ANCHORKV_OK && g_fi_tripped)
      return fail(ANCHORKV_ERR_HIP, "fault injected at kernel " + g_fi_kernel + " (ANCHORKV_FAULT_INJECT)");
    return s;
  }
};
}  // namespace

bool akv::launch_blocked(const char* kernel) {
  if (g_fi_tripped) return true;
  if (!g_fi_target.empty() && g_fi_target == kernel) {
    g_fi_tripped = true;
    g_fi_kernel = kernel;
    return true;
  }
  return false;
}

static anchorkv_status need_bytes(size_t have, size_t want, const char* what) {
  if (have < want)
    return fail(ANCHORKV_ERR_BUFFER_TOO_SMALL,
                std::string(what) + ": " + std::to_string(have) + " bytes, the plan needs " + std::to_string(want));
  return ANCHORKV_OK;
}

struct Layout {
  std::vector<size_t> off;
  size_t total = 0;
  size_t add(size_t bytes) {
    size_t o = total;
    off.push_back(o);
    total += (bytes + 255) & ~(size_t)255;
    return o;
  }
};

struct anchorkv_plan {
  anchorkv_config cfg;
  Geo geo;
  std::vector<anchorkv_request_info> req;
  // cache blob offsets
  size_t c_header, c_anc_pos, c_ancK, c_ancV, c_nrmK, c_nrmV, c_invK, c_invV, c_idxK, c_idxV, c_gK, c_gV, c_pos,
      c_maskK, c_maskV, c_pcK, c_pcV, c_codesK, c_codesV, c_scalesK, c_scalesV, c_tidxK, c_tidxV, c_tgK, c_tgV, c_tkd, c_tvd,
      c_stats;
  size_t cache_bytes;
  // encode workspace offsets
  size_t w_o64M, w_o64Z, w_o64O, w_M64, w_Z64, w_Y64, w_Y, w_Yhi, w_Ylo, w_ynp, w_qt,
      w_cw, w_qn, w_uL, w_uU, w_bandpos, w_bandu, w_brank, w_sc, w_rank, w_flag, w_sband, w_sbscore, w_sstate, w_sghist, w_scand, w_rkey, w_rpos, w_slcnt, w_QA, w_apos,
      w_fix, w_fixcount, w_gpos, w_xn2, w_u, w_sel, w_srec, w_bhist, w_bstate, w_bcval, w_bcpos, w_tiecnt, w_shist, w_wcnt,
      w_krot, w_cs;
  size_t ws_bytes;
  // decode workspace offsets
  size_t d_SK, d_RK, d_part, d_asc, d_atop, d_LK;
  size_t dws_bytes;
};

static int64_t theta_residuals(int S, int H, int D, int W, int k, int G, int eb, double theta) {
  // Eq. byte-budget with M_base from Eq. mfixed (b_a = 2, b_gamma = element size).
  const double P = (double)(S - W);
  const double words = ceil(P / 64.0);
  const double Mbase = (double)H * (2.0 * eb * k * D + 8.0 * (k - W) + 2.0 * P * (2.0 + eb)) + 24.0 * H * words +
                       8.0 * (H + 1) + 4.0 * P;
  const double Mfull = 2.0 * eb * (double)S * H * D;
  const double cK = D / 4.0 + 4.0 * (D / G);
  const double bres = 0.5 * (cK + (cK + 1.0));
  const double n = floor((theta * Mfull - Mbase) / bres);
  return n > 0 ? (int64_t)n : 0;
}

static uint64_t mix64(uint64_t x) { return akv::splitmix64(x); }

extern "C" anchorkv_status anchorkv_plan_create(const anchorkv_config* cfg, int32_t batch, const int32_t* seq_lens,
                                                anchorkv_plan** out) {
  if (!cfg || !seq_lens || !out) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  const anchorkv_config& c = *cfg;
  if (batch < 1 || batch > AKV_MAXB) return fail(ANCHORKV_ERR_INVALID_ARG, "batch must be in [1, 64]");
  if (c.num_kv_heads < 1 || c.num_kv_heads > 255) return fail(ANCHORKV_ERR_INVALID_ARG, "num_kv_heads must be in [1, 255]");
  if (c.num_q_heads < c.num_kv_heads || c.num_q_heads % c.num_kv_heads)
    return fail(ANCHORKV_ERR_INVALID_ARG, "num_q_heads must be a positive multiple of num_kv_heads");
  const int g = c.num_q_heads / c.num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8)
    return fail(ANCHORKV_ERR_UNSUPPORTED, "query heads per KV head must be 1, 2, 4 or 8");
  if (c.head_dim <= 0 || (c.head_dim & (c.head_dim - 1)))
    return fail(ANCHORKV_ERR_INVALID_ARG, "head_dim must be a power of two");
  if (c.head_dim != AKV_D) return fail(ANCHORKV_ERR_UNSUPPORTED, "this build supports head_dim = 128");
  if (c.window < 1) return fail(ANCHORKV_ERR_INVALID_ARG, "window must be >= 1");
  if (c.window * g > 256) return fail(ANCHORKV_ERR_UNSUPPORTED, "window * (Hq/H) must be <= 256");
  if (c.kappa < 1 || (c.kappa & 1) == 0 || c.kappa > 255)
    return fail(ANCHORKV_ERR_INVALID_ARG, "kappa must be odd, in [1, 255]");
  if (!(c.rho >= 0.0f && c.rho <= 1.0f)) return fail(ANCHORKV_ERR_INVALID_ARG, "rho must be in [0, 1]");
  if (c.dtype != ANCHORKV_F32 && c.dtype != ANCHORKV_BF16) return fail(ANCHORKV_ERR_INVALID_ARG, "bad dtype");
  const int G = c.quant_group ? c.quant_group : c.head_dim;
  if (G < 4 || G % 4 || c.head_dim % G) return fail(ANCHORKV_ERR_INVALID_ARG, "quant_group must divide head_dim and be a multiple of 4");
  if (G < 32) return fail(ANCHORKV_ERR_UNSUPPORTED, "this build supports quant_group 32, 64 or 128");
  if (c.scale_mode < 0 || c.scale_mode > 3) return fail(ANCHORKV_ERR_INVALID_ARG, "bad scale_mode");
  if (c.rank_mode < 0 || c.rank_mode > 4) return fail(ANCHORKV_ERR_INVALID_ARG, "bad rank_mode");
  if (c.head_budget != 0 && c.head_budget != 1) return fail(ANCHORKV_ERR_INVALID_ARG, "head_budget must be 0 or 1");
  if (c.append_mode != ANCHORKV_APPEND_ENCODED && c.append_mode != ANCHORKV_APPEND_DENSE)
    return fail(ANCHORKV_ERR_INVALID_ARG, "bad append_mode");
  if (c.head_budget && (int64_t)batch * c.num_kv_heads > AKV_MAXB)
    return fail(ANCHORKV_ERR_UNSUPPORTED, "equal per-head budgets need batch * num_kv_heads <= 64");
  if (c.budget_mode < 0 || c.budget_mode > 2) return fail(ANCHORKV_ERR_INVALID_ARG, "bad budget_mode");
  if (!(c.budget >= 0.0f) || (c.budget_mode != ANCHORKV_BUDGET_COUNT && c.budget > 1.0f))
    return fail(ANCHORKV_ERR_INVALID_ARG, "budget must be in [0, 1]");
  if (c.budget_mode == ANCHORKV_BUDGET_COUNT && c.budget_count < 0)
    return fail(ANCHORKV_ERR_INVALID_ARG, "budget_count must be >= 0");
  if (c.max_append < 0) return fail(ANCHORKV_ERR_INVALID_ARG, "max_append must be >= 0");
  if (c.anchor_count == 0 && !(c.anchor_frac > 0.0f && c.anchor_frac <= 1.0f))
    return fail(ANCHORKV_ERR_INVALID_ARG, "anchor_frac must be in (0, 1] when anchor_count = 0");
  if (c.anchor_count < 0) return fail(ANCHORKV_ERR_INVALID_ARG, "anchor_count must be >= 0");
  if (c.rope != 0 && c.rope != 1) return fail(ANCHORKV_ERR_INVALID_ARG, "rope must be 0 or 1");
  if (c.rope)
    for (int f = 0; f < c.head_dim / 2 && f < 64; ++f)
      if (!(c.rope_inv_freq[f] >= 0.0f && c.rope_inv_freq[f] <= 1e6f))
        return fail(ANCHORKV_ERR_INVALID_ARG, "rope_inv_freq must be finite and >= 0");

  anchorkv_plan* p = new (std::nothrow) anchorkv_plan();
  if (!p) return fail(ANCHORKV_ERR_INVALID_ARG, "out of host memory");
  p->cfg = c;
  Geo& geo = p->geo;
  memset(&geo, 0, sizeof(geo));
  const int H = c.num_kv_heads, D = c.head_dim, W = c.window;
  geo.B = batch;
  geo.H = H;
  geo.Hq = c.num_q_heads;
  geo.g = g;
  geo.D = D;
  geo.W = W;
  geo.G = G;
  geo.m = W * g;
  geo.dtype = c.dtype;
  geo.esz = c.dtype == ANCHORKV_BF16 ? 2 : 4;
  geo.kappa = c.kappa;
  geo.scale_mode = c.scale_mode;
  // Codec levels and threshold in units of the stored scale: the Lloyd-Max
  // pair for the rotated codec, the uniform grid {1, 3} (threshold 2) for the
  // naive one, whose scale is a quarter of the group absmax.
  geo.rot = c.scale_mode != ANCHORKV_SCALE_NAIVE;
  geo.lev0 = geo.rot ? AKV_L0 : 1.0f;
  geo.lev1 = geo.rot ? AKV_L1 : 3.0f;
  geo.thr = geo.rot ? AKV_T : 2.0f;
  geo.rank_mode = c.rank_mode;
  geo.hdiv = c.head_budget ? c.num_kv_heads : 1;
  geo.seed_rank = mix64(c.seed ^ 3ull);
  geo.dense_tail = c.append_mode == ANCHORKV_APPEND_DENSE;
  geo.max_append = c.max_append;
  geo.seed_anchor = mix64(c.seed ^ 1ull);
  geo.seed_sign = mix64(c.seed ^ 2ull);
  geo.rope = c.rope;
  for (int f = 0; f < D / 2; ++f) geo.invf[f] = c.rope ? c.rope_inv_freq[f] : 0.0f;
  geo.sgnbits[0] = geo.sgnbits[1] = 0;
  for (int j = 0; j < D; ++j)
    if (mix64(geo.seed_sign ^ (uint64_t)j) >> 63) geo.sgnbits[j >> 6] |= 1ull << (j & 63);
  int64_t totS = 0;
  for (int b = 0; b < batch; ++b) {
    const int S = seq_lens[b];
    if (S <= W) {
      delete p;
      return fail(ANCHORKV_ERR_INVALID_ARG, "every sequence must be longer than the window");
    }
    if (S > (1 << 22)) {
      delete p;
      return fail(ANCHORKV_ERR_UNSUPPORTED, "sequence length above 4M");
    }
    int k;
    if (c.anchor_count > 0) {
      k = c.anchor_count < S ? c.anchor_count : S;
    } else {
      k = (int)floor((double)c.anchor_frac * (double)S);
      if (k < W) k = W;
      if (k > S) k = S;
    }
    if (k < W) {
      delete p;
      return fail(ANCHORKV_ERR_INVALID_ARG, "anchor count must include the window (k >= W)");
    }
    if (k > AKV_MAXK) {
      delete p;
      return fail(ANCHORKV_ERR_UNSUPPORTED, "more than 16384 anchors per head");
    }
    const int ntop = (int)floor((double)c.rho * (double)(k - W));
    const int64_t ncand = (int64_t)H * (S - k);
    int64_t NK, NV;
    if (c.budget_mode == ANCHORKV_BUDGET_FRACTION) {
      NK = NV = (int64_t)floor((double)c.budget * (double)H * (double)S);
    } else if (c.budget_mode == ANCHORKV_BUDGET_THETA) {
      const int64_t N = theta_residuals(S, H, D, W, k, G, geo.esz, (double)c.budget);
      NK = N / 2;
      NV = N - NK;
    } else {
      NK = NV = c.budget_count;
    }
    if (NK > ncand) NK = ncand;
    if (NV > ncand) NV = ncand;
    if (c.head_budget) {  // every head takes floor(N_side / H)
      NK = NK / H * H;
      NV = NV / H * H;
    }
    anchorkv_request_info ri;
    ri.seq_len = S;
    ri.anchors = k;
    ri.n_top = ntop;
    ri.n_rand = k - W - ntop;
    ri.residuals_k = NK;
    ri.residuals_v = NV;
    p->req.push_back(ri);
    geo.S[b] = S;
    geo.k[b] = k;
    geo.ntop[b] = ntop;
    geo.nrand[b] = k - W - ntop;
    geo.maxS = S > geo.maxS ? S : geo.maxS;
    geo.maxK = k > geo.maxK ? k : geo.maxK;
    totS += S;
  }
  if (totS * H >= (1ll << 30)) {
    delete p;
    return fail(ANCHORKV_ERR_UNSUPPORTED, "total tokens x heads above 2^30");
  }
  // Every prefix sum below must fit the int32 offsets the kernels use.
  {
    int64_t kt = 0;
    for (int b = 0; b < batch; ++b)
      kt += (int64_t)H * geo.k[b] * ((geo.S[b] + akv::SORT_CHUNK - 1) / akv::SORT_CHUNK + 1);
    if (kt >= (1ll << 31) - 1) {
      delete p;
      return fail(ANCHORKV_ERR_UNSUPPORTED, "anchors x heads x sort chunks above 2^31");
    }
  }
  for (int b = 0; b < batch; ++b) {
    const int S = geo.S[b], k = geo.k[b];
    geo.prefS[b + 1] = geo.prefS[b] + S;
    geo.prefK[b + 1] = geo.prefK[b] + k;
    geo.prefW[b + 1] = geo.prefW[b] + (S + 63) / 64;
    geo.prefC[b + 1] = geo.prefC[b] + (S + akv::OBS_CHUNK - 1) / akv::OBS_CHUNK;
    geo.prefKT[b + 1] = geo.prefKT[b] + H * k * ((S + akv::SORT_CHUNK - 1) / akv::SORT_CHUNK + 1);
    geo.prefBC[b + 1] = geo.prefBC[b] + geo.hdiv * ((H / geo.hdiv * S + kBudgetChunk - 1) / kBudgetChunk);
    geo.prefKp[b + 1] = geo.prefKp[b] + ((k + 3) & ~3);
    geo.prefAB[b + 1] = geo.prefAB[b] + (k + 255) / 256;
    geo.prefNK[b + 1] = geo.prefNK[b] + (int)p->req[b].residuals_k;
    geo.prefNV[b + 1] = geo.prefNV[b] + (int)p->req[b].residuals_v;
  }
  // fp64 observation chunks: the smallest power of two (>= 256 tokens) that
  // keeps the launch at about 1024 workgroups of 64 rows and a head at <= 256
  // chunks (the partial outputs are 1 KB per chunk and row).
  {
    geo.mpad = (geo.m + 15) / 16 * 16;
    const int nrg = (geo.m + 63) / 64;
    int oc = 256;
    for (;;) {
      int64_t n = 0;
      for (int b = 0; b < batch; ++b) n += (int64_t)H * nrg * ((geo.S[b] + oc - 1) / oc);
      if ((n <= 1024 && (geo.maxS + oc - 1) / oc <= 256) || oc >= (1 << 16)) break;
      oc *= 2;
    }
    geo.oc64 = oc;
    for (int b = 0; b < batch; ++b) geo.prefC64[b + 1] = geo.prefC64[b] + (geo.S[b] + oc - 1) / oc;
  }
  // Decode split: 2048 sorted slots per workgroup when that still gives at
  // least 256 workgroups (one per CU), else 1024.
  {
    int Lsel = 1024;
    int64_t n = 0;
    for (int b = 0; b < batch; ++b) n += (int64_t)H * ((geo.S[b] + 2047) / 2048);
    if (n >= 256) Lsel = 2048;
    geo.dsplit = Lsel;
    // split records per query head: the splits plus one for the appended tail
    for (int b = 0; b < batch; ++b) geo.prefSp[b + 1] = geo.prefSp[b] + (geo.S[b] + Lsel - 1) / Lsel + 1;
  }
  const size_t TS = (size_t)geo.prefS[batch] * H, TK = (size_t)geo.prefK[batch] * H,
               TW = (size_t)geo.prefW[batch] * H;
  const size_t NKt = geo.prefNK[batch], NVt = geo.prefNV[batch];
  const size_t esz = geo.esz, m = geo.m, cap = c.max_append;
  Layout L;
  p->c_header = L.add(256);
  p->c_anc_pos = L.add(4 * TK);
  p->c_ancK = L.add(esz * TK * D);
  p->c_ancV = L.add(esz * TK * D);
  p->c_nrmK = L.add(8 * TK);
  p->c_nrmV = L.add(8 * TK);
  p->c_invK = L.add(4 * TK);
  p->c_invV = L.add(4 * TK);
  const size_t TSP = TW * 64;  // per-slot arrays: each head padded to whole mask words
  p->c_idxK = L.add(2 * TSP);
  p->c_idxV = L.add(2 * TSP);
  p->c_gK = L.add(esz * TSP);
  p->c_gV = L.add(esz * TSP);
  p->c_pos = L.add(4 * TSP);
  p->c_maskK = L.add(8 * TW);
  p->c_maskV = L.add(8 * TW);
  p->c_pcK = L.add(4 * TW);
  p->c_pcV = L.add(4 * TW);
  p->c_codesK = L.add(NKt * (D / 4));
  p->c_codesV = L.add(NVt * (D / 4));
  p->c_scalesK = L.add(4 * NKt * (D / G));
  p->c_scalesV = L.add(4 * NVt * (D / G));
  p->c_tidxK = L.add(2 * batch * H * cap);
  p->c_tidxV = L.add(2 * batch * H * cap);
  p->c_tgK = L.add(esz * batch * H * cap);
  p->c_tgV = L.add(esz * batch * H * cap);
  const size_t dcap = geo.dense_tail ? (size_t)cap : 0;
  p->c_tkd = L.add(esz * batch * H * dcap * D);
  p->c_tvd = L.add(esz * batch * H * dcap * D);
  p->c_stats = L.add(4 * 4 * batch);
  p->cache_bytes = L.total;

  Layout Wl;
  {
    const size_t TC64 = (size_t)geo.prefC64[batch] * H, mp = geo.mpad;
    p->w_o64M = Wl.add(8 * TC64 * mp);
    p->w_o64Z = Wl.add(8 * TC64 * mp);
    p->w_o64O = Wl.add(8 * TC64 * mp * D);
  }
  p->w_M64 = Wl.add(8 * batch * H * m);
  p->w_Z64 = Wl.add(8 * batch * H * m);
  p->w_Y64 = Wl.add(8 * batch * H * m * D);
  p->w_cw = Wl.add(4 * batch * H * m);
  p->w_qn = Wl.add(4 * batch * H * m);
  p->w_Y = Wl.add(4 * batch * H * m * D);
  p->w_Yhi = Wl.add(2 * batch * H * m * D);
  p->w_Ylo = Wl.add(2 * batch * H * m * D);
  p->w_ynp = Wl.add(8 * 4 * batch * H * m);
  p->w_qt = Wl.add(esz * batch * H * m * D);
  p->w_sc = Wl.add(4 * TS);
  p->w_rank = Wl.add(4 * TS);
  p->w_flag = Wl.add(TS);
  p->w_sband = Wl.add(4 * (size_t)batch * H * akv::SEL_BAND_MAX);
  p->w_sbscore = Wl.add(8 * (size_t)batch * H * akv::SEL_BAND_MAX);
  p->w_sstate = Wl.add(4 * akv::SS_N * (size_t)batch * H);
  p->w_sghist = Wl.add(4 * 4096 * (size_t)batch * H);
  p->w_scand = Wl.add(4 * (size_t)akv::SEL_CMAX * batch * H);
  p->w_rkey = Wl.add(8 * (size_t)akv::SEL_CAND * batch * H);
  p->w_rpos = Wl.add(4 * (size_t)akv::SEL_CAND * batch * H);
  p->w_slcnt = Wl.add(4 * (size_t)((geo.maxS + akv::SEL_SLICE - 1) / akv::SEL_SLICE) * batch * H);
  p->w_QA = Wl.add(4 * TK * m);
  p->w_apos = Wl.add(4 * 2 * TS);
  p->w_fix = Wl.add(8 * 2 * TS);
  p->w_fixcount = Wl.add(4 * 2 * (size_t)H * batch);
  p->w_gpos = Wl.add(4 * 2 * TS);
  p->w_xn2 = Wl.add(4 * 2 * TS);
  p->w_u = Wl.add(4 * 2 * TS);
  p->w_uL = Wl.add(4 * 2 * TS);
  p->w_uU = Wl.add(4 * 2 * TS);
  p->w_sel = Wl.add(2 * TS);
  p->w_srec = Wl.add(16 * TW * 64);
  // budget lists: one per request and side, or one per request, head and
  // side with equal per-head budgets
  const size_t nlist = (size_t)batch * geo.hdiv;
  p->w_bhist = Wl.add(4 * 2 * 4096 * nlist);
  p->w_bstate = Wl.add(4 * 2 * akv::BST_N * nlist);
  p->w_bandpos = Wl.add(4 * 2 * (size_t)akv::BAND_CAP * nlist);
  p->w_bandu = Wl.add(8 * 2 * (size_t)akv::BAND_CAP * nlist);
  p->w_brank = Wl.add(4 * 2 * (size_t)akv::BAND_CAP * nlist);
  p->w_bcval = Wl.add(4 * 2 * (size_t)32768 * nlist);
  p->w_bcpos = Wl.add(4 * 2 * (size_t)32768 * nlist);
  p->w_tiecnt = Wl.add(4 * 2 * (size_t)geo.prefBC[batch]);
  p->w_shist = Wl.add(4 * (size_t)geo.prefKT[batch]);
  p->w_wcnt = Wl.add(4 * 2 * TW);
  p->w_krot = Wl.add(c.rope ? esz * TS * D : 0);
  p->w_cs = Wl.add(c.rope ? 4 * (size_t)geo.maxS * D : 0);
  p->ws_bytes = Wl.total;

  Layout Dl;
  p->d_SK = Dl.add(4 * (size_t)geo.prefKp[batch] * H * g);
  p->d_RK = Dl.add(4 * (size_t)geo.prefNK[batch] * g);
  p->d_part = Dl.add(4 * (size_t)geo.prefSp[batch] * geo.Hq * (4 + D));
  p->d_asc = Dl.add(4 * 2 * (size_t)geo.prefKp[batch] * H);
  p->d_atop = Dl.add(16 * 2 * 4 * (size_t)geo.prefAB[batch] * H);
  p->d_LK = Dl.add(c.rope ? 4 * TSP * g : 0);
  p->dws_bytes = Dl.total;
  *out = p;
  return ANCHORKV_OK;
}

extern "C" void anchorkv_plan_destroy(anchorkv_plan* plan) { delete plan; }
extern "C" size_t anchorkv_cache_bytes(const anchorkv_plan* p) { return p ? p->cache_bytes : 0; }
extern "C" size_t anchorkv_encode_workspace_bytes(const anchorkv_plan* p) { return p ? p->ws_bytes : 0; }
extern "C" size_t anchorkv_decode_workspace_bytes(const anchorkv_plan* p) { return p ? p->dws_bytes : 0; }

extern "C" anchorkv_status anchorkv_plan_request(const anchorkv_plan* p, int32_t request, anchorkv_request_info* info) {
  if (!p || !info) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  if (request < 0 || request >= p->geo.B) return fail(ANCHORKV_ERR_INVALID_ARG, "request out of range");
  *info = p->req[request];
  return ANCHORKV_OK;
}

template <typename T>
static T* at(void* base, size_t off) {
  return (T*)((char*)base + off);
}

static akv::Cache cache_ptrs(const anchorkv_plan* p, void* base) {
  akv::Cache c;
  c.header = at<uint32_t>(base, p->c_header);
  c.anc_pos = at<int32_t>(base, p->c_anc_pos);
  c.ancK = at<void>(base, p->c_ancK);
  c.ancV = at<void>(base, p->c_ancV);
  c.nrmK = at<double>(base, p->c_nrmK);
  c.nrmV = at<double>(base, p->c_nrmV);
  c.invK = at<float>(base, p->c_invK);
  c.invV = at<float>(base, p->c_invV);
  c.idxK = at<uint16_t>(base, p->c_idxK);
  c.idxV = at<uint16_t>(base, p->c_idxV);
  c.gK = at<void>(base, p->c_gK);
  c.gV = at<void>(base, p->c_gV);
  c.pos = at<int32_t>(base, p->c_pos);
  c.maskK = at<uint64_t>(base, p->c_maskK);
  c.maskV = at<uint64_t>(base, p->c_maskV);
  c.pcK = at<int32_t>(base, p->c_pcK);
  c.pcV = at<int32_t>(base, p->c_pcV);
  c.codesK = at<uint8_t>(base, p->c_codesK);
  c.codesV = at<uint8_t>(base, p->c_codesV);
  c.scalesK = at<float>(base, p->c_scalesK);
  c.scalesV = at<float>(base, p->c_scalesV);
  c.tidxK = at<uint16_t>(base, p->c_tidxK);
  c.tidxV = at<uint16_t>(base, p->c_tidxV);
  c.tgK = at<void>(base, p->c_tgK);
  c.tgV = at<void>(base, p->c_tgV);
  c.tkd = at<void>(base, p->c_tkd);
  c.tvd = at<void>(base, p->c_tvd);
  c.stats = at<int32_t>(base, p->c_stats);
  return c;
}

static akv::Ws ws_ptrs(const anchorkv_plan* p, void* base) {
  akv::Ws w;
  w.o64M = at<double>(base, p->w_o64M);
  w.o64Z = at<double>(base, p->w_o64Z);
  w.o64O = at<double>(base, p->w_o64O);
  w.M64 = at<double>(base, p->w_M64);
  w.Z64 = at<double>(base, p->w_Z64);
  w.Y64 = at<double>(base, p->w_Y64);
  w.cw = at<float>(base, p->w_cw);
  w.qn = at<float>(base, p->w_qn);
  w.Y = at<float>(base, p->w_Y);
  w.Yhi = at<uint16_t>(base, p->w_Yhi);
  w.Ylo = at<uint16_t>(base, p->w_Ylo);
  w.ynp = at<double>(base, p->w_ynp);
  w.qt = at<uint8_t>(base, p->w_qt);
  w.sc = at<float>(base, p->w_sc);
  w.rank = at<int32_t>(base, p->w_rank);
  w.flag = at<uint8_t>(base, p->w_flag);
  w.sband = at<int32_t>(base, p->w_sband);
  w.sbscore = at<double>(base, p->w_sbscore);
  w.sstate = at<int32_t>(base, p->w_sstate);
  w.sghist = at<uint32_t>(base, p->w_sghist);
  w.scand = at<float>(base, p->w_scand);
  w.rkey = at<unsigned long long>(base, p->w_rkey);
  w.rpos = at<int32_t>(base, p->w_rpos);
  w.slcnt = at<int32_t>(base, p->w_slcnt);
  w.QA = at<float>(base, p->w_QA);
  w.apos = at<int32_t>(base, p->w_apos);
  w.fixt = at<int32_t>(base, p->w_fix);
  w.fixb = (float*)(w.fixt + 2 * (size_t)p->geo.H * p->geo.prefS[p->geo.B]);
  w.fixcount = at<int32_t>(base, p->w_fixcount);
  w.gpos = at<float>(base, p->w_gpos);
  w.xn2 = at<float>(base, p->w_xn2);
  w.u = at<float>(base, p->w_u);
  w.uL = at<float>(base, p->w_uL);
  w.uU = at<float>(base, p->w_uU);
  w.sel = at<uint8_t>(base, p->w_sel);
  w.srec = at<uint4>(base, p->w_srec);
  w.bhist = at<uint32_t>(base, p->w_bhist);
  w.bstate = at<int32_t>(base, p->w_bstate);
  w.bandpos = at<int32_t>(base, p->w_bandpos);
  w.bandu = at<double>(base, p->w_bandu);
  w.brank = at<int32_t>(base, p->w_brank);
  w.bcval = at<float>(base, p->w_bcval);
  w.bcpos = at<int32_t>(base, p->w_bcpos);
  w.tiecnt = at<int32_t>(base, p->w_tiecnt);
  w.shist = at<int32_t>(base, p->w_shist);
  w.wcnt = at<int32_t>(base, p->w_wcnt);
  w.krot = at<void>(base, p->w_krot);
  w.cs = at<float>(base, p->w_cs);
  return w;
}

static akv::DecWs dws_ptrs(const anchorkv_plan* p, void* base) {
  akv::DecWs d;
  d.SK = at<float>(base, p->d_SK);
  d.RK = at<float>(base, p->d_RK);
  d.part = at<float>(base, p->d_part);
  d.asc = at<float>(base, p->d_asc);
  d.atop = at<float4>(base, p->d_atop);
  d.LK = at<float>(base, p->d_LK);
  return d;
}

static anchorkv_status hip_status(hipError_t e, const char* what) {
  if (g_fi_tripped)  // an injected fault: nothing was launched from that kernel on
    return fail(ANCHORKV_ERR_HIP, "fault injected at kernel " + g_fi_kernel + " (ANCHORKV_FAULT_INJECT)");
  if (e == hipSuccess) return ANCHORKV_OK;
  return fail(ANCHORKV_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Bytes the plan needs for each caller buffer.
static size_t kv_need(const anchorkv_plan* p) { return (size_t)p->geo.prefS[p->geo.B] * p->geo.H * p->geo.D * p->geo.esz; }
static size_t qobs_need(const anchorkv_plan* p) {
  return (size_t)p->geo.B * p->geo.Hq * p->geo.W * p->geo.D * p->geo.esz;
}
static size_t override_need(const anchorkv_plan* p) { return 4 * (size_t)p->geo.prefK[p->geo.B] * p->geo.H; }
static size_t new_need(const anchorkv_plan* p) { return (size_t)p->geo.B * p->geo.H * p->geo.D * p->geo.esz; }
static size_t q_need(const anchorkv_plan* p) { return (size_t)p->geo.B * p->geo.Hq * p->geo.D * p->geo.esz; }
static size_t out_need(const anchorkv_plan* p, int out_dtype) {
  return (size_t)p->geo.B * p->geo.Hq * p->geo.D * (out_dtype == ANCHORKV_F32 ? 4 : 2);
}

extern "C" anchorkv_status anchorkv_encode(const anchorkv_plan* p, const void* K, const void* V, size_t kv_bytes,
                                           const void* Q_obs, size_t q_obs_bytes, const int32_t* anchor_pos_override,
                                           size_t override_bytes, void* cache, size_t cache_bytes, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  if (!p || !K || !V || !Q_obs || !cache || !workspace) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  anchorkv_status s;
  if ((s = need_bytes(kv_bytes, kv_need(p), "K / V")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(q_obs_bytes, qobs_need(p), "Q_obs")) != ANCHORKV_OK) return s;
  if (anchor_pos_override && (s = need_bytes(override_bytes, override_need(p), "anchor override")) != ANCHORKV_OK)
    return s;
  if ((s = need_bytes(cache_bytes, p->cache_bytes, "cache")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(workspace_bytes, p->ws_bytes, "encode workspace")) != ANCHORKV_OK) return s;
  const FaultScope fs;
  const hipStream_t st = (hipStream_t)stream;
  const akv::Cache c = cache_ptrs(p, cache);
  const akv::Ws w = ws_ptrs(p, workspace);
  const Geo& g = p->geo;
  (void)hipGetLastError();
  if ((s = hip_status(akv::launch_init(g, c, w, st), "init")) != ANCHORKV_OK) return s;
  // With positions encoded the observation pass, the selection band and the
  // attention weights of the utilities read the rotated keys; assignment,
  // anchors, coefficients and residuals read the keys as given.
  const void* Kobs = K;
  if (g.rope) {
    if ((s = hip_status(akv::launch_rope(g, w, K, st), "rotation")) != ANCHORKV_OK) return s;
    Kobs = w.krot;
  }
  if ((s = hip_status(akv::launch_obs64(g, w, Kobs, V, Q_obs, st), "fp64 observation pass")) != ANCHORKV_OK) return s;
  if ((s = hip_status(akv::launch_obs(g, w, Kobs, Q_obs, st), "observation pass")) != ANCHORKV_OK) return s;
  if ((s = hip_status(akv::launch_select(g, w, c, K, Kobs, V, Q_obs, anchor_pos_override, st), "anchor selection")) !=
      ANCHORKV_OK)
    return s;
  if ((s = hip_status(akv::launch_assign(g, w, c, K, V, st), "assignment")) != ANCHORKV_OK) return s;
  if ((s = hip_status(akv::launch_epilogue(g, w, c, K, Kobs, V, Q_obs, st), "utilities")) != ANCHORKV_OK) return s;
  if ((s = hip_status(akv::launch_budget(g, w, c, K, Kobs, V, st), "budget")) != ANCHORKV_OK) return s;
  if ((s = hip_status(akv::launch_layout(g, w, c, K, V, st), "layout")) != ANCHORKV_OK) return s;
  return fs.finish(ANCHORKV_OK);
}

extern "C" anchorkv_status anchorkv_append(const anchorkv_plan* p, void* cache, size_t cache_bytes, int32_t n_appended,
                                           const void* k_new, const void* v_new, size_t new_bytes, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  if (!p || !cache || !k_new || !v_new || !workspace) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  if (n_appended < 0) return fail(ANCHORKV_ERR_INVALID_ARG, "n_appended must be >= 0");
  if (n_appended >= p->cfg.max_append) return fail(ANCHORKV_ERR_CAPACITY, "append capacity exhausted");
  anchorkv_status s;
  if ((s = need_bytes(cache_bytes, p->cache_bytes, "cache")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(new_bytes, new_need(p), "k_new / v_new")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(workspace_bytes, p->dws_bytes, "decode workspace")) != ANCHORKV_OK) return s;
  const FaultScope fs;
  (void)hipGetLastError();
  return fs.finish(hip_status(akv::launch_decode(p->geo, cache_ptrs(p, cache), dws_ptrs(p, workspace), nullptr, k_new,
                                                 v_new, nullptr, 0, 0.0f, n_appended, (hipStream_t)stream),
                              "append"));
}

extern "C" anchorkv_status anchorkv_decode_attn(const anchorkv_plan* p, const void* cache, size_t cache_bytes,
                                                int32_t n_appended, const void* q, size_t q_bytes, void* out,
                                                size_t out_bytes, int32_t out_dtype, float softmax_scale,
                                                void* workspace, size_t workspace_bytes, void* stream) {
  if (!p || !cache || !q || !out || !workspace) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  if (n_appended < 0 || n_appended > p->cfg.max_append)
    return fail(ANCHORKV_ERR_INVALID_ARG, "n_appended must be in [0, max_append]");
  if (out_dtype != ANCHORKV_F32 && out_dtype != ANCHORKV_BF16) return fail(ANCHORKV_ERR_INVALID_ARG, "bad out_dtype");
  anchorkv_status s;
  if ((s = need_bytes(cache_bytes, p->cache_bytes, "cache")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(q_bytes, q_need(p), "q")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(out_bytes, out_need(p, out_dtype), "out")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(workspace_bytes, p->dws_bytes, "decode workspace")) != ANCHORKV_OK) return s;
  const float scale = softmax_scale > 0.0f ? softmax_scale : 1.0f / sqrtf((float)p->geo.D);
  const FaultScope fs;
  (void)hipGetLastError();
  return fs.finish(hip_status(akv::launch_decode(p->geo, cache_ptrs(p, (void*)cache), dws_ptrs(p, workspace), q,
                                                 nullptr, nullptr, out, out_dtype, scale, n_appended,
                                                 (hipStream_t)stream),
                              "decode"));
}

extern "C" anchorkv_status anchorkv_decode_step(const anchorkv_plan* p, void* cache, size_t cache_bytes,
                                                int32_t n_appended, const void* k_new, const void* v_new,
                                                size_t new_bytes, const void* q, size_t q_bytes, void* out,
                                                size_t out_bytes, int32_t out_dtype, float softmax_scale,
                                                void* workspace, size_t workspace_bytes, void* stream) {
  if (!p || !cache || !k_new || !v_new || !q || !out || !workspace)
    return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  if (n_appended < 0) return fail(ANCHORKV_ERR_INVALID_ARG, "n_appended must be >= 0");
  if (n_appended >= p->cfg.max_append) return fail(ANCHORKV_ERR_CAPACITY, "append capacity exhausted");
  if (out_dtype != ANCHORKV_F32 && out_dtype != ANCHORKV_BF16) return fail(ANCHORKV_ERR_INVALID_ARG, "bad out_dtype");
  anchorkv_status s;
  if ((s = need_bytes(cache_bytes, p->cache_bytes, "cache")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(new_bytes, new_need(p), "k_new / v_new")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(q_bytes, q_need(p), "q")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(out_bytes, out_need(p, out_dtype), "out")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(workspace_bytes, p->dws_bytes, "decode workspace")) != ANCHORKV_OK) return s;
  const float scale = softmax_scale > 0.0f ? softmax_scale : 1.0f / sqrtf((float)p->geo.D);
  const FaultScope fs;
  (void)hipGetLastError();
  return fs.finish(hip_status(akv::launch_decode(p->geo, cache_ptrs(p, cache), dws_ptrs(p, workspace), q, k_new,
                                                 v_new, out, out_dtype, scale, n_appended, (hipStream_t)stream),
                              "decode step"));
}

// ------------------------------------------------------------------ no-allocation decode step
// The scratch of anchorkv_decode_step_noalloc: one static device array per
// GPU.  In host code `scratch` only names the symbol; its device address is
// looked up once per device (with that device current) and kept.
static __device__ __align__(256) unsigned char scratch[ANCHORKV_NOALLOC_SCRATCH_BYTES];
namespace {
std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

static anchorkv_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(ANCHORKV_ERR_UNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(ANCHORKV_ERR_HIP, "hipGetSymbolAddress(scratch) returned no address");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return ANCHORKV_OK;
}

extern "C" anchorkv_status anchorkv_decode_step_noalloc(const anchorkv_plan* p, void* cache, size_t cache_bytes,
                                                        int32_t n_appended, const void* k_new, const void* v_new,
                                                        size_t new_bytes, const void* q, size_t q_bytes, void* out,
                                                        size_t out_bytes, int32_t out_dtype, float softmax_scale,
                                                        void* stream) {
  if (!p || !cache || !k_new || !v_new || !q || !out) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  if (n_appended < 0) return fail(ANCHORKV_ERR_INVALID_ARG, "n_appended must be >= 0");
  if (n_appended >= p->cfg.max_append) return fail(ANCHORKV_ERR_CAPACITY, "append capacity exhausted");
  if (out_dtype != ANCHORKV_F32 && out_dtype != ANCHORKV_BF16) return fail(ANCHORKV_ERR_INVALID_ARG, "bad out_dtype");
  anchorkv_status s;
  if ((s = need_bytes(cache_bytes, p->cache_bytes, "cache")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(new_bytes, new_need(p), "k_new / v_new")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(q_bytes, q_need(p), "q")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(out_bytes, out_need(p, out_dtype), "out")) != ANCHORKV_OK) return s;
  if ((s = need_bytes(ANCHORKV_NOALLOC_SCRATCH_BYTES, p->dws_bytes, "static decode scratch")) != ANCHORKV_OK)
    return s;
  void* ws = nullptr;
  if ((s = scratch_address(&ws)) != ANCHORKV_OK) return s;
  const float scale = softmax_scale > 0.0f ? softmax_scale : 1.0f / sqrtf((float)p->geo.D);
  const FaultScope fs;
  (void)hipGetLastError();
  return fs.finish(hip_status(akv::launch_decode(p->geo, cache_ptrs(p, cache), dws_ptrs(p, ws), q, k_new, v_new, out,
                                                 out_dtype, scale, n_appended, (hipStream_t)stream),
                              "decode step (no allocation)"));
}

extern "C" anchorkv_status anchorkv_reconstruct(const anchorkv_plan* p, const void* cache, size_t cache_bytes,
                                                int32_t n_appended, int32_t request, int32_t side, float* out,
                                                size_t out_bytes, void* stream) {
  if (!p || !cache || !out) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  if (request < 0 || request >= p->geo.B) return fail(ANCHORKV_ERR_INVALID_ARG, "request out of range");
  if (side != 0 && side != 1) return fail(ANCHORKV_ERR_INVALID_ARG, "side must be 0 (keys) or 1 (values)");
  if (n_appended < 0 || n_appended > p->cfg.max_append)
    return fail(ANCHORKV_ERR_INVALID_ARG, "n_appended must be in [0, max_append]");
  anchorkv_status s;
  if ((s = need_bytes(cache_bytes, p->cache_bytes, "cache")) != ANCHORKV_OK) return s;
  const size_t want = (size_t)p->geo.H * (p->geo.S[request] + n_appended) * p->geo.D * 4;
  if ((s = need_bytes(out_bytes, want, "out")) != ANCHORKV_OK) return s;
  const FaultScope fs;
  (void)hipGetLastError();
  return fs.finish(hip_status(
      akv::launch_reconstruct(p->geo, cache_ptrs(p, (void*)cache), request, side, n_appended, out, (hipStream_t)stream),
      "reconstruct"));
}

static float coef_host(const void* base, size_t i, int dtype) {
  if (dtype == ANCHORKV_BF16) return akv::bf2f(((const uint16_t*)base)[i]);
  return ((const float*)base)[i];
}

extern "C" anchorkv_status anchorkv_export(const anchorkv_plan* p, const void* cache_host, size_t cache_bytes,
                                           int32_t b, int32_t n_appended, anchorkv_export_arrays* o) {
  if (!p || !cache_host || !o) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  {
    const anchorkv_status s = need_bytes(cache_bytes, p->cache_bytes, "cache");
    if (s != ANCHORKV_OK) return s;
  }
  if (b < 0 || b >= p->geo.B) return fail(ANCHORKV_ERR_INVALID_ARG, "request out of range");
  if (n_appended < 0 || n_appended > p->cfg.max_append)
    return fail(ANCHORKV_ERR_INVALID_ARG, "n_appended must be in [0, max_append]");
  const akv::Cache c = cache_ptrs(p, (void*)cache_host);
  const Geo& g = p->geo;
  if (c.header[0] != kMagic || c.header[1] != kVersion || (int)c.header[3] != g.B || (int)c.header[4] != g.H ||
      (int)c.header[5] != g.D || (int)c.header[6] != g.dtype)
    return fail(ANCHORKV_ERR_CORRUPT_CACHE, "cache header does not match the plan");
  if (c.header[2] & 1u) return fail(ANCHORKV_ERR_CORRUPT_CACHE, "invalid anchor override");
  if (c.header[2] & 2u) return fail(ANCHORKV_ERR_CORRUPT_CACHE, "anchor selection count mismatch");
  const int H = g.H, S = g.S[b], k = g.k[b], D = g.D, G = g.G, nw = (S + 63) / 64;
  const size_t ko = (size_t)g.prefK[b] * H, wo = (size_t)g.prefW[b] * H;
  if (o->anchors) memcpy(o->anchors, c.anc_pos + ko, sizeof(int32_t) * H * k);
  for (int side = 0; side < 2; ++side) {
    int32_t* a_out = side ? o->a_v : o->a_k;
    float* g_out = side ? o->gamma_v : o->gamma_k;
    uint8_t* s_out = side ? o->sel_v : o->sel_k;
    uint8_t* c_out = side ? o->codes_v : o->codes_k;
    float* sc_out = side ? o->scales_v : o->scales_k;
    const uint16_t* idx = side ? c.idxV : c.idxK;
    const void* gm = side ? c.gV : c.gK;
    const uint64_t* mask = side ? c.maskV : c.maskK;
    const int32_t* pc = side ? c.pcV : c.pcK;
    const uint8_t* codes = side ? c.codesV : c.codesK;
    const float* scales = side ? c.scalesV : c.scalesK;
    const int ntot = side ? g.prefNV[g.B] : g.prefNK[g.B];
    if (c_out) memset(c_out, 0, (size_t)H * S * (D / 4));
    if (sc_out) memset(sc_out, 0, sizeof(float) * (size_t)H * S * (D / G));
    for (int h = 0; h < H; ++h)
      for (int i = 0; i < S; ++i) {
        const size_t e = akv::slot_base(g, b, h) + i;
        const int t = c.pos[e];
        if (t < 0 || t >= S) return fail(ANCHORKV_ERR_CORRUPT_CACHE, "position id out of range");
        const size_t te = (size_t)h * S + t;
        if (a_out) a_out[te] = idx[e];
        if (g_out) g_out[te] = coef_host(gm, e, g.dtype);
        const size_t wi = wo + (size_t)h * nw + (i >> 6);
        const uint64_t wm = mask[wi];
        const bool sel = (wm >> (i & 63)) & 1u;
        if (s_out) s_out[te] = sel;
        if (sel) {
          const int slot = pc[wi] + __builtin_popcountll(wm & ((1ull << (i & 63)) - 1ull));
          if (slot < 0 || slot >= ntot) return fail(ANCHORKV_ERR_CORRUPT_CACHE, "residual slot out of range");
          if (c_out) memcpy(c_out + te * (D / 4), codes + (size_t)slot * (D / 4), D / 4);
          if (sc_out) memcpy(sc_out + te * (D / G), scales + (size_t)slot * (D / G), sizeof(float) * (D / G));
        }
      }
    int32_t* ta = side ? o->tail_a_v : o->tail_a_k;
    float* tg = side ? o->tail_gamma_v : o->tail_gamma_k;
    const uint16_t* tidx = side ? c.tidxV : c.tidxK;
    const void* tgm = side ? c.tgV : c.tgK;
    for (int h = 0; h < H; ++h)
      for (int n = 0; n < n_appended; ++n) {
        const size_t ti = ((size_t)b * H + h) * g.max_append + n;
        // a dense tail stores the tokens themselves: no anchor, no coefficient
        if (ta) ta[(size_t)h * n_appended + n] = g.dense_tail ? -1 : tidx[ti];
        if (tg) tg[(size_t)h * n_appended + n] = g.dense_tail ? 0.0f : coef_host(tgm, ti, g.dtype);
      }
  }
  if (o->stats) {
    o->stats[0] = c.stats[b * 4 + 0];
    o->stats[1] = c.stats[b * 4 + 1];
    o->stats[2] = p->req[b].residuals_k;
    o->stats[3] = p->req[b].residuals_v;
    o->stats[4] = c.stats[b * 4 + 2];
    o->stats[5] = c.stats[b * 4 + 3];
  }
  return ANCHORKV_OK;
}

extern "C" const char* anchorkv_status_string(anchorkv_status s) {
  switch (s) {
    case ANCHORKV_OK: return "ok";
    case ANCHORKV_ERR_INVALID_ARG: return "invalid argument";
    case ANCHORKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case ANCHORKV_ERR_CAPACITY: return "append capacity exhausted";
    case ANCHORKV_ERR_CORRUPT_CACHE: return "corrupt cache";
    case ANCHORKV_ERR_HIP: return "HIP runtime error";
    case ANCHORKV_ERR_BUFFER_TOO_SMALL: return "buffer too small";
  }
  return "unknown status";
}

extern "C" const char* anchorkv_last_error(void) { return g_last_error.c_str(); }

// ------------------------------------------------------------------ kernel timing
namespace {
struct KernelEvents {
  std::string name;
  std::vector<hipEvent_t> ev;  // 2 per launch
  int used = 0;
};
struct Profiler {
  std::mutex mu;
  std::atomic<bool> on{false};
  std::vector<KernelEvents> k;
};
Profiler& profiler() {
  static Profiler p;
  return p;
}
void release_events(Profiler& p) {
  for (auto& ke : p.k)
    for (hipEvent_t e : ke.ev)
      if (e) (void)hipEventDestroy(e);
  p.k.clear();
}
}  // namespace

bool akv::prof_events(const char* kernel, hipEvent_t* start, hipEvent_t* stop) {
  Profiler& p = profiler();
  if (!p.on.load(std::memory_order_acquire)) return false;
  std::lock_guard<std::mutex> lk(p.mu);
  for (auto& ke : p.k) {
    if (ke.name != kernel || 2 * ke.used + 1 >= (int)ke.ev.size()) continue;
    *start = ke.ev[2 * ke.used];
    *stop = ke.ev[2 * ke.used + 1];
    ++ke.used;
    return true;
  }
  return false;
}

extern "C" anchorkv_status anchorkv_profile_enable(const char* kernels, int32_t max_launches) {
  if (!kernels || max_launches < 1) return fail(ANCHORKV_ERR_INVALID_ARG, "bad profile request");
  Profiler& p = profiler();
  std::lock_guard<std::mutex> lk(p.mu);
  p.on.store(false);
  release_events(p);
  std::string all(kernels);
  size_t pos = 0;
  while (pos <= all.size()) {
    size_t e = all.find(',', pos);
    if (e == std::string::npos) e = all.size();
    if (e > pos) {
      KernelEvents ke;
      ke.name = all.substr(pos, e - pos);
      ke.ev.assign(2 * (size_t)max_launches, nullptr);
      p.k.push_back(ke);
      for (auto& ev : p.k.back().ev) {
        if (hipEventCreate(&ev) != hipSuccess) {
          ev = nullptr;
          release_events(p);
          return fail(ANCHORKV_ERR_HIP, "hipEventCreate failed");
        }
      }
    }
    pos = e + 1;
  }
  if (p.k.empty()) return fail(ANCHORKV_ERR_INVALID_ARG, "no kernel named");
  p.on.store(true, std::memory_order_release);
  return ANCHORKV_OK;
}

extern "C" anchorkv_status anchorkv_profile_read(const char* kernel, float* total_ms, int32_t* launches) {
  if (!kernel || !total_ms || !launches) return fail(ANCHORKV_ERR_INVALID_ARG, "null argument");
  Profiler& p = profiler();
  std::lock_guard<std::mutex> lk(p.mu);
  for (auto& ke : p.k) {
    if (ke.name != kernel) continue;
    float tot = 0.0f;
    for (int i = 0; i < ke.used; ++i) {
      if (hipEventSynchronize(ke.ev[2 * i + 1]) != hipSuccess) return fail(ANCHORKV_ERR_HIP, "hipEventSynchronize failed");
      float ms = 0.0f;
      if (hipEventElapsedTime(&ms, ke.ev[2 * i], ke.ev[2 * i + 1]) != hipSuccess)
        return fail(ANCHORKV_ERR_HIP, "hipEventElapsedTime failed");
      tot += ms;
    }
    *total_ms = tot;
    *launches = ke.used;
    return ANCHORKV_OK;
  }
  return fail(ANCHORKV_ERR_INVALID_ARG, "kernel is not being profiled");
}

extern "C" anchorkv_status anchorkv_profile_disable(void) {
  Profiler& p = profiler();
  std::lock_guard<std::mutex> lk(p.mu);
  p.on.store(false);
  release_events(p);
  return ANCHORKV_OK;
}

// ------------------------------------------------------------------ init kernel
namespace akv {
__global__ void k_init(Geo g, Cache c, Ws w) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) {
    c.header[0] = kMagic;
    c.header[1] = kVersion;
    c.header[2] = 0;
    c.header[3] = (uint32_t)g.B;
    c.header[4] = (uint32_t)g.H;
    c.header[5] = (uint32_t)g.D;
    c.header[6] = (uint32_t)g.dtype;
  }
  if (i < 4 * g.B) c.stats[i] = 0;
  if (i < 2 * g.H * g.B) w.fixcount[i] = 0;
  if (i < akv::SS_N * g.H * g.B) w.sstate[i] = 0;
  if (i < 4096 * g.H * g.B) w.sghist[i] = 0u;
  const int nl = g.B * g.hdiv;
  if (i < 2 * 4096 * nl) w.bhist[i] = 0u;
  if (i < 2 * akv::BST_N * nl) w.bstate[i] = (i % akv::BST_N) == akv::BST_A ? 0x7F800000 : 0;
}
hipError_t launch_init(const Geo& g, const Cache& c, const Ws& w, hipStream_t st) {
  int n = 4 * g.B > 2 * g.H * g.B ? 4 * g.B : 2 * g.H * g.B;
  if (4096 * g.H * g.B > n) n = 4096 * g.H * g.B;
  if (2 * 4096 * g.B * g.hdiv > n) n = 2 * 4096 * g.B * g.hdiv;
  if (2 * akv::BST_N * g.B * g.hdiv > n) n = 2 * akv::BST_N * g.B * g.hdiv;
  launch("k_init", k_init, dim3((n + 255) / 256), dim3(256), 0, st, g, c, w);
  return hipGetLastError();
}
}  // namespace akv
