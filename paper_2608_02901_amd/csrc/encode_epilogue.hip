// Per-token epilogue of the compression: projection coefficient and
// residual (Sec. 3.1 Eq. projection) and the attention-output-aware
// utilities (Sec. 3.3 Eq. utilities, App. A.3), for EPI_TOK tokens of one
// (request, head) per workgroup.
//
// Coefficient (bit-exact with the CPU oracle): d = sequential fp64 dot of the
// token and its anchor, gamma = d / ||a||^2 in fp64, rounded to fp32 and, for
// a bf16 cache, to bf16 (round to nearest even).  Anchor positions keep
// gamma = 1.  An estimate of d with a proven error bound (an fp32 sum of the
// exact bf16 products for a bf16 cache, an fp64 sum of the exact fp32
// products for an fp32 cache, in a lane tree) decides the rounded value when
// its whole error interval rounds alike (nearly always); otherwise the
// sequential fp64 sum is formed.
//
// Utilities (fp32):
//   uK_t = (1/m) sum_w alpha_wt^2 (q_w . R_t rK_t)^2 / D * ||v_t - y_w||^2
//   uV_t = (1/m) sum_w alpha_wt^2 ||rV_t||^2
// with ||v_t - y_w||^2 = ||v_t||^2 - 2 v_t . y_w + ||y_w||^2 and the logits and
// v_t . y_w on MFMA; anchors get u = -1 and never compete.  Without positions
// (R_t = I) q_w . rK_t = q_w . k_t - gamma_t (q_w . abar_a(t)), the second term
// from the QA table.  With positions encoded (RP) the logits come from the
// rotated keys and q_w . R_t rK_t from a second contraction over the tile of
// rotated residuals R_t (k_t - fp32(gamma abar)), split into bf16 hi + lo parts
// for a bf16 cache.
//
// Schedule: first the 2 x EPI_TOK coefficient chains of the workgroup's
// tokens, 32 tokens per step, each chain's row split over a group of lanes
// (16-byte chunks, so that a wave's loads cover whole rows), then the
// utilities tile by tile (32 tokens), with the observation rows staged in LDS
// once, each wave's y fragments in registers and its rows' softmax constants
// in LDS for all tiles.  In both phases the next step's rows are loaded while
// the current one is processed; the loads are issued by every lane alike
// (rows past the workgroup's last token repeat that token's row), so that the
// waits for the current rows leave them in flight.
#include "akv_common.h"

namespace akv {

constexpr int EPI_TOK = 512;  // tokens per workgroup: 16 tiles of 32

// The canonical sequential fp64 dot of a token row and an anchor row, read
// from memory (fp64 fused multiply-add on the exact products, j = 0..D-1): the
// rare fallback of the certified coefficient, one 16-byte chunk per step so
// that it holds few registers in the caller.
template <int DT>
__device__ inline double dot64_rows(const typename Elem<DT>::T* x, const typename Elem<DT>::T* a) {
  constexpr int PER = 16 / sizeof(typename Elem<DT>::T);
  double s = 0.0;
#pragma unroll 1
  for (int j = 0; j < AKV_D; j += PER) {
    const uint4 xv = *(const uint4*)(x + j), av = *(const uint4*)(a + j);
#pragma unroll
    for (int e = 0; e < PER; ++e) s = fma((double)Elem<DT>::get(&xv, e), (double)Elem<DT>::get(&av, e), s);
  }
  return s;
}

// Lane exchange of a 64-bit value (two 32-bit moves).
template <int M>
__device__ inline double lane_xor_d(double v) {
  const unsigned long long u = __builtin_bit_cast(unsigned long long, v);
  const int lo = __builtin_bit_cast(int, lane_xor<M>(__builtin_bit_cast(float, (int)(unsigned)u)));
  const int hi = __builtin_bit_cast(int, lane_xor<M>(__builtin_bit_cast(float, (int)(unsigned)(u >> 32))));
  return __builtin_bit_cast(double, (unsigned long long)(unsigned)lo | ((unsigned long long)(unsigned)hi << 32));
}
template <int M>
__device__ inline float lane_xor_v(float v) { return lane_xor<M>(v); }
template <int M>
__device__ inline double lane_xor_v(double v) { return lane_xor_d<M>(v); }

// Reduce-scatter of NC chains over a group of G lanes (G a power of two,
// NC <= G): on entry v[c] is this lane's partial of chain c; on exit v[0]
// holds, in lane j of the group, the whole sum of chain rev(j mod NC) (the
// bit-reversed index).  At each level a lane keeps half of its chains and adds
// its partner's half; the remaining levels add whole sums.  Every addition
// pairs a lane's value with its partner's, and fp addition commutes, so all
// lanes that hold a chain hold the same bits; the summation tree has depth
// log2(G) above the lanes' own partial sums.
template <int M, int CNT, int NC, typename T>
__device__ inline void rs_level(T (&v)[NC], int lane) {
  const bool hi = lane & M;
#pragma unroll
  for (int q = 0; q < CNT / 2; ++q) {
    const T keep = hi ? v[q + CNT / 2] : v[q];
    const T send = hi ? v[q] : v[q + CNT / 2];
    v[q] = keep + lane_xor_v<M>(send);
  }
}
template <int G, int NC, typename T>
__device__ inline void group_reduce_scatter(T (&v)[NC], int lane) {
  static_assert(NC == 4 || NC == 8, "two or four rows per lane, two sides each");
  rs_level<1, NC>(v, lane);
  rs_level<2, NC / 2>(v, lane);
  if constexpr (NC == 8) rs_level<4, 2>(v, lane);
  if constexpr (NC < 8 && G > 4) v[0] += lane_xor_v<4>(v[0]);
  if constexpr (G > 8) v[0] += lane_xor_v<8>(v[0]);
  if constexpr (G > 16) v[0] += lane_xor_v<16>(v[0]);
}
template <int NC>
__device__ constexpr int chain_of(int j) {  // chain held by lane j after the reduce-scatter
  return NC == 4 ? (((j & 1) << 1) | ((j >> 1) & 1)) : (((j & 1) << 2) | (j & 2) | ((j >> 2) & 1));
}
// Chain C's value from the lane of this lane's NC-block that holds it.
template <int NC, int C>
__device__ inline float chain_bcast(float v, int lane) {
  constexpr int src = chain_of<NC>(C);  // the bit reversal is its own inverse
  if constexpr (NC == 4) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), src * 0x55, 0xF, 0xF, false));
  } else {
    return __shfl(v, (lane & ~(NC - 1)) | src, 64);
  }
}

template <int NC, int C = 0>
__device__ inline void chain_bcast_all(float (&gc)[NC], float v, int lane) {
  gc[C] = chain_bcast<NC, C>(v, lane);
  if constexpr (C + 1 < NC) chain_bcast_all<NC, C + 1>(gc, v, lane);
}

template <int DT, int R, bool RP>
__global__ __launch_bounds__(256, R == 1 ? 2 : 1) void k_epilogue(Geo g, Ws w, Cache c, const void* Kin,
                                                                  const void* Kobs, const void* Vin, const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = AKV_D + (DT ? 8 : 4);
  constexpr int PER = 16 / sizeof(E);
  constexpr int CPR = AKV_D / PER;          // 16-byte chunks per row
  constexpr int RPT = 32 * CPR / 256;       // chunks per thread of one 32-row tile
  constexpr int NKS = AKV_D / M::KS;
  constexpr int NT = EPI_TOK / 32;
  __shared__ __align__(16) E KT[32 * LD];
  __shared__ __align__(16) E VT[32 * LD];
  // rotated key residuals of the tile (RP): fp32, or bf16 hi and lo parts
  __shared__ __align__(16) E RTh[RP ? 32 * LD : 1];
  __shared__ __align__(16) E RTl[RP && DT == 1 ? 32 * LD : 1];
  constexpr int NC = 2 * RPT;  // coefficient chains per lane group: RPT rows x (K, V)
  // Per token and side: the anchor row to gather (0 for an invalid
  // assignment) and flags.
  constexpr int F_IDX = 0x0FFFFFFF, F_BAD = 1 << 28, F_PAST = 1 << 29, F_ANC = 1 << 30;
  __shared__ int fa_s[2][EPI_TOK];
  __shared__ float gK_s[EPI_TOK], gV_s[EPI_TOK], rv2_s[EPI_TOK], vn_s[EPI_TOK], rk2_s[EPI_TOK];
  // Row sums per token: each wave leaves its partials of a tile in tpart
  // (double-buffered by tile parity); 32 threads add the four waves' partials
  // in a fixed order into sumK (sum a2 vv qr^2), sumV (sum a2) and sumQ
  // (sum a2 qr^2) after the next tile's first barrier.
  __shared__ float tpart[2][3][4][32];
  __shared__ float sumK[EPI_TOK], sumV[EPI_TOK], sumQ[EPI_TOK];
  __shared__ __align__(16) float CVS[256], YVS[256];  // per observation row: softmax constant, ||y_w||^2
  __shared__ unsigned hmax[3];  // head maxima (float bits): ||q_w||, ||y_w||^2, |c_w|
  extern __shared__ __align__(16) char qlds_raw[];  // the m observation rows, row stride LD
  E* QS = (E*)qlds_raw;

  // Consecutive logical blocks (the chunks of one head) share an XCD, so the
  // head's anchor rows, gathered by every token's coefficient chain, stay in
  // that XCD's L2.
  int idx = blockIdx.x;
  {
    const int n8 = gridDim.x & ~7;
    if (idx < n8) idx = (idx & 7) * (n8 >> 3) + (idx >> 3);
  }
  const int b = locate(g, EPI_TOK, 1, idx);
  const int S = g.S[b], k = g.k[b], D = AKV_D, m = g.m;
  const int nchunk = (S + EPI_TOK - 1) / EPI_TOK;
  const int h = idx / nchunk, tb = (idx % nchunk) * EPI_TOK;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* Kx = (const E*)Kin + xoff;
  const E* Vx = (const E*)Vin + xoff;
  const E* Ko = (const E*)(RP ? Kobs : Kin) + xoff;  // keys of the logits
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;  // per-side stride of the position arrays
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D;
  // the observation rows into LDS (row stride LD), eight 16-byte loads in
  // flight per thread before any is stored
  for (int c0 = threadIdx.x; c0 < m * CPR; c0 += 8 * 256) {
    u32x4 qv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int ch = min(c0 + 256 * u, m * CPR - 1);
      qv[u] = *(const u32x4*)(Q + (size_t)(ch / CPR) * D + (ch % CPR) * PER);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int ch = c0 + 256 * u;
      if (ch < m * CPR) *(u32x4*)(&QS[(ch / CPR) * LD + (ch % CPR) * PER]) = qv[u];
    }
  }

  for (int tl = threadIdx.x; tl < EPI_TOK; tl += 256) {
    const int t = tb + tl;
    int fk = F_PAST, fv = F_PAST;
    if (t < S) {
      const int anc = w.rank[po + t] >= 0 ? F_ANC : 0;
      const int apk = w.apos[po + t], apv = w.apos[TS + po + t];
      fk = anc | ((apk < 0 || apk >= k) ? F_BAD : apk);
      fv = anc | ((apv < 0 || apv >= k) ? F_BAD : apv);
    }
    fa_s[0][tl] = fk;
    fa_s[1][tl] = fv;
  }
  __syncthreads();
  const int ntl = min(NT, (S - tb + 31) / 32);
  const int tlast = min(tb + EPI_TOK, S) - 1;  // the workgroup's last token

  // ---- coefficients, 32 tokens per step.  Lane gj of a CPR-lane group holds
  // elements PER gj .. PER gj + PER - 1 of rows tid / CPR + (256 / CPR) i of
  // the step (i < RPT) and of their anchors; chain c = 2 i + side is the dot
  // of row i's token and its anchor on that side, summed over the group by
  // the reduce-scatter.  Each lane certifies chain cc and the group shares
  // the coefficients.  The next step's rows are loaded while the current one
  // is processed.
  {
    const int gj = threadIdx.x % CPR;
    const int cc = chain_of<NC>(gj % NC);  // certified chain: row cc >> 1, side cc & 1
    struct Rows {
      u32x4 x[2][RPT], a[2][RPT];
      float x2;
      double n;
    };
    // Every lane issues the same loads (rows past the workgroup's last token
    // read that token's row; chains of tokens past S or of anchors are
    // discarded), so that the wait for one step's rows leaves the next step's
    // loads in flight.
    auto load = [&](Rows& q, int t0) {
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const int t = min(t0 + threadIdx.x / CPR + (256 / CPR) * i, tlast), col = gj * PER;
        const int fk = fa_s[0][t - tb], fv = fa_s[1][t - tb];
        q.x[0][i] = *(const u32x4*)(Kx + (size_t)t * D + col);
        q.x[1][i] = *(const u32x4*)(Vx + (size_t)t * D + col);
        q.a[0][i] = *(const u32x4*)((const E*)c.ancK + (ko + (fk & F_IDX)) * D + col);
        q.a[1][i] = *(const u32x4*)((const E*)c.ancV + (ko + (fv & F_IDX)) * D + col);
      }
      const int side = cc & 1, t = min(t0 + threadIdx.x / CPR + (256 / CPR) * (cc >> 1), tlast);
      q.x2 = w.xn2[side * TS + po + t];
      q.n = (side ? c.nrmV : c.nrmK)[ko + (fa_s[side][t - tb] & F_IDX)];
    };
    auto chains = [&](const Rows& q, int it) {
      using P = typename std::conditional<DT == 1, float, double>::type;
      float xs[NC][PER], as[NC][PER];
#pragma unroll
      for (int i = 0; i < RPT; ++i)
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          xs[2 * i][e] = chunk_elem<DT>(q.x[0][i], e);
          xs[2 * i + 1][e] = chunk_elem<DT>(q.x[1][i], e);
          as[2 * i][e] = chunk_elem<DT>(q.a[0][i], e);
          as[2 * i + 1][e] = chunk_elem<DT>(q.a[1][i], e);
        }
      P dp[NC];
#pragma unroll
      for (int j = 0; j < NC; ++j) {
        dp[j] = (P)0;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          if constexpr (DT == 1) dp[j] = fmaf(xs[j][e], as[j][e], dp[j]);
          else dp[j] = fma((double)xs[j][e], (double)as[j][e], dp[j]);
        }
      }
      group_reduce_scatter<CPR>(dp, lane);
      const int side = cc & 1, tl = 32 * it + threadIdx.x / CPR + (256 / CPR) * (cc >> 1), t = tb + tl;
      const int fa = fa_s[side][tl];
      const bool cand = !(fa & (F_PAST | F_ANC));
      float gb = 1.0f;
      if (cand) {
        // Certified coefficient.  The lanes' products are exact (bf16 in
        // fp32, fp32 in fp64) up to fp32 underflow (at most D 2^-126 in all);
        // the group sum has a summation tree of depth PER + log2(CPR) <= 12,
        // so its error is at most 12 u (1 + 12 u) sum|x_j a_j| (u = 2^-24 for
        // fp32, 2^-53 for fp64), and the canonical sequential fp64 sum lies
        // within 128 * 2^-53 (1 + 2^-46) sum|x_j a_j| of the exact dot.
        // sum|x_j a_j| <= sqrt(xx n), with xx the token's fp32 squared norm
        // (within 130 u of the exact one above fp32 underflow, which leaves at
        // most D 2^-126 < 2e-36) and n the anchor's fp64 one.  Eb below bounds
        // the distance of the canonical dot from the estimate; the stored
        // value round(fp32(fl64(d / n))) is monotone in d, so when both ends
        // of [est - Eb, est + Eb] give the same bits those are the canonical
        // bits; otherwise the sequential fp64 chain decides.
        const double n = q.n, est = (double)dp[0];
        bool done = false;
        if (n > 0.0 && __builtin_isfinite(est)) {
          const double rxn = sqrt(((double)q.x2 + 2e-36) * n);
          const double Eb = DT == 1 ? 2.1482e-6 * rxn + 3e-36 : 1.6e-14 * rxn;
          const float lo = Elem<DT>::round_coef((float)((est - Eb) / n));
          const float hi = Elem<DT>::round_coef((float)((est + Eb) / n));
          if (__float_as_uint(lo) == __float_as_uint(hi)) {
            gb = lo;
            done = true;
          }
        } else if (!(n > 0.0)) {
          gb = 0.0f;  // canonical gamma of a zero anchor
          done = true;
        }
        if (!done) {
          const E* xrow = (side ? Vx : Kx) + (size_t)t * D;
          const E* arow = (const E*)(side ? c.ancV : c.ancK) + (ko + (fa & F_IDX)) * D;
          const double d = dot64_rows<DT>(xrow, arow);
          gb = Elem<DT>::round_coef((float)(n > 0.0 ? d / n : 0.0));
        }
      }
      float gc[NC];
      chain_bcast_all(gc, gb, lane);
      // ||r||^2 of each chain's fp32 residual (the key side bounds q.r_K,
      // the value side is the value utility's factor)
      float rs[NC];
#pragma unroll
      for (int j = 0; j < NC; ++j) {
        rs[j] = 0.0f;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const float r = fmaf(-gc[j], as[j][e], xs[j][e]);
          rs[j] = fmaf(r, r, rs[j]);
        }
      }
      group_reduce_scatter<CPR>(rs, lane);
      if (gj < NC) {  // one lane per chain
        const bool in = t < S;
        if (in) w.gpos[side * TS + po + t] = gb;
        if (cand && (fa & F_BAD)) atomicOr(&c.header[2], 4u);
        const float rsv = cand ? rs[0] : 0.0f;
        if (side == 0) {
          gK_s[tl] = in ? gb : 0.0f;
          rk2_s[tl] = rsv;
        } else {
          gV_s[tl] = in ? gb : 0.0f;
          rv2_s[tl] = rsv;
          vn_s[tl] = in ? q.x2 : 0.0f;
        }
      }
    };
    Rows q0, q1;
    load(q0, tb);
#pragma unroll 1
    for (int it = 0; it < ntl; it += 2) {
      load(q1, tb + 32 * (it + 1));
      chains(q0, it);
      load(q0, tb + 32 * (it + 2));
      if (it + 1 < ntl) chains(q1, it + 1);
    }
  }

  // ---- utilities.  Wave rows: row block rb = wave + 4 r; lane l supplies
  // row rb*32 + l%32 of the fragments and owns the accumulator rows
  // rb*32 + crow(e, l) of token column l%32.
  const int nrb = (m + 31) / 32;
  constexpr float LOG2E = 1.4426950408889634f;
  const float isl = LOG2E / sqrtf((float)D);  // logit scale in base 2
  const float* cw = w.cw + (size_t)(b * g.H + h) * m;
  const float* qn = w.qn + (size_t)(b * g.H + h) * m;
  const double* ynp = w.ynp + (size_t)(b * g.H + h) * m * 4;  // quarters of ||y_w||^2
  const float* QA = w.QA + ko * m;
  // alpha = exp(l / sqrt(D) - M_w) / Z_w is taken as exp2(l log2(e) / sqrt(D)
  // - c_w) with c_w = (M_w + ln Z_w) log2(e) from the fp64 row statistics;
  // rows past m get c_w = 1e30, hence alpha = 0.  c_w and ||y_w||^2 sit in
  // LDS, the y fragments in registers; the head maxima of ||q_w||, ||y_w||^2
  // and |c_w| feed the error bounds.
  if (threadIdx.x < 3) hmax[threadIdx.x] = 0u;
  __syncthreads();
  for (int wr = threadIdx.x; wr < nrb * 32; wr += 256) {
    // ||y_w||^2: the fp32 rounding of the fp64 sum of the four quarters
    const float yn = wr < m ? (float)((ynp[4 * wr] + ynp[4 * wr + 1]) + (ynp[4 * wr + 2] + ynp[4 * wr + 3])) : 0.0f;
    CVS[wr] = wr < m ? cw[wr] : 1e30f;
    YVS[wr] = yn;
    if (wr < m) {
      atomicMax(&hmax[0], __float_as_uint(qn[wr]));
      atomicMax(&hmax[1], __float_as_uint(yn));
      atomicMax(&hmax[2], __float_as_uint(fabsf(cw[wr])));
    }
  }
  typename M::frag yh[R][NKS], yl[R][DT ? NKS : 1];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int rb = wave + 4 * r;
    const int arow = min(rb * 32 + (lane & 31), m - 1);
    const size_t yo = ((size_t)(b * g.H + h) * m + arow) * D;
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      const int k0 = kofs(M::KS, s, lane);
      if constexpr (DT == 1) {
        yh[r][s] = M::load(w.Yhi + yo, k0);
        yl[r][s] = M::load(w.Ylo + yo, k0);
      } else {
        yh[r][s] = w.Y[yo + k0];
      }
    }
  }
  // Next tile's keys and values, 16-byte chunks.  Every lane issues the same
  // loads (rows past the workgroup's last token read that token's row; their
  // columns are never used), so the waits of the current tile leave them in
  // flight.
  u32x4 kpre[RPT], vpre[RPT];
  auto fetch = [&](int t0) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int ch = threadIdx.x + 256 * i, r = min(t0 + ch / CPR, tlast), col = (ch % CPR) * PER;
      kpre[i] = *(const u32x4*)(Ko + (size_t)r * D + col);
      vpre[i] = *(const u32x4*)(Vx + (size_t)r * D + col);
    }
  };
  fetch(tb);
  auto fold = [&](int tt) {  // tile tt's partials into the per-token sums
    const int tl = 32 * tt + threadIdx.x;
    const float(*pp)[4][32] = tpart[tt & 1];
    sumK[tl] = (pp[0][0][threadIdx.x] + pp[0][1][threadIdx.x]) + (pp[0][2][threadIdx.x] + pp[0][3][threadIdx.x]);
    sumV[tl] = (pp[1][0][threadIdx.x] + pp[1][1][threadIdx.x]) + (pp[1][2][threadIdx.x] + pp[1][3][threadIdx.x]);
    sumQ[tl] = (pp[2][0][threadIdx.x] + pp[2][1][threadIdx.x]) + (pp[2][2][threadIdx.x] + pp[2][3][threadIdx.x]);
  };
  for (int it = 0; it < ntl; ++it) {
    const int t0 = tb + 32 * it;
    __syncthreads();  // previous tile's LDS reads are done (and, at it = 0, the coefficients are in LDS)
    if (it > 0 && threadIdx.x < 32) fold(it - 1);
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int ch = threadIdx.x + 256 * i, r = ch / CPR, col = (ch % CPR) * PER;
      *(u32x4*)(&KT[r * LD + col]) = kpre[i];
      *(u32x4*)(&VT[r * LD + col]) = vpre[i];
    }
    if constexpr (RP) {
      // Rotated key residuals: thread = (token tid / 8, pairs 8 (tid % 8) ..
      // +7).  r = x - fp32(gamma abar) (the residual the codec sees), then
      // (c r_f - s r_{f+64}, s r_f + c r_{f+64}) in fp32; zero for anchors and
      // rows past S.
      const int rr = threadIdx.x >> 3, f0 = 8 * (threadIdx.x & 7);
      const int tl = 32 * it + rr, t = t0 + rr;
      const int fk0 = fa_s[0][tl];
      const int ak = (fk0 & (F_PAST | F_ANC)) ? -1 : (fk0 & F_IDX);
      float xr[16], ar[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) xr[i] = ar[i] = 0.0f;
      float2 csv[8];
      if (ak >= 0) {
        const E* xrow = Kx + (size_t)t * D;
        const E* arow = (const E*)c.ancK + (ko + ak) * D;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int i = 0; i < 8; i += PER) {
            const uint4 xv4 = *(const uint4*)(xrow + f0 + 64 * hf + i);
            const uint4 av4 = *(const uint4*)(arow + f0 + 64 * hf + i);
#pragma unroll
            for (int e = 0; e < PER && i + e < 8; ++e) {
              xr[8 * hf + i + e] = Elem<DT>::get(&xv4, e);
              ar[8 * hf + i + e] = Elem<DT>::get(&av4, e);
            }
          }
#pragma unroll
        for (int i = 0; i < 8; i += 2) {
          const float4 cv = *(const float4*)&w.cs[(size_t)t * D + 2 * (f0 + i)];
          csv[i] = make_float2(cv.x, cv.y);
          csv[i + 1] = make_float2(cv.z, cv.w);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) csv[i] = make_float2(0.0f, 0.0f);
      }
      const float gk = gK_s[tl];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float r0 = xr[i] - gk * ar[i], r1 = xr[8 + i] - gk * ar[8 + i];
        const float o0 = fmaf(csv[i].x, r0, -(csv[i].y * r1));
        const float o1 = fmaf(csv[i].y, r0, csv[i].x * r1);
        if constexpr (DT == 1) {
          const uint16_t h0 = f2bf(o0), h1 = f2bf(o1);
          RTh[rr * LD + f0 + i] = h0;
          RTh[rr * LD + f0 + 64 + i] = h1;
          RTl[rr * LD + f0 + i] = f2bf(o0 - bf2f(h0));
          RTl[rr * LD + f0 + 64 + i] = f2bf(o1 - bf2f(h1));
        } else {
          RTh[rr * LD + f0 + i] = o0;
          RTh[rr * LD + f0 + 64 + i] = o1;
        }
      }
    }
    __syncthreads();
    const int tl = 32 * it + (lane & 31);
    const int fk0 = fa_s[0][tl];
    const int ak = (fk0 & (F_PAST | F_ANC)) ? -1 : (fk0 & F_IDX);  // -1: no utility
    const float gk = gK_s[tl], vn = vn_s[tl];
    // The token's QA row (rows of accumulator entries 4j .. 4j+3 are
    // consecutive) is read before the next tile's rows are requested, for
    // every token (anchor 0 stands in for an anchor position), so that its
    // wait leaves those in flight and its latency overlaps the MFMAs.
    const float* qa = QA + (size_t)max(ak, 0) * m;
    float qv[R][RP ? 1 : 16];
    if constexpr (!RP) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int rb = wave + 4 * r;
        if (rb >= nrb) break;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int w0 = rb * 32 + j * 8 + (lane >> 5) * 4;
          if ((m & 3) == 0) {
            const float4 q4 = *(const float4*)(qa + min(w0, m - 4));
            qv[r][4 * j] = q4.x; qv[r][4 * j + 1] = q4.y; qv[r][4 * j + 2] = q4.z; qv[r][4 * j + 3] = q4.w;
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) qv[r][4 * j + i] = qa[min(w0 + i, m - 1)];
          }
        }
      }
    }
    fetch(t0 + 32);
    float tk = 0.0f, tv = 0.0f, tq = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= nrb) break;
      f32x16 accL = {}, accY = {}, accR = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const int k0 = kofs(M::KS, s, lane);
        const auto kb = M::load_lds(&KT[(lane & 31) * LD], k0);
        const auto vb = M::load_lds(&VT[(lane & 31) * LD], k0);
        const auto qf = M::load_lds(&QS[(min(rb * 32 + (lane & 31), m - 1)) * LD], k0);
        accL = M::mma(qf, kb, accL);
        accY = M::mma(yh[r][s], vb, accY);
        if constexpr (DT == 1) accY = M::mma(yl[r][s], vb, accY);
        if constexpr (RP) {
          accR = M::mma(qf, M::load_lds(&RTh[(lane & 31) * LD], k0), accR);
          if constexpr (DT == 1) accR = M::mma(qf, M::load_lds(&RTl[(lane & 31) * LD], k0), accR);
        }
      }
      if (ak >= 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int w0 = rb * 32 + j * 8 + (lane >> 5) * 4;
          const float4 c4 = *(const float4*)&CVS[w0];
          const float4 y4 = *(const float4*)&YVS[w0];
          const float cq[4] = {c4.x, c4.y, c4.z, c4.w}, yq[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int e = 4 * j + i;
            const float l = accL[e];
            const float al = __builtin_amdgcn_exp2f(fmaf(l, isl, -cq[i]));
            const float a2 = al * al;
            float qr;
            if constexpr (RP) qr = accR[e];
            else qr = fmaf(-gk, qv[r][e], l);
            // ||v - y||^2 >= 0: the cancellation form can dip below zero
            // when y nearly equals v; the bounds below cover the clamp.
            const float vv = fmaxf(fmaf(-2.0f, accY[e], vn + yq[i]), 0.0f);
            const float q2 = qr * qr;
            tk = fmaf(a2 * vv, q2, tk);
            tq = fmaf(a2, q2, tq);
            tv += a2;
          }
        }
      }
    }
    tk += __shfl_xor(tk, 32, 64);
    tv += __shfl_xor(tv, 32, 64);
    tq += __shfl_xor(tq, 32, 64);
    if (lane < 32) {
      tpart[it & 1][0][wave][lane] = tk;
      tpart[it & 1][1][wave][lane] = tv;
      tpart[it & 1][2][wave][lane] = tq;
    }
  }
  __syncthreads();
  if (threadIdx.x < 32) fold(ntl - 1);
  __syncthreads();
  // ---- per token: the fp32 estimates and proven bounds [uL, uU] of the
  // canonical fp64 utilities (Sec. 3.3 Eq. utilities computed in fp64 from
  // the exact fp64 logits, y_w, M_w and Z_w).  With u = 2^-24:
  //   alpha: |ln(alpha32 / alpha)| <= eta = ln2 [c1 qmax |k| isl
  //          + u (3 qmax |k| isl + 2 cmax)] + 4u  (logit MFMA error c1 |q||k|:
  //          twice the error bound of a sequential fp32 sum of the 128
  //          products, which are exact for bf16 (c1 = 256u) and rounded for
  //          fp32 (c1 = 512u); the roundings of isl, the fma and c_w; exp2);
  //   q.r_K: |qr32 - qr| <= e = qmax (|k| + |gamma| |a|) (c1 + 4u) (logit and
  //          QA-table MFMA errors, the residual's rounding);
  //   vv   : |vv32 - ||v - y||^2| <= dvv = 258u |v|^2 + 4u ymax^2
  //          + 9.3e-5 |v| ymax (|v|^2 and ||y||^2 roundings, the bf16 hi/lo
  //          split of y and the MFMA error of v.y, the fp32 combination);
  // and with tk = sum a2 vv qr^2 (a2 = alpha32^2), tv = sum a2, S2 = sum a2
  // qr^2 (fp32 sums of non-negative terms, relative error <= 301u), S0 = sum
  // a2 vv <= V2 tv, S3 = sum a2 |qr| <= sqrt(S2 tv) and sum a2 vv |qr| <=
  // sqrt(tk S0) (Cauchy-Schwarz):
  //   m D uK <= (1+ea)^2 [tk + 2e sqrt(tk S0) + e^2 S0 + dvv (S2 + 2e S3 + e^2 tv)]
  //   m D uK >= (1-ea)^2 [tk - 2e sqrt(tk S0) - dvv S2]
  // (ea = eta (1 + eta)); the value side scales ||r_V||^2 tv / m likewise.
  {
    constexpr float U = 5.9604645e-8f;  // 2^-24
    constexpr float C1 = (DT == 1 ? 256.0f : 512.0f) * U;
    const float qmax = __uint_as_float(hmax[0]);
    const float ymax2 = __uint_as_float(hmax[1]) * (1.0f + 8.0f * U);
    const float ymax = sqrtf(ymax2) * (1.0f + 2.0f * U);
    const float cmax = __uint_as_float(hmax[2]);
    const float isl1 = LOG2E / sqrtf((float)D) * (1.0f + 4.0f * U);
    for (int tl = threadIdx.x; tl < EPI_TOK; tl += 256) {
      const int t = tb + tl;
      if (t >= S) continue;
      float uk = -1.0f, uv = -1.0f, ukl = -1.0f, uku = -1.0f, uvl = -1.0f, uvu = -1.0f;
      const int fk0 = fa_s[0][tl];
      const int ak = (fk0 & (F_PAST | F_ANC)) ? -1 : (fk0 & F_IDX);
      if (ak >= 0) {
        const float sk = sumK[tl], sv = sumV[tl], sq = sumQ[tl];
        uk = sk / ((float)m * (float)D);
        uv = rv2_s[tl] * sv / (float)m;
        // token quantities (upper bounds of the norms)
        // the logits' keys: the token, or its rotation rounded to the dtype
        // (|R_t k| = |k| up to the fp32 table, then one fp32 and one bf16 rounding)
        const float kn = sqrtf(w.xn2[po + t] * (1.0f + 300.0f * U)) * (1.0f + 2.0f * U) *
                         (RP ? (DT == 1 ? 1.0079f : 1.0001f) : 1.0f);
        const float vn2 = vn_s[tl] * (1.0f + 300.0f * U);
        const float vnm = sqrtf(vn2) * (1.0f + 2.0f * U);
        const float gk = fabsf(gK_s[tl]);
        const float an = (float)sqrt((c.nrmK)[ko + ak]) * (1.0f + 2.0f * U);
        const float rkn = sqrtf(rk2_s[tl] * (1.0f + 300.0f * U)) * (1.0f + 2.0f * U);
        const float qk = qmax * kn * isl1;
        const float eta = 0.6931472f * (C1 * qk + U * (3.0f * qk + 2.0f * cmax)) + 4.0f * U;
        const float ea = eta * (1.0f + eta) * 1.0001f;
        // |qr32 - q.R_t r| <= e.  Without positions: the logit and QA-table
        // MFMA errors and the residual's rounding.  With positions: the
        // rotation's two fp32 roundings per coordinate (2u |r|), the hi/lo
        // split (2^-18 |r|), the MFMA over the hi and lo chains (2 C1, or C1
        // for fp32) and, for an fp32 cache, the difference of the fused and
        // the canonical residual (2u |gamma| |a|).
        const float e = RP ? qmax * (rkn + (DT == 1 ? 0.0f : 2.1f * U * gk * an)) *
                                 (2.0002f * U + (DT == 1 ? 3.82e-6f + 2.0079f * C1 : C1) + 1e-15f) * 1.0001f
                           : qmax * (kn + gk * an) * (C1 + 4.0f * U) * 1.0001f;
        const float dvv = (258.0f * U * vn2 + 4.0f * U * ymax2 + 9.3e-5f * vnm * ymax) * 1.0001f;
        const float V2 = (vnm + ymax) * (vnm + ymax) * 1.0001f + dvv;
        const float qr1 = qmax * rkn + e;
        const float Qr2 = qr1 * qr1 * 1.0001f;
        const float r1 = 301.0f * U * 1.01f;
        const float tkh = sk * (1.0f + r1), tkl = sk * (1.0f - r1);
        const float tvh = sv * (1.0f + r1), tvl = sv * (1.0f - r1);
        const float S0 = V2 * tvh;
        const float cs = sqrtf(tkh * S0) * (1.0f + 2.0f * U);
        const float S2 = sq * (1.0f + r1);
        const float S3 = sqrtf(S2 * tvh) * (1.0f + 2.0f * U);
        const float hiK = tkh + 2.0f * e * cs + e * e * S0 + dvv * (S2 + 2.0f * e * S3 + e * e * tvh);
        const float loK = tkl - 2.0f * e * cs - dvv * S2;
        const float md = (float)m * (float)D;
        // fp32 underflow (flushed or subnormal intermediates) leaves at most
        // 2^-126 (Qr2 V2 + Qr2 + 1) per row term, m terms, / (m D)
        const float ufK = fmaxf(2.4e-38f, 2.4e-38f * (Qr2 * V2 + Qr2 + 1.0f) / (float)D);
        uku = (1.0f + ea) * (1.0f + ea) * hiK / md * (1.0f + 8.0f * U) + ufK;
        ukl = fmaxf(0.0f, (1.0f - ea) * (1.0f - ea) * loK / md * (1.0f - 8.0f * U) - ufK);
        // value side: ||r_V||^2 (fp32 sum of squares of the fp32 residual; for
        // an fp32 cache the residual's product rounding differs from the
        // canonical form by <= 2u |gamma| |a| per coordinate)
        const int fv = fa_s[1][tl];
        const float gv = fabsf(gV_s[tl]);
        const float anv = (fv & F_BAD) ? 0.0f : (float)sqrt((c.nrmV)[ko + (fv & F_IDX)]) * (1.0f + 2.0f * U);
        const float rv2 = rv2_s[tl];
        const float drv = 300.0f * U * rv2 + (DT == 1 ? 0.0f : 4.1f * U * sqrtf(rv2) * gv * anv * 1.01f);
        const float ufV = fmaxf(2.4e-38f, 2.4e-38f * (rv2 + drv + 1.0f));
        uvu = (1.0f + ea) * (1.0f + ea) * (rv2 + drv) * tvh / (float)m * (1.0f + 8.0f * U) + ufV;
        uvl = fmaxf(0.0f, (1.0f - ea) * (1.0f - ea) * (rv2 - drv) * tvl / (float)m * (1.0f - 8.0f * U) - ufV);
      }
      w.u[po + t] = uk;
      w.u[TS + po + t] = uv;
      w.uL[po + t] = ukl;
      w.uU[po + t] = uku;
      w.uL[TS + po + t] = uvl;
      w.uU[TS + po + t] = uvu;
    }
  }
}

template <int DT, int R, bool RP>
static hipError_t launch_epi_t(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs,
                               const void* V, const void* Q, int nblk, uint32_t qlds, hipStream_t st) {
  // With 256 observation rows the staged rows and the kernel's static arrays
  // pass 64 KiB; the kernel then asks for the larger LDS allocation gfx950
  // offers.
  if (qlds > 32768) {
    const hipError_t e =
        hipFuncSetAttribute((const void*)k_epilogue<DT, R, RP>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)qlds);
    if (e != hipSuccess) return e;
  }
  launch("k_epilogue", k_epilogue<DT, R, RP>, dim3(nblk), dim3(256), qlds, st, g, w, c, K, Kobs, V, Q);
  return hipGetLastError();
}

hipError_t launch_epilogue(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs, const void* V,
                           const void* Q, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * ((g.S[b] + EPI_TOK - 1) / EPI_TOK);
  const bool r2 = g.m > 128;  // 4 waves x 2 row blocks of 32 for up to 256 rows
  const uint32_t qlds = (uint32_t)g.m * (AKV_D + (g.dtype == 1 ? 8 : 4)) * (g.dtype == 1 ? 2 : 4);
  const bool rp = g.rope != 0;
  if (g.dtype == 1) {
    if (rp) return r2 ? launch_epi_t<1, 2, true>(g, w, c, K, Kobs, V, Q, nblk, qlds, st)
                      : launch_epi_t<1, 1, true>(g, w, c, K, Kobs, V, Q, nblk, qlds, st);
    return r2 ? launch_epi_t<1, 2, false>(g, w, c, K, Kobs, V, Q, nblk, qlds, st)
              : launch_epi_t<1, 1, false>(g, w, c, K, Kobs, V, Q, nblk, qlds, st);
  }
  if (rp) return r2 ? launch_epi_t<0, 2, true>(g, w, c, K, Kobs, V, Q, nblk, qlds, st)
                    : launch_epi_t<0, 1, true>(g, w, c, K, Kobs, V, Q, nblk, qlds, st);
  return r2 ? launch_epi_t<0, 2, false>(g, w, c, K, Kobs, V, Q, nblk, qlds, st)
            : launch_epi_t<0, 1, false>(g, w, c, K, Kobs, V, Q, nblk, qlds, st);
}

}  // namespace akv
