// Per-token epilogue of the compression: projection coefficient and
// residual (Sec. 3.1 Eq. projection) and the attention-output-aware
// utilities (Sec. 3.3 Eq. utilities, App. A.3), for EPI_TOK tokens of one
// (request, head) per workgroup.
//
// Coefficient (bit-exact with the CPU oracle): d = sequential fp64 dot of the
// token and its anchor, gamma = d / ||a||^2 in fp64, rounded to fp32 and, for
// a bf16 cache, to bf16 (round to nearest even).  Anchor positions keep
// gamma = 1.  For a bf16 cache an fp32 estimate of d with a proven error
// bound decides the rounded value when its whole error interval rounds alike
// (nearly always); otherwise the sequential fp64 sum is formed.
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
// tokens (four per thread, spread over all waves), then the utilities tile by
// tile (32 tokens), with the observation rows staged in LDS once, each wave's
// y fragments in registers and its rows' softmax constants in LDS for all
// tiles, and the next tile's keys and values loaded while the current tile is
// processed.
#include "akv_common.h"

namespace akv {

constexpr int EPI_TOK = 512;  // tokens per workgroup: 16 tiles of 32

// The canonical sequential fp64 dot of a token row and an anchor row, read
// from memory: the rare fallback of the certified coefficient, kept out of
// line so that it holds no registers in the caller.
template <int DT>
__device__ __attribute__((noinline)) double dot64_rows(const typename Elem<DT>::T* x, const typename Elem<DT>::T* a) {
  return dot64_seq<DT, true>(x, a, AKV_D);
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
  __shared__ float gK_s[EPI_TOK], rv2_s[EPI_TOK], vn_s[EPI_TOK], rk2_s[EPI_TOK];
  __shared__ int aK_s[EPI_TOK];
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
  for (int ch = threadIdx.x; ch < m * CPR; ch += 256) {
    const int r = ch / CPR, col = (ch % CPR) * PER;
    *(uint4*)(&QS[r * LD + col]) = *(const uint4*)(Q + (size_t)r * D + col);
  }

  // ---- coefficients: thread = token tb + tid + 256 p (p < EPI_TOK / 256),
  // both sides.  A token with
  // an invalid assignment raises the error bit and uses anchor 0; the
  // K side marks utility candidates (non-anchors), the V side also leaves
  // ||rV||^2 and ||v||^2 (the latter from the assignment pass).
  {
#pragma unroll 1
  for (int pp = 0; pp < EPI_TOK / 256; ++pp) {
    const int tl = threadIdx.x + 256 * pp, t = tb + tl;
    const bool in = t < S;
    const int tc = in ? t : S - 1;
    const int rk = w.rank[po + tc];
#pragma unroll 1
    for (int side = 0; side < 2; ++side) {
      const int ap = w.apos[side * TS + po + tc];
      const bool bad = ap < 0 || ap >= k;
      const int a = bad ? 0 : ap;
      const E* xrow = (side ? Vx : Kx) + (size_t)tc * D;
      const E* arow = (const E*)(side ? c.ancV : c.ancK) + (ko + a) * D;
      const double n = (side ? c.nrmV : c.nrmK)[ko + a];
      uint4 xv[CPR], av[CPR];
#pragma unroll
      for (int i = 0; i < CPR; ++i) {
        const uint4 x4 = *(const uint4*)(xrow + i * PER);
        const uint4 a4 = *(const uint4*)(arow + i * PER);
        xv[i] = make_uint4(x4.x, x4.y, x4.z, x4.w);
        av[i] = make_uint4(a4.x, a4.y, a4.z, a4.w);
      }
      const E* xe = (const E*)xv;
      const E* ae = (const E*)av;
      float gb = 1.0f;
      if (in && rk < 0) {
        if (bad) atomicOr(&c.header[2], 4u);
        bool done = false;
        if constexpr (DT == 1) {
          // Certified shortcut for a bf16 cache.  Four interleaved fp32 FMA
          // chains over the exact bf16 products give d32 with |d32 - d| <=
          // 35 u (1 + 35 u) sum|x_j a_j| <= 36 u sqrt(xx n) (u = 2^-24; 32
          // steps per chain and three combining adds; xx is the token's fp32
          // sum of squares, within 130 u of the exact one), and the
          // sequential fp64 sum lies within 2^-44 sqrt(xx n) of d.  The
          // stored value bf16(fp32(fl64(d / n))) is monotone in d, so when
          // both ends of the interval round to the same bits, those are the
          // canonical bits; otherwise the sequential fp64 chain decides.
          float e0 = 0.0f, e1 = 0.0f, e2 = 0.0f, e3 = 0.0f;
#pragma unroll
          for (int j = 0; j < AKV_D; j += 4) {
            e0 = fmaf(Elem<DT>::get(xe, j), Elem<DT>::get(ae, j), e0);
            e1 = fmaf(Elem<DT>::get(xe, j + 1), Elem<DT>::get(ae, j + 1), e1);
            e2 = fmaf(Elem<DT>::get(xe, j + 2), Elem<DT>::get(ae, j + 2), e2);
            e3 = fmaf(Elem<DT>::get(xe, j + 3), Elem<DT>::get(ae, j + 3), e3);
          }
          const float f32 = (e0 + e1) + (e2 + e3);
          const double d32 = (double)f32;
          if (n > 0.0 && __builtin_isfinite(f32)) {
            // + 128 * 2^-126 for products flushed to zero below the fp32
            // normal range
            const double E = 2.1482e-6 * sqrt((double)w.xn2[side * TS + po + tc] * n) + 3e-36;
            const float lo = Elem<DT>::round_coef((float)((d32 - E) / n));
            const float hi = Elem<DT>::round_coef((float)((d32 + E) / n));
            if (__float_as_uint(lo) == __float_as_uint(hi)) {
              gb = lo;
              done = true;
            }
          } else if (!(n > 0.0)) {
            gb = 0.0f;  // canonical gamma of a zero anchor
            done = true;
          }
        }
        if (!done) {
          const double d = DT == 1 ? dot64_rows<DT>(xrow, arow) : dot64_seq<DT, true>(xe, ae, D);
          const double g64 = n > 0.0 ? d / n : 0.0;
          gb = Elem<DT>::round_coef((float)g64);
        }
      }
      if (in) w.gpos[side * TS + po + t] = gb;
      // ||r||^2 of the side's fp32 residual (the key side bounds q.r_K, the
      // value side is the value utility's factor)
      float rs = 0.0f;
#pragma unroll
      for (int j = 0; j < AKV_D; ++j) {
        const float r = fmaf(-gb, Elem<DT>::get(ae, j), Elem<DT>::get(xe, j));
        rs = fmaf(r, r, rs);
      }
      rs = (in && rk < 0) ? rs : 0.0f;
      if (side == 0) {
        gK_s[tl] = in ? gb : 0.0f;
        aK_s[tl] = (in && rk < 0) ? a : -1;  // -1: no utility (anchor or past S)
        rk2_s[tl] = rs;
      } else {
        vn_s[tl] = w.xn2[TS + po + tc];
        rv2_s[tl] = rs;
      }
    }
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
  const float* yn = w.ynorm + (size_t)(b * g.H + h) * m;
  const float* QA = w.QA + ko * m;
  // alpha = exp(l / sqrt(D) - M_w) / Z_w is taken as exp2(l log2(e) / sqrt(D)
  // - c_w) with c_w = (M_w + ln Z_w) log2(e) from the fp64 row statistics;
  // rows past m get c_w = 1e30, hence alpha = 0.  c_w and ||y_w||^2 sit in
  // LDS, the y fragments in registers; the head maxima of ||q_w||, ||y_w||^2
  // and |c_w| feed the error bounds.
  if (threadIdx.x < 3) hmax[threadIdx.x] = 0u;
  __syncthreads();
  for (int wr = threadIdx.x; wr < nrb * 32; wr += 256) {
    CVS[wr] = wr < m ? cw[wr] : 1e30f;
    YVS[wr] = wr < m ? yn[wr] : 0.0f;
    if (wr < m) {
      atomicMax(&hmax[0], __float_as_uint(qn[wr]));
      atomicMax(&hmax[1], __float_as_uint(yn[wr]));
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
  // Next tile's keys and values, 16-byte chunks (rows past S are zero).
  uint4 kpre[RPT], vpre[RPT];
  auto fetch = [&](int t0) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int ch = threadIdx.x + 256 * i, r = ch / CPR, col = (ch % CPR) * PER;
      kpre[i] = make_uint4(0, 0, 0, 0);
      vpre[i] = make_uint4(0, 0, 0, 0);
      if (t0 + r < S) {
        kpre[i] = *(const uint4*)(Ko + (size_t)(t0 + r) * D + col);
        vpre[i] = *(const uint4*)(Vx + (size_t)(t0 + r) * D + col);
      }
    }
  };
  const int ntl = min(NT, (S - tb + 31) / 32);
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
      *(uint4*)(&KT[r * LD + col]) = kpre[i];
      *(uint4*)(&VT[r * LD + col]) = vpre[i];
    }
    if constexpr (RP) {
      // Rotated key residuals: thread = (token tid / 8, pairs 8 (tid % 8) ..
      // +7).  r = x - fp32(gamma abar) (the residual the codec sees), then
      // (c r_f - s r_{f+64}, s r_f + c r_{f+64}) in fp32; zero for anchors and
      // rows past S.
      const int rr = threadIdx.x >> 3, f0 = 8 * (threadIdx.x & 7);
      const int tl = 32 * it + rr, t = t0 + rr;
      const int ak = aK_s[tl];
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
    if (it + 1 < ntl) fetch(t0 + 32);
    const int tl = 32 * it + (lane & 31);
    const int ak = aK_s[tl];
    const float gk = gK_s[tl], vn = vn_s[tl];
    // The token's QA row (rows of accumulator entries 4j .. 4j+3 are
    // consecutive) is read before the contraction, for every token (anchor 0
    // stands in for an anchor position), so its latency overlaps the MFMAs.
    const float* qa = QA + (size_t)max(ak, 0) * m;
    float tk = 0.0f, tv = 0.0f, tq = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= nrb) break;
      float qv[RP ? 1 : 16];
      if constexpr (!RP) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int w0 = rb * 32 + j * 8 + (lane >> 5) * 4;
          if ((m & 3) == 0) {
            const float4 q4 = *(const float4*)(qa + min(w0, m - 4));
            qv[4 * j] = q4.x; qv[4 * j + 1] = q4.y; qv[4 * j + 2] = q4.z; qv[4 * j + 3] = q4.w;
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) qv[4 * j + i] = qa[min(w0 + i, m - 1)];
          }
        }
      }
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
            else qr = fmaf(-gk, qv[e], l);
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
      const int ak = aK_s[tl];
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
        const int av = w.apos[TS + po + t];
        const float gv = fabsf(w.gpos[TS + po + t]);
        const float anv = (av >= 0 && av < k) ? (float)sqrt((c.nrmV)[ko + av]) * (1.0f + 2.0f * U) : 0.0f;
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
