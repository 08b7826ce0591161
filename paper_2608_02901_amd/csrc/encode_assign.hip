// Nearest-anchor assignment (Sec. 3.1 Eq. nearest-anchor; Algorithm 1,
// second step), per request, KV head and side.
//
// k_assign: the dense tokens x anchors similarity contraction on MFMA, anchors
// on the M axis (staged through LDS, double buffered) and tokens on N (held in
// VGPRs for the whole anchor loop), so every lane's accumulators hold 16
// anchors of one token.  The epilogue keeps, per token, the best score
// s^_a = |x.a| / ||a|| with its index and the second best, without ever
// materializing the S x k score matrix.
//
// Certified argmax: the fp32 score differs from the exact |x.a|/||a|| by at
// most eps = (D 2^-23 + 2^-22) ||x|| (accumulation of D exact bf16 products,
// or rounded fp32 products, in any order, plus the inverse-norm and product
// roundings; inflated by 1 %).  When the best exceeds the second best by more
// than 2 eps (+ 2^-40 of the best, far above fp64 rounding), the winner is the
// exact argmax.  Otherwise the token goes to k_fixup, which rescans all anchors
// in fp32, and re-scores every anchor within the 2 eps band with the canonical
// fp64 formula (sequential fp64 dot d, c = d*d / ||a||^2, ties to the lowest
// index) -- the same formula as the CPU oracle, so the index is bit-exact.
#include "akv_common.h"

namespace akv {

// A score with its low 4 mantissa bits replaced by a tag is within 2^-19 of
// its value; the bound used is 2^-18 (inflated by 1 %).
__device__ inline float tag_score(float v, uint32_t tag) {
  return __uint_as_float((__float_as_uint(v) & ~15u) | tag);
}
__device__ inline float tag_eps(float b1) { return b1 * 3.8528442e-6f; }

// Token groups of 32 per wave and tokens per workgroup of k_assign.
constexpr int ASSIGN_NT = 2;
constexpr int ASSIGN_TOK = 4 * 32 * ASSIGN_NT;

__device__ inline float score_eps(float xnorm2, int D) {
  float xn = sqrtf(xnorm2) * (1.0f + 1e-5f);
  return xn * ((float)D * 1.1920929e-7f + 2.3841858e-7f) * 1.01f + 1e-30f;
}

template <int DT>
__global__ __launch_bounds__(256) void k_assign(Geo g, Ws w, Cache c, const void* Kin, const void* Vin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LDA = AKV_D + (DT ? 8 : 4);
  constexpr int NKS = AKV_D / M::KS;
  constexpr int PER = 16 / sizeof(E);
  constexpr int STAGE = 64;                                 // anchors per LDS stage
  constexpr int NLD = STAGE * AKV_D / PER / 256;            // 16-byte loads per thread per stage
  __shared__ __align__(16) E AS[2][STAGE * LDA];
  __shared__ float WS[2][STAGE];

  int idx = blockIdx.x;
  const int b = locate(g, ASSIGN_TOK, 2, idx);
  const int side = idx & 1;
  idx >>= 1;
  const int S = g.S[b], k = g.k[b], D = AKV_D;
  const int ntile = (S + ASSIGN_TOK - 1) / ASSIGN_TOK;
  const int h = idx / ntile, tile = idx % ntile;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)(side ? Vin : Kin) + xoff;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  const float* inv = (side ? c.invV : c.invK) + ko;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  // Token fragments (B operand) of the wave's ASSIGN_NT groups of 32 tokens,
  // and the tokens' squared norms.
  typename M::frag xf[ASSIGN_NT][NKS];
  float ss[ASSIGN_NT];
#pragma unroll
  for (int n = 0; n < ASSIGN_NT; ++n) {
    const int t = tile * ASSIGN_TOK + (wave * ASSIGN_NT + n) * 32 + (lane & 31);
    const int tc = min(t, S - 1);
    ss[n] = 0.0f;
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      xf[n][s] = M::load(X + (size_t)tc * D, kofs(M::KS, s, lane));
      if constexpr (DT == 1) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float v = (float)xf[n][s][i];
          ss[n] = fmaf(v, v, ss[n]);
        }
      } else {
        ss[n] = fmaf(xf[n][s], xf[n][s], ss[n]);
      }
    }
    ss[n] += __shfl_xor(ss[n], 32, 64);
  }

  const int nstage = (k + STAGE - 1) / STAGE;
  uint4 pre[NLD];
  float prew = 0.0f;
  auto fetch = [&](int st) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      int ch = threadIdx.x + 256 * i;
      int r = ch / (AKV_D / PER), col = (ch % (AKV_D / PER)) * PER;
      int a = st * STAGE + r;
      // rows past k repeat row k - 1; their inverse norm is 0, so they score 0
      const uint4* src = (const uint4*)(A + (size_t)min(a, k - 1) * D + col);
      pre[i] = make_uint4(src->x, src->y, src->z, src->w);
    }
    if (threadIdx.x < STAGE) {
      int a = st * STAGE + threadIdx.x;
      prew = a < k ? inv[a] : 0.0f;
    }
  };
  auto commit = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      int ch = threadIdx.x + 256 * i;
      int r = ch / (AKV_D / PER), col = (ch % (AKV_D / PER)) * PER;
      *(uint4*)(&AS[buf][r * LDA + col]) = pre[i];
    }
    if (threadIdx.x < STAGE) WS[buf][threadIdx.x] = prew;
  };

  // Scores carry their accumulator slot e (15 - e: within a lane the row
  // grows with e, so equal scores favour the lower row) in the low 4
  // mantissa bits; the tile of the best score is tracked per tile.  The tag
  // moves a score by less than 2^-18 of its value, which the certification
  // bound includes.  Every anchor fragment read from LDS feeds the MFMAs of
  // all ASSIGN_NT token groups, and the scores of a tile are processed while
  // the MFMAs of the next tile run (two accumulator sets, P and Q).
  float b1[ASSIGN_NT], b2[ASSIGN_NT];
  int tb1[ASSIGN_NT];
#pragma unroll
  for (int n = 0; n < ASSIGN_NT; ++n) {
    b1[n] = b2[n] = -1.0f;
    tb1[n] = 0;
  }
  auto mma_tile = [&](f32x16 (&acc)[ASSIGN_NT], int buf, int blk) {
#pragma unroll
    for (int n = 0; n < ASSIGN_NT; ++n) acc[n] = f32x16{};
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      auto af = M::load_lds(&AS[buf][(blk * 32 + (lane & 31)) * LDA], kofs(M::KS, s, lane));
#pragma unroll
      for (int n = 0; n < ASSIGN_NT; ++n) acc[n] = M::mma(af, xf[n][s], acc[n]);
    }
  };
  auto load_ws = [&](float (&wsr)[16], int buf, int blk) {
#pragma unroll
    for (int e = 0; e < 16; ++e) wsr[e] = WS[buf][blk * 32 + crow(e, lane)];
  };
  // Two scores at a time: the runner-up of {b1, b2, v0, v1} (b1 >= b2) is
  // max(b2, med3(b1, v0, v1)) and the best is max3(b1, v0, v1), three VALU
  // operations per pair instead of four.
  auto scores = [&](const f32x16 (&acc)[ASSIGN_NT], const float (&wsr)[16], int abase) {
#pragma unroll
    for (int n = 0; n < ASSIGN_NT; ++n) {
      const float b1o = b1[n];
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float v0 = tag_score(fabsf(acc[n][e]) * wsr[e], 15u - (uint32_t)e);
        const float v1 = tag_score(fabsf(acc[n][e + 1]) * wsr[e + 1], 14u - (uint32_t)e);
        b2[n] = fmaxf(b2[n], __builtin_amdgcn_fmed3f(b1[n], v0, v1));
        b1[n] = fmaxf(fmaxf(b1[n], v0), v1);
      }
      tb1[n] = b1[n] != b1o ? abase >> 5 : tb1[n];
    }
  };
  // Before the first tile, P holds a tile of zero scores, so that every
  // stage has the same branch-free schedule; it only matters for a token
  // whose every score is 0, which the certification sends to the fixup.
  f32x16 accP[ASSIGN_NT], accQ[ASSIGN_NT];
  float wsP[16], wsQ[16];
#pragma unroll
  for (int n = 0; n < ASSIGN_NT; ++n) accP[n] = f32x16{};
#pragma unroll
  for (int e = 0; e < 16; ++e) wsP[e] = 0.0f;
  int pend = 0;         // anchor base of the tile whose scores are pending
  bool pendQ = false;   // pending tile sits in Q (a last stage with one tile)
  fetch(0);
  commit(0);
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    const int cur = st & 1;
    if (st + 1 < nstage) fetch(st + 1);
    const int a0 = st * STAGE, a1 = a0 + 32;
    // tile 0 of the stage into Q; the pending tile (P) is scored meanwhile
    mma_tile(accQ, cur, 0);
    scores(accP, wsP, pend);
    load_ws(wsQ, cur, 0);
    pend = a0;
    pendQ = true;
    if (a1 < k) {
      mma_tile(accP, cur, 1);
      scores(accQ, wsQ, a0);
      load_ws(wsP, cur, 1);
      pend = a1;
      pendQ = false;
    }
    if (st + 1 < nstage) commit(cur ^ 1);
    __syncthreads();
  }
  if (pendQ) scores(accQ, wsQ, pend);
  else scores(accP, wsP, pend);
#pragma unroll
  for (int n = 0; n < ASSIGN_NT; ++n) {
    const int t = tile * ASSIGN_TOK + (wave * ASSIGN_NT + n) * 32 + (lane & 31);
    int i1 = tb1[n] * 32 + crow(15 - (int)(__float_as_uint(b1[n]) & 15u), lane);
    float B1 = b1[n], B2 = b2[n];
    // Merge the two lanes holding the same token (rows 0-3 / 4-7 of each 8).
    {
      const float ob1 = __shfl_xor(B1, 32, 64), ob2 = __shfl_xor(B2, 32, 64);
      const int oi1 = __shfl_xor(i1, 32, 64);
      const float top2 = fmaxf(fmaxf(B2, ob2), fminf(B1, ob1));
      if (ob1 > B1 || (ob1 == B1 && oi1 < i1)) i1 = oi1;
      B1 = fmaxf(B1, ob1);
      B2 = top2;
    }
    if (lane < 32 && t < S) {
      const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S + t;
      int32_t* apos = w.apos + (size_t)side * g.H * g.prefS[g.B] + po;
      w.xn2[(size_t)side * g.H * g.prefS[g.B] + po] = ss[n];  // the token's squared norm (fp32 sum)
      const int rk = w.rank[po];
      if (rk >= 0) {
        *apos = rk;
      } else {
        const float eps = score_eps(ss[n], D) + tag_eps(B1);
        if (B1 - B2 > 2.0f * eps + B1 * 9.094947e-13f && i1 < k) {
          *apos = i1;
        } else {
          *apos = -1;
          const int grp = (side * g.B + b) * g.H + h;
          const int slot = atomicAdd(&w.fixcount[grp], 1);  // < S: a token is listed once
          const size_t lo = (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H + (size_t)h * S;
          w.fixt[lo + slot] = t;
          w.fixb[lo + slot] = B1;
          atomicAdd(&c.stats[b * 4 + side], 1);
        }
      }
    }
  }
}

// Exact resolution of the tokens whose fp32 margin did not certify the argmax.
//
// The fixup lists are kept per (side, request, head), so a task of 32 listed
// tokens shares one anchor set.  One workgroup per task recomputes the
// tokens' scores against every anchor of the head with the same MFMA
// contraction as k_assign (its four waves take interleaved 32-anchor tiles,
// read straight from memory with a two-tile prefetch).  With b1 the best fp32
// score found for the token and eps its error bound, the exact argmax has an
// fp32 score of at least b1 - 2 eps: its exact score is >= the exact score of
// b1's anchor, which is >= b1 - eps, and the fp32 score is within eps of the
// exact one.  Every anchor in that band is re-scored with the canonical fp64
// formula (sequential fp64 dot d, c = d*d / ||a||^2, -1 for a zero anchor;
// largest c, then lowest index).  A token with more than FIX_SLOTS band
// members (a zero vector, many equal anchors) is resolved by a full scan.
// The number of tasks is read on the device; the grid strides over them and
// every workgroup exits once they are done.
constexpr int FIX_SLOTS = 8;

__device__ inline int wave_incl_scan_i(int v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

constexpr int FIX_NW = 8;  // waves per k_fixup workgroup (interleaved anchor tiles)

template <int DT>
__global__ __launch_bounds__(64 * FIX_NW) void k_fixup(Geo g, Ws w, Cache c, const void* Kin, const void* Vin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int NKS = AKV_D / M::KS;
  constexpr int PER = 16 / sizeof(E);
  __shared__ int ccnt[32];
  __shared__ int cidx[32][FIX_SLOTS];
  __shared__ double cval[32][FIX_SLOTS];
  __shared__ int task[3];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int D = AKV_D;
  const int ngrp = 2 * g.B * g.H;

  // Total number of 32-token tasks (every wave computes it; the loop bound is uniform).
  int ntask = 0;
  for (int g0 = 0; g0 < ngrp; g0 += 64) {
    const int gi = g0 + lane;
    ntask += wave_sum_i(gi < ngrp ? (w.fixcount[gi] + 31) >> 5 : 0);
  }

  for (int q = blockIdx.x; q < ntask; q += gridDim.x) {
    if (wave == 0) {
      // The task's group: the first group whose inclusive task prefix exceeds q.
      int grp = 0, first = 0, base = 0;
      for (int g0 = 0; g0 < ngrp; g0 += 64) {
        const int gi = g0 + lane;
        const int v = gi < ngrp ? (w.fixcount[gi] + 31) >> 5 : 0;
        const int incl = wave_incl_scan_i(v, lane);
        const unsigned long long hit = __ballot(base + incl > q);
        if (hit) {
          const int L = __ffsll((long long)hit) - 1;
          grp = g0 + L;
          first = base + __shfl(incl - v, L, 64);
          break;
        }
        base += __shfl(incl, 63, 64);
      }
      if (lane == 0) {
        task[0] = grp;
        task[1] = q - first;
      }
      if (lane < 32) ccnt[lane] = 0;
    }
    __syncthreads();
    const int grp = task[0], chunk = task[1];
    const int h = grp % g.H, b = (grp / g.H) % g.B, side = grp / (g.H * g.B);
    const int S = g.S[b], k = g.k[b];
    const size_t lo = (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H + (size_t)h * S;
    const int r0 = chunk * 32, nr = min(32, w.fixcount[grp] - r0);
    const int n = lane & 31, nn = min(n, nr - 1);
    const int t = w.fixt[lo + r0 + nn];
    const float b1 = w.fixb[lo + r0 + nn];
    const E* X = (const E*)(side ? Vin : Kin) + ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
    const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
    const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
    const float* inv = (side ? c.invV : c.invK) + ko;
    const double* nrm = (side ? c.nrmV : c.nrmK) + ko;
    int32_t* apos = w.apos + lo;

    typename M::frag xf[NKS];
    float ss = 0.0f;
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      xf[s] = M::load(X + (size_t)t * D, kofs(M::KS, s, lane));
      if constexpr (DT == 1) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float v = (float)xf[s][i];
          ss = fmaf(v, v, ss);
        }
      } else {
        ss = fmaf(xf[s], xf[s], ss);
      }
    }
    ss += __shfl_xor(ss, 32, 64);
    const float eps = score_eps(ss, D) + tag_eps(b1);
    const float bnd = b1 - 2.0f * eps - b1 * 9.094947e-13f;

    // Band collection: wave w takes anchor tiles w, w + FIX_NW, ... (rows of
    // the tile on M, tokens on N), prefetching two tiles ahead together with
    // the inverse norms of the lane's 16 rows (rows past k read 0: score 0).
    typename M::frag f0[NKS], f1[NKS];
    float i0[16], i1[16];
    auto fetch = [&](typename M::frag (&f)[NKS], float (&iv)[16], int a0) {
      const E* arow = A + (size_t)min(a0 + (lane & 31), k - 1) * D;
#pragma unroll
      for (int s = 0; s < NKS; ++s) f[s] = M::load(arow, kofs(M::KS, s, lane));
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = a0 + crow(e, lane);
        iv[e] = inv[min(r, k - 1)] * (r < k ? 1.0f : 0.0f);
      }
    };
    auto tile = [&](const typename M::frag (&f)[NKS], const float (&iv)[16], int a0) {
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) acc = M::mma(f[s], xf[s], acc);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = a0 + crow(e, lane);
        if (r < k && n < nr && fabsf(acc[e]) * iv[e] >= bnd) {
          const int j = atomicAdd(&ccnt[n], 1);
          if (j < FIX_SLOTS) cidx[n][j] = r;
        }
      }
    };
    constexpr int TS = 32 * FIX_NW;  // anchors between a wave's consecutive tiles
    int a0 = wave * 32;
    if (a0 < k) fetch(f0, i0, a0);
    if (a0 + TS < k) fetch(f1, i1, a0 + TS);
    for (; a0 < k; a0 += 2 * TS) {
      tile(f0, i0, a0);
      if (a0 + 2 * TS < k) fetch(f0, i0, a0 + 2 * TS);
      if (a0 + TS >= k) break;
      tile(f1, i1, a0 + TS);
      if (a0 + 3 * TS < k) fetch(f1, i1, a0 + 3 * TS);
    }
    __syncthreads();

    // Canonical fp64 scores of the band members (one thread per member).
    {
      const int pn = threadIdx.x / FIX_SLOTS, pj = threadIdx.x % FIX_SLOTS;
      const int cn = pn < nr ? ccnt[pn] : 0;
      if (pn < nr && cn <= FIX_SLOTS && pj < cn) {
        const int a = cidx[pn][pj];
        const int tp = w.fixt[lo + r0 + pn];
        const double d = dot64_seq<DT>(X + (size_t)tp * D, A + (size_t)a * D, D);
        cval[pn][pj] = nrm[a] > 0.0 ? (d * d) / nrm[a] : -1.0;
      }
    }
    __syncthreads();
    if (wave == 0) {
      if (lane < nr) {
        const int cn = ccnt[lane];
        if (cn <= FIX_SLOTS) {
          double bc = -INFINITY;
          int bi = 0x7fffffff;
          for (int j = 0; j < cn; ++j) {
            const double cc = cval[lane][j];
            const int a = cidx[lane][j];
            if (cc > bc || (cc == bc && a < bi)) { bc = cc; bi = a; }
          }
          apos[t] = bi;
        }
      }
      // Tokens with an overflowing band: full scan by the wave.
      unsigned long long big = __ballot(lane < nr && ccnt[lane] > FIX_SLOTS);
      while (big) {
        const int L = __ffsll((long long)big) - 1;
        big &= big - 1;
        const int tp = __shfl(t, L, 64);
        const float bl = __shfl(bnd, L, 64);
        const E* x = X + (size_t)tp * D;
        double bc = -INFINITY;
        int bi = 0x7fffffff;
        for (int a = lane; a < k; a += 64) {
          const uint4* row = (const uint4*)(A + (size_t)a * D);
          const uint4* xr = (const uint4*)x;
          float s = 0.0f;
          for (int i = 0; i < AKV_D / PER; ++i) {
            const uint4 av = row[i], xv = xr[i];
            const E* ea = (const E*)&av;
            const E* ex = (const E*)&xv;
#pragma unroll
            for (int j = 0; j < PER; ++j) s = fmaf(Elem<DT>::get(ex, j), Elem<DT>::get(ea, j), s);
          }
          if (fabsf(s) * inv[a] < bl) continue;
          const double d = dot64_seq<DT>(x, A + (size_t)a * D, D);
          const double cc = nrm[a] > 0.0 ? (d * d) / nrm[a] : -1.0;
          if (cc > bc || (cc == bc && a < bi)) { bc = cc; bi = a; }
        }
        for (int o = 32; o > 0; o >>= 1) {
          const double oc = __shfl_xor(bc, o, 64);
          const int oi = __shfl_xor(bi, o, 64);
          if (oc > bc || (oc == bc && oi < bi)) { bc = oc; bi = oi; }
        }
        if (lane == 0) apos[tp] = bi;
      }
    }
    __syncthreads();
  }
}

hipError_t launch_assign(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * ((g.S[b] + ASSIGN_TOK - 1) / ASSIGN_TOK) * 2;
  if (g.dtype == 1) {
    launch("k_assign", k_assign<1>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V);
    launch("k_fixup", k_fixup<1>, dim3(512), dim3(64 * FIX_NW), 0, st, g, w, c, K, V);
  } else {
    launch("k_assign", k_assign<0>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V);
    launch("k_fixup", k_fixup<0>, dim3(512), dim3(64 * FIX_NW), 0, st, g, w, c, K, V);
  }
  return hipGetLastError();
}

}  // namespace akv
