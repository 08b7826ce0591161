// Head-pooled residual budget (Sec. 3.4; Algorithm 1, "top N by utility
// pooled over heads").  Per request and side, the N_side candidates of highest
// utility among the non-anchor positions of all H heads get a residual; ties
// go to the lower head, then the lower position (the flattened (h, t) order).
// The utility ranked is the canonical fp64 one (Sec. 3.3 Eq. utilities in fp64
// from exact fp64 logits and the fp64 observation statistics).
//
// First the fp32 estimates u are cut by an exact radix select on their bit
// patterns (utilities are >= 0, so their bits order like the values; anchors
// carry -1 and are skipped):
//   k_bhist : per chunk of the flattened (h, t) range, histogram of the first
//             12-bit digit [31:20], added to the request's;
//   k_bcand : every workgroup finds the digit of the N-th largest from that
//             histogram; utilities inside its bin are appended (value and
//             flattened index) as candidates;
//   k_bcut  : one workgroup per request and side: the remaining digits [19:8]
//             and [7:0] among the candidates (or, when the list overflowed,
//             among all utilities: same digits, same result), the count still
//             to take at the threshold, and per chunk the number of
//             threshold ties in the earlier chunks;
//   k_bmark : marks: above the threshold taken, ties taken in flattened order
//             while the count lasts.
// N <= 0 takes nothing; N at least the number of candidates takes them all.
//
// Then the fp32 order is corrected to the fp64 one.  The epilogue gives every
// candidate proven bounds uL <= u64 <= uU.  With T the N-th largest fp32
// estimate, A = min{uL : u >= T} is at most the N-th largest fp64 utility X
// (the N candidates with u >= T all have u64 >= A) and B = max{uU : u <= T} is
// at least X (only the fewer than N candidates with u > T can exceed B).  So
// uL > B is surely selected, uU < A surely not (both agree with the fp32
// marks), and the band of the rest holds X and every candidate whose order
// matters:
//   k_bbound   : A and B per request and side;
//   k_bmark    : also lists the band and counts the band members the fp32
//                order selected (the selections the band must supply);
//   k_brescore : the fp64 utility of every band member, computed as the
//                oracle does (sequential fp64 dots, one wave per member);
//   k_brank    : each band member's rank in (fp64 utility descending,
//                flattened index ascending) order;
//   k_bsel     : re-marks the band: ranks below `need` are selected.
// A band above BAND_CAP keeps the fp32 marks and raises HDR_BAND_OVERFLOW.
//
// Ranking keys other than the utility (the residual-ranking ablations of
// Sec. 4.3) go through the same cut: k_rankkeys replaces u, uL, uU by the
// key's fp32 rounding and an interval that holds its exact fp64 value, and
// k_brescore computes the exact fp64 key of the band members.  With equal
// per-head budgets (the head-pooling ablation of Sec. 4.3) every (request,
// head, side) is a list of its own, ranked in position order.
#include "akv_common.h"

namespace akv {

constexpr int BCHUNK = 4096;
constexpr int BCMAX = 32768;  // first-digit candidates kept per list and side

// Budget list L: request L / hdiv; heads [h0, h0 + hp) of it, hp = H / hdiv
// (all heads with pooled budgets, one head with equal per-head budgets).
// Its elements are the flattened (h - h0, t) positions, n = hp * S of them,
// at offset `off` of a side's per-position arrays.
struct BList {
  int b, hp, h0, S, n, nch;
  size_t off;
};
__device__ inline BList blist(const Geo& g, int L) {
  BList q;
  q.b = L / g.hdiv;
  q.hp = g.H / g.hdiv;
  q.h0 = (L % g.hdiv) * q.hp;
  q.S = g.S[q.b];
  q.n = q.hp * q.S;
  q.nch = (q.n + BCHUNK - 1) / BCHUNK;
  q.off = (size_t)g.prefS[q.b] * g.H + (size_t)q.h0 * q.S;
  return q;
}
__device__ inline int nside(const Geo& g, const BList& q, int side) {
  const int b = q.b;
  return (side ? g.prefNV[b + 1] - g.prefNV[b] : g.prefNK[b + 1] - g.prefNK[b]) / g.hdiv;
}
// 0: radix select, 1: take every candidate, 2: take none.
__device__ inline int bmode(const Geo& g, const BList& q, int side) {
  const int N = nside(g, q, side);
  const int ncand = q.hp * (q.S - g.k[q.b]);
  return N <= 0 ? 2 : (N >= ncand ? 1 : 0);
}
// Threshold-tie counts of the list's chunks.
__device__ inline int32_t* btie(const Geo& g, const Ws& w, int L, const BList& q, int side) {
  return w.tiecnt + 2 * g.prefBC[q.b] + (2 * (L % g.hdiv) + side) * q.nch;
}

// Workgroup idx -> list (chunks of both sides of every list in turn).
__device__ inline int locate_l(const Geo& g, int& idx) {
  const int nl = g.B * g.hdiv;
  for (int L = 0; L < nl; ++L) {
    const int n = 2 * (((g.H / g.hdiv) * g.S[L / g.hdiv] + BCHUNK - 1) / BCHUNK);
    if (idx < n) return L;
    idx -= n;
  }
  return -1;
}

__device__ inline size_t bbase(const Geo& g, const BList& q, int side) {
  return (size_t)side * g.H * g.prefS[g.B] + q.off;
}

// ------------------------------------------------------------------ rank keys
// Exact fp64 keys of the ranking ablations, as the oracle defines them:
//   COSINE  : 1 - |d| / sqrt(xx nn) with d, xx, nn sequential fp64 dots of
//             the token and its anchor (1 when a norm is zero);
//   RESNORM : sequential fp64 sum of the squared fp32 residual
//             r = x - fp32(gamma a);
//   RANDOM  : 53 bits of splitmix64(seed ^ (side + 1) << 60 ^ h << 40 ^ t).
// Products of two fp32 (or bf16) values are exact in fp64, so a fused
// multiply-add accumulates exactly as a product followed by an add.
template <int DT>
__device__ double rank_key64(const Geo& g, int side, int h, int t, const typename Elem<DT>::T* x,
                             const typename Elem<DT>::T* a, float gm) {
  if (g.rank_mode == RANK_RANDOM) {
    const unsigned long long key =
        splitmix64(g.seed_rank ^ ((unsigned long long)(side + 1) << 60) ^ ((unsigned long long)h << 40) ^
                   (unsigned long long)t);
    return (double)(key >> 11) * 0x1p-53;
  }
  constexpr int PER = 16 / sizeof(typename Elem<DT>::T);
  double d = 0.0, xx = 0.0, nn = 0.0;
  for (int c = 0; c < AKV_D / PER; ++c) {
    const uint4 xv = ((const uint4*)x)[c], av = ((const uint4*)a)[c];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const float xf = Elem<DT>::get(&xv, e), af = Elem<DT>::get(&av, e);
      if (g.rank_mode == RANK_COSINE) {
        d = fma((double)xf, (double)af, d);
        xx = fma((double)xf, (double)xf, xx);
        nn = fma((double)af, (double)af, nn);
      } else {
        const float p = gm * af;
        const float r = xf - p;
        d = fma((double)r, (double)r, d);
      }
    }
  }
  if (g.rank_mode != RANK_COSINE) return d;
  const double den = __dsqrt_rn(xx * nn);
  return den > 0.0 ? 1.0 - fabs(d) / den : 1.0;
}

// Relative and absolute slack of the fp32 selector score against its fp64
// value (logit error of fp32 MFMA dots, fp32 exp and sums; the absolute part
// covers terms that underflow in fp32).
constexpr float ATT_REL = 1e-2f;
constexpr float ATT_ABS = 1e-30f;

// Replaces the utilities of the non-anchor positions (u >= 0) by the key of
// the configured ranking: its fp32 rounding and an fp32 interval around the
// exact value.  Thread = position, grid = (request, head, 256 positions).
template <int DT>
__global__ __launch_bounds__(256) void k_rankkeys(Geo g, Ws w, Cache c, const void* Kin, const void* Vin) {
  using E = typename Elem<DT>::T;
  int idx = blockIdx.x, b = 0;
  for (; b < g.B; ++b) {
    const int n = g.H * ((g.S[b] + 255) / 256);
    if (idx < n) break;
    idx -= n;
  }
  const int S = g.S[b], k = g.k[b], P = S - g.W;
  const int nc = (S + 255) / 256, h = idx / nc, t = (idx % nc) * 256 + threadIdx.x;
  if (t >= S) return;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  for (int side = 0; side < 2; ++side) {
    const size_t e = side * TS + po + t;
    if (!(w.u[e] >= 0.0f)) continue;  // anchor
    float u, lo, hi;
    if (g.rank_mode == RANK_ATTENTION) {
      const float sc = t < P ? w.sc[po + t] : 0.0f;
      u = sc;
      lo = fmaxf(sc * (1.0f - ATT_REL) - ATT_ABS, 0.0f);
      hi = sc * (1.0f + ATT_REL) + ATT_ABS;
      if (t >= P) lo = hi = 0.0f;
    } else {
      const int a = min(max(w.apos[e], 0), k - 1);
      const E* x = (const E*)(side ? Vin : Kin) + (po + t) * AKV_D;
      const E* ar = (const E*)(side ? c.ancV : c.ancK) + (ko + a) * AKV_D;
      const double key = rank_key64<DT>(g, side, h, t, x, ar, w.gpos[e]);
      u = __double2float_rn(key);
      lo = __double2float_rd(key);
      hi = __double2float_ru(key);
    }
    w.u[e] = u;
    w.uL[e] = lo;
    w.uU[e] = hi;
  }
}

__global__ __launch_bounds__(256) void k_bhist(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  int idx = blockIdx.x;
  const int L = locate_l(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const BList q = blist(g, L);
  if (bmode(g, q, side) != 0) return;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  const int n = q.n;
  const float* u = w.u + bbase(g, q, side);
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  constexpr int per = BCHUNK / 256;  // all loads issued before any is counted
  float v[per];
#pragma unroll
  for (int j = 0; j < per; ++j) v[j] = u[min(e0 + j * 256 + (int)threadIdx.x, e1 - 1)];
#pragma unroll
  for (int j = 0; j < per; ++j)
    if (e0 + j * 256 + (int)threadIdx.x < e1 && v[j] >= 0.0f) atomicAdd(&hist[__float_as_uint(v[j]) >> 20], 1u);
  __syncthreads();
  uint32_t* gh = w.bhist + (size_t)(L * 2 + side) * SEL_NBIN;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x)
    if (hist[i]) atomicAdd(&gh[i], hist[i]);
}

__global__ __launch_bounds__(256) void k_bcand(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[8], pick[2];
  static_assert(BCHUNK % 256 == 0, "whole rounds of 256 elements per chunk");
  int idx = blockIdx.x;
  const int L = locate_l(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const BList q = blist(g, L);
  if (bmode(g, q, side) != 0) return;
  const int bs = L * 2 + side;
  const uint32_t* gh = w.bhist + (size_t)bs * SEL_NBIN;
  stage_lds(hist, gh, SEL_NBIN);
  __syncthreads();
  digit_pick(hist, SEL_NBIN, nside(g, q, side), true, tmp, pick);
  const uint32_t bin1 = (uint32_t)pick[0];
  const int n = q.n;
  const float* u = w.u + bbase(g, q, side);
  float* cv = w.bcval + (size_t)bs * BCMAX;
  int32_t* cp = w.bcpos + (size_t)bs * BCMAX;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  constexpr int per = BCHUNK / 256;
  float v[per];
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    const int e = e0 + j * 256 + threadIdx.x;
    v[j] = e < e1 ? u[e] : -1.0f;
    cnt += v[j] >= 0.0f && (__float_as_uint(v[j]) >> 20) == bin1;
  }
  int slot = wg_reserve(cnt, &w.bstate[bs * BST_N + BST_NCAND], tmp);
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (v[j] >= 0.0f && (__float_as_uint(v[j]) >> 20) == bin1) {
      if (slot < BCMAX) {
        cv[slot] = v[j];
        cp[slot] = e0 + j * 256 + threadIdx.x;
      }
      ++slot;
    }
  }
}

__global__ __launch_bounds__(1024) void k_bcut(Geo g, Ws w, Cache c) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[20], pick[2];
  const int bs = blockIdx.x, L = bs >> 1, side = bs & 1;
  const BList q = blist(g, L);
  const int n = q.n;
  const int nch = q.nch;
  int32_t* tc = btie(g, w, L, q, side);
  int32_t* st = w.bstate + bs * BST_N;
  if (bmode(g, q, side) != 0) return;
  const int N = nside(g, q, side);
  const uint32_t* gh = w.bhist + (size_t)bs * SEL_NBIN;
  stage_lds(hist, gh, SEL_NBIN);
  __syncthreads();
  digit_pick(hist, SEL_NBIN, N, true, tmp, pick);
  if (pick[0] < 0) {  // fewer candidates than N: cannot happen with N < candidates
    if (threadIdx.x == 0) {
      atomicOr(&c.header[2], HDR_BUDGET_CUT);
      st[BST_T] = 0x7F800000;
      st[BST_REMAIN] = 0;
    }
    return;
  }
  int remaining = N - pick[1];
  uint32_t prefix = (uint32_t)pick[0] << 20, pmask = 0xFFF00000u;
  const int nc = st[0];
  const float* cv = w.bcval + (size_t)bs * BCMAX;
  const int32_t* cp = w.bcpos + (size_t)bs * BCMAX;
  const float* u = w.u + bbase(g, q, side);
  // Anchors carry -1 (sign bit set): they never match a prefix of a
  // non-negative utility.
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 8 : 0, nbin = pass == 0 ? SEL_NBIN : 256;
    if (nc <= BCMAX)
      digit_hist(hist, nbin, nc, [&](int i) { return __float_as_uint(cv[i]); }, pmask, prefix, shift);
    else
      digit_hist(hist, nbin, n, [&](int e) { return __float_as_uint(u[e]); }, pmask, prefix, shift);
    digit_pick(hist, nbin, remaining, true, tmp, pick);
    if (pick[0] < 0) {
      if (threadIdx.x == 0) {
        atomicOr(&c.header[2], HDR_BUDGET_CUT);
        st[BST_T] = 0x7F800000;
        st[BST_REMAIN] = 0;
      }
      return;
    }
    remaining -= pick[1];
    prefix |= (uint32_t)pick[0] << shift;
    pmask |= (uint32_t)(nbin - 1) << shift;
    __syncthreads();
  }
  // Threshold ties per chunk, then their exclusive scan over the chunks (in
  // rounds of SEL_NBIN chunks).
  int carry = 0;
  for (int c0 = 0; c0 < nch; c0 += SEL_NBIN) {
    const int c1 = min(nch, c0 + SEL_NBIN);
    for (int i = threadIdx.x; i < c1 - c0; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    if (nc <= BCMAX) {
      for (int i = threadIdx.x; i < nc; i += blockDim.x) {
        const int c = cp[i] / BCHUNK;
        if (__float_as_uint(cv[i]) == prefix && c >= c0 && c < c1) atomicAdd(&hist[c - c0], 1u);
      }
    } else {
      for (int e = c0 * BCHUNK + threadIdx.x; e < min(n, c1 * BCHUNK); e += blockDim.x)
        if (__float_as_uint(u[e]) == prefix) atomicAdd(&hist[e / BCHUNK - c0], 1u);
    }
    __syncthreads();
    // exclusive scan of the round's counts: each thread takes `per`
    // consecutive chunks
    const int ncc = c1 - c0, per = (ncc + (int)blockDim.x - 1) / (int)blockDim.x;
    int loc = 0;
    for (int i = 0; i < per; ++i) {
      const int ci = (int)threadIdx.x * per + i;
      if (ci < ncc) loc += (int)hist[ci];
    }
    int tot;
    int run = carry + block_excl_scan(loc, tmp, tot);
    for (int i = 0; i < per; ++i) {
      const int ci = (int)threadIdx.x * per + i;
      if (ci < ncc) {
        tc[c0 + ci] = run;
        run += (int)hist[ci];
      }
    }
    carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    st[BST_T] = (int)prefix;
    st[BST_REMAIN] = remaining;
  }
}

// Band limits A = min{uL : u >= T}, B = max{uU : u <= T} (float bits of
// non-negative values order like the values).
__global__ __launch_bounds__(256) void k_bbound(Geo g, Ws w) {
  __shared__ unsigned red[2][4];
  int idx = blockIdx.x;
  const int L = locate_l(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const BList q = blist(g, L);
  if (bmode(g, q, side) != 0) return;
  const int bs = L * 2 + side;
  const uint32_t T = (uint32_t)w.bstate[bs * BST_N + BST_T];
  const int n = q.n;
  const size_t base = bbase(g, q, side);
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  unsigned amin = 0x7F800000u, bmax = 0u;
  // the chunk's 16 elements per thread: estimates and both bounds are loaded
  // before any is compared (positions past the list end are skipped)
  constexpr int per = BCHUNK / 256;
  float v[per];
  unsigned lb[per], ub[per];
#pragma unroll
  for (int j = 0; j < per; ++j) {
    const int e = min(e0 + j * 256 + (int)threadIdx.x, e1 - 1);
    v[j] = w.u[base + e];
    lb[j] = __float_as_uint(w.uL[base + e]);
    ub[j] = __float_as_uint(w.uU[base + e]);
  }
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (!(e0 + j * 256 + (int)threadIdx.x < e1 && v[j] >= 0.0f)) continue;
    const uint32_t vb = __float_as_uint(v[j]);
    if (vb >= T) amin = min(amin, lb[j]);
    if (vb <= T) bmax = max(bmax, ub[j]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    amin = min(amin, (unsigned)__shfl_xor((int)amin, o, 64));
    bmax = max(bmax, (unsigned)__shfl_xor((int)bmax, o, 64));
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    red[0][wave] = amin;
    red[1][wave] = bmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 4; ++i) {
      amin = min(amin, red[0][i]);
      bmax = max(bmax, red[1][i]);
    }
    atomicMin((unsigned*)&w.bstate[bs * BST_N + BST_A], amin);
    atomicMax((unsigned*)&w.bstate[bs * BST_N + BST_B], bmax);
  }
}

__global__ __launch_bounds__(256) void k_bmark(Geo g, Ws w) {
  __shared__ int wtot[4];
  __shared__ int tmp[8];
  // the chunk's estimates and bounds, read coalesced and then taken by each
  // thread as 16 consecutive elements; the marks go back the same way
  __shared__ __align__(16) float s_u[BCHUNK];
  __shared__ __align__(16) uint32_t s_lb[BCHUNK], s_ub[BCHUNK];
  __shared__ __align__(16) uint8_t s_sel[BCHUNK];
  int idx = blockIdx.x;
  const int L = locate_l(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const BList q = blist(g, L);
  const int bs = L * 2 + side;
  int32_t* st = w.bstate + bs * BST_N;
  const int mode = bmode(g, q, side);
  const uint32_t T = (uint32_t)st[BST_T];
  const int need = st[BST_REMAIN];
  const uint32_t A = (uint32_t)st[BST_A], Bb = (uint32_t)st[BST_B];
  const int n = q.n;
  const int32_t* tc = btie(g, w, L, q, side);
  const int tie0 = mode == 0 ? tc[ch] : 0;  // threshold ties in the earlier chunks
  const size_t base = bbase(g, q, side);
  const float* u = w.u + base;
  uint8_t* sel = w.sel + base;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  // Each thread owns 16 consecutive elements; ranks of ties follow (h, t) order.
  constexpr int per = BCHUNK / 256;
  const int lo = e0 + threadIdx.x * per;
  {
    float cu[per];
    uint32_t cl[per], ch2[per];
#pragma unroll
    for (int j = 0; j < per; ++j) {
      const int e = min(e0 + j * 256 + (int)threadIdx.x, e1 - 1);
      cu[j] = u[e];
      cl[j] = mode == 0 ? __float_as_uint(w.uL[base + e]) : 0u;
      ch2[j] = mode == 0 ? __float_as_uint(w.uU[base + e]) : 0u;
    }
#pragma unroll
    for (int j = 0; j < per; ++j) {
      const int i = j * 256 + threadIdx.x;
      const bool in = e0 + i < e1;
      s_u[i] = in ? cu[j] : -1.0f;
      s_lb[i] = cl[j];
      s_ub[i] = ch2[j];
    }
  }
  __syncthreads();
  float v[per];
  uint32_t lbv[per], ubv[per];
#pragma unroll
  for (int j = 0; j < per; j += 4) {
    const int i = threadIdx.x * per + j;
    const float4 a4 = *(const float4*)&s_u[i];
    const uint4 l4 = *(const uint4*)&s_lb[i], h4 = *(const uint4*)&s_ub[i];
    v[j] = a4.x; v[j + 1] = a4.y; v[j + 2] = a4.z; v[j + 3] = a4.w;
    lbv[j] = l4.x; lbv[j + 1] = l4.y; lbv[j + 2] = l4.z; lbv[j + 3] = l4.w;
    ubv[j] = h4.x; ubv[j + 1] = h4.y; ubv[j + 2] = h4.z; ubv[j + 3] = h4.w;
  }
  int eq = 0;
  if (mode == 0)
#pragma unroll
    for (int j = 0; j < per; ++j) eq += (v[j] >= 0.0f && __float_as_uint(v[j]) == T);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = eq;
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wtot[wave] = x;
  __syncthreads();
  int before = x - eq + tie0;
  for (int i = 0; i < wave; ++i) before += wtot[i];
  unsigned bandbits = 0;  // element j of the thread is a band member
  int nb = 0, nsel = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    uint8_t s = 0;
    if (lo + j < e1 && v[j] >= 0.0f) {  // (v is -1 past the list end as well)
      if (mode == 1) {
        s = 1;
      } else if (mode == 0) {
        const uint32_t bits = __float_as_uint(v[j]);
        if (bits > T) {
          s = 1;
        } else if (bits == T) {
          s = before < need;
          ++before;
        }
        if (!(lbv[j] > Bb) && !(ubv[j] < A)) {
          bandbits |= 1u << j;
          ++nb;
          nsel += s;
        }
      }
    }
    s_sel[threadIdx.x * per + j] = s;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < per; ++j) {
    const int i = j * 256 + threadIdx.x;
    if (e0 + i < e1) sel[e0 + i] = s_sel[i];
  }
  if (mode != 0) return;  // uniform per workgroup
  // List the band members (one slot reservation per workgroup).
  int slot = wg_reserve(nb, &st[BST_NBAND], tmp);
  int32_t* bp = w.bandpos + (size_t)bs * BAND_CAP;
#pragma unroll
  for (int j = 0; j < per; ++j)
    if ((bandbits >> j) & 1u) {
      if (slot < BAND_CAP) {
        bp[slot] = lo + j;
        w.brank[(size_t)bs * BAND_CAP + slot] = 0;
      }
      ++slot;
    }
  const int ns = wave_sum_i(nsel);
  if (lane == 0 && ns) atomicAdd(&st[BST_NEED], ns);
}

// Sequential fp64 dots of a query row (16-byte chunks, chunk c at q4[c m]) with the
// member's key row x and, when R is set, its residual r (both fp64 in LDS):
// l = sum_j q_j x_j and qr = sum_j q_j r_j, products rounded, then added in
// j order.  The row is loaded 8 chunks at a time (half a bf16 row) before
// any is consumed (with 16 the kernel needs more than 168 registers and fits
// two waves per SIMD instead of three); the scheduling fences keep each
// chunk's LDS operands from being read ahead of earlier chunks' work.
template <int DT, bool R>
__device__ inline void qrow_dots(const u32x4* q4, int m, const double* xd, const double* rr, double& l, double& qr) {
  constexpr int PER = 16 / sizeof(typename Elem<DT>::T), NC = AKV_D / PER, QB = 8;
#pragma unroll 1
  for (int c0 = 0; c0 < NC; c0 += QB) {
    u32x4 qc[QB];
#pragma unroll
    for (int u = 0; u < QB; ++u) qc[u] = q4[(size_t)(c0 + u) * m];
#pragma unroll
    for (int u = 0; u < QB; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("" : "+v"(qc[u]));  // unpack this chunk here, not all at once
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const double qe = (double)chunk_elem<DT>(qc[u], e);
        l += qe * xd[(c0 + u) * PER + e];
        if constexpr (R) qr += qe * rr[(c0 + u) * PER + e];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// fp64 utility of every listed band member, one wave per member, computed as
// the oracle computes it (Sec. 3.3 Eq. utilities): the stored coefficient's
// residual r = x - fp32(gamma a) in fp32; per observation row w (lane w, w + 64,
// ...) the sequential fp64 dots l = q_w.k_t / sqrt(D), alpha = exp(l - M_w) /
// Z_w, and for keys q_w.r and ||v_t - y_w||^2, for values ||r||^2; the row
// terms alpha^2 (q.r)^2 / D ||v - y||^2 (or alpha^2 ||r||^2) summed in row
// order and divided by m.  The ATTENTION ranking sums alpha itself (the raw
// selector score, 0 inside the window); the other ablation keys come from
// rank_key64 on one lane.
template <int DT>
__global__ __launch_bounds__(256) void k_brescore(Geo g, Ws w, Cache c, const void* Kin, const void* Kobs,
                                                  const void* Vin) {
  using E = typename Elem<DT>::T;
  // the member's rows widened to fp64 once (exact), so the per-row loops
  // below convert only the query elements
  __shared__ float rs[4][AKV_D];
  __shared__ double xd[4][AKV_D], vd[4][AKV_D];
  __shared__ double rr[4][AKV_D];  // r, or R_t r_K when positions are encoded
  __shared__ double terms[4][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = gridDim.x * 4;
  const int gw = blockIdx.x * 4 + wave;
  const int m = g.m, D = AKV_D;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;
  const double sqd = sqrt((double)D);
  int base = 0;  // members of the earlier lists
  for (int bs = 0; bs < 2 * g.B * g.hdiv; ++bs) {
    const int L = bs >> 1, side = bs & 1;
    const BList bl = blist(g, L);
    const int b = bl.b;
    const int nl = w.bstate[bs * BST_N + BST_NBAND];
    const int n = (bmode(g, bl, side) == 0 && nl <= BAND_CAP) ? nl : 0;
    int i0 = gw - base;
    if (i0 < 0) i0 += ((-i0 + nw - 1) / nw) * nw;
    for (int i = i0; i < n; i += nw) {
      const int S = g.S[b], k = g.k[b];
      const int f = w.bandpos[(size_t)bs * BAND_CAP + i];
      const int h = bl.h0 + f / S, t = f % S;
      const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
      const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
      const size_t xo = (po + t) * D;
      const int a = min(max(w.apos[side * TS + po + t], 0), k - 1);
      const float gm = w.gpos[side * TS + po + t];
      const E* xr = (const E*)(side ? Vin : Kin) + xo;
      const E* ar = (const E*)(side ? c.ancV : c.ancK) + (ko + a) * D;
      const E* kr = (const E*)Kobs + xo;  // the keys of the logits (rotated when positions are encoded)
      const E* vr = (const E*)Vin + xo;
      const bool att = g.rank_mode == RANK_ATTENTION;
      if ((g.rank_mode != RANK_UTILITY && !att) || (att && t >= S - g.W)) {  // uniform per wave
        if (lane == 0) w.bandu[(size_t)bs * BAND_CAP + i] = att ? 0.0 : rank_key64<DT>(g, side, h, t, xr, ar, gm);
        continue;
      }
      for (int j = lane; j < D; j += 64) {
        const float p = gm * Elem<DT>::get(ar, j);
        const float r = Elem<DT>::get(xr, j) - p;
        rs[wave][j] = r;
        rr[wave][j] = r;
        xd[wave][j] = Elem<DT>::get(kr, j);
        vd[wave][j] = Elem<DT>::get(vr, j);
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      const bool rot = g.rope && side == 0;
      if (rot) {
        // (c r_f - s r_{f+D/2}, s r_f + c r_{f+D/2}) in fp64: exact products
        // of fp32 factors, one rounding per coordinate, as the oracle forms it
        const int f = lane;
        const float2 cv = *(const float2*)&w.cs[(size_t)t * D + 2 * f];
        const double cd = cv.x, sd = cv.y, a = rs[wave][f], bb = rs[wave][f + D / 2];
        rr[wave][f] = cd * a - sd * bb;
        rr[wave][f + D / 2] = sd * a + cd * bb;
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      }
      double rvn = 0.0;
      if (side == 1)
        for (int j = 0; j < D; ++j) rvn += rr[wave][j] * rr[wave][j];
      const size_t bh = (size_t)b * g.H + h;
      for (int wr = lane; wr < m; wr += 64) {
        // q.k (and q.r_K for keys) over the lane's query row
        const u32x4* q4 = (const u32x4*)w.qt + bh * m * (AKV_D * sizeof(E) / 16) + wr;
        double l = 0.0, qr = 0.0;
        if (side == 0 && !att)
          qrow_dots<DT, true>(q4, m, xd[wave], rr[wave], l, qr);
        else
          qrow_dots<DT, false>(q4, m, xd[wave], rr[wave], l, qr);
        l = l / sqd;
        const double al = exp(l - w.M64[bh * m + wr]) / w.Z64[bh * m + wr];
        const double a2 = al * al;
        double term;
        if (att) {
          term = al;
        } else if (side == 0) {
          // ||v_t - y_w||^2 (sequential); y_w is stored in dimension pairs
          // with the rows innermost, so that one load of the wave reads 64
          // rows' pair p as 1 KB of contiguous memory.  Sixteen pairs are
          // loaded before any is consumed.
          const double2* y2 = (const double2*)(w.Y64 + bh * m * D) + wr;
          double vy = 0.0;
          constexpr int YB = 16;
#pragma unroll 1
          for (int p0 = 0; p0 < AKV_D / 2; p0 += YB) {
            double2 yc[YB];
#pragma unroll
            for (int u = 0; u < YB; ++u) yc[u] = y2[(size_t)(p0 + u) * m];
#pragma unroll
            for (int u = 0; u < YB; ++u) {
              __builtin_amdgcn_sched_barrier(0);
              const double d0 = vd[wave][2 * (p0 + u)] - yc[u].x;
              vy += d0 * d0;
              const double d1 = vd[wave][2 * (p0 + u) + 1] - yc[u].y;
              vy += d1 * d1;
            }
            __builtin_amdgcn_sched_barrier(0);
          }
          term = a2 * (qr * qr / D) * vy;
        } else {
          term = a2 * rvn;
        }
        terms[wave][wr] = term;
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      if (lane == 0) {
        // row order, the terms read 16 at a time
        double su = 0.0;
        for (int w0 = 0; w0 < m; w0 += 16) {
          double tv[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) tv[u] = terms[wave][w0 + u];
#pragma unroll
          for (int u = 0; u < 16; ++u)
            if (w0 + u < m) su += tv[u];
        }
        w.bandu[(size_t)bs * BAND_CAP + i] = su / m;
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
    base += n;
  }
}

// Exact ranks inside the band: member i is selected when fewer than `need`
// members precede it in (fp64 utility descending, flattened index ascending)
// order.  k_brank counts, per 256 x 256 tile of (member i, member j) pairs,
// the j that precede each i and adds the counts to brank[i] (zeroed when the
// member was listed); the tiles of all lists are spread over a fixed grid.
// k_bsel then marks the band members from their ranks.
constexpr int RANK_T = 256;
__global__ __launch_bounds__(RANK_T) void k_brank(Geo g, Ws w) {
  __shared__ double su[RANK_T];
  __shared__ int sp[RANK_T];
  int tile0 = 0;
  for (int bs = 0; bs < 2 * g.B * g.hdiv; ++bs) {
    const int side = bs & 1;
    const BList bl = blist(g, bs >> 1);
    const int nl = w.bstate[bs * BST_N + BST_NBAND];
    const int n = (bmode(g, bl, side) == 0 && nl <= BAND_CAP) ? nl : 0;
    const int nt = (n + RANK_T - 1) / RANK_T;
    const int32_t* bp = w.bandpos + (size_t)bs * BAND_CAP;
    const double* bu = w.bandu + (size_t)bs * BAND_CAP;
    int32_t* br = w.brank + (size_t)bs * BAND_CAP;
    int t = (int)blockIdx.x - tile0;
    if (t < 0) t += ((-t + (int)gridDim.x - 1) / (int)gridDim.x) * (int)gridDim.x;
    for (; t < nt * nt; t += gridDim.x) {  // uniform per workgroup
      const int ti = t / nt, tj = t % nt;
      const int j = tj * RANK_T + threadIdx.x;
      __syncthreads();
      su[threadIdx.x] = j < n ? bu[j] : 0.0;
      sp[threadIdx.x] = j < n ? bp[j] : 0x7FFFFFFF;
      __syncthreads();
      const int i = ti * RANK_T + threadIdx.x;
      if (i < n) {
        const double ui = bu[i];
        const int pi = bp[i];
        const int nj = min(RANK_T, n - tj * RANK_T);
        // eight members per step, read before any is compared, no branches
        int r = 0;
        for (int j0 = 0; j0 < nj; j0 += 8) {
          double uj[8];
          int pj[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            uj[u] = su[j0 + u];
            pj[u] = sp[j0 + u];
          }
#pragma unroll
          for (int u = 0; u < 8; ++u)
            r += (j0 + u < nj) & ((uj[u] > ui) | ((uj[u] == ui) & (pj[u] < pi)));
        }
        if (r) atomicAdd(&br[i], r);
      }
    }
    tile0 += nt * nt;
  }
}

__global__ __launch_bounds__(256) void k_bsel(Geo g, Ws w, Cache c) {
  const int bs = blockIdx.y, side = bs & 1;
  const BList bl = blist(g, bs >> 1);
  if (bmode(g, bl, side) != 0) return;
  const int n = w.bstate[bs * BST_N + BST_NBAND];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    atomicAdd(&c.stats[bl.b * 4 + 2 + side], n);  // band size (summed over heads), reported by the export
    if (n > BAND_CAP) atomicOr(&c.header[2], HDR_BAND_OVERFLOW);
  }
  if (n > BAND_CAP) return;
  const int need = w.bstate[bs * BST_N + BST_NEED];
  uint8_t* sel = w.sel + bbase(g, bl, side);
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    sel[w.bandpos[(size_t)bs * BAND_CAP + i]] = w.brank[(size_t)bs * BAND_CAP + i] < need ? 1 : 0;
}

hipError_t launch_budget(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs, const void* V,
                         hipStream_t st) {
  int nblk = 0, nkey = 0;
  const int nl = g.B * g.hdiv;
  for (int L = 0; L < nl; ++L) nblk += 2 * (((g.H / g.hdiv) * g.S[L / g.hdiv] + BCHUNK - 1) / BCHUNK);
  for (int b = 0; b < g.B; ++b) nkey += g.H * ((g.S[b] + 255) / 256);
  if (g.rank_mode != RANK_UTILITY) {
    if (g.dtype == 1)
      launch("k_rankkeys", k_rankkeys<1>, dim3(nkey), dim3(256), 0, st, g, w, c, K, V);
    else
      launch("k_rankkeys", k_rankkeys<0>, dim3(nkey), dim3(256), 0, st, g, w, c, K, V);
  }
  launch("k_bhist", k_bhist, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bcand", k_bcand, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bcut", k_bcut, dim3(nl * 2), dim3(1024), 0, st, g, w, c);
  launch("k_bbound", k_bbound, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bmark", k_bmark, dim3(nblk), dim3(256), 0, st, g, w);
  if (g.dtype == 1)
    launch("k_brescore", k_brescore<1>, dim3(1024), dim3(256), 0, st, g, w, c, K, Kobs, V);
  else
    launch("k_brescore", k_brescore<0>, dim3(1024), dim3(256), 0, st, g, w, c, K, Kobs, V);
  launch("k_brank", k_brank, dim3(2048), dim3(RANK_T), 0, st, g, w);
  launch("k_bsel", k_bsel, dim3(64, nl * 2), dim3(256), 0, st, g, w, c);
  return hipGetLastError();
}

}  // namespace akv
