// Anchor selection (Sec. 3.2 "Anchor selection"; App. A.2 Eq. selector-score;
// Algorithm 1, first step) and anchor preparation.
//
// Selection: average-pool the observation score over kappa positions (zero
// padding, divided by kappa), take the floor(rho (k - W)) best pooled
// positions of [0, S - W) (ties to the lower position) by an exact radix
// select on the fp32 bits, sample the rest of the non-window budget uniformly
// without replacement (the positions with the smallest SplitMix64 hash), add
// the window, and write the ascending anchor list and the position ->
// anchor-index map.  Every pass runs on SEL_SLICE-position slices of all
// (request, head) pairs at once.  A decision that needs a whole head (a digit
// of the radix select, the exact cut among candidates, the ranking of hash
// candidates) is taken by every workgroup of the next pass from the totals
// and lists the previous pass left in memory (the kernel boundary publishes
// them), so no workgroup waits for another:
//   k_sel_pool  : marks reset, pooled scores, histogram of their first 12-bit
//                 digit;
//   k_sel_cand  : the digit of the n_top-th largest; scores inside its bin
//                 appended as candidates;
//   k_sel_class : the exact cut (remaining two digits) among the candidates;
//                 positions clearly above it taken, the band around it listed
//                 for the fp64 re-scoring (k_sel_band);
//   k_sel_rhist : band decisions (fp32 order on a band overflow), histogram of
//                 the hash's top 12 bits over the untaken positions;
//   k_sel_rcand : the bin of the n_rand-th smallest key; keys below it taken,
//                 keys inside it appended; per-slice anchor counts;
//   k_sel_list  : the bin's keys ranked and the smallest taken; the anchor
//                 list and the map, slices placed by the counts.
//   k_anchor_prep : copies anchor keys/values into the cache, their canonical
//                   fp64 squared norms and fp32 inverse norms, and the table
//                   QA[a][w] = q_w . abar^K_a used by the key utilities.
#include "akv_common.h"

namespace akv {

// Positions whose fp32 pooled score lies within SEL_BAND (relative) of the
// cut are re-scored in fp64 (at most SEL_BAND_MAX of them).  The fp32 score's
// error is below 1e-4 relative: fp32 accumulation of 128 exact bf16 products
// (at most 128 * 2^-24 * sum |q_i k_i| / sqrt(D) on a logit), fp32 exp and
// sums; the band is ten times wider.  The fp64 scores use exact fp64 logits
// and the row maxima M_w and sums Z_w of the fp64 observation pass (fp64
// logits and exponentials throughout), so they match the canonical fp64
// definition to rounding order, far below the gaps between real scores.
constexpr float SEL_BAND = 1e-3f;

// fp64 pooled selector score of band member i of (request b, head h), one
// workgroup per member (k_sel_band): (1/kappa) sum_{|d| <= kappa/2,
// 0 <= t+d < P} (1/m) sum_w exp(dot64(q_w, k_{t+d}) / sqrt(D) - M_w) / Z_w,
// with the row statistics of the fp64 observation pass.  The m query rows and the
// kappa key rows are staged in LDS when they fit; thread = (row, offset)
// pair.  The dot products are exact fp64 products (fused multiply-add of an
// exact product rounds once, like an add) in four interleaved partial sums
// (the order differs from a sequential sum by ~1e-16 relative, far below the
// band's resolution); the terms are combined in a fixed order.
constexpr int SEL_QLDS = 32768;  // bytes of staged query rows
constexpr int SEL_KLDS = 8192;   // bytes of staged key rows

template <int DT>
__global__ __launch_bounds__(256) void k_sel_band(Geo g, Ws w, const void* Kin, const void* Qin) {
  using E = typename Elem<DT>::T;
  constexpr int PER = 16 / sizeof(E), NCH = AKV_D / PER;
  __shared__ __align__(16) unsigned char qlds[SEL_QLDS];
  __shared__ __align__(16) unsigned char klds[SEL_KLDS];
  __shared__ double part[256 * 2];
  const int bh = blockIdx.x / SEL_BAND_MAX, i = blockIdx.x % SEL_BAND_MAX;
  const int b = bh / g.H, h = bh % g.H;
  const int nb = w.sstate[bh * SS_N + SS_NBAND];
  if (i >= nb || nb > SEL_BAND_MAX) return;  // past the band, or an overflowed band
  const int S = g.S[b], P = S - g.W, m = g.m;
  const int tid = threadIdx.x, nt = blockDim.x, half = g.kappa / 2, nk = 2 * half + 1;
  const int t = w.sband[(size_t)bh * SEL_BAND_MAX + i];
  const E* X = (const E*)Kin + ((size_t)g.prefS[b] * g.H + (size_t)h * S) * AKV_D;
  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * AKV_D;
  const double* M64 = w.M64 + (size_t)bh * m;
  const double* Z64 = w.Z64 + (size_t)bh * m;
  const double isd = 1.0 / sqrt((double)AKV_D);
  const bool qst = (size_t)m * AKV_D * sizeof(E) <= SEL_QLDS;
  const bool kst = (size_t)nk * AKV_D * sizeof(E) <= SEL_KLDS;
  E* qs = (E*)qlds;
  E* ks = (E*)klds;
  if (qst) stage_lds((uint4*)qs, (const uint4*)Q, m * NCH);
  if (kst)
    for (int c = tid; c < nk * NCH; c += nt) {
      const int u = min(max(t + c / NCH - half, 0), P - 1);
      ((uint4*)ks)[c] = ((const uint4*)(X + (size_t)u * AKV_D))[c % NCH];
    }
  __syncthreads();
  double acc = 0.0;
  for (int wr = tid; wr < m; wr += nt) {
    const E* q = qst ? qs + (size_t)wr * AKV_D : Q + (size_t)wr * AKV_D;
    double rs = 0.0;
    for (int r = 0; r < nk; ++r) {
      const int u = t + r - half;
      if (u < 0 || u >= P) continue;
      const E* x = kst ? ks + (size_t)r * AKV_D : X + (size_t)u * AKV_D;
      double p4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
      for (int ch = 0; ch < NCH; ++ch) {
        const uint4 qv = ((const uint4*)q)[ch], xv = ((const uint4*)x)[ch];
        const E* qe = (const E*)&qv;
        const E* xe = (const E*)&xv;
#pragma unroll
        for (int e = 0; e < PER; ++e)
          p4[e & 3] = fma((double)Elem<DT>::get(qe, e), (double)Elem<DT>::get(xe, e), p4[e & 3]);
      }
      const double l = ((p4[0] + p4[1]) + (p4[2] + p4[3])) * isd;
      rs += exp(l - M64[wr]) / Z64[wr];
    }
    acc += rs;
  }
  // rows summed per thread (rows tid, tid + nt, ...), then over threads in order
  part[tid] = acc;
  __syncthreads();
  if (tid == 0) {
    // in thread order, the partials read 16 at a time (nt is a multiple of 16)
    double tot = 0.0;
    for (int r0 = 0; r0 < nt; r0 += 16) {
      double pv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) pv[u] = part[r0 + u];
#pragma unroll
      for (int u = 0; u < 16; ++u) tot += pv[u];
    }
    w.sbscore[(size_t)bh * SEL_BAND_MAX + i] = tot / (double)m / (double)g.kappa;
  }
}

// ------------------------------------------------------------------ slice passes
// Slice sl of (request b, head h): positions [sl * SEL_SLICE, ...) of [0, S).
struct SelSlice {
  int b, h, bh, sl, nsl, S, P, k, t0, t1;  // [t0, t1) = the slice's part of [0, P)
  size_t so;                                // offset of the head's position arrays
};
__device__ inline SelSlice sel_slice(const Geo& g) {
  SelSlice q;
  int idx = blockIdx.x;
  q.b = locate(g, SEL_SLICE, 1, idx);
  q.S = g.S[q.b];
  q.P = q.S - g.W;
  q.k = g.k[q.b];
  q.nsl = (q.S + SEL_SLICE - 1) / SEL_SLICE;
  q.h = idx / q.nsl;
  q.sl = idx % q.nsl;
  q.bh = q.b * g.H + q.h;
  q.t0 = q.sl * SEL_SLICE;
  q.t1 = min(q.P, q.t0 + SEL_SLICE);
  q.so = (size_t)g.prefS[q.b] * g.H + (size_t)q.h * q.S;
  return q;
}

// Appends the lanes' `take` values to a per-head list: one atomic per wave.
// Returns the slot (or -1 for lanes that append nothing).
__device__ inline int wave_append(bool take, int32_t* count) {
  const unsigned long long bal = __ballot(take);
  if (!bal) return -1;
  const int lane = threadIdx.x & 63;
  const int leader = __ffsll((long long)bal) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(count, __popcll(bal));
  base = __shfl(base, leader, 64);
  return take ? base + __popcll(bal & ((1ull << lane) - 1ull)) : -1;
}

// The bin of a head's summed histogram where the running count (from the
// top when `desc`) reaches `need`, and the count before it; whole workgroup.
__device__ inline void pick_global(const uint32_t* gh, uint32_t* hist, int need, bool desc, int* tmp, int* pick) {
  stage_lds(hist, gh, SEL_NBIN);
  __syncthreads();
  digit_pick(hist, SEL_NBIN, need, desc, tmp, pick);
}

// Marks reset over the slice's positions of [0, S), pooled scores over its
// part of [0, P) (the scores with their halo staged in LDS; terms added in
// offset order from -kappa/2), and the histogram of their first digit
// [31:20] (non-negative scores order as their bits) added to the head's.
__global__ __launch_bounds__(256) void k_sel_pool(Geo g, Ws w, int override_anchors) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ float stile[SEL_SLICE + SEL_HALO];
  const SelSlice q = sel_slice(g);
  const int tid = threadIdx.x, nt = blockDim.x;
  int32_t* rank = w.rank + q.so;
  uint8_t* flag = w.flag + q.so;
  for (int t = q.t0 + tid; t < min(q.S, q.t0 + SEL_SLICE); t += nt) {
    rank[t] = -1;
    flag[t] = 0;
  }
  if (override_anchors) return;
  const int half = g.kappa / 2;
  const float* sc = w.sc + q.so;
  float* pooled = w.u + q.so;  // the utility buffer is free until the epilogue
  // the slice's scores and halo, eight loads in flight per thread (indices
  // clamped into the head's row; positions outside [0, P) read as 0)
  const int ntile = q.t1 - q.t0 + 2 * half;
  for (int j0 = tid; j0 < ntile; j0 += 8 * nt) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = sc[min(max(q.t0 - half + j0 + e * nt, 0), max(q.P - 1, 0))];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int j = j0 + e * nt, u = q.t0 - half + j;
      if (j < ntile) stile[j] = (u >= 0 && u < q.P) ? v[e] : 0.0f;
    }
  }
  for (int i = tid; i < SEL_NBIN; i += nt) hist[i] = 0;
  __syncthreads();
  const int ntop = g.ntop[q.b];
  for (int t = q.t0 + tid; t < q.t1; t += nt) {
    float s = 0.0f;
    for (int d = 0; d <= 2 * half; ++d) s += stile[t - q.t0 + d];
    const float v = s / (float)g.kappa;
    pooled[t] = v;
    if (ntop > 0) atomicAdd(&hist[__float_as_uint(v) >> 20], 1u);
  }
  __syncthreads();
  uint32_t* gh = w.sghist + (size_t)q.bh * SEL_NBIN;
  if (ntop > 0)
    for (int i = tid; i < SEL_NBIN; i += nt)
      if (hist[i]) atomicAdd(&gh[i], hist[i]);
}

// The first digit of the n_top-th largest score and the count above its bin
// (every workgroup, from the head's histogram); the slice's scores inside
// the bin are appended as candidates.
__global__ __launch_bounds__(256) void k_sel_cand(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[8], pick[2];
  const SelSlice q = sel_slice(g);
  const int ntop = g.ntop[q.b];
  if (ntop <= 0) return;
  const int tid = threadIdx.x;
  int32_t* st = w.sstate + q.bh * SS_N;
  pick_global(w.sghist + (size_t)q.bh * SEL_NBIN, hist, ntop, true, tmp, pick);
  const uint32_t bin1 = (uint32_t)pick[0];
  if (q.sl == 0 && tid == 0) {
    st[SS_BIN1] = pick[0];
    st[SS_ABOVE1] = pick[1];
  }
  const float* pooled = w.u + q.so;
  float* cand = w.scand + (size_t)q.bh * SEL_CMAX;
  constexpr int per = SEL_SLICE / 256;
  float v[per];
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    const int t = q.t0 + j * 256 + tid;
    v[j] = t < q.t1 ? pooled[t] : -1.0f;
    cnt += v[j] >= 0.0f && (__float_as_uint(v[j]) >> 20) == bin1;
  }
  int slot = wg_reserve(cnt, &st[SS_NCAND], tmp);
#pragma unroll
  for (int j = 0; j < per; ++j)
    if (v[j] >= 0.0f && (__float_as_uint(v[j]) >> 20) == bin1) {
      if (slot < SEL_CMAX) cand[slot] = v[j];
      ++slot;
    }
}

// The exact cut (every workgroup): digits [19:8] and [7:0] of the n_top-th
// largest score and the count still to take among scores equal to it, from
// the candidate list or, when it overflowed, from all of [0, P) (same
// digits, same result).  Then the slice's scores clearly above the band
// around the cut are taken and the band's members listed.
__global__ __launch_bounds__(256) void k_sel_class(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[8], pick[2];
  const SelSlice q = sel_slice(g);
  const int ntop = g.ntop[q.b];
  if (ntop <= 0) return;
  const int tid = threadIdx.x, nt = blockDim.x;
  int32_t* st = w.sstate + q.bh * SS_N;
  const float* pooled = w.u + q.so;
  const float* cand = w.scand + (size_t)q.bh * SEL_CMAX;
  const int nc = st[SS_NCAND];
  int remaining = ntop - st[SS_ABOVE1];
  uint32_t prefix = (uint32_t)st[SS_BIN1] << 20, pmask = 0xFFF00000u;
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 8 : 0, nbin = pass == 0 ? SEL_NBIN : 256;
    if (nc <= SEL_CMAX)
      digit_hist(hist, nbin, nc, [&](int i) { return __float_as_uint(cand[i]); }, pmask, prefix, shift);
    else
      digit_hist(hist, nbin, q.P, [&](int t) { return __float_as_uint(pooled[t]); }, pmask, prefix, shift);
    digit_pick(hist, nbin, remaining, true, tmp, pick);
    remaining -= pick[1];
    prefix |= (uint32_t)pick[0] << shift;
    pmask |= (uint32_t)(nbin - 1) << shift;
    __syncthreads();
  }
  if (q.sl == 0 && tid == 0) {
    st[SS_PREFIX] = (int)prefix;
    st[SS_REMAIN] = remaining;
  }
  // The head's histogram is read by no later workgroup of this pass; clear it
  // for the hash histogram.
  if (q.sl == 0)
    for (int i = tid; i < SEL_NBIN; i += nt) w.sghist[(size_t)q.bh * SEL_NBIN + i] = 0u;
  const float cut = __uint_as_float(prefix);
  const float bhi = cut * (1.0f + SEL_BAND), blo = cut * (1.0f - SEL_BAND);
  uint8_t* flag = w.flag + q.so;
  int32_t* band = w.sband + (size_t)q.bh * SEL_BAND_MAX;
  int above = 0;
  for (int t0 = q.t0; t0 < q.t1; t0 += nt) {
    const int t = t0 + tid;
    const float v = t < q.t1 ? pooled[t] : -1.0f;
    if (v > bhi) {
      flag[t] = 1;
      ++above;
    }
    const int slot = wave_append(v <= bhi && v >= blo, &st[SS_NBAND]);
    if (slot >= 0 && slot < SEL_BAND_MAX) band[slot] = t;
  }
  above = wave_sum_i(above);
  if ((tid & 63) == 0 && above) atomicAdd(&st[SS_NABOVE], above);
}

// Band decisions for the slice's members: rank by fp64 score (ties to the
// lower position) against all members.  On a band overflow the fp32 order
// decides instead: scores above the cut are taken, and of those equal to it
// the first `remaining` in position order (equal scores in earlier slices
// counted here).  Then the histogram of the hash's top 12 bits over the
// slice's untaken positions is added to the head's.
__global__ __launch_bounds__(256) void k_sel_rhist(Geo g, Ws w, Cache c) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ uint8_t sflag[SEL_SLICE];
  __shared__ int tmp[8];
  const SelSlice q = sel_slice(g);
  const int tid = threadIdx.x, nt = blockDim.x;
  int32_t* st = w.sstate + q.bh * SS_N;
  uint8_t* flag = w.flag + q.so;
  const int ntop = g.ntop[q.b];
  const int nb = ntop > 0 ? st[SS_NBAND] : 0;
  if (nb > SEL_BAND_MAX) {
    if (q.sl == 0 && tid == 0) atomicOr(&c.header[2], 32u);
    const uint32_t prefix = (uint32_t)st[SS_PREFIX];
    const float* pooled = w.u + q.so;
    int eq = 0;
    for (int t = tid; t < q.t0 && t < q.P; t += nt) eq += __float_as_uint(pooled[t]) == prefix;
    int before_slice;
    block_excl_scan(eq, tmp, before_slice);
    const int per = SEL_SLICE / 256;
    const int lo = min(q.t1, q.t0 + tid * per), hi = min(q.t1, lo + per);
    int e2 = 0;
    for (int t = lo; t < hi; ++t) e2 += __float_as_uint(pooled[t]) == prefix;
    int tot;
    int before = before_slice + block_excl_scan(e2, tmp, tot);
    const int remaining = st[SS_REMAIN];
    for (int t = lo; t < hi; ++t) {
      const uint32_t u = __float_as_uint(pooled[t]);
      uint8_t f = 0;
      if (u > prefix) {
        f = 1;
      } else if (u == prefix) {
        if (before < remaining) f = 1;
        ++before;
      }
      flag[t] = f;
      sflag[t - q.t0] = f;
    }
  } else {
    if (q.t1 > q.t0) {  // the slice's flags, all loaded before any is stored
      constexpr int NJ = SEL_SLICE / 256;
      uint8_t fv[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) fv[j] = flag[min(q.t0 + j * 256 + tid, q.t1 - 1)];
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if (q.t0 + j * 256 + tid < q.t1) sflag[j * 256 + tid] = fv[j];
    }
    if (nb > 0) {
      const int need = ntop - st[SS_NABOVE];
      const int32_t* band = w.sband + (size_t)q.bh * SEL_BAND_MAX;
      const double* bscore = w.sbscore + (size_t)q.bh * SEL_BAND_MAX;
      __syncthreads();
      for (int i = tid; i < nb; i += nt) {
        const int t = band[i];
        if (t < q.t0 || t >= q.t1) continue;
        const double si = bscore[i];
        int r = 0;
        for (int j = 0; j < nb; ++j) r += bscore[j] > si || (bscore[j] == si && band[j] < t);
        if (r < need) {
          flag[t] = 1;
          sflag[t - q.t0] = 1;
        }
      }
    }
  }
  const int nrand = g.nrand[q.b];
  if (nrand <= 0) return;
  for (int i = tid; i < SEL_NBIN; i += nt) hist[i] = 0;
  __syncthreads();
  const unsigned long long hs = g.seed_anchor ^ ((unsigned long long)q.h << 40);
  for (int t = q.t0 + tid; t < q.t1; t += nt)
    if (!sflag[t - q.t0]) atomicAdd(&hist[splitmix64(hs ^ (unsigned long long)t) >> 52], 1u);
  __syncthreads();
  uint32_t* gh = w.sghist + (size_t)q.bh * SEL_NBIN;
  for (int i = tid; i < SEL_NBIN; i += nt)
    if (hist[i]) atomicAdd(&gh[i], hist[i]);
}

// The bin of the n_rand-th smallest key (every workgroup, from the head's
// histogram); the slice's untaken positions with a key below it are taken,
// those inside it appended (keys are distinct: SplitMix64 is a bijection).
// Each workgroup leaves its slice's anchor count (bin members excluded).
__global__ __launch_bounds__(256) void k_sel_rcand(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[8], pick[2], wcnt[4];
  const SelSlice q = sel_slice(g);
  const int tid = threadIdx.x, nt = blockDim.x;
  int32_t* st = w.sstate + q.bh * SS_N;
  uint8_t* flag = w.flag + q.so;
  const int nrand = g.nrand[q.b];
  unsigned long long bin = ~0ull;
  if (nrand > 0) {
    pick_global(w.sghist + (size_t)q.bh * SEL_NBIN, hist, nrand, false, tmp, pick);
    bin = (unsigned long long)pick[0];
    if (q.sl == 0 && tid == 0) {
      st[SS_RBIN] = pick[0];
      st[SS_RNEED] = nrand - pick[1];
    }
  }
  const unsigned long long hs = g.seed_anchor ^ ((unsigned long long)q.h << 40);
  unsigned long long* ckey = w.rkey + (size_t)q.bh * SEL_CAND;
  int32_t* cpos = w.rpos + (size_t)q.bh * SEL_CAND;
  int cnt = 0;
  for (int t0 = q.t0; t0 < q.t1; t0 += nt) {
    const int t = t0 + tid;
    uint8_t f = t < q.t1 ? flag[t] : 1;
    bool app = false;
    if (!f && nrand > 0) {
      const unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
      if ((key >> 52) < bin) {
        flag[t] = 2;
        f = 2;
      } else if ((key >> 52) == bin) {
        app = true;
      }
    }
    const int slot = wave_append(app, &st[SS_NRC]);
    if (slot >= 0 && slot < SEL_CAND) {
      ckey[slot] = splitmix64(hs ^ (unsigned long long)t);
      cpos[slot] = t;
    }
    cnt += (t < q.t1 && f != 0);
  }
  cnt = wave_sum_i(cnt);
  if ((tid & 63) == 0) wcnt[tid >> 6] = cnt;
  __syncthreads();
  const int nslmax = (g.maxS + SEL_SLICE - 1) / SEL_SLICE;
  if (tid == 0) w.slcnt[(size_t)q.bh * nslmax + q.sl] = (wcnt[0] + wcnt[1]) + (wcnt[2] + wcnt[3]);
}

// The hash bin's keys are ranked (every workgroup; on a candidate overflow
// the radix select finishes on the remaining 52 bits over all of [0, P), in
// digits of 12, 12, 12, 12 and 4 bits) and the smallest taken.  The slice's
// flagged positions then go after those of the earlier slices (their counts
// plus the bin members taken there), in position order (wave ballots and a
// scan of the per-wave counts); then the window.  The slice holding
// position P - 1 (or the first slice when P = 0) checks the total.
__global__ __launch_bounds__(256) void k_sel_list(Geo g, Ws w, Cache c) {
  constexpr int NJ = SEL_SLICE / 256;  // positions per thread of the slice
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ unsigned long long skey[SEL_CAND];  // the bin's keys, staged for the ranking
  __shared__ int tmp[8], pick[2], wc[NJ][4], wpre[NJ][4], wtot, basev, extra;
  const SelSlice q = sel_slice(g);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int W = g.W, k = g.k[q.b];
  const int nslmax = (g.maxS + SEL_SLICE - 1) / SEL_SLICE;
  const int32_t* slc = w.slcnt + (size_t)q.bh * nslmax;
  const int32_t* st = w.sstate + q.bh * SS_N;
  int32_t* rank = w.rank + q.so;
  uint8_t* flag = w.flag + q.so;
  int32_t* anc = c.anc_pos + (size_t)g.prefK[q.b] * g.H + (size_t)q.h * k;
  if (tid == 0) extra = 0;
  __syncthreads();
  const int nrand = g.nrand[q.b];
  if (nrand > 0) {
    const int need = st[SS_RNEED];
    const int nc = st[SS_NRC];
    const unsigned long long bin = (unsigned long long)st[SS_RBIN];
    const unsigned long long* ckey = w.rkey + (size_t)q.bh * SEL_CAND;
    const int32_t* cpos = w.rpos + (size_t)q.bh * SEL_CAND;
    if (nc <= SEL_CAND) {
      if (nc > 0) stage_lds(skey, ckey, nc);
      __syncthreads();
      int ex = 0;
      for (int i = tid; i < nc; i += blockDim.x) {
        const unsigned long long ki = skey[i];
        int r = 0;
        for (int j = 0; j < nc; ++j) r += skey[j] < ki;
        if (r < need) {
          const int t = cpos[i];
          if (t < q.t0) ++ex;
          else if (t < q.t1) flag[t] = 2;
        }
      }
      ex = wave_sum_i(ex);
      if (lane == 0 && ex) atomicAdd(&extra, ex);
    } else {
      if (q.sl == 0 && tid == 0) atomicOr(&c.header[2], 64u);
      const unsigned long long hs = g.seed_anchor ^ ((unsigned long long)q.h << 40);
      unsigned long long prefix = bin << 52, pmask = 0xfffull << 52;
      int remaining = need;
      for (int dgt = 0; dgt < 5; ++dgt) {
        const int shift = dgt < 4 ? 40 - 12 * dgt : 0;
        const int nbin = dgt < 4 ? SEL_NBIN : 16;
        for (int i = tid; i < nbin; i += blockDim.x) hist[i] = 0;
        __syncthreads();
        for (int t = tid; t < q.P; t += blockDim.x) {
          if (flag[t] == 1) continue;  // bin members may be taken meanwhile (2)
          const unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
          if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & (unsigned long long)(nbin - 1)], 1u);
        }
        __syncthreads();
        digit_pick(hist, nbin, remaining, false, tmp, pick);
        remaining -= pick[1];
        prefix |= (unsigned long long)pick[0] << shift;
        pmask |= (unsigned long long)(nbin - 1) << shift;
        __syncthreads();
      }
      // Positions in the bin with a key up to the threshold are taken:
      // counted in the earlier slices, flagged in this one.  Keys in the bin
      // mark exactly the positions left untaken by the earlier passes, so
      // the 2s other workgroups write meanwhile change nothing here.
      int ex = 0;
      for (int t = tid; t < q.t1; t += blockDim.x) {
        if (flag[t] == 1) continue;
        const unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
        if ((key & (0xfffull << 52)) == (bin << 52) && key <= prefix) {
          if (t < q.t0) ++ex;
          else flag[t] = 2;
        }
      }
      ex = wave_sum_i(ex);
      if (lane == 0 && ex) atomicAdd(&extra, ex);
    }
  }
  if (tid < 64) {
    int s = 0;
    const int nbefore = min(q.sl, (q.P + SEL_SLICE - 1) / SEL_SLICE);
    for (int i = lane; i < nbefore; i += 64) s += slc[i];
    s = wave_sum_i(s);
    if (lane == 0) basev = s;
  }
  __syncthreads();
  int base = basev + extra;
  // The slice's flags, all loaded before any is used (one round trip), then
  // the ranks of the flagged positions in position order: wave ballots per
  // round of 256 positions and one scan over (round, wave).
  uint8_t fl[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) fl[j] = flag[min(q.t0 + j * 256 + tid, max(q.t1 - 1, 0))];
  unsigned long long bal[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int t = q.t0 + j * 256 + tid;
    bal[j] = __ballot(t < q.t1 && fl[j] != 0);
    if (lane == 0) wc[j][wave] = __popcll(bal[j]);
  }
  __syncthreads();
  if (tid == 0) {
    int s = 0;
    for (int j = 0; j < NJ; ++j)
      for (int i = 0; i < 4; ++i) {
        wpre[j][i] = s;
        s += wc[j][i];
      }
    wtot = s;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int t = q.t0 + j * 256 + tid;
    const bool f = t < q.t1 && fl[j] != 0;
    const int r = base + wpre[j][wave] + __popcll(bal[j] & ((1ull << lane) - 1ull));
    if (f && r < k - W) {
      anc[r] = t;
      rank[t] = r;
    }
  }
  base += wtot;
  const bool tail = q.P > 0 ? (q.t0 <= q.P - 1 && q.P - 1 < q.t0 + SEL_SLICE) : q.sl == 0;
  if (tail) {
    if (tid == 0 && base + W != k) atomicOr(&c.header[2], 2u);
    for (int i = tid; i < W; i += blockDim.x) {
      anc[k - W + i] = q.P + i;
      rank[q.P + i] = k - W + i;
    }
  }
}

// An anchor override replaces the selection: validated (ascending, inside
// [0, S), the window last) and copied; the marks were reset by k_sel_pool.
__global__ __launch_bounds__(256) void k_sel_override(Geo g, Ws w, Cache c, const int32_t* ovr) {
  const int bh = blockIdx.x, b = bh / g.H, h = bh % g.H;
  const int S = g.S[b], W = g.W, P = S - W, k = g.k[b];
  const size_t so = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  int32_t* rank = w.rank + so;
  int32_t* anc = c.anc_pos + (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int32_t* o = ovr + (size_t)g.prefK[b] * g.H + (size_t)h * k;
  bool bad = false;
  for (int a = threadIdx.x; a < k; a += blockDim.x) {
    const int p = o[a];
    const bool ok = p >= 0 && p < S && (a == 0 || o[a - 1] < p) && (a < k - W || p == P + (a - (k - W)));
    if (!ok) bad = true;
    anc[a] = p;
    if (p >= 0 && p < S) rank[p] = a;
  }
  if (bad) atomicOr(&c.header[2], 1u);
}

template <int DT>
__global__ __launch_bounds__(256) void k_anchor_prep(Geo g, Ws w, Cache c, const void* Kin, const void* Vin,
                                                     const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int PER = 16 / sizeof(E), CPR = AKV_D / PER;
  constexpr int LD = AKV_D + (DT ? 8 : 4);  // LDS row stride (16-byte aligned rows)
  __shared__ __align__(16) E AK[64 * LD];
  __shared__ __align__(16) E AV[64 * LD];
  int idx = blockIdx.x;
  int b = 0;
  for (; b < g.B; ++b) {
    int n = g.H * ((g.k[b] + 63) / 64);
    if (idx < n) break;
    idx -= n;
  }
  const int k = g.k[b], S = g.S[b], D = AKV_D, m = g.m;
  const int nch = (k + 63) / 64;
  const int h = idx / nch, a0 = (idx % nch) * 64;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int32_t* anc = c.anc_pos + ko;
  const int na = min(64, k - a0);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Copy the 64 anchor rows in 16-byte chunks and stage them in LDS (rows
  // past na are zero).
#pragma unroll
  for (int i = threadIdx.x; i < 64 * CPR; i += 256) {
    const int a = i / CPR, col = (i % CPR) * PER;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (a < na) {
      const int p = min(max(anc[a0 + a], 0), S - 1);
      kv = *(const uint4*)((const E*)Kin + xoff + (size_t)p * D + col);
      vv = *(const uint4*)((const E*)Vin + xoff + (size_t)p * D + col);
      *(uint4*)((E*)c.ancK + (ko + a0 + a) * D + col) = kv;
      *(uint4*)((E*)c.ancV + (ko + a0 + a) * D + col) = vv;
    }
    *(uint4*)&AK[a * LD + col] = kv;
    *(uint4*)&AV[a * LD + col] = vv;
  }
  __syncthreads();
  // Canonical squared norms (fp64, sequential) and fp32 inverse norms.
  if (threadIdx.x < 2 * na) {
    const int a = threadIdx.x % na, side = threadIdx.x / na;
    const E* row = &(side ? AV : AK)[a * LD];
    double n = dot64_seq<DT>(row, row, D);
    (side ? c.nrmV : c.nrmK)[ko + a0 + a] = n;
    (side ? c.invV : c.invK)[ko + a0 + a] = n > 0.0 ? (float)(1.0 / sqrt(n)) : 0.0f;
  }
  // QA[a][w] = q_w . abar^K_a (fp32 accumulation of exact products), anchor-
  // major so that a token reads the m values of its anchor contiguously: one
  // 32x32 MFMA tile (anchors x observation rows) per wave and step.
  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D;
  float* QA = w.QA + ko * m;
  const int nrb = (m + 31) / 32, nat = (na + 31) / 32;
  for (int ti = wave; ti < nat * nrb; ti += 4) {
    const int at = ti % nat, wt = ti / nat;
    const int wr = wt * 32 + (lane & 31);
    const E* qrow = Q + (size_t)min(wr, m - 1) * D;
    f32x16 acc = {};
#pragma unroll
    for (int s = 0; s < AKV_D / M::KS; ++s) {
      const int k0 = kofs(M::KS, s, lane);
      acc = M::mma(M::load_lds(&AK[(at * 32 + (lane & 31)) * LD], k0), M::load(qrow, k0), acc);
    }
    if (wr < m) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int a = at * 32 + crow(e, lane);
        if (a < na) QA[(size_t)(a0 + a) * m + wr] = acc[e];
      }
    }
  }
}

hipError_t launch_select(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* Kobs, const void* V,
                         const void* Q, const int32_t* ovr, hipStream_t st) {
  int nblk = 0, nsel = 0;
  for (int b = 0; b < g.B; ++b) {
    nblk += g.H * ((g.k[b] + 63) / 64);
    nsel += g.H * ((g.S[b] + SEL_SLICE - 1) / SEL_SLICE);
  }
  const int nbh = g.B * g.H;
  launch("k_sel_pool", k_sel_pool, dim3(nsel), dim3(256), 0, st, g, w, ovr ? 1 : 0);
  if (ovr) {
    launch("k_sel_override", k_sel_override, dim3(nbh), dim3(256), 0, st, g, w, c, ovr);
  } else {
    launch("k_sel_cand", k_sel_cand, dim3(nsel), dim3(256), 0, st, g, w);
    launch("k_sel_class", k_sel_class, dim3(nsel), dim3(256), 0, st, g, w);
    if (g.dtype == 1) launch("k_sel_band", k_sel_band<1>, dim3(nbh * SEL_BAND_MAX), dim3(256), 0, st, g, w, Kobs, Q);
    else launch("k_sel_band", k_sel_band<0>, dim3(nbh * SEL_BAND_MAX), dim3(256), 0, st, g, w, Kobs, Q);
    launch("k_sel_rhist", k_sel_rhist, dim3(nsel), dim3(256), 0, st, g, w, c);
    launch("k_sel_rcand", k_sel_rcand, dim3(nsel), dim3(256), 0, st, g, w);
    launch("k_sel_list", k_sel_list, dim3(nsel), dim3(256), 0, st, g, w, c);
  }
  if (g.dtype == 1) {
    launch("k_anchor_prep", k_anchor_prep<1>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V, Q);
  } else {
    launch("k_anchor_prep", k_anchor_prep<0>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V, Q);
  }
  return hipGetLastError();
}

}  // namespace akv
