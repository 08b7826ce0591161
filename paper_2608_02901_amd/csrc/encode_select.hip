// Anchor selection (Sec. 3.2 "Anchor selection"; App. A.2 Eq. selector-score;
// Algorithm 1, first step) and anchor preparation.
//   k_select      : one workgroup per (request, head).  Average-pools the
//                   observation score over kappa positions (zero padding,
//                   divided by kappa), takes the floor(rho (k - W)) best pooled
//                   positions of [0, S - W) (ties to the lower position) by an
//                   exact radix select on the fp32 bits, samples the rest of the
//                   non-window budget uniformly without replacement (the
//                   positions with the smallest SplitMix64 hash), adds the
//                   window and writes the ascending anchor list and the
//                   position -> anchor-index map.
//   k_anchor_prep : copies anchor keys/values into the cache, their canonical
//                   fp64 squared norms and fp32 inverse norms, and the table
//                   QA[a][w] = q_w . abar^K_a used by the key utilities.
#include "akv_common.h"

namespace akv {

// Exclusive scan of one int per thread over a 1024-thread block.
__device__ inline int block_excl_scan(int v, int* tmp /* >= 16 ints */, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) tmp[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int i = 0; i < nw; ++i) {
      int t = tmp[i];
      tmp[i] = s;
      s += t;
    }
    tmp[nw] = s;
  }
  __syncthreads();
  int r = x - v + tmp[wave];
  total = tmp[nw];
  __syncthreads();
  return r;
}

// Positions whose fp32 pooled score lies within SEL_BAND (relative) of the
// cut are re-scored in fp64 (at most SEL_BAND_MAX of them).  The fp32 score's
// error is below 1e-4 relative: fp32 accumulation of 128 exact bf16 products
// (at most 128 * 2^-24 * sum |q_i k_i| / sqrt(D) on a logit), fp32 exp and
// sums; the band is ten times wider.  The fp64 scores use exact fp64 logits
// and the row sums Z_w of the observation pass (fp64 sums of fp32-logit
// exponentials, ~1e-9 relative), so they match the canonical fp64 definition
// to far better than the gaps between real scores.
constexpr float SEL_BAND = 1e-3f;

// fp64 pooled selector score of band member i of (request b, head h), one
// workgroup per member (k_sel_band): (1/kappa) sum_{|d| <= kappa/2,
// 0 <= t+d < P} (1/m) sum_w exp(dot64(q_w, k_{t+d}) / sqrt(D) - M_w) / Z_w,
// with the row statistics of the observation pass.  The m query rows and the
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
  const int nb = w.sstate[bh * 4 + 3];
  if (i >= nb) return;  // also an overflowed band (nb < 0)
  const int S = g.S[b], P = S - g.W, m = g.m;
  const int tid = threadIdx.x, nt = blockDim.x, half = g.kappa / 2, nk = 2 * half + 1;
  const int t = w.sband[(size_t)bh * SEL_BAND_MAX + i];
  const E* X = (const E*)Kin + ((size_t)g.prefS[b] * g.H + (size_t)h * S) * AKV_D;
  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * AKV_D;
  const float* oM = w.oM + (size_t)bh * m;
  const double* oiZ = w.oiZ64 + (size_t)bh * m;
  const double isd = 1.0 / sqrt((double)AKV_D);
  const bool qst = (size_t)m * AKV_D * sizeof(E) <= SEL_QLDS;
  const bool kst = (size_t)nk * AKV_D * sizeof(E) <= SEL_KLDS;
  E* qs = (E*)qlds;
  E* ks = (E*)klds;
  if (qst)
    for (int c = tid; c < m * NCH; c += nt) ((uint4*)qs)[c] = ((const uint4*)Q)[c];
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
      rs += exp(l - (double)oM[wr]) * oiZ[wr];
    }
    acc += rs;
  }
  // rows summed per thread (rows tid, tid + nt, ...), then over threads in order
  part[tid] = acc;
  __syncthreads();
  if (tid == 0) {
    double tot = 0.0;
    for (int r = 0; r < nt; ++r) tot += part[r];
    w.sbscore[(size_t)bh * SEL_BAND_MAX + i] = tot / (double)m / (double)g.kappa;
  }
}

// Radix digit search over a 4096-bin histogram: the bin where the running
// count (from the top when `desc`, else from the bottom) reaches `need`.
// Writes (bin, count before it) to out[0..1].  Whole workgroup.
__device__ inline void digit_pick(const uint32_t* hist, int nbin, int need, bool desc, int* tmp, int* out) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int per = (nbin + nt - 1) / nt;
  int loc = 0;
  for (int i = 0; i < per; ++i) {
    const int bin = tid * per + i;
    if (bin < nbin) loc += (int)hist[desc ? nbin - 1 - bin : bin];
  }
  int tot;
  const int before = block_excl_scan(loc, tmp, tot);
  int run = before;
  for (int i = 0; i < per; ++i) {
    const int bin = tid * per + i;
    if (bin >= nbin) break;
    const int c = (int)hist[desc ? nbin - 1 - bin : bin];
    if (run < need && run + c >= need) {
      out[0] = desc ? nbin - 1 - bin : bin;
      out[1] = run;
    }
    run += c;
  }
  __syncthreads();
}

constexpr int SEL_NBIN = 4096;  // 12-bit radix digits
constexpr int SEL_TILE = 3840;  // pooled positions per LDS tile (tile + halo fit the histogram)
constexpr int SEL_HALO = 254;   // 2 * (kappa / 2) for kappa <= 255
constexpr int SEL_CAND = 1024;  // hash candidates kept in the last digit's bin
constexpr int SEL_U = 8;        // elements per thread per batch (independent loads)

// Passes over [0, n) visit t = t0 + u * nt (u < SEL_U) per batch: coalesced
// across lanes, SEL_U independent loads in flight per thread.
template <typename F>
__device__ inline void sel_batches(int n, F&& body) {
  for (int t0 = threadIdx.x; t0 < n; t0 += SEL_U * blockDim.x) body(t0);
}

// Selection, first half (one workgroup per request and head): marks reset,
// pooled scores, the exact n_top-th largest pooled fp32 value, the positions
// clearly above it (taken) and the band around it, whose members k_sel_band
// re-scores in fp64.  An anchor override replaces the selection.
template <int DT>
__global__ __launch_bounds__(1024) void k_sel_top(Geo g, Ws w, Cache c, const int32_t* ovr) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[20];
  __shared__ int pick[2];
  __shared__ int nband, nabove;
  const int bh = blockIdx.x, b = bh / g.H, h = bh % g.H;
  const int S = g.S[b], W = g.W, P = S - W, k = g.k[b];
  const size_t so = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  int32_t* rank = w.rank + so;
  uint8_t* flag = w.flag + so;
  const float* sc = w.sc + so;
  float* pooled = w.u + so;  // the utility buffer is free until the epilogue
  int32_t* anc = c.anc_pos + (size_t)g.prefK[b] * g.H + (size_t)h * k;
  int32_t* st = w.sstate + bh * 4;  // prefix, remaining, nabove, nband (-1: none / overflow)
  const int tid = threadIdx.x, nt = blockDim.x;

  sel_batches(S, [&](int t0) {
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) {
      const int t = t0 + u * nt;
      if (t < S) {
        rank[t] = -1;
        flag[t] = 0;
      }
    }
  });
  if (tid == 0) st[3] = -1;
  __syncthreads();
  if (ovr) {
    const int32_t* o = ovr + (size_t)g.prefK[b] * g.H + (size_t)h * k;
    bool bad = false;
    for (int a = tid; a < k; a += nt) {
      int p = o[a];
      bool ok = p >= 0 && p < S && (a == 0 || o[a - 1] < p) && (a < k - W || p == P + (a - (k - W)));
      if (!ok) bad = true;
      anc[a] = p;
      if (p >= 0 && p < S) rank[p] = a;
    }
    if (bad) atomicOr(&c.header[2], 1u);
    return;
  }

  // Average pooling of width kappa over [0, P), zero padded, divided by kappa
  // (terms added in offset order, from -kappa/2), in tiles of SEL_TILE
  // positions staged through LDS with their halo; the next tile's values are
  // loaded while the current one is pooled.
  const int half = g.kappa / 2;
  {
    float* stile = (float*)hist;  // the histogram is not in use yet
    constexpr int TV = (SEL_TILE + SEL_HALO + 1023) / 1024;  // staged values per thread
    float nxt[TV];
    auto load_tile = [&](int c0) {
#pragma unroll
      for (int i = 0; i < TV; ++i) {
        const int j = tid + i * nt, u = c0 - half + j;
        nxt[i] = (j < SEL_TILE + 2 * half && u >= 0 && u < P) ? sc[u] : 0.0f;
      }
    };
    load_tile(0);
    for (int c0 = 0; c0 < P; c0 += SEL_TILE) {
      __syncthreads();
#pragma unroll
      for (int i = 0; i < TV; ++i) {
        const int j = tid + i * nt;
        if (j < SEL_TILE + 2 * half) stile[j] = nxt[i];
      }
      __syncthreads();
      if (c0 + SEL_TILE < P) load_tile(c0 + SEL_TILE);
      for (int t = tid; t < SEL_TILE && c0 + t < P; t += nt) {
        float s = 0.0f;
        for (int d = 0; d <= 2 * half; ++d) s += stile[t + d];
        pooled[c0 + t] = s / (float)g.kappa;
      }
    }
  }
  __syncthreads();

  // ---- top n_top by pooled score, ties to the lower position: radix select
  // on the fp32 bits (non-negative scores order as their bits), digits
  // [31:20], [19:8], [7:0].
  const int ntop = g.ntop[b];
  if (ntop <= 0) return;
  uint32_t prefix = 0, pmask = 0;
  int remaining = ntop;
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 20 : (pass == 1 ? 8 : 0);
    const int nbin = pass == 2 ? 256 : SEL_NBIN;
    for (int i = tid; i < nbin; i += nt) hist[i] = 0;
    __syncthreads();
    sel_batches(P, [&](int t0) {
      uint32_t v[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) v[u] = t0 + u * nt < P ? __float_as_uint(pooled[t0 + u * nt]) : 0u;
#pragma unroll
      for (int u = 0; u < SEL_U; ++u)
        if (t0 + u * nt < P && (v[u] & pmask) == prefix) atomicAdd(&hist[(v[u] >> shift) & (nbin - 1)], 1u);
    });
    __syncthreads();
    digit_pick(hist, nbin, remaining, true, tmp, pick);
    remaining -= pick[1];
    prefix |= (uint32_t)pick[0] << shift;
    pmask |= (uint32_t)(nbin - 1) << shift;
    __syncthreads();
  }
  // prefix is the bit pattern of the n_top-th largest fp32 score.  Scores
  // clearly above the band are taken; inside the band the decision uses the
  // fp64 scores (ties to the lower position).
  const float cut = __uint_as_float(prefix);
  const float bhi = cut * (1.0f + SEL_BAND), blo = cut * (1.0f - SEL_BAND);
  if (tid == 0) {
    nband = 0;
    nabove = 0;
  }
  __syncthreads();
  int32_t* band = w.sband + (size_t)bh * SEL_BAND_MAX;
  sel_batches(P, [&](int t0) {
    float v[SEL_U];
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) v[u] = t0 + u * nt < P ? pooled[t0 + u * nt] : -1.0f;
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) {
      const int t = t0 + u * nt;
      if (t >= P) continue;
      if (v[u] > bhi) {
        atomicAdd(&nabove, 1);
        flag[t] = 1;
      } else if (v[u] >= blo) {
        const int i = atomicAdd(&nband, 1);
        if (i < SEL_BAND_MAX) band[i] = t;
      }
    }
  });
  __syncthreads();
  const int nb = nband;
  if (nb > SEL_BAND_MAX) {
    // Band overflow: the fp32 order decides (ties to the lower position).
    if (tid == 0) atomicOr(&c.header[2], 32u);
    const int per = (P + nt - 1) / nt;
    const int lo = min(P, tid * per), hi = min(P, lo + per);
    for (int t = lo; t < hi; ++t) flag[t] = 0;
    __syncthreads();
    int eq = 0;
    for (int t = lo; t < hi; ++t) eq += (__float_as_uint(pooled[t]) == prefix);
    int tot;
    int before = block_excl_scan(eq, tmp, tot);
    for (int t = lo; t < hi; ++t) {
      uint32_t u = __float_as_uint(pooled[t]);
      if (u > prefix) {
        flag[t] = 1;
      } else if (u == prefix) {
        if (before < remaining) flag[t] = 1;
        ++before;
      }
    }
  } else if (tid == 0) {
    st[0] = (int)prefix;
    st[1] = remaining;
    st[2] = nabove;
    st[3] = nb;
  }
}

// Selection, second half: the band members ranked by their fp64 scores, the
// uniform share (the n_rand unflagged positions with the smallest SplitMix64
// key: the top 12 bits locate the bin holding the n_rand-th smallest key, keys
// below it are taken, the keys inside it are ranked exactly; keys are
// distinct since SplitMix64 is a bijection), and the ascending anchor list
// with the position -> anchor-index map.
template <int DT>
__global__ __launch_bounds__(1024) void k_sel_rest(Geo g, Ws w, Cache c, const int32_t* ovr) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[20];
  __shared__ int pick[2];
  __shared__ unsigned long long ckey[SEL_CAND];
  __shared__ int cpos[SEL_CAND];
  __shared__ int ncand;
  __shared__ int cnts[SEL_U * 16];     // flags per (u, wave) of a batch (16 waves of 1024 threads)
  __shared__ int cpre[SEL_U * 16 + 1];  // their exclusive prefix, then the batch total
  if (ovr) return;
  const int bh = blockIdx.x, b = bh / g.H, h = bh % g.H;
  const int S = g.S[b], W = g.W, P = S - W, k = g.k[b];
  const size_t so = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  int32_t* rank = w.rank + so;
  uint8_t* flag = w.flag + so;
  int32_t* anc = c.anc_pos + (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int tid = threadIdx.x, nt = blockDim.x;

  const int nb = w.sstate[bh * 4 + 3];
  if (nb > 0) {
    const int need = g.ntop[b] - w.sstate[bh * 4 + 2];
    const int32_t* band = w.sband + (size_t)bh * SEL_BAND_MAX;
    const double* bscore = w.sbscore + (size_t)bh * SEL_BAND_MAX;
    for (int i = tid; i < nb; i += nt) {
      int r = 0;
      for (int j = 0; j < nb; ++j)
        r += bscore[j] > bscore[i] || (bscore[j] == bscore[i] && band[j] < band[i]);
      if (r < need) flag[band[i]] = 1;
    }
    __syncthreads();
  }

  const int nrand = g.nrand[b];
  const unsigned long long hs = g.seed_anchor ^ ((unsigned long long)h << 40);
  if (nrand > 0) {
    for (int i = tid; i < SEL_NBIN; i += nt) hist[i] = 0;
    if (tid == 0) ncand = 0;
    __syncthreads();
    sel_batches(P, [&](int t0) {
      uint8_t f[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) f[u] = t0 + u * nt < P ? flag[t0 + u * nt] : 1;
#pragma unroll
      for (int u = 0; u < SEL_U; ++u)
        if (!f[u]) atomicAdd(&hist[splitmix64(hs ^ (unsigned long long)(t0 + u * nt)) >> 52], 1u);
    });
    __syncthreads();
    digit_pick(hist, SEL_NBIN, nrand, false, tmp, pick);
    const unsigned long long bin = (unsigned long long)pick[0];
    const int need = nrand - pick[1];
    sel_batches(P, [&](int t0) {
      uint8_t f[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) f[u] = t0 + u * nt < P ? flag[t0 + u * nt] : 1;
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) {
        if (f[u]) continue;
        const int t = t0 + u * nt;
        const unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
        if ((key >> 52) < bin) {
          flag[t] = 2;
        } else if ((key >> 52) == bin) {
          const int i = atomicAdd(&ncand, 1);
          if (i < SEL_CAND) {
            ckey[i] = key;
            cpos[i] = t;
          }
        }
      }
    });
    __syncthreads();
    const int nc = ncand;
    if (nc <= SEL_CAND) {
      for (int i = tid; i < nc; i += nt) {
        int r = 0;
        for (int j = 0; j < nc; ++j) r += ckey[j] < ckey[i];
        if (r < need) flag[cpos[i]] = 2;
      }
    } else {
      // More candidates than the buffer holds (far from the expected P/4096):
      // finish the radix select on the remaining 52 bits (digits of 12, 12,
      // 12, 12 and 4 bits).
      if (tid == 0) atomicOr(&c.header[2], 64u);
      unsigned long long prefix = bin << 52, pmask = 0xfffull << 52;
      int remaining = need;
      for (int dgt = 0; dgt < 5; ++dgt) {
        const int shift = dgt < 4 ? 40 - 12 * dgt : 0;
        const int nbin = dgt < 4 ? SEL_NBIN : 16;
        for (int i = tid; i < nbin; i += nt) hist[i] = 0;
        __syncthreads();
        for (int t = tid; t < P; t += nt) {
          if (flag[t]) continue;
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
      for (int t = tid; t < P; t += nt) {
        if (flag[t]) continue;
        const unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
        if ((key & (0xfffull << 52)) == (bin << 52) && key <= prefix) flag[t] = 2;
      }
    }
    __syncthreads();
  }

  // ---- ascending anchor list: flagged positions of [0, P), then the window.
  // Batches of SEL_U x nt positions in (u, thread) order; a flag's rank is the
  // count before its batch plus the flags before it inside the batch (wave
  // ballots, then per-(u, wave) counts in LDS).
  {
    static_assert(SEL_U * 16 == 128, "two scan entries per lane of one wave");
    const int lane = tid & 63, wv = tid >> 6;
    int base = 0;
    for (int t0 = tid; t0 - tid < P; t0 += SEL_U * nt) {
      uint8_t f[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) f[u] = t0 + u * nt < P ? flag[t0 + u * nt] : 0;
      unsigned long long bal[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) {
        bal[u] = __ballot(f[u] != 0);
        if (lane == 0) cnts[u * 16 + wv] = __popcll(bal[u]);
      }
      __syncthreads();
      if (wv == 0) {  // exclusive scan of the (u, wave) counts, u-major
        const int c0 = cnts[2 * lane], c1 = cnts[2 * lane + 1];
        int x = c0 + c1;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(x, o, 64);
          if (lane >= o) x += y;
        }
        const int ex = x - c0 - c1;
        cpre[2 * lane] = ex;
        cpre[2 * lane + 1] = ex + c0;
        if (lane == 63) cpre[SEL_U * 16] = x;
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) {
        const int r = base + cpre[u * 16 + wv] + __popcll(bal[u] & ((1ull << lane) - 1ull));
        if (f[u] && r < k - W) {
          const int t = t0 + u * nt;
          anc[r] = t;
          rank[t] = r;
        }
      }
      base += cpre[SEL_U * 16];
      __syncthreads();
    }
    if (tid == 0 && base + W != k) atomicOr(&c.header[2], 2u);
  }
  for (int i = tid; i < W; i += nt) {
    anc[k - W + i] = P + i;
    rank[P + i] = k - W + i;
  }
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

hipError_t launch_select(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, const void* Q,
                         const int32_t* ovr, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * ((g.k[b] + 63) / 64);
  const int nbh = g.B * g.H;
  if (g.dtype == 1) {
    launch("k_select", k_sel_top<1>, dim3(nbh), dim3(1024), 0, st, g, w, c, ovr);
    if (!ovr) launch("k_sel_band", k_sel_band<1>, dim3(nbh * SEL_BAND_MAX), dim3(256), 0, st, g, w, K, Q);
    launch("k_sel_rest", k_sel_rest<1>, dim3(nbh), dim3(1024), 0, st, g, w, c, ovr);
  } else {
    launch("k_select", k_sel_top<0>, dim3(nbh), dim3(1024), 0, st, g, w, c, ovr);
    if (!ovr) launch("k_sel_band", k_sel_band<0>, dim3(nbh * SEL_BAND_MAX), dim3(256), 0, st, g, w, K, Q);
    launch("k_sel_rest", k_sel_rest<0>, dim3(nbh), dim3(1024), 0, st, g, w, c, ovr);
  }
  if (g.dtype == 1) {
    launch("k_anchor_prep", k_anchor_prep<1>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V, Q);
  } else {
    launch("k_anchor_prep", k_anchor_prep<0>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V, Q);
  }
  return hipGetLastError();
}

}  // namespace akv
