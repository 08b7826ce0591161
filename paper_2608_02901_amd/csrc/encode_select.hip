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
constexpr int SEL_BAND_MAX = 256;

// fp64 pooled selector score of position t (t < P, so every observation row
// sees it): (1/kappa) sum_{|d| <= kappa/2, 0 <= t+d < P} (1/m) sum_w
// exp(dot64(q_w, k_{t+d}) / sqrt(D) - M_w) / Z_w, with the row statistics of
// the observation pass.  One wave; lane l takes rows l, l + 64, ...; the
// lane partials are summed in a fixed order.
template <int DT>
__device__ double pooled64(const Geo& g, const typename Elem<DT>::T* X, const typename Elem<DT>::T* Q,
                           const float* oM, const double* oiZ, int t, int P, int m) {
  const int lane = threadIdx.x & 63, half = g.kappa / 2;
  double acc = 0.0;
  for (int wr = lane; wr < m; wr += 64) {
    const auto* q = Q + (size_t)wr * AKV_D;
    double rs = 0.0;
    for (int d = -half; d <= half; ++d) {
      const int u = t + d;
      if (u < 0 || u >= P) continue;
      const double l = dot64_seq<DT>(q, X + (size_t)u * AKV_D, AKV_D) / sqrt((double)AKV_D);
      rs += exp(l - (double)oM[wr]) * oiZ[wr];
    }
    acc += rs;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  return acc / (double)m / (double)g.kappa;
}

template <int DT>
__global__ __launch_bounds__(1024) void k_select(Geo g, Ws w, Cache c, const int32_t* ovr, const void* Kin,
                                                 const void* Qin) {
  using E = typename Elem<DT>::T;
  __shared__ uint32_t hist[256];
  __shared__ int tmp[20];
  __shared__ unsigned long long bcast[2];
  __shared__ int band[SEL_BAND_MAX];
  __shared__ double bscore[SEL_BAND_MAX];
  __shared__ int nband, nabove;
  const int b = blockIdx.x / g.H, h = blockIdx.x % g.H;
  const int S = g.S[b], W = g.W, P = S - W, k = g.k[b];
  const size_t so = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  int32_t* rank = w.rank + so;
  uint8_t* flag = w.flag + so;
  const float* sc = w.sc + so;
  float* pooled = w.u + so;  // the utility buffer is free until the epilogue
  int32_t* anc = c.anc_pos + (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int tid = threadIdx.x, nt = blockDim.x;

  for (int t = tid; t < S; t += nt) {
    rank[t] = -1;
    flag[t] = 0;
  }
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

  // Average pooling of width kappa over [0, P), zero padded, divided by kappa.
  const int half = g.kappa / 2;
  for (int t = tid; t < P; t += nt) {
    float s = 0.0f;
    for (int d = -half; d <= half; ++d) {
      int u = t + d;
      if (u >= 0 && u < P) s += sc[u];
    }
    pooled[t] = s / (float)g.kappa;
  }
  __syncthreads();

  // Contiguous range of [0, P) owned by this thread (for ordered ranks).
  const int per = (P + nt - 1) / nt;
  const int lo = min(P, tid * per), hi = min(P, lo + per);

  // ---- top n_top by pooled score, ties to the lower position.
  const int ntop = g.ntop[b];
  if (ntop > 0) {
    uint32_t prefix = 0, pmask = 0;
    int remaining = ntop;
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      for (int i = tid; i < 256; i += nt) hist[i] = 0;
      __syncthreads();
      for (int t = tid; t < P; t += nt) {
        uint32_t u = __float_as_uint(pooled[t]);
        if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        int cum = 0, dg = 255;
        for (; dg > 0; --dg) {
          if (cum + (int)hist[dg] >= remaining) break;
          cum += hist[dg];
        }
        remaining -= cum;
        bcast[0] = ((unsigned long long)dg << 32) | (unsigned)remaining;
      }
      __syncthreads();
      const uint32_t dg = (uint32_t)(bcast[0] >> 32);
      remaining = (int)(bcast[0] & 0xffffffffu);
      prefix |= dg << shift;
      pmask |= 255u << shift;
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
    for (int t = tid; t < P; t += nt) {
      const float v = pooled[t];
      if (v > bhi) {
        atomicAdd(&nabove, 1);
      } else if (v >= blo) {
        const int i = atomicAdd(&nband, 1);
        if (i < SEL_BAND_MAX) band[i] = t;
      }
    }
    __syncthreads();
    const int nb = nband;
    if (nb <= SEL_BAND_MAX) {
      const E* X = (const E*)Kin + ((size_t)g.prefS[b] * g.H + (size_t)h * S) * AKV_D;
      const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * AKV_D;
      const float* oM = w.oM + (size_t)(b * g.H + h) * g.m;
      const double* oiZ = w.oiZ64 + (size_t)(b * g.H + h) * g.m;
      for (int i = tid >> 6; i < nb; i += nt >> 6) {
        const double v = pooled64<DT>(g, X, Q, oM, oiZ, band[i], P, g.m);
        if ((tid & 63) == 0) bscore[i] = v;
      }
      __syncthreads();
      const int need = ntop - nabove;
      for (int t = tid; t < P; t += nt) flag[t] = pooled[t] > bhi ? 1 : 0;
      __syncthreads();
      for (int i = tid; i < nb; i += nt) {
        int r = 0;
        for (int j = 0; j < nb; ++j)
          r += bscore[j] > bscore[i] || (bscore[j] == bscore[i] && band[j] < band[i]);
        if (r < need) flag[band[i]] = 1;
      }
      __syncthreads();
    } else {
    if (tid == 0) atomicOr(&c.header[2], 32u);  // band overflow: the fp32 order decides
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
    __syncthreads();
    }
  }

  // ---- uniform share: the n_rand unflagged positions with the smallest hash.
  const int nrand = g.nrand[b];
  const unsigned long long hs = g.seed_anchor ^ ((unsigned long long)h << 40);
  if (nrand > 0) {
    unsigned long long prefix = 0, pmask = 0;
    int remaining = nrand;
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      for (int i = tid; i < 256; i += nt) hist[i] = 0;
      __syncthreads();
      for (int t = tid; t < P; t += nt) {
        if (flag[t]) continue;
        unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255ull], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        int cum = 0, dg = 0;
        for (; dg < 255; ++dg) {
          if (cum + (int)hist[dg] >= remaining) break;
          cum += hist[dg];
        }
        remaining -= cum;
        bcast[1] = ((unsigned long long)dg << 32) | (unsigned)remaining;
      }
      __syncthreads();
      const unsigned long long dg = bcast[1] >> 32;
      remaining = (int)(bcast[1] & 0xffffffffu);
      prefix |= dg << shift;
      pmask |= 255ull << shift;
      __syncthreads();
    }
    // Keys are distinct (SplitMix64 is a bijection), so exactly the keys
    // <= prefix are taken.
    for (int t = tid; t < P; t += nt) {
      if (flag[t]) continue;
      unsigned long long key = splitmix64(hs ^ (unsigned long long)t);
      if (key <= prefix) flag[t] = 2;
    }
    __syncthreads();
  }

  // ---- ascending anchor list: flagged positions of [0, P), then the window.
  int cnt = 0;
  for (int t = lo; t < hi; ++t) cnt += flag[t] != 0;
  int tot;
  int at = block_excl_scan(cnt, tmp, tot);
  for (int t = lo; t < hi; ++t)
    if (flag[t]) {
      if (at < k - W) {
        anc[at] = t;
        rank[t] = at;
      }
      ++at;
    }
  for (int i = tid; i < W; i += nt) {
    anc[k - W + i] = P + i;
    rank[P + i] = k - W + i;
  }
  if (tid == 0 && tot + W != k) atomicOr(&c.header[2], 2u);
}

template <int DT>
__global__ __launch_bounds__(256) void k_anchor_prep(Geo g, Ws w, Cache c, const void* Kin, const void* Vin,
                                                     const void* Qin) {
  using E = typename Elem<DT>::T;
  __shared__ float AK[64][AKV_D + 1];
  int idx = blockIdx.x;
  int b = 0;
  for (; b < g.B; ++b) {
    int n = g.H * ((g.k[b] + 63) / 64);
    if (idx < n) break;
    idx -= n;
  }
  const int k = g.k[b], S = g.S[b], D = g.D, m = g.m;
  const int nch = (k + 63) / 64;
  const int h = idx / nch, a0 = (idx % nch) * 64;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int32_t* anc = c.anc_pos + ko;
  const int na = min(64, k - a0);
  // Copy rows and stage the keys in LDS as fp32.
  for (int i = threadIdx.x; i < na * D; i += blockDim.x) {
    int a = i / D, d = i % D;
    int p = anc[a0 + a];
    p = min(max(p, 0), S - 1);
    E kv = ((const E*)Kin)[xoff + (size_t)p * D + d];
    E vv = ((const E*)Vin)[xoff + (size_t)p * D + d];
    ((E*)c.ancK)[(ko + a0 + a) * D + d] = kv;
    ((E*)c.ancV)[(ko + a0 + a) * D + d] = vv;
    AK[a][d] = Elem<DT>::get(&kv, 0);
  }
  __syncthreads();
  // Canonical squared norms (fp64, sequential) and fp32 inverse norms.
  if (threadIdx.x < 2 * na) {
    const int a = threadIdx.x % na, side = threadIdx.x / na;
    const E* row = (const E*)(side ? c.ancV : c.ancK) + (ko + a0 + a) * D;
    double n = dot64_seq<DT>(row, row, D);
    (side ? c.nrmV : c.nrmK)[ko + a0 + a] = n;
    (side ? c.invV : c.invK)[ko + a0 + a] = n > 0.0 ? (float)(1.0 / sqrt(n)) : 0.0f;
  }
  // QA[a][w] = q_w . abar^K_a (raw dot, fp32), anchor-major so that a token
  // reads the m values of its anchor contiguously.
  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D;
  float* QA = w.QA + ko * m;
  for (int i = threadIdx.x; i < m * na; i += blockDim.x) {
    int a = i / m, wr = i % m;
    const E* q = Q + (size_t)wr * D;
    float s = 0.0f;
    for (int d = 0; d < D; ++d) s = fmaf(Elem<DT>::get(q, d), AK[a][d], s);
    QA[(size_t)(a0 + a) * m + wr] = s;
  }
}

hipError_t launch_select(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, const void* Q,
                         const int32_t* ovr, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * ((g.k[b] + 63) / 64);
  if (g.dtype == 1) {
    AKV_TIMED("k_select", st, k_select<1><<<g.B * g.H, 1024, 0, st>>>(g, w, c, ovr, K, Q));
  } else {
    AKV_TIMED("k_select", st, k_select<0><<<g.B * g.H, 1024, 0, st>>>(g, w, c, ovr, K, Q));
  }
  if (g.dtype == 1) {
    AKV_TIMED("k_anchor_prep", st, k_anchor_prep<1><<<nblk, 256, 0, st>>>(g, w, c, K, V, Q));
  } else {
    AKV_TIMED("k_anchor_prep", st, k_anchor_prep<0><<<nblk, 256, 0, st>>>(g, w, c, K, V, Q));
  }
  return hipGetLastError();
}

}  // namespace akv
