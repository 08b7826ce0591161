// Observation-window pass of the compression (Sec. 3.2 anchor selection,
// App. A.2 Eq. selector-score; Sec. 3.3 needs the same attention for the
// utilities).  For every KV head the m = W * (Hq/H) observation rows (the
// queries of the last W positions, causal inside the window) attend to all
// positions:
//   k_obs_stats   : per half chunk (1024 tokens), MFMA logits q_w.k_t / sqrt(D)
//                   and the per-row running max and sum of exp;
//   k_obs_reduce  : merges the chunk statistics into M_w and 1/Z_w;
//   k_obs_pass    : recomputes the logits, alpha = exp(l - M)/Z and the SnapKV
//                   column score sc(t) = (1/m) sum_w alpha_wt.
// The outputs y_w and the fp64 row statistics come from the fp64 pass
// (encode_obs64.hip).
#include "akv_common.h"

namespace akv {

template <int DT> struct TileLD { static constexpr int v = AKV_D + (DT ? 8 : 4); };

// A tile of 32 token rows held in registers between its load and its LDS
// store (RPT 16-byte chunks per thread), so the next tile's loads are in
// flight while the current tile is processed.
template <int DT>
struct RowTile {
  using E = typename Elem<DT>::T;
  static constexpr int PER = 16 / sizeof(E), CPR = AKV_D / PER, RPT = 32 * CPR / 256;
  uint4 v[RPT];
  __device__ void load(const E* X, int t0, int S) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int c = threadIdx.x + 256 * i, r = c / CPR, col = (c % CPR) * PER;
      v[i] = t0 + r < S ? *(const uint4*)(X + (size_t)(t0 + r) * AKV_D + col) : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ void store(E* lds, int LD) const {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int c = threadIdx.x + 256 * i, r = c / CPR, col = (c % CPR) * PER;
      *(uint4*)(lds + r * LD + col) = v[i];
    }
  }
};

// Query row w of KV head h (rows w = jj*W + i are contiguous in [Hq][W][D]).
template <int DT>
__device__ inline const typename Elem<DT>::T* qrows(const Geo& g, const void* Qin, int b, int h) {
  return (const typename Elem<DT>::T*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * g.D;
}

// Last position observation row wr attends to (the rows are the queries of
// positions P .. P+W-1, causal inside the window); -1 for padding rows.
__device__ inline int obs_limit(int wr, int m, int P, int W) { return wr < m ? P + wr % W : -1; }

constexpr float NEG = -1e30f;

template <int CTRL>
__device__ inline float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Sum of v[e] over the 16 lanes of each DPP row: four exchanges (row mirror,
// half-row mirror, quad reversal, quad swap) in which a lane keeps half of its
// entries and adds the partner's copy of them; lane l ends with the row sum of
// entry l & 15.
__device__ inline float row_reduce_scatter16(const float (&v)[16], int lane) {
  float a[8], b[4], c[2];
  const bool s3 = lane & 8, s2 = lane & 4, s1 = lane & 2, s0 = lane & 1;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (s3 ? v[8 + i] : v[i]) + dpp_mov<0x140>(s3 ? v[i] : v[8 + i]);
#pragma unroll
  for (int i = 0; i < 4; ++i) b[i] = (s2 ? a[4 + i] : a[i]) + dpp_mov<0x141>(s2 ? a[i] : a[4 + i]);
#pragma unroll
  for (int i = 0; i < 2; ++i) c[i] = (s1 ? b[2 + i] : b[i]) + dpp_mov<0x1B>(s1 ? b[i] : b[2 + i]);
  return (s0 ? c[1] : c[0]) + dpp_mov<0xB1>(s0 ? c[0] : c[1]);
}

// R = row blocks of 32 observation rows per wave (4 waves cover 128 R rows).
template <int DT, int R>
__global__ __launch_bounds__(256) void k_obs_stats(Geo g, Ws w, const void* Kin, const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = TileLD<DT>::v;
  __shared__ __align__(16) E KT[2][32 * LD];  // double-buffered key tile
  int idx = blockIdx.x >> 1;
  const int hs = blockIdx.x & 1;  // half of the chunk (OBS_CHUNK / 2 tokens)
  const int b = locate(g, OBS_CHUNK, 1, idx);
  const int S = g.S[b], P = S - g.W, D = g.D, m = g.m;
  const int nch = (S + OBS_CHUNK - 1) / OBS_CHUNK;
  const int h = idx / nch, ch = idx % nch;
  const E* X = (const E*)Kin + ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* Q = qrows<DT>(g, Qin, b, h);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (m + 31) / 32;
  const float isd = 1.0f / sqrtf((float)D);
  // Running max (fp32 logits) and sum of exp in fp64 of the lane's row over
  // its tokens; the max moves at most once per tile and then rescales the sum
  // by an fp64 exp, so the sum keeps ~1e-9 relative accuracy (the anchor
  // selection re-scores near-ties against it).
  float mx[R];
  double sm[R];
  int lim[R];
  constexpr int NKS = AKV_D / M::KS;
  typename M::frag qf[R][NKS];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    mx[r] = NEG;
    sm[r] = 0.0;
    const int wr = (wave + 4 * r) * 32 + (lane & 31);
    lim[r] = obs_limit(wr, m, P, g.W);
    const int arow = min(wr, m - 1);
#pragma unroll
    for (int s = 0; s < NKS; ++s) qf[r][s] = M::load(Q + (size_t)arow * D, kofs(M::KS, s, lane));
  }
  const int tb = ch * OBS_CHUNK + hs * (OBS_CHUNK / 2), te = min(S, tb + OBS_CHUNK / 2);
  // Tile it sits in KT[it & 1]; the tile after it is stored into the other
  // buffer right after the barrier that ends the reads of tile it - 1, so
  // one barrier per tile suffices.
  RowTile<DT> kt;
  kt.load(X, tb, S);
  kt.store(KT[0], LD);
  if (tb + 32 < te) kt.load(X, tb + 32, S);
  int it = 0;
  for (int t0 = tb; t0 < te; t0 += 32, ++it) {
    const int cb = it & 1;
    __syncthreads();
    if (t0 + 32 < te) kt.store(KT[cb ^ 1], LD);
    if (t0 + 64 < te) kt.load(X, t0 + 64, S);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= nrb) break;
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        auto kb = M::load_lds(&KT[cb][(lane & 31) * LD], kofs(M::KS, s, lane));
        acc = M::mma(kb, qf[r][s], acc);
      }
      float l[16];
      float tm = NEG;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        l[e] = t0 + crow(e, lane) <= lim[r] ? acc[e] * isd : NEG;
        tm = fmaxf(tm, l[e]);
      }
      if (tm > mx[r]) {
        sm[r] *= exp((double)mx[r] - (double)tm);
        mx[r] = tm;
      }
      double p[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) p[e] = l[e] > NEG ? (double)__expf(l[e] - mx[r]) : 0.0;
#pragma unroll
      for (int o = 8; o > 0; o >>= 1)
#pragma unroll
        for (int e = 0; e < o; ++e) p[e] += p[e + o];
      sm[r] += p[0];
    }
  }
  // Merge the two lanes (l, l + 32) that share each row.
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int rb = wave + 4 * r;
    if (rb >= nrb) break;
    const float a = mx[r], oa = __shfl_xor(a, 32, 64);
    const double s = sm[r], os = __shfl_xor(s, 32, 64);
    const float nm = fmaxf(a, oa);
    const double z = (a == nm ? s : s * exp((double)a - (double)nm)) + (oa == nm ? os : os * exp((double)oa - (double)nm));
    const int wr = rb * 32 + lane;
    if (lane < 32 && wr < m) {
      size_t o = ((size_t)(g.prefC[b] * g.H + h * nch + ch) * 2 + hs) * m + wr;
      w.opmax[o] = nm;
      w.opsum[o] = z;
    }
  }
}

// Row statistics from the chunk statistics: per workgroup 64 rows of one
// (request, head); the 16 waves take every 16th half-chunk entry, and their
// partial (max, sum) pairs are merged in LDS.
__global__ __launch_bounds__(1024) void k_obs_reduce(Geo g, Ws w) {
  constexpr int NP = 16;
  __shared__ float pm[NP][64];
  __shared__ double ps[NP][64];
  const int nrg = (g.m + 63) / 64;
  const int bh = blockIdx.x / nrg, b = bh / g.H, h = bh % g.H;
  const int lane = threadIdx.x & 63, part = threadIdx.x >> 6;
  const int wr = (blockIdx.x % nrg) * 64 + lane;
  const int nch = (g.S[b] + OBS_CHUNK - 1) / OBS_CHUNK;
  const int wc = min(wr, g.m - 1);
  const size_t base = ((size_t)(g.prefC[b] * g.H + h * nch)) * 2 * g.m + wc;
  float M = NEG;
  for (int c = part; c < 2 * nch; c += NP) M = fmaxf(M, w.opmax[base + (size_t)c * g.m]);
  double Z = 0.0;
  for (int c = part; c < 2 * nch; c += NP) {
    const float mc = w.opmax[base + (size_t)c * g.m];
    const double sc = w.opsum[base + (size_t)c * g.m];
    Z += mc == M ? sc : sc * exp((double)mc - (double)M);
  }
  pm[part][lane] = M;
  ps[part][lane] = Z;
  __syncthreads();
  if (part == 0 && wr < g.m) {
    float Mt = pm[0][lane];
    for (int p = 1; p < NP; ++p) Mt = fmaxf(Mt, pm[p][lane]);
    double Zt = 0.0;
    for (int p = 0; p < NP; ++p) {
      const float mp = pm[p][lane];
      if (mp == NEG) continue;  // a part without entries
      Zt += mp == Mt ? ps[p][lane] : ps[p][lane] * exp((double)mp - (double)Mt);
    }
    w.oM[(size_t)(b * g.H + h) * g.m + wr] = Mt;
    w.oiZ[(size_t)(b * g.H + h) * g.m + wr] = (float)(1.0 / Zt);
  }
}

template <int DT, int R>
__global__ __launch_bounds__(256) void k_obs_pass(Geo g, Ws w, const void* Kin, const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = TileLD<DT>::v;
  __shared__ __align__(16) E KT[2][32 * LD];  // double-buffered key tiles
  __shared__ float scw[2][4][32];
  int idx = blockIdx.x;
  const int b = locate(g, OBS_CHUNK, 1, idx);
  const int S = g.S[b], P = S - g.W, D = g.D, m = g.m;
  const int nch = (S + OBS_CHUNK - 1) / OBS_CHUNK;
  const int h = idx / nch, ch = idx % nch;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)Kin + xoff;
  const E* Q = qrows<DT>(g, Qin, b, h);
  const float* oM = w.oM + (size_t)(b * g.H + h) * m;
  const float* oiZ = w.oiZ + (size_t)(b * g.H + h) * m;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (m + 31) / 32;
  const float isd = 1.0f / sqrtf((float)D);
  // The lane's row of each row block: query fragments, row max, 1/Z and
  // causal limit stay in registers; the next key tile is loaded while the
  // current one is used.
  constexpr int NKS = AKV_D / M::KS;
  typename M::frag qf[R][NKS];
  float rmax[R], riz[R];
  int lim[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int wr = (wave + 4 * r) * 32 + (lane & 31);
    const int arow = min(wr, m - 1);
    lim[r] = obs_limit(wr, m, P, g.W);
    rmax[r] = oM[arow];
    riz[r] = oiZ[arow];
#pragma unroll
    for (int s = 0; s < NKS; ++s) qf[r][s] = M::load(Q + (size_t)arow * D, kofs(M::KS, s, lane));
  }
  const int tb = ch * OBS_CHUNK, te = min(S, tb + OBS_CHUNK);
  float* sc = w.sc + (size_t)g.prefS[b] * g.H + (size_t)h * S;
  // Tile it sits in KT[it & 1] and leaves its column sums in scw[it & 1];
  // after the barrier that starts tile it, the next tile is stored into the
  // other buffer and the column sums of tile it - 1 are final.  One barrier
  // per tile.
  RowTile<DT> kt;
  kt.load(X, tb, S);
  kt.store(KT[0], LD);
  if (tb + 32 < te) kt.load(X, tb + 32, S);
  int it = 0;
  for (int t0 = tb; t0 < te; t0 += 32, ++it) {
    const int cb = it & 1;
    __syncthreads();
    if (it > 0 && threadIdx.x < 32 && t0 - 32 + threadIdx.x < S)
      sc[t0 - 32 + threadIdx.x] = (scw[cb ^ 1][0][threadIdx.x] + scw[cb ^ 1][1][threadIdx.x] +
                                   scw[cb ^ 1][2][threadIdx.x] + scw[cb ^ 1][3][threadIdx.x]) / (float)m;
    if (t0 + 32 < te) kt.store(KT[cb ^ 1], LD);
    if (t0 + 64 < te) kt.load(X, t0 + 64, S);
    float cs[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) cs[e] = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= nrb) break;
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        auto kb = M::load_lds(&KT[cb][(lane & 31) * LD], kofs(M::KS, s, lane));
        acc = M::mma(kb, qf[r][s], acc);
      }
      // alpha of the lane's row and tokens t0 + crow(e, lane).
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float a = __expf(acc[e] * isd - rmax[r]) * riz[r];
        cs[e] += t0 + crow(e, lane) <= lim[r] ? a : 0.0f;
      }
    }
    // Column sums over the wave's rows: the 16 lanes of a DPP row, then the
    // two rows of each half; lanes 0-15 and 32-47 hold tokens crow(l & 15, l).
    float csum = row_reduce_scatter16(cs, lane);
    csum += lane_xor<16>(csum);
    if ((lane & 16) == 0) scw[cb][wave][crow(lane & 15, lane)] = csum;
  }
  __syncthreads();
  {
    const int tl = tb + 32 * (it - 1);  // first token of the last tile
    const int cl = (it - 1) & 1;
    if (threadIdx.x < 32 && tl + threadIdx.x < S)
      sc[tl + threadIdx.x] = (scw[cl][0][threadIdx.x] + scw[cl][1][threadIdx.x] + scw[cl][2][threadIdx.x] +
                              scw[cl][3][threadIdx.x]) / (float)m;
  }
}

// ------------------------------------------------------------------ launchers
hipError_t launch_obs(const Geo& g, const Ws& w, const void* K, const void* V, const void* Q, hipStream_t st) {
  int nblk = g.H * g.prefC[g.B];
  const bool r2 = g.m > 128;  // 4 waves x 2 row blocks of 32 for up to 256 rows
  if (g.dtype == 1) {
    if (r2) launch("k_obs_stats", k_obs_stats<1, 2>, dim3(2 * nblk), dim3(256), 0, st, g, w, K, Q);
    else launch("k_obs_stats", k_obs_stats<1, 1>, dim3(2 * nblk), dim3(256), 0, st, g, w, K, Q);
  } else {
    if (r2) launch("k_obs_stats", k_obs_stats<0, 2>, dim3(2 * nblk), dim3(256), 0, st, g, w, K, Q);
    else launch("k_obs_stats", k_obs_stats<0, 1>, dim3(2 * nblk), dim3(256), 0, st, g, w, K, Q);
  }
  launch("k_obs_reduce", k_obs_reduce, dim3(g.B * g.H * ((g.m + 63) / 64)), dim3(1024), 0, st, g, w);
  if (g.dtype == 1) {
    if (r2) launch("k_obs_pass", k_obs_pass<1, 2>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
    else launch("k_obs_pass", k_obs_pass<1, 1>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
  } else {
    if (r2) launch("k_obs_pass", k_obs_pass<0, 2>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
    else launch("k_obs_pass", k_obs_pass<0, 1>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
  }
  return hipGetLastError();
}

}  // namespace akv
