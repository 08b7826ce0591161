// Selector score of the compression (Sec. 3.2 anchor selection, App. A.2
// Eq. selector-score): for every KV head the m = W * (Hq/H) observation rows
// (the queries of the last W positions, causal inside the window) attend to
// all positions, and k_obs_pass takes fp32 MFMA logits q_w.k_t / sqrt(D),
// alpha = exp(l - M_w) / Z_w with the row statistics of the fp64 pass
// (encode_obs64.hip, which runs first; as c_w = (M_w + ln Z_w) log2(e)) and
// the SnapKV column score sc(t) = (1/m) sum_w alpha_wt.
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
  const float* cw = w.cw + (size_t)(b * g.H + h) * m;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (m + 31) / 32;
  // alpha = exp(l / sqrt(D) - M_w) / Z_w is taken as exp2(l log2(e) / sqrt(D)
  // - c_w) with c_w = (M_w + ln Z_w) log2(e) from the fp64 row statistics
  // (one fused multiply-add and one exp2 per pair); rows past m get
  // c_w = +inf, hence alpha = 0.
  const float isl = 1.4426950408889634f / sqrtf((float)D);
  // The lane's row of each row block: query fragments, c_w and causal limit
  // stay in registers; the next key tile is loaded while the current one is
  // used.
  constexpr int NKS = AKV_D / M::KS;
  typename M::frag qf[R][NKS];
  float cwr[R];
  int lim[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int wr = (wave + 4 * r) * 32 + (lane & 31);
    const int arow = min(wr, m - 1);
    lim[r] = obs_limit(wr, m, P, g.W);
    cwr[r] = wr < m ? cw[arow] : INFINITY;
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
      // alpha of the lane's row and tokens t0 + crow(e, lane); a tile before
      // the window (every row attends to all of it) needs no causal mask.
      if (t0 + 32 <= P) {
#pragma unroll
        for (int e = 0; e < 16; ++e) cs[e] += __builtin_amdgcn_exp2f(fmaf(acc[e], isl, -cwr[r]));
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float a = __builtin_amdgcn_exp2f(fmaf(acc[e], isl, -cwr[r]));
          cs[e] += t0 + crow(e, lane) <= lim[r] ? a : 0.0f;
        }
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
hipError_t launch_obs(const Geo& g, const Ws& w, const void* K, const void* Q, hipStream_t st) {
  const int nblk = g.H * g.prefC[g.B];
  const bool r2 = g.m > 128;  // 4 waves x 2 row blocks of 32 for up to 256 rows
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
