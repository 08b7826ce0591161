// Observation-window pass of the compression (Sec. 3.2 anchor selection,
// App. A.2 Eq. selector-score; Sec. 3.3 needs the same attention for the
// utilities).  For every KV head the m = W * (Hq/H) observation rows (the
// queries of the last W positions, causal inside the window) attend to all
// positions:
//   k_obs_stats   : per half chunk (1024 tokens), MFMA logits q_w.k_t / sqrt(D)
//                   and the per-row running max and sum of exp;
//   k_obs_reduce  : merges the chunk statistics into M_w and 1/Z_w;
//   k_obs_pass    : recomputes the logits, alpha = exp(l - M)/Z, the SnapKV
//                   column score sc(t) = (1/m) sum_w alpha_wt, and the partial
//                   outputs y_w = sum_t alpha_wt v_t on MFMA (alpha split into two
//                   bf16 terms so y keeps about 16 bits);
//   k_obs_yreduce : sums the partial outputs, ||y_w||^2 and the bf16 hi/lo split
//                   of y used by the utility epilogue.
#include "akv_common.h"

namespace akv {

template <int DT> struct TileLD { static constexpr int v = AKV_D + (DT ? 8 : 4); };

// Orientation of the observation logits: the MFMA takes the key tile as its
// row operand and the query fragments as its column operand, so lane l holds
// the logits of observation row w = l % 32 (of its row block) against the 16
// tokens crow(e, l), e = 0..15, of the 32-token tile.  A lane's row max, 1/Z
// and causal limit are then single registers, and its 16 probabilities serve
// directly as the row operand of the value contraction, whose k index kappa
// runs over the tokens in the order the accumulator entries are taken:
// kappa = KS s + KL (l / 32) + j holds entry e = KL s + j, i.e. token
// kap_tok(kappa); the value tile is stored in that order.
template <int DT>
__device__ inline int tok_kap(int t) {  // token -> kappa (inverse of the entry order)
  if constexpr (DT == 1) {
    return (t & ~12) | ((t >> 2) & 1) << 3 | ((t >> 3) & 1) << 2;  // bits 2 and 3 swapped
  } else {
    return (t & ~7) | (t & 3) << 1 | ((t >> 2) & 1);
  }
}

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

// Position of contraction index kappa in row d of the transposed value tile:
// groups of 8 stay contiguous (one MFMA operand load) and are permuted by d,
// which spreads the stores of one wave over the LDS banks.
__device__ inline int vt_pos(int d, int kap) { return (((kap >> 3) ^ (d >> 3)) & 3) * 8 + (kap & 7); }

// Value tile, transposed: lds[d * LDT + vt_pos(d, tok_kap(r))] = X[t0 + r][d].
// Thread c takes rows 2p, 2p+1 (p = c / CPR) of one 16-byte column chunk; for
// bf16 the two tokens have adjacent kappa and are stored as one 32-bit word.
template <int DT>
struct PairTile {
  using E = typename Elem<DT>::T;
  static constexpr int PER = 16 / sizeof(E), CPR = AKV_D / PER, NP = 16 * CPR / 256;
  uint4 v0[NP], v1[NP];
  __device__ void load(const E* X, int t0, int S) {
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int c = threadIdx.x + 256 * i, p = c / CPR, col = (c % CPR) * PER;
      const int r0 = t0 + 2 * p;
      v0[i] = r0 < S ? *(const uint4*)(X + (size_t)r0 * AKV_D + col) : make_uint4(0, 0, 0, 0);
      v1[i] = r0 + 1 < S ? *(const uint4*)(X + (size_t)(r0 + 1) * AKV_D + col) : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ void store_t(E* lds, int LDT) const {
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int c = threadIdx.x + 256 * i, p = c / CPR, col = (c % CPR) * PER;
      const E* e0 = (const E*)&v0[i];
      const E* e1 = (const E*)&v1[i];
      const int k0 = tok_kap<DT>(2 * p), k1 = tok_kap<DT>(2 * p + 1);
      if constexpr (sizeof(E) == 2) {
#pragma unroll
        for (int j = 0; j < PER; ++j)
          *(uint32_t*)(lds + (col + j) * LDT + vt_pos(col + j, k0)) = (uint32_t)e0[j] | ((uint32_t)e1[j] << 16);
      } else {
#pragma unroll
        for (int j = 0; j < PER; ++j) {
          lds[(col + j) * LDT + vt_pos(col + j, k0)] = e0[j];
          lds[(col + j) * LDT + vt_pos(col + j, k1)] = e1[j];
        }
      }
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

// Two fp32 values rounded to nearest-even bf16, packed low | high << 16.
__device__ inline uint32_t pk_bf16(float x0, float x1) {
  typedef __attribute__((ext_vector_type(2))) float f32x2;
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
  const f32x2 v = {x0, x1};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
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
    w.oiZ64[(size_t)(b * g.H + h) * g.m + wr] = 1.0 / Zt;
  }
}

template <int DT, int R>
__global__ __launch_bounds__(256) void k_obs_pass(Geo g, Ws w, const void* Kin, const void* Vin, const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = TileLD<DT>::v;
  constexpr int LDT = 32 + (DT ? 8 : 4);  // transposed value tile row stride (16-byte aligned rows)
  __shared__ __align__(16) E KT[2][32 * LD];      // double-buffered tiles
  __shared__ __align__(16) E VT[2][AKV_D * LDT];
  __shared__ float scw[2][4][32];
  int idx = blockIdx.x;
  const int b = locate(g, OBS_CHUNK, 1, idx);
  const int S = g.S[b], P = S - g.W, D = g.D, m = g.m;
  const int nch = (S + OBS_CHUNK - 1) / OBS_CHUNK;
  const int h = idx / nch, ch = idx % nch;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)Kin + xoff;
  const E* Vx = (const E*)Vin + xoff;
  const E* Q = qrows<DT>(g, Qin, b, h);
  const float* oM = w.oM + (size_t)(b * g.H + h) * m;
  const float* oiZ = w.oiZ + (size_t)(b * g.H + h) * m;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (m + 31) / 32;
  const float isd = 1.0f / sqrtf((float)D);
  f32x16 yacc[R][4];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int db = 0; db < 4; ++db) yacc[r][db] = f32x16{};
  // The lane's row of each row block: query fragments, row max, 1/Z and
  // causal limit stay in registers; the next token tile's keys and values are
  // loaded while the current one is used.
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
  // Tile it sits in KT/VT[it & 1] and leaves its column sums in scw[it & 1];
  // after the barrier that starts tile it, the next tile is stored into the
  // other buffer and the column sums of tile it - 1 are final.  One barrier
  // per tile.
  RowTile<DT> kt;
  PairTile<DT> vt;
  kt.load(X, tb, S);
  vt.load(Vx, tb, S);
  kt.store(KT[0], LD);
  vt.store_t(VT[0], LDT);
  if (tb + 32 < te) {
    kt.load(X, tb + 32, S);
    vt.load(Vx, tb + 32, S);
  }
  int it = 0;
  for (int t0 = tb; t0 < te; t0 += 32, ++it) {
    const int cb = it & 1;
    __syncthreads();
    if (it > 0 && threadIdx.x < 32 && t0 - 32 + threadIdx.x < S)
      sc[t0 - 32 + threadIdx.x] = (scw[cb ^ 1][0][threadIdx.x] + scw[cb ^ 1][1][threadIdx.x] +
                                   scw[cb ^ 1][2][threadIdx.x] + scw[cb ^ 1][3][threadIdx.x]) / (float)m;
    if (t0 + 32 < te) {
      kt.store(KT[cb ^ 1], LD);
      vt.store_t(VT[cb ^ 1], LDT);
    }
    if (t0 + 64 < te) {
      kt.load(X, t0 + 64, S);
      vt.load(Vx, t0 + 64, S);
    }
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
      float al[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float a = __expf(acc[e] * isd - rmax[r]) * riz[r];
        al[e] = t0 + crow(e, lane) <= lim[r] ? a : 0.0f;
        cs[e] += al[e];
      }
      // y_w += sum_t alpha[w][t] V[t][d]: row operand = alpha (entries KL s ..
      // KL s + KL - 1 for step s), column operand = the value tile in kappa order.
#pragma unroll
      for (int s = 0; s < 32 / M::KS; ++s) {
        typename M::frag ah, alo;
        if constexpr (DT == 1) {
          uint32_t hw[4], lw[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float x0 = al[8 * s + 2 * j], x1 = al[8 * s + 2 * j + 1];
            hw[j] = pk_bf16(x0, x1);
            lw[j] = pk_bf16(x0 - __builtin_bit_cast(float, hw[j] << 16),
                            x1 - __builtin_bit_cast(float, hw[j] & 0xFFFF0000u));
          }
          ah = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
          alo = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
        } else {
          ah = al[s];
        }
        const int k0 = kofs(M::KS, s, lane);
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const int d = db * 32 + (lane & 31);
          auto vb = M::load_lds(&VT[cb][d * LDT + vt_pos(d, k0)], 0);
          yacc[r][db] = M::mma(ah, vb, yacc[r][db]);
          if constexpr (DT == 1) yacc[r][db] = M::mma(alo, vb, yacc[r][db]);
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
  // Partial outputs of this chunk.
  float* yp = w.ypart + ((size_t)(g.prefC[b] * g.H + h * nch + ch)) * m * D;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int rb = wave + 4 * r;
    if (rb >= nrb) break;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int wr = rb * 32 + crow(e, lane);
        if (wr < m) yp[(size_t)wr * D + db * 32 + (lane & 31)] = yacc[r][db][e];
      }
  }
}

__global__ __launch_bounds__(128) void k_obs_yreduce(Geo g, Ws w) {
  const int bh = blockIdx.x / g.m, wr = blockIdx.x % g.m;
  const int b = bh / g.H, h = bh % g.H;
  const int nch = (g.S[b] + OBS_CHUNK - 1) / OBS_CHUNK;
  const int D = g.D;
  __shared__ float red[2];
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    // Chunks added in order, their partial outputs loaded 16 at a time.
    const float* yp = w.ypart + (((size_t)(g.prefC[b] * g.H + h * nch)) * g.m + wr) * D + d;
    const size_t cs = (size_t)g.m * D;
    float y = 0.0f;
    for (int c0 = 0; c0 < nch; c0 += 16) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = c0 + u < nch ? yp[(size_t)(c0 + u) * cs] : 0.0f;
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (c0 + u < nch) y += v[u];
    }
    size_t o = ((size_t)bh * g.m + wr) * D + d;
    w.Y[o] = y;
    uint16_t hi = f2bf(y);
    w.Yhi[o] = hi;
    w.Ylo[o] = f2bf(y - bf2f(hi));
    float sq = wave_sum(y * y);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sq;
  }
  __syncthreads();
  if (threadIdx.x == 0) w.ynorm[(size_t)bh * g.m + wr] = red[0] + (D > 64 ? red[1] : 0.0f);
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
    if (r2) launch("k_obs_pass", k_obs_pass<1, 2>, dim3(nblk), dim3(256), 0, st, g, w, K, V, Q);
    else launch("k_obs_pass", k_obs_pass<1, 1>, dim3(nblk), dim3(256), 0, st, g, w, K, V, Q);
  } else {
    if (r2) launch("k_obs_pass", k_obs_pass<0, 2>, dim3(nblk), dim3(256), 0, st, g, w, K, V, Q);
    else launch("k_obs_pass", k_obs_pass<0, 1>, dim3(nblk), dim3(256), 0, st, g, w, K, V, Q);
  }
  launch("k_obs_yreduce", k_obs_yreduce, dim3(g.B * g.H * g.m), dim3(128), 0, st, g, w);
  return hipGetLastError();
}

}  // namespace akv
