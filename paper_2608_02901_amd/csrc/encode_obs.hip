// Observation-window pass of the compression (Sec. 3.2 anchor selection,
// App. A.2 Eq. selector-score; Sec. 3.3 needs the same attention for the
// utilities).  For every KV head the m = W * (Hq/H) observation rows (the
// queries of the last W positions, causal inside the window) attend to all
// positions:
//   k_obs_stats   : per chunk of 2048 tokens, MFMA logits q_w.k_t / sqrt(D) and
//                   the per-row running max and sum of exp;
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

// Loads 32 token rows [t0, t0+32) of X ([S][D], row-major) into LDS with row
// stride LD; rows at or past S are zero.
template <int DT>
__device__ inline void load_rows(typename Elem<DT>::T* lds, const typename Elem<DT>::T* X, int t0, int S, int D,
                                 int LD) {
  using E = typename Elem<DT>::T;
  constexpr int PER = 16 / sizeof(E);  // elements per 16-byte chunk
  const int cpr = D / PER;             // chunks per row
  for (int c = threadIdx.x; c < 32 * cpr; c += blockDim.x) {
    int r = c / cpr, col = (c % cpr) * PER;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t0 + r < S) v = *(const uint4*)(X + (size_t)(t0 + r) * D + col);
    *(uint4*)(lds + r * LD + col) = v;
  }
}

// Loads 32 token rows transposed: lds[d * LDT + r] = X[t0 + r][d].
template <int DT>
__device__ inline void load_rows_t(typename Elem<DT>::T* lds, const typename Elem<DT>::T* X, int t0, int S, int D,
                                   int LDT) {
  using E = typename Elem<DT>::T;
  constexpr int PER = 16 / sizeof(E);
  const int cpr = D / PER;
  for (int c = threadIdx.x; c < 32 * cpr; c += blockDim.x) {
    int r = c / cpr, col = (c % cpr) * PER;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t0 + r < S) v = *(const uint4*)(X + (size_t)(t0 + r) * D + col);
    const E* e = (const E*)&v;
#pragma unroll
    for (int i = 0; i < PER; ++i) lds[(col + i) * LDT + r] = e[i];
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
  // Transposed: lds[d * LDT + r] = X[t0 + r][d].
  __device__ void store_t(E* lds, int LDT) const {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int c = threadIdx.x + 256 * i, r = c / CPR, col = (c % CPR) * PER;
      const E* e = (const E*)&v[i];
#pragma unroll
      for (int j = 0; j < PER; ++j) lds[(col + j) * LDT + r] = e[j];
    }
  }
};

// Position of token r in row d of the transposed value tile: groups of 8
// tokens stay contiguous (one MFMA operand load) and are permuted by d, which
// spreads the stores of one wave over the LDS banks.
__device__ inline int vt_pos(int d, int r) { return (((r >> 3) ^ (d >> 3)) & 3) * 8 + (r & 7); }

// Value tile for the transposed LDS layout lds[d * LDT + vt_pos(d, r)] = X[t0 + r][d]:
// thread c takes rows 2p, 2p+1 (p = c / CPR) of one 16-byte column chunk, so
// for bf16 the two tokens of a column are stored as one 32-bit word.
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
      if constexpr (sizeof(E) == 2) {
#pragma unroll
        for (int j = 0; j < PER; ++j)
          *(uint32_t*)(lds + (col + j) * LDT + vt_pos(col + j, 2 * p)) = (uint32_t)e0[j] | ((uint32_t)e1[j] << 16);
      } else {
#pragma unroll
        for (int j = 0; j < PER; ++j)
          *(float2*)(lds + (col + j) * LDT + vt_pos(col + j, 2 * p)) = make_float2(e0[j], e1[j]);
      }
    }
  }
};

template <int DT>
__device__ inline typename MF<DT>::frag zero_frag() {
  if constexpr (DT == 1) {
    return __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
  } else {
    return 0.0f;
  }
}

// Query row w of KV head h (rows w = jj*W + i are contiguous in [Hq][W][D]).
template <int DT>
__device__ inline const typename Elem<DT>::T* qrows(const Geo& g, const void* Qin, int b, int h) {
  return (const typename Elem<DT>::T*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * g.D;
}

__device__ inline bool obs_visible(int t, int S, int P, int wr, int m, int W) {
  return t < S && wr < m && (t < P || t <= P + (wr % W));
}

constexpr float NEG = -1e30f;

// R = row blocks of 32 observation rows per wave (4 waves cover 128 R rows).
template <int DT, int R>
__global__ __launch_bounds__(256) void k_obs_stats(Geo g, Ws w, const void* Kin, const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = TileLD<DT>::v;
  __shared__ __align__(16) E KT[32 * LD];
  int idx = blockIdx.x;
  const int b = locate(g, OBS_CHUNK, 1, idx);
  const int S = g.S[b], P = S - g.W, D = g.D, m = g.m;
  const int nch = (S + OBS_CHUNK - 1) / OBS_CHUNK;
  const int h = idx / nch, ch = idx % nch;
  const E* X = (const E*)Kin + ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* Q = qrows<DT>(g, Qin, b, h);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (m + 31) / 32;
  const float isd = 1.0f / sqrtf((float)D);
  // Running row max (fp32 logits) and sum of exp in fp64; a change of the
  // max rescales the sum by an fp64 exp, so the sum keeps ~1e-9 relative
  // accuracy (the anchor selection re-scores near-ties against it).
  float mx[R][16];
  double sm[R][16];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int e = 0; e < 16; ++e) { mx[r][e] = NEG; sm[r][e] = 0.0; }
  // Query fragments of the wave's row blocks stay in registers.
  constexpr int NKS = AKV_D / M::KS;
  typename M::frag qf[R][NKS];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int arow = min((wave + 4 * r) * 32 + (lane & 31), m - 1);
#pragma unroll
    for (int s = 0; s < NKS; ++s) qf[r][s] = M::load(Q + (size_t)arow * D, kofs(M::KS, s, lane));
  }
  const int tb = ch * OBS_CHUNK, te = min(S, tb + OBS_CHUNK);
  RowTile<DT> kt;
  kt.load(X, tb, S);
  for (int t0 = tb; t0 < te; t0 += 32) {
    __syncthreads();
    kt.store(KT, LD);
    __syncthreads();
    if (t0 + 32 < te) kt.load(X, t0 + 32, S);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= nrb) break;
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        auto bb = M::load_lds(&KT[(lane & 31) * LD], kofs(M::KS, s, lane));
        acc = M::mma(qf[r][s], bb, acc);
      }
      const int t = t0 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int wr = rb * 32 + crow(e, lane);
        if (obs_visible(t, S, P, wr, m, g.W)) {
          const float l = acc[e] * isd;
          if (l > mx[r][e]) {
            sm[r][e] *= exp((double)mx[r][e] - (double)l);
            mx[r][e] = l;
          }
          sm[r][e] += (double)__expf(l - mx[r][e]);
        }
      }
    }
  }
  // Merge the 32 lanes that share each row.
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int rb = wave + 4 * r;
    if (rb >= nrb) break;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float a = mx[r][e];
      double s = sm[r][e];
      for (int o = 1; o < 32; o <<= 1) {
        const float oa = __shfl_xor(a, o, 64);
        const double os = __shfl_xor(s, o, 64);
        const float nm = fmaxf(a, oa);
        s = (a == nm ? s : s * exp((double)a - (double)nm)) + (oa == nm ? os : os * exp((double)oa - (double)nm));
        a = nm;
      }
      const int wr = rb * 32 + crow(e, lane);
      if ((lane & 31) == 0 && wr < m) {
        size_t o = ((size_t)(g.prefC[b] * g.H + h * nch + ch)) * m + wr;
        w.opmax[o] = a;
        w.opsum[o] = s;
      }
    }
  }
}

__global__ __launch_bounds__(256) void k_obs_reduce(Geo g, Ws w) {
  const int b = blockIdx.x / g.H, h = blockIdx.x % g.H;
  const int nch = (g.S[b] + OBS_CHUNK - 1) / OBS_CHUNK;
  for (int wr = threadIdx.x; wr < g.m; wr += blockDim.x) {
    size_t base = ((size_t)(g.prefC[b] * g.H + h * nch)) * g.m + wr;
    float M = NEG;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, w.opmax[base + (size_t)c * g.m]);
    double Z = 0.0;
    for (int c = 0; c < nch; ++c) {
      const float mc = w.opmax[base + (size_t)c * g.m];
      const double sc = w.opsum[base + (size_t)c * g.m];
      Z += mc == M ? sc : sc * exp((double)mc - (double)M);
    }
    w.oM[(size_t)(b * g.H + h) * g.m + wr] = M;
    w.oiZ[(size_t)(b * g.H + h) * g.m + wr] = (float)(1.0 / Z);
    w.oiZ64[(size_t)(b * g.H + h) * g.m + wr] = 1.0 / Z;
  }
}

template <int DT, int R>
__global__ __launch_bounds__(256) void k_obs_pass(Geo g, Ws w, const void* Kin, const void* Vin, const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = TileLD<DT>::v;
  constexpr int LDT = 32 + (DT ? 8 : 4);  // transposed value tile / alpha tile row stride (16-byte aligned rows)
  __shared__ __align__(16) E KT[32 * LD];
  __shared__ __align__(16) E VT[AKV_D * LDT];
  __shared__ __align__(16) E AH[4][R][32 * LDT];  // alpha (hi part for bf16)
  __shared__ __align__(16) E AL[DT ? 4 : 1][R][DT ? 32 * LDT : 1];  // alpha lo part (bf16 only)
  __shared__ float scb[32];
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
  // Query fragments of the wave's row blocks stay in registers; the next
  // token tile's keys and values are loaded while the current one is used.
  constexpr int NKS = AKV_D / M::KS;
  typename M::frag qf[R][NKS];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int arow = min((wave + 4 * r) * 32 + (lane & 31), m - 1);
#pragma unroll
    for (int s = 0; s < NKS; ++s) qf[r][s] = M::load(Q + (size_t)arow * D, kofs(M::KS, s, lane));
  }
  const int tb = ch * OBS_CHUNK, te = min(S, tb + OBS_CHUNK);
  float* sc = w.sc + (size_t)g.prefS[b] * g.H + (size_t)h * S;
  RowTile<DT> kt;
  PairTile<DT> vt;
  kt.load(X, tb, S);
  vt.load(Vx, tb, S);
  for (int t0 = tb; t0 < te; t0 += 32) {
    __syncthreads();
    kt.store(KT, LD);
    vt.store_t(VT, LDT);
    if (threadIdx.x < 32) scb[threadIdx.x] = 0.0f;
    __syncthreads();
    if (t0 + 32 < te) {
      kt.load(X, t0 + 32, S);
      vt.load(Vx, t0 + 32, S);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= nrb) break;
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        auto bb = M::load_lds(&KT[(lane & 31) * LD], kofs(M::KS, s, lane));
        acc = M::mma(qf[r][s], bb, acc);
      }
      const int tl = lane & 31, t = t0 + tl;
      float col = 0.0f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int wl = crow(e, lane), wr = rb * 32 + wl;
        float al = 0.0f;
        if (obs_visible(t, S, P, wr, m, g.W)) al = __expf(acc[e] * isd - oM[wr]) * oiZ[wr];
        col += al;
        if constexpr (DT == 1) {
          uint16_t hi = f2bf(al);
          AH[wave][r][wl * LDT + tl] = hi;
          AL[wave][r][wl * LDT + tl] = f2bf(al - bf2f(hi));
        } else {
          AH[wave][r][wl * LDT + tl] = al;
        }
      }
      col += __shfl_xor(col, 32, 64);
      if (lane < 32) atomicAdd(&scb[lane], col);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // y_w += alpha[w][t] V[t][d]: A = alpha (rows w, k = tokens), B = V^T tile.
      for (int s = 0; s < 32 / M::KS; ++s) {
        const int k0 = kofs(M::KS, s, lane);
        auto ah = M::load_lds(&AH[wave][r][(lane & 31) * LDT], k0);
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const int d = db * 32 + (lane & 31);
          auto vb = M::load_lds(&VT[d * LDT + vt_pos(d, k0)], 0);
          yacc[r][db] = M::mma(ah, vb, yacc[r][db]);
          if constexpr (DT == 1) {
            auto alo = M::load_lds(&AL[wave][r][(lane & 31) * LDT], k0);
            yacc[r][db] = M::mma(alo, vb, yacc[r][db]);
          }
        }
      }
    }
    __syncthreads();
    if (threadIdx.x < 32 && t0 + threadIdx.x < S) sc[t0 + threadIdx.x] = scb[threadIdx.x] / (float)m;
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
    float y = 0.0f;
    for (int c = 0; c < nch; ++c)
      y += w.ypart[(((size_t)(g.prefC[b] * g.H + h * nch + c)) * g.m + wr) * D + d];
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
    if (r2) launch("k_obs_stats", k_obs_stats<1, 2>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
    else launch("k_obs_stats", k_obs_stats<1, 1>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
  } else {
    if (r2) launch("k_obs_stats", k_obs_stats<0, 2>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
    else launch("k_obs_stats", k_obs_stats<0, 1>, dim3(nblk), dim3(256), 0, st, g, w, K, Q);
  }
  launch("k_obs_reduce", k_obs_reduce, dim3(g.B * g.H), dim3(256), 0, st, g, w);
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
