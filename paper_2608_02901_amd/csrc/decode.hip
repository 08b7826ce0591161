// Decode attention over the compressed cache (Sec. 3.4 "Storage and
// Decoding"; App. E.1), the append of generated tokens, and the dense
// reconstruction of Eq. (reconstruction).
//
// Attention of query j (KV head h = j / g) over every stored entry t:
//   logit_t = scale * (gamma^K_t (q_j . abar^K_a(t)) + [t in R_K] q_rot . zhat^K_t / D)
//   out     = (sum_a w_a abar^V_a + s * FWHT(sum_t p_t zhat^V_t) / D) / sum_t p_t
// with p_t = exp(logit_t - max), w_a = sum over tokens of value anchor a of
// p_t gamma^V_t, zhat the dequantized rotated residual and q_rot = FWHT(s * q).
// This is the exact algebra of attention over the reconstructed cache: U is
// orthogonal and linear, so the inverse rotation of the value residuals is
// applied once per query and split instead of once per token, and the key
// residual term is a dot product in the rotated basis.
//
// One decode step is two launches:
//   k_dec_front  : work that depends only on the new query and token, fully
//                  parallel: anchor scores S_K[a][j] = q_j . abar^K_a (bf16:
//                  one MFMA contraction of 16-anchor tiles with the queries and
//                  the appended token as columns; fp32: one thread per anchor,
//                  the row in registers), key-residual terms q_rot . zhat^K_e / D
//                  (one thread per stored key residual), and, when a token is
//                  appended, its screening similarity to every anchor of both
//                  sides with a per-64-anchor top-2;
//   k_dec_stream : split-K pass over the value-anchor-grouped records.  Loads
//                  come in two rounds (records and flag words; then anchor
//                  scores, key-residual terms, value-anchor rows and value
//                  residual codes).  Each split writes (max, sum, output) with
//                  the rotation of its value residuals already undone.  All
//                  splits of a head run on one XCD.  Extra workgroups resolve
//                  the appended token's anchors meanwhile (certified argmax,
//                  canonical fp64 coefficient);
//   k_dec_merge  : merges the splits of each query head and the appended tail;
//   k_app_finish : the argmax resolution alone, for a standalone append.
//   k_reconstruct: dense x^ of one side of one request (Eq. reconstruction).
#include "akv_common.h"

namespace akv {

constexpr int PS = 4 + AKV_D;  // split record: max, sum, 2 pad, output[D]

__device__ inline float level(const Geo& g, int code) {
  // 0 -> -l1, 1 -> -l0, 2 -> +l0, 3 -> +l1 (the Lloyd-Max pair, or 1 and 3
  // for the naive uniform codec)
  const float mag = (code == 0 || code == 3) ? g.lev1 : g.lev0;
  return code < 2 ? -mag : mag;
}


// ------------------------------------------------------------------ positions
// x - floor(x) for the finite, non-negative angles (in revolutions) below:
// v_fract_f64 itself, without the compiler's guard for inputs just below an
// integer (a result of 1.0 turns by a whole revolution, the same rotation).
__device__ inline double fract64(double x) {
  double r;
  asm("v_fract_f64 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

// Keys are stored before the rotation when positions are encoded (Sec. 3.2
// "RoPE"); decode rotates each key at its position (App. E
// "Implementation").  The rotation of position p turns the coordinate pair
// (f, f + D/2) by p * inv_freq[f].  Its cosine and sine are evaluated in
// fp32 from the angle in revolutions, reduced in fp64 (p * inv_freq / 2 pi,
// fractional part, centred to [-1/2, 1/2)) and passed to the hardware sine
// and cosine, which take revolutions: within about 1e-6 of the fp32 table
// of the compression pass, well inside attention's tolerance.
__device__ inline void rope_cs(float invf, int p, float& c, float& s) {
  const float r = (float)fract64((double)p * ((double)invf * 0.15915494309189535));
  c = __builtin_amdgcn_cosf(r);
  s = __builtin_amdgcn_sinf(r);
}

// Base-2 logits sl2 * q_j . R_p x of tail tokens n0 .. n1-1 into dst[n - n0][j]:
// one wave per token (tokens wave, wave + 4, ...), lane f takes the pair
// (f, f + 64) of x = fp32(gm a) (row and gm from row_of(n), p from pos_of(n))
// and the GQ staged queries (qs: [j][D] fp32), then a wave sum per query.
// Whole workgroup of 256 threads; dst is LDS, complete after the call.
template <int DT, int GQ, typename RowOf, typename PosOf>
__device__ inline void rope_tail_logits(const float* qs, const float* invs, RowOf row_of, PosOf pos_of, float sl2,
                                        float (*dst)[GQ], int n0, int n1) {
  using E = typename Elem<DT>::T;
  constexpr int F = AKV_D / 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float qa[GQ], qb[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    qa[jj] = qs[jj * AKV_D + lane];
    qb[jj] = qs[jj * AKV_D + lane + F];
  }
  const float invf = invs[lane];
  for (int n = n0 + wave; n < n1; n += 4) {
    float gm;
    const E* row = row_of(n, gm);
    const float a = gm * Elem<DT>::get(row, lane), bb = gm * Elem<DT>::get(row, lane + F);
    float c, s;
    rope_cs(invf, pos_of(n), c, s);
    const float k0 = fmaf(c, a, -(s * bb)), k1 = fmaf(s, a, c * bb);
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) {
      const float t = wave_sum_dpp(fmaf(qa[jj], k0, qb[jj] * k1));
      if (lane == 0) dst[n - n0][jj] = t * sl2;
    }
  }
  __syncthreads();
}

// Merge of two (best, second best, index of best) summaries of screening
// scores; ties of the best go to the lower anchor index.
__device__ inline void top2_merge(float& b1, float& b2, int& i1, float c1, float c2, int j1) {
  const float t2 = fmaxf(fmaxf(b2, c2), fminf(b1, c1));
  if (c1 > b1 || (c1 == b1 && j1 < i1)) i1 = j1;
  b1 = fmaxf(b1, c1);
  b2 = t2;
}
__device__ inline void top2_wave(float& b1, float& b2, int& i1) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float c1 = __shfl_xor(b1, o, 64), c2 = __shfl_xor(b2, o, 64);
    const int j1 = __shfl_xor(i1, o, 64);
    top2_merge(b1, b2, i1, c1, c2, j1);
  }
}

// GQ consecutive floats (16-byte aligned when GQ >= 4) as a vector load/store.
template <int GQ>
__device__ inline void load_g(const float* p, float* v) {
  if constexpr (GQ % 4 == 0) {
#pragma unroll
    for (int i = 0; i < GQ / 4; ++i) {
      const float4 t = *(const float4*)(p + 4 * i);
      v[4 * i] = t.x;
      v[4 * i + 1] = t.y;
      v[4 * i + 2] = t.z;
      v[4 * i + 3] = t.w;
    }
  } else if constexpr (GQ == 2) {
    const float2 t = *(const float2*)p;
    v[0] = t.x;
    v[1] = t.y;
  } else {
    v[0] = p[0];
  }
}
template <int GQ>
__device__ inline void store_g(float* p, const float* v) {
  if constexpr (GQ % 4 == 0) {
#pragma unroll
    for (int i = 0; i < GQ / 4; ++i) *(float4*)(p + 4 * i) = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
  } else if constexpr (GQ == 2) {
    *(float2*)p = make_float2(v[0], v[1]);
  } else {
    p[0] = v[0];
  }
}

// ------------------------------------------------------------------ front
// Dot products of one anchor row (in registers) with the g staged queries
// ([d][j] layout) and with the appended token.
template <int DT, int GQ, bool DOQ, bool APP>
__device__ inline void anchor_dots(const uint4* rv, const float* qs, const float* xs, float* acc, float& s) {
  using E = typename Elem<DT>::T;
  constexpr int PER = 16 / sizeof(E), NV = AKV_D / PER;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const E* e = (const E*)&rv[i];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const float x = Elem<DT>::get(e, j);
      if constexpr (DOQ) {
        float qv[GQ];
        load_g<GQ>(&qs[(i * PER + j) * GQ], qv);
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) acc[jj] = fmaf(qv[jj], x, acc[jj]);
      }
      if constexpr (APP) s = fmaf(xs[i * PER + j], x, s);
    }
  }
}

template <int M>
__device__ inline int lane_xor_i(int v) {
  return __builtin_bit_cast(int, lane_xor<M>(__builtin_bit_cast(float, v)));
}
template <int M>
__device__ inline void top2_step(float& b1, float& b2, int& i1) {
  const float c1 = lane_xor<M>(b1), c2 = lane_xor<M>(b2);
  const int j1 = lane_xor_i<M>(i1);
  top2_merge(b1, b2, i1, c1, c2, j1);
}
__device__ inline void top2_wave_dpp(float& b1, float& b2, int& i1) {
  top2_step<1>(b1, b2, i1);
  top2_step<2>(b1, b2, i1);
  top2_step<4>(b1, b2, i1);
  top2_step<8>(b1, b2, i1);
  top2_step<16>(b1, b2, i1);
  top2_step<32>(b1, b2, i1);
}

// Screening top-2 records of the appended token: one per 64 anchors (a wave's
// share of a 256-anchor block), [side][b][h][4 ceil(k_b / 256)].
__device__ inline size_t atop_index(const Geo& g, int side, int b, int h, int chunk) {
  const int nab = (g.k[b] + 255) / 256;
  return 4 * ((size_t)side * g.H * g.prefAB[g.B] + (size_t)g.prefAB[b] * g.H + (size_t)h * nab) + chunk;
}

// One block of 256 bf16 anchors of (request b, head h, side) on MFMA
// (v_mfma_f32_16x16x32_bf16).  Wave w takes anchors ch * 256 + 64 w .. +63 as
// four 16-row tiles, loaded straight into A fragments; B holds the g queries
// in columns 0 .. g-1 (key side, attention) and the appended token in column
// g (append), zeros elsewhere.  One contraction gives the anchor scores
// S_K[a][j] (stored scaled by sl2) and the screening products x . abar_a; the
// screening score |x . abar_a| / ||abar_a|| and the block's top-2 follow.  fp32
// accumulation of exact bf16 products in any order stays within the error
// bound the appended token's certification assumes.
template <int GQ>
__device__ void anchor_block_mfma(const Geo& g, const Cache& c, const DecWs& dw, const void* q, const void* kin,
                                  const void* vin, bool attn, bool app, int side, int b, int h, int ch, float sl2) {
  static_assert(GQ < 16, "queries and the appended token share one 16-column tile");
  constexpr int D = AKV_D;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int k = g.k[b], kp = (k + 3) & ~3;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const size_t ab = (size_t)g.prefKp[b] * g.H + (size_t)h * kp;
  const uint16_t* A = (const uint16_t*)(side ? c.ancV : c.ancK) + ko * D;
  const bool doq = attn && side == 0;
  const int col = lane & 15, kq = lane >> 4;
  const uint16_t* bsrc = nullptr;
  if (doq && col < GQ) bsrc = (const uint16_t*)q + ((size_t)b * g.Hq + (size_t)h * GQ + col) * D;
  if (app && col == GQ) bsrc = (const uint16_t*)(side ? vin : kin) + ((size_t)b * g.H + h) * D;
  bf16x8 bf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const uint4 v = bsrc ? *(const uint4*)(bsrc + 32 * ks + 8 * kq) : make_uint4(0, 0, 0, 0);
    bf[ks] = __builtin_bit_cast(bf16x8, v);
  }
  const int a0 = ch * 256 + wave * 64;
  // inverse norms of the lane's 16 anchors, issued with the rows; loaded and
  // used by every lane (only column g keeps them), so the loads stay here
  const float* inv = (side ? c.invV : c.invK) + ko;
  float ivs[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) ivs[t][i] = inv[min(a0 + 16 * t + 4 * kq + i, k - 1)];
  bf16x8 af[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint16_t* row = A + (size_t)min(a0 + 16 * t + col, k - 1) * D + 8 * kq;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) af[t][ks] = __builtin_bit_cast(bf16x8, *(const uint4*)(row + 32 * ks));
  }
  float* ascp = dw.asc + (size_t)side * g.H * g.prefKp[g.B] + ab + a0 + 4 * kq;
  float4* atopp = dw.atop + atop_index(g, side, b, h, 4 * ch + wave);
  // Anchor the inverse-norm loads here (issued before the rows, so waiting
  // for them costs nothing the contraction would not wait for anyway);
  // otherwise they are sunk to the screening and pay a full round trip there.
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) asm volatile("" ::"v"(ivs[t][i]));
  f32x4 acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    acc[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[t][ks], bf[ks], acc[t], 0, 0, 0);
  }
  // lane holds column col of anchors a0 + 16 t + 4 kq + i, i = 0..3; a
  // wave whose 64 anchors all exist (every wave but a head's last) stores
  // without per-element guards.  The screening math (which waits for the
  // inverse norms) comes before every store: loads and stores share one
  // completion counter, so a wait issued after the stores would wait for them.
  const bool full = a0 + 63 < k;
  float b1 = -1.0f, b2 = -1.0f;
  int i1 = 0x7fffffff;
  float sc[4][4];
  if (app) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int a = a0 + 16 * t + 4 * kq + i;
        const bool ok = col == GQ && (full || a < k);
        sc[t][i] = ok ? fabsf(acc[t][i]) * ivs[t][i] : -1.0f;
        top2_merge(b1, b2, i1, sc[t][i], -1.0f, ok ? a : 0x7fffffff);
      }
    top2_wave_dpp(b1, b2, i1);
  }
  if (doq && col < GQ) {
    float* skp = dw.SK + (ab + a0 + 4 * kq) * GQ + col;
    if (full) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) skp[(16 * t + i) * GQ] = acc[t][i] * sl2;
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (a0 + 16 * t + 4 * kq + i < k) skp[(16 * t + i) * GQ] = acc[t][i] * sl2;
    }
  }
  if (!app) return;
  if (col == GQ) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (full || a0 + 16 * t + 4 * kq + i < k) ascp[16 * t + i] = sc[t][i];
  }
  if (lane == 0) *atopp = make_float4(b1, b2, __int_as_float(i1), 0.0f);
}

constexpr int RK_PER_BLOCK = 128;  // stored key residuals per key-residual block

// Grid: nAK key-anchor blocks, nAV value-anchor blocks (append only), then
// ceil(sum N_K / 128) key-residual blocks (attention only).  flags: bit 0 =
// attention (q given), bit 1 = append (k_new, v_new given).  sl2 = softmax
// scale * log2(e): the stored anchor scores and key-residual terms are logits
// in base 2.
template <int DT, int GQ>
__global__ __launch_bounds__(256) void k_dec_front(Geo g, Cache c, DecWs dw, const void* q, const void* kin,
                                                   const void* vin, int flags, int nAK, int nAV, float sl2) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D, PER = 16 / sizeof(E), NV = D / PER;
  constexpr int RK_TABS = GQ <= 4 ? 2 : 1;            // key-residual tables built per pass
  __shared__ __align__(16) float qs[RK_TABS * D * GQ];          // [head][d][j] queries, or rotated queries
  __shared__ __align__(16) float tab[RK_TABS * 64 * 16 * GQ];   // [head][pair][nibble][j] residual-term table
  __shared__ float xs[D];
  __shared__ __align__(16) E qraw[64 * D];            // queries of one request (key-residual blocks)
  __shared__ int bhr[2];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool attn = flags & 1, app = (flags & 2) != 0;
  int idx = blockIdx.x;
  if (idx < nAK + nAV) {
    const int side = idx >= nAK ? 1 : 0;
    if (side) idx -= nAK;
    int b = 0;
    for (; b < g.B - 1; ++b) {
      const int n = g.H * ((g.k[b] + 255) / 256);
      if (idx < n) break;
      idx -= n;
    }
    const int k = g.k[b], kp = (k + 3) & ~3, nab = (k + 255) / 256;
    const int h = idx / nab, ch = idx % nab;
    if constexpr (DT == 1) {
      anchor_block_mfma<GQ>(g, c, dw, q, kin, vin, attn, app, side, b, h, ch, sl2);
      return;
    }
    const int a = ch * 256 + tid;
    const bool valid = a < k;
    const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
    const E* row = (const E*)(side ? c.ancV : c.ancK) + (ko + min(a, k - 1)) * D;
    uint4 rv[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) rv[i] = *(const uint4*)(row + i * PER);
    const bool doq = attn && side == 0;
    if (doq) {
      const E* qp = (const E*)q + ((size_t)b * g.Hq + (size_t)h * GQ) * D;
      for (int i = tid; i < GQ * D; i += 256) qs[(i % D) * GQ + i / D] = Elem<DT>::get(qp, i);
    }
    if (app && tid < D) xs[tid] = Elem<DT>::get((const E*)(side ? vin : kin) + ((size_t)b * g.H + h) * D, tid);
    __syncthreads();
    const size_t ab = (size_t)g.prefKp[b] * g.H + (size_t)h * kp;  // anchor-table row of anchor 0
    float acc[GQ], s = 0.0f;
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) acc[jj] = 0.0f;
    if (doq && app) anchor_dots<DT, GQ, true, true>(rv, qs, xs, acc, s);
    else if (doq) anchor_dots<DT, GQ, true, false>(rv, qs, xs, acc, s);
    else anchor_dots<DT, GQ, false, true>(rv, qs, xs, acc, s);
    if (doq && valid) {
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) acc[jj] *= sl2;
      store_g<GQ>(dw.SK + (ab + a) * GQ, acc);
    }
    if (app) {
      const float* inv = (side ? c.invV : c.invK) + ko;
      const float sc = valid ? fabsf(s) * inv[a] : -1.0f;
      if (valid) dw.asc[(size_t)side * g.H * g.prefKp[g.B] + ab + a] = sc;
      float b1 = sc, b2 = -1.0f;
      int i1 = valid ? a : 0x7fffffff;
      top2_wave_dpp(b1, b2, i1);
      if (lane == 0) dw.atop[atop_index(g, side, b, h, 4 * ch + wave)] = make_float4(b1, b2, __int_as_float(i1), 0.0f);
    }
    return;
  }

  // ---- key-residual terms: two threads per stored key residual (global index
  // e), 128 residuals per block.  q_rot . zhat = sum over coordinate pairs of
  // a table entry indexed by the pair's 4-bit code (its two levels times the
  // two rotated query values), scaled by the group scale; each thread sums 32
  // pairs and the partner's sum is added with a lane swap.
  idx -= nAK + nAV;
  const int NKt = g.prefNK[g.B];
  const int e0 = idx * RK_PER_BLOCK;
  const int e = e0 + (tid >> 1), half = tid & 1;
  const bool valid = e < NKt;
  const int ec = min(e, NKt - 1);
  const int G = g.G;
  // The queries of the block's first request, loaded beside the codes so that
  // the rotation below does not wait for them (at most 64 query heads).
  int bq = 0;
  while (bq < g.B - 1 && e0 >= g.prefNK[bq + 1]) ++bq;
  const bool qpre = g.Hq <= 64;
  constexpr int QPT = 64 * D / PER / 256;  // 16-byte chunks per thread at 64 query heads
  const int nq4 = g.Hq * D / PER;
  uint4 qv[QPT];
  if (qpre) {
    const uint4* qsrc = (const uint4*)((const E*)q + (size_t)bq * g.Hq * D);
#pragma unroll
    for (int u = 0; u < QPT; ++u) {  // past the end: reload the last chunk, not stored
      const uint4 t = qsrc[min(tid + 256 * u, nq4 - 1)];
      qv[u] = make_uint4(t.x, t.y, t.z, t.w);
    }
  }
  __builtin_amdgcn_sched_barrier(0);  // issue the query loads first
  // this thread's half of the codes (pairs 32 half .. +31) and its two scales
  const uint4 ch4 = *(const uint4*)(c.codesK + (size_t)ec * (D / 4) + 16 * half);
  float sg[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) sg[u] = c.scalesK[(size_t)ec * (D / G) + ((2 * half + u) * 32) / G];
  // (request, head) of a residual index: the last head whose first residual
  // index (the flag-word prefix of its first word) is at most the index.
  // Each wave reads the head starts of its first residual's request one per
  // lane (one round trip) and counts them; residuals of a later request (a
  // wave straddling requests) scan that request's starts.
  int bw = 0;
  const int ew = min(e0 + wave * 32, NKt - 1);
  while (bw < g.B - 1 && ew >= g.prefNK[bw + 1]) ++bw;
  const size_t wbw = (size_t)g.prefW[bw] * g.H;
  const int nww = (g.S[bw] + 63) / 64;
  int hst = 0x7fffffff;  // start of head `lane` (lanes 1 .. H-1; H <= 64 heads per ballot)
  for (int hh = lane; hh < g.H; hh += 64)
    if (hh == lane && hh >= 1) hst = c.pcK[wbw + (size_t)hh * nww];
  int b = bw;
  while (b < g.B - 1 && ec >= g.prefNK[b + 1]) ++b;
  int hcnt = 0;
  if (b == bw && g.H <= 64) {
    for (int l = 1; l < g.H; ++l) hcnt += __builtin_amdgcn_readlane(hst, l) <= ec ? 1 : 0;
  } else {
    const int nw = (g.S[b] + 63) / 64;
    const size_t wb = (size_t)g.prefW[b] * g.H;
    for (int hh = 1; hh < g.H; ++hh) hcnt += c.pcK[wb + (size_t)hh * nw] <= ec ? 1 : 0;
  }
  const int bh = b * g.H + hcnt;
  const int lastv = 2 * min(RK_PER_BLOCK - 1, NKt - 1 - e0);
  if (tid == 0) bhr[0] = bh;
  if (tid == lastv) bhr[1] = bh;
  if (qpre) {
#pragma unroll
    for (int u = 0; u < QPT; ++u)
      if (tid + 256 * u < nq4) ((uint4*)qraw)[tid + 256 * u] = qv[u];
  }
  __syncthreads();
  const int lo = bhr[0], hi = bhr[1];
  const uint32_t cw[4] = {ch4.x, ch4.y, ch4.z, ch4.w};
  // the rotated codec's residual dot is q_rot . zhat / D; the naive codec's
  // is q . zhat (no rotation)
  const float qscale = g.rot ? sl2 * (1.0f / (float)D) : sl2;
  const float s0v = sign_bit(g.sgnbits, 2 * lane), s1v = sign_bit(g.sgnbits, 2 * lane + 1);
  float dot[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) dot[jj] = 0.0f;
  for (int p0 = lo; p0 <= hi; p0 += RK_TABS) {  // RK_TABS heads per pass
    for (int f = wave; f < RK_TABS * GQ; f += 4) {
      const int p = p0 + f / GQ, jj = f % GQ;
      if (p > hi) continue;
      const int b2 = p / g.H, h2 = p % g.H;
      float z0, z1;
      if (qpre && b2 == bq) {
        const E* qp = qraw + ((size_t)h2 * GQ + jj) * D;
        z0 = Elem<DT>::get(qp, 2 * lane);
        z1 = Elem<DT>::get(qp, 2 * lane + 1);
      } else {
        const E* qp = (const E*)q + ((size_t)b2 * g.Hq + (size_t)h2 * GQ + jj) * D;
        z0 = Elem<DT>::get(qp, 2 * lane);
        z1 = Elem<DT>::get(qp, 2 * lane + 1);
      }
      if (g.rot) {
        z0 *= s0v;
        z1 *= s1v;
        fwht_wave_dpp(z0, z1, lane);
      }
      float* qt = qs + (f / GQ) * D * GQ;
      qt[(2 * lane) * GQ + jj] = z0 * qscale;
      qt[(2 * lane + 1) * GQ + jj] = z1 * qscale;
    }
    __syncthreads();
    for (int t = 0; t < RK_TABS && p0 + t <= hi; ++t) {  // table: thread = (pair t/4, nibbles 4 (t%4) .. +3)
      const float* qt = qs + t * D * GQ;
      float* tb = tab + t * 64 * 16 * GQ;
      const int pr = tid >> 2, n0 = 4 * (tid & 3);
      float qa[GQ], qb[GQ];
      load_g<GQ>(&qt[(2 * pr) * GQ], qa);
      load_g<GQ>(&qt[(2 * pr + 1) * GQ], qb);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int nib = n0 + u;
        const float la = level(g, nib & 3), lb = level(g, nib >> 2);
        float tv[GQ];
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) tv[jj] = fmaf(lb, qb[jj], la * qa[jj]);
        store_g<GQ>(&tb[(pr * 16 + nib) * GQ], tv);
      }
    }
    __syncthreads();
    if (bh >= p0 && bh < p0 + RK_TABS) {
      const float* tb = tab + (bh - p0) * 64 * 16 * GQ;
#pragma unroll
      for (int qh = 0; qh < 2; ++qh) {  // 32-coordinate quarters lie inside one group (G >= 32)
        const int qd = 2 * half + qh;
        float part[GQ];
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) part[jj] = 0.0f;
#pragma unroll
        for (int n = 0; n < 16; ++n) {
          const int pr = qd * 16 + n, lp = qh * 16 + n;  // lp: pair within this thread's half
          const int nib = (cw[lp >> 3] >> (4 * (lp & 7))) & 15;
          float tv[GQ];
          load_g<GQ>(&tb[(pr * 16 + nib) * GQ], tv);
#pragma unroll
          for (int jj = 0; jj < GQ; ++jj) part[jj] += tv[jj];
        }
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) dot[jj] = fmaf(sg[qh], part[jj], dot[jj]);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) dot[jj] += lane_xor<1>(dot[jj]);
  if (valid && half == 0) store_g<GQ>(dw.RK + (size_t)e * GQ, dot);
}

// ------------------------------------------------------------------ append resolution
// Resolves the appended token of (request b, head h) on both sides at once
// (waves 0-1: keys, waves 2-3: values) from the screening scores of
// k_dec_front: the best anchor by |cos| is certified when its margin over the
// runner-up exceeds the fp32 error bound; otherwise every anchor within the
// bound is rescored with the canonical fp64 formula (ties to the lowest
// index).  The coefficient is the canonical fp64 projection rounded to the
// stored dtype.  Whole-workgroup call; the records go to tail slot n_app and
// to out_idx[side] / out_gamma[side] (LDS).
template <int DT>
__device__ void append_resolve(const Geo& g, const Cache& c, const DecWs& dw, int b, int h, int n_app,
                               const void* kin, const void* vin, int* out_idx, float* out_gamma) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D;
  __shared__ float fr[2][3];
  __shared__ int ir[2];
  __shared__ double dr[4];
  __shared__ int di[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int side = wave >> 1, lt = tid & 127;
  const int k = g.k[b], kp = (k + 3) & ~3, nab = (k + 255) / 256;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const size_t ab = (size_t)g.prefKp[b] * g.H + (size_t)h * kp;
  const E* x = (const E*)(side ? vin : kin) + ((size_t)b * g.H + h) * D;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  const double* nrm = (side ? c.nrmV : c.nrmK) + ko;
  const float* sc = dw.asc + (size_t)side * g.H * g.prefKp[g.B] + ab;
  if ((wave & 1) == 0) {
    const float x0 = Elem<DT>::get(x, 2 * lane), x1 = Elem<DT>::get(x, 2 * lane + 1);
    const float ss = wave_sum(x0 * x0 + x1 * x1);
    const float xn = sqrtf(ss) * (1.0f + 1e-5f);
    float b1 = -1.0f, b2 = -1.0f;
    int i1 = 0x7fffffff;
    for (int ci = lane; ci < 4 * nab; ci += 64) {
      const float4 t = dw.atop[atop_index(g, side, b, h, ci)];
      top2_merge(b1, b2, i1, t.x, t.y, __float_as_int(t.z));
    }
    top2_wave(b1, b2, i1);
    if (lane == 0) {
      fr[side][0] = b1;
      fr[side][1] = b2;
      fr[side][2] = xn * ((float)D * 1.1920929e-7f + 2.3841858e-7f) * 1.01f + 1e-30f;
      ir[side] = i1;
    }
  }
  __syncthreads();
  const float b1 = fr[side][0], b2 = fr[side][1], eps = fr[side][2];
  const bool certified = b1 - b2 > 2.0f * eps + b1 * 9.094947e-13f;
  double bc = -INFINITY;
  int bi = 0x7fffffff;
  if (!certified) {
    const float band = b1 - 2.0f * eps - b1 * 9.094947e-13f;
    for (int a = lt; a < k; a += 128) {
      if (sc[a] < band) continue;
      const double d = dot64_seq<DT>(x, A + (size_t)a * D, D);
      const double cc = nrm[a] > 0.0 ? (d * d) / nrm[a] : -1.0;
      if (cc > bc) {
        bc = cc;
        bi = a;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const double oc = __shfl_xor(bc, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (oc > bc || (oc == bc && oi < bi)) {
        bc = oc;
        bi = oi;
      }
    }
    if (lane == 0) {
      dr[wave] = bc;
      di[wave] = bi;
    }
  }
  __syncthreads();
  if (lt == 0) {
    int best = ir[side];
    if (!certified) {
      const int w0 = 2 * side;
      best = (dr[w0 + 1] > dr[w0] || (dr[w0 + 1] == dr[w0] && di[w0 + 1] < di[w0])) ? di[w0 + 1] : di[w0];
    }
    const double n = nrm[best];
    const double d = dot64_seq<DT>(x, A + (size_t)best * D, D);
    const double g64 = n > 0.0 ? d / n : 0.0;
    const float gb = Elem<DT>::round_coef((float)g64);
    const size_t ti = ((size_t)b * g.H + h) * g.max_append + n_app;
    (side ? c.tidxV : c.tidxK)[ti] = (uint16_t)best;
    Elem<DT>::put(side ? c.tgV : c.tgK, ti, gb);
    out_idx[side] = best;
    out_gamma[side] = gb;
  }
  __syncthreads();
}

template <int DT>
__global__ __launch_bounds__(256) void k_app_finish(Geo g, Cache c, DecWs dw, int n_app, const void* kin,
                                                    const void* vin) {
  __shared__ int oi[2];
  __shared__ float og[2];
  append_resolve<DT>(g, c, dw, blockIdx.x / g.H, blockIdx.x % g.H, n_app, kin, vin, oi, og);
}

// ------------------------------------------------------------------ tail
// The appended tokens of one (request, KV head) as one more split record
// (index nsp) for each of its g query heads.  When this step appends a token
// (kin != nullptr), its anchors are resolved first and it joins the tail as
// slot n_app.  Tail tokens carry no residual: logit = gamma^K S_K[a^K], value
// gamma^V abar^V_{a^V}.  Runs beside the split workgroups of the stream pass.
template <int DT, int GQ>
__device__ void tail_block(const Geo& g, const Cache& c, const DecWs& dw, int bh, int n_app, const void* kin,
                           const void* vin, const void* q, float sl2, unsigned char* pool) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D, TCH = 256;
  __shared__ int t_idx[2];
  __shared__ float t_g[2];
  __shared__ float red[4][GQ];
  // Carved from the caller's LDS pool (>= 9 KB): weights p * gamma^V per
  // tail token, their value anchors, and the per-group output partials.
  float(*tl)[GQ] = (float(*)[GQ])pool;
  int* tav = (int*)(pool + TCH * GQ * 4);
  float(*acc)[D] = (float(*)[D])(pool + TCH * GQ * 4 + TCH * 4);
  // positions encoded: the queries, the frequencies and a chunk's logits
  float* qsr = (float*)(pool + TCH * GQ * 4 + TCH * 4 + 8 * D * 4);
  float* invs = qsr + GQ * D;
  float(*tlg)[GQ] = (float(*)[GQ])(invs + D / 2);
  const int b = bh / g.H, h = bh % g.H;
  const int S = g.S[b], k = g.k[b], kp = (k + 3) & ~3;
  const int nsp = (S + g.dsplit - 1) / g.dsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool app = kin != nullptr;
  if (app) append_resolve<DT>(g, c, dw, b, h, n_app, kin, vin, t_idx, t_g);
  const int ntail = n_app + (app ? 1 : 0);
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const float* SKh = dw.SK + ((size_t)g.prefKp[b] * g.H + (size_t)h * kp) * GQ;
  const E* AVg = (const E*)c.ancV + ko * D;
  const size_t tb = ((size_t)b * g.H + h) * g.max_append;
  if (g.rope) {
    const typename Elem<DT>::T* qg = (const typename Elem<DT>::T*)q + ((size_t)b * g.Hq + (size_t)h * GQ) * D;
    for (int i = tid; i < GQ * D; i += 256) qsr[i] = Elem<DT>::get(qg, i);
    if (tid < D / 2) invs[tid] = g.invf[tid];
    __syncthreads();
  }
  auto rec = [&](int n, int& ak, float& gk, int& av, float& gv) {
    if (app && n == n_app) {
      ak = t_idx[0];
      gk = t_g[0];
      av = t_idx[1];
      gv = t_g[1];
    } else {
      ak = min((int)c.tidxK[tb + n], k - 1);
      gk = Elem<DT>::get(c.tgK, tb + n);
      av = min((int)c.tidxV[tb + n], k - 1);
      gv = Elem<DT>::get(c.tgV, tb + n);
    }
  };
  // With positions encoded the logits q . R_{S+n} (gamma abar_a) of a chunk
  // of 256 tail tokens are formed first (one wave per token) into tlg.
  auto rope_chunk = [&](int c0) {
    rope_tail_logits<DT, GQ>(
        qsr, invs,
        [&](int n, float& gmo) {
          int ak, av;
          float gk, gv;
          rec(n, ak, gk, av, gv);
          gmo = gk;
          return (const E*)c.ancK + (ko + ak) * D;
        },
        [&](int n) { return S + n; }, sl2, tlg, c0, min(ntail, c0 + TCH));
  };
  // Base-2 logit of tail token n (chunk c0): gamma S_K[a], or from tlg.
  auto tlogit = [&](int n, int c0, int ak, float gk, float* l) {
    if (g.rope) {
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) l[jj] = tlg[n - c0][jj];
    } else {
      float sk[GQ];
      load_g<GQ>(SKh + (size_t)ak * GQ, sk);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) l[jj] = gk * sk[jj];
    }
  };
  // Maxima over the whole tail (log2-domain logits).
  float mloc[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) mloc[jj] = -INFINITY;
  for (int c0 = 0; c0 < ntail; c0 += TCH) {
    if (g.rope) rope_chunk(c0);
    const int n = c0 + tid;
    if (n < ntail) {
      int ak, av;
      float gk, gv;
      rec(n, ak, gk, av, gv);
      float sk[GQ];
      tlogit(n, c0, ak, gk, sk);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) mloc[jj] = fmaxf(mloc[jj], sk[jj]);
    }
    if (g.rope) __syncthreads();  // tlg is refilled by the next chunk
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float v = wave_max_dpp(mloc[jj]);
    if (lane == 0) red[wave][jj] = v;
  }
  __syncthreads();
  float M[GQ], lsum[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    M[jj] = fmaxf(fmaxf(red[0][jj], red[1][jj]), fmaxf(red[2][jj], red[3][jj]));
    lsum[jj] = 0.0f;
  }
  // Outputs: thread = (coordinate quad cq, token group sg of 8).
  const int cq = tid & 31, sg = tid >> 5;
  float o[GQ][4];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) o[jj][0] = o[jj][1] = o[jj][2] = o[jj][3] = 0.0f;
  for (int c0 = 0; c0 < ntail; c0 += TCH) {
    const int n = c0 + tid;
    __syncthreads();
    if (g.rope) rope_chunk(c0);
    if (n < ntail) {
      int ak, av;
      float gk, gv;
      rec(n, ak, gk, av, gv);
      float sk[GQ];
      tlogit(n, c0, ak, gk, sk);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        const float p = __builtin_amdgcn_exp2f(sk[jj] - M[jj]);
        lsum[jj] += p;
        tl[tid][jj] = p * gv;
      }
      tav[tid] = av;
    }
    __syncthreads();
    const int cn = min(TCH, ntail - c0);
    for (int u = sg; u < cn; u += 8) {
      const E* row = AVg + (size_t)tav[u] * D + 4 * cq;
      float v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = Elem<DT>::get(row, i);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        const float w = tl[u][jj];
#pragma unroll
        for (int i = 0; i < 4; ++i) o[jj][i] = fmaf(w, v[i], o[jj][i]);
      }
    }
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float v = wave_sum_dpp(lsum[jj]);
    __syncthreads();
    if (lane == 0) red[wave][jj] = v;
    __syncthreads();
    lsum[jj] = (red[0][jj] + red[1][jj]) + (red[2][jj] + red[3][jj]);
  }
  const int Hq = g.Hq;
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[sg][4 * cq + i] = o[jj][i];
    __syncthreads();
    float* pr = dw.part + ((size_t)g.prefSp[b] * Hq + (size_t)(h * GQ + jj) * (nsp + 1) + nsp) * PS;
    if (tid < D) {
      float y = 0.0f;
#pragma unroll
      for (int q = 0; q < 8; ++q) y += acc[q][tid];
      pr[4 + tid] = y;
    }
    if (tid == 0) {
      pr[0] = ntail > 0 ? M[jj] : -INFINITY;
      pr[1] = lsum[jj];
    }
  }
}

// The appended tokens of one (request, KV head) when they are stored exactly
// (App. E "Generated Tokens"): one more split record per query head of the
// group with the exact logits sl2 q_j . k_n (fp32, sequential over the
// coordinates) and the exact values.  When this step appends (kin !=
// nullptr), the token is written to tail slot n_app and attended straight
// from kin / vin.
template <int DT, int GQ>
__device__ void tail_dense(const Geo& g, const Cache& c, const DecWs& dw, int bh, int n_app, const void* kin,
                           const void* vin, const void* q, float sl2, unsigned char* pool) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D, TCH = 256;
  __shared__ float red[4][GQ];
  float(*qs)[D] = (float(*)[D])pool;
  float(*tl)[GQ] = (float(*)[GQ])(pool + GQ * D * 4);
  float(*acc)[D] = (float(*)[D])(pool + GQ * D * 4 + TCH * GQ * 4);
  float* invs = (float*)(pool + GQ * D * 4 + TCH * GQ * 4 + 8 * D * 4);  // positions encoded
  float(*tlg)[GQ] = (float(*)[GQ])(invs + D / 2);                          // a chunk's rotated logits
  const int b = bh / g.H, h = bh % g.H;
  const int S = g.S[b];
  const int nsp = (S + g.dsplit - 1) / g.dsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool app = kin != nullptr;
  const int ntail = n_app + (app ? 1 : 0);
  const size_t tb = ((size_t)b * g.H + h) * g.max_append;
  const E* TK = (const E*)c.tkd + tb * D;
  const E* TV = (const E*)c.tvd + tb * D;
  const E* kn = app ? (const E*)kin + ((size_t)b * g.H + h) * D : nullptr;
  const E* vn = app ? (const E*)vin + ((size_t)b * g.H + h) * D : nullptr;
  if (app && tid < D) {
    Elem<DT>::put(c.tkd, (tb + n_app) * D + tid, Elem<DT>::get(kn, tid));
    Elem<DT>::put(c.tvd, (tb + n_app) * D + tid, Elem<DT>::get(vn, tid));
  }
  const E* qg = (const E*)q + ((size_t)b * g.Hq + (size_t)h * GQ) * D;
  for (int i = tid; i < GQ * D; i += 256) qs[i / D][i % D] = Elem<DT>::get(qg, i);
  if (tid < D / 2) invs[tid] = g.invf[tid];
  __syncthreads();
  // With positions encoded the stored keys are unrotated: the logits
  // q . R_{S+n} k_n of a chunk of 256 tokens are formed first (one wave per
  // token) into tlg.
  auto rope_chunk = [&](int c0) {
    rope_tail_logits<DT, GQ>(
        &qs[0][0], invs,
        [&](int n, float& gmo) {
          gmo = 1.0f;
          return (app && n == n_app) ? kn : TK + (size_t)n * D;
        },
        [&](int n) { return S + n; }, sl2, tlg, c0, min(ntail, c0 + TCH));
  };
  auto logits = [&](int n, int c0, float* l) {
    const E* kr = (app && n == n_app) ? kn : TK + (size_t)n * D;
    if (g.rope) {
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) l[jj] = tlg[n - c0][jj];
      return;
    }
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) l[jj] = 0.0f;
    for (int d = 0; d < D; ++d) {
      const float kd = Elem<DT>::get(kr, d);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) l[jj] = fmaf(qs[jj][d], kd, l[jj]);
    }
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) l[jj] *= sl2;
  };
  float mloc[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) mloc[jj] = -INFINITY;
  for (int c0 = 0; c0 < ntail; c0 += TCH) {
    if (g.rope) rope_chunk(c0);
    const int n = c0 + tid;
    if (n < ntail) {
      float l[GQ];
      logits(n, c0, l);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) mloc[jj] = fmaxf(mloc[jj], l[jj]);
    }
    if (g.rope) __syncthreads();  // tlg is refilled by the next chunk
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float v = wave_max_dpp(mloc[jj]);
    if (lane == 0) red[wave][jj] = v;
  }
  __syncthreads();
  float M[GQ], lsum[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    M[jj] = fmaxf(fmaxf(red[0][jj], red[1][jj]), fmaxf(red[2][jj], red[3][jj]));
    lsum[jj] = 0.0f;
  }
  const int cq = tid & 31, sg = tid >> 5;
  float o[GQ][4];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) o[jj][0] = o[jj][1] = o[jj][2] = o[jj][3] = 0.0f;
  for (int c0 = 0; c0 < ntail; c0 += TCH) {
    const int n = c0 + tid;
    __syncthreads();
    if (g.rope) rope_chunk(c0);
    if (n < ntail) {
      float l[GQ];
      logits(n, c0, l);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        const float p = __builtin_amdgcn_exp2f(l[jj] - M[jj]);
        lsum[jj] += p;
        tl[tid][jj] = p;
      }
    }
    __syncthreads();
    const int cn = min(TCH, ntail - c0);
    for (int u = sg; u < cn; u += 8) {
      const int nn = c0 + u;
      const E* row = ((app && nn == n_app) ? vn : TV + (size_t)nn * D) + 4 * cq;
      float v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = Elem<DT>::get(row, i);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        const float w = tl[u][jj];
#pragma unroll
        for (int i = 0; i < 4; ++i) o[jj][i] = fmaf(w, v[i], o[jj][i]);
      }
    }
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float v = wave_sum_dpp(lsum[jj]);
    __syncthreads();
    if (lane == 0) red[wave][jj] = v;
    __syncthreads();
    lsum[jj] = (red[0][jj] + red[1][jj]) + (red[2][jj] + red[3][jj]);
  }
  const int Hq = g.Hq;
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[sg][4 * cq + i] = o[jj][i];
    __syncthreads();
    float* pr = dw.part + ((size_t)g.prefSp[b] * Hq + (size_t)(h * GQ + jj) * (nsp + 1) + nsp) * PS;
    if (tid < D) {
      float y = 0.0f;
#pragma unroll
      for (int qq = 0; qq < 8; ++qq) y += acc[qq][tid];
      pr[4 + tid] = y;
    }
    if (tid == 0) {
      pr[0] = ntail > 0 ? M[jj] : -INFINITY;
      pr[1] = lsum[jj];
    }
  }
}

// Append only, dense tail: copies the new key and value of every (request,
// KV head) into tail slot n_app.  Grid: B * H workgroups of D threads.
template <int DT>
__global__ __launch_bounds__(AKV_D) void k_app_dense(Geo g, Cache c, int n_app, const void* kin, const void* vin) {
  const size_t bh = blockIdx.x, d = threadIdx.x;
  const size_t ti = (bh * g.max_append + n_app) * AKV_D + d;
  Elem<DT>::put(c.tkd, ti, Elem<DT>::get(kin, bh * AKV_D + d));
  Elem<DT>::put(c.tvd, ti, Elem<DT>::get(vin, bh * AKV_D + d));
}

// Two fp32 values rounded to bf16 (round to nearest even) and packed, low first.
__device__ inline uint32_t pk_bf16(float a, float b) {
  typedef __attribute__((ext_vector_type(2))) float f2;
  typedef __attribute__((ext_vector_type(2))) __bf16 b2;
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){a, b}, b2));
}

// Key logits of every stored slot with positions encoded: LK[slot][j] =
// sl2 * q_j . R_p x^_p, p the slot's position and x^ = gamma abar (+ the
// dequantized residual r~ for a slot in R_K) the unrotated reconstruction of
// Eq. (reconstruction); R_p is linear, so the anchor part and the residual
// part are rotated and contracted separately.  One wave per 64 slots (one
// mask word):
//  - residuals first, one at a time (about 3 per word at a 5 % budget): lane l
//    holds coordinates 2l, 2l+1 of z^, the inverse Hadamard transform runs on
//    DPP lane moves, lanes l and l ^ 32 exchange the halves of each
//    rotate-half pair, and q_j . R_p r~ is a wave sum, kept in LDS per slot;
//  - then four 16-slot MFMA tiles of gamma abar: lane l holds coordinates
//    32 ks + 8 (l / 16) + e (ks < 4, e < 8) of slot l % 16, which pairs
//    coordinate f with f + 64 inside the lane; the rotated rows are contracted
//    with the g queries (bf16: hi and lo parts on v_mfma_f32_16x16x32_bf16;
//    fp32: v_mfma_f32_16x16x4f32 in the same coordinate order).
template <int DT, int GQ>
__global__ __launch_bounds__(256) void k_dec_rope_scores(Geo g, Cache c, DecWs dw, const void* q, float sl2) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D, F = AKV_D / 2;
  __shared__ float invs[F];
  __shared__ float rl[4][64][GQ];  // per wave: residual logit terms of its 64 slots
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < F) invs[tid] = g.invf[tid];
  for (int i = lane; i < 64 * GQ; i += 64) (&rl[wave][0][0])[i] = 0.0f;
  __syncthreads();
  // Consecutive logical blocks (the words of one head) share an XCD, so a
  // head's anchor rows stay in that XCD's L2.
  int blk = blockIdx.x;
  const int n8 = gridDim.x & ~7;
  if (blk < n8) blk = (blk & 7) * (n8 >> 3) + (blk >> 3);
  int gw = blk * 4 + wave;  // global mask word
  int b = 0;
  for (; b < g.B; ++b) {
    const int n = g.H * ((g.S[b] + 63) / 64);
    if (gw < n) break;
    gw -= n;
  }
  if (b >= g.B) return;
  const int S = g.S[b], k = g.k[b], nw = (S + 63) / 64;
  const int h = gw / nw, wi = gw % nw;
  const size_t so = slot_base(g, b, h) + (size_t)wi * 64;
  const size_t wo = (size_t)g.prefW[b] * g.H + (size_t)h * nw + wi;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const E* qg = (const E*)q + ((size_t)b * g.Hq + (size_t)h * GQ) * D;
  const uint2 mw2 = *(const uint2*)&c.maskK[wo];
  const unsigned long long mword = ((unsigned long long)__builtin_amdgcn_readfirstlane(mw2.y) << 32) |
                                   (unsigned)__builtin_amdgcn_readfirstlane(mw2.x);  // wave-uniform

  // ---- key residuals of the word: q_j . R_p r~
  if (mword) {
    const int pc0 = __builtin_amdgcn_readfirstlane(c.pcK[wo]);
    float q0[GQ], q1[GQ];
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) {
      q0[jj] = Elem<DT>::get(qg, (size_t)jj * D + 2 * lane);
      q1[jj] = Elem<DT>::get(qg, (size_t)jj * D + 2 * lane + 1);
    }
    const float if0 = invs[(2 * lane) & (F - 1)], if1 = invs[(2 * lane + 1) & (F - 1)];
    const float sg0 = sign_bit(g.sgnbits, 2 * lane), sg1 = sign_bit(g.sgnbits, 2 * lane + 1);
    const float invD = 1.0f / (float)D;
    const bool lo_half = lane < 32;
    unsigned long long m = mword;
    int rank = 0;
    while (m) {
      const int bit = __builtin_ctzll(m);
      m &= m - 1ull;
      const int slot = pc0 + rank++;
      const int p = c.pos[so + bit];
      const int nib = (c.codesK[(size_t)slot * (D / 4) + (lane >> 1)] >> (4 * (lane & 1))) & 15;
      const float sc = c.scalesK[(size_t)slot * (D / g.G) + (2 * lane) / g.G];
      float z0 = sc * level(g, nib & 3), z1 = sc * level(g, nib >> 2);
      if (g.rot) {
        fwht_wave_dpp(z0, z1, lane);
        z0 = (z0 * invD) * sg0;
        z1 = (z1 * invD) * sg1;
      }
      const float o0 = lane_xor<32>(z0), o1 = lane_xor<32>(z1);
      float c0, s0, c1, s1;
      rope_cs(if0, p, c0, s0);
      rope_cs(if1, p, c1, s1);
      // (r_f, r_{f+64}) -> (c r_f - s r_{f+64}, s r_f + c r_{f+64})
      const float r0 = lo_half ? fmaf(c0, z0, -(s0 * o0)) : fmaf(s0, o0, c0 * z0);
      const float r1 = lo_half ? fmaf(c1, z1, -(s1 * o1)) : fmaf(s1, o1, c1 * z1);
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        const float t = wave_sum_dpp(fmaf(q0[jj], r0, q1[jj] * r1));
        if (lane == 0) rl[wave][bit][jj] = t;
      }
    }
    // the tiles below read these terms from other lanes of this wave
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // ---- anchor parts: four 16-slot MFMA tiles
  const int i = lane & 15, kq = lane >> 4, col = i;
  // frequencies of the lane's 16 pairs, in revolutions per position
  double cf[2][8];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int e = 0; e < 8; ++e) cf[ks][e] = (double)invs[32 * ks + 8 * kq + e] * 0.15915494309189535;
  // queries as the B operand: lane supplies q_col[32 ks + 8 kq + e]
  const bool qv = col < GQ;
  const E* qp = qg + (size_t)(qv ? col : 0) * D;
  bf16x8 bq[DT == 1 ? 4 : 1];
  float qf[DT == 1 ? 1 : 4][8];
  if constexpr (DT == 1) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 v = qv ? *(const uint4*)((const uint16_t*)qp + 32 * ks + 8 * kq) : make_uint4(0, 0, 0, 0);
      bq[ks] = __builtin_bit_cast(bf16x8, v);
    }
  } else {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[ks][e] = qv ? Elem<DT>::get(qp, 32 * ks + 8 * kq + e) : 0.0f;
  }
  // records and anchor row chunks of one tile (loading the next tile's while
  // processing the current one measured slower: 89 against 78 us per 128K
  // layer-step, at three instead of four waves per SIMD)
  constexpr int NCH = DT == 1 ? 4 : 8;  // 16-byte chunks of the lane's 32 coordinates
  uint4 nxt[NCH];
  float ngm = 0.0f;
  int np = 0;
  auto fetch = [&](int tile) {
    const bool valid = wi * 64 + tile * 16 + i < S;
    const size_t sl = so + tile * 16 + i;
    const int a = valid ? min((int)c.idxK[sl], k - 1) : 0;
    ngm = valid ? Elem<DT>::get(c.gK, sl) : 0.0f;
    np = valid ? c.pos[sl] : 0;
    const E* ar = (const E*)c.ancK + (ko + a) * D;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int ks = DT == 1 ? u : u >> 1;
      nxt[u] = *(const uint4*)(ar + 32 * ks + 8 * kq + (DT == 1 ? 0 : 4 * (u & 1)));
    }
  };
  for (int tile = 0; tile < 4; ++tile) {
    fetch(tile);
    uint4 cur[NCH];
#pragma unroll
    for (int u = 0; u < NCH; ++u) cur[u] = nxt[u];
    const float gm = ngm;
    const int p = np;
    float x[4][8];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if constexpr (DT == 1) {
        const uint4 v = cur[ks];
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          x[ks][2 * u] = gm * __uint_as_float(w4[u] << 16);
          x[ks][2 * u + 1] = gm * __uint_as_float(w4[u] & 0xffff0000u);
        }
      } else {
        const uint4 v0 = cur[2 * ks], v1 = cur[2 * ks + 1];
        const float t8[8] = {__uint_as_float(v0.x), __uint_as_float(v0.y), __uint_as_float(v0.z),
                             __uint_as_float(v0.w), __uint_as_float(v1.x), __uint_as_float(v1.y),
                             __uint_as_float(v1.z), __uint_as_float(v1.w)};
#pragma unroll
        for (int e = 0; e < 8; ++e) x[ks][e] = gm * t8[e];
      }
    }
    // rotation of the pairs (f, f + 64) held as (x[ks][e], x[ks + 2][e])
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // revolutions in [0, 1): inside the hardware sine's input range
        const float r = (float)fract64((double)p * cf[ks][e]);
        const float cc = __builtin_amdgcn_cosf(r), ss = __builtin_amdgcn_sinf(r);
        const float u = x[ks][e], v = x[ks + 2][e];
        x[ks][e] = fmaf(cc, u, -(ss * v));
        x[ks + 2][e] = fmaf(ss, u, cc * v);
      }
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (DT == 1) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        uint32_t hw[4], lw[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float a0 = x[ks][2 * u], a1 = x[ks][2 * u + 1];
          hw[u] = pk_bf16(a0, a1);
          lw[u] = pk_bf16(a0 - __uint_as_float(hw[u] << 16), a1 - __uint_as_float(hw[u] & 0xffff0000u));
        }
        const bf16x8 ah = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
        const bf16x8 al = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bq[ks], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bq[ks], acc, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(x[ks][e], qf[ks][e], acc, 0, 0, 0);
    }
    // lane holds rows 4 kq + r (slots) of column col (query head)
    if (qv) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = tile * 16 + 4 * kq + r;
        if (wi * 64 + row < S) dw.LK[(so + row) * GQ + col] = (acc[r] + rl[wave][row][col]) * sl2;
      }
    }
  }
}

// ------------------------------------------------------------------ stream
// R uint16 values starting at p (R * 2 bytes, 8-byte aligned).
template <int R>
__device__ inline void load_u16(const uint16_t* p, uint16_t* v) {
#pragma unroll
  for (int i = 0; i < R / 4; ++i) {
    const uint2 x = *(const uint2*)(p + 4 * i);
    v[4 * i + 0] = (uint16_t)(x.x & 0xffff);
    v[4 * i + 1] = (uint16_t)(x.x >> 16);
    v[4 * i + 2] = (uint16_t)(x.y & 0xffff);
    v[4 * i + 3] = (uint16_t)(x.y >> 16);
  }
}
template <int DT, int R>
__device__ inline void load_coef(const void* base, size_t i0, float* v) {
  if constexpr (DT == 1) {
    uint16_t t[R];
    load_u16<R>((const uint16_t*)base + i0, t);
#pragma unroll
    for (int i = 0; i < R; ++i) v[i] = bf2f(t[i]);
  } else {
#pragma unroll
    for (int i = 0; i < R / 4; ++i) {
      const float4 x = *(const float4*)((const float*)base + i0 + 4 * i);
      v[4 * i] = x.x;
      v[4 * i + 1] = x.y;
      v[4 * i + 2] = x.z;
      v[4 * i + 3] = x.w;
    }
  }
}
__device__ inline unsigned long long low_bits(int n) { return n >= 64 ? ~0ull : ((1ull << n) - 1ull); }

// Per-wave LDS of the streaming kernel.
constexpr int SW_VCH = 64;  // value residuals staged per chunk
constexpr int SW_ACH = 64;  // anchors per weight window
constexpr int SW_AST = 16;  // value-anchor rows staged per wave
template <int DT, int GQ>
struct alignas(16) StreamWaveLds {
  uint32_t vcode[SW_VCH][8];
  float vsc[SW_VCH][4];
  float vp[SW_VCH][GQ];
  float wacc[SW_ACH][GQ];
  float2 lvl[16];  // the two levels of a coordinate pair, by its 4-bit code
  typename Elem<DT>::T avs[SW_AST * AKV_D];
};

// Orders this wave's LDS writes before its later LDS reads (and vice versa).
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Grid: nst split workgroups, then one tail workgroup per (request, KV head)
// (which first resolves this step's appended token when kin != nullptr).
// A split of 256 R sorted slots is processed as four independent wave
// sub-splits of 64 R slots (own softmax statistics, value residuals, anchor
// weights); one barrier at the end combines them, and the inverse rotation is
// applied once per query head.
template <int DT, int GQ, int R>
__global__ __launch_bounds__(256) void k_dec_stream(Geo g, Cache c, DecWs dw, int nst, int n_app, const void* kin,
                                                    const void* vin, const void* q, float sl2) {
  using E = typename Elem<DT>::T;
  using WL = StreamWaveLds<DT, GQ>;
  constexpr int D = AKV_D, LW = 64 * R, L = 4 * LW, PER = 16 / sizeof(E);
  constexpr int NAVW = SW_AST * D / PER / 64;  // 16-byte anchor-row chunks per lane
  constexpr int ZY_B = 2 * 4 * GQ * D * 4;
  constexpr int WL_B = 4 * (int)sizeof(WL);
  constexpr int TAIL_E = 256 * GQ * 4 + 256 * 4 + 8 * D * 4 + GQ * D * 4 + D * 2 + 256 * GQ * 4,
                TAIL_D = GQ * D * 4 + 256 * GQ * 4 + 8 * D * 4 + D * 2 + 256 * GQ * 4;
  constexpr int TAIL_B = TAIL_E > TAIL_D ? TAIL_E : TAIL_D;
  constexpr int POOL_B = (WL_B > ZY_B ? WL_B : ZY_B) > TAIL_B ? (WL_B > ZY_B ? WL_B : ZY_B) : TAIL_B;
  __shared__ __align__(16) unsigned char pool[POOL_B];
  __shared__ float wm[4][GQ], wl[4][GQ];
  if ((int)blockIdx.x >= nst) {
    if (g.dense_tail)
      tail_dense<DT, GQ>(g, c, dw, (int)blockIdx.x - nst, n_app, kin, vin, q, sl2, pool);
    else
      tail_block<DT, GQ>(g, c, dw, (int)blockIdx.x - nst, n_app, kin, vin, q, sl2, pool);
    return;
  }
  // Logical block id: consecutive ids (the splits of one head) share an XCD.
  int id = blockIdx.x;
  const int n8 = nst & ~7;
  if (id < n8) id = (id & 7) * (n8 >> 3) + (id >> 3);
  const int b = locate(g, L, 1, id);
  const int S = g.S[b], k = g.k[b], G = g.G, kp = (k + 3) & ~3;
  const int nsp = (S + L - 1) / L;
  const int h = id / nsp, sp = id % nsp;
  const int s0 = sp * L, s1 = min(S, s0 + L);
  const int nw = (S + 63) / 64;
  const size_t so = slot_base(g, b, h);
  const size_t wo = (size_t)g.prefW[b] * g.H + (size_t)h * nw;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const float* SKh = dw.SK + ((size_t)g.prefKp[b] * g.H + (size_t)h * kp) * GQ;
  const E* AVg = (const E*)c.ancV + ko * D;
  WL& W = ((WL*)pool)[wave];

  float za[GQ][2], ya[GQ][2], mw[GQ], lsw[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    za[jj][0] = za[jj][1] = ya[jj][0] = ya[jj][1] = 0.0f;
    mw[jj] = -INFINITY;
    lsw[jj] = 0.0f;
  }
  const int ws0 = s0 + wave * LW, ws1 = min(s1, ws0 + LW);
  if (ws0 < ws1) {
    for (int i = lane; i < SW_ACH * GQ; i += 64) (&W.wacc[0][0])[i] = 0.0f;
    if (lane < 16) W.lvl[lane] = make_float2(level(g, lane & 3), level(g, lane >> 2));

    // ---- round 1: records and flag words of this wave's slots.  Every
    // lane reads raw words (a lane past the split end re-reads the wave's
    // first group and discards it), all loads are issued before any is
    // unpacked.
    const int i0 = ws0 + lane * R;
    const bool any = i0 < ws1;
    const int i0c = any ? i0 : ws0;
    uint16_t ik[R], iv[R];
    float gk[R], gv[R];
    unsigned long long wk, wv;
    int pck, pcv;
    float lg[R][GQ];
    if (g.rope) {  // positions encoded: the slots' whole key logits (residuals included), by slot index
#pragma unroll
      for (int r = 0; r < R; ++r) load_g<GQ>(dw.LK + (so + i0c + r) * GQ, lg[r]);
    }
    {
      constexpr int NU = R / 4;                       // uint2 words per index array
      constexpr int NG = DT == 1 ? R / 4 : R / 2;     // uint2 words per coefficient array
      uint2 rik[NU], riv[NU], rgk[NG], rgv[NG];
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        rik[u] = ((const uint2*)(c.idxK + so + i0c))[u];
        riv[u] = ((const uint2*)(c.idxV + so + i0c))[u];
      }
#pragma unroll
      for (int u = 0; u < NG; ++u) {
        rgk[u] = ((const uint2*)((const E*)c.gK + so + i0c))[u];
        rgv[u] = ((const uint2*)((const E*)c.gV + so + i0c))[u];
      }
      wk = c.maskK[wo + (i0c >> 6)];
      wv = c.maskV[wo + (i0c >> 6)];
      pck = c.pcK[wo + (i0c >> 6)];
      pcv = c.pcV[wo + (i0c >> 6)];
      __builtin_amdgcn_sched_barrier(0);  // all loads above are issued before the unpacking
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        ik[4 * u] = (uint16_t)(rik[u].x & 0xffff);
        ik[4 * u + 1] = (uint16_t)(rik[u].x >> 16);
        ik[4 * u + 2] = (uint16_t)(rik[u].y & 0xffff);
        ik[4 * u + 3] = (uint16_t)(rik[u].y >> 16);
        iv[4 * u] = (uint16_t)(riv[u].x & 0xffff);
        iv[4 * u + 1] = (uint16_t)(riv[u].x >> 16);
        iv[4 * u + 2] = (uint16_t)(riv[u].y & 0xffff);
        iv[4 * u + 3] = (uint16_t)(riv[u].y >> 16);
      }
#pragma unroll
      for (int u = 0; u < NG; ++u) {
        if constexpr (DT == 1) {
          gk[4 * u] = bf2f((uint16_t)(rgk[u].x & 0xffff));
          gk[4 * u + 1] = bf2f((uint16_t)(rgk[u].x >> 16));
          gk[4 * u + 2] = bf2f((uint16_t)(rgk[u].y & 0xffff));
          gk[4 * u + 3] = bf2f((uint16_t)(rgk[u].y >> 16));
          gv[4 * u] = bf2f((uint16_t)(rgv[u].x & 0xffff));
          gv[4 * u + 1] = bf2f((uint16_t)(rgv[u].x >> 16));
          gv[4 * u + 2] = bf2f((uint16_t)(rgv[u].y & 0xffff));
          gv[4 * u + 3] = bf2f((uint16_t)(rgv[u].y >> 16));
        } else {
          gk[2 * u] = __uint_as_float(rgk[u].x);
          gk[2 * u + 1] = __uint_as_float(rgk[u].y);
          gv[2 * u] = __uint_as_float(rgv[u].x);
          gv[2 * u + 1] = __uint_as_float(rgv[u].y);
        }
      }
      if (!any) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          ik[r] = iv[r] = 0;
          gk[r] = gv[r] = 0.0f;
        }
        wk = wv = 0;
        pck = pcv = 0;
      }
    }
    const int nval = max(0, min(R, ws1 - i0));  // valid slots of this lane (a prefix)
    const int sh = i0 & 63;
    const uint32_t vmask = nval >= 32 ? ~0u : ((1u << nval) - 1u);
    const uint32_t bk = (uint32_t)(wk >> sh) & vmask, bv = (uint32_t)(wv >> sh) & vmask;
    pck += __popcll(wk & low_bits(sh));
    pcv += __popcll(wv & low_bits(sh));
    int aLast = iv[0];
#pragma unroll
    for (int r = 1; r < R; ++r)
      if (r < nval) aLast = iv[r];
    const int lastl = (ws1 - ws0 - 1) / R;  // last lane with a valid slot (uniform)
    const int a_lo = __builtin_amdgcn_readfirstlane(iv[0]);
    const int a_hi = __builtin_amdgcn_readlane(aLast, lastl);
    const int pv_lo = __builtin_amdgcn_readfirstlane(pcv);
    const int pv_hi = __builtin_amdgcn_readlane(pcv + __popc(bv), lastl);
    const int nrange = a_hi - a_lo + 1, nstage = min(nrange, SW_AST), nvres = pv_hi - pv_lo;

    // ---- round 2: anchor scores, key-residual terms, anchor rows, first value residuals.
    float rk[R][GQ];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (g.rope) {  // the logits were loaded with the records
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) rk[r][jj] = 0.0f;
        continue;
      }
      load_g<GQ>(SKh + (size_t)min((int)ik[r], k - 1) * GQ, lg[r]);
      if ((bk >> r) & 1u) {
        load_g<GQ>(dw.RK + (size_t)(pck + __popc(bk & ((1u << r) - 1u))) * GQ, rk[r]);
      } else {
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) rk[r][jj] = 0.0f;
      }
    }
    uint4 avr[NAVW];
#pragma unroll
    for (int i = 0; i < NAVW; ++i) {
      const int ch = lane + 64 * i;
      const int row = ch / (D / PER), col = (ch % (D / PER)) * PER;
      avr[i] = row < nstage ? *(const uint4*)(AVg + (size_t)(a_lo + row) * D + col) : make_uint4(0, 0, 0, 0);
    }
    auto load_vchunk = [&](int cb, uint4& c0, uint4& c1, float* sv) {
      const int nv = min(SW_VCH, nvres - cb);
      if (lane < nv) {
        const uint4* cp = (const uint4*)(c.codesV + (size_t)(pv_lo + cb + lane) * (D / 4));
        c0 = cp[0];
        c1 = cp[1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int f = lane + 64 * u;
        sv[u] = f < nv * (D / G) ? c.scalesV[(size_t)(pv_lo + cb) * (D / G) + f] : 0.0f;
      }
    };
    auto stage_vchunk = [&](int cb, const uint4& c0, const uint4& c1, const float* sv) {
      const int nv = min(SW_VCH, nvres - cb);
      if (lane < nv) {
        *(uint4*)&W.vcode[lane][0] = c0;
        *(uint4*)&W.vcode[lane][4] = c1;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int f = lane + 64 * u;
        if (f < nv * (D / G)) W.vsc[f / (D / G)][f % (D / G)] = sv[u];
      }
    };
    uint4 vc0 = make_uint4(0, 0, 0, 0), vc1 = make_uint4(0, 0, 0, 0);
    float vsv[4];
    load_vchunk(0, vc0, vc1, vsv);

    // ---- logits (base 2) and this wave's softmax statistics.
    if (!g.rope) {
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) lg[r][jj] = fmaf(gk[r], lg[r][jj], rk[r][jj]);
    }
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) {
      float v = -INFINITY;
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (r < nval) v = fmaxf(v, lg[r][jj]);
      mw[jj] = wave_max_dpp(v);
      float sum = 0.0f;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const float p = r < nval ? __builtin_amdgcn_exp2f(lg[r][jj] - mw[jj]) : 0.0f;
        lg[r][jj] = p;
        sum += p;
      }
      lsw[jj] = wave_sum_dpp(sum);
    }
    // Stage the anchor rows and the first residual chunk.
#pragma unroll
    for (int i = 0; i < NAVW; ++i) {
      const int ch = lane + 64 * i;
      const int row = ch / (D / PER), col = (ch % (D / PER)) * PER;
      *(uint4*)&W.avs[row * D + col] = avr[i];
    }
    stage_vchunk(0, vc0, vc1, vsv);

    // ---- value residuals in the rotated basis: lane = coordinate pair.
    const int grp = (2 * lane) / G, nsh = 4 * (lane & 7);
    auto vres_acc = [&](uint32_t word, float sgv, const float* pv) {
      const float2 lv = W.lvl[(word >> nsh) & 15];
      const float z0 = sgv * lv.x, z1 = sgv * lv.y;
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        za[jj][0] = fmaf(pv[jj], z0, za[jj][0]);
        za[jj][1] = fmaf(pv[jj], z1, za[jj][1]);
      }
    };
    for (int cb = 0; cb < nvres; cb += SW_VCH) {
      const int nv = min(SW_VCH, nvres - cb);
      if (cb > 0) {
        wave_lds_sync();
        load_vchunk(cb, vc0, vc1, vsv);
        stage_vchunk(cb, vc0, vc1, vsv);
      }
#pragma unroll
      for (int r = 0; r < R; ++r)
        if ((bv >> r) & 1u) {
          const int li = pcv + __popc(bv & ((1u << r) - 1u)) - pv_lo - cb;
          if (li >= 0 && li < nv) store_g<GQ>(&W.vp[li][0], lg[r]);
        }
      wave_lds_sync();
      int e = 0;
      for (; e + 3 < nv; e += 4) {
        uint32_t wd[4];
        float sg4[4], pv[4][GQ];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          wd[u] = W.vcode[e + u][lane >> 3];
          sg4[u] = W.vsc[e + u][grp];
          load_g<GQ>(&W.vp[e + u][0], pv[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) vres_acc(wd[u], sg4[u], pv[u]);
      }
      for (; e < nv; ++e) {
        float pv[GQ];
        load_g<GQ>(&W.vp[e][0], pv);
        vres_acc(W.vcode[e][lane >> 3], W.vsc[e][grp], pv);
      }
    }

    // ---- per-anchor value weights (first/last run of each lane's slots) and
    // y = sum_a w_a abar^V_a, in windows of SW_ACH anchors.
    auto vpair = [&](const E* p, float& v0, float& v1) {
      if constexpr (DT == 1) {
        const uint32_t t = *(const uint32_t*)(p + 2 * lane);
        v0 = bf2f((uint16_t)(t & 0xffffu));
        v1 = bf2f((uint16_t)(t >> 16));
      } else {
        const float2 t = *(const float2*)(p + 2 * lane);
        v0 = t.x;
        v1 = t.y;
      }
    };
    auto yacc = [&](float v0, float v1, const float* w) {
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        ya[jj][0] = fmaf(w[jj], v0, ya[jj][0]);
        ya[jj][1] = fmaf(w[jj], v1, ya[jj][1]);
      }
    };
    const int aF = iv[0];
    float rf[GQ], rl[GQ];
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) rf[jj] = rl[jj] = 0.0f;
    bool mid = false;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const bool v = r < nval;
      const bool isF = v && (int)iv[r] == aF, isL = v && !isF && (int)iv[r] == aLast;
      mid |= v && !isF && !isL;
      const float wF = isF ? gv[r] : 0.0f, wL = isL ? gv[r] : 0.0f;
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) {
        rf[jj] = fmaf(lg[r][jj], wF, rf[jj]);
        rl[jj] = fmaf(lg[r][jj], wL, rl[jj]);
      }
    }
    for (int wb = 0; wb < nrange; wb += SW_ACH) {
      const int wn = min(SW_ACH, nrange - wb);
      if (wb > 0) {
        wave_lds_sync();
        for (int i = lane; i < SW_ACH * GQ; i += 64) (&W.wacc[0][0])[i] = 0.0f;
        wave_lds_sync();
      }
      const int oF = aF - a_lo - wb, oL = aLast - a_lo - wb;
      if (nval > 0 && oF >= 0 && oF < wn) {
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) atomicAdd(&W.wacc[oF][jj], rf[jj]);
      }
      if (nval > 0 && aLast != aF && oL >= 0 && oL < wn) {
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) atomicAdd(&W.wacc[oL][jj], rl[jj]);
      }
      if (mid) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int o = (int)iv[r] - a_lo - wb;
          if (r < nval && (int)iv[r] != aF && (int)iv[r] != aLast && o >= 0 && o < wn) {
#pragma unroll
            for (int jj = 0; jj < GQ; ++jj) atomicAdd(&W.wacc[o][jj], lg[r][jj] * gv[r]);
          }
        }
      }
      wave_lds_sync();
      const int wl_ = max(0, min(wn, nstage - wb));  // rows of this window staged in LDS
      int a = 0;
      for (; a + 3 < wl_; a += 4) {
        float v0[4], v1[4], w[4][GQ];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          vpair(W.avs + (size_t)(wb + a + u) * D, v0[u], v1[u]);
          load_g<GQ>(&W.wacc[a + u][0], w[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) yacc(v0[u], v1[u], w[u]);
      }
      for (; a < wl_; ++a) {
        float v0, v1, w[GQ];
        vpair(W.avs + (size_t)(wb + a) * D, v0, v1);
        load_g<GQ>(&W.wacc[a][0], w);
        yacc(v0, v1, w);
      }
      for (; a < wn; ++a) {  // rows past the staged ones
        float v0, v1, w[GQ];
        vpair(AVg + (size_t)(a_lo + wb + a) * D, v0, v1);
        load_g<GQ>(&W.wacc[a][0], w);
        yacc(v0, v1, w);
      }
    }
  }

  // ---- combine the four wave sub-splits: o = y + s * FWHT(zacc) / D per query head.
  if (lane == 0) {
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) {
      wm[wave][jj] = mw[jj];
      wl[wave][jj] = lsw[jj];
    }
  }
  __syncthreads();  // the pool now holds the per-wave partials
  float(*zp)[GQ][D] = (float(*)[GQ][D])pool;
  float(*yp)[GQ][D] = (float(*)[GQ][D])(pool + 4 * GQ * D * 4);
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    *(float2*)&zp[wave][jj][2 * lane] = make_float2(za[jj][0], za[jj][1]);
    *(float2*)&yp[wave][jj][2 * lane] = make_float2(ya[jj][0], ya[jj][1]);
  }
  __syncthreads();
  const int Hq = g.Hq;
  const float s0v = sign_bit(g.sgnbits, 2 * lane), s1v = sign_bit(g.sgnbits, 2 * lane + 1);
  const float invD = 1.0f / (float)D;
  for (int jj = wave; jj < GQ; jj += 4) {
    const float M = fmaxf(fmaxf(wm[0][jj], wm[1][jj]), fmaxf(wm[2][jj], wm[3][jj]));
    float z0 = 0.0f, z1 = 0.0f, y0 = 0.0f, y1 = 0.0f, l = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = wm[w][jj] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(wm[w][jj] - M);
      z0 = fmaf(f, zp[w][jj][2 * lane], z0);
      z1 = fmaf(f, zp[w][jj][2 * lane + 1], z1);
      y0 = fmaf(f, yp[w][jj][2 * lane], y0);
      y1 = fmaf(f, yp[w][jj][2 * lane + 1], y1);
      l = fmaf(f, wl[w][jj], l);
    }
    float o0, o1;
    if (g.rot) {
      fwht_wave_dpp(z0, z1, lane);
      o0 = y0 + s0v * (z0 * invD);
      o1 = y1 + s1v * (z1 * invD);
    } else {
      o0 = y0 + z0;
      o1 = y1 + z1;
    }
    float* pr = dw.part + ((size_t)g.prefSp[b] * Hq + (size_t)(h * GQ + jj) * (nsp + 1) + sp) * PS;
    if (lane == 0) {
      pr[0] = M;
      pr[1] = l;
    }
    *(float2*)&pr[4 + 2 * lane] = make_float2(o0, o1);
  }
}

// ------------------------------------------------------------------ merge
// One workgroup per (request, query head): merges its nsp + 1 split records
// (the last one holds the appended tail) in one pass.  Thread t owns output
// coordinates 4 (t % 32) .. +3 of every 8th record; the record maxima and
// values are loaded together, 128 records per round.
template <int DT, int GQ>
__global__ __launch_bounds__(256) void k_dec_merge(Geo g, DecWs dw, void* out, int out_dtype) {
  constexpr int D = AKV_D, RCH = 128;
  __shared__ float red[4];
  __shared__ __align__(16) float acc[8][D];
  const int b = blockIdx.x / g.Hq, jq = blockIdx.x % g.Hq;
  const int nrec = (g.S[b] + g.dsplit - 1) / g.dsplit + 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cq = tid & 31, sg = tid >> 5;
  const float* pb = dw.part + ((size_t)g.prefSp[b] * g.Hq + (size_t)jq * nrec) * PS;
  // Maxima and sums of the first 256 records are loaded once, beside the
  // first round of record values (issued before the max is known).
  const float m0 = tid < nrec ? pb[(size_t)tid * PS] : -INFINITY;
  const float l0 = tid < nrec ? pb[(size_t)tid * PS + 1] : 0.0f;
  float M = m0;
  for (int s = tid + 256; s < nrec; s += 256) M = fmaxf(M, pb[(size_t)s * PS]);
  float4 v[RCH / 8];
  float mv[RCH / 8];
#pragma unroll
  for (int j = 0; j < RCH / 8; ++j) {
    const int s = min(sg + 8 * j, nrec - 1);
    v[j] = *(const float4*)&pb[(size_t)s * PS + 4 + 4 * cq];
    mv[j] = pb[(size_t)s * PS];
  }
  M = wave_max_dpp(M);
  if (lane == 0) red[wave] = M;
  __syncthreads();
  M = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float l = tid < nrec ? __builtin_amdgcn_exp2f(m0 - M) * l0 : 0.0f;
  for (int s = tid + 256; s < nrec; s += 256) l = fmaf(__builtin_amdgcn_exp2f(pb[(size_t)s * PS] - M), pb[(size_t)s * PS + 1], l);
  float o[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int c0 = 0; c0 < nrec; c0 += RCH) {
    if (c0 > 0) {
#pragma unroll
      for (int j = 0; j < RCH / 8; ++j) {
        const int s = min(c0 + sg + 8 * j, nrec - 1);
        v[j] = *(const float4*)&pb[(size_t)s * PS + 4 + 4 * cq];
        mv[j] = pb[(size_t)s * PS];
      }
    }
#pragma unroll
    for (int j = 0; j < RCH / 8; ++j) {
      const float w = c0 + sg + 8 * j < nrec ? __builtin_amdgcn_exp2f(mv[j] - M) : 0.0f;
      o[0] = fmaf(w, v[j].x, o[0]);
      o[1] = fmaf(w, v[j].y, o[1]);
      o[2] = fmaf(w, v[j].z, o[2]);
      o[3] = fmaf(w, v[j].w, o[3]);
    }
  }
  l = wave_sum_dpp(l);
  __syncthreads();
  if (lane == 0) red[wave] = l;
  *(float4*)&acc[sg][4 * cq] = make_float4(o[0], o[1], o[2], o[3]);
  __syncthreads();
  if (tid < D) {
    const float lt = (red[0] + red[1]) + (red[2] + red[3]);
    float y = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) y += acc[q][tid];
    const size_t oi = ((size_t)b * g.Hq + jq) * D + tid;
    if (out_dtype == 1) ((uint16_t*)out)[oi] = f2bf(y / lt); else ((float*)out)[oi] = y / lt;
  }
}

// ------------------------------------------------------------------ reconstruct
template <int DT>
__global__ __launch_bounds__(256) void k_reconstruct(Geo g, Cache c, int b, int side, int n_app, float* out) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D;
  const int lane = threadIdx.x & 63;
  const int S = g.S[b], k = g.k[b], G = g.G;
  const int rows = S + n_app;
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int h = gw / rows, i = gw % rows;
  if (h >= g.H) return;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  int a, t;
  float gb;
  bool res = false;
  int slot = 0;
  if (i < S) {
    const size_t so = slot_base(g, b, h);
    t = min(max(c.pos[so + i], 0), S - 1);
    a = min((int)(side ? c.idxV : c.idxK)[so + i], k - 1);
    gb = Elem<DT>::get(side ? c.gV : c.gK, so + i);
    const size_t wo = (size_t)g.prefW[b] * g.H + (size_t)h * ((S + 63) / 64) + (i >> 6);
    const unsigned long long wm = (side ? c.maskV : c.maskK)[wo];
    res = (wm >> (i & 63)) & 1ull;
    slot = (side ? c.pcV : c.pcK)[wo] + __popcll(wm & ((1ull << (i & 63)) - 1ull));
  } else {
    const size_t ti = ((size_t)b * g.H + h) * g.max_append + (i - S);
    if (g.dense_tail) {  // stored exactly
      const void* X = side ? c.tvd : c.tkd;
      float* o = out + ((size_t)h * rows + i) * D;
      o[2 * lane] = Elem<DT>::get(X, ti * D + 2 * lane);
      o[2 * lane + 1] = Elem<DT>::get(X, ti * D + 2 * lane + 1);
      return;
    }
    t = i;
    a = min((int)(side ? c.tidxV : c.tidxK)[ti], k - 1);
    gb = Elem<DT>::get(side ? c.tgV : c.tgK, ti);
  }
  const E* ar = A + (size_t)a * D;
  float x0 = gb * Elem<DT>::get(ar, 2 * lane), x1 = gb * Elem<DT>::get(ar, 2 * lane + 1);
  if (res) {
    const uint8_t* cd = (side ? c.codesV : c.codesK) + (size_t)slot * (D / 4);
    const float sg = (side ? c.scalesV : c.scalesK)[(size_t)slot * (D / G) + (2 * lane) / G];
    const int nib = (cd[lane / 2] >> (4 * (lane & 1))) & 15;
    float z0 = sg * level(g, nib & 3), z1 = sg * level(g, nib >> 2);
    if (g.rot) {
      fwht_wave(z0, z1, lane);
      const float invD = 1.0f / (float)D;
      z0 = (z0 * invD) * hsign(g.seed_sign, 2 * lane);
      z1 = (z1 * invD) * hsign(g.seed_sign, 2 * lane + 1);
    }
    x0 = x0 + z0;
    x1 = x1 + z1;
  }
  float* o = out + ((size_t)h * rows + t) * D;
  o[2 * lane] = x0;
  o[2 * lane + 1] = x1;
}

// ------------------------------------------------------------------ launchers
template <int DT, int GQ>
static void launch_steps(const Geo& g, const Cache& c, const DecWs& dw, const void* q, const void* kn,
                         const void* vn, void* out, int out_dtype, float scale, int n_app, bool attn, bool app,
                         hipStream_t st) {
  // A dense tail needs no anchor screening for the appended token: the tail
  // workgroups store it (or k_app_dense, for an append alone).
  const bool screen = app && !g.dense_tail;
  if (!attn && !screen) {
    launch("k_app_dense", k_app_dense<DT>, dim3(g.B * g.H), dim3(AKV_D), 0, st, g, c, n_app, kn, vn);
    return;
  }
  // With positions encoded the anchor scores and key-residual terms are
  // replaced by the per-slot logits of k_dec_rope_scores; the front kernel
  // then only screens an appended token.
  const bool sk = attn && !g.rope;
  const int nAK = (sk || screen) ? g.H * g.prefAB[g.B] : 0;
  const int nAV = screen ? g.H * g.prefAB[g.B] : 0;
  const int nR = sk ? (g.prefNK[g.B] + RK_PER_BLOCK - 1) / RK_PER_BLOCK : 0;
  const int flags = (sk ? 1 : 0) | (screen ? 2 : 0);
  const float sl2 = scale * 1.4426950408889634f;
  if (nAK + nAV + nR > 0)
    launch("k_dec_front", k_dec_front<DT, GQ>, dim3(nAK + nAV + nR), dim3(256), 0, st, g, c, dw, q, kn, vn, flags, nAK,
           nAV, sl2);
  if (!attn) {
    launch("k_app_finish", k_app_finish<DT>, dim3(g.B * g.H), dim3(256), 0, st, g, c, dw, n_app, kn, vn);
    return;
  }
  if (g.rope) {
    const int nwords = g.H * g.prefW[g.B];
    launch("k_dec_rope_scores", k_dec_rope_scores<DT, GQ>, dim3((nwords + 3) / 4), dim3(256), 0, st, g, c, dw, q, sl2);
  }
  const int L = g.dsplit;
  int nst = 0;
  for (int b = 0; b < g.B; ++b) nst += g.H * ((g.S[b] + L - 1) / L);
  const int ntb = g.B * g.H;  // tail workgroups
  if (L == 2048) {
    launch("k_dec_stream", k_dec_stream<DT, GQ, 8>, dim3(nst + ntb), dim3(256), 0, st, g, c, dw, nst, n_app, kn, vn, q,
           sl2);
  } else {
    launch("k_dec_stream", k_dec_stream<DT, GQ, 4>, dim3(nst + ntb), dim3(256), 0, st, g, c, dw, nst, n_app, kn, vn, q,
           sl2);
  }
  launch("k_dec_merge", k_dec_merge<DT, GQ>, dim3(g.B * g.Hq), dim3(256), 0, st, g, dw, out, out_dtype);
}

template <int DT>
static void launch_steps_g(const Geo& g, const Cache& c, const DecWs& dw, const void* q, const void* kn,
                           const void* vn, void* out, int out_dtype, float scale, int n_app, bool attn, bool app,
                           hipStream_t st) {
  // An append alone needs no query-head grouping: one instantiation serves.
  const int gq = attn ? g.g : 1;
  switch (gq) {
    case 1: launch_steps<DT, 1>(g, c, dw, q, kn, vn, out, out_dtype, scale, n_app, attn, app, st); break;
    case 2: launch_steps<DT, 2>(g, c, dw, q, kn, vn, out, out_dtype, scale, n_app, attn, app, st); break;
    case 4: launch_steps<DT, 4>(g, c, dw, q, kn, vn, out, out_dtype, scale, n_app, attn, app, st); break;
    default: launch_steps<DT, 8>(g, c, dw, q, kn, vn, out, out_dtype, scale, n_app, attn, app, st); break;
  }
}

// q == nullptr: append only; kn == nullptr: attention only; both: append the
// token as tail slot n_app, then attend over it too.
hipError_t launch_decode(const Geo& g, const Cache& c, const DecWs& dw, const void* q, const void* kn,
                         const void* vn, void* out, int out_dtype, float scale, int n_app, hipStream_t st) {
  const bool attn = q != nullptr, app = kn != nullptr;
  if (g.dtype == 1)
    launch_steps_g<1>(g, c, dw, q, kn, vn, out, out_dtype, scale, n_app, attn, app, st);
  else
    launch_steps_g<0>(g, c, dw, q, kn, vn, out, out_dtype, scale, n_app, attn, app, st);
  return hipGetLastError();
}

hipError_t launch_reconstruct(const Geo& g, const Cache& c, int b, int side, int n_app, float* out, hipStream_t st) {
  const int rows = g.S[b] + n_app;
  const int nblk = (g.H * rows + 3) / 4;
  if (g.dtype == 1) {
    launch("k_reconstruct", k_reconstruct<1>, dim3(nblk), dim3(256), 0, st, g, c, b, side, n_app, out);
  } else {
    launch("k_reconstruct", k_reconstruct<0>, dim3(nblk), dim3(256), 0, st, g, c, b, side, n_app, out);
  }
  return hipGetLastError();
}

}  // namespace akv
