// Decode attention over the compressed cache (Sec. 3.4 "Storage and
// Decoding"; App. E.1) and the two cache services around it.
//
// Attention of query j (KV head h = j / g) over every stored entry t:
//   logit_t = scale * (gamma^K_t (q_j . abar^K_a(t)) + [t in R_K] q_rot . zhat^K_t / D)
//   out     = (sum_a w_a abar^V_a + s * FWHT(sum_t p_t zhat^V_t) / D) / sum_t p_t
// with p_t = exp(logit_t - max), w_a = sum over tokens of value anchor a of
// p_t gamma^V_t, zhat the dequantized rotated residual and q_rot = FWHT(s * q).
// This is the exact algebra of attention over the reconstructed cache (Eq.
// reconstruction): U is orthogonal and linear, so the inverse rotation of the
// value residuals is applied once per query instead of once per token, and
// the key residual term is a dot product in the rotated basis.
//
//   k_dec_scores : everything that depends only on the queries, fully parallel:
//                  the anchor scores S_K[j][a] = q_j . abar^K_a (one thread per
//                  anchor, the row in registers) and the key-residual terms
//                  q_rot . zhat^K_t / D (one thread per stored key residual);
//   k_dec_stream : split-K pass over the value-anchor-grouped records.  Loads
//                  are issued in two rounds (records, flags, the score table;
//                  then key-residual terms, value-anchor rows and value
//                  residual codes); per split it writes the partial (max, sum,
//                  sum_a w_a abar^V_a, rotated value-residual sum).  Blocks are
//                  mapped so that all splits of one head share one XCD (and its
//                  L2) for the score table and the anchor rows;
//   k_dec_combine: merges the splits, adds appended tokens, applies the
//                  inverse rotation once and normalizes.
//   k_append     : encodes one new key/value per head against the existing
//                  anchors (certified argmax, canonical fp64 coefficient).
//   k_reconstruct: dense x^ of one side of one request (Eq. reconstruction).
#include "akv_common.h"

namespace akv {

__device__ inline float level(int code) {
  // 0 -> -L1, 1 -> -L0, 2 -> +L0, 3 -> +L1
  const float mag = (code == 0 || code == 3) ? AKV_L1 : AKV_L0;
  return code < 2 ? -mag : mag;
}

// sigma * level(code) from the group's four precomputed values.
__device__ inline float scaled_level(int code, float n1, float n0, float p0, float p1) {
  const float lo = (code & 1) ? n0 : n1;
  const float hi = (code & 1) ? p1 : p0;
  return (code & 2) ? hi : lo;
}

// ------------------------------------------------------------------ D1
template <int DT>
__global__ __launch_bounds__(256) void k_dec_scores(Geo g, Cache c, DecWs dw, const void* qin) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D;
  constexpr int PER = 16 / sizeof(E);
  __shared__ float qs[8][D];
  const int gq = g.g;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int idx = blockIdx.x;
  int nsc = 0;
  for (int b = 0; b < g.B; ++b) nsc += g.H * ((g.k[b] + 255) / 256);
  if (idx < nsc) {
    // ---- anchor scores
    int b = 0;
    for (; b < g.B; ++b) {
      const int n = g.H * ((g.k[b] + 255) / 256);
      if (idx < n) break;
      idx -= n;
    }
    const int k = g.k[b], kp = (k + 3) & ~3;
    const int nch = (k + 255) / 256;
    const int h = idx / nch, a0 = (idx % nch) * 256;
    const int a = a0 + threadIdx.x;
    const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
    const E* row = (const E*)c.ancK + (ko + min(a, k - 1)) * D;
    uint4 rv[D / PER];
#pragma unroll
    for (int i = 0; i < D / PER; ++i) rv[i] = *(const uint4*)(row + i * PER);
    const E* q = (const E*)qin + ((size_t)b * g.Hq + (size_t)h * gq) * D;
    for (int i = threadIdx.x; i < gq * D; i += 256) qs[i / D][i % D] = Elem<DT>::get(q, i);
    __syncthreads();
    float acc[8];
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) acc[jj] = 0.0f;
#pragma unroll
    for (int i = 0; i < D / PER; ++i) {
      const E* e = (const E*)&rv[i];
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const float x = Elem<DT>::get(e, j);
#pragma unroll
        for (int jj = 0; jj < 8; ++jj)
          if (jj < gq) acc[jj] = fmaf(qs[jj][i * PER + j], x, acc[jj]);
      }
    }
    if (a < k) {
      float* SK = dw.SK + ((size_t)g.prefKp[b] * g.H + (size_t)h * kp) * gq;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (jj < gq) SK[(size_t)jj * kp + a] = acc[jj];
    }
    return;
  }
  // ---- key-residual terms of one (request, head), 256 residuals per block
  idx -= nsc;
  const int rb = idx % g.maxRB, bh = idx / g.maxRB;
  const int b = bh / g.H, h = bh % g.H;
  const int S = g.S[b], G = g.G;
  const int nw = (S + 63) / 64;
  const size_t wo = (size_t)g.prefW[b] * g.H + (size_t)h * nw;
  const int e0 = c.pcK[wo];
  const int e1 = h + 1 < g.H ? c.pcK[wo + nw] : g.prefNK[b + 1];
  if (e0 + rb * 256 >= e1) return;
  // Rotated queries q_rot = FWHT(s * q): one wave per query head.
  for (int jj = wave; jj < gq; jj += 4) {
    const E* q = (const E*)qin + ((size_t)b * g.Hq + (size_t)h * gq + jj) * D;
    float z0 = hsign(g.seed_sign, 2 * lane) * Elem<DT>::get(q, 2 * lane);
    float z1 = hsign(g.seed_sign, 2 * lane + 1) * Elem<DT>::get(q, 2 * lane + 1);
    fwht_wave(z0, z1, lane);
    qs[jj][2 * lane] = z0;
    qs[jj][2 * lane + 1] = z1;
  }
  __syncthreads();
  const int e = e0 + rb * 256 + threadIdx.x;
  if (e >= e1) return;
  const uint4* cp = (const uint4*)(c.codesK + (size_t)e * (D / 4));
  const uint4 c0 = cp[0], c1 = cp[1];
  const uint32_t cw[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
  float sg[4];
#pragma unroll
  for (int qd = 0; qd < 4; ++qd) sg[qd] = qd < D / G ? c.scalesK[(size_t)e * (D / G) + qd] : 0.0f;
  float dot[8];
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) dot[jj] = 0.0f;
#pragma unroll
  for (int qd = 0; qd < 4; ++qd) {  // 32-coordinate quarters lie inside one group (G >= 32)
    const float s = sg[(qd * 32) / G];
    const float n1 = -s * AKV_L1, n0 = -s * AKV_L0, p0 = s * AKV_L0, p1 = s * AKV_L1;
#pragma unroll
    for (int dd = 0; dd < 32; ++dd) {
      const int d = qd * 32 + dd;
      const int code = (cw[d >> 4] >> (2 * (d & 15))) & 3;
      const float z = scaled_level(code, n1, n0, p0, p1);
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (jj < gq) dot[jj] = fmaf(qs[jj][d], z, dot[jj]);
    }
  }
  const float invD = 1.0f / (float)D;
#pragma unroll
  for (int jj = 0; jj < 8; ++jj)
    if (jj < gq) dw.RK[(size_t)e * gq + jj] = dot[jj] * invD;
}

// ------------------------------------------------------------------ D2
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

constexpr int DEC_ASTG = 64;   // value-anchor rows staged in LDS per split
constexpr int DEC_RCW = 512;   // anchor window of the per-anchor value weights
constexpr int DEC_VCH = 128;   // value residuals staged per chunk

template <int DT, int GQ, int R>
__global__ __launch_bounds__(256) void k_dec_stream(Geo g, Cache c, DecWs dw, float scale) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D, L = 256 * R, PER = 16 / sizeof(E);
  constexpr int NAV = DEC_ASTG * D / PER / 256;
  constexpr int NY = (GQ * D + 255) / 256;  // outputs per thread
  constexpr int JG = GQ < 4 ? GQ : 4;       // query heads covered by the 4 thread groups
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ float wacc[GQ][DEC_RCW];
  __shared__ __align__(16) E avs[DEC_ASTG * D];
  __shared__ __align__(16) uint32_t vcode[DEC_VCH][8];
  __shared__ float vsc[DEC_VCH][4];
  __shared__ float vp[DEC_VCH][GQ];
  __shared__ float red[4][GQ];
  __shared__ float mfin[GQ];

  // Logical block id: consecutive ids (the splits of one head) share an XCD.
  int id = blockIdx.x;
  const int n8 = gridDim.x & ~7;
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
  const int kpm = (g.maxK + 3) & ~3;
  float* SKs = (float*)smem;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* SKg = dw.SK + ((size_t)g.prefKp[b] * g.H + (size_t)h * kp) * GQ;
  const E* AVg = (const E*)c.ancV + ko * D;

  // ---- round 1: records, flag words, the split's residual ranges, the score table.
  const int i0 = s0 + tid * R;
  const bool any = i0 < s1;
  uint16_t ik[R], iv[R];
  float gk[R], gv[R];
  unsigned long long wk = 0, wv = 0;
  int pck = 0, pcv = 0;
  if (any) {
    load_u16<R>(c.idxK + so + i0, ik);
    load_u16<R>(c.idxV + so + i0, iv);
    load_coef<DT, R>(c.gK, so + i0, gk);
    load_coef<DT, R>(c.gV, so + i0, gv);
    wk = c.maskK[wo + (i0 >> 6)];
    wv = c.maskV[wo + (i0 >> 6)];
    pck = c.pcK[wo + (i0 >> 6)];
    pcv = c.pcV[wo + (i0 >> 6)];
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      ik[r] = 0;
      iv[r] = 0;
      gk[r] = 0.0f;
      gv[r] = 0.0f;
    }
  }
  const int a_lo = c.idxV[so + s0], a_hi = c.idxV[so + s1 - 1];
  const int pv_lo = c.pcV[wo + (s0 >> 6)];
  const int w1 = (s1 - 1) >> 6;
  const int pv_hi = c.pcV[wo + w1] + __popcll(c.maskV[wo + w1] & low_bits(s1 - 64 * w1));
  if (g.dsk_lds) {
    const int n4 = GQ * kp / 4;
    for (int i = tid; i < n4; i += 4 * 256) {
      float4 t[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i + u * 256 < n4) t[u] = *(const float4*)(SKg + 4 * (size_t)(i + u * 256));
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i + u * 256 < n4) {
          const int f = 4 * (i + u * 256);
          *(float4*)(&SKs[(f / kp) * kpm + (f % kp)]) = t[u];
        }
    }
  }
  const int nrange = a_hi - a_lo + 1;
  const int nstage = min(nrange, DEC_ASTG);
  const int nvres = pv_hi - pv_lo;

  // ---- round 2: key-residual terms, value-anchor rows, first value-residual chunk.
  const int sh = i0 & 63;
  uint32_t vmask = 0;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (i0 + r < s1) vmask |= 1u << r;
  const uint32_t bk = any ? ((uint32_t)(wk >> sh) & vmask) : 0u;
  const uint32_t bv = any ? ((uint32_t)(wv >> sh) & vmask) : 0u;
  pck += __popcll(wk & low_bits(sh));
  pcv += __popcll(wv & low_bits(sh));
  float rk[R][GQ];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int ri = pck + __popc(bk & ((1u << r) - 1u));
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) rk[r][jj] = ((bk >> r) & 1u) ? dw.RK[(size_t)ri * GQ + jj] : 0.0f;
  }
  uint4 avr[NAV];
#pragma unroll
  for (int i = 0; i < NAV; ++i) {
    const int ch = tid + 256 * i;
    const int r = ch / (D / PER), col = (ch % (D / PER)) * PER;
    avr[i] = r < nstage ? *(const uint4*)(AVg + (size_t)(a_lo + r) * D + col) : make_uint4(0, 0, 0, 0);
  }
  const int nv0 = min(nvres, DEC_VCH);
  uint4 vcr = make_uint4(0, 0, 0, 0);
  if (tid < 2 * nv0) vcr = ((const uint4*)(c.codesV + (size_t)(pv_lo + (tid >> 1)) * (D / 4)))[tid & 1];
  float vsr[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int f = tid + 256 * u;
    vsr[u] = f < nv0 * (D / G) ? c.scalesV[(size_t)pv_lo * (D / G) + f] : 0.0f;
  }
  __syncthreads();

  // ---- logits.
  float lg[R][GQ];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int a = min((int)ik[r], k - 1);
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) {
      const float s = g.dsk_lds ? SKs[jj * kpm + a] : SKg[(size_t)jj * kp + a];
      lg[r][jj] = (gk[r] * s + rk[r][jj]) * scale;
    }
  }
  // ---- softmax statistics of the split.
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    float v = -INFINITY;
#pragma unroll
    for (int r = 0; r < R; ++r)
      if ((vmask >> r) & 1u) v = fmaxf(v, lg[r][jj]);
    v = wave_max(v);
    if (lane == 0) red[wave][jj] = v;
  }
  __syncthreads();
  if (tid < GQ) mfin[tid] = fmaxf(fmaxf(red[0][tid], red[1][tid]), fmaxf(red[2][tid], red[3][tid]));
  __syncthreads();
  float ls[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float m = mfin[jj];
    ls[jj] = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float p = ((vmask >> r) & 1u) ? __expf(lg[r][jj] - m) : 0.0f;
      lg[r][jj] = p;
      ls[jj] += p;
    }
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float v = wave_sum(ls[jj]);
    if (lane == 0) red[wave][jj] = v;
  }
  // Stage the value-anchor rows and the first value-residual chunk.
#pragma unroll
  for (int i = 0; i < NAV; ++i) {
    const int ch = tid + 256 * i;
    const int r = ch / (D / PER), col = (ch % (D / PER)) * PER;
    *(uint4*)(&avs[r * D + col]) = avr[i];
  }
  if (tid < 2 * nv0) *(uint4*)(&vcode[tid >> 1][4 * (tid & 1)]) = vcr;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int f = tid + 256 * u;
    if (f < nv0 * (D / G)) vsc[f / (D / G)][f % (D / G)] = vsr[u];
  }

  // ---- value residuals: thread (coordinate pair, query head) accumulates over
  // the split's stored value residuals, staged DEC_VCH at a time.
  const int pair = tid & 63, jg = tid >> 6;
  const int grp = (2 * pair) / G;
  float za[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
  for (int cb = 0; cb < nvres; cb += DEC_VCH) {
    const int nv = min(DEC_VCH, nvres - cb);
    if (cb > 0) {
      __syncthreads();
      if (tid < 2 * nv) *(uint4*)(&vcode[tid >> 1][4 * (tid & 1)]) =
          ((const uint4*)(c.codesV + (size_t)(pv_lo + cb + (tid >> 1)) * (D / 4)))[tid & 1];
      for (int f = tid; f < nv * (D / G); f += 256)
        vsc[f / (D / G)][f % (D / G)] = c.scalesV[(size_t)(pv_lo + cb) * (D / G) + f];
    }
    // probabilities of this chunk's residual slots, written by their owners
#pragma unroll
    for (int r = 0; r < R; ++r)
      if ((bv >> r) & 1u) {
        const int li = pcv + __popc(bv & ((1u << r) - 1u)) - pv_lo - cb;
        if (li >= 0 && li < nv) {
#pragma unroll
          for (int jj = 0; jj < GQ; ++jj) vp[li][jj] = lg[r][jj];
        }
      }
    __syncthreads();
    if (jg < JG) {
      for (int e = 0; e < nv; ++e) {
        const uint32_t word = vcode[e][pair >> 3];
        const int nib = (word >> (4 * (pair & 7))) & 15;
        const float sg = vsc[e][grp];
        const float z0 = sg * level(nib & 3), z1 = sg * level(nib >> 2);
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int jj = jg + 4 * u;
          if (jj < GQ) {
            const float p = vp[e][jj];
            za[u][0] = fmaf(p, z0, za[u][0]);
            za[u][1] = fmaf(p, z1, za[u][1]);
          }
        }
      }
    }
  }

  // ---- per-anchor value weights over anchor windows, and y = sum_a w_a abar^V_a.
  float y[NY];
#pragma unroll
  for (int u = 0; u < NY; ++u) y[u] = 0.0f;
  for (int wb = 0; wb < nrange; wb += DEC_RCW) {
    const int wn = min(DEC_RCW, nrange - wb);
    __syncthreads();
    for (int i = tid; i < GQ * DEC_RCW; i += 256) (&wacc[0][0])[i] = 0.0f;
    __syncthreads();
    {
      int cur = -1;
      float run[GQ];
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) run[jj] = 0.0f;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int off = (int)iv[r] - a_lo - wb;
        const bool in = ((vmask >> r) & 1u) && off >= 0 && off < wn;
        if (in && off != cur) {
          if (cur >= 0) {
#pragma unroll
            for (int jj = 0; jj < GQ; ++jj)
              if (run[jj] != 0.0f) atomicAdd(&wacc[jj][cur], run[jj]);
          }
#pragma unroll
          for (int jj = 0; jj < GQ; ++jj) run[jj] = 0.0f;
          cur = off;
        }
        if (in) {
#pragma unroll
          for (int jj = 0; jj < GQ; ++jj) run[jj] = fmaf(lg[r][jj], gv[r], run[jj]);
        }
      }
      if (cur >= 0) {
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj)
          if (run[jj] != 0.0f) atomicAdd(&wacc[jj][cur], run[jj]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NY; ++u) {
      const int p = tid + 256 * u;
      if (p < GQ * D) {
        const int jj = p / D, d = p % D;
        float acc = y[u];
        for (int a = 0; a < wn; ++a) {
          const int ra = wb + a;
          const float av = ra < nstage ? Elem<DT>::get(avs, (size_t)ra * D + d)
                                       : Elem<DT>::get(AVg, (size_t)(a_lo + ra) * D + d);
          acc = fmaf(wacc[jj][a], av, acc);
        }
        y[u] = acc;
      }
    }
  }

  // ---- partial outputs.
  const int Hq = g.Hq;
#pragma unroll
  for (int u = 0; u < NY; ++u) {
    const int p = tid + 256 * u;
    if (p < GQ * D) {
      const int jj = p / D, d = p % D;
      const size_t pi = ((size_t)(g.prefSp[b] * Hq + (h * GQ + jj) * nsp + sp)) * (2 + 2 * D);
      if (d == 0) {
        dw.part[pi] = mfin[jj];
        dw.part[pi + 1] = red[0][jj] + red[1][jj] + red[2][jj] + red[3][jj];
      }
      dw.part[pi + 2 + d] = y[u];
    }
  }
  if (jg < JG) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int jj = jg + 4 * u;
      if (jj < GQ) {
        const size_t pi = ((size_t)(g.prefSp[b] * Hq + (h * GQ + jj) * nsp + sp)) * (2 + 2 * D);
        dw.part[pi + 2 + D + 2 * pair] = za[u][0];
        dw.part[pi + 2 + D + 2 * pair + 1] = za[u][1];
      }
    }
  }
}

// ------------------------------------------------------------------ D3
template <int DT>
__global__ __launch_bounds__(256) void k_dec_combine(Geo g, Cache c, DecWs dw, float scale, int n_app, void* out,
                                                     int out_dtype) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D;
  __shared__ float zb[D];
  __shared__ float yb[D];
  __shared__ float rmax[4], rsum[4];
  const int b = blockIdx.x / g.Hq, jq = blockIdx.x % g.Hq;
  const int h = jq / g.g, jj = jq % g.g;
  const int S = g.S[b], k = g.k[b], kp = (k + 3) & ~3;
  const int L = g.dsplit;
  const int nsp = (S + L - 1) / L;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const size_t pb = (size_t)(g.prefSp[b] * g.Hq + jq * nsp) * (2 + 2 * D);
  const float* part = dw.part + pb;
  const size_t tb = ((size_t)b * g.H + h) * g.max_append;
  const float* SK = dw.SK + ((size_t)g.prefKp[b] * g.H + (size_t)h * kp) * g.g + (size_t)jj * kp;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Global max over the splits and the appended tokens.
  float M = -INFINITY;
  for (int s = tid; s < nsp; s += 256) M = fmaxf(M, part[(size_t)s * (2 + 2 * D)]);
  for (int n = tid; n < n_app; n += 256)
    M = fmaxf(M, scale * (Elem<DT>::get(c.tgK, tb + n) * SK[min((int)c.tidxK[tb + n], k - 1)]));
  M = wave_max(M);
  if (lane == 0) rmax[wave] = M;
  __syncthreads();
  M = fmaxf(fmaxf(rmax[0], rmax[1]), fmaxf(rmax[2], rmax[3]));
  float l = 0.0f;
  for (int s = tid; s < nsp; s += 256) {
    const float* pp = part + (size_t)s * (2 + 2 * D);
    l += __expf(pp[0] - M) * pp[1];
  }
  // Each thread owns one output: y[d] (threads 0..127) or zacc[d] (128..255).
  float acc = 0.0f;
  int s = 0;
  for (; s + 8 <= nsp; s += 8) {
    float mv[8], vv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float* pp = part + (size_t)(s + u) * (2 + 2 * D);
      mv[u] = pp[0];
      vv[u] = pp[2 + tid];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc = fmaf(__expf(mv[u] - M), vv[u], acc);
  }
  for (; s < nsp; ++s) {
    const float* pp = part + (size_t)s * (2 + 2 * D);
    acc = fmaf(__expf(pp[0] - M), pp[2 + tid], acc);
  }
  // Appended tokens: encoded against the anchors, no residual.
  const E* AV = (const E*)c.ancV + ko * D;
  for (int n = 0; n < n_app; ++n) {
    const float lgt = scale * (Elem<DT>::get(c.tgK, tb + n) * SK[min((int)c.tidxK[tb + n], k - 1)]);
    const float p = __expf(lgt - M);
    if (tid == 0) l += p;
    if (tid < D) {
      const int av = min((int)c.tidxV[tb + n], k - 1);
      acc = fmaf(p * Elem<DT>::get(c.tgV, tb + n), Elem<DT>::get(AV, (size_t)av * D + tid), acc);
    }
  }
  l = wave_sum(l);
  if (lane == 0) rsum[wave] = l;
  if (tid < D) yb[tid] = acc; else zb[tid - D] = acc;
  // Inverse rotation of the value-residual sum: s * FWHT(z) / D.
  for (int hh = 1; hh < D; hh <<= 1) {
    __syncthreads();
    float v = 0.0f;
    if (tid < D) {
      const float x0 = zb[tid & ~hh], x1 = zb[tid | hh];
      v = (tid & hh) ? x0 - x1 : x0 + x1;
    }
    __syncthreads();
    if (tid < D) zb[tid] = v;
  }
  __syncthreads();
  if (tid < D) {
    const float lt = rsum[0] + rsum[1] + rsum[2] + rsum[3];
    const float y = yb[tid] + hsign(g.seed_sign, tid) * zb[tid] * (1.0f / (float)D);
    const float o = y / lt;
    const size_t oi = ((size_t)b * g.Hq + jq) * D + tid;
    if (out_dtype == 1) ((uint16_t*)out)[oi] = f2bf(o); else ((float*)out)[oi] = o;
  }
}

// ------------------------------------------------------------------ append
template <int DT>
__global__ __launch_bounds__(256) void k_append(Geo g, Cache c, int n_app, const void* kin, const void* vin) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D;
  __shared__ float xs[D];
  __shared__ float rb1[4], rb2[4];
  __shared__ int ri1[4];
  __shared__ double rc[4];
  __shared__ int rci[4];
  const int side = blockIdx.x & 1, bh = blockIdx.x >> 1;
  const int b = bh / g.H, h = bh % g.H;
  const int k = g.k[b];
  const E* x = (const E*)(side ? vin : kin) + (size_t)bh * D;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  const float* inv = (side ? c.invV : c.invK) + ko;
  const double* nrm = (side ? c.nrmV : c.nrmK) + ko;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (threadIdx.x < D) xs[threadIdx.x] = Elem<DT>::get(x, threadIdx.x);
  __syncthreads();
  float ss = 0.0f;
  for (int d = 0; d < D; ++d) ss = fmaf(xs[d], xs[d], ss);
  const float xn = sqrtf(ss) * (1.0f + 1e-5f);
  const float eps = xn * ((float)D * 1.1920929e-7f + 2.3841858e-7f) * 1.01f + 1e-30f;
  auto score = [&](int a) {
    const E* row = A + (size_t)a * D;
    float s = 0.0f;
    for (int d = 0; d < D; ++d) s = fmaf(xs[d], Elem<DT>::get(row, d), s);
    return fabsf(s) * inv[a];
  };
  float b1 = -1.0f, b2 = -1.0f;
  int i1 = 0x7fffffff;
  for (int a = threadIdx.x; a < k; a += 256) {
    const float v = score(a);
    b2 = __builtin_amdgcn_fmed3f(b1, b2, v);
    if (v > b1) { b1 = v; i1 = a; }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float ob1 = __shfl_xor(b1, o, 64), ob2 = __shfl_xor(b2, o, 64);
    const int oi = __shfl_xor(i1, o, 64);
    const float t2 = fmaxf(fmaxf(b2, ob2), fminf(b1, ob1));
    if (ob1 > b1 || (ob1 == b1 && oi < i1)) i1 = oi;
    b1 = fmaxf(b1, ob1);
    b2 = t2;
  }
  if (lane == 0) { rb1[wave] = b1; rb2[wave] = b2; ri1[wave] = i1; }
  __syncthreads();
  b1 = rb1[0]; b2 = rb2[0]; i1 = ri1[0];
  for (int v = 1; v < 4; ++v) {
    const float t2 = fmaxf(fmaxf(b2, rb2[v]), fminf(b1, rb1[v]));
    if (rb1[v] > b1 || (rb1[v] == b1 && ri1[v] < i1)) i1 = ri1[v];
    b1 = fmaxf(b1, rb1[v]);
    b2 = t2;
  }
  int best = i1;
  if (!(b1 - b2 > 2.0f * eps + b1 * 9.094947e-13f)) {
    const float band = b1 - 2.0f * eps - b1 * 9.094947e-13f;
    double bc = -INFINITY;
    int bi = 0x7fffffff;
    for (int a = threadIdx.x; a < k; a += 256) {
      if (score(a) < band) continue;
      const double d = dot64_seq<DT>(x, A + (size_t)a * D, D);
      const double cc = nrm[a] > 0.0 ? (d * d) / nrm[a] : -1.0;
      if (cc > bc) { bc = cc; bi = a; }
    }
    for (int o = 32; o > 0; o >>= 1) {
      const double oc = __shfl_xor(bc, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (oc > bc || (oc == bc && oi < bi)) { bc = oc; bi = oi; }
    }
    __syncthreads();
    if (lane == 0) { rc[wave] = bc; rci[wave] = bi; }
    __syncthreads();
    bc = rc[0];
    bi = rci[0];
    for (int v = 1; v < 4; ++v)
      if (rc[v] > bc || (rc[v] == bc && rci[v] < bi)) { bc = rc[v]; bi = rci[v]; }
    best = bi;
  }
  if (threadIdx.x == 0) {
    const double n = nrm[best];
    const double d = dot64_seq<DT>(x, A + (size_t)best * D, D);
    const double g64 = n > 0.0 ? d / n : 0.0;
    const float gb = Elem<DT>::round_coef((float)g64);
    const size_t ti = ((size_t)b * g.H + h) * g.max_append + n_app;
    (side ? c.tidxV : c.tidxK)[ti] = (uint16_t)best;
    Elem<DT>::put(side ? c.tgV : c.tgK, ti, gb);
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
    float z0 = sg * level(nib & 3), z1 = sg * level(nib >> 2);
    fwht_wave(z0, z1, lane);
    const float invD = 1.0f / (float)D;
    const float r0 = (z0 * invD) * hsign(g.seed_sign, 2 * lane);
    const float r1 = (z1 * invD) * hsign(g.seed_sign, 2 * lane + 1);
    x0 = x0 + r0;
    x1 = x1 + r1;
  }
  float* o = out + ((size_t)h * rows + t) * D;
  o[2 * lane] = x0;
  o[2 * lane + 1] = x1;
}

// ------------------------------------------------------------------ launchers
template <int DT, int GQ, int R>
static void launch_stream(const Geo& g, const Cache& c, const DecWs& dw, float scale, int nblk, size_t lds,
                          hipStream_t st) {
  (void)hipFuncSetAttribute((const void*)k_dec_stream<DT, GQ, R>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
  AKV_TIMED("k_dec_stream", st, k_dec_stream<DT, GQ, R><<<nblk, 256, lds, st>>>(g, c, dw, scale));
}

template <int DT, int GQ>
static void launch_stream_r(const Geo& g, const Cache& c, const DecWs& dw, float scale, int nblk, size_t lds,
                            hipStream_t st) {
  switch (g.dsplit) {
    case 2048: launch_stream<DT, GQ, 8>(g, c, dw, scale, nblk, lds, st); break;
    default: launch_stream<DT, GQ, 4>(g, c, dw, scale, nblk, lds, st); break;
  }
}

template <int DT>
static void launch_stream_g(const Geo& g, const Cache& c, const DecWs& dw, float scale, int nblk, size_t lds,
                            hipStream_t st) {
  switch (g.g) {
    case 1: launch_stream_r<DT, 1>(g, c, dw, scale, nblk, lds, st); break;
    case 2: launch_stream_r<DT, 2>(g, c, dw, scale, nblk, lds, st); break;
    case 4: launch_stream_r<DT, 4>(g, c, dw, scale, nblk, lds, st); break;
    default: launch_stream_r<DT, 8>(g, c, dw, scale, nblk, lds, st); break;
  }
}

// Dynamic LDS of the streaming kernel: the anchor-score table when it is kept
// in LDS (the rest of its LDS is static).
size_t decode_stream_lds(const Geo& g, int L, bool sk_in_lds) {
  (void)L;
  const size_t kpm = (size_t)((g.maxK + 3) & ~3);
  return sk_in_lds ? g.g * kpm * 4 : 0;
}

hipError_t launch_decode(const Geo& g, const Cache& c, const DecWs& dw, const void* q, void* out, int out_dtype,
                         float scale, int n_app, hipStream_t st) {
  const int L = g.dsplit;
  int nsc = g.B * g.H * g.maxRB, nst = 0;
  for (int b = 0; b < g.B; ++b) {
    nsc += g.H * ((g.k[b] + 255) / 256);
    nst += g.H * ((g.S[b] + L - 1) / L);
  }
  if (g.dtype == 1) {
    AKV_TIMED("k_dec_scores", st, k_dec_scores<1><<<nsc, 256, 0, st>>>(g, c, dw, q));
    launch_stream_g<1>(g, c, dw, scale, nst, decode_stream_lds(g, L, g.dsk_lds != 0), st);
    AKV_TIMED("k_dec_combine", st,
              k_dec_combine<1><<<g.B * g.Hq, 256, 0, st>>>(g, c, dw, scale, n_app, out, out_dtype));
  } else {
    AKV_TIMED("k_dec_scores", st, k_dec_scores<0><<<nsc, 256, 0, st>>>(g, c, dw, q));
    launch_stream_g<0>(g, c, dw, scale, nst, decode_stream_lds(g, L, g.dsk_lds != 0), st);
    AKV_TIMED("k_dec_combine", st,
              k_dec_combine<0><<<g.B * g.Hq, 256, 0, st>>>(g, c, dw, scale, n_app, out, out_dtype));
  }
  return hipGetLastError();
}

hipError_t launch_append(const Geo& g, const Cache& c, int n_app, const void* kn, const void* vn, hipStream_t st) {
  if (g.dtype == 1) {
    AKV_TIMED("k_append", st, k_append<1><<<g.B * g.H * 2, 256, 0, st>>>(g, c, n_app, kn, vn));
  } else {
    AKV_TIMED("k_append", st, k_append<0><<<g.B * g.H * 2, 256, 0, st>>>(g, c, n_app, kn, vn));
  }
  return hipGetLastError();
}

hipError_t launch_reconstruct(const Geo& g, const Cache& c, int b, int side, int n_app, float* out, hipStream_t st) {
  const int rows = g.S[b] + n_app;
  const int nblk = (g.H * rows + 3) / 4;
  if (g.dtype == 1) {
    AKV_TIMED("k_reconstruct", st, k_reconstruct<1><<<nblk, 256, 0, st>>>(g, c, b, side, n_app, out));
  } else {
    AKV_TIMED("k_reconstruct", st, k_reconstruct<0><<<nblk, 256, 0, st>>>(g, c, b, side, n_app, out));
  }
  return hipGetLastError();
}

}  // namespace akv
