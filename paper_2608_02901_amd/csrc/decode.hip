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
//   k_dec_scores : anchor scores S_K[j][a] = q_j . abar^K_a for every query of
//                  the group, once per step, and the rotated queries;
//   k_dec_stream : split-K pass over the value-anchor-grouped records (8 per
//                  lane, coalesced), S_K gathered from LDS, online softmax
//                  partials (max, sum, per-anchor value weights turned into
//                  sum_a w_a abar^V_a over the split's anchor range, rotated
//                  value residual sum);
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

// ------------------------------------------------------------------ D1
template <int DT>
__global__ __launch_bounds__(256) void k_dec_scores(Geo g, Cache c, DecWs dw, const void* qin) {
  using E = typename Elem<DT>::T;
  __shared__ float qs[8][AKV_D];
  __shared__ float zb[AKV_D];
  int idx = blockIdx.x;
  int b = 0;
  for (; b < g.B; ++b) {
    const int n = g.H * ((g.k[b] + 63) / 64);
    if (idx < n) break;
    idx -= n;
  }
  const int k = g.k[b], D = AKV_D, gq = g.g;
  const int nch = (k + 63) / 64;
  const int h = idx / nch, a0 = (idx % nch) * 64;
  const E* q = (const E*)qin + ((size_t)b * g.Hq + (size_t)h * gq) * D;
  for (int i = threadIdx.x; i < gq * D; i += blockDim.x) qs[i / D][i % D] = Elem<DT>::get(q, i);
  __syncthreads();
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const E* A = (const E*)c.ancK + ko * D;
  float* SK = dw.SK + ko * gq;
  for (int p = threadIdx.x; p < 64 * gq; p += blockDim.x) {
    const int a = a0 + (p & 63), jj = p >> 6;
    if (a >= k) continue;
    const E* row = A + (size_t)a * D;
    float s = 0.0f;
    for (int d = 0; d < D; d += 8) {
      if constexpr (DT == 1) {
        uint4 v = *(const uint4*)(row + d);
        const uint16_t* e = (const uint16_t*)&v;
#pragma unroll
        for (int i = 0; i < 8; ++i) s = fmaf(qs[jj][d + i], bf2f(e[i]), s);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) s = fmaf(qs[jj][d + i], row[d + i], s);
      }
    }
    SK[(size_t)jj * k + a] = s;
  }
  // Rotated queries, by the first block of each head.
  if (a0 == 0) {
    for (int jj = 0; jj < gq; ++jj) {
      __syncthreads();
      if (threadIdx.x < D) zb[threadIdx.x] = hsign(g.seed_sign, threadIdx.x) * qs[jj][threadIdx.x];
      for (int hh = 1; hh < D; hh <<= 1) {
        __syncthreads();
        float v = 0.0f;
        if (threadIdx.x < D) {
          const int i = threadIdx.x;
          const float a = zb[i & ~hh], bb = zb[i | hh];
          v = (i & hh) ? a - bb : a + bb;
        }
        __syncthreads();
        if (threadIdx.x < D) zb[threadIdx.x] = v;
      }
      __syncthreads();
      if (threadIdx.x < D) dw.qrot[((size_t)b * g.Hq + h * gq + jj) * D + threadIdx.x] = zb[threadIdx.x];
    }
  }
}

// ------------------------------------------------------------------ D2
template <int DT, int GQ, int R>
__global__ __launch_bounds__(256) void k_dec_stream(Geo g, Cache c, DecWs dw, float scale) {
  using E = typename Elem<DT>::T;
  constexpr int L = 256 * R;
  constexpr int D = AKV_D;
  extern __shared__ float lds[];
  __shared__ float red[4][GQ];
  __shared__ float mfin[GQ];
  __shared__ float zred[4][GQ][2 * 64];
  int idx = blockIdx.x;
  const int b = locate(g, L, 1, idx);
  const int S = g.S[b], k = g.k[b], G = g.G;
  const int nsp = (S + L - 1) / L;
  const int h = idx / nsp, sp = idx % nsp;
  const int s0 = sp * L, s1 = min(S, s0 + L);
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int range_cap = min(g.maxK, L);
  float* SKs = lds;                      // [GQ][k]
  float* wacc = lds + GQ * g.maxK;       // [GQ][range_cap]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  // Anchor scores of this head's queries.
  const float* SK = dw.SK + ko * GQ;
  for (int i = threadIdx.x; i < GQ * k; i += 256) SKs[(i / k) * g.maxK + (i % k)] = SK[i];
  const int a_lo = c.idxV[po + s0], a_hi = c.idxV[po + s1 - 1];
  const int nrange = a_hi - a_lo + 1;
  for (int i = threadIdx.x; i < GQ * range_cap; i += 256) wacc[i] = 0.0f;
  // Rotated query coordinates of this lane (2l, 2l+1).
  float qr0[GQ], qr1[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float* qr = dw.qrot + ((size_t)b * g.Hq + h * GQ + jj) * D;
    qr0[jj] = qr[2 * lane];
    qr1[jj] = qr[2 * lane + 1];
  }

  // Records of this lane's R consecutive slots.
  const int i0 = s0 + (wave * 64 + lane) * R;
  uint16_t ik[R], iv[R];
  float gk[R], gv[R];
  uint32_t bk = 0, bv = 0;  // residual flag bits of the R slots
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = i0 + r;
    const bool ok = i < s1;
    ik[r] = ok ? c.idxK[po + i] : 0;
    iv[r] = ok ? c.idxV[po + i] : (uint16_t)a_lo;
    gk[r] = ok ? Elem<DT>::get(c.gK, po + i) : 0.0f;
    gv[r] = ok ? Elem<DT>::get(c.gV, po + i) : 0.0f;
  }
  const size_t wo0 = (size_t)g.prefW[b] * g.H + (size_t)h * ((S + 63) / 64);
  unsigned long long wk = 0, wv = 0;
  int pck = 0, pcv = 0;
  if (i0 < s1) {
    const int word = i0 >> 6;
    wk = c.maskK[wo0 + word];
    wv = c.maskV[wo0 + word];
    pck = c.pcK[wo0 + word];
    pcv = c.pcV[wo0 + word];
    const int sh = i0 & 63;
    const unsigned long long lowm = (1ull << sh) - 1ull;
    pck += __popcll(wk & lowm);
    pcv += __popcll(wv & lowm);
    const uint32_t rm = (R >= 32) ? 0xffffffffu : ((1u << R) - 1u);
    bk = (uint32_t)(wk >> sh) & rm;
    bv = (uint32_t)(wv >> sh) & rm;
    const int valid = s1 - i0;
    if (valid < R) {
      bk &= (1u << valid) - 1u;
      bv &= (1u << valid) - 1u;
    }
  }
  __syncthreads();

  float lg[R][GQ];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) lg[r][jj] = gk[r] * SKs[jj * g.maxK + min((int)ik[r], k - 1)];

  // Key residuals: the wave takes each flagged slot in turn.
  const float invD = 1.0f / (float)D;
  const int grp = (2 * lane) / G;
  {
    uint32_t my = bk;
    int myslot = pck;
    for (int r = 0; r < R; ++r) {
      unsigned long long bal = __ballot((my >> r) & 1u);
      while (bal) {
        const int src = __ffsll((long long)bal) - 1;
        bal &= bal - 1;
        const int slot = __shfl(myslot + __popc(my & ((1u << r) - 1u)), src, 64);
        const uint8_t byte = c.codesK[(size_t)slot * (D / 4) + lane / 2];
        const int nib = (lane & 1) ? (byte >> 4) : (byte & 15);
        const float sg = c.scalesK[(size_t)slot * (D / G) + grp];
        const float z0 = sg * level(nib & 3), z1 = sg * level(nib >> 2);
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) {
          const float part = wave_sum(fmaf(qr0[jj], z0, qr1[jj] * z1));
          if (lane == src) lg[r][jj] += part * invD;
        }
      }
    }
  }
  // Softmax statistics of the split.
  float mx[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    float v = -INFINITY;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      lg[r][jj] *= scale;
      if (i0 + r < s1) v = fmaxf(v, lg[r][jj]);
    }
    v = wave_max(v);
    if (lane == 0) red[wave][jj] = v;
  }
  __syncthreads();
  if (threadIdx.x < GQ)
    mfin[threadIdx.x] = fmaxf(fmaxf(red[0][threadIdx.x], red[1][threadIdx.x]), fmaxf(red[2][threadIdx.x], red[3][threadIdx.x]));
  __syncthreads();
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) mx[jj] = mfin[jj];
  float ls[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) ls[jj] = 0.0f;
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) {
      const float p = (i0 + r < s1) ? __expf(lg[r][jj] - mx[jj]) : 0.0f;
      lg[r][jj] = p;
      ls[jj] += p;
    }
  // Per-anchor value weights: runs of equal value anchors accumulate in
  // registers and are flushed to LDS when the anchor changes.
  {
    int cur = iv[0];
    float run[GQ];
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj) run[jj] = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (iv[r] != cur) {
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) {
          if (run[jj] != 0.0f) atomicAdd(&wacc[jj * range_cap + (cur - a_lo)], run[jj]);
          run[jj] = 0.0f;
        }
        cur = iv[r];
      }
#pragma unroll
      for (int jj = 0; jj < GQ; ++jj) run[jj] = fmaf(lg[r][jj], gv[r], run[jj]);
    }
#pragma unroll
    for (int jj = 0; jj < GQ; ++jj)
      if (run[jj] != 0.0f) atomicAdd(&wacc[jj * range_cap + (cur - a_lo)], run[jj]);
  }
  // Value residuals: rotated-domain accumulation, two coordinates per lane.
  float za0[GQ], za1[GQ];
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) { za0[jj] = 0.0f; za1[jj] = 0.0f; }
  {
    uint32_t my = bv;
    int myslot = pcv;
    for (int r = 0; r < R; ++r) {
      unsigned long long bal = __ballot((my >> r) & 1u);
      while (bal) {
        const int src = __ffsll((long long)bal) - 1;
        bal &= bal - 1;
        const int slot = __shfl(myslot + __popc(my & ((1u << r) - 1u)), src, 64);
        const uint8_t byte = c.codesV[(size_t)slot * (D / 4) + lane / 2];
        const int nib = (lane & 1) ? (byte >> 4) : (byte & 15);
        const float sg = c.scalesV[(size_t)slot * (D / G) + grp];
        const float z0 = sg * level(nib & 3), z1 = sg * level(nib >> 2);
#pragma unroll
        for (int jj = 0; jj < GQ; ++jj) {
          const float p = __shfl(lg[r][jj], src, 64);
          za0[jj] = fmaf(p, z0, za0[jj]);
          za1[jj] = fmaf(p, z1, za1[jj]);
        }
      }
    }
  }
#pragma unroll
  for (int jj = 0; jj < GQ; ++jj) {
    const float v = wave_sum(ls[jj]);
    zred[wave][jj][2 * lane] = za0[jj];
    zred[wave][jj][2 * lane + 1] = za1[jj];
    if (lane == 0) red[wave][jj] = v;
  }
  __syncthreads();
  // Outputs: thread (jj, d) pairs.
  float* part = dw.part;
  const int Hq = g.Hq;
  for (int p = threadIdx.x; p < GQ * D; p += 256) {
    const int jj = p / D, d = p % D;
    const E* AV = (const E*)c.ancV + (ko + a_lo) * D + d;
    float y = 0.0f;
    for (int a = 0; a < nrange; ++a) y = fmaf(wacc[jj * range_cap + a], Elem<DT>::get(AV, (size_t)a * D), y);
    const float z = zred[0][jj][d] + zred[1][jj][d] + zred[2][jj][d] + zred[3][jj][d];
    const int jq = h * GQ + jj;
    const size_t pi = ((size_t)(g.prefSp[b] * Hq + jq * nsp + sp)) * (2 + 2 * D);
    if (d == 0) {
      part[pi] = mx[jj];
      part[pi + 1] = red[0][jj] + red[1][jj] + red[2][jj] + red[3][jj];
    }
    part[pi + 2 + d] = y;
    part[pi + 2 + D + d] = z;
  }
}

// ------------------------------------------------------------------ D3
template <int DT>
__global__ __launch_bounds__(128) void k_dec_combine(Geo g, Cache c, DecWs dw, float scale, int L, int n_app,
                                                     void* out, int out_dtype) {
  using E = typename Elem<DT>::T;
  constexpr int D = AKV_D;
  __shared__ float zb[D];
  const int b = blockIdx.x / g.Hq, jq = blockIdx.x % g.Hq;
  const int h = jq / g.g, jj = jq % g.g;
  const int S = g.S[b], k = g.k[b];
  const int nsp = (S + L - 1) / L;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int d = threadIdx.x;
  const size_t pb = (size_t)(g.prefSp[b] * g.Hq + jq * nsp) * (2 + 2 * D);
  float M = -INFINITY;
  for (int s = 0; s < nsp; ++s) M = fmaxf(M, dw.part[pb + (size_t)s * (2 + 2 * D)]);
  // Appended tokens (encoded against the anchors, no residual).
  const size_t tb = ((size_t)b * g.H + h) * g.max_append;
  const float* SK = dw.SK + ko * g.g + (size_t)jj * k;
  for (int n = 0; n < n_app; ++n) {
    const float l = scale * (Elem<DT>::get(c.tgK, tb + n) * SK[min((int)c.tidxK[tb + n], k - 1)]);
    M = fmaxf(M, l);
  }
  float l = 0.0f, y = 0.0f, z = 0.0f;
  for (int s = 0; s < nsp; ++s) {
    const float* pp = dw.part + pb + (size_t)s * (2 + 2 * D);
    const float f = __expf(pp[0] - M);
    l += f * pp[1];
    y += f * pp[2 + d];
    z += f * pp[2 + D + d];
  }
  const E* AV = (const E*)c.ancV + ko * D;
  for (int n = 0; n < n_app; ++n) {
    const float lg = scale * (Elem<DT>::get(c.tgK, tb + n) * SK[min((int)c.tidxK[tb + n], k - 1)]);
    const float p = __expf(lg - M);
    l += p;
    const int av = min((int)c.tidxV[tb + n], k - 1);
    y = fmaf(p * Elem<DT>::get(c.tgV, tb + n), Elem<DT>::get(AV, (size_t)av * D + d), y);
  }
  // Inverse rotation of the value-residual sum: s * FWHT(z) / D.
  zb[d] = z;
  for (int hh = 1; hh < D; hh <<= 1) {
    __syncthreads();
    const float a = zb[d & ~hh], bb = zb[d | hh];
    const float v = (d & hh) ? a - bb : a + bb;
    __syncthreads();
    zb[d] = v;
  }
  __syncthreads();
  y += hsign(g.seed_sign, d) * zb[d] * (1.0f / (float)D);
  const float o = y / l;
  const size_t oi = ((size_t)b * g.Hq + jq) * D + d;
  if (out_dtype == 1) ((uint16_t*)out)[oi] = f2bf(o); else ((float*)out)[oi] = o;
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
    const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
    t = min(max(c.pos[po + i], 0), S - 1);
    a = min((int)(side ? c.idxV : c.idxK)[po + i], k - 1);
    gb = Elem<DT>::get(side ? c.gV : c.gK, po + i);
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
    {
      const float p = z0, q = z1;
      z0 = p + q;
      z1 = p - q;
    }
    for (int hh = 1; hh < 64; hh <<= 1) {
      const float o0 = __shfl_xor(z0, hh, 64), o1 = __shfl_xor(z1, hh, 64);
      if (lane & hh) {
        z0 = o0 - z0;
        z1 = o1 - z1;
      } else {
        z0 = z0 + o0;
        z1 = z1 + o1;
      }
    }
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
template <int DT, int GQ>
static void launch_stream(const Geo& g, const Cache& c, const DecWs& dw, float scale, int nblk, size_t lds,
                          hipStream_t st) {
  (void)hipFuncSetAttribute((const void*)k_dec_stream<DT, GQ, 8>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  AKV_TIMED("k_dec_stream", st, k_dec_stream<DT, GQ, 8><<<nblk, 256, lds, st>>>(g, c, dw, scale));
}

hipError_t launch_decode(const Geo& g, const Cache& c, const DecWs& dw, const void* q, void* out, int out_dtype,
                         float scale, int n_app, hipStream_t st) {
  const int L = g.dsplit;
  int nsc = 0, nst = 0;
  for (int b = 0; b < g.B; ++b) {
    nsc += g.H * ((g.k[b] + 63) / 64);
    nst += g.H * ((g.S[b] + L - 1) / L);
  }
  if (g.dtype == 1) {
    AKV_TIMED("k_dec_scores", st, k_dec_scores<1><<<nsc, 256, 0, st>>>(g, c, dw, q));
  } else {
    AKV_TIMED("k_dec_scores", st, k_dec_scores<0><<<nsc, 256, 0, st>>>(g, c, dw, q));
  }
  const size_t lds = ((size_t)g.g * g.maxK + (size_t)g.g * (size_t)min(g.maxK, L)) * sizeof(float);
#define AKV_STREAM(DT)                                                   \
  switch (g.g) {                                                         \
    case 1: launch_stream<DT, 1>(g, c, dw, scale, nst, lds, st); break;  \
    case 2: launch_stream<DT, 2>(g, c, dw, scale, nst, lds, st); break;  \
    case 4: launch_stream<DT, 4>(g, c, dw, scale, nst, lds, st); break;  \
    default: launch_stream<DT, 8>(g, c, dw, scale, nst, lds, st); break; \
  }
  if (g.dtype == 1) {
    AKV_STREAM(1)
  } else {
    AKV_STREAM(0)
  }
#undef AKV_STREAM
  if (g.dtype == 1) {
    AKV_TIMED("k_dec_combine", st, k_dec_combine<1><<<g.B * g.Hq, 128, 0, st>>>(g, c, dw, scale, L, n_app, out, out_dtype));
  } else {
    AKV_TIMED("k_dec_combine", st, k_dec_combine<0><<<g.B * g.Hq, 128, 0, st>>>(g, c, dw, scale, L, n_app, out, out_dtype));
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
