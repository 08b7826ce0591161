// Per-token epilogue of the compression: projection coefficient and
// residual (Sec. 3.1 Eq. projection) and the attention-output-aware
// utilities (Sec. 3.3 Eq. utilities, App. A.3), for 32 tokens of one
// (request, head) per workgroup.
//
// Coefficient (bit-exact with the CPU oracle): d = sequential fp64 dot of the
// token and its anchor, gamma = d / ||a||^2 in fp64, rounded to fp32 and, for
// a bf16 cache, to bf16 (round to nearest even).  Anchor positions keep
// gamma = 1.
//
// Utilities (fp32, no positional rotation on this path, R_t = I):
//   uK_t = (1/m) sum_w alpha_wt^2 (q_w . rK_t)^2 / D * ||v_t - y_w||^2
//   uV_t = (1/m) sum_w alpha_wt^2 ||rV_t||^2
// with q_w . rK_t = q_w . k_t - gamma_t (q_w . abar_a(t)) (the second term from
// the QA table), ||v_t - y_w||^2 = ||v_t||^2 - 2 v_t . y_w + ||y_w||^2 and the
// logits and v_t . y_w on MFMA; anchors get u = -1 and never compete.
#include "akv_common.h"

namespace akv {

template <int DT>
__global__ __launch_bounds__(256) void k_epilogue(Geo g, Ws w, Cache c, const void* Kin, const void* Vin,
                                                  const void* Qin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LD = AKV_D + (DT ? 8 : 4);
  constexpr int PER = 16 / sizeof(E);
  __shared__ __align__(16) E KT[32 * LD];
  __shared__ __align__(16) E VT[32 * LD];
  __shared__ float gK_s[32], rv2_s[32], vn_s[32], sumK[32], sumV[32];
  __shared__ int aK_s[32], cand_s[32];

  int idx = blockIdx.x;
  const int b = locate(g, 32, 1, idx);
  const int S = g.S[b], k = g.k[b], D = AKV_D, m = g.m;
  const int ntile = (S + 31) / 32;
  const int h = idx / ntile, t0 = (idx % ntile) * 32;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* Kx = (const E*)Kin + xoff;
  const E* Vx = (const E*)Vin + xoff;
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;  // per-side stride of the position arrays
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  // Threads 0..63 = (token, side): the anchor rank and the assigned anchor
  // are read first, and the anchor row right after them, so that the
  // coefficient below waits for no memory (the rows of K and V load meanwhile).
  int rk0 = -1, ap0 = 0;
  uint4 arv[AKV_D / PER];
  double nrm0 = 0.0;
  if (threadIdx.x < 64) {
    const int side = threadIdx.x >> 5, t = min(t0 + (threadIdx.x & 31), S - 1);
    rk0 = w.rank[po + t];
    ap0 = w.apos[side * TS + po + t];
    const int a = (ap0 < 0 || ap0 >= k) ? 0 : ap0;
    const E* arow = (const E*)(side ? c.ancV : c.ancK) + (ko + a) * D;
#pragma unroll
    for (int i = 0; i < AKV_D / PER; ++i) {
      const uint4 v = *(const uint4*)(arow + i * PER);
      arv[i] = make_uint4(v.x, v.y, v.z, v.w);
    }
    nrm0 = (side ? c.nrmV : c.nrmK)[ko + a];
  }

#pragma unroll
  for (int ch = threadIdx.x; ch < 32 * (AKV_D / PER); ch += 256) {
    int r = ch / (D / PER), col = (ch % (D / PER)) * PER;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (t0 + r < S) {
      kv = *(const uint4*)(Kx + (size_t)(t0 + r) * D + col);
      vv = *(const uint4*)(Vx + (size_t)(t0 + r) * D + col);
    }
    *(uint4*)(&KT[r * LD + col]) = kv;
    *(uint4*)(&VT[r * LD + col]) = vv;
  }
  if (threadIdx.x < 32) {
    sumK[threadIdx.x] = 0.0f;
    sumV[threadIdx.x] = 0.0f;
  }
  __syncthreads();

  // Coefficients: threads 0..63 = (token, side).
  if (threadIdx.x < 64) {
    const int tl = threadIdx.x & 31, side = threadIdx.x >> 5, t = t0 + tl;
    if (t < S) {
      const int rk = rk0;
      const size_t o = side * TS + po + t;
      const E* xrow = &(side ? VT : KT)[tl * LD];
      if (rk >= 0) {
        w.gpos[o] = 1.0f;
        if (side == 0) { gK_s[tl] = 1.0f; aK_s[tl] = rk; cand_s[tl] = 0; }
        if (side == 1) rv2_s[tl] = 0.0f;
      } else {
        int a = ap0;
        if (a < 0 || a >= k) {
          atomicOr(&c.header[2], 4u);
          a = 0;
        }
        const E* arow = (const E*)arv;  // the prefetched row of anchor a
        const double n = nrm0;
        const double d = dot64_seq<DT>(xrow, arow, D);
        const double g64 = n > 0.0 ? d / n : 0.0;
        const float gb = Elem<DT>::round_coef((float)g64);
        w.gpos[o] = gb;
        if (side == 0) { gK_s[tl] = gb; aK_s[tl] = a; cand_s[tl] = 1; }
        if (side == 1) {
          float s = 0.0f;
#pragma unroll
          for (int j0 = 0; j0 < AKV_D; j0 += PER) {
            const uint4 av = *(const uint4*)(arow + j0);
            const uint4 xv = *(const uint4*)(xrow + j0);
            const E* ea = (const E*)&av;
            const E* ex = (const E*)&xv;
#pragma unroll
            for (int j = 0; j < PER; ++j) {
              float p = gb * Elem<DT>::get(ea, j);
              float r = Elem<DT>::get(ex, j) - p;
              s = fmaf(r, r, s);
            }
          }
          rv2_s[tl] = s;
        }
      }
    } else if (side == 0) {
      cand_s[tl] = 0;
      gK_s[tl] = 0.0f;
      aK_s[tl] = 0;
    }
  } else if (threadIdx.x < 96) {
    const int tl = threadIdx.x - 64;
    float s = 0.0f;
    for (int j = 0; j < D; ++j) {
      float v = Elem<DT>::get(&VT[tl * LD], j);
      s = fmaf(v, v, s);
    }
    vn_s[tl] = s;
  }
  __syncthreads();

  const int nrb = (m + 31) / 32;
  const float isd = 1.0f / sqrtf((float)D);
  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D;
  const float* oM = w.oM + (size_t)(b * g.H + h) * m;
  const float* oiZ = w.oiZ + (size_t)(b * g.H + h) * m;
  const float* yn = w.ynorm + (size_t)(b * g.H + h) * m;
  const float* QA = w.QA + ko * m;
  const int tl = lane & 31;
  const bool cand = cand_s[tl] != 0;
  const float gk = gK_s[tl];
  const int ak = aK_s[tl];
  const float vn = vn_s[tl];
  const bool vec = (m & 3) == 0;  // the row tables can be read as float4
  for (int rb = wave; rb < nrb; rb += 4) {
    // Rows past m (a partial last block) load row m - 1 and contribute 0.
    const int arow = min(rb * 32 + (lane & 31), m - 1);
    const E* qrow = Q + (size_t)arow * D;
    const size_t yo = ((size_t)(b * g.H + h) * m + arow) * D;
    f32x16 accL = {}, accY = {};
#pragma unroll
    for (int s = 0; s < D / M::KS; ++s) {
      const int k0 = kofs(M::KS, s, lane);
      auto qa = M::load(qrow, k0);
      auto kb = M::load_lds(&KT[tl * LD], k0);
      auto vb = M::load_lds(&VT[tl * LD], k0);
      accL = M::mma(qa, kb, accL);
      if constexpr (DT == 1) {
        accY = M::mma(M::load(w.Yhi + yo, k0), vb, accY);
        accY = M::mma(M::load(w.Ylo + yo, k0), vb, accY);
      } else {
        accY = M::mma(w.Y[yo + k0], vb, accY);
      }
    }
    float tk = 0.0f, tv = 0.0f;
    if (cand) {
      // Rows of accumulator entries 4j .. 4j+3 are consecutive.
      const float* qa = QA + (size_t)ak * m;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int w0 = rb * 32 + j * 8 + (lane >> 5) * 4;
        float qv[4], mv[4], zv[4], yv[4];
        if (vec && w0 < m) {
          const float4 q4 = *(const float4*)(qa + w0), m4 = *(const float4*)(oM + w0);
          const float4 z4 = *(const float4*)(oiZ + w0), y4 = *(const float4*)(yn + w0);
          qv[0] = q4.x; qv[1] = q4.y; qv[2] = q4.z; qv[3] = q4.w;
          mv[0] = m4.x; mv[1] = m4.y; mv[2] = m4.z; mv[3] = m4.w;
          zv[0] = z4.x; zv[1] = z4.y; zv[2] = z4.z; zv[3] = z4.w;
          yv[0] = y4.x; yv[1] = y4.y; yv[2] = y4.z; yv[3] = y4.w;
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int wr = min(w0 + i, m - 1);
            qv[i] = qa[wr];
            mv[i] = oM[wr];
            zv[i] = oiZ[wr];
            yv[i] = yn[wr];
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * j + i;
          const float l = accL[e];
          const float al = __expf(l * isd - mv[i]) * zv[i];
          const float a2 = w0 + i < m ? al * al : 0.0f;
          const float qr = l - gk * qv[i];
          const float vv = vn - 2.0f * accY[e] + yv[i];
          tk += a2 * (qr * qr) * vv;
          tv += a2;
        }
      }
    }
    tk += __shfl_xor(tk, 32, 64);
    tv += __shfl_xor(tv, 32, 64);
    if (lane < 32) {
      atomicAdd(&sumK[tl], tk);
      atomicAdd(&sumV[tl], tv);
    }
  }
  __syncthreads();
  if (threadIdx.x < 32) {
    const int t = t0 + threadIdx.x;
    if (t < S) {
      float uk = -1.0f, uv = -1.0f;
      if (cand_s[threadIdx.x]) {
        uk = sumK[threadIdx.x] / ((float)m * (float)D);
        uv = rv2_s[threadIdx.x] * sumV[threadIdx.x] / (float)m;
      }
      w.u[po + t] = uk;
      w.u[TS + po + t] = uv;
    }
  }
}

hipError_t launch_epilogue(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, const void* Q,
                           hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * ((g.S[b] + 31) / 32);
  if (g.dtype == 1) {
    launch("k_epilogue", k_epilogue<1>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V, Q);
  } else {
    launch("k_epilogue", k_epilogue<0>, dim3(nblk), dim3(256), 0, st, g, w, c, K, V, Q);
  }
  return hipGetLastError();
}

}  // namespace akv
