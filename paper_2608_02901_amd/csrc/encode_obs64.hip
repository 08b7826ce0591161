// fp64 observation attention of the compression pass: for every KV head the
// m = W * (Hq/H) observation rows (the queries of the last W positions,
// causal inside the window; Sec. 3.2, App. A.2) attend to all positions, and
// this pass returns per row a reference M_w of the logits (at most 20 below
// their maximum), Z_w = sum_t exp(l_wt - M_w) and y_w = sum_t alpha_wt v_t in
// fp64, alpha_wt = exp(l_wt - M_w) / Z_w (Sec. 3.3 Eq. utilities uses alpha_wt
// and y_w; the softmax does not depend on the reference).  The utility epilogue reads them to bound its fp32 utilities, the
// residual budget re-scores the candidates at its cut with them, and the
// anchor selection re-scores its near-ties with M_w and Z_w.
//
//   k_obs64        : one workgroup per (request, head, 64 rows, chunk of
//                    oc64 tokens); each wave owns 16 rows and runs an online
//                    softmax over the chunk on v_mfma_f64_16x16x4_f64:
//                    S^T = K Q^T per 16-key tile (A = keys, B = queries), then
//                    O^T += V^T P^T (A = values, B = the probabilities, which
//                    the S^T accumulators already hold in the B layout).
//                    The key and value tiles sit in LDS in fp32 (one
//                    conversion to fp64 per operand), the query fragment in
//                    fp32 registers, the accumulators in VGPRs, and the
//                    softmax uses a table-driven exp (exp_tab);
//   k_obs64_reduce : merges the chunk statistics and outputs of 16 rows and
//                    derives the fp32 forms the epilogue uses.
//
// f64 16x16x4 MFMA operand layout: lane l supplies A[l%16][l/16] and
// B[l/16][l%16]; accumulator register r of lane l holds D[l/16 + 4r][l%16].
#include "akv_common.h"

namespace akv {

typedef __attribute__((ext_vector_type(4))) double f64x4;

constexpr int O64_KT = 32;          // keys per LDS tile (two MFMA key tiles)
constexpr int O64_MAXCH = 256;      // most chunks per head (the reduce keeps their scales in LDS)
constexpr double O64_NEG = -1e300;  // reference sentinel (finite: exp of differences stays defined)
// A row's reference lags its running maximum by at most this much (logit
// units), so p = exp(l - reference) <= exp(20).
constexpr double O64_SLACK = 20.0;

template <int DT>
__device__ inline double e2d(const void* p, int i) {
  if constexpr (DT == 1) return (double)bf2f(((const uint16_t*)p)[i]);
  else return (double)((const float*)p)[i];
}

// exp(x) in fp64 for -inf < x <= 20, within a few ulp: x is clamped below at
// -745 (the result underflows to zero there), then split as x = n ln2/64 + r
// with n = round(64 x / ln2) and |r| <= ln2/128 (Cody-Waite: ln2/64 in a
// 29-bit head, exact times any |n| < 2^24, and a tail), so that
// exp(x) = 2^(n >> 6) * 2^((n & 63)/64) * e^r, e^r by its degree-6 Taylor
// polynomial (truncation below 1e-19 relative) and 2^(j/64) from a table of
// 64 values.  About half the instructions of the library exp, which also
// guards the overflow range that the softmax here never reaches.
__device__ inline double exp_tab(double x, const double* tab) {
  constexpr double L64E = 92.332482616893656;                 // 64 / ln2
  constexpr double LN2H = 0.010830424696905538;               // ln2/64, head (0x3f862e42ff000000)
  constexpr double LN2L = -6.563929801064195e-13;             // ln2/64 - head
  x = fmax(x, -745.0);
  const double n = __builtin_rint(x * L64E);
  double r = fma(-n, LN2H, x);
  r = fma(-n, LN2L, r);
  const int ni = (int)n;
  double p = 1.0 / 720;
  p = fma(p, r, 1.0 / 120);
  p = fma(p, r, 1.0 / 24);
  p = fma(p, r, 1.0 / 6);
  p = fma(p, r, 0.5);
  p = fma(p, r, 1.0);
  p = fma(p, r, 1.0);
  return ldexp(tab[ni & 63] * p, ni >> 6);
}

// Four bf16 values (two packed words) as fp32.
__device__ inline float4 bf16x4_f(unsigned a, unsigned b) {
  return float4{__uint_as_float(a << 16), __uint_as_float(a & 0xFFFF0000u), __uint_as_float(b << 16),
                __uint_as_float(b & 0xFFFF0000u)};
}

__device__ inline f64x4 mfma64(double a, double b, f64x4 c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

template <int DT>
__global__ __launch_bounds__(256) void k_obs64(Geo g, Ws w, const void* Kin, const void* Vin, const void* Qin) {
  using E = typename Elem<DT>::T;
  constexpr int PER = 16 / sizeof(E);      // elements per 16-byte chunk
  constexpr int LDK = AKV_D + 4;           // LDS row stride in floats (16 bytes of padding)
  constexpr int CPR = AKV_D / PER;         // chunks per row
  constexpr int NLD = O64_KT * CPR / 256;  // chunks per thread per tile and side
  // key and value tiles in fp32 (bf16 widened once per tile, exactly), so
  // that the contractions convert each element with one instruction
  __shared__ __align__(16) float KT[2][O64_KT * LDK];
  __shared__ __align__(16) float VT[2][O64_KT * LDK];
  __shared__ double etab[64];  // 2^(j/64), the table of exp_tab
  if (threadIdx.x < 64) etab[threadIdx.x] = exp2(threadIdx.x / 64.0);
  const int nrg = (g.m + 63) / 64;
  int idx = blockIdx.x;
  int b = 0;
  for (; b < g.B; ++b) {
    const int n = g.H * nrg * ((g.S[b] + g.oc64 - 1) / g.oc64);
    if (idx < n) break;
    idx -= n;
  }
  const int S = g.S[b], P = S - g.W, m = g.m, D = AKV_D;
  const int nch = (S + g.oc64 - 1) / g.oc64;
  const int rg = idx % nrg, hc = idx / nrg, h = hc / nch, ch = hc % nch;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)Kin + xoff;
  const E* Vx = (const E*)Vin + xoff;
  const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rbase = rg * 64 + wave * 16;
  const bool active = rbase < m;  // wave-uniform: the wave owns at least one row
  const int row = rbase + (lane & 15);
  const int lim = row < m ? P + row % g.W : -1;  // last position the row attends to
  const int kq = lane >> 4;                      // contraction group of the lane
  const double isd = 1.0 / sqrt((double)D);

  // Query fragment of the lane: Q[row][32 kq + s], s = 0..31 (the contraction
  // index d = 32 (l/16) + s, the same bijection on both operands).
  float qf[32];
  {
    const E* qr = Q + (size_t)min(row, m - 1) * D + 32 * kq;
#pragma unroll
    for (int c = 0; c < 32 / PER; ++c) {
      const uint4 v = *(const uint4*)(qr + c * PER);
      if constexpr (DT == 1) {
        const float4 a = bf16x4_f(v.x, v.y), bq = bf16x4_f(v.z, v.w);
        qf[8 * c] = a.x; qf[8 * c + 1] = a.y; qf[8 * c + 2] = a.z; qf[8 * c + 3] = a.w;
        qf[8 * c + 4] = bq.x; qf[8 * c + 5] = bq.y; qf[8 * c + 6] = bq.z; qf[8 * c + 7] = bq.w;
      } else {
        qf[4 * c] = __uint_as_float(v.x); qf[4 * c + 1] = __uint_as_float(v.y);
        qf[4 * c + 2] = __uint_as_float(v.z); qf[4 * c + 3] = __uint_as_float(v.w);
      }
    }
  }

  const int tb = ch * g.oc64, te = min(S, tb + g.oc64);
  uint4 kpre[NLD], vpre[NLD];
  auto fetch = [&](int t0) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int c = threadIdx.x + 256 * i, r = c / CPR, col = (c % CPR) * PER;
      const bool in = t0 + r < S;
      kpre[i] = in ? *(const uint4*)(X + (size_t)(t0 + r) * D + col) : make_uint4(0, 0, 0, 0);
      vpre[i] = in ? *(const uint4*)(Vx + (size_t)(t0 + r) * D + col) : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int c = threadIdx.x + 256 * i, r = c / CPR, col = (c % CPR) * PER;
      if constexpr (DT == 1) {
        const uint4 k = kpre[i], v = vpre[i];
        *(float4*)&KT[buf][r * LDK + col] = bf16x4_f(k.x, k.y);
        *(float4*)&KT[buf][r * LDK + col + 4] = bf16x4_f(k.z, k.w);
        *(float4*)&VT[buf][r * LDK + col] = bf16x4_f(v.x, v.y);
        *(float4*)&VT[buf][r * LDK + col + 4] = bf16x4_f(v.z, v.w);
      } else {
        *(uint4*)&KT[buf][r * LDK + col] = kpre[i];
        *(uint4*)&VT[buf][r * LDK + col] = vpre[i];
      }
    }
  };

  double mrow = O64_NEG, zl = 0.0;  // reference of the row (same on its 4 lanes), lane-partial sum
  f64x4 O[8];
#pragma unroll
  for (int blk = 0; blk < 8; ++blk) O[blk] = f64x4{0.0, 0.0, 0.0, 0.0};

  fetch(tb);
  stash(0);
  if (tb + O64_KT < te) fetch(tb + O64_KT);
  int it = 0;
  for (int t0 = tb; t0 < te; t0 += O64_KT, ++it) {
    const int cb = it & 1;
    __syncthreads();  // tile it - 1 is no longer read: its buffer takes tile it + 1
    if (t0 + O64_KT < te) stash(cb ^ 1);
    if (t0 + 2 * O64_KT < te) fetch(t0 + 2 * O64_KT);
    if (!active) continue;
    // Two 16-key steps per LDS tile, unrolled so that the scheduler can
    // overlap one step's softmax with the other's contractions.
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      // ---- logits: register r of acc is key t0 + 16u + kq + 4r against row l%16
      const float* kr = &KT[cb][(16 * u + (lane & 15)) * LDK + 32 * kq];
      // The query fragment stays in fp32: widening it to fp64 once outside
      // the loop would hold 32 more registers for the whole chunk.
#pragma unroll
      for (int s = 0; s < 32; ++s) asm volatile("" : "+v"(qf[s]));
      // two independent accumulation chains (even and odd s)
      f64x4 acc = {0.0, 0.0, 0.0, 0.0}, acc1 = {0.0, 0.0, 0.0, 0.0};
      // the key fragment in two halves of 16 floats (fewer registers live)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        float4 kraw[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) kraw[c] = *(const float4*)(kr + 16 * hf + 4 * c);
#pragma unroll
        for (int s = 0; s < 16; s += 2) {
          acc = mfma64((double)((const float*)kraw)[s], (double)qf[16 * hf + s], acc);
          acc1 = mfma64((double)((const float*)kraw)[s + 1], (double)qf[16 * hf + s + 1], acc1);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      acc += acc1;
      double lg[4];
      bool ok[4];
      double tmax = O64_NEG;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        ok[r] = t0 + 16 * u + kq + 4 * r <= lim;
        lg[r] = acc[r] * isd;
        if (ok[r]) tmax = fmax(tmax, lg[r]);
      }
      tmax = fmax(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmax(tmax, __shfl_xor(tmax, 32, 64));
      // The row's reference mrow moves only when a logit exceeds it by more
      // than O64_SLACK (then to the running maximum, rescaling the sums), so
      // the rescale of the eight accumulators is rare: every p stays below
      // exp(O64_SLACK), far inside fp64 (and fp32) range.
      const bool up = tmax > mrow + O64_SLACK;
      if (__ballot(up)) {  // some row's reference moves (factor 1 on the others)
        const double nr = up ? tmax : mrow;
        const double scl = exp(mrow - nr);
        zl *= scl;
#pragma unroll
        for (int blk = 0; blk < 8; ++blk) O[blk] *= scl;
        mrow = nr;
      }
      double p[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const double e = exp_tab(lg[r] - mrow, etab);
        p[r] = ok[r] ? e : 0.0;
        zl += p[r];
      }
      // ---- values: MFMA r contracts the keys 16u + kq + 4r (k = kq); lane l
      // supplies V[key][8 (l%16) + blk] as A and its own p as B, so output
      // register r' of O[blk] is O^T[dim 8 (l/16 + 4 r') + blk][row l%16].
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float* vr = &VT[cb][(16 * u + kq + 4 * r) * LDK + 8 * (lane & 15)];
        const float4 v0 = *(const float4*)vr, v1 = *(const float4*)(vr + 4);
        const float vf[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int blk = 0; blk < 8; ++blk) O[blk] = mfma64((double)vf[blk], p[r], O[blk]);
      }
    }
  }
  if (!active) return;
  zl += __shfl_xor(zl, 16, 64);
  zl += __shfl_xor(zl, 32, 64);
  const size_t gc = ((size_t)g.prefC64[b] * g.H + (size_t)h * nch + ch);
  if (lane < 16 && row < m) {
    w.o64M[gc * g.mpad + row] = mrow;
    w.o64Z[gc * g.mpad + row] = zl;
  }
  double* op = w.o64O + (gc * (g.mpad / 16) + rbase / 16) * 2048;
#pragma unroll
  for (int blk = 0; blk < 8; ++blk)
#pragma unroll
    for (int r = 0; r < 4; ++r) op[(blk * 4 + r) * 64 + lane] = O[blk][r];
}

// One workgroup of 512 threads per (request, head, 16 rows, quarter of the
// dimensions), one output per thread:
// M_w = max of the chunk references, Z_w = sum_c Z_c exp(M_c - M_w) (every
// quarter forms them alike), y_w = sum_c O_c exp(M_c - M_w) / Z_w over the
// quarter's 32 dimensions (chunks in order), then the fp32 forms: y rounded
// and its bf16 hi/lo split, and the quarter's fp64 partial of ||y_w||^2.  The
// first quarter also writes M_w, Z_w, (M + ln Z) log2(e), ||q_w|| and the
// chunk-transposed copy of q_w (qt) that the band re-scoring reads.
template <int DT>
__global__ __launch_bounds__(512) void k_obs64_reduce(Geo g, Ws w, const void* Qin) {
  using E = typename Elem<DT>::T;
  __shared__ double scl[O64_MAXCH][16];
  __shared__ double red[16][16];
  __shared__ double Msh[16], Zsh[16];
  __shared__ double ysq[256];  // y^2 of the upper half's outputs
  const int nrb = g.mpad / 16;
  const int qd = blockIdx.x & 3, blk16 = blockIdx.x >> 2;
  const int bh = blk16 / nrb, rb16 = blk16 % nrb, b = bh / g.H, h = bh % g.H;
  const int m = g.m, D = AKV_D;
  const int nch = (g.S[b] + g.oc64 - 1) / g.oc64;
  const size_t gc0 = (size_t)g.prefC64[b] * g.H + (size_t)h * nch;
  const int tid = threadIdx.x, r16 = tid & 15, part = tid >> 4;
  const int row = rb16 * 16 + r16;
  const bool rok = row < m;
  const bool low = tid < 256;  // the row statistics use the first 256 threads
  double mx = O64_NEG;
  if (low && rok)
    for (int c = part; c < nch; c += 16) mx = fmax(mx, w.o64M[(gc0 + c) * g.mpad + row]);
  if (low) red[part][r16] = mx;
  __syncthreads();
  if (tid < 16) {
    double M = red[0][tid];
    for (int p = 1; p < 16; ++p) M = fmax(M, red[p][tid]);
    Msh[tid] = M;
  }
  __syncthreads();
  double za = 0.0;
  if (low)
    for (int c = part; c < nch; c += 16) {
      const double s = rok ? exp(w.o64M[(gc0 + c) * g.mpad + row] - Msh[r16]) : 0.0;
      scl[c][r16] = s;
      za += rok ? w.o64Z[(gc0 + c) * g.mpad + row] * s : 0.0;
    }
  if (low) red[part][r16] = za;
  __syncthreads();
  if (tid < 16) {
    double Z = 0.0;
    for (int p = 0; p < 16; ++p) Z += red[p][tid];
    Zsh[tid] = Z;
  }
  __syncthreads();
  // Outputs: in the chunk layout, register slot (blk * 4 + r) of lane l holds
  // dimension 8 (l / 16 + 4 r) + blk of row l % 16; the quarter qd takes
  // blk = 2 qd, 2 qd + 1 (512 contiguous values per chunk), one per thread
  // (threads t and t + 256 hold the two blocks).
  const int lane = tid & 63;
  const size_t bhm = (size_t)bh * m;
  const int slot = 8 * qd + (tid >> 6);  // blk * 4 + r
  const double* op = w.o64O + (gc0 * nrb + rb16) * 2048 + slot * 64 + lane;
  double acc = 0.0;
  const size_t cstride = (size_t)nrb * 2048;
  for (int c0 = 0; c0 < nch; c0 += 16) {
    double v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = c0 + u < nch ? op[(size_t)(c0 + u) * cstride] : 0.0;
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (c0 + u < nch) acc += v[u] * scl[c0 + u][r16];
  }
  {
    const int blk = slot >> 2, r = slot & 3;
    const double y = acc / Zsh[r16];
    const int dim = 8 * ((lane >> 4) + 4 * r) + blk;
    if (rok) {
      const size_t o = (bhm + row) * D + dim;
      w.Y64[(bhm * D + (size_t)(dim >> 1) * m * 2) + row * 2 + (dim & 1)] = y;
      const float y32 = (float)y;
      w.Y[o] = y32;
      const uint16_t hi = f2bf(y32);
      w.Yhi[o] = hi;
      w.Ylo[o] = f2bf(y32 - bf2f(hi));
    }
    acc = y * y;
  }
  // per thread of the lower half: y^2 of its block, then that of its partner
  if (!low) ysq[tid - 256] = acc;
  __syncthreads();
  if (low) red[part][r16] = acc + ysq[tid];
  __syncthreads();
  if (tid < 16 && rok) {
    double t = 0.0;
    for (int p = 0; p < 16; ++p) t += red[p][tid];
    w.ynp[(bhm + rb16 * 16 + tid) * 4 + qd] = t;
  }
  if (qd == 0) {
    // ||q_w||: 16 threads per row (the lower half), 8 coordinates each, then
    // a fixed-order sum
    __syncthreads();
    const E* q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D + (size_t)min(row, m - 1) * D;
    if (low) {
      double qq = 0.0;
      for (int j = 8 * part; j < 8 * part + 8; ++j) {
        const double x = e2d<DT>(q, j);
        qq += x * x;
      }
      // the same 8 coordinates: one 16-byte chunk (bf16) or two (fp32)
      constexpr int CPT = sizeof(E) / 2, NCH = AKV_D * sizeof(E) / 16;
      if (rok)
#pragma unroll
        for (int u = 0; u < CPT; ++u) {
          const int c = part * CPT + u;
          ((u32x4*)w.qt)[((size_t)bh * NCH + c) * m + row] = ((const u32x4*)q)[c];
        }
      red[part][r16] = qq;
    }
    __syncthreads();
    if (tid < 16 && rok) {
      double t = 0.0;
      for (int p = 0; p < 16; ++p) t += red[p][tid];
      const int rw = rb16 * 16 + tid;
      w.M64[bhm + rw] = Msh[tid];
      w.Z64[bhm + rw] = Zsh[tid];
      w.cw[bhm + rw] = (float)((Msh[tid] + log(Zsh[tid])) * 1.4426950408889634);
      w.qn[bhm + rw] = (float)(sqrt(t) * (1.0 + 1e-6));
    }
  }
}

hipError_t launch_obs64(const Geo& g, const Ws& w, const void* K, const void* V, const void* Q, hipStream_t st) {
  const int nrg = (g.m + 63) / 64;
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * nrg * ((g.S[b] + g.oc64 - 1) / g.oc64);
  const int nred = g.B * g.H * (g.mpad / 16) * 4;
  if (g.dtype == 1) {
    launch("k_obs64", k_obs64<1>, dim3(nblk), dim3(256), 0, st, g, w, K, V, Q);
    launch("k_obs64_reduce", k_obs64_reduce<1>, dim3(nred), dim3(512), 0, st, g, w, Q);
  } else {
    launch("k_obs64", k_obs64<0>, dim3(nblk), dim3(256), 0, st, g, w, K, V, Q);
    launch("k_obs64_reduce", k_obs64_reduce<0>, dim3(nred), dim3(512), 0, st, g, w, Q);
  }
  return hipGetLastError();
}

}  // namespace akv
