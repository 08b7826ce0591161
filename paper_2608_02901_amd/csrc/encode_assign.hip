// Nearest-anchor assignment (Sec. 3.1 Eq. nearest-anchor; Algorithm 1,
// second step), per request, KV head and side.
//
// k_assign: the dense tokens x anchors similarity contraction on MFMA, anchors
// on the M axis (staged through LDS, double buffered) and tokens on N (held in
// VGPRs for the whole anchor loop), so every lane's accumulators hold 16
// anchors of one token.  The epilogue keeps, per token, the best score
// s^_a = |x.a| / ||a|| with its index and the second best, without ever
// materializing the S x k score matrix.
//
// Certified argmax: the fp32 score differs from the exact |x.a|/||a|| by at
// most eps = (D 2^-23 + 2^-22) ||x|| (accumulation of D exact bf16 products,
// or rounded fp32 products, in any order, plus the inverse-norm and product
// roundings; inflated by 1 %).  When the best exceeds the second best by more
// than 2 eps (+ 2^-40 of the best, far above fp64 rounding), the winner is the
// exact argmax.  Otherwise the token goes to k_fixup, which rescans all anchors
// in fp32, and re-scores every anchor within the 2 eps band with the canonical
// fp64 formula (sequential fp64 dot d, c = d*d / ||a||^2, ties to the lowest
// index) -- the same formula as the CPU oracle, so the index is bit-exact.
#include "akv_common.h"

namespace akv {

__device__ inline float score_eps(float xnorm2, int D) {
  float xn = sqrtf(xnorm2) * (1.0f + 1e-5f);
  return xn * ((float)D * 1.1920929e-7f + 2.3841858e-7f) * 1.01f + 1e-30f;
}

template <int DT>
__global__ __launch_bounds__(256) void k_assign(Geo g, Ws w, Cache c, const void* Kin, const void* Vin) {
  using E = typename Elem<DT>::T;
  using M = MF<DT>;
  constexpr int LDA = AKV_D + (DT ? 8 : 4);
  constexpr int NKS = AKV_D / M::KS;
  constexpr int PER = 16 / sizeof(E);
  constexpr int STAGE = 64;                                 // anchors per LDS stage
  constexpr int NLD = STAGE * AKV_D / PER / 256;            // 16-byte loads per thread per stage
  __shared__ __align__(16) E AS[2][STAGE * LDA];
  __shared__ float WS[2][STAGE];

  int idx = blockIdx.x;
  const int b = locate(g, 128, 2, idx);
  const int side = idx & 1;
  idx >>= 1;
  const int S = g.S[b], k = g.k[b], D = AKV_D;
  const int ntile = (S + 127) / 128;
  const int h = idx / ntile, tile = idx % ntile;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)(side ? Vin : Kin) + xoff;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  const float* inv = (side ? c.invV : c.invK) + ko;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t = tile * 128 + wave * 32 + (lane & 31);
  const int tc = min(t, S - 1);

  // Token fragments (B operand) and the token's squared norm.
  typename M::frag xf[NKS];
  float ss = 0.0f;
#pragma unroll
  for (int s = 0; s < NKS; ++s) {
    xf[s] = M::load(X + (size_t)tc * D, kofs(M::KS, s, lane));
    if constexpr (DT == 1) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float v = (float)xf[s][i];
        ss = fmaf(v, v, ss);
      }
    } else {
      ss = fmaf(xf[s], xf[s], ss);
    }
  }
  ss += __shfl_xor(ss, 32, 64);

  const int nstage = (k + STAGE - 1) / STAGE;
  uint4 pre[NLD];
  float prew = 0.0f;
  auto fetch = [&](int st) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      int ch = threadIdx.x + 256 * i;
      int r = ch / (AKV_D / PER), col = (ch % (AKV_D / PER)) * PER;
      int a = st * STAGE + r;
      pre[i] = a < k ? *(const uint4*)(A + (size_t)a * D + col) : make_uint4(0, 0, 0, 0);
    }
    if (threadIdx.x < STAGE) {
      int a = st * STAGE + threadIdx.x;
      prew = a < k ? inv[a] : 0.0f;
    }
  };
  auto commit = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      int ch = threadIdx.x + 256 * i;
      int r = ch / (AKV_D / PER), col = (ch % (AKV_D / PER)) * PER;
      *(uint4*)(&AS[buf][r * LDA + col]) = pre[i];
    }
    if (threadIdx.x < STAGE) WS[buf][threadIdx.x] = prew;
  };

  float b1 = -1.0f, b2 = -1.0f;
  int i1 = 0;
  fetch(0);
  commit(0);
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    const int cur = st & 1;
    if (st + 1 < nstage) fetch(st + 1);
#pragma unroll
    for (int blk = 0; blk < STAGE / 32; ++blk) {
      const int abase = st * STAGE + blk * 32;
      if (abase >= k) break;
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        auto af = M::load_lds(&AS[cur][(blk * 32 + (lane & 31)) * LDA], kofs(M::KS, s, lane));
        acc = M::mma(af, xf[s], acc);
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = blk * 32 + crow(e, lane);
        const float v = fabsf(acc[e]) * WS[cur][r];
        const float nb2 = __builtin_amdgcn_fmed3f(b1, b2, v);
        const bool gt = v > b1;
        i1 = gt ? st * STAGE + r : i1;
        b1 = fmaxf(b1, v);
        b2 = nb2;
      }
    }
    if (st + 1 < nstage) commit(cur ^ 1);
    __syncthreads();
  }
  // Merge the two lanes holding the same token (rows 0-3 / 4-7 of each 8).
  {
    const float ob1 = __shfl_xor(b1, 32, 64), ob2 = __shfl_xor(b2, 32, 64);
    const int oi1 = __shfl_xor(i1, 32, 64);
    const float top2 = fmaxf(fmaxf(b2, ob2), fminf(b1, ob1));
    if (ob1 > b1 || (ob1 == b1 && oi1 < i1)) i1 = oi1;
    b1 = fmaxf(b1, ob1);
    b2 = top2;
  }
  if (lane < 32 && t < S) {
    const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S + t;
    int32_t* apos = w.apos + (size_t)side * g.H * g.prefS[g.B] + po;
    const int rk = w.rank[po];
    if (rk >= 0) {
      *apos = rk;
    } else {
      const float eps = score_eps(ss, D);
      if (b1 - b2 > 2.0f * eps + b1 * 9.094947e-13f) {
        *apos = i1;
      } else {
        *apos = -1;
        int slot = atomicAdd(&w.fixcount[0], 1);
        w.fix[slot] = ((unsigned long long)b << 48) | ((unsigned long long)side << 40) |
                      ((unsigned long long)h << 32) | (unsigned long long)t;
        atomicAdd(&c.stats[b * 4 + side], 1);
      }
    }
  }
}

// Exact resolution of the tokens whose fp32 margin did not certify the argmax.
// One wave per listed token; the grid strides over the list (its length is
// read on the device), so every wave exits once the list is exhausted.
template <int DT>
__global__ __launch_bounds__(256) void k_fixup(Geo g, Ws w, Cache c, const void* Kin, const void* Vin) {
  using E = typename Elem<DT>::T;
  __shared__ float xs[4][AKV_D];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = w.fixcount[0];
  const int D = AKV_D;
  for (int e = blockIdx.x * 4 + wave; e < n; e += gridDim.x * 4) {
    const unsigned long long ent = w.fix[e];
    const int b = (int)(ent >> 48), side = (int)((ent >> 40) & 0xff), h = (int)((ent >> 32) & 0xff);
    const int t = (int)(ent & 0xffffffffu);
    const int S = g.S[b], k = g.k[b];
    const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
    const E* x = (const E*)(side ? Vin : Kin) + xoff + (size_t)t * D;
    const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
    const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
    const float* inv = (side ? c.invV : c.invK) + ko;
    const double* nrm = (side ? c.nrmV : c.nrmK) + ko;
    float x0 = Elem<DT>::get(x, 2 * lane), x1 = Elem<DT>::get(x, 2 * lane + 1);
    xs[wave][2 * lane] = x0;
    xs[wave][2 * lane + 1] = x1;
    const float ss = wave_sum(fmaf(x0, x0, x1 * x1));
    const float eps = score_eps(ss, D);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    auto score = [&](int a) {
      const E* row = A + (size_t)a * D;
      float s = 0.0f;
      for (int d = 0; d < D; ++d) s = fmaf(xs[wave][d], Elem<DT>::get(row, d), s);
      return fabsf(s) * inv[a];
    };
    float smax = -1.0f;
    for (int a = lane; a < k; a += 64) smax = fmaxf(smax, score(a));
    smax = wave_max(smax);
    const float band = smax - 2.0f * eps - smax * 9.094947e-13f;
    double bc = -INFINITY;
    int bi = 0x7fffffff;
    for (int a = lane; a < k; a += 64) {
      if (score(a) < band) continue;
      const double d = dot64_seq<DT>(x, A + (size_t)a * D, D);
      const double cc = nrm[a] > 0.0 ? (d * d) / nrm[a] : -1.0;
      if (cc > bc) { bc = cc; bi = a; }
    }
    // Wave argmax: largest c, then lowest index.
    for (int o = 32; o > 0; o >>= 1) {
      double oc = __shfl_xor(bc, o, 64);
      int oi = __shfl_xor(bi, o, 64);
      if (oc > bc || (oc == bc && oi < bi)) { bc = oc; bi = oi; }
    }
    if (lane == 0) {
      w.apos[(size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H + (size_t)h * S + t] = bi;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

hipError_t launch_assign(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += g.H * ((g.S[b] + 127) / 128) * 2;
  if (g.dtype == 1) {
    AKV_TIMED("k_assign", st, k_assign<1><<<nblk, 256, 0, st>>>(g, w, c, K, V));
    AKV_TIMED("k_fixup", st, k_fixup<1><<<1024, 256, 0, st>>>(g, w, c, K, V));
  } else {
    AKV_TIMED("k_assign", st, k_assign<0><<<nblk, 256, 0, st>>>(g, w, c, K, V));
    AKV_TIMED("k_fixup", st, k_fixup<0><<<1024, 256, 0, st>>>(g, w, c, K, V));
  }
  return hipGetLastError();
}

}  // namespace akv
