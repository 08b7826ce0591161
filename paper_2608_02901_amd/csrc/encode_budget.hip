// Head-pooled residual budget (Sec. 3.4; Algorithm 1, "top N by utility
// pooled over heads").  Per request and side, the N_side candidates of highest
// utility among the non-anchor positions of all H heads get a residual; ties
// go to the lower head, then the lower position (the flattened (h, t) order).
// The utility ranked is the canonical fp64 one (Sec. 3.3 Eq. utilities in fp64
// from exact fp64 logits and the fp64 observation statistics).
//
// First the fp32 estimates u are cut by an exact radix select on their bit
// patterns (utilities are >= 0, so their bits order like the values; anchors
// carry -1 and are skipped):
//   k_bhist : per chunk of the flattened (h, t) range, histogram of the first
//             12-bit digit [31:20], added to the request's;
//   k_bcand : every workgroup finds the digit of the N-th largest from that
//             histogram; utilities inside its bin are appended (value and
//             flattened index) as candidates;
//   k_bcut  : one workgroup per request and side: the remaining digits [19:8]
//             and [7:0] among the candidates (or, when the list overflowed,
//             among all utilities: same digits, same result), the count still
//             to take at the threshold, and per chunk the number of
//             threshold ties in the earlier chunks;
//   k_bmark : marks: above the threshold taken, ties taken in flattened order
//             while the count lasts.
// N <= 0 takes nothing; N at least the number of candidates takes them all.
//
// Then the fp32 order is corrected to the fp64 one.  The epilogue gives every
// candidate proven bounds uL <= u64 <= uU.  With T the N-th largest fp32
// estimate, A = min{uL : u >= T} is at most the N-th largest fp64 utility X
// (the N candidates with u >= T all have u64 >= A) and B = max{uU : u <= T} is
// at least X (only the fewer than N candidates with u > T can exceed B).  So
// uL > B is surely selected, uU < A surely not (both agree with the fp32
// marks), and the band of the rest holds X and every candidate whose order
// matters:
//   k_bbound   : A and B per request and side;
//   k_bmark    : also lists the band and counts the band members the fp32
//                order selected (the selections the band must supply);
//   k_brescore : the fp64 utility of every band member, computed as the
//                oracle does (sequential fp64 dots, one wave per member);
//   k_brank    : each band member's rank in (fp64 utility descending,
//                flattened index ascending) order;
//   k_bsel     : re-marks the band: ranks below `need` are selected.
// A band above BAND_CAP keeps the fp32 marks and raises HDR_BAND_OVERFLOW.
#include "akv_common.h"

namespace akv {

constexpr int BCHUNK = 4096;
constexpr int BCMAX = 32768;  // first-digit candidates kept per request and side

__device__ inline int nside(const Geo& g, int b, int side) {
  return side ? g.prefNV[b + 1] - g.prefNV[b] : g.prefNK[b + 1] - g.prefNK[b];
}
// 0: radix select, 1: take every candidate, 2: take none.
__device__ inline int bmode(const Geo& g, int b, int side) {
  const int N = nside(g, b, side);
  const int ncand = g.H * (g.S[b] - g.k[b]);
  return N <= 0 ? 2 : (N >= ncand ? 1 : 0);
}

__device__ inline int locate_b(const Geo& g, int& idx) {
  for (int b = 0; b < g.B; ++b) {
    int n = 2 * ((g.H * g.S[b] + BCHUNK - 1) / BCHUNK);
    if (idx < n) return b;
    idx -= n;
  }
  return -1;
}

__device__ inline const float* butil(const Geo& g, const Ws& w, int b, int side) {
  return w.u + (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
}

__global__ __launch_bounds__(256) void k_bhist(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  if (bmode(g, b, side) != 0) return;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  const int n = g.H * g.S[b];
  const float* u = butil(g, w, b, side);
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  for (int e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
    const float v = u[e];
    if (v >= 0.0f) atomicAdd(&hist[__float_as_uint(v) >> 20], 1u);
  }
  __syncthreads();
  uint32_t* gh = w.bhist + (size_t)(b * 2 + side) * SEL_NBIN;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x)
    if (hist[i]) atomicAdd(&gh[i], hist[i]);
}

__global__ __launch_bounds__(256) void k_bcand(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[8], pick[2];
  static_assert(BCHUNK % 256 == 0, "whole rounds of 256 elements per chunk");
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  if (bmode(g, b, side) != 0) return;
  const int bs = b * 2 + side;
  const uint32_t* gh = w.bhist + (size_t)bs * SEL_NBIN;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x) hist[i] = gh[i];
  __syncthreads();
  digit_pick(hist, SEL_NBIN, nside(g, b, side), true, tmp, pick);
  const uint32_t bin1 = (uint32_t)pick[0];
  const int n = g.H * g.S[b];
  const float* u = butil(g, w, b, side);
  float* cv = w.bcval + (size_t)bs * BCMAX;
  int32_t* cp = w.bcpos + (size_t)bs * BCMAX;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  constexpr int per = BCHUNK / 256;
  float v[per];
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    const int e = e0 + j * 256 + threadIdx.x;
    v[j] = e < e1 ? u[e] : -1.0f;
    cnt += v[j] >= 0.0f && (__float_as_uint(v[j]) >> 20) == bin1;
  }
  int slot = wg_reserve(cnt, &w.bstate[bs * BST_N + BST_NCAND], tmp);
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (v[j] >= 0.0f && (__float_as_uint(v[j]) >> 20) == bin1) {
      if (slot < BCMAX) {
        cv[slot] = v[j];
        cp[slot] = e0 + j * 256 + threadIdx.x;
      }
      ++slot;
    }
  }
}

__global__ __launch_bounds__(1024) void k_bcut(Geo g, Ws w, Cache c) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[20], pick[2];
  const int bs = blockIdx.x, b = bs >> 1, side = bs & 1;
  const int n = g.H * g.S[b];
  const int nch = (n + BCHUNK - 1) / BCHUNK;
  int32_t* tc = w.tiecnt + 2 * g.prefBC[b] + side * nch;
  int32_t* st = w.bstate + bs * BST_N;
  if (bmode(g, b, side) != 0) return;
  const int N = nside(g, b, side);
  const uint32_t* gh = w.bhist + (size_t)bs * SEL_NBIN;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x) hist[i] = gh[i];
  __syncthreads();
  digit_pick(hist, SEL_NBIN, N, true, tmp, pick);
  if (pick[0] < 0) {  // fewer candidates than N: cannot happen with N < candidates
    if (threadIdx.x == 0) {
      atomicOr(&c.header[2], HDR_BUDGET_CUT);
      st[BST_T] = 0x7F800000;
      st[BST_REMAIN] = 0;
    }
    return;
  }
  int remaining = N - pick[1];
  uint32_t prefix = (uint32_t)pick[0] << 20, pmask = 0xFFF00000u;
  const int nc = st[0];
  const float* cv = w.bcval + (size_t)bs * BCMAX;
  const int32_t* cp = w.bcpos + (size_t)bs * BCMAX;
  const float* u = butil(g, w, b, side);
  // Anchors carry -1 (sign bit set): they never match a prefix of a
  // non-negative utility.
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 8 : 0, nbin = pass == 0 ? SEL_NBIN : 256;
    if (nc <= BCMAX)
      digit_hist(hist, nbin, nc, [&](int i) { return __float_as_uint(cv[i]); }, pmask, prefix, shift);
    else
      digit_hist(hist, nbin, n, [&](int e) { return __float_as_uint(u[e]); }, pmask, prefix, shift);
    digit_pick(hist, nbin, remaining, true, tmp, pick);
    if (pick[0] < 0) {
      if (threadIdx.x == 0) {
        atomicOr(&c.header[2], HDR_BUDGET_CUT);
        st[BST_T] = 0x7F800000;
        st[BST_REMAIN] = 0;
      }
      return;
    }
    remaining -= pick[1];
    prefix |= (uint32_t)pick[0] << shift;
    pmask |= (uint32_t)(nbin - 1) << shift;
    __syncthreads();
  }
  // Threshold ties per chunk, then their exclusive scan over the chunks (in
  // rounds of SEL_NBIN chunks).
  int carry = 0;
  for (int c0 = 0; c0 < nch; c0 += SEL_NBIN) {
    const int c1 = min(nch, c0 + SEL_NBIN);
    for (int i = threadIdx.x; i < c1 - c0; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    if (nc <= BCMAX) {
      for (int i = threadIdx.x; i < nc; i += blockDim.x) {
        const int c = cp[i] / BCHUNK;
        if (__float_as_uint(cv[i]) == prefix && c >= c0 && c < c1) atomicAdd(&hist[c - c0], 1u);
      }
    } else {
      for (int e = c0 * BCHUNK + threadIdx.x; e < min(n, c1 * BCHUNK); e += blockDim.x)
        if (__float_as_uint(u[e]) == prefix) atomicAdd(&hist[e / BCHUNK - c0], 1u);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      for (int i = c0; i < c1; ++i) {
        const int v = (int)hist[i - c0];
        tc[i] = carry;
        carry += v;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    st[BST_T] = (int)prefix;
    st[BST_REMAIN] = remaining;
  }
}

// Band limits A = min{uL : u >= T}, B = max{uU : u <= T} (float bits of
// non-negative values order like the values).
__global__ __launch_bounds__(256) void k_bbound(Geo g, Ws w) {
  __shared__ unsigned red[2][4];
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  if (bmode(g, b, side) != 0) return;
  const int bs = b * 2 + side;
  const uint32_t T = (uint32_t)w.bstate[bs * BST_N + BST_T];
  const int n = g.H * g.S[b];
  const size_t base = (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  unsigned amin = 0x7F800000u, bmax = 0u;
  for (int e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
    const float v = w.u[base + e];
    if (!(v >= 0.0f)) continue;
    const uint32_t vb = __float_as_uint(v);
    if (vb >= T) amin = min(amin, __float_as_uint(w.uL[base + e]));
    if (vb <= T) bmax = max(bmax, __float_as_uint(w.uU[base + e]));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    amin = min(amin, (unsigned)__shfl_xor((int)amin, o, 64));
    bmax = max(bmax, (unsigned)__shfl_xor((int)bmax, o, 64));
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    red[0][wave] = amin;
    red[1][wave] = bmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 4; ++i) {
      amin = min(amin, red[0][i]);
      bmax = max(bmax, red[1][i]);
    }
    atomicMin((unsigned*)&w.bstate[bs * BST_N + BST_A], amin);
    atomicMax((unsigned*)&w.bstate[bs * BST_N + BST_B], bmax);
  }
}

__global__ __launch_bounds__(256) void k_bmark(Geo g, Ws w) {
  __shared__ int wtot[4];
  __shared__ int tmp[8];
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const int bs = b * 2 + side;
  int32_t* st = w.bstate + bs * BST_N;
  const int mode = bmode(g, b, side);
  const uint32_t T = (uint32_t)st[BST_T];
  const int need = st[BST_REMAIN];
  const uint32_t A = (uint32_t)st[BST_A], Bb = (uint32_t)st[BST_B];
  const int n = g.H * g.S[b];
  const int nch = (n + BCHUNK - 1) / BCHUNK;
  const int32_t* tc = w.tiecnt + 2 * g.prefBC[b] + side * nch;
  const size_t base = (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
  const float* u = w.u + base;
  uint8_t* sel = w.sel + base;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  // Each thread owns 16 consecutive elements; ranks of ties follow (h, t) order.
  constexpr int per = BCHUNK / 256;
  const int lo = e0 + threadIdx.x * per;
  float v[per];
#pragma unroll
  for (int j = 0; j < per; ++j) v[j] = lo + j < e1 ? u[lo + j] : -1.0f;
  int eq = 0;
  if (mode == 0)
#pragma unroll
    for (int j = 0; j < per; ++j) eq += (v[j] >= 0.0f && __float_as_uint(v[j]) == T);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = eq;
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wtot[wave] = x;
  __syncthreads();
  int before = x - eq + (mode == 0 ? tc[ch] : 0);
  for (int i = 0; i < wave; ++i) before += wtot[i];
  unsigned bandbits = 0;  // element j of the thread is a band member
  int nb = 0, nsel = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (lo + j >= e1) break;
    uint8_t s = 0;
    if (v[j] >= 0.0f) {
      if (mode == 1) {
        s = 1;
      } else if (mode == 0) {
        const uint32_t bits = __float_as_uint(v[j]);
        if (bits > T) {
          s = 1;
        } else if (bits == T) {
          s = before < need;
          ++before;
        }
        const uint32_t lb = __float_as_uint(w.uL[base + lo + j]), ub = __float_as_uint(w.uU[base + lo + j]);
        if (!(lb > Bb) && !(ub < A)) {
          bandbits |= 1u << j;
          ++nb;
          nsel += s;
        }
      }
    }
    sel[lo + j] = s;
  }
  if (mode != 0) return;  // uniform per workgroup
  // List the band members (one slot reservation per workgroup).
  int slot = wg_reserve(nb, &st[BST_NBAND], tmp);
  int32_t* bp = w.bandpos + (size_t)bs * BAND_CAP;
#pragma unroll
  for (int j = 0; j < per; ++j)
    if ((bandbits >> j) & 1u) {
      if (slot < BAND_CAP) {
        bp[slot] = lo + j;
        w.brank[(size_t)bs * BAND_CAP + slot] = 0;
      }
      ++slot;
    }
  const int ns = wave_sum_i(nsel);
  if (lane == 0 && ns) atomicAdd(&st[BST_NEED], ns);
}

// fp64 utility of every listed band member, one wave per member, computed as
// the oracle computes it (Sec. 3.3 Eq. utilities): the stored coefficient's
// residual r = x - fp32(gamma a) in fp32; per observation row w (lane w, w + 64,
// ...) the sequential fp64 dots l = q_w.k_t / sqrt(D), alpha = exp(l - M_w) /
// Z_w, and for keys q_w.r and ||v_t - y_w||^2, for values ||r||^2; the row
// terms alpha^2 (q.r)^2 / D ||v - y||^2 (or alpha^2 ||r||^2) summed in row
// order and divided by m.
template <int DT>
__global__ __launch_bounds__(256) void k_brescore(Geo g, Ws w, Cache c, const void* Kin, const void* Vin,
                                                  const void* Qin) {
  using E = typename Elem<DT>::T;
  __shared__ float xs[4][AKV_D], vs[4][AKV_D], rs[4][AKV_D];
  __shared__ double terms[4][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = gridDim.x * 4;
  const int gw = blockIdx.x * 4 + wave;
  const int m = g.m, D = AKV_D;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;
  const double sqd = sqrt((double)D);
  int base = 0;  // members of the earlier lists
  for (int bs = 0; bs < 2 * g.B; ++bs) {
    const int b = bs >> 1, side = bs & 1;
    const int nl = w.bstate[bs * BST_N + BST_NBAND];
    const int n = (bmode(g, b, side) == 0 && nl <= BAND_CAP) ? nl : 0;
    int i0 = gw - base;
    if (i0 < 0) i0 += ((-i0 + nw - 1) / nw) * nw;
    for (int i = i0; i < n; i += nw) {
      const int S = g.S[b], k = g.k[b];
      const int f = w.bandpos[(size_t)bs * BAND_CAP + i];
      const int h = f / S, t = f % S;
      const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
      const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
      const size_t xo = (po + t) * D;
      const int a = min(max(w.apos[side * TS + po + t], 0), k - 1);
      const float gm = w.gpos[side * TS + po + t];
      const E* xr = (const E*)(side ? Vin : Kin) + xo;
      const E* ar = (const E*)(side ? c.ancV : c.ancK) + (ko + a) * D;
      const E* kr = (const E*)Kin + xo;
      const E* vr = (const E*)Vin + xo;
      for (int j = lane; j < D; j += 64) {
        const float p = gm * Elem<DT>::get(ar, j);
        rs[wave][j] = Elem<DT>::get(xr, j) - p;
        xs[wave][j] = Elem<DT>::get(kr, j);
        vs[wave][j] = Elem<DT>::get(vr, j);
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      double rvn = 0.0;
      if (side == 1)
        for (int j = 0; j < D; ++j) rvn += (double)rs[wave][j] * (double)rs[wave][j];
      const size_t bh = (size_t)b * g.H + h;
      const E* Q = (const E*)Qin + ((size_t)b * g.Hq + (size_t)h * g.g) * g.W * D;
      constexpr int PER = 16 / sizeof(E);
      constexpr int NC = AKV_D / PER;
      for (int wr = lane; wr < m; wr += 64) {
        // q.k and q.r_K in one pass over the lane's query row, 16 bytes at a
        // time with the next chunk's load in flight (sequential sums)
        const uint4* q4 = (const uint4*)(Q + (size_t)wr * D);
        double l = 0.0, qr = 0.0;
        uint4 cur = q4[0];
        for (int c4 = 0; c4 < NC; ++c4) {
          const uint4 nxt = q4[min(c4 + 1, NC - 1)];
#pragma unroll
          for (int e = 0; e < PER; ++e) {
            const double qe = (double)Elem<DT>::get(&cur, e);
            l += qe * (double)xs[wave][c4 * PER + e];
            qr += qe * (double)rs[wave][c4 * PER + e];
          }
          cur = nxt;
        }
        l = l / sqd;
        const double al = exp(l - w.M64[bh * m + wr]) / w.Z64[bh * m + wr];
        const double a2 = al * al;
        double term;
        if (side == 0) {
          const double4* y4 = (const double4*)(w.Y64 + (bh * m + wr) * D);
          double vy = 0.0;
          double4 yc = y4[0];
          for (int c4 = 0; c4 < AKV_D / 4; ++c4) {
            const double4 yn = y4[min(c4 + 1, AKV_D / 4 - 1)];
            const double ye[4] = {yc.x, yc.y, yc.z, yc.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const double dv = (double)vs[wave][4 * c4 + e] - ye[e];
              vy += dv * dv;
            }
            yc = yn;
          }
          term = a2 * (qr * qr / D) * vy;
        } else {
          term = a2 * rvn;
        }
        terms[wave][wr] = term;
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      if (lane == 0) {
        double su = 0.0;
        for (int wr = 0; wr < m; ++wr) su += terms[wave][wr];
        w.bandu[(size_t)bs * BAND_CAP + i] = su / m;
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
    base += n;
  }
}

// Exact ranks inside the band: member i is selected when fewer than `need`
// members precede it in (fp64 utility descending, flattened index ascending)
// order.  k_brank counts, per 256 x 256 tile of (member i, member j) pairs,
// the j that precede each i and adds the counts to brank[i] (zeroed when the
// member was listed); the tiles of all lists are spread over a fixed grid.
// k_bsel then marks the band members from their ranks.
constexpr int RANK_T = 256;
__global__ __launch_bounds__(RANK_T) void k_brank(Geo g, Ws w) {
  __shared__ double su[RANK_T];
  __shared__ int sp[RANK_T];
  int tile0 = 0;
  for (int bs = 0; bs < 2 * g.B; ++bs) {
    const int b = bs >> 1, side = bs & 1;
    const int nl = w.bstate[bs * BST_N + BST_NBAND];
    const int n = (bmode(g, b, side) == 0 && nl <= BAND_CAP) ? nl : 0;
    const int nt = (n + RANK_T - 1) / RANK_T;
    const int32_t* bp = w.bandpos + (size_t)bs * BAND_CAP;
    const double* bu = w.bandu + (size_t)bs * BAND_CAP;
    int32_t* br = w.brank + (size_t)bs * BAND_CAP;
    int t = (int)blockIdx.x - tile0;
    if (t < 0) t += ((-t + (int)gridDim.x - 1) / (int)gridDim.x) * (int)gridDim.x;
    for (; t < nt * nt; t += gridDim.x) {  // uniform per workgroup
      const int ti = t / nt, tj = t % nt;
      const int j = tj * RANK_T + threadIdx.x;
      __syncthreads();
      su[threadIdx.x] = j < n ? bu[j] : 0.0;
      sp[threadIdx.x] = j < n ? bp[j] : 0x7FFFFFFF;
      __syncthreads();
      const int i = ti * RANK_T + threadIdx.x;
      if (i < n) {
        const double ui = bu[i];
        const int pi = bp[i];
        const int nj = min(RANK_T, n - tj * RANK_T);
        int r = 0;
        for (int jj = 0; jj < nj; ++jj) r += (su[jj] > ui || (su[jj] == ui && sp[jj] < pi)) ? 1 : 0;
        if (r) atomicAdd(&br[i], r);
      }
    }
    tile0 += nt * nt;
  }
}

__global__ __launch_bounds__(256) void k_bsel(Geo g, Ws w, Cache c) {
  const int bs = blockIdx.y, b = bs >> 1, side = bs & 1;
  if (bmode(g, b, side) != 0) return;
  const int n = w.bstate[bs * BST_N + BST_NBAND];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    c.stats[b * 4 + 2 + side] = n;  // band size, reported by the export
    if (n > BAND_CAP) atomicOr(&c.header[2], HDR_BAND_OVERFLOW);
  }
  if (n > BAND_CAP) return;
  const int need = w.bstate[bs * BST_N + BST_NEED];
  uint8_t* sel = w.sel + (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    sel[w.bandpos[(size_t)bs * BAND_CAP + i]] = w.brank[(size_t)bs * BAND_CAP + i] < need ? 1 : 0;
}

hipError_t launch_budget(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, const void* Q,
                         hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += 2 * ((g.H * g.S[b] + BCHUNK - 1) / BCHUNK);
  launch("k_bhist", k_bhist, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bcand", k_bcand, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bcut", k_bcut, dim3(g.B * 2), dim3(1024), 0, st, g, w, c);
  launch("k_bbound", k_bbound, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bmark", k_bmark, dim3(nblk), dim3(256), 0, st, g, w);
  if (g.dtype == 1)
    launch("k_brescore", k_brescore<1>, dim3(1024), dim3(256), 0, st, g, w, c, K, V, Q);
  else
    launch("k_brescore", k_brescore<0>, dim3(1024), dim3(256), 0, st, g, w, c, K, V, Q);
  launch("k_brank", k_brank, dim3(2048), dim3(RANK_T), 0, st, g, w);
  launch("k_bsel", k_bsel, dim3(64, g.B * 2), dim3(256), 0, st, g, w, c);
  return hipGetLastError();
}

}  // namespace akv
