// Head-pooled residual budget (Sec. 3.4; Algorithm 1, "top N by utility
// pooled over heads").  Per request and side, the N_side candidates of highest
// utility among the non-anchor positions of all H heads get a residual; ties
// go to the lower head, then the lower position (the flattened (h, t) order).
//
// The cut is an exact radix select on the fp32 bit patterns (utilities are
// >= 0, so their bits order like the values; anchors carry -1 and are
// skipped):
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
  int slot = wg_reserve(cnt, &w.bstate[bs * 4], tmp);
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

__global__ __launch_bounds__(1024) void k_bcut(Geo g, Ws w) {
  __shared__ uint32_t hist[SEL_NBIN];
  __shared__ int tmp[20], pick[2];
  const int bs = blockIdx.x, b = bs >> 1, side = bs & 1;
  const int n = g.H * g.S[b];
  const int nch = (n + BCHUNK - 1) / BCHUNK;
  int32_t* tc = w.tiecnt + 2 * g.prefBC[b] + side * nch;
  int32_t* st = w.bstate + bs * 4;
  if (bmode(g, b, side) != 0) return;
  const int N = nside(g, b, side);
  const uint32_t* gh = w.bhist + (size_t)bs * SEL_NBIN;
  for (int i = threadIdx.x; i < SEL_NBIN; i += blockDim.x) hist[i] = gh[i];
  __syncthreads();
  digit_pick(hist, SEL_NBIN, N, true, tmp, pick);
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
    st[1] = (int)prefix;
    st[2] = remaining;
  }
}

__global__ __launch_bounds__(256) void k_bmark(Geo g, Ws w) {
  __shared__ int wtot[4];
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const int bs = b * 2 + side;
  const int32_t* st = w.bstate + bs * 4;
  const int mode = bmode(g, b, side);
  const uint32_t T = (uint32_t)st[1];
  const int need = st[2];
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
      }
    }
    sel[lo + j] = s;
  }
}

hipError_t launch_budget(const Geo& g, const Ws& w, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += 2 * ((g.H * g.S[b] + BCHUNK - 1) / BCHUNK);
  launch("k_bhist", k_bhist, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bcand", k_bcand, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_bcut", k_bcut, dim3(g.B * 2), dim3(1024), 0, st, g, w);
  launch("k_bmark", k_bmark, dim3(nblk), dim3(256), 0, st, g, w);
  return hipGetLastError();
}

}  // namespace akv
