// Head-pooled residual budget (Sec. 3.4; Algorithm 1, "top N by utility
// pooled over heads").  Per request and side, the N_side candidates of highest
// utility among the non-anchor positions of all H heads get a residual; ties
// go to the lower head, then the lower position (the flattened (h, t) order).
//
// The cut is an exact radix select on the fp32 bit patterns (utilities are
// >= 0, so their bits order like the values; anchors carry -1 and are
// skipped): four 8-bit passes (histogram + pick), then the equal-to-threshold
// candidates are ranked in flattened order by a chunk count and scan.
#include "akv_common.h"

namespace akv {

constexpr int BCHUNK = 4096;

__device__ inline int nside(const Geo& g, int b, int side) {
  return side ? g.prefNV[b + 1] - g.prefNV[b] : g.prefNK[b + 1] - g.prefNK[b];
}

// bstate[b][side] = {prefix, mask, remaining, mode}; mode 0: radix select,
// 1: take every candidate, 2: take none.
__global__ void k_binit(Geo g, Ws w) {
  const int bs = blockIdx.x;  // b * 2 + side
  const int b = bs >> 1, side = bs & 1;
  for (int i = threadIdx.x; i < 256; i += blockDim.x) w.bhist[bs * 256 + i] = 0;
  if (threadIdx.x == 0) {
    const int N = nside(g, b, side);
    const int ncand = g.H * (g.S[b] - g.k[b]);
    int32_t* st = w.bstate + bs * 4;
    st[0] = 0;
    st[1] = 0;
    st[2] = N;
    st[3] = N <= 0 ? 2 : (N >= ncand ? 1 : 0);
  }
}

__device__ inline int locate_b(const Geo& g, int& idx) {
  for (int b = 0; b < g.B; ++b) {
    int n = 2 * ((g.H * g.S[b] + BCHUNK - 1) / BCHUNK);
    if (idx < n) return b;
    idx -= n;
  }
  return -1;
}

__global__ __launch_bounds__(256) void k_bhist(Geo g, Ws w, int shift) {
  __shared__ uint32_t hist[256];
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const int bs = b * 2 + side;
  const int32_t* st = w.bstate + bs * 4;
  if (st[3] != 0) return;
  const uint32_t prefix = (uint32_t)st[0], mask = (uint32_t)st[1];
  for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  const int n = g.H * g.S[b];
  const float* u = w.u + (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  for (int e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
    const float v = u[e];
    if (v < 0.0f) continue;
    const uint32_t bits = __float_as_uint(v);
    if ((bits & mask) == prefix) atomicAdd(&hist[(bits >> shift) & 255u], 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 256; i += blockDim.x)
    if (hist[i]) atomicAdd(&w.bhist[bs * 256 + i], hist[i]);
}

__global__ void k_bpick(Geo g, Ws w, int shift) {
  const int bs = blockIdx.x;
  int32_t* st = w.bstate + bs * 4;
  if (threadIdx.x == 0 && st[3] == 0) {
    const uint32_t* hist = w.bhist + bs * 256;
    int remaining = st[2];
    int cum = 0, dg = 255;
    for (; dg > 0; --dg) {
      if (cum + (int)hist[dg] >= remaining) break;
      cum += hist[dg];
    }
    st[0] = (int32_t)((uint32_t)st[0] | ((uint32_t)dg << shift));
    st[1] = (int32_t)((uint32_t)st[1] | (255u << shift));
    st[2] = remaining - cum;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 256; i += blockDim.x) w.bhist[bs * 256 + i] = 0;
}

// Equal-to-threshold count per chunk.
__global__ __launch_bounds__(256) void k_btie(Geo g, Ws w) {
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const int bs = b * 2 + side;
  const int32_t* st = w.bstate + bs * 4;
  const int n = g.H * g.S[b];
  const int nch = (n + BCHUNK - 1) / BCHUNK;
  int32_t* tc = w.tiecnt + 2 * g.prefBC[b] + side * nch;
  if (st[3] != 0) {
    if (threadIdx.x == 0) tc[ch] = 0;
    return;
  }
  const uint32_t T = (uint32_t)st[0];
  const float* u = w.u + (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  int cnt = 0;
  for (int e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
    const float v = u[e];
    cnt += (v >= 0.0f && __float_as_uint(v) == T);
  }
  cnt = wave_sum_i(cnt);
  __shared__ int red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) tc[ch] = red[0] + red[1] + red[2] + red[3];
}

__global__ void k_btscan(Geo g, Ws w) {
  const int bs = blockIdx.x, b = bs >> 1, side = bs & 1;
  const int n = g.H * g.S[b];
  const int nch = (n + BCHUNK - 1) / BCHUNK;
  int32_t* tc = w.tiecnt + 2 * g.prefBC[b] + side * nch;
  if (threadIdx.x == 0) {
    int s = 0;
    for (int i = 0; i < nch; ++i) {
      int v = tc[i];
      tc[i] = s;
      s += v;
    }
  }
}

__global__ __launch_bounds__(256) void k_bmark(Geo g, Ws w) {
  __shared__ int wtot[4];
  int idx = blockIdx.x;
  const int b = locate_b(g, idx);
  const int side = idx & 1, ch = idx >> 1;
  const int bs = b * 2 + side;
  const int32_t* st = w.bstate + bs * 4;
  const int mode = st[3];
  const uint32_t T = (uint32_t)st[0];
  const int need = st[2];
  const int n = g.H * g.S[b];
  const int nch = (n + BCHUNK - 1) / BCHUNK;
  const int32_t* tc = w.tiecnt + 2 * g.prefBC[b] + side * nch;
  const size_t base = (size_t)side * g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H;
  const float* u = w.u + base;
  uint8_t* sel = w.sel + base;
  const int e0 = ch * BCHUNK, e1 = min(n, e0 + BCHUNK);
  // Each thread owns 16 consecutive elements; ranks of ties follow (h, t) order.
  const int per = BCHUNK / 256;
  const int lo = e0 + threadIdx.x * per, hi = min(e1, lo + per);
  int eq = 0;
  if (mode == 0)
    for (int e = lo; e < hi; ++e) {
      const float v = u[e];
      eq += (v >= 0.0f && __float_as_uint(v) == T);
    }
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
  for (int e = lo; e < hi; ++e) {
    const float v = u[e];
    uint8_t s = 0;
    if (v >= 0.0f) {
      if (mode == 1) {
        s = 1;
      } else if (mode == 0) {
        const uint32_t bits = __float_as_uint(v);
        if (bits > T) {
          s = 1;
        } else if (bits == T) {
          s = before < need;
          ++before;
        }
      }
    }
    sel[e] = s;
  }
}

hipError_t launch_budget(const Geo& g, const Ws& w, hipStream_t st) {
  int nblk = 0;
  for (int b = 0; b < g.B; ++b) nblk += 2 * ((g.H * g.S[b] + BCHUNK - 1) / BCHUNK);
  launch("k_binit", k_binit, dim3(g.B * 2), dim3(256), 0, st, g, w);
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    launch("k_bhist", k_bhist, dim3(nblk), dim3(256), 0, st, g, w, shift);
    launch("k_bpick", k_bpick, dim3(g.B * 2), dim3(256), 0, st, g, w, shift);
  }
  launch("k_btie", k_btie, dim3(nblk), dim3(256), 0, st, g, w);
  launch("k_btscan", k_btscan, dim3(g.B * 2), dim3(64), 0, st, g, w);
  launch("k_bmark", k_bmark, dim3(nblk), dim3(256), 0, st, g, w);
  return hipGetLastError();
}

}  // namespace akv
