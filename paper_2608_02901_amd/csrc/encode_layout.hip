// Compressed layout build (App. A.1 "Layout" and Table of the layout) and the
// residual codec (Sec. 3.1 "Residual quantization"; App. A.1 Eqs. hadamard,
// arc-tuple).
//
// Decode order.  Attention is invariant to the order of its entries once
// positions are explicit (the layout keeps them as position ids), so each head
// stores its S records grouped by value anchor: a stable counting sort of the
// positions by a_V(t) (ties in position order).  The decode kernel then sees
// every anchor's value-side tokens contiguously and reads each anchor value
// row once.  Per sorted slot the cache keeps (a_K, gamma_K, a_V, gamma_V), the
// position, one residual flag bit per side in 64-bit words, and per word the
// global residual slot of its first flagged entry (prefix counts with the head
// offsets folded in), which makes slot lookup O(1).
//
//   k_shist    : per 2048-token chunk, histogram of a_V over the k anchors;
//   k_sscan    : per head, exclusive scan in (anchor, chunk) order;
//   k_sscatter : stable scatter of the positions, 64 tokens at a time;
//   k_lrec     : records, flag words and popcounts per sorted slot;
//   k_lscan    : per request and side, slot bases of every word;
//   k_codec    : one wave per flagged token: r = x - gamma * abar (fp32),
//                z = FWHT(s * r), per-group scale, 2-bit codes packed four per
//                byte (coordinate j in byte j/4, bits 2(j%4)..2(j%4)+1).
#include "akv_common.h"

namespace akv {

__device__ inline int locate_sort(const Geo& g, int& idx) {
  for (int b = 0; b < g.B; ++b) {
    int n = g.H * ((g.S[b] + SORT_CHUNK - 1) / SORT_CHUNK);
    if (idx < n) return b;
    idx -= n;
  }
  return -1;
}

__device__ inline int32_t* shist_base(const Geo& g, const Ws& w, int b, int h) {
  const int nT = (g.S[b] + SORT_CHUNK - 1) / SORT_CHUNK;
  return w.shist + (size_t)g.prefKT[b] + (size_t)h * g.k[b] * nT;
}

__global__ __launch_bounds__(256) void k_shist(Geo g, Ws w) {
  extern __shared__ int hist[];
  int idx = blockIdx.x;
  const int b = locate_sort(g, idx);
  const int S = g.S[b], k = g.k[b];
  const int nT = (S + SORT_CHUNK - 1) / SORT_CHUNK;
  const int h = idx / nT, ch = idx % nT;
  for (int a = threadIdx.x; a < k; a += blockDim.x) hist[a] = 0;
  __syncthreads();
  const int32_t* av = w.apos + (size_t)g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const int t0 = ch * SORT_CHUNK, t1 = min(S, t0 + SORT_CHUNK);
  for (int t = t0 + threadIdx.x; t < t1; t += blockDim.x) {
    const int a = av[t];
    if (a >= 0 && a < k) atomicAdd(&hist[a], 1);
  }
  __syncthreads();
  int32_t* out = shist_base(g, w, b, h);
  for (int a = threadIdx.x; a < k; a += blockDim.x) out[(size_t)a * nT + ch] = hist[a];
}

// Per head, the (anchor, chunk) histogram becomes its exclusive prefix sums,
// in place.  Batches of 8 x 1024 entries in (u, thread) order: coalesced
// loads (the next batch's issued before the current one is scanned), wave
// scans, and one scan of the per-(u, wave) totals per batch.
__global__ __launch_bounds__(1024) void k_sscan(Geo g, Ws w) {
  constexpr int U = 8;
  __shared__ int cnts[U * 16];
  __shared__ int cpre[U * 16 + 1];
  const int b = blockIdx.x / g.H, h = blockIdx.x % g.H;
  const int nT = (g.S[b] + SORT_CHUNK - 1) / SORT_CHUNK;
  const int n = g.k[b] * nT;
  int32_t* a = shist_base(g, w, b, h);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, nt = blockDim.x;  // nt = 1024
  int cur[U], nxt[U];
#pragma unroll
  for (int u = 0; u < U; ++u) nxt[u] = u * nt + tid < n ? a[u * nt + tid] : 0;
  int base = 0;
  for (int c0 = 0; c0 < n; c0 += U * nt) {
#pragma unroll
    for (int u = 0; u < U; ++u) cur[u] = nxt[u];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = c0 + U * nt + u * nt + tid;
      nxt[u] = i < n ? a[i] : 0;
    }
    int x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      x[u] = cur[u];
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x[u], o, 64);
        if (lane >= o) x[u] += y;
      }
      if (lane == 63) cnts[u * 16 + wv] = x[u];
    }
    __syncthreads();
    if (wv == 0) {
      const int v0 = cnts[2 * lane], v1 = cnts[2 * lane + 1];
      int y = v0 + v1;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int z = __shfl_up(y, o, 64);
        if (lane >= o) y += z;
      }
      cpre[2 * lane] = y - v0 - v1;
      cpre[2 * lane + 1] = y - v1;
      if (lane == 63) cpre[U * 16] = y;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = c0 + u * nt + tid;
      if (i < n) a[i] = base + cpre[u * 16 + wv] + x[u] - cur[u];
    }
    base += cpre[U * 16];
    __syncthreads();
  }
}

// One wave per chunk: tokens in groups of 64 in position order; the rank of a
// token among equal anchors of its group comes from a lane scan, a running
// per-anchor count in LDS carries it across groups.
__global__ __launch_bounds__(64) void k_sscatter(Geo g, Ws w, Cache c) {
  extern __shared__ int run[];
  int idx = blockIdx.x;
  const int b = locate_sort(g, idx);
  const int S = g.S[b], k = g.k[b];
  const int nT = (S + SORT_CHUNK - 1) / SORT_CHUNK;
  const int h = idx / nT, ch = idx % nT;
  const int lane = threadIdx.x;
  for (int a = lane; a < k; a += 64) run[a] = 0;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  const int32_t* av = w.apos + (size_t)g.H * g.prefS[g.B] + (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const int32_t* off = shist_base(g, w, b, h);
  int32_t* pos = c.pos + slot_base(g, b, h);
  const int t0 = ch * SORT_CHUNK, t1 = min(S, t0 + SORT_CHUNK);
  for (int tb = t0; tb < t1; tb += 64) {
    const int t = tb + lane;
    int a = t < t1 ? av[t] : -1;
    if (a >= k) a = -1;
    int before = 0, after = 0;
    for (int o = 0; o < 64; ++o) {
      const int ao = __shfl(a, o, 64);
      before += (o < lane && ao == a);
      after += (o > lane && ao == a);
    }
    if (a >= 0) {
      const int dest = off[(size_t)a * nT + ch] + run[a] + before;
      if (dest >= 0 && dest < S) pos[dest] = t;
    }
    __syncthreads();
    if (a >= 0 && after == 0) run[a] += before + 1;
    __syncthreads();
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_lrec(Geo g, Ws w, Cache c) {
  int idx = blockIdx.x;
  const int b = locate(g, 256, 1, idx);
  const int S = g.S[b];
  const int nt = (S + 255) / 256;
  const int h = idx / nt, i = (idx % nt) * 256 + threadIdx.x;
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t so = slot_base(g, b, h);
  const size_t TS = (size_t)g.prefS[g.B] * g.H;
  bool fk = false, fv = false;
  if (i < S) {
    int t = c.pos[so + i];
    if (t < 0 || t >= S) {
      atomicOr(&c.header[2], 8u);
      t = 0;
    }
    c.idxK[so + i] = (uint16_t)w.apos[po + t];
    c.idxV[so + i] = (uint16_t)w.apos[TS + po + t];
    Elem<DT>::put(c.gK, so + i, w.gpos[po + t]);
    Elem<DT>::put(c.gV, so + i, w.gpos[TS + po + t]);
    fk = w.sel[po + t] != 0;
    fv = w.sel[TS + po + t] != 0;
  } else if (i < ((S + 63) & ~63)) {
    // Padding slots of the head's last word: anchor 0 with coefficient 0.
    c.pos[so + i] = 0;
    c.idxK[so + i] = 0;
    c.idxV[so + i] = 0;
    Elem<DT>::put(c.gK, so + i, 0.0f);
    Elem<DT>::put(c.gV, so + i, 0.0f);
  }
  const unsigned long long mk = __ballot(fk), mv = __ballot(fv);
  if ((threadIdx.x & 63) == 0 && i < S) {
    const int word = i >> 6;
    const size_t wo = (size_t)g.prefW[b] * g.H + (size_t)h * ((S + 63) / 64) + word;
    c.maskK[wo] = mk;
    c.maskV[wo] = mv;
    const size_t WT = (size_t)g.prefW[g.B] * g.H;
    w.wcnt[wo] = __popcll(mk);
    w.wcnt[WT + wo] = __popcll(mv);
  }
}

// Slot base of every word: the request's first slot plus an exclusive scan
// over its (head, word) sequence.
__global__ __launch_bounds__(1024) void k_lscan(Geo g, Ws w, Cache c) {
  __shared__ int tmp[20];
  const int b = blockIdx.x >> 1, side = blockIdx.x & 1;
  const int nw = g.H * ((g.S[b] + 63) / 64);
  const size_t WT = (size_t)g.prefW[g.B] * g.H;
  const size_t wo = (size_t)g.prefW[b] * g.H;
  const int32_t* cnt = w.wcnt + side * WT + wo;
  int32_t* pc = (side ? c.pcV : c.pcK) + wo;
  const int per = (nw + blockDim.x - 1) / blockDim.x;
  const int lo = min(nw, (int)threadIdx.x * per), hi = min(nw, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += cnt[i];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = s;
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) tmp[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
      int v = tmp[i];
      tmp[i] = acc;
      acc += v;
    }
  }
  __syncthreads();
  int run = x - s + tmp[wave] + (side ? g.prefNV[b] : g.prefNK[b]);
  for (int i = lo; i < hi; ++i) {
    int v = cnt[i];
    pc[i] = run;
    run += v;
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_codec(Geo g, Ws w, Cache c, const void* Kin, const void* Vin) {
  using E = typename Elem<DT>::T;
  const int lane = threadIdx.x & 63;
  // One wave per 64-slot word; flattened over (side, request, head, word).
  int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int WTH = g.prefW[g.B] * g.H;
  if (wid >= 2 * WTH) return;
  const int side = wid >= WTH;
  if (side) wid -= WTH;
  int b = 0;
  for (; b < g.B; ++b) {
    const int n = g.H * ((g.S[b] + 63) / 64);
    if (wid < n) break;
    wid -= n;
  }
  const int S = g.S[b], k = g.k[b], D = AKV_D, G = g.G;
  const int nw = (S + 63) / 64;
  const int h = wid / nw, word = wid % nw;
  const size_t wo = (size_t)g.prefW[b] * g.H + (size_t)h * nw + word;
  unsigned long long mask = (side ? c.maskV : c.maskK)[wo];
  if (!mask) return;
  int slot = (side ? c.pcV : c.pcK)[wo];
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)(side ? Vin : Kin) + xoff;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  uint8_t* codes = side ? c.codesV : c.codesK;
  float* scales = side ? c.scalesV : c.scalesK;
  const float s0 = hsign(g.seed_sign, 2 * lane), s1 = hsign(g.seed_sign, 2 * lane + 1);
  while (mask) {
    const int bit = __ffsll((long long)mask) - 1;
    mask &= mask - 1;
    const int i = word * 64 + bit;
    const int t = min(max(c.pos[slot_base(g, b, h) + i], 0), S - 1);
    const int a = min(max(w.apos[side * TS + po + t], 0), k - 1);
    const float gb = w.gpos[side * TS + po + t];
    const E* x = X + (size_t)t * D;
    const E* ar = A + (size_t)a * D;
    float p0 = gb * Elem<DT>::get(ar, 2 * lane), p1 = gb * Elem<DT>::get(ar, 2 * lane + 1);
    float r0 = Elem<DT>::get(x, 2 * lane) - p0, r1 = Elem<DT>::get(x, 2 * lane + 1) - p1;
    float z0 = s0 * r0, z1 = s1 * r1;
    fwht_wave(z0, z1, lane);
    // Group scale (G coordinates = G/2 lanes).
    const int gl = G / 2;
    float sigma;
    if (g.scale_mode == 2) {
      // Sequential fp32 sum of squares over the group, in coordinate order.
      const int gbase = (lane / gl) * gl;
      float acc = 0.0f;
      for (int j = 0; j < gl; ++j) {
        const float a0 = __shfl(z0, gbase + j, 64), a1 = __shfl(z1, gbase + j, 64);
        const float q0 = a0 * a0;
        acc = acc + q0;
        const float q1 = a1 * a1;
        acc = acc + q1;
      }
      const float ms = acc / (float)G;
      sigma = sqrtf(ms);
    } else {
      float am = fmaxf(fabsf(z0), fabsf(z1));
      for (int o = 1; o < gl; o <<= 1) am = fmaxf(am, __shfl_xor(am, o, 64));
      sigma = g.scale_mode == 1 ? am : am / AKV_L1;
    }
    const float T = sigma * AKV_T;
    const int c0 = z0 < 0.0f ? (fabsf(z0) > T ? 0 : 1) : (fabsf(z0) > T ? 3 : 2);
    const int c1 = z1 < 0.0f ? (fabsf(z1) > T ? 0 : 1) : (fabsf(z1) > T ? 3 : 2);
    const int nib = c0 | (c1 << 2);
    const int onib = __shfl_xor(nib, 1, 64);
    if ((lane & 1) == 0) codes[(size_t)slot * (D / 4) + lane / 2] = (uint8_t)(nib | (onib << 4));
    if (lane % gl == 0) scales[(size_t)slot * (D / G) + lane / gl] = sigma;
    ++slot;
  }
}

hipError_t launch_layout(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, hipStream_t st) {
  int nsort = 0, nrec = 0;
  for (int b = 0; b < g.B; ++b) {
    nsort += g.H * ((g.S[b] + SORT_CHUNK - 1) / SORT_CHUNK);
    nrec += g.H * ((g.S[b] + 255) / 256);
  }
  const size_t lds = (size_t)g.maxK * sizeof(int);
  launch("k_shist", k_shist, dim3(nsort), dim3(256), lds, st, g, w);
  launch("k_sscan", k_sscan, dim3(g.B * g.H), dim3(1024), 0, st, g, w);
  launch("k_sscatter", k_sscatter, dim3(nsort), dim3(64), lds, st, g, w, c);
  if (g.dtype == 1) {
    launch("k_lrec", k_lrec<1>, dim3(nrec), dim3(256), 0, st, g, w, c);
  } else {
    launch("k_lrec", k_lrec<0>, dim3(nrec), dim3(256), 0, st, g, w, c);
  }
  launch("k_lscan", k_lscan, dim3(g.B * 2), dim3(1024), 0, st, g, w, c);
  const int nwords = 2 * g.prefW[g.B] * g.H;
  if (g.dtype == 1) {
    launch("k_codec", k_codec<1>, dim3((nwords + 3) / 4), dim3(256), 0, st, g, w, c, K, V);
  } else {
    launch("k_codec", k_codec<0>, dim3((nwords + 3) / 4), dim3(256), 0, st, g, w, c, K, V);
  }
  return hipGetLastError();
}

}  // namespace akv
