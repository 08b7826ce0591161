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
//   k_sscan    : per block of 256 anchors, each anchor's column of chunk
//                counts becomes its exclusive prefix, its total goes to the
//                table's last row;
//   k_sscatter : per chunk, the anchors' start slots (scan of the totals plus
//                the column prefix), then a stable scatter of the chunk's
//                tokens 64 at a time, one 16-byte record per token;
//   k_lrec     : per sorted slot, the record spread over the layout's arrays,
//                flag words and popcounts;
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
  return w.shist + (size_t)g.prefKT[b] + (size_t)h * g.k[b] * (nT + 1);
}

// Table of a head: rows = sort chunks, columns = anchors (row nT: totals).
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
  int32_t* out = shist_base(g, w, b, h) + (size_t)ch * k;
  for (int a = threadIdx.x; a < k; a += blockDim.x) out[a] = hist[a];
}

// One thread per (request, head, anchor): the anchor's column of chunk counts
// becomes its exclusive prefix sum in place (the counts of its tokens in the
// earlier chunks), and its total goes to row nT; loads are issued 32 rows at
// a time.
__global__ __launch_bounds__(256) void k_sscan(Geo g, Ws w) {
  int idx = blockIdx.x;
  int b = 0;
  for (; b < g.B; ++b) {
    const int n = g.H * ((g.k[b] + 255) / 256);
    if (idx < n) break;
    idx -= n;
  }
  const int k = g.k[b];
  const int nT = (g.S[b] + SORT_CHUNK - 1) / SORT_CHUNK;
  const int nab = (k + 255) / 256;
  const int h = idx / nab, a = (idx % nab) * 256 + threadIdx.x;
  if (a >= k) return;
  int32_t* col = shist_base(g, w, b, h) + a;
  constexpr int U = 32;
  int s = 0;
  for (int c0 = 0; c0 < nT; c0 += U) {
    int v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = c0 + u < nT ? col[(size_t)(c0 + u) * k] : 0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (c0 + u < nT) col[(size_t)(c0 + u) * k] = s;
      s += v[u];
    }
  }
  col[(size_t)nT * k] = s;
}

// One workgroup per chunk.  The anchors' start slots for this chunk (first
// slot of the anchor plus its column prefix) and the chunk's token records
// (anchor indices, stored coefficients, residual flags) are staged in LDS by
// all four waves; then one wave takes the tokens in groups of 64 in position
// order.  Lanes holding the same anchor find each other with one ballot per
// bit of the anchor index; a token's slot is its anchor's start plus the
// equal tokens before it in the group, and the group's last such lane
// advances the start.  The token's record goes to its slot as one 16-byte
// write, so the records are read in position order and each token costs one
// scattered write; k_lrec then spreads them over the layout's arrays.
template <int DT>
__global__ __launch_bounds__(256) void k_sscatter(Geo g, Ws w, Cache c) {
  extern __shared__ __align__(16) int lds[];
  __shared__ int wsum[64], wpre[65];
  int* sa = lds;                       // [SORT_CHUNK] value-side anchor
  int* ska = sa + SORT_CHUNK;          // [SORT_CHUNK] key-side anchor
  float* sgk = (float*)(ska + SORT_CHUNK);
  float* sgv = sgk + SORT_CHUNK;
  uint8_t* sfk = (uint8_t*)(sgv + SORT_CHUNK);
  uint8_t* sfv = sfk + SORT_CHUNK;
  int* run = (int*)(sfv + SORT_CHUNK);  // [k] running start slot per anchor
  int idx = blockIdx.x;
  const int b = locate_sort(g, idx);
  const int S = g.S[b], k = g.k[b];
  const int nT = (S + SORT_CHUNK - 1) / SORT_CHUNK;
  const int h = idx / nT, ch = idx % nT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int32_t* tab = shist_base(g, w, b, h);
  const int32_t* first = tab + (size_t)nT * k;
  const int32_t* colp = tab + (size_t)ch * k;
  const size_t TS = (size_t)g.prefS[g.B] * g.H;
  const size_t po = (size_t)g.prefS[b] * g.H + (size_t)h * S;
  const size_t so = slot_base(g, b, h);
  const int t0 = ch * SORT_CHUNK, t1 = min(S, t0 + SORT_CHUNK), nt = t1 - t0;
  constexpr int RU = SORT_CHUNK / 256;
  {
    float gk[RU], gv[RU];
    int ak[RU], av[RU];
    uint8_t fk[RU], fv[RU];
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int i = min(u * 256 + tid, nt - 1);
      av[u] = w.apos[TS + po + t0 + i];
      ak[u] = w.apos[po + t0 + i];
      gk[u] = w.gpos[po + t0 + i];
      gv[u] = w.gpos[TS + po + t0 + i];
      fk[u] = w.sel[po + t0 + i];
      fv[u] = w.sel[TS + po + t0 + i];
    }
    // First slot of each anchor: exclusive scan of the anchor totals, up to
    // TU tiles of 256 per round (all loaded before the wave scans, then one
    // scan of the (tile, wave) sums); plus the column prefix of this chunk.
    constexpr int TU = 16;
    int carry = 0;
    for (int a0 = 0; a0 < k; a0 += TU * 256) {
      int v[TU], x[TU], cp[TU];
#pragma unroll
      for (int u = 0; u < TU; ++u) {
        const int a = a0 + u * 256 + tid;
        v[u] = a < k ? first[a] : 0;
        cp[u] = a < k ? colp[a] : 0;
      }
#pragma unroll
      for (int u = 0; u < TU; ++u) {
        x[u] = v[u];
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(x[u], o, 64);
          if (lane >= o) x[u] += y;
        }
        if (lane == 63) wsum[u * 4 + (tid >> 6)] = x[u];
      }
      __syncthreads();
      if (tid < 64) {
        const int c0 = wsum[lane];
        int y = c0;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int z = __shfl_up(y, o, 64);
          if (lane >= o) y += z;
        }
        wpre[lane] = y - c0;
        if (lane == 63) wpre[TU * 4] = y;
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < TU; ++u) {
        const int a = a0 + u * 256 + tid;
        if (a < k) run[a] = carry + wpre[u * 4 + (tid >> 6)] + x[u] - v[u] + cp[u];
      }
      carry += wpre[TU * 4];
      __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int i = u * 256 + tid;
      sa[i] = av[u];
      ska[i] = ak[u];
      sgk[i] = gk[u];
      sgv[i] = gv[u];
      sfk[i] = fk[u];
      sfv[i] = fv[u];
    }
  }
  __syncthreads();
  if (tid >= 64) return;
  const int nbits = 32 - __clz(k);  // key a + 1 lies in [0, k]
  for (int i0 = 0; i0 < nt; i0 += 64) {
    const int i = i0 + lane;
    const int a = (i >= nt || sa[i] >= k) ? -1 : sa[i];
    const unsigned key = (unsigned)(a + 1);
    unsigned long long peers = ~0ull;
    for (int bit = 0; bit < nbits; ++bit) {
      const bool on = (key >> bit) & 1u;
      const unsigned long long bb = __ballot(on);
      peers &= on ? bb : ~bb;
    }
    const int before = __popcll(peers & ((1ull << lane) - 1ull));
    const bool lastp = (peers >> lane) == 1ull;
    if (a >= 0) {
      const int dest = run[a] + before;
      if (dest >= 0 && dest < S) {
        // One 16-byte record per token: position with the residual flags in
        // bits 30 and 31, the two anchor indices, the two coefficients.
        const uint32_t w0 = (uint32_t)(t0 + i) | (sfk[i] ? 1u << 30 : 0u) | (sfv[i] ? 1u << 31 : 0u);
        const uint32_t w1 = (uint32_t)(uint16_t)ska[i] | ((uint32_t)a << 16);
        w.srec[so + dest] = make_uint4(w0, w1, __float_as_uint(sgk[i]), __float_as_uint(sgv[i]));
      }
      if (lastp) run[a] = dest + 1;
    }
  }
}

// Per 256 sorted slots: the records become the layout's per-slot arrays,
// and the residual flag words and their popcounts; a slot holding an
// out-of-range position raises the layout error bit.  Padding slots of the
// head's last word get anchor 0 with coefficient 0.
template <int DT>
__global__ __launch_bounds__(256) void k_lrec(Geo g, Ws w, Cache c) {
  int idx = blockIdx.x;
  const int b = locate(g, 256, 1, idx);
  const int S = g.S[b];
  const int nt = (S + 255) / 256;
  const int h = idx / nt, i = (idx % nt) * 256 + threadIdx.x;
  const size_t so = slot_base(g, b, h);
  bool fk = false, fv = false;
  if (i < S) {
    const uint4 r = w.srec[so + i];
    const int t = (int)(r.x & 0x3FFFFFFFu);
    if (t >= S) atomicOr(&c.header[2], 8u);
    fk = (r.x >> 30) & 1u;
    fv = r.x >> 31;
    c.pos[so + i] = t;
    c.idxK[so + i] = (uint16_t)(r.y & 0xFFFFu);
    c.idxV[so + i] = (uint16_t)(r.y >> 16);
    Elem<DT>::put(c.gK, so + i, __uint_as_float(r.z));
    Elem<DT>::put(c.gV, so + i, __uint_as_float(r.w));
  } else if (i < ((S + 63) & ~63)) {
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
// over its (head, word) sequence.  Words are read coalesced, up to 16 tiles
// of 1024 per round (all loads issued before the wave scans), then one scan
// of the (tile, wave) sums.
__global__ __launch_bounds__(1024) void k_lscan(Geo g, Ws w, Cache c) {
  constexpr int TU = 16;
  __shared__ int wsum[TU * 16], wpre[TU * 16 + 1];
  const int b = blockIdx.x >> 1, side = blockIdx.x & 1;
  const int nw = g.H * ((g.S[b] + 63) / 64);
  const size_t WT = (size_t)g.prefW[g.B] * g.H;
  const size_t wo = (size_t)g.prefW[b] * g.H;
  const int32_t* cnt = w.wcnt + side * WT + wo;
  int32_t* pc = (side ? c.pcV : c.pcK) + wo;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int carry = side ? g.prefNV[b] : g.prefNK[b];
  for (int a0 = 0; a0 < nw; a0 += TU * 1024) {
    int v[TU], x[TU];
#pragma unroll
    for (int u = 0; u < TU; ++u) {
      const int i = a0 + u * 1024 + tid;
      v[u] = i < nw ? cnt[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < TU; ++u) {
      x[u] = v[u];
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x[u], o, 64);
        if (lane >= o) x[u] += y;
      }
      if (lane == 63) wsum[u * 16 + wave] = x[u];
    }
    __syncthreads();
    if (tid < 64) {  // 256 sums, four per lane in order
      int c4[4], t4 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c4[j] = wsum[4 * lane + j];
        t4 += c4[j];
      }
      int y = t4;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int z = __shfl_up(y, o, 64);
        if (lane >= o) y += z;
      }
      int run = y - t4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        wpre[4 * lane + j] = run;
        run += c4[j];
      }
      if (lane == 63) wpre[TU * 16] = y;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < TU; ++u) {
      const int i = a0 + u * 1024 + tid;
      if (i < nw) pc[i] = carry + wpre[u * 16 + wave] + x[u] - v[u];
    }
    carry += wpre[TU * 16];
    __syncthreads();
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
  // The word's mask, first residual slot and the records of its 64 slots
  // (position, anchors, coefficients, as the scatter left them) are read
  // together, the records without waiting for the mask.
  unsigned long long mask = (side ? c.maskV : c.maskK)[wo];
  int slot = (side ? c.pcV : c.pcK)[wo];
  const uint4 rec = w.srec[slot_base(g, b, h) + (size_t)word * 64 + lane];
  if (!mask) return;
  const size_t ko = (size_t)g.prefK[b] * g.H + (size_t)h * k;
  const size_t xoff = ((size_t)g.prefS[b] * g.H + (size_t)h * S) * D;
  const E* X = (const E*)(side ? Vin : Kin) + xoff;
  const E* A = (const E*)(side ? c.ancV : c.ancK) + ko * D;
  uint8_t* codes = side ? c.codesV : c.codesK;
  float* scales = side ? c.scalesV : c.scalesK;
  const float s0 = sign_bit(g.sgnbits, 2 * lane), s1 = sign_bit(g.sgnbits, 2 * lane + 1);
  // Position, anchor and coefficient of every slot of the word, one lane each
  // (clamped: padding slots of the last word hold no record and no flag).
  const int tj = min((int)(rec.x & 0x3FFFFFFFu), S - 1);
  const int aj = min((int)(side ? rec.y >> 16 : rec.y & 0xFFFFu), k - 1);
  const float gj = __uint_as_float(side ? rec.w : rec.z);
  // Up to CB flagged slots per round; their token and anchor coordinates
  // (2 per lane) are loaded together before any is encoded.
  constexpr int CB = 4;
  while (mask) {
    int bit[CB];
    float x0[CB], x1[CB], a0[CB], a1[CB], gq[CB];
#pragma unroll
    for (int q = 0; q < CB; ++q) {
      bit[q] = mask ? __ffsll((long long)mask) - 1 : -1;
      mask &= mask - 1;
      x0[q] = x1[q] = a0[q] = a1[q] = gq[q] = 0.0f;
      if (bit[q] >= 0) {
        const int t = __builtin_amdgcn_readlane(tj, bit[q]);
        const int a = __builtin_amdgcn_readlane(aj, bit[q]);
        gq[q] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gj), bit[q]));
        const E* x = X + (size_t)t * D;
        const E* ar = A + (size_t)a * D;
        x0[q] = Elem<DT>::get(x, 2 * lane);
        x1[q] = Elem<DT>::get(x, 2 * lane + 1);
        a0[q] = Elem<DT>::get(ar, 2 * lane);
        a1[q] = Elem<DT>::get(ar, 2 * lane + 1);
      }
    }
#pragma unroll
    for (int q = 0; q < CB; ++q) {
      if (bit[q] < 0) break;
      const float p0 = gq[q] * a0[q], p1 = gq[q] * a1[q];
      const float r0 = x0[q] - p0, r1 = x1[q] - p1;
      float z0 = r0, z1 = r1;
      if (g.rot) {  // randomized Hadamard rotation (uniform branch)
        z0 = s0 * r0;
        z1 = s1 * r1;
        fwht_wave_dpp(z0, z1, lane);
      }
      // Group scale (G coordinates = G/2 lanes).
      const int gl = G / 2;
      float sigma;
      if (g.scale_mode == 2) {
        // Sequential fp32 sum of squares over the group, in coordinate order.
        const int gbase = (lane / gl) * gl;
        float acc = 0.0f;
        for (int j = 0; j < gl; ++j) {
          const float b0 = __shfl(z0, gbase + j, 64), b1 = __shfl(z1, gbase + j, 64);
          const float q0 = b0 * b0;
          acc = acc + q0;
          const float q1 = b1 * b1;
          acc = acc + q1;
        }
        const float ms = acc / (float)G;
        sigma = sqrtf(ms);
      } else {
        float am = fmaxf(fabsf(z0), fabsf(z1));
        for (int o = 1; o < gl; o <<= 1) am = fmaxf(am, __shfl_xor(am, o, 64));
        sigma = g.scale_mode == 1 ? am : (g.scale_mode == 3 ? am * 0.25f : am / AKV_L1);
      }
      const float T = sigma * g.thr;
      const int c0 = z0 < 0.0f ? (fabsf(z0) > T ? 0 : 1) : (fabsf(z0) > T ? 3 : 2);
      const int c1 = z1 < 0.0f ? (fabsf(z1) > T ? 0 : 1) : (fabsf(z1) > T ? 3 : 2);
      const int nib = c0 | (c1 << 2);
      const int onib = __shfl_xor(nib, 1, 64);
      if ((lane & 1) == 0) codes[(size_t)slot * (D / 4) + lane / 2] = (uint8_t)(nib | (onib << 4));
      if (lane % gl == 0) scales[(size_t)slot * (D / G) + lane / gl] = sigma;
      ++slot;
    }
  }
}

hipError_t launch_layout(const Geo& g, const Ws& w, const Cache& c, const void* K, const void* V, hipStream_t st) {
  int nsort = 0, nrec = 0;
  for (int b = 0; b < g.B; ++b) {
    nsort += g.H * ((g.S[b] + SORT_CHUNK - 1) / SORT_CHUNK);
    nrec += g.H * ((g.S[b] + 255) / 256);
  }
  const size_t lds = (size_t)g.maxK * sizeof(int);
  int nscan = 0;
  for (int b = 0; b < g.B; ++b) nscan += g.H * ((g.k[b] + 255) / 256);
  const size_t lds_scatter = (size_t)SORT_CHUNK * 18 + (size_t)g.maxK * sizeof(int);
  launch("k_shist", k_shist, dim3(nsort), dim3(256), lds, st, g, w);
  launch("k_sscan", k_sscan, dim3(nscan), dim3(256), 0, st, g, w);
  // Above 64 KiB (more than about 7000 anchors per head) the kernel asks
  // for the larger LDS allocation gfx950 offers.
  if (lds_scatter > 65536) {
    const hipError_t e = g.dtype == 1
        ? hipFuncSetAttribute((const void*)k_sscatter<1>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_scatter)
        : hipFuncSetAttribute((const void*)k_sscatter<0>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_scatter);
    if (e != hipSuccess) return e;
  }
  if (g.dtype == 1) {
    launch("k_sscatter", k_sscatter<1>, dim3(nsort), dim3(256), lds_scatter, st, g, w, c);
    launch("k_lrec", k_lrec<1>, dim3(nrec), dim3(256), 0, st, g, w, c);
  } else {
    launch("k_sscatter", k_sscatter<0>, dim3(nsort), dim3(256), lds_scatter, st, g, w, c);
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
