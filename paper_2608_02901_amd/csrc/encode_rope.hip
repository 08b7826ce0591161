// Positional rotation of the compression pass (Sec. 3.2 "RoPE"): the keys
// arrive before the rotation; the observation pass needs them rotated, as
// attention sees them, while assignment, projection and storage keep the
// unrotated ones.
//
// k_rope_prep writes, for every position t < max S, the fp32 cosines and
// sines of the rotation R_t (the fp32 roundings of the fp64 cos and sin of
// the fp64 angle t * inv_freq[f]; pair f is the coordinate pair (f, f + D/2))
// and, for every (request, head) with t < S_b, the rotated key
//   (c x_f - s x_{f+D/2}, s x_f + c x_{f+D/2})
// formed in fp64 (exact products of fp32 factors, one rounding per
// coordinate), rounded to fp32 and then to the cache dtype.  Thread = (t, f);
// a workgroup covers four positions, its 64 lanes the 64 pairs of one of
// them, so the key reads and writes of a head are 128-byte runs.
#include "akv_common.h"

namespace akv {

template <int DT>
__global__ __launch_bounds__(256) void k_rope_prep(Geo g, Ws w, const void* Kin) {
  constexpr int D = AKV_D, F = AKV_D / 2;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6), f = threadIdx.x & 63;
  if (t >= g.maxS) return;
  const double ang = (double)t * (double)g.invf[f];
  const float c = (float)cos(ang), s = (float)sin(ang);
  *(float2*)&w.cs[(size_t)t * D + 2 * f] = make_float2(c, s);
  const double cd = c, sd = s;
  for (int b = 0; b < g.B; ++b) {
    const int S = g.S[b];
    if (t >= S) continue;
    for (int h = 0; h < g.H; ++h) {
      const size_t row = ((size_t)g.prefS[b] * g.H + (size_t)h * S + t) * D;
      const double a = Elem<DT>::get(Kin, row + f), bb = Elem<DT>::get(Kin, row + f + F);
      const float r0 = (float)(cd * a - sd * bb), r1 = (float)(sd * a + cd * bb);
      Elem<DT>::put(w.krot, row + f, r0);
      Elem<DT>::put(w.krot, row + f + F, r1);
    }
  }
}

hipError_t launch_rope(const Geo& g, const Ws& w, const void* K, hipStream_t st) {
  const int nblk = (g.maxS + 3) / 4;
  if (g.dtype == 1)
    launch("k_rope_prep", k_rope_prep<1>, dim3(nblk), dim3(256), 0, st, g, w, K);
  else
    launch("k_rope_prep", k_rope_prep<0>, dim3(nblk), dim3(256), 0, st, g, w, K);
  return hipGetLastError();
}

}  // namespace akv
