// Gumbel keys of the random eviction (NaCl Section 5.2): a token's key is
// binary32(log-weight + g) with g = -ln(-ln u) in binary64,
// u = (word + 1/2) / 2^32 and word = Philox4x32-10 output j mod 4 at counter
// (j / 4, h, b, layer) under key = seed.  Keys are stored as order-preserving
// uint32 bits.  Shared by the stand-alone key kernel and the column
// reduction, which draws the keys of its chunk when it runs inside a whole
// eviction.
#pragma once

#include "device_common.h"
#include "philox.h"

namespace nacl {

// ln(x) in binary64 for x >= 0 (ln 0 = -inf, ln inf = inf), to within a
// few units in the last place: x = m 2^e with m in [sqrt(1/2), sqrt(2)),
// ln m = 2 atanh(s) with s = (m - 1) / (m + 1), |s| < 0.172, summed as the
// odd series 2 s (1 + s^2/3 + s^4/5 + ... + s^20/21) (the next term is
// below 2^-59 relative), and e ln 2 added in two parts (ln 2 rounded to
// binary64 and the rest).  The quotient takes a hardware reciprocal, two
// Newton steps and one residual correction.  The keys are rounded to
// binary32 afterwards, so a few binary64 units never matter except for a
// key within that distance of a binary32 rounding boundary.
__device__ __forceinline__ double ln_f64(double x) {
  constexpr double kLn2 = 0.6931471805599453094172321;         // rounded to binary64
  constexpr double kLn2Rest = 2.319046813846299558e-17;        // ln 2 - kLn2
  constexpr double kSqrtHalf = 0.70710678118654752440;
  double m = __builtin_amdgcn_frexp_mant(x);                   // [1/2, 1)
  int e = __builtin_amdgcn_frexp_exp(x);
  if (m < kSqrtHalf) {
    m *= 2.0;
    --e;
  }
  const double f = m - 1.0;                                    // exact
  const double d = f + 2.0;
  double r = __builtin_amdgcn_rcp(d);
  r = fma(r, fma(-d, r, 1.0), r);
  r = fma(r, fma(-d, r, 1.0), r);
  double s = f * r;
  s = fma(fma(-s, d, f), r, s);
  const double z = s * s;
  double q = 1.0 / 21;
  q = fma(q, z, 1.0 / 19);
  q = fma(q, z, 1.0 / 17);
  q = fma(q, z, 1.0 / 15);
  q = fma(q, z, 1.0 / 13);
  q = fma(q, z, 1.0 / 11);
  q = fma(q, z, 1.0 / 9);
  q = fma(q, z, 1.0 / 7);
  q = fma(q, z, 1.0 / 5);
  q = fma(q, z, 1.0 / 3);
  const double s2 = 2.0 * s;
  const double lnm = fma(s2 * z, q, s2);
  const double ed = (double)e;
  const double p = ed * kLn2;
  const double perr = fma(ed, kLn2, -p);                       // exact rounding error of p
  const double res = p + (lnm + fma(ed, kLn2Rest, perr));
  if (x == 0.0) return -INFINITY;
  if (x == INFINITY) return INFINITY;
  return res;
}

// Key of one token.  MODE selects the log-weight: 0 = F (weights
// Softmax(F)), 1 = ln F (weights F), 2 = none (uniform).
template <int MODE>
__device__ __forceinline__ uint32_t gumbel_order_key(float f, uint32_t word) {
  const double u = ((double)word + 0.5) * 0x1p-32;
  const double g = -ln_f64(-ln_f64(u));
  double key = g;
  if constexpr (MODE == 0) key = (double)f + g;
  if constexpr (MODE == 1) key = ln_f64((double)f) + g;
  return float_order_key((float)key);
}

// The keys of tokens j0 .. j0 + n - 1 (j0 a multiple of 4, n <= 4: one
// Philox block) of head (b, h) with scores f[0 .. n), into out[0 .. n).
// `mode` is uniform across the calling wave.
__device__ __forceinline__ void gumbel_block_keys(int mode, int j0, int n, int b, int h, uint32_t layer,
                                                  uint32_t k0, uint32_t k1, const float (&f)[4],
                                                  uint32_t (&out)[4]) {
  const U32x4 w = philox4x32_10(U32x4{(uint32_t)(j0 >> 2), (uint32_t)h, (uint32_t)b, layer}, k0, k1);
  const uint32_t word[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (e < n) {
      if (mode == 0) out[e] = gumbel_order_key<0>(f[e], word[e]);
      else if (mode == 1) out[e] = gumbel_order_key<1>(f[e], word[e]);
      else out[e] = gumbel_order_key<2>(f[e], word[e]);
    }
  }
}

}  // namespace nacl
