// Reproducible elementary functions for gfx950, built only from IEEE-754
// binary32 basic operations (add, multiply, fused multiply-add, correctly
// rounded divide, round-to-integral) whose results every conforming unit
// returns bit for bit.  No hardware approximation (v_exp_f32, v_rcp_f32,
// v_rsq_f32) is used.
//
// exp:  Cody and Waite's additive reduction x = n ln2 + r with ln2 split in a
//       high and a low binary32 part, then the degree-7 Taylor polynomial of
//       exp(r) by Horner's rule, then scaling by 2^n in two exact-exponent
//       steps (RepOps rebuilds exp with a controlled order, Section 3.1 of the
//       Verde paper; the method is Cody-Waite + Taylor).
// gelu: tanh form through 0.5 (1 + tanh z) = 1 / (1 + exp(-2z)).
// gelu': with s = 1 / (1 + exp(-2z)) the forward is x * s, so its derivative
//       is s + x s (1 - s) * 2 sqrt(2/pi) (1 + 3 * 0.044715 x^2).
// sin/cos: Cody and Waite's additive reduction by pi/2 (pi/2 split in three
//       binary32 parts), Taylor polynomials of degree 9 and 10 on |r| <= pi/4
//       by Horner's rule, quadrant selection.
// silu: x / (1 + exp(-x)); silu' = s + x s (1 - s) with s = 1 / (1 + exp(-x)).
// erf: Taylor series below 0.5; beyond, erfc(z) = exp(-z^2) R(z) with R =
//       exp(z^2) erfc(z) from Chebyshev interpolants on [0.5, 2.5] and
//       [2.5, 10.5]; exp(-c x^2) from a split of x so that x^2 is never rounded.
// gelu_erf: x Phi(x), Phi's lower tail taken directly (no 1 + erf).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace repops {

// Nearest binary32 values to log2(e), ln2 (high part) and ln2 - ln2_hi.
constexpr float kLog2e = 0x1.715476p+0f;
constexpr float kLn2Hi = 0x1.62e43p-1f;
constexpr float kLn2Lo = -0x1.05c61p-29f;
// 1/k! rounded to binary32, k = 2..7 (the k = 0, 1 coefficients are 1).
constexpr float kInvFact2 = 0x1p-1f;
constexpr float kInvFact3 = 0x1.555556p-3f;
constexpr float kInvFact4 = 0x1.555556p-5f;
constexpr float kInvFact5 = 0x1.111112p-7f;
constexpr float kInvFact6 = 0x1.6c16c2p-10f;
constexpr float kInvFact7 = 0x1.a01a02p-13f;
// Nearest binary32 values to 0.044715 and sqrt(2/pi).
constexpr float kGeluCubic = 0x1.6e4e26p-5f;
constexpr float kGeluScale = 0x1.988454p-1f;
// Nearest binary32 value to 3 * 0.044715 = 0.134145, and 2 * kGeluScale (exact).
constexpr float kGeluCubic3 = 0x1.12ba9ep-3f;
constexpr float kGeluScale2 = 0x1.988454p+0f;

__device__ __forceinline__ float pow2_exact(int e) {
  // 2^e for e in [-126, 127] from the exponent field alone.
  return __int_as_float((e + 127) << 23);
}

__device__ __forceinline__ float rep_exp(float x) {
  const float t = x * kLog2e;
  const float nf = __builtin_rintf(t);  // v_rndne_f32: nearest, ties to even
  // Clamp before the integer conversion so that every lane takes the same
  // straight-line path; out-of-range lanes are replaced below.
  const float nc = __builtin_fminf(__builtin_fmaxf(nf, -151.0f), 128.0f);
  float r = __builtin_fmaf(nc, -kLn2Hi, x);
  r = __builtin_fmaf(nc, -kLn2Lo, r);
  float p = __builtin_fmaf(kInvFact7, r, kInvFact6);
  p = __builtin_fmaf(p, r, kInvFact5);
  p = __builtin_fmaf(p, r, kInvFact4);
  p = __builtin_fmaf(p, r, kInvFact3);
  p = __builtin_fmaf(p, r, kInvFact2);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  const int n = static_cast<int>(nc);
  const int lo = n >> 1;  // floor(n / 2): arithmetic shift
  const int hi = n - lo;
  float y = (p * pow2_exact(lo)) * pow2_exact(hi);
  y = (nf > 128.0f) ? __builtin_huge_valf() : y;
  y = (nf < -151.0f) ? 0.0f : y;
  y = (x != x) ? x : y;  // NaN in, NaN out
  return y;
}

__device__ __forceinline__ float rep_gelu(float x) {
  float u = x * x;
  u = u * x;
  float z = __builtin_fmaf(kGeluCubic, u, x);
  z = z * kGeluScale;
  const float w = z * -2.0f;
  const float d = 1.0f + rep_exp(w);
  return x / d;  // correctly rounded division
}

// Nearest binary32 value to 2/pi; pi/2 = kHalfPi1 + kHalfPi2 + kHalfPi3 + O(2^-76),
// each part the binary32 value nearest the remainder.
constexpr float kTwoOverPi = 0x1.45f306p-1f;
constexpr float kHalfPi1 = 0x1.921fb6p+0f;
constexpr float kHalfPi2 = -0x1.777a5cp-25f;
constexpr float kHalfPi3 = -0x1.ee59dap-50f;
// (-1)^k / (2k+1)! and (-1)^k / (2k)! rounded to binary32.
constexpr float kSin3 = -0x1.555556p-3f;
constexpr float kSin5 = 0x1.111112p-7f;
constexpr float kSin7 = -0x1.a01a02p-13f;
constexpr float kSin9 = 0x1.71de3ap-19f;
constexpr float kCos2 = -0x1p-1f;
constexpr float kCos4 = 0x1.555556p-5f;
constexpr float kCos6 = -0x1.6c16c2p-10f;
constexpr float kCos8 = 0x1.a01a02p-16f;
constexpr float kCos10 = -0x1.27e4fcp-22f;

// sin and cos of x.  n = rint(x * 2/pi); r = x - n pi/2 in three fused steps
// (r = x when n = 0); u = r*r; s = r + (r u) P(u), c = 1 + u Q(u); the quadrant
// n mod 4 picks (s, c), (c, -s), (-s, -c) or (-c, s).  x = +-0 gives (x, 1);
// non-finite x gives NaN.  Straight-line code: every lane takes the same path.
__device__ __forceinline__ void rep_sincos(float x, float& sin_out, float& cos_out) {
  const bool finite = __builtin_isfinite(x);
  const float xs = finite ? x : 0.0f;
  const float t = xs * kTwoOverPi;
  const float n = __builtin_rintf(t);
  float r = __builtin_fmaf(n, -kHalfPi1, xs);
  r = __builtin_fmaf(n, -kHalfPi2, r);
  r = __builtin_fmaf(n, -kHalfPi3, r);
  r = (n != 0.0f) ? r : xs;
  const float u = r * r;
  float ps = __builtin_fmaf(kSin9, u, kSin7);
  ps = __builtin_fmaf(ps, u, kSin5);
  ps = __builtin_fmaf(ps, u, kSin3);
  const float r3 = r * u;
  const float sv = __builtin_fmaf(r3, ps, r);
  float pc = __builtin_fmaf(kCos10, u, kCos8);
  pc = __builtin_fmaf(pc, u, kCos6);
  pc = __builtin_fmaf(pc, u, kCos4);
  pc = __builtin_fmaf(pc, u, kCos2);
  const float cv = __builtin_fmaf(u, pc, 1.0f);
  const float quarter = n * 0.25f;
  const float fq = n - 4.0f * __builtin_floorf(quarter);  // exact, in {0, 1, 2, 3}
  const int q = static_cast<int>(fq);
  float so = (q & 1) ? cv : sv;
  float co = (q & 1) ? sv : cv;
  so = (q & 2) ? -so : so;
  co = (q == 1 || q == 2) ? -co : co;
  so = (x == 0.0f) ? x : so;
  co = (x == 0.0f) ? 1.0f : co;
  const float qnan = __builtin_nanf("");
  sin_out = finite ? so : qnan;
  cos_out = finite ? co : qnan;
}

// Taylor coefficients 2/sqrt(pi) (-1)^n / (n! (2n + 1)), n = 0..7.
constexpr float kErfT0 = 0x1.20dd76p+0f, kErfT1 = -0x1.812746p-2f, kErfT2 = 0x1.ce2f22p-4f,
                kErfT3 = -0x1.b82ce4p-6f, kErfT4 = 0x1.565bcep-8f, kErfT5 = -0x1.c02db4p-11f,
                kErfT6 = 0x1.f9a326p-14f, kErfT7 = -0x1.f4d25cp-17f;
// exp(z^2) erfc(z): degree-12 Chebyshev interpolant in s = z - 1.5 on [0.5, 2.5]
// and degree-8 interpolant in s = (1/(1+z) - 3/16) * 9.5 on [2.5, 10.5],
// binary32-rounded monomial coefficients, constant term first.
constexpr float kErfcA[13] = {
    0x1.494db0p-2f, -0x1.4f1988p-3f, 0x1.37ea26p-4f, -0x1.0dc542p-5f, 0x1.b6596ep-7f,
    -0x1.5135c2p-8f, 0x1.ee6646p-10f, -0x1.5c00ccp-11f, 0x1.d5624ap-13f, -0x1.243bd4p-14f,
    0x1.71a8d4p-16f, -0x1.364e28p-17f, 0x1.6a86acp-19f};
constexpr float kErfcB[9] = {
    0x1.040c3ap-3f, 0x1.565eecp-4f, 0x1.c46bacp-8f, -0x1.24aa48p-13f, -0x1.44b7dap-14f,
    0x1.7d0926p-19f, 0x1.82a7a8p-20f, -0x1.1ebc20p-23f, -0x1.dd0088p-26f};
constexpr float kInvSqrt2 = 0x1.6a09e6p-1f;
constexpr float kInvSqrt2Pi = 0x1.988454p-2f;

__device__ __forceinline__ float rep_erf_small(float z) {
  const float u = z * z;
  float p = __builtin_fmaf(kErfT7, u, kErfT6);
  p = __builtin_fmaf(p, u, kErfT5);
  p = __builtin_fmaf(p, u, kErfT4);
  p = __builtin_fmaf(p, u, kErfT3);
  p = __builtin_fmaf(p, u, kErfT2);
  p = __builtin_fmaf(p, u, kErfT1);
  p = __builtin_fmaf(p, u, kErfT0);
  return z * p;
}

// exp(-c x^2), c = 1 or 1/2: h = x with its low 12 significand bits cleared,
// so h*h is exact; exp(-c x^2) = exp(-(h h) c) exp(-(x - h)(x + h) c).
__device__ __forceinline__ float rep_exp_neg_sq(float x, float c) {
  const float h = __uint_as_float(__float_as_uint(x) & 0xFFFFF000u);
  const float hh = h * h;
  const float a = -(hh * c);
  const float dl = x - h;
  const float ds = x + h;
  const float d = dl * ds;
  const float b = -(d * c);
  return rep_exp(a) * rep_exp(b);
}

// exp(z^2) erfc(z) for z >= 0.5: each interval's Horner chain from its
// leading coefficient.  Every lane evaluates both (straight-line code, the
// coefficients as instruction literals) and keeps the one for its interval.
__device__ __forceinline__ float rep_erfc_scaled(float z) {
  const bool lo = z < 2.5f;
  const float t = 1.0f / (1.0f + z);
  const float sa = z - 1.5f;
  const float sb = (t - 0.1875f) * 9.5f;
  float pa = kErfcA[12];
#pragma unroll
  for (int j = 11; j >= 0; --j) pa = __builtin_fmaf(pa, sa, kErfcA[j]);
  float pb = kErfcB[8];
#pragma unroll
  for (int j = 7; j >= 0; --j) pb = __builtin_fmaf(pb, sb, kErfcB[j]);
  return lo ? pa : pb;
}

__device__ __forceinline__ float rep_erf(float x) {
  const float a = __builtin_fabsf(x);
  const float small = rep_erf_small(x);
  const float q = (a >= 10.5f) ? 0.0f : rep_exp_neg_sq(a, 1.0f) * rep_erfc_scaled(a);
  const float r = 1.0f - q;
  float y = (x < 0.0f) ? -r : r;
  y = (a < 0.5f) ? small : y;
  return (x != x) ? x : y;
}

// Phi(x), the standard normal distribution function.
__device__ __forceinline__ float rep_normal_cdf(float x, float a, float e) {
  const float z = a * kInvSqrt2;
  const float xs = x * kInvSqrt2;
  const float mid = __builtin_fmaf(0.5f, rep_erf_small(xs), 0.5f);
  const float er = e * rep_erfc_scaled(z);
  const float q = (z >= 10.5f) ? 0.0f : er * 0.5f;
  const float tail = (x > 0.0f) ? 1.0f - q : q;
  return (z < 0.5f) ? mid : tail;
}

__device__ __forceinline__ float rep_gelu_erf(float x) {
  const float a = __builtin_fabsf(x);
  const float y = x * rep_normal_cdf(x, a, rep_exp_neg_sq(a, 0.5f));
  return (x != x) ? x : y;
}

__device__ __forceinline__ float rep_gelu_erf_grad(float x) {
  const float a = __builtin_fabsf(x);
  const float e = rep_exp_neg_sq(a, 0.5f);
  const float phi = e * kInvSqrt2Pi;
  const float g = __builtin_fmaf(x, phi, rep_normal_cdf(x, a, e));
  return (x != x) ? x : g;
}

__device__ __forceinline__ float rep_silu(float x) {
  const float w = -x;
  const float d = 1.0f + rep_exp(w);
  return x / d;
}

__device__ __forceinline__ float rep_silu_grad(float x) {
  const float w = -x;
  const float d = 1.0f + rep_exp(w);
  const float s = 1.0f / d;
  const float om = 1.0f - s;
  const float xs = x * s;
  return __builtin_fmaf(xs, om, s);
}

// Derivative of rep_gelu, one fixed operation sequence.
__device__ __forceinline__ float rep_gelu_grad(float x) {
  const float u = x * x;
  const float u3 = u * x;
  float z = __builtin_fmaf(kGeluCubic, u3, x);
  z = z * kGeluScale;
  const float w = z * -2.0f;
  const float d = 1.0f + rep_exp(w);
  const float s = 1.0f / d;
  const float om = 1.0f - s;
  const float v = __builtin_fmaf(kGeluCubic3, u, 1.0f);
  const float t1 = x * s;
  const float t2 = t1 * om;
  const float t3 = kGeluScale2 * v;
  return __builtin_fmaf(t2, t3, s);
}

}  // namespace repops
