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
