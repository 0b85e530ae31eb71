// Wave-level helpers shared by the tiled kernels (gfx950, wave64): compile-time
// loops, DPP row moves, exponentials and the XCD-aware workgroup numbering.
#pragma once

#include <hip/hip_runtime.h>

#include <utility>

namespace vtrace {

// A native 16-byte vector: plain vector loads and stores, kept in registers.
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// Calls f(std::integral_constant<int, i>) for i = 0..N-1, unrolled at compile
// time so that arrays indexed by i stay in registers.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// DPP row moves on a double (two 32-bit halves).  Lanes whose source falls
// outside their row of 16 read 0 (bound_ctrl), so the move needs no copy of
// the old value; every caller overrides or ignores those lanes.
//   0x100 + k (row_shl:k): lane i of a row reads lane i+k;
//   kRowShr15 (row_shr:15): lane 15 of a row reads lane 0.
template <int kCtrl>
__device__ __forceinline__ double dpp_f64(double x) {
  const unsigned long long u = __double_as_longlong(x);
  int lo = static_cast<int>(u & 0xffffffffu);
  int hi = static_cast<int>(u >> 32);
  lo = __builtin_amdgcn_update_dpp(0, lo, kCtrl, 0xF, 0xF, true);
  hi = __builtin_amdgcn_update_dpp(0, hi, kCtrl, 0xF, 0xF, true);
  return __longlong_as_double(static_cast<long long>(
      (static_cast<unsigned long long>(static_cast<unsigned>(hi)) << 32) | static_cast<unsigned>(lo)));
}
constexpr int kRowShl1 = 0x101;
constexpr int kRowShr15 = 0x11F;

// e^x from the hardware base-2 exponential (about one ulp; results below the
// normal range flush to zero, harmless where every term joins a sum >= 1).
__device__ __forceinline__ float exp_fast(float x) {
  constexpr float kLog2e = 1.44269504088896340736f;
  return __builtin_amdgcn_exp2f(x * kLog2e);
}

// e^x in float64 for finite x <= 0: Cody-Waite reduction x = k ln2 + r with
// |r| <= ln2/2 (ln2 split into a 32-bit head, so k*head is exact, and a tail),
// then the Taylor series of e^r to degree 9 (truncation below 7e-12 relative)
// and a scaling by 2^k.  Arguments below -1000 are raised to -1000, where the
// result has already underflowed to zero; NaN stays NaN.
__device__ __forceinline__ double exp_nonpos_f64(double x) {
  constexpr double kLog2e = 1.4426950408889634;
  constexpr double kLn2Hi = 0.6931471803691238;      // ln2 rounded to 32 bits
  constexpr double kLn2Lo = 1.9082149292705877e-10;  // ln2 - kLn2Hi
  x = x < -1000.0 ? -1000.0 : x;
  const double k = __builtin_rint(x * kLog2e);
  double r = fma(-k, kLn2Hi, x);
  r = fma(-k, kLn2Lo, r);
  double p = 2.7557319223985893e-06;  // 1/9!
  p = fma(p, r, 2.48015873015873e-05);
  p = fma(p, r, 0.0001984126984126984);
  p = fma(p, r, 0.001388888888888889);
  p = fma(p, r, 0.008333333333333333);
  p = fma(p, r, 0.041666666666666664);
  p = fma(p, r, 0.16666666666666666);
  p = fma(p, r, 0.5);
  p = fma(p, r, 1.0);
  p = fma(p, r, 1.0);
  return __builtin_ldexp(p, static_cast<int>(k));
}

// 2^x in float64 for |x| <= 1100 (the caller bounds x).  x = k + f with k the
// nearest integer and |f| <= 1/2; 2^f is the polynomial of degree kDegree that
// interpolates 2^f at the kDegree + 1 Chebyshev nodes of [-1/2, 1/2] (relative
// error below 6e-11 over the interval for degree 7, below 2.6e-9 for degree
// 6); the result is scaled by 2^k.  k is formed by adding 1.5 * 2^52, which
// leaves the nearest integer to x in the low word of the sum (no
// float-to-integer conversion; NaN gives NaN).
template <int kDegree = 7>
__device__ __forceinline__ double exp2_f64_bounded(double x) {
  static_assert(kDegree == 6 || kDegree == 7, "degree 6 or 7");
  constexpr double kRound = 6755399441055744.0;  // 1.5 * 2^52
  const double t = x + kRound;
  const int k = static_cast<int>(static_cast<unsigned>(__double_as_longlong(t) & 0xffffffffu));
  const double f = x - (t - kRound);
  double p;
  if constexpr (kDegree == 7) {
    p = 1.5303701161442145e-05;
    p = fma(p, f, 1.5469729221575116e-04);
    p = fma(p, f, 1.3333478471058548e-03);
    p = fma(p, f, 9.6180256132689674e-03);
    p = fma(p, f, 5.5504109063307244e-02);
    p = fma(p, f, 2.4022651213498578e-01);
    p = fma(p, f, 6.9314718055682956e-01);
    p = fma(p, f, 9.9999999995956212e-01);
  } else {
    p = 1.5461444698569130e-04;
    p = fma(p, f, 1.3400428177615838e-03);
    p = fma(p, f, 9.6180566785246370e-03);
    p = fma(p, f, 5.5503272266703020e-02);
    p = fma(p, f, 2.4022650922288757e-01);
    p = fma(p, f, 6.9314720670283260e-01);
    p = fma(p, f, 1.0);
  }
  return __builtin_ldexp(p, k);
}

// 2^x in float64 for any x: arguments are held to [-1100, 1100], beyond which
// 2^x has underflowed to 0 or overflowed to +inf; the comparisons keep NaN as
// NaN.
__device__ __forceinline__ double exp2_f64(double x) {
  x = x < -1100.0 ? -1100.0 : x;
  x = x > 1100.0 ? 1100.0 : x;
  return exp2_f64_bounded(x);
}

// 2^x for a term of an exponent sum, x <= 0 up to rounding, from the degree-6
// polynomial (a sum of such terms is within 2.6e-9 of itself, twenty times
// below a float32 rounding): arguments below -1100 (-inf included) are raised
// by the hardware maximum, one instruction, which also turns NaN into a term
// of 0.  Callers find rows with NaN logits
// from the row's maximum instead (row_max propagates NaN).
// kClamp false: for callers that know x is finite (a term of a row whose
// logits are all finite), where no clamp is needed: a finite x below -1100
// gives 2^k p(f) with k below -1100, which underflows to 0 all the same.
template <bool kClamp = true>
__device__ __forceinline__ double exp2_f64_term(double x) {
  if constexpr (kClamp) return exp2_f64_bounded<6>(__builtin_fmax(x, -1100.0));
  return exp2_f64_bounded<6>(x);
}

// log s in float64 for an exponent sum s in [1, 2^64) (a sum whose largest
// term is 1): the hardware float32 base-2 logarithm as the start, l = log2 s
// to about 1e-7, then one Newton step for f(y) = e^y - s from y0 = l ln2,
// y1 = y0 - 1 + s e^{-y0} with e^{-y0} = 2^{-l} from the degree-7 exponential:
// the step squares the start's error, so what remains is that exponential's
// relative error (below 6e-11) and a few float64 roundings.  NaN stays NaN.
__device__ __forceinline__ double log_sum_f64(double s) {
  constexpr double kLn2 = 0.6931471805599453;
  const double l = static_cast<double>(__builtin_amdgcn_logf(static_cast<float>(s)));
  const double y0 = l * kLn2;
  return fma(s, exp2_f64_bounded<7>(-l), y0 - 1.0);
}

// Workgroups are handed to the 8 XCDs round-robin; number the lane tiles so
// that neighbouring tiles (which share 128-byte lines of the [T,B] arrays) run
// on the same XCD and meet in its L2.
__device__ __forceinline__ int64_t xcd_tile(int64_t block, int64_t nblocks) {
  constexpr int64_t kXcd = 8;
  const int64_t per = nblocks / kXcd;
  if (block >= per * kXcd) return block;
  return (block % kXcd) * per + block / kXcd;
}

}  // namespace vtrace
