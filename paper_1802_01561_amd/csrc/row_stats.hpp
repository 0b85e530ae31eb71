// Per-step row statistics of the target and behaviour logits, shared by the
// tiled and time-parallel V-trace kernels.
#pragma once

#include <type_traits>

#include "device_common.hpp"
#include "wave_ops.hpp"

namespace vtrace {

// Row statistics of one step: what the rest of the step needs from the logits.
struct RowStats {
  double ratio;       // pi(a|x) / mu(a|x)
  double log_pa;      // log pi(a|x)
  double sum, inv;    // s = sum_j exp(z_j - m_z) and 1/s
  double dza;         // z_a - m_z
  float inv_s;        // 1 / sum_j exp(z_j - m_z)
  float log_s;        // log of that sum
  float H;            // entropy of pi
  float one_minus_pa; // 1 - pi(a|x), formed without cancellation
  float e_a;          // exp(z_a - m_z)
  float mz;
};

// Maximum of a row of logits, NaN if any logit is NaN (the IEEE maximum,
// v_maximum3_f32 on gfx950).
template <int A_, typename In>
__device__ __forceinline__ float row_max(const In* r) {
  float m = logit_to_float(r[0]);
#pragma unroll
  for (int j = 1; j < A_; ++j) m = __builtin_elementwise_maximum(m, logit_to_float(r[j]));
  return m;
}

// kPrecise: the exponent sums, and from them the importance ratio and
// log pi(a|x), are formed in float64 from float64 exponentials of exact
// float64 differences (relative error near 1e-10).  Two things need this.  The
// loss sums over a lane's steps (Sec. 4.2, App. D) can cancel to a few
// hundredths from a thousand terms of order one, and a float32 ratio (a few
// 1e-7 relative) then moves them by more than 1e-5; and when the weights can
// exceed 1 (lambda * c_bar > 1, or rho left unclipped above 1), products of c
// amplify errors in the ratio.  Otherwise (a targets-only call whose weights
// are all at most 1) float32 exponentials from the hardware exp2 are accurate
// enough.  Both modes write the float32 e_j = exp(z_j - m_z) to e[0..A) (the
// precise mode rounds its float64 ones) for the gradient and the entropy.
//
// A row whose maximum is not finite (a NaN or +inf logit, or every logit
// -inf) gets NaN statistics; -inf logits elsewhere are zero-probability
// actions.
//
// With behaviour log-probabilities (beh_lp) there is no behaviour row: the
// ratio is exp(log pi(a|x) - lmu), lmu = log mu(a|x) as given.  Variants that
// do not use the ratio (no_ratio) skip the behaviour row too; their ratio is 1.
constexpr double kLog2eF64 = 1.4426950408889634;
constexpr double kLn2F64 = 0.6931471805599453;

// The precise mode's statistics of a target row: everything of RowStats but the
// ratio.  e_j = 2^((z_j - m_z) log2 e), the fused multiply-add forming the
// exponent from the exact product z_j log2 e; their float32 roundings go to e.
// The precise mode reads a row once into registers (one batch of LDS reads and
// one wait) and forms its terms fully unrolled.  An empty asm statement after
// each term pins the running sums in place: otherwise the compiler sinks the
// additions below all A_ exponentials and keeps every term live, more
// registers than two waves per SIMD have.
template <int A_, typename In>
__device__ __forceinline__ float read_row_max(const In* r, float (&v)[A_]) {
#pragma unroll
  for (int j = 0; j < A_; ++j) v[j] = logit_to_float(r[j]);
  float m = v[0];
#pragma unroll
  for (int j = 1; j < A_; ++j) m = __builtin_elementwise_maximum(m, v[j]);
  return m;
}

// Whether every row of the wave is finite (its maximum m and its minimum
// both finite): then no exponent-sum term needs the clamp against -inf and
// NaN logits, and the whole wave takes the unclamped terms (A + 1 VALU
// instructions fewer per row for the A - 1 that find its minimum, fewer for
// three-operand minima).  Called by every thread of the wave.
template <int A_>
__device__ __forceinline__ bool wave_rows_finite(const float (&v)[A_], float m) {
  float mn = v[0];
#pragma unroll
  for (int j = 1; j < A_; ++j) mn = __builtin_elementwise_minimum(mn, v[j]);
  return __all(__builtin_isfinite(mn) && __builtin_isfinite(m)) != 0;
}

template <int A_, typename In>
__device__ __forceinline__ RowStats target_row_stats(const In* zr, int act_c, float* e, float* zo) {
  RowStats st;
  const float za = logit_to_float(zr[act_c]);
  float z[A_];
  const float mz = read_row_max<A_>(zr, z);
  if (zo != nullptr) {
#pragma unroll
    for (int j = 0; j < A_; ++j) zo[j] = z[j];
  }
  st.mz = mz;
  const double mzl = static_cast<double>(mz) * kLog2eF64;
  // The sums start from -0.0, the additive identity, which lets the compiler
  // drop the first addition.
  double sz = -0.0;
  double ed = -0.0;  // sum_j e_j (z_j - m_z) log2 e, for the entropy
  double ea;
  auto terms = [&](auto clamp) {
    constexpr bool kClamp = decltype(clamp)::value;
    static_for<A_>([&](auto J) {
      constexpr int j = decltype(J)::value;
      const double xj = fma(static_cast<double>(z[j]), kLog2eF64, -mzl);
      const double ej = exp2_f64_term<kClamp>(xj);
      sz += ej;
      e[j] = static_cast<float>(ej);
      ed = fma(ej, xj, ed);
      asm volatile("" : "+v"(sz), "+v"(ed));
    });
    ea = exp2_f64_term<kClamp>(fma(static_cast<double>(za), kLog2eF64, -mzl));
  };
  if (wave_rows_finite<A_>(z, mz))
    terms(std::false_type{});
  else
    terms(std::true_type{});
  if (!__builtin_isfinite(mz)) sz = NAN;
  const double dza = static_cast<double>(za) - static_cast<double>(mz);  // exact
  // 1/s from the hardware reciprocal and two Newton steps.
  double inv = __builtin_amdgcn_rcp(sz);
  inv = fma(inv, fma(-sz, inv, 1.0), inv);
  inv = fma(inv, fma(-sz, inv, 1.0), inv);
  const double log_sz = log_sum_f64(sz);
  st.log_pa = dza - log_sz;
  st.inv_s = static_cast<float>(inv);
  st.log_s = static_cast<float>(log_sz);
  st.one_minus_pa = static_cast<float>((sz - ea) * inv);
  st.e_a = static_cast<float>(ea);
  st.H = static_cast<float>(fma(-ed * kLn2F64, inv, log_sz));
  st.ratio = 0.0;
  st.sum = sz;
  st.inv = inv;
  st.dza = dza;
  return st;
}

// Sum of the behaviour row's exponentials in float64 (precise mode), NaN when
// the row's maximum is not finite; *dya receives y_a - m_y (exact).
template <int A_, typename In>
__device__ __forceinline__ double behaviour_exp_sum(const In* yr, int act_c, double* dya) {
  float y[A_];
  const float my = read_row_max<A_>(yr, y);
  const double myl = static_cast<double>(my) * kLog2eF64;
  double sy = -0.0;
  auto terms = [&](auto clamp) {
    constexpr bool kClamp = decltype(clamp)::value;
    static_for<A_>([&](auto J) {
      constexpr int j = decltype(J)::value;
      sy += exp2_f64_term<kClamp>(fma(static_cast<double>(y[j]), kLog2eF64, -myl));
      asm volatile("" : "+v"(sy));
    });
  };
  if (wave_rows_finite<A_>(y, my))
    terms(std::false_type{});
  else
    terms(std::true_type{});
  if (!__builtin_isfinite(my)) sy = NAN;
  *dya = static_cast<double>(logit_to_float(yr[act_c])) - static_cast<double>(my);
  return sy;
}

//
// zo (precise mode; may be null) receives the target row as float32, for
// callers that keep it in registers until the gradient.
template <int A_, bool kPrecise, typename In>
__device__ __forceinline__ RowStats row_stats(const In* zr, const In* yr, int act_c, bool act_ok,
                                              bool beh_lp, bool no_ratio, float lmu, float* e,
                                              float* zo = nullptr) {
  if constexpr (kPrecise) {
    RowStats st = target_row_stats<A_>(zr, act_c, e, zo);
    if (no_ratio) {
      st.ratio = act_ok ? 1.0 : NAN;
    } else if (beh_lp) {
      st.ratio = act_ok ? exp2_f64((st.log_pa - static_cast<double>(lmu)) * kLog2eF64) : NAN;
    } else {
      double dya;
      const double sy = behaviour_exp_sum<A_>(yr, act_c, &dya);
      st.ratio = act_ok ? exp2_f64((st.dza - dya) * kLog2eF64) * (sy * st.inv) : NAN;
    }
    return st;
  } else {
    RowStats st;
    const float za = logit_to_float(zr[act_c]);
    const float mz = row_max<A_>(zr);
    st.mz = mz;
    float ed = 0.f;  // sum_j e_j (z_j - m_z), for the entropy
    float sz = 0.f, sy = 0.f;
#pragma unroll
    for (int j = 0; j < A_; ++j) {
      const float d = logit_to_float(zr[j]) - mz;
      e[j] = exp_fast(d);
      sz += e[j];
      ed = fmaf(e[j], d, ed);
    }
    const float inv = __builtin_amdgcn_rcpf(sz);
    const float ea = exp_fast(za - mz);
    const float log_s = __logf(sz);
    st.log_pa = static_cast<double>(za - mz) - static_cast<double>(log_s);
    if (no_ratio) {
      st.ratio = act_ok ? 1.0 : NAN;
    } else if (beh_lp) {
      st.ratio = act_ok ? static_cast<double>(exp_fast((za - mz) - log_s - lmu)) : NAN;
    } else {
      const float ya = logit_to_float(yr[act_c]);
      const float my = row_max<A_>(yr);
#pragma unroll
      for (int j = 0; j < A_; ++j) sy += exp_fast(logit_to_float(yr[j]) - my);
      st.ratio = act_ok ? static_cast<double>(exp_fast((za - mz) - (ya - my)) * (sy * inv)) : NAN;
    }
    st.inv_s = inv;
    st.log_s = log_s;
    st.one_minus_pa = (sz - ea) * inv;
    st.e_a = ea;
    st.H = log_s - ed * inv;
    st.sum = sz;
    st.inv = inv;
    st.dza = za - mz;
    return st;
  }
}

// log(pi(a|x) + eps), the epsilon-correction's policy-gradient log-probability,
// in the precision of the row statistics.
template <bool kPrecise>
__device__ __forceinline__ double log_prob_plus_eps(const RowStats& st, float eps) {
  if constexpr (kPrecise) return log(exp(st.log_pa) + static_cast<double>(eps));
  return static_cast<double>(logf(st.e_a * st.inv_s + eps));
}

}  // namespace vtrace
