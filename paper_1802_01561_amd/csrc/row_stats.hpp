// Per-step row statistics of the target and behaviour logits, shared by the
// tiled and time-parallel V-trace kernels.
#pragma once

#include "device_common.hpp"
#include "wave_ops.hpp"

namespace vtrace {

// Row statistics of one step: what the rest of the step needs from the logits.
struct RowStats {
  double ratio;       // pi(a|x) / mu(a|x)
  float inv_s;        // 1 / sum_j exp(z_j - m_z)
  float log_s;        // log of that sum
  float H;            // entropy of pi
  float one_minus_pa; // 1 - pi(a|x), formed without cancellation
  float e_a;          // exp(z_a - m_z)
  float mz;
};

// kPrecise: the importance ratio feeds products of c over many steps (lambda *
// c_bar > 1) or is left unclipped above 1 (rho_bar > 1), so errors in it are
// amplified; the exponent sums are then formed from float64 exponentials of
// exact float64 differences.  Otherwise every weight is at most 1, nothing is
// amplified, and float32 exponentials are accurate enough.
//
// With behaviour log-probabilities (beh_lp) there is no behaviour row: the
// ratio is exp(log pi(a|x) - lmu), lmu = log mu(a|x) as given.  Variants that
// do not use the ratio (no_ratio) skip the behaviour row too; their ratio is 1.
template <int A_, bool kPrecise, typename In>
__device__ __forceinline__ RowStats row_stats(const In* zr, const In* yr, int act_c, bool act_ok,
                                              bool beh_lp, bool no_ratio, float lmu,
                                              float (&e)[A_]) {
  RowStats st;
  const float za = logit_to_float(zr[act_c]);
  float mz = logit_to_float(zr[0]);
#pragma unroll
  for (int j = 1; j < A_; ++j) mz = fmaxf(mz, logit_to_float(zr[j]));
  float ya = 0.f, my = 0.f;
  if (!beh_lp && !no_ratio) {
    ya = logit_to_float(yr[act_c]);
    my = logit_to_float(yr[0]);
#pragma unroll
    for (int j = 1; j < A_; ++j) my = fmaxf(my, logit_to_float(yr[j]));
  }
  st.mz = mz;
  float ed = 0.f;  // sum_j e_j (z_j - m_z), for the entropy
  if constexpr (kPrecise) {
    // The exponent sums decide the ratio and are formed in float64; a short
    // unroll keeps their float64 temporaries from crowding out the registers
    // the rest of the step needs.  The e_j themselves only enter the gradient
    // and the entropy, where float32 exponentials are accurate enough.
    double sz = 0.0, sy = 0.0;
#pragma unroll 3
    for (int j = 0; j < A_; ++j)
      sz += exp_nonpos_f64(static_cast<double>(logit_to_float(zr[j])) - static_cast<double>(mz));
#pragma unroll
    for (int j = 0; j < A_; ++j) {
      const float d = logit_to_float(zr[j]) - mz;
      e[j] = exp_fast(d);
      ed = fmaf(e[j], d, ed);
    }
    const double inv = 1.0 / sz;
    const double dza = static_cast<double>(za) - static_cast<double>(mz);
    const double ea = exp_nonpos_f64(dza);
    if (no_ratio) {
      st.ratio = act_ok ? 1.0 : NAN;
    } else if (beh_lp) {
      st.ratio = act_ok ? exp(dza - log(sz) - static_cast<double>(lmu)) : NAN;
    } else {
#pragma unroll 3
      for (int j = 0; j < A_; ++j)
        sy += exp_nonpos_f64(static_cast<double>(logit_to_float(yr[j])) - static_cast<double>(my));
      const double dya = static_cast<double>(ya) - static_cast<double>(my);
      st.ratio = act_ok ? exp(dza - dya) * (sy * inv) : NAN;
    }
    st.inv_s = static_cast<float>(inv);
    st.log_s = static_cast<float>(log(sz));
    st.one_minus_pa = static_cast<float>((sz - ea) * inv);
    st.e_a = static_cast<float>(ea);
  } else {
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
    if (no_ratio) {
      st.ratio = act_ok ? 1.0 : NAN;
    } else if (beh_lp) {
      st.ratio = act_ok ? static_cast<double>(exp_fast((za - mz) - log_s - lmu)) : NAN;
    } else {
#pragma unroll
      for (int j = 0; j < A_; ++j) sy += exp_fast(logit_to_float(yr[j]) - my);
      st.ratio = act_ok ? static_cast<double>(exp_fast((za - mz) - (ya - my)) * (sy * inv)) : NAN;
    }
    st.inv_s = inv;
    st.log_s = log_s;
    st.one_minus_pa = (sz - ea) * inv;
    st.e_a = ea;
  }
  st.H = st.log_s - ed * st.inv_s;
  return st;
}

}  // namespace vtrace
