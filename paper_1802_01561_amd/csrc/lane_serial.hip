// Generic V-trace kernel: one thread per lane, walking time backwards.
//
// This is the any-A path (and the reference point for the tiled kernel).  Each
// thread owns lane b and visits t = T-1 .. 0, so the reverse recursion of
// Remark 1 is a plain loop and v_{t+1} is already known when step t needs it
// for its advantage: the whole step (log-softmaxes, ratio, delta, recursion,
// advantage, gradients, loss partials) is one pass over the lane's data.  Rows
// are read straight from global memory; that is simple but not coalesced, which
// is why the common action counts use the tiled kernel instead.
#include "device_common.hpp"
#include "wave_ops.hpp"

namespace vtrace {
namespace {

constexpr int kLaneSerialThreads = 64;

template <typename In, bool kGrad>
__global__ __launch_bounds__(kLaneSerialThreads) void lane_serial_kernel(StepArgs a) {
  __shared__ double red_scratch[3 * (kLaneSerialThreads / kWave)];
  const int64_t b = static_cast<int64_t>(blockIdx.x) * kLaneSerialThreads + threadIdx.x;
  const int64_t T = a.T, B = a.B, A = a.A;
  const In* __restrict__ zlog = static_cast<const In*>(a.target_logits);
  const In* __restrict__ ylog = static_cast<const In*>(a.behaviour_logits);
  const float* __restrict__ lmu_g = static_cast<const float*>(a.behaviour_logits);
  const bool beh_lp = a.behaviour_log_probs != 0;
  const double rho_bar = a.rho_bar, c_bar = a.c_bar, lam = a.lambda;
  const float ce = a.entropy_cost;

  double acc_pg = 0.0, acc_base = 0.0, acc_ent = 0.0;
  if (b < B) {
    // Carries from step t+1: V(x_{t+1}), v_{t+1} and v_{t+1} - V(x_{t+1}).
    const double boot = a.bootstrap_value[b];
    double V_next = boot, v_next = boot, A_next = 0.0;
    for (int64_t t = T - 1; t >= 0; --t) {
      const int64_t idx = t * B + b;
      const In* zr = zlog + idx * A;
      const In* yr = ylog + idx * A;
      const int32_t act = a.actions[idx];
      const bool valid = act >= 0 && act < A;

      // Row maxima and the logits at the taken action.
      float mz = -INFINITY, my = -INFINITY, za = 0.f, ya = 0.f;
      for (int64_t j = 0; j < A; ++j) {
        const float z = logit_to_float(zr[j]);
        mz = __builtin_elementwise_maximum(mz, z);  // NaN if any logit is NaN
        if (j == act) za = z;
        if (!beh_lp) {
          const float y = logit_to_float(yr[j]);
          my = __builtin_elementwise_maximum(my, y);
          if (j == act) ya = y;
        }
      }
      // Exponent sums in float64 (e_j = 2^((l_j - m) log2 e), as the tiled
      // kernel's precise mode); also sum_j e_j (z_j - m_z) in float32, which
      // gives the entropy as H = log s - (sum_j e_j (z_j - m_z)) / s.
      constexpr double kLog2e = 1.4426950408889634;
      const double mzl = static_cast<double>(mz) * kLog2e;
      const double myl = static_cast<double>(my) * kLog2e;
      double sz = 0.0, sy = 0.0;
      float ed = 0.f;
      for (int64_t j = 0; j < A; ++j) {
        const float z = logit_to_float(zr[j]);
        sz += exp2_f64_term(fma(static_cast<double>(z), kLog2e, -mzl));
        const float dz = z - mz;
        ed += expf(dz) * dz;
        if (!beh_lp) sy += exp2_f64_term(fma(static_cast<double>(logit_to_float(yr[j])), kLog2e, -myl));
      }
      // A row whose maximum is not finite (NaN or +inf logits) gets NaN sums.
      if (!__builtin_isfinite(mz)) sz = NAN;
      if (!beh_lp && !__builtin_isfinite(my)) sy = NAN;
      const double dza = static_cast<double>(za) - static_cast<double>(mz);  // exact
      const double ea = exp2_f64_term(fma(static_cast<double>(za), kLog2e, -mzl));
      const double log_pa_d = dza - log(sz);

      // With behaviour log-probabilities the ratio is exp(log pi(a) - log mu(a)).
      const double ratio =
          !valid ? NAN
          : beh_lp ? exp2_f64((log_pa_d - static_cast<double>(lmu_g[idx])) * kLog2e)
                   : exp2_f64((dza - (static_cast<double>(ya) - static_cast<double>(my))) * kLog2e) *
                         (sy / sz);
      if (!valid) raise_error_flag(a.error_flag);
      const StepWeights w = variant_weights(a.correction, clip_above(ratio, rho_bar),
                                            lam * clip_above(ratio, c_bar), lam, valid);

      const double r = transform_reward(a.rewards[idx], a.reward_transform);
      const double g = a.discounts[idx], V = a.values[idx];
      const double delta = w.rho_v * (r + g * V_next - V);
      const double A_t = delta + g * w.c_v * A_next;  // v_t - V(x_t)
      const double v_t = V + A_t;
      const double q_next = a.q_estimate == kQBaseline ? V_next : v_next;
      const double adv = w.rho_pg * (r + g * q_next - V);

      if (a.vs) a.vs[idx] = static_cast<float>(v_t);
      if (a.pg_adv) a.pg_adv[idx] = static_cast<float>(adv);

      if constexpr (kGrad) {
        a.d_values[idx] = static_cast<float>(a.baseline_cost * (V - v_t));
        const float szf = static_cast<float>(sz);
        const float inv = 1.0f / szf;
        const float log_s = logf(szf);
        const float H = log_s - ed * inv;
        // 1 - pi(a): the other actions' mass, without cancellation.
        const float one_minus_pa = static_cast<float>((sz - ea) / sz);
        // epsilon-correction: -adv log(pi_a + eps) has gradient adv pi_a/(pi_a + eps) (pi_j - 1[j=a]).
        const float pa = static_cast<float>(ea / sz);
        const bool eps_mode = a.correction == kCorrEpsilon;
        const float pg_w = eps_mode ? pa / (pa + a.epsilon) : 1.0f;
        const float adv32 = valid ? static_cast<float>(adv) * pg_w : NAN;
        for (int64_t j = 0; j < A; ++j) {
          const float dz = logit_to_float(zr[j]) - mz;
          const float p = expf(dz) * inv;
          const float pg_term = (j == act) ? -one_minus_pa : p;
          const float d = adv32 * pg_term + ce * p * ((dz - log_s) + H);
          if (a.grad_bf16)
            static_cast<uint16_t*>(a.d_logits)[idx * A + j] = to_bf16(d);
          else
            static_cast<float*>(a.d_logits)[idx * A + j] = d;
        }
        const double log_pa = !valid ? NAN
                              : eps_mode ? log(exp(log_pa_d) + static_cast<double>(a.epsilon))
                                         : log_pa_d;
        acc_pg += -adv * log_pa;
        acc_base += 0.5 * (v_t - V) * (v_t - V);
        acc_ent += -static_cast<double>(H);
      }
      V_next = V;
      v_next = v_t;
      A_next = A_t;
    }
    if constexpr (kGrad) {
      acc_base *= a.baseline_cost;
      acc_ent *= a.entropy_cost;
      if (a.lane_losses) {
        a.lane_losses[3 * b + 0] = static_cast<float>(acc_pg);
        a.lane_losses[3 * b + 1] = static_cast<float>(acc_base);
        a.lane_losses[3 * b + 2] = static_cast<float>(acc_ent);
      }
    }
  }
  if constexpr (kGrad) finish_losses<kLaneSerialThreads>(a, acc_pg, acc_base, acc_ent, red_scratch);
}

template <typename In>
hipError_t launch_typed(const StepArgs& a, Mode mode, hipStream_t s, int64_t* nwg) {
  const int64_t blocks = (a.B + kLaneSerialThreads - 1) / kLaneSerialThreads;
  *nwg = blocks;
  if (mode == Mode::LossGrad) {
    hipLaunchKernelGGL((lane_serial_kernel<In, true>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kLaneSerialThreads), 0, s, a);
  } else {
    hipLaunchKernelGGL((lane_serial_kernel<In, false>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kLaneSerialThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lane_serial(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                              int64_t* num_workgroups) {
  if (lt == LogitsType::BF16) return launch_typed<uint16_t>(a, mode, s, num_workgroups);
  return launch_typed<float>(a, mode, s, num_workgroups);
}

}  // namespace vtrace
