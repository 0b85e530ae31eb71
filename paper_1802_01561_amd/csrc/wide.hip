// Time-parallel V-trace kernel for short unrolls (T <= 256): one thread per
// (lane, step), so a batch of B lanes runs its T steps at once instead of
// walking 16-step chunks one after another.  This is the shape of the paper's
// learner batches (B = 32 trajectories of 100 or 20 steps), where the chunk
// walk leaves the GPU idle and the call is latency-bound.
//
// A workgroup of 256 threads holds 256 / TP lanes of TP steps each, TP the
// power of two >= max(T, 16); thread (lane, t) handles step t, and the 16
// consecutive steps of one DPP row never straddle two lanes.  The reverse
// recursion v_t - V(x_t) = delta_t + gamma_t c_t (v_{t+1} - V(x_{t+1}))
// (Remark 1) is an affine map per step; it is composed in two levels:
//  1. a DPP suffix scan within each row of 16 steps (as in the tiled kernel);
//  2. the rows' composites go through LDS, where one thread per lane walks its
//     TP / 16 rows from the last and leaves each row the value at the next
//     row's first step; applying it finishes every step.
// Steps at or beyond T carry the identity-breaking map (0, 0), which makes
// v_{T-1} use V(x_T) exactly as Eq. (1) does.  Each thread reads its own logit
// rows straight from global memory: at these sizes latency, not bandwidth,
// sets the time.  The loss kernel's outputs go through LDS instead: the first
// wave reduces the losses and takes the cross-workgroup ticket while the
// other three store every output in runs of whole time rows, so that the
// wait before the ticket and the gradient stores overlap instead of adding.
#include "device_common.hpp"
#include "row_stats.hpp"
#include "wave_ops.hpp"

namespace vtrace {
namespace {

constexpr int kWideLog2 = 8;
constexpr int kWideThreads = 1 << kWideLog2;
constexpr int kRow = 16;
constexpr int kRows = kWideThreads / kRow;

// The loss reduction of the loss kernel, run by its first wave alone while the
// other waves store the outputs: each lane passes its share of the
// workgroup's three sums (added in a fixed order), and the cross-workgroup
// step is finish_losses' ticket.  This wave stores nothing but lane losses
// before its partial, so the wait for the partial's stores before the ticket
// does not also wait for the gradient stores.
__device__ void finish_losses_first_wave(const StepArgs& a, double pg, double base, double ent) {
  pg = wave_sum(pg);
  base = wave_sum(base);
  ent = wave_sum(ent);
  const bool lead = threadIdx.x == 0;
  if (gridDim.x == 1) {
    if (lead) {
      a.losses[0] = static_cast<float>(pg + base + ent);
      a.losses[1] = static_cast<float>(pg);
      a.losses[2] = static_cast<float>(base);
      a.losses[3] = static_cast<float>(ent);
    }
    return;
  }
  int last = 0;
  if (lead) {
    double* p = a.partials + 3 * static_cast<size_t>(blockIdx.x);
    __hip_atomic_store(p + 0, pg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 1, base, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 2, ent, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // the partial stores have completed
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    const unsigned prev = __hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = prev == gridDim.x - 1;
  }
  if (__shfl(last, 0, kWave) == 0) return;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0;
  for (unsigned i = threadIdx.x; i < gridDim.x; i += kWave) {
    const double* p = a.partials + 3 * static_cast<size_t>(i);
    s0 += __hip_atomic_load(p + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s1 += __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s2 += __hip_atomic_load(p + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  s0 = wave_sum(s0);
  s1 = wave_sum(s1);
  s2 = wave_sum(s2);
  if (lead) {
    a.losses[0] = static_cast<float>(s0 + s1 + s2);
    a.losses[1] = static_cast<float>(s0);
    a.losses[2] = static_cast<float>(s1);
    a.losses[3] = static_cast<float>(s2);
    __hip_atomic_store(a.ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int A_, typename In, bool kGrad, bool kPrecise>
__global__ __launch_bounds__(kWideThreads) void wide_kernel(StepArgs a, int tp_log2) {
  __shared__ double s_x[kWideThreads];    // V(x_t), then v_t, by thread
  __shared__ double s_g[kRows], s_d[kRows], s_c[kRows];
  __shared__ double s_loss[3 * kRows];
  // Loss kernel outputs by time row (position t * lanes + lane): d_logits
  // rows, then d_values, v_s and the advantages.
  __shared__ float s_out[kGrad ? kWideThreads * (A_ + 3) : 1];

  const int tp = 1 << tp_log2;
  const int tid = threadIdx.x;
  const int lane_local = tid >> tp_log2;
  const int t = tid & (tp - 1);
  const int s = tid % kRow;
  const int row = tid / kRow;
  const int rows_per_lane = tp / kRow;
  const int lanes = kWideThreads >> tp_log2;
  const int64_t T = a.T, B = a.B;
  const int64_t b = static_cast<int64_t>(blockIdx.x) * lanes + lane_local;
  const bool lane_ok = b < B;
  const bool step_ok = lane_ok && t < T;
  const int64_t idx = step_ok ? static_cast<int64_t>(t) * B + b : 0;  // element 0 stands in

  const bool beh_lp = a.behaviour_log_probs != 0;
  const bool no_ratio = a.correction == kCorrNone || a.correction == kCorrEpsilon;
  int32_t act = step_ok ? a.actions[idx] : 0;
  float r32 = step_ok ? a.rewards[idx] : 0.f;
  const float g32 = step_ok ? a.discounts[idx] : 0.f;
  const float V32 = step_ok ? a.values[idx] : 0.f;
  const float lmu = (step_ok && beh_lp && !no_ratio) ? static_cast<const float*>(a.behaviour_logits)[idx] : 0.f;
  r32 = transform_reward(r32, a.reward_transform);
  const bool act_ok = act >= 0 && act < A_;
  const int act_c = act_ok ? act : 0;
  if (step_ok && !act_ok) raise_error_flag(a.error_flag);

  const In* zr = static_cast<const In*>(a.target_logits) + idx * A_;
  const In* yr = static_cast<const In*>(a.behaviour_logits) + idx * A_;
  float e[A_];
  RowStats st = row_stats<A_, kPrecise>(zr, yr, act_c, act_ok, beh_lp, no_ratio, lmu, e);
  const double lam = a.lambda;
  const StepWeights w = variant_weights(a.correction, clip_above(st.ratio, static_cast<double>(a.rho_bar)),
                                        lam * clip_above(st.ratio, static_cast<double>(a.c_bar)), lam, act_ok);

  const double boot = lane_ok ? static_cast<double>(a.bootstrap_value[b]) : 0.0;
  const double r = r32, gm = g32, V = V32;
  const bool last = t == T - 1;
  s_x[tid] = V;
  __syncthreads();
  const double V_next = last ? boot : (t + 1 < tp ? s_x[tid + 1] : 0.0);

  // 1. Suffix scan of the affine maps within the row.
  double G = step_ok ? gm * w.c_v : 0.0;
  double D = step_ok ? w.rho_v * (r + gm * V_next - V) : 0.0;
  static_for<4>([&](auto I) {
    constexpr int off = 1 << decltype(I)::value;
    const double Gn = dpp_f64<0x100 + off>(G);
    const double Dn = dpp_f64<0x100 + off>(D);
    if (s + off < kRow) {
      D = fma(G, Dn, D);
      G = G * Gn;
    }
  });
  if (s == 0) {
    s_g[row] = G;
    s_d[row] = D;
  }
  __syncthreads();
  // 2. Carries between the rows of a lane, from its last row backwards.
  if (t == 0) {
    double carry = 0.0;  // v - V just past the lane's last thread: beyond T, zero
    for (int rr = rows_per_lane - 1; rr >= 0; --rr) {
      s_c[row + rr] = carry;
      carry = fma(s_g[row + rr], carry, s_d[row + rr]);
    }
  }
  __syncthreads();
  const double A_t = fma(G, s_c[row], D);  // v_t - V(x_t)
  const double v_t = V + A_t;
  s_x[tid] = v_t;
  __syncthreads();
  const double v_next = last ? boot : (t + 1 < tp ? s_x[tid + 1] : 0.0);
  const double q_next = a.q_estimate == kQBaseline ? V_next : v_next;
  const double adv = w.rho_pg * (r + gm * q_next - V);

  if constexpr (!kGrad) {
    if (step_ok) {
      if (a.vs) a.vs[idx] = static_cast<float>(v_t);
      if (a.pg_adv) a.pg_adv[idx] = static_cast<float>(adv);
    }
  } else {
    // d_logits_j = adv (pi_j - 1[j=a]) + ce pi_j (log pi_j + H): e_j (alpha +
    // beta z_j) off the taken action, as in the tiled kernel.
    const float ce = a.entropy_cost;
    const float K = st.mz + st.log_s - st.H;
    const float pa = st.e_a * st.inv_s;
    const bool eps_mode = a.correction == kCorrEpsilon;
    const float pg_w = eps_mode ? pa / (pa + a.epsilon) : 1.0f;
    const float adv32 = static_cast<float>(adv) * pg_w;
    const float beta = st.inv_s * ce;
    const float alpha = st.inv_s * adv32 - beta * K;
    const float za = logit_to_float(zr[act_c]);
    const float out_a = -adv32 * st.one_minus_pa + ce * pa * (za - K);
    // The outputs go to LDS in time-row order, where the workgroup's lanes of
    // one step are one contiguous run, as in memory.
    const int lanes_log2 = kWideLog2 - tp_log2;
    const int pos = (t << lanes_log2) + lane_local;
    float* const s_dl = s_out;                           // [tp * lanes][A]
    float* const s_dv = s_out + kWideThreads * A_;      // [tp * lanes]
    float* const s_vs = s_dv + kWideThreads;
    float* const s_pa = s_vs + kWideThreads;
    double l_pg = 0.0, l_base = 0.0, l_ent = 0.0;
    if (step_ok) {
      s_dv[pos] = static_cast<float>(a.baseline_cost * (V - v_t));
      s_vs[pos] = static_cast<float>(v_t);
      s_pa[pos] = static_cast<float>(adv);
      const double log_pa = !act_ok ? NAN : eps_mode ? log_prob_plus_eps<kPrecise>(st, a.epsilon) : st.log_pa;
      l_pg = -adv * log_pa;
      l_base = 0.5 * A_t * A_t;
      l_ent = -static_cast<double>(st.H);
#pragma unroll
      for (int j = 0; j < A_; ++j) {
        float x = e[j] * fmaf(beta, logit_to_float(zr[j]), alpha);
        if (j == act_c) x = act_ok ? out_a : NAN;
        s_dl[pos * A_ + j] = x;
      }
    }
    // Loss sums: per row (fixed butterfly), per lane (rows in order), then
    // over the workgroup's lanes and the batch.
#pragma unroll
    for (int off = kRow / 2; off > 0; off >>= 1) {
      l_pg += __shfl_xor(l_pg, off, kRow);
      l_base += __shfl_xor(l_base, off, kRow);
      l_ent += __shfl_xor(l_ent, off, kRow);
    }
    if (s == 0) {
      s_loss[3 * row + 0] = l_pg;
      s_loss[3 * row + 1] = l_base;
      s_loss[3 * row + 2] = l_ent;
    }
    __syncthreads();
    const int64_t b0 = static_cast<int64_t>(blockIdx.x) * lanes;
    if (tid < kWave) {
      // First wave: the loss sums, lane tid of the workgroup in thread tid.
      double pg = 0.0, base = 0.0, ent = 0.0;
      if (tid < lanes) {
        for (int rr = 0; rr < rows_per_lane; ++rr) {
          const int q = tid * rows_per_lane + rr;
          pg += s_loss[3 * q + 0];
          base += s_loss[3 * q + 1];
          ent += s_loss[3 * q + 2];
        }
        base *= a.baseline_cost;
        ent *= a.entropy_cost;
        const int64_t bl = b0 + tid;
        if (bl < B && a.lane_losses) {
          a.lane_losses[3 * bl + 0] = static_cast<float>(pg);
          a.lane_losses[3 * bl + 1] = static_cast<float>(base);
          a.lane_losses[3 * bl + 2] = static_cast<float>(ent);
        }
        if (bl >= B) pg = base = ent = 0.0;
      }
      finish_losses_first_wave(a, pg, base, ent);
    } else {
      // The other waves: coalesced stores of the outputs, time row by time row.
      constexpr int kCopy = kWideThreads - kWave;
      const int k = tid - kWave;
      const bool bf16 = a.grad_bf16 != 0;
      for (int f = k; f < kWideThreads * A_; f += kCopy) {
        const int q = f / A_;
        const int tt = q >> lanes_log2;
        const int ll = q & (lanes - 1);
        if (tt < T && b0 + ll < B) {
          const int64_t g = (static_cast<int64_t>(tt) * B + b0 + ll) * A_ + (f - q * A_);
          if (bf16)
            static_cast<uint16_t*>(a.d_logits)[g] = to_bf16(s_dl[f]);
          else
            static_cast<float*>(a.d_logits)[g] = s_dl[f];
        }
      }
      for (int q = k; q < kWideThreads; q += kCopy) {
        const int tt = q >> lanes_log2;
        const int ll = q & (lanes - 1);
        if (tt < T && b0 + ll < B) {
          const int64_t g = static_cast<int64_t>(tt) * B + b0 + ll;
          a.d_values[g] = s_dv[q];
          if (a.vs) a.vs[g] = s_vs[q];
          if (a.pg_adv) a.pg_adv[g] = s_pa[q];
        }
      }
    }
  }
}

// Loss kernels always take the float64 exponent sums (precise_row_sums).
template <int A_, typename In, bool kGrad>
void launch_wide_mode(const StepArgs& a, hipStream_t st, unsigned blocks, int tp_log2) {
  if constexpr (kGrad) {
    hipLaunchKernelGGL((wide_kernel<A_, In, true, true>), dim3(blocks), dim3(kWideThreads), 0, st, a, tp_log2);
  } else {
    if (precise_row_sums(a, false))
      hipLaunchKernelGGL((wide_kernel<A_, In, false, true>), dim3(blocks), dim3(kWideThreads), 0, st, a,
                         tp_log2);
    else
      hipLaunchKernelGGL((wide_kernel<A_, In, false, false>), dim3(blocks), dim3(kWideThreads), 0, st, a,
                         tp_log2);
  }
}

template <int A_, typename In>
hipError_t launch_wide_shape(const StepArgs& a, Mode mode, hipStream_t st, int64_t* nwg) {
  int tp_log2 = 4;
  while ((int64_t(1) << tp_log2) < a.T) ++tp_log2;
  const int64_t lanes = kWideThreads >> tp_log2;
  const int64_t blocks = (a.B + lanes - 1) / lanes;
  *nwg = blocks;
  if (mode == Mode::LossGrad)
    launch_wide_mode<A_, In, true>(a, st, static_cast<unsigned>(blocks), tp_log2);
  else
    launch_wide_mode<A_, In, false>(a, st, static_cast<unsigned>(blocks), tp_log2);
  return hipGetLastError();
}

}  // namespace

bool wide_supported(const StepArgs& a, LogitsType) {
  return (a.A == 9 || a.A == 18) && a.T <= kWideThreads && a.B <= (int64_t(1) << 31);
}

hipError_t launch_wide(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st,
                       int64_t* num_workgroups) {
  if (lt == LogitsType::F32) {
    if (a.A == 18) return launch_wide_shape<18, float>(a, mode, st, num_workgroups);
    if (a.A == 9) return launch_wide_shape<9, float>(a, mode, st, num_workgroups);
  } else {
    if (a.A == 18) return launch_wide_shape<18, uint16_t>(a, mode, st, num_workgroups);
    if (a.A == 9) return launch_wide_shape<9, uint16_t>(a, mode, st, num_workgroups);
  }
  return hipErrorNotSupported;
}

}  // namespace vtrace
