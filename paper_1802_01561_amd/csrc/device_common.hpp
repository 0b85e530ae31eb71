// Device helpers shared by the V-trace kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "launch.hpp"

namespace vtrace {

constexpr int kWave = 64;

__device__ __forceinline__ float logit_to_float(float x) { return x; }
__device__ __forceinline__ float logit_to_float(uint16_t bits) {
  return __uint_as_float(static_cast<uint32_t>(bits) << 16);
}

// min(bar, x) as in the truncated weights of Sec. 4.1, written so that a NaN
// ratio stays NaN (fmin would return `bar`).  min(+inf, x) = x.
__device__ __forceinline__ double clip_above(double x, double bar) { return x > bar ? bar : x; }

// Pointers into global memory.  An access through a generic pointer is a flat
// instruction, which the hardware also counts as an LDS operation, so every
// wait for an LDS read would wait for the loads in flight as well.
template <typename T>
using gptr = __attribute__((address_space(1))) T*;

// p + n elements (or bytes) for an n that may put the result before the array:
// a chunk's row 0 lies before t = 0 in a lane's last chunk, where only rows
// from t = 0 on are accessed.  Integer arithmetic, so that no out-of-range
// pointer is formed; the result is a global pointer (see gptr).
template <typename T>
__device__ __forceinline__ gptr<T> offset_elems(T* p, int64_t n) {
  return (gptr<T>)(reinterpret_cast<T*>(reinterpret_cast<uintptr_t>(p) +
                                        static_cast<uintptr_t>(n * int64_t(sizeof(T)))));
}
__device__ __forceinline__ gptr<const char> offset_bytes(const void* p, int64_t bytes) {
  return (gptr<const char>)(reinterpret_cast<const char*>(reinterpret_cast<uintptr_t>(p) +
                                                          static_cast<uintptr_t>(bytes)));
}
__device__ __forceinline__ gptr<char> offset_bytes(void* p, int64_t bytes) {
  return (gptr<char>)(reinterpret_cast<char*>(reinterpret_cast<uintptr_t>(p) + static_cast<uintptr_t>(bytes)));
}

// Correction variants of Sec. 5.2.3 (values of StepArgs::correction).
constexpr int kCorrVtrace = 0, kCorrNone = 1, kCorrEpsilon = 2, kCorrOneStepIs = 3;
constexpr int kQBaseline = 1;  // StepArgs::q_estimate: q_s = r_s + gamma_s V(x_{s+1})

// Which ratio mode a call takes (the same rule for every kernel; Args is
// StepArgs or HeadArgs).  float32 ratios suffice unless V-trace's weights can
// exceed 1: products of c can then grow and amplify rounding (lambda c_bar > 1),
// or rho is left unclipped above 1.  The other variants use the ratio, if at
// all, only as one factor of one step's advantage.
template <typename Args>
inline bool ratio_needs_fp64(const Args& a) {
  return a.correction == kCorrVtrace && !(a.rho_bar <= 1.0f && a.lambda * a.c_bar <= 1.0f);
}

// Which row statistics a plain V-trace call takes: the float64 exponent sums
// (precise mode) whenever it forms loss sums, whose terms over a lane's steps
// can cancel (Sec. 4.2, App. D: losses summed over batch and time) so that a
// float32 ratio's rounding moves them by more than the outputs' tolerance, and
// whenever the weights can amplify ratio errors (ratio_needs_fp64).  Only a
// targets-only call with every weight at most 1 takes the float32 mode.
inline bool precise_row_sums(const StepArgs& a, bool losses) { return losses || ratio_needs_fp64(a); }

// A call with none of the variants but possibly a reward transform and
// bfloat16 gradients: V-trace, behaviour logits, q_s from v_{s+1}.
inline bool is_plain_vtrace_any_rewards(const StepArgs& a) {
  return a.correction == kCorrVtrace && a.q_estimate == 0 && a.behaviour_log_probs == 0;
}

// The same with behaviour log-probabilities instead of behaviour logits.
inline bool is_plain_vtrace_log_probs(const StepArgs& a) {
  return a.correction == kCorrVtrace && a.q_estimate == 0 && a.behaviour_log_probs != 0;
}

// A call with none of the variants: the above with rewards as given and
// float32 gradients.
inline bool is_plain_vtrace(const StepArgs& a) {
  return is_plain_vtrace_any_rewards(a) && a.reward_transform == 0 && a.grad_bf16 == 0;
}

// The weights a step contributes under a correction variant: rho and c in the
// value target, and the weight on the advantage.  V-trace uses the truncated
// rho_t and c_t everywhere; the uncorrected variants use rho = 1 and c = lambda
// in the target, and one-step importance sampling weights the advantage by
// rho_t.  A step with an invalid action gets NaN weights in every variant.
struct StepWeights {
  double rho_v, c_v, rho_pg;
};
__device__ __forceinline__ StepWeights variant_weights(int correction, double rho, double c,
                                                       double lam, bool act_ok) {
  StepWeights w;
  if (correction == kCorrVtrace) {
    w.rho_v = rho;
    w.c_v = c;
    w.rho_pg = rho;
  } else {
    w.rho_v = act_ok ? 1.0 : NAN;
    w.c_v = act_ok ? lam : NAN;
    w.rho_pg = correction == kCorrOneStepIs ? rho : w.rho_v;
  }
  return w;
}

// Reward preprocessing of App. D (values of StepArgs::reward_transform).  NaN
// stays NaN.
constexpr int kRewardClip = 1, kRewardAsymmetric = 2;
__device__ __forceinline__ float transform_reward(float r, int kind) {
  if (kind == kRewardClip) return r < -1.0f ? -1.0f : (r > 1.0f ? 1.0f : r);
  if (kind == kRewardAsymmetric) {
    const float t = tanhf(r);
    return t < 0.0f ? 0.3f * t : 5.0f * t;  // 0.3 min(t, 0) + 5 max(t, 0)
  }
  return r;
}

// Two floats to two bfloat16 (round to nearest even), packed low-first.
typedef float v2f_t __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ unsigned pack_bf16x2(float lo, float hi) {
  const v2f_t f = {lo, hi};
  return __builtin_bit_cast(unsigned, __builtin_convertvector(f, v2bf_t));
}
__device__ __forceinline__ uint16_t to_bf16(float x) {
  return static_cast<uint16_t>(pack_bf16x2(x, 0.0f) & 0xffffu);
}

// Butterfly sum over a wave.  Every lane ends with the same value, and the
// order of additions is fixed, so the result is reproducible bit for bit.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Sum of three per-thread values over the block, in a fixed order.  The result
// is valid in thread 0.  `scratch` holds 3 doubles per wave.
template <int kThreads>
__device__ __forceinline__ void block_sum3(double& x0, double& x1, double& x2, double* scratch) {
  x0 = wave_sum(x0);
  x1 = wave_sum(x1);
  x2 = wave_sum(x2);
  if constexpr (kThreads > kWave) {
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) {
      scratch[3 * w + 0] = x0;
      scratch[3 * w + 1] = x1;
      scratch[3 * w + 2] = x2;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      x0 = scratch[0];
      x1 = scratch[1];
      x2 = scratch[2];
      for (int i = 1; i < kThreads / kWave; ++i) {
        x0 += scratch[3 * i + 0];
        x1 += scratch[3 * i + 1];
        x2 += scratch[3 * i + 2];
      }
    }
    __syncthreads();
  }
}

// s_waitcnt immediate for vmcnt(0) alone (expcnt and lgkmcnt at their maxima).
constexpr int kWaitVmcnt0 = 0x0F70;

// Cross-workgroup loss reduction in the same launch.  Each workgroup stores its
// three partial sums, then takes a ticket; the workgroup that draws the last
// ticket adds all partials in workgroup order, writes `losses` and rearms the
// counter for the next call.  Every thread of every workgroup must call this.
//
// Ordering without fences: the partials are written and read only with
// device-scope atomic stores and loads, which the hardware performs where the
// accesses of all XCDs meet (not in one XCD's L2).  A workgroup takes its
// ticket only after its partial stores have completed (vmcnt(0)), so the
// workgroup that draws the last ticket reads every partial.  A device-scope
// fence would in addition write back and invalidate the XCD's L2 for ordinary
// accesses, which nothing here needs; in a short call those fences cost
// several microseconds.
template <int kThreads>
__device__ void finish_losses(const StepArgs& a, double pg, double base, double ent,
                              double* scratch) {
  __shared__ int s_last;
  block_sum3<kThreads>(pg, base, ent, scratch);
  if (gridDim.x == 1) {
    // One workgroup: its sums are the totals (the same values the ticket path
    // would add to zero), without the round trips through memory.
    if (threadIdx.x == 0) {
      a.losses[0] = static_cast<float>(pg + base + ent);
      a.losses[1] = static_cast<float>(pg);
      a.losses[2] = static_cast<float>(base);
      a.losses[3] = static_cast<float>(ent);
    }
    return;
  }
  if (threadIdx.x == 0) {
    double* p = a.partials + 3 * static_cast<size_t>(blockIdx.x);
    __hip_atomic_store(p + 0, pg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 1, base, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 2, ent, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);  // keep the compiler from moving them past the wait
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // the partial stores have completed
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    const unsigned prev = __hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == gridDim.x - 1);
  }
  __syncthreads();
  if (!s_last) return;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0;
  for (unsigned i = threadIdx.x; i < gridDim.x; i += kThreads) {
    const double* p = a.partials + 3 * static_cast<size_t>(i);
    s0 += __hip_atomic_load(p + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s1 += __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s2 += __hip_atomic_load(p + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  block_sum3<kThreads>(s0, s1, s2, scratch);
  if (threadIdx.x == 0) {
    a.losses[0] = static_cast<float>(s0 + s1 + s2);
    a.losses[1] = static_cast<float>(s0);
    a.losses[2] = static_cast<float>(s1);
    a.losses[3] = static_cast<float>(s2);
    __hip_atomic_store(a.ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ __forceinline__ void raise_error_flag(unsigned int* flag) {
  if (flag != nullptr) atomicOr(flag, 1u);
}

}  // namespace vtrace
