// Host-side declarations shared by the C ABI and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace vtrace {

// Everything one V-trace launch needs, passed by value to the kernels.
struct StepArgs {
  int64_t T, B, A;
  const void* target_logits;     // [T,B,A] f32 or bf16
  const void* behaviour_logits;  // [T,B,A]
  const int32_t* actions;        // [T,B]
  const float* rewards;          // [T,B]
  const float* discounts;        // [T,B]
  const float* values;           // [T,B]
  const float* bootstrap_value;  // [B]
  float rho_bar, c_bar, lambda;
  float baseline_cost, entropy_cost;
  // Correction variant (0 = V-trace, 1 = none, 2 = epsilon, 3 = one-step IS),
  // Q estimate (0: r + gamma v_{s+1}, 1: r + gamma V(x_{s+1})) and epsilon.
  int correction, q_estimate;
  float epsilon;
  // 1: behaviour_logits holds [T,B] float32 log mu(a_t|x_t) instead of logits.
  int behaviour_log_probs;
  // Reward preprocessing: 0 none, 1 clip to [-1, 1], 2 optimistic asymmetric.
  int reward_transform;
  // 1: d_logits is written as bfloat16.
  int grad_bf16;
  // outputs (any may be null except where a kernel variant requires them)
  float* losses;       // [4]
  void* d_logits;      // [T,B,A] float32 or bfloat16
  float* d_values;     // [T,B]
  float* vs;           // [T,B]
  float* pg_adv;       // [T,B]
  float* lane_losses;  // [B,3]
  // workspace pieces (null when no workspace was given)
  unsigned int* ticket;
  unsigned int* error_flag;
  double* partials;  // [num_workgroups, 3]
};

// Workspace layout: a 256-byte header (completion counter, error flag) and then
// three float64 partial sums per workgroup.
constexpr size_t kWsHeaderBytes = 256;
constexpr size_t kWsTicketOffset = 0;
constexpr size_t kWsFlagOffset = 4;
// Every loss kernel covers at least this many lanes per workgroup, so the
// partials array is sized by ceil(B / kMinLanesPerWorkgroup).  (The
// time-parallel kernel holds a single lane per workgroup for T > 128.)
constexpr int64_t kMinLanesPerWorkgroup = 1;

enum class LogitsType { F32, BF16 };
enum class Mode { Targets, LossGrad };

// Kernel launchers.  They return the HIP status of the launch.
hipError_t launch_lane_serial(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                              int64_t* num_workgroups);
bool tiled_supported(const StepArgs& a, LogitsType lt);
// The tiled kernel covers 2 <= A <= kTiledMaxActions (beyond, its per-thread
// prefetch no longer fits the registers of two waves per SIMD).  allow_multi
// false keeps one workgroup per tile (no multi-tile walk).
constexpr int64_t kTiledMaxActions = 20;
// allow_long false keeps the 16-step tiles of 16 or 32 lanes (no long-run
// tile shapes).
hipError_t launch_tiled(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                        int64_t* num_workgroups, bool allow_multi, bool allow_long);
// Long-run tile shapes for A = 9 and A = 18 (targets-only calls in the float32
// ratio mode; loss calls by a rule of their own): true (with the launch
// status in *err) when one applies and was launched.
bool launch_tiled_long_f32(const StepArgs& a, Mode mode, hipStream_t s, int64_t* num_workgroups,
                           bool allow_multi, hipError_t* err);
bool launch_tiled_long_bf16(const StepArgs& a, Mode mode, hipStream_t s, int64_t* num_workgroups,
                            bool allow_multi, hipError_t* err);
hipError_t launch_tiled_a2_8(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                             int64_t* num_workgroups, bool allow_multi);
hipError_t launch_tiled_a10_14(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                               int64_t* num_workgroups, bool allow_multi);
hipError_t launch_tiled_a15_20(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                               int64_t* num_workgroups, bool allow_multi);
bool wide_supported(const StepArgs& a, LogitsType lt);
hipError_t launch_wide(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s,
                       int64_t* num_workgroups);
hipError_t launch_gather(int64_t T, int64_t B, int64_t A, LogitsType lt, const void* target,
                         const void* behaviour, const int32_t* actions, void* gathered,
                         hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);

}  // namespace vtrace
