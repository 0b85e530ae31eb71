// Host-side declarations of the fused output-layer + V-trace kernel.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "launch.hpp"

namespace vtrace {

// Everything one launch of the fused output-layer kernel needs.  The layer maps
// hidden[t, b, :] to o = hidden @ weight + bias: A policy logits, then the
// baseline.
struct HeadArgs {
  int64_t T, B, A, H;
  const uint16_t* hidden;        // [T,B,H] bfloat16
  const uint16_t* weight;        // [H,A+1] bfloat16
  const float* bias;             // [A+1]
  const void* behaviour;         // [T,B,A] logits (float32 or bfloat16) or [T,B] float32 log mu
  const int32_t* actions;        // [T,B]
  const float* rewards;          // [T,B]
  const float* discounts;        // [T,B]
  const float* bootstrap_value;  // [B]
  float rho_bar, c_bar, lambda;
  float baseline_cost, entropy_cost;
  int correction, q_estimate;
  float epsilon;
  int behaviour_log_probs;
  int behaviour_bf16;  // behaviour logits are bfloat16
  int reward_transform;
  int grad_bf16;       // d_hidden is written as bfloat16
  // outputs
  float* losses;       // [4]
  void* d_hidden;      // [T,B,H]
  float* d_weight;     // [H,A+1]
  float* d_bias;       // [A+1]
  float* vs;           // [T,B] or null
  float* pg_adv;       // [T,B] or null
  float* lane_losses;  // [B,3] or null
  float* outputs;      // [T,B,A+1] or null: the layer's outputs
  // workspace pieces
  unsigned int* error_flag;
  double* loss_partials;  // [workgroups, 3]
  float* grad_partials;   // [workgroups, H+1, C]: d_weight rows, then d_bias
};

// The fused output-layer kernel runs at most this many workgroups (two per CU
// of a 256-CU part); each loops over groups of four lanes.
constexpr int64_t kHeadMaxWorkgroups = 512;
// Hidden sizes with a kernel instance, and the largest A (A + 1 output columns
// fill at most two 16-column MFMA tiles).
constexpr int64_t kHeadMaxActions = 31;
// The kernel addresses a chunk's 16 time rows of one array through one buffer
// descriptor with 32-bit offsets: 16 rows of B*H float32 must stay below
// 0xFFFFF000 bytes, so B*H is at most this.
constexpr int64_t kHeadMaxBatchTimesHidden = 0xFFFFF000LL / 64;
bool head_hidden_supported(int64_t H);
int64_t head_workgroups(int64_t B);
// Workspace of the fused kernel: the 256-byte header, then float64 loss
// partials and float32 gradient partials per workgroup.
size_t head_workspace_bytes(int64_t B, int64_t A, int64_t H);
void head_attach_workspace(HeadArgs* a, void* ws);
hipError_t launch_head(const HeadArgs& a, hipStream_t s);

}  // namespace vtrace
