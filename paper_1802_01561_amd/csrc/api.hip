// C ABI of libvtrace: argument validation, kernel choice and launch.
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "vtrace.h"
#include "head.hpp"
#include "launch.hpp"

namespace {

using vtrace::LogitsType;
using vtrace::Mode;
using vtrace::StepArgs;

constexpr int kAbiVersion = 1;
constexpr int64_t kMaxElements = int64_t(1) << 40;

bool shape_ok(int64_t T, int64_t B, int64_t A) {
  if (T < 1 || B < 1 || A < 1) return false;
  if (T > kMaxElements || B > kMaxElements || A > kMaxElements) return false;
  const __int128 n = static_cast<__int128>(T) * B * A;
  return n <= kMaxElements;
}

bool aligned(const void* p, uintptr_t k) { return (reinterpret_cast<uintptr_t>(p) % k) == 0; }

bool truncation_ok(float x) { return !std::isnan(x) && x >= 0.0f; }

hipStream_t as_hip(vtrace_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

bool dtype_of(vtrace_dtype d, LogitsType* lt) {
  if (d == VTRACE_F32) {
    *lt = LogitsType::F32;
    return true;
  }
  if (d == VTRACE_BF16) {
    *lt = LogitsType::BF16;
    return true;
  }
  return false;
}

// Kernel choice: the time-parallel kernel for short unrolls of small batches,
// the tiled kernel where it applies, else the generic one.  VTRACE_KERNEL
// (lane_serial, tiled, tiled_single, tiled_short, tiled_short_single or wide)
// forces a kernel where it applies, to cross-check them: tiled_single is the
// tiled kernel with one workgroup per tile, never the multi-tile walk;
// tiled_short keeps its 16-step tiles, never the long-run tile shapes;
// tiled_short_single both.
enum class Kernel { Auto, LaneSerial, Tiled, TiledSingle, TiledShort, TiledShortSingle, Wide };
Kernel forced_kernel() {
  const char* k = std::getenv("VTRACE_KERNEL");
  if (k == nullptr) return Kernel::Auto;
  if (std::strcmp(k, "lane_serial") == 0) return Kernel::LaneSerial;
  if (std::strcmp(k, "tiled") == 0) return Kernel::Tiled;
  if (std::strcmp(k, "tiled_single") == 0) return Kernel::TiledSingle;
  if (std::strcmp(k, "tiled_short") == 0) return Kernel::TiledShort;
  if (std::strcmp(k, "tiled_short_single") == 0) return Kernel::TiledShortSingle;
  if (std::strcmp(k, "wide") == 0) return Kernel::Wide;
  return Kernel::Auto;
}

// Where both apply, the time-parallel kernel wins while the tiled kernel's
// serial walk over T / 16 chunks costs more than the time-parallel kernel's
// uncoalesced row reads.  Measured on MI355X (cold, A = 9 and 18, T from 16
// to 256, B from 8 to 2048, fp32 logits): batches of fewer than 16 lanes (less
// than one lane tile) at every T; loss calls of more than one chunk and
// targets-only calls of more than two, with B <= 512, or with B <= 1024 and
// T <= 128 (for loss calls only with A = 18).  The DMLab- and Atari-shaped
// batches (B = 32, T = 100 and 20) take it.
bool prefer_wide(const StepArgs& a, Mode mode) {
  if (a.B < 16) return true;
  const bool loss = mode == Mode::LossGrad;
  if (a.T <= (loss ? 16 : 32)) return false;
  return a.B <= 512 || (a.B <= 1024 && a.T <= 128 && (!loss || a.A >= 18));
}

size_t workspace_bytes_for(int64_t B) {
  const int64_t max_wg = (B + vtrace::kMinLanesPerWorkgroup - 1) / vtrace::kMinLanesPerWorkgroup;
  return vtrace::kWsHeaderBytes + 3 * sizeof(double) * static_cast<size_t>(max_wg);
}

vtrace_status check_common(int64_t T, int64_t B, int64_t A, vtrace_dtype dt, const void* tl,
                           const void* bl, const int32_t* act, const float* r, const float* d,
                           const float* v, const float* boot, float rho_bar, float c_bar,
                           float lambda, LogitsType* lt) {
  if (!tl || !bl || !act || !r || !d || !v || !boot) return VTRACE_ERR_NULL;
  if (!shape_ok(T, B, A)) return VTRACE_ERR_SHAPE;
  if (!dtype_of(dt, lt)) return VTRACE_ERR_DTYPE;
  if (!truncation_ok(rho_bar) || !truncation_ok(c_bar)) return VTRACE_ERR_PARAM;
  if (std::isnan(lambda) || lambda < 0.0f || lambda > 1.0f) return VTRACE_ERR_PARAM;
  if (!aligned(tl, 16) || !aligned(bl, 4)) return VTRACE_ERR_ALIGN;
  if (!aligned(act, 4) || !aligned(r, 4) || !aligned(d, 4) || !aligned(v, 4) || !aligned(boot, 4))
    return VTRACE_ERR_ALIGN;
  return VTRACE_OK;
}

StepArgs make_args(int64_t T, int64_t B, int64_t A, const void* tl, const void* bl,
                   const int32_t* act, const float* r, const float* d, const float* v,
                   const float* boot, float rho_bar, float c_bar, float lambda) {
  StepArgs a;
  std::memset(&a, 0, sizeof(a));
  a.T = T;
  a.B = B;
  a.A = A;
  a.target_logits = tl;
  a.behaviour_logits = bl;
  a.actions = act;
  a.rewards = r;
  a.discounts = d;
  a.values = v;
  a.bootstrap_value = boot;
  a.rho_bar = rho_bar;
  a.c_bar = c_bar;
  a.lambda = lambda;
  return a;
}

void attach_workspace(StepArgs* a, void* ws) {
  char* base = static_cast<char*>(ws);
  a->ticket = reinterpret_cast<unsigned int*>(base + vtrace::kWsTicketOffset);
  a->error_flag = reinterpret_cast<unsigned int*>(base + vtrace::kWsFlagOffset);
  a->partials = reinterpret_cast<double*>(base + vtrace::kWsHeaderBytes);
}

// A caller's variant, checked (NULL = V-trace with float32 gradients).
struct Variant {
  int correction = VTRACE_CORRECTION_VTRACE;
  int q_estimate = VTRACE_Q_VTRACE;
  float epsilon = 0.0f;
  int behaviour_log_probs = 0;
  int reward_transform = VTRACE_REWARD_RAW;
  int grad_bf16 = 0;
};

vtrace_status parse_variant(const vtrace_variant* v, Variant* out) {
  *out = Variant{};
  if (v == nullptr) return VTRACE_OK;
  if (v->correction < VTRACE_CORRECTION_VTRACE || v->correction > VTRACE_CORRECTION_ONE_STEP_IS)
    return VTRACE_ERR_PARAM;
  if (v->q_estimate != VTRACE_Q_VTRACE && v->q_estimate != VTRACE_Q_BASELINE) return VTRACE_ERR_PARAM;
  if (v->correction == VTRACE_CORRECTION_EPSILON && !(std::isfinite(v->epsilon) && v->epsilon > 0.0f))
    return VTRACE_ERR_PARAM;
  if (v->behaviour_input != VTRACE_BEHAVIOUR_LOGITS && v->behaviour_input != VTRACE_BEHAVIOUR_LOG_PROBS)
    return VTRACE_ERR_PARAM;
  if (v->reward_transform < VTRACE_REWARD_RAW || v->reward_transform > VTRACE_REWARD_ASYMMETRIC)
    return VTRACE_ERR_PARAM;
  if (v->grad_dtype != VTRACE_F32 && v->grad_dtype != VTRACE_BF16) return VTRACE_ERR_DTYPE;
  out->correction = v->correction;
  out->q_estimate = v->q_estimate;
  out->epsilon = v->epsilon;
  out->behaviour_log_probs = v->behaviour_input == VTRACE_BEHAVIOUR_LOG_PROBS;
  out->reward_transform = v->reward_transform;
  out->grad_bf16 = v->grad_dtype == VTRACE_BF16;
  return VTRACE_OK;
}

// Copies a caller's variant into the launch arguments.
vtrace_status apply_variant(const vtrace_variant* v, StepArgs* a) {
  Variant f;
  const vtrace_status st = parse_variant(v, &f);
  if (st != VTRACE_OK) return st;
  // Logit rows are read with 16-byte vectors; log-probabilities are plain floats.
  if (!f.behaviour_log_probs && !aligned(a->behaviour_logits, 16)) return VTRACE_ERR_ALIGN;
  a->correction = f.correction;
  a->q_estimate = f.q_estimate;
  a->epsilon = f.epsilon;
  a->behaviour_log_probs = f.behaviour_log_probs;
  a->reward_transform = f.reward_transform;
  a->grad_bf16 = f.grad_bf16;
  return VTRACE_OK;
}

bool head_shape_ok(int64_t T, int64_t B, int64_t A, int64_t H) {
  return A >= 1 && A <= vtrace::kHeadMaxActions && vtrace::head_hidden_supported(H) &&
         B <= vtrace::kHeadMaxBatchTimesHidden / H && shape_ok(T, B, H) &&
         shape_ok(T, B, A + 1);
}

vtrace_status launch(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t s) {
  (void)hipGetLastError();  // do not report an earlier, unrelated error
  int64_t nwg = 0;
  hipError_t e;
  const Kernel k = forced_kernel();
  const bool wide = vtrace::wide_supported(a, lt);
  const bool tiled = vtrace::tiled_supported(a, lt);
  if (k == Kernel::LaneSerial)
    e = vtrace::launch_lane_serial(a, lt, mode, s, &nwg);
  else if (wide && (k == Kernel::Wide || (k == Kernel::Auto && prefer_wide(a, mode))))
    e = vtrace::launch_wide(a, lt, mode, s, &nwg);
  else if (tiled)
    e = vtrace::launch_tiled(a, lt, mode, s, &nwg, k != Kernel::TiledSingle && k != Kernel::TiledShortSingle,
                             k != Kernel::TiledShort && k != Kernel::TiledShortSingle);
  else
    e = vtrace::launch_lane_serial(a, lt, mode, s, &nwg);
  return e == hipSuccess ? VTRACE_OK : VTRACE_ERR_HIP;
}

// Validation and launch arguments of a loss call, except the workspace and
// the variant.
vtrace_status loss_grad_args(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype, const void* target_logits,
                             const void* behaviour_logits, const int32_t* actions, const float* rewards,
                             const float* discounts, const float* values, const float* bootstrap_value,
                             float rho_bar, float c_bar, float lambda, float baseline_cost, float entropy_cost,
                             float* losses, void* d_logits, float* d_values, float* vs, float* pg_advantages,
                             float* lane_losses, StepArgs* a, LogitsType* lt) {
  LogitsType lt_local;
  vtrace_status st = check_common(T, B, A, logits_dtype, target_logits, behaviour_logits, actions, rewards,
                                  discounts, values, bootstrap_value, rho_bar, c_bar, lambda, &lt_local);
  if (st != VTRACE_OK) return st;
  if (!std::isfinite(baseline_cost) || !std::isfinite(entropy_cost)) return VTRACE_ERR_PARAM;
  if (!losses || !d_logits || !d_values) return VTRACE_ERR_NULL;
  if (!aligned(d_logits, 16)) return VTRACE_ERR_ALIGN;
  if (!aligned(losses, 4) || !aligned(d_values, 4) || !aligned(vs, 4) || !aligned(pg_advantages, 4) ||
      !aligned(lane_losses, 4))
    return VTRACE_ERR_ALIGN;
  StepArgs args = make_args(T, B, A, target_logits, behaviour_logits, actions, rewards, discounts, values,
                            bootstrap_value, rho_bar, c_bar, lambda);
  args.baseline_cost = baseline_cost;
  args.entropy_cost = entropy_cost;
  args.losses = losses;
  args.d_logits = d_logits;
  args.d_values = d_values;
  args.vs = vs;
  args.pg_adv = pg_advantages;
  args.lane_losses = lane_losses;
  *a = args;
  *lt = lt_local;
  return VTRACE_OK;
}

// The workspace of vtrace_loss_grad_static: a device array of fixed size,
// allocated with the library's code object (each device that runs the library
// holds its own copy until the process ends), so that the call itself
// allocates nothing.  Layout as a caller's workspace: the 256-byte header
// (completion counter, error flag) and three float64 partials per workgroup,
// at most one workgroup per lane.
constexpr size_t kStaticWorkspaceBytes =
    vtrace::kWsHeaderBytes + 3 * sizeof(double) * static_cast<size_t>(VTRACE_STATIC_MAX_LANES);
static_assert(kStaticWorkspaceBytes == VTRACE_STATIC_WORKSPACE_BYTES, "header states the array's size");
static __device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

// In host code `scratch` names a host-side stand-in, not the device array: the
// array's address on a device is asked of the runtime once per device, with
// that device current, and only that address is ever handed to kernels.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_address[kMaxDevices];

// This device's address of `scratch`.  The first call on a device asks for it
// and clears the array's header with the fill kernel on `s` (the completion
// counter must start at zero; every loss launch leaves it at zero again).
vtrace_status static_workspace(hipStream_t s, void** ws) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return VTRACE_ERR_HIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_address[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return VTRACE_ERR_HIP;
    }
    (void)hipGetLastError();
    if (vtrace::launch_fill_zero(p, vtrace::kWsHeaderBytes, s) != hipSuccess) return VTRACE_ERR_HIP;
    g_scratch_address[dev] = p;
  }
  *ws = g_scratch_address[dev];
  return VTRACE_OK;
}

}  // namespace

extern "C" {

int vtrace_abi_version(void) { return kAbiVersion; }

const char* vtrace_status_string(int32_t status) {
  switch (status) {
    case VTRACE_OK: return "ok";
    case VTRACE_ERR_NULL: return "a required pointer is NULL";
    case VTRACE_ERR_SHAPE:
      return "T, B and A must be >= 1 and T*B*A within vtrace_max_elements(); the fused output "
             "layer also needs A <= 31 and H in {64, 128, 256}";
    case VTRACE_ERR_DTYPE: return "unknown logits dtype";
    case VTRACE_ERR_PARAM:
      return "bad parameter: rho_bar, c_bar must be >= 0 (inf allowed), lambda in [0,1], "
             "costs finite, none NaN; a variant needs a known correction and Q estimate and, "
             "for epsilon-correction, a finite epsilon > 0";
    case VTRACE_ERR_ALIGN:
      return "misaligned pointer: logits/d_logits/gathered/hidden/d_hidden need 16 bytes, "
             "others their element size";
    case VTRACE_ERR_WORKSPACE: return "workspace missing or smaller than vtrace_workspace_bytes()";
    case VTRACE_ERR_HIP: return "the HIP runtime rejected the kernel launch";
  }
  return "unknown status";
}

int64_t vtrace_max_elements(void) { return kMaxElements; }

size_t vtrace_workspace_bytes(int64_t T, int64_t B, int64_t A) {
  if (!shape_ok(T, B, A)) return 0;
  return workspace_bytes_for(B);
}

vtrace_status vtrace_workspace_init(void* workspace, size_t workspace_bytes, vtrace_stream_t stream) {
  if (!workspace) return VTRACE_ERR_NULL;
  if (!aligned(workspace, 16)) return VTRACE_ERR_ALIGN;
  if (workspace_bytes < vtrace::kWsHeaderBytes) return VTRACE_ERR_WORKSPACE;
  (void)hipGetLastError();
  return vtrace::launch_fill_zero(workspace, workspace_bytes, as_hip(stream)) == hipSuccess
             ? VTRACE_OK
             : VTRACE_ERR_HIP;
}

vtrace_status vtrace_targets(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
                             const void* target_logits, const void* behaviour_logits,
                             const int32_t* actions, const float* rewards, const float* discounts,
                             const float* values, const float* bootstrap_value, float rho_bar,
                             float c_bar, float lambda, float* vs, float* pg_advantages,
                             void* workspace, size_t workspace_bytes, vtrace_stream_t stream) {
  return vtrace_targets_ex(T, B, A, logits_dtype, target_logits, behaviour_logits, actions,
                           rewards, discounts, values, bootstrap_value, rho_bar, c_bar, lambda,
                           nullptr, vs, pg_advantages, workspace, workspace_bytes, stream);
}

vtrace_status vtrace_targets_ex(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
                                const void* target_logits, const void* behaviour_logits,
                                const int32_t* actions, const float* rewards,
                                const float* discounts, const float* values,
                                const float* bootstrap_value, float rho_bar, float c_bar,
                                float lambda, const vtrace_variant* variant, float* vs,
                                float* pg_advantages, void* workspace, size_t workspace_bytes,
                                vtrace_stream_t stream) {
  LogitsType lt;
  vtrace_status st = check_common(T, B, A, logits_dtype, target_logits, behaviour_logits, actions,
                                  rewards, discounts, values, bootstrap_value, rho_bar, c_bar,
                                  lambda, &lt);
  if (st != VTRACE_OK) return st;
  if (!vs || !pg_advantages) return VTRACE_ERR_NULL;
  if (!aligned(vs, 4) || !aligned(pg_advantages, 4)) return VTRACE_ERR_ALIGN;
  StepArgs a = make_args(T, B, A, target_logits, behaviour_logits, actions, rewards, discounts,
                         values, bootstrap_value, rho_bar, c_bar, lambda);
  a.vs = vs;
  a.pg_adv = pg_advantages;
  st = apply_variant(variant, &a);
  if (st != VTRACE_OK) return st;
  if (workspace) {
    if (!aligned(workspace, 16)) return VTRACE_ERR_ALIGN;
    if (workspace_bytes < vtrace::kWsHeaderBytes) return VTRACE_ERR_WORKSPACE;
    attach_workspace(&a, workspace);
    a.partials = nullptr;
    a.ticket = nullptr;
  }
  return launch(a, lt, Mode::Targets, as_hip(stream));
}

vtrace_status vtrace_loss_grad(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
                               const void* target_logits, const void* behaviour_logits,
                               const int32_t* actions, const float* rewards,
                               const float* discounts, const float* values,
                               const float* bootstrap_value, float rho_bar, float c_bar,
                               float lambda, float baseline_cost, float entropy_cost,
                               float* losses, float* d_logits, float* d_values, float* vs,
                               float* pg_advantages, float* lane_losses, void* workspace,
                               size_t workspace_bytes, vtrace_stream_t stream) {
  return vtrace_loss_grad_ex(T, B, A, logits_dtype, target_logits, behaviour_logits, actions,
                             rewards, discounts, values, bootstrap_value, rho_bar, c_bar, lambda,
                             baseline_cost, entropy_cost, nullptr, losses, d_logits, d_values, vs,
                             pg_advantages, lane_losses, workspace, workspace_bytes, stream);
}

vtrace_status vtrace_loss_grad_ex(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
                                  const void* target_logits, const void* behaviour_logits,
                                  const int32_t* actions, const float* rewards,
                                  const float* discounts, const float* values,
                                  const float* bootstrap_value, float rho_bar, float c_bar,
                                  float lambda, float baseline_cost, float entropy_cost,
                                  const vtrace_variant* variant, float* losses, void* d_logits,
                                  float* d_values, float* vs, float* pg_advantages,
                                  float* lane_losses, void* workspace, size_t workspace_bytes,
                                  vtrace_stream_t stream) {
  StepArgs a;
  LogitsType lt;
  vtrace_status st = loss_grad_args(T, B, A, logits_dtype, target_logits, behaviour_logits, actions, rewards,
                                    discounts, values, bootstrap_value, rho_bar, c_bar, lambda, baseline_cost,
                                    entropy_cost, losses, d_logits, d_values, vs, pg_advantages, lane_losses, &a,
                                    &lt);
  if (st != VTRACE_OK) return st;
  if (!workspace) return VTRACE_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return VTRACE_ERR_ALIGN;
  if (workspace_bytes < workspace_bytes_for(B)) return VTRACE_ERR_WORKSPACE;
  st = apply_variant(variant, &a);
  if (st != VTRACE_OK) return st;
  attach_workspace(&a, workspace);
  return launch(a, lt, Mode::LossGrad, as_hip(stream));
}

vtrace_status vtrace_loss_grad_static(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
                                      const void* target_logits, const void* behaviour_logits,
                                      const int32_t* actions, const float* rewards,
                                      const float* discounts, const float* values,
                                      const float* bootstrap_value, float rho_bar, float c_bar,
                                      float lambda, float baseline_cost, float entropy_cost,
                                      const vtrace_variant* variant, float* losses, void* d_logits,
                                      float* d_values, float* vs, float* pg_advantages,
                                      float* lane_losses, vtrace_stream_t stream) {
  StepArgs a;
  LogitsType lt;
  vtrace_status st = loss_grad_args(T, B, A, logits_dtype, target_logits, behaviour_logits, actions, rewards,
                                    discounts, values, bootstrap_value, rho_bar, c_bar, lambda, baseline_cost,
                                    entropy_cost, losses, d_logits, d_values, vs, pg_advantages, lane_losses, &a,
                                    &lt);
  if (st != VTRACE_OK) return st;
  if (B > VTRACE_STATIC_MAX_LANES) return VTRACE_ERR_WORKSPACE;
  st = apply_variant(variant, &a);
  if (st != VTRACE_OK) return st;
  void* ws = nullptr;
  st = static_workspace(as_hip(stream), &ws);
  if (st != VTRACE_OK) return st;
  attach_workspace(&a, ws);
  a.error_flag = nullptr;  // nothing reads a flag in the shared array
  return launch(a, lt, Mode::LossGrad, as_hip(stream));
}

vtrace_status vtrace_gather_logits(int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
                                   const void* target_logits, const void* behaviour_logits,
                                   const int32_t* actions, void* gathered, vtrace_stream_t stream) {
  if (!target_logits || !behaviour_logits || !actions || !gathered) return VTRACE_ERR_NULL;
  if (!shape_ok(T, B, A)) return VTRACE_ERR_SHAPE;
  LogitsType lt;
  if (!dtype_of(logits_dtype, &lt)) return VTRACE_ERR_DTYPE;
  if (!aligned(target_logits, 16) || !aligned(behaviour_logits, 16) || !aligned(gathered, 16))
    return VTRACE_ERR_ALIGN;
  if (!aligned(actions, 4)) return VTRACE_ERR_ALIGN;
  (void)hipGetLastError();
  return vtrace::launch_gather(T, B, A, lt, target_logits, behaviour_logits, actions, gathered,
                               as_hip(stream)) == hipSuccess
             ? VTRACE_OK
             : VTRACE_ERR_HIP;
}

size_t vtrace_head_workspace_bytes(int64_t T, int64_t B, int64_t A, int64_t H) {
  if (!head_shape_ok(T, B, A, H)) return 0;
  return vtrace::head_workspace_bytes(B, A, H);
}

vtrace_status vtrace_head_loss_grad(
    int64_t T, int64_t B, int64_t A, int64_t H, vtrace_dtype behaviour_dtype, const void* hidden,
    const void* head_weight, const float* head_bias, const void* behaviour, const int32_t* actions,
    const float* rewards, const float* discounts, const float* bootstrap_value, float rho_bar,
    float c_bar, float lambda, float baseline_cost, float entropy_cost,
    const vtrace_variant* variant, float* losses, void* d_hidden, float* d_weight, float* d_bias,
    float* vs, float* pg_advantages, float* lane_losses, float* outputs, void* workspace,
    size_t workspace_bytes, vtrace_stream_t stream) {
  if (!hidden || !head_weight || !head_bias || !behaviour || !actions || !rewards || !discounts ||
      !bootstrap_value || !losses || !d_hidden || !d_weight || !d_bias)
    return VTRACE_ERR_NULL;
  if (!head_shape_ok(T, B, A, H)) return VTRACE_ERR_SHAPE;
  LogitsType lt;
  if (!dtype_of(behaviour_dtype, &lt)) return VTRACE_ERR_DTYPE;
  if (!truncation_ok(rho_bar) || !truncation_ok(c_bar)) return VTRACE_ERR_PARAM;
  if (std::isnan(lambda) || lambda < 0.0f || lambda > 1.0f) return VTRACE_ERR_PARAM;
  if (!std::isfinite(baseline_cost) || !std::isfinite(entropy_cost)) return VTRACE_ERR_PARAM;
  Variant f;
  vtrace_status st = parse_variant(variant, &f);
  if (st != VTRACE_OK) return st;
  const uintptr_t beh_align = (f.behaviour_log_probs || lt == LogitsType::F32) ? 4 : 2;
  if (!aligned(hidden, 16) || !aligned(d_hidden, 16) || !aligned(head_weight, 2) ||
      !aligned(behaviour, beh_align))
    return VTRACE_ERR_ALIGN;
  if (!aligned(head_bias, 4) || !aligned(actions, 4) || !aligned(rewards, 4) ||
      !aligned(discounts, 4) || !aligned(bootstrap_value, 4) || !aligned(losses, 4) ||
      !aligned(d_weight, 4) || !aligned(d_bias, 4) || !aligned(vs, 4) ||
      !aligned(pg_advantages, 4) || !aligned(lane_losses, 4) || !aligned(outputs, 4))
    return VTRACE_ERR_ALIGN;
  if (!workspace) return VTRACE_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return VTRACE_ERR_ALIGN;
  if (workspace_bytes < vtrace::head_workspace_bytes(B, A, H)) return VTRACE_ERR_WORKSPACE;

  vtrace::HeadArgs a;
  std::memset(&a, 0, sizeof(a));
  a.T = T;
  a.B = B;
  a.A = A;
  a.H = H;
  a.hidden = static_cast<const uint16_t*>(hidden);
  a.weight = static_cast<const uint16_t*>(head_weight);
  a.bias = head_bias;
  a.behaviour = behaviour;
  a.actions = actions;
  a.rewards = rewards;
  a.discounts = discounts;
  a.bootstrap_value = bootstrap_value;
  a.rho_bar = rho_bar;
  a.c_bar = c_bar;
  a.lambda = lambda;
  a.baseline_cost = baseline_cost;
  a.entropy_cost = entropy_cost;
  a.correction = f.correction;
  a.q_estimate = f.q_estimate;
  a.epsilon = f.epsilon;
  a.behaviour_log_probs = f.behaviour_log_probs;
  a.behaviour_bf16 = !f.behaviour_log_probs && lt == LogitsType::BF16;
  a.reward_transform = f.reward_transform;
  a.grad_bf16 = f.grad_bf16;
  a.losses = losses;
  a.d_hidden = d_hidden;
  a.d_weight = d_weight;
  a.d_bias = d_bias;
  a.vs = vs;
  a.pg_adv = pg_advantages;
  a.lane_losses = lane_losses;
  a.outputs = outputs;
  vtrace::head_attach_workspace(&a, workspace);
  (void)hipGetLastError();
  return vtrace::launch_head(a, as_hip(stream)) == hipSuccess ? VTRACE_OK : VTRACE_ERR_HIP;
}

vtrace_status vtrace_error_flag(const void* workspace, int32_t* flag, vtrace_stream_t stream) {
  if (!workspace || !flag) return VTRACE_ERR_NULL;
  if (!aligned(workspace, 16)) return VTRACE_ERR_ALIGN;
  uint32_t v = 0;
  hipStream_t s = as_hip(stream);
  if (hipMemcpyAsync(&v, static_cast<const char*>(workspace) + vtrace::kWsFlagOffset, sizeof(v),
                     hipMemcpyDeviceToHost, s) != hipSuccess)
    return VTRACE_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return VTRACE_ERR_HIP;
  *flag = static_cast<int32_t>(v);
  return VTRACE_OK;
}

}  // extern "C"
