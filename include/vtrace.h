/*
 * libvtrace: the learner-side V-trace actor-critic step of IMPALA
 * (Espeholt et al., 2018, "IMPALA: Scalable Distributed Deep-RL with Importance
 * Weighted Actor-Learner Architectures"), on AMD Instinct MI355X (gfx950).
 *
 * C ABI.  Every array argument is a DEVICE pointer owned by the caller; the
 * library allocates nothing and keeps no global mutable state, except the
 * fixed device array behind vtrace_loss_grad_static.  Each call
 * validates its arguments on the host, enqueues its kernel(s) on `stream`
 * (NULL = the null stream) and returns without synchronising.  A returned
 * VTRACE_OK means the arguments were valid and the launch was accepted; device
 * faults surface on the caller's next synchronisation.
 *
 * Layout.  Batches are time-major and row-major: element (t, b) of a [T,B] array
 * is at index t*B + b, and element (t, b, j) of a [T,B,A] array at
 * (t*B + b)*A + j, the action axis innermost (the learner folds time into the
 * batch, paper Sec. 3.1).
 *
 * Inputs (shared by vtrace_targets and vtrace_loss_grad):
 *   target_logits     [T,B,A]  logits of the learner policy pi, dtype `logits_dtype`
 *   behaviour_logits  [T,B,A]  logits of the actor policy mu the actions were drawn from
 *   actions           [T,B]    int32, 0 <= a < A
 *   rewards           [T,B]    float32, r_t
 *   discounts         [T,B]    float32, gamma_t: discount between x_t and x_{t+1};
 *                              0 marks an episode that ended after step t
 *   values            [T,B]    float32, V(x_t)
 *   bootstrap_value   [B]      float32, V(x_T)
 *   rho_bar, c_bar             truncation levels of Sec. 4.1; >= 0, +INFINITY allowed
 *                              (no truncation).  rho_bar < c_bar is accepted.
 *   lambda                     trace discount of Remark 2, in [0, 1]; scales c only.
 *
 * Definitions computed (Sec. 4.1, Eq. (1), Remarks 1-2, Sec. 4.2):
 *   ratio_t = pi(a_t|x_t) / mu(a_t|x_t)             (from the two log-softmaxes)
 *   rho_t   = min(rho_bar, ratio_t)
 *   c_t     = lambda * min(c_bar, ratio_t)
 *   delta_t = rho_t (r_t + gamma_t V(x_{t+1}) - V(x_t)),  V(x_T) = bootstrap_value
 *   v_s     = V(x_s) + sum_{t=s}^{T-1} (gamma_s..gamma_{t-1})(c_s..c_{t-1}) delta_t
 *             (every v_s uses the rest of the unroll; v_T = V(x_T))
 *   pg_adv_s = rho_s (r_s + gamma_s v_{s+1} - V(x_s))
 *
 * Numerics.  The recursion, advantages and loss partial sums are float64.  The
 * exponent sums of both log-softmaxes, and from them the importance ratio and
 * log pi(a_t|x_t), are float64 (float64 exponentials of exact differences,
 * about 1e-10 relative) in every call that forms losses, and in a targets-only
 * call whose weights can exceed 1 (V-trace with rho_bar > 1 or
 * lambda * c_bar > 1, where products of c_t amplify the ratio's rounding).  A
 * targets-only call with every weight at most 1 forms them from float32
 * exponentials.  The per-element softmax work of the gradient and the entropy
 * is float32.  Outputs are float32 (or bfloat16 where a variant asks for it).
 * NaN or Inf inputs are propagated, not sanitised.
 *
 * Errors that only the device can see.  An action outside [0, A) makes that
 * step's importance ratio NaN; the NaN reaches that step's outputs, every
 * earlier step of the same lane, and the policy-gradient, baseline and total
 * losses (the entropy loss does not depend on actions).  When a workspace is
 * passed the kernel also raises a sticky flag in it (vtrace_error_flag).
 *
 * Outputs must not alias inputs or each other.  Base pointers of logits,
 * d_logits and gathered arrays must be 16-byte aligned; all others 4-byte.
 * Calls are re-entrant; concurrent calls need distinct workspaces.
 */
#ifndef VTRACE_H_
#define VTRACE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t. */
typedef struct ihipStream_t* vtrace_stream_t;

typedef enum {
  VTRACE_OK = 0,
  VTRACE_ERR_NULL = 1,      /* a required pointer is NULL */
  VTRACE_ERR_SHAPE = 2,     /* T, B or A < 1, or T*B*A beyond the supported range */
  VTRACE_ERR_DTYPE = 3,     /* unknown logits dtype */
  VTRACE_ERR_PARAM = 4,     /* NaN or out-of-range scalar parameter */
  VTRACE_ERR_ALIGN = 5,     /* a base pointer breaks the alignment rule above */
  VTRACE_ERR_WORKSPACE = 6, /* workspace NULL or smaller than vtrace_workspace_bytes */
  VTRACE_ERR_HIP = 7        /* the HIP runtime rejected the launch */
} vtrace_status;

typedef enum {
  VTRACE_F32 = 0,  /* IEEE binary32 logits */
  VTRACE_BF16 = 1, /* bfloat16 logits (upper half of a binary32) */
  /* Not dtypes: they give the type the range of int32_t, so that any int32
     value a caller passes is a defined value (rejected with VTRACE_ERR_DTYPE). */
  VTRACE_DTYPE_RANGE_MIN_ = -0x7fffffff - 1,
  VTRACE_DTYPE_RANGE_MAX_ = 0x7fffffff
} vtrace_dtype;

/*
 * Off-policy correction variants compared in the paper (Sec. 5.2.3) and the
 * choice of the Q estimate in the advantage (App. E.3).  The default, V-trace
 * with q_s = r_s + gamma_s v_{s+1}, is what vtrace_targets and vtrace_loss_grad
 * compute.
 */
typedef enum {
  VTRACE_CORRECTION_VTRACE = 0,     /* V-trace (Sec. 4) */
  VTRACE_CORRECTION_NONE = 1,       /* no correction: rho = c = 1 in the target (c = lambda with
                                       lambda < 1), no weight on the advantage */
  VTRACE_CORRECTION_EPSILON = 2,    /* as NONE, with log(pi(a|x) + epsilon) in place of
                                       log pi(a|x) in the policy-gradient term */
  VTRACE_CORRECTION_ONE_STEP_IS = 3 /* uncorrected target (as NONE), advantage times rho_s */
} vtrace_correction;

typedef enum {
  VTRACE_Q_VTRACE = 0,  /* q_s = r_s + gamma_s v_{s+1} (Sec. 4.2) */
  VTRACE_Q_BASELINE = 1 /* q_s = r_s + gamma_s V(x_{s+1}) (App. E.3) */
} vtrace_q_estimate;

/*
 * What the behaviour-policy argument holds.  The paper's actors send the
 * behaviour policy's probabilities of the actions they took (Sec. 3); with
 * LOG_PROBS the caller passes log mu(a_t|x_t) directly and the kernel reads
 * 4 bytes per step instead of a whole logit row.
 */
typedef enum {
  VTRACE_BEHAVIOUR_LOGITS = 0,   /* [T,B,A] logits of mu, in logits_dtype, 16-byte aligned */
  VTRACE_BEHAVIOUR_LOG_PROBS = 1 /* [T,B] float32 log mu(a_t|x_t), 4-byte aligned */
} vtrace_behaviour_input;

/* Reward preprocessing applied inside the kernel (App. D). */
typedef enum {
  VTRACE_REWARD_RAW = 0,       /* rewards used as given */
  VTRACE_REWARD_CLIP = 1,      /* clipped to [-1, 1] (single tasks) */
  VTRACE_REWARD_ASYMMETRIC = 2 /* 0.3 min(tanh r, 0) + 5 max(tanh r, 0) (DMLab-30) */
} vtrace_reward_transform;

typedef struct {
  int32_t correction;       /* a vtrace_correction */
  int32_t q_estimate;       /* a vtrace_q_estimate */
  float epsilon;            /* VTRACE_CORRECTION_EPSILON only: finite and > 0 (paper: 1e-6) */
  int32_t behaviour_input;  /* a vtrace_behaviour_input */
  int32_t reward_transform; /* a vtrace_reward_transform */
  int32_t grad_dtype;       /* element type of d_logits: VTRACE_F32 or VTRACE_BF16 (rounded to
                               nearest even); vtrace_loss_grad_ex only */
} vtrace_variant;

/* Version of this interface; bumped on any incompatible change. */
int vtrace_abi_version(void);

/*
 * Static, never-NULL description of a status code.  Takes any int32 value (a
 * vtrace_status converts implicitly); values that are not a vtrace_status give
 * "unknown status".
 */
const char* vtrace_status_string(int32_t status);

/* Largest T*B*A the kernels accept. */
int64_t vtrace_max_elements(void);

/*
 * Bytes of device workspace that vtrace_loss_grad needs for a [T,B,A] batch
 * (the cross-workgroup loss partials, a completion counter and the error
 * flag).  Returns 0 for invalid sizes.
 */
size_t vtrace_workspace_bytes(int64_t T, int64_t B, int64_t A);

/*
 * Clears a workspace (counter, error flag, partials) with a fill kernel on
 * `stream`.  Call once after allocating it; vtrace_loss_grad leaves the counter
 * at zero again after every call, so a workspace can be reused without clearing.
 */
vtrace_status vtrace_workspace_init(void* workspace, size_t workspace_bytes,
                                    vtrace_stream_t stream);

/*
 * V-trace targets and policy-gradient advantages (Sec. 4.1, Eq. (1), Remark 1;
 * Sec. 4.2 for pg_adv).
 *   vs, pg_advantages  [T,B] float32 outputs (both required)
 *   workspace          optional (may be NULL, then workspace_bytes is ignored):
 *                      when given, receives the out-of-range-action flag.
 */
vtrace_status vtrace_targets(
    int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
    const void* target_logits, const void* behaviour_logits, const int32_t* actions,
    const float* rewards, const float* discounts, const float* values,
    const float* bootstrap_value, float rho_bar, float c_bar, float lambda,
    float* vs, float* pg_advantages,
    void* workspace, size_t workspace_bytes, vtrace_stream_t stream);

/*
 * The V-trace actor-critic losses and their gradients (Sec. 4.2), fused with the
 * targets into one pass over the batch.
 *
 * Losses, each a sum (not a mean) over batch and time, as the caption of the
 * hyperparameter-range table in App. D states:
 *   policy gradient  L_pg  = -sum pg_adv_s * log pi(a_s|x_s)
 *   baseline         L_v   = baseline_cost * 1/2 * sum (v_s - V(x_s))^2
 *   entropy          L_ent = entropy_cost * sum_s sum_a pi(a|x_s) log pi(a|x_s)
 * Descending these moves along the paper's three update directions: the
 * importance-weighted policy gradient, the value direction (v_s - V)grad V and
 * the entropy bonus.  The paper's settings are baseline_cost = 0.5 and
 * entropy_cost = 0.01 (App. D).  rho, c, v_s and pg_adv are targets: no gradient
 * flows through them, and none reaches behaviour_logits or bootstrap_value.
 *
 *   baseline_cost, entropy_cost  finite floats
 *   losses        [4] float32 device: {L_pg + L_v + L_ent, L_pg, L_v, L_ent}
 *   d_logits      [T,B,A] float32: dL/d target_logits
 *                 = pg_adv_t (pi_j - 1[j = a_t]) + entropy_cost pi_j (log pi_j + H_t),
 *                 H_t = -sum_j pi_j log pi_j
 *   d_values      [T,B] float32: dL/dV(x_t) = baseline_cost (V(x_t) - v_t)
 *   vs, pg_advantages  optional [T,B] float32 outputs (NULL to skip)
 *   lane_losses   optional [B,3] float32: per-lane {L_pg, L_v, L_ent} over time
 *   workspace     required, >= vtrace_workspace_bytes(T,B,A) bytes, cleared once
 *                 by vtrace_workspace_init.
 * The loss totals are reduced in a fixed order: repeated calls on the same
 * inputs give bit-identical results.
 */
vtrace_status vtrace_loss_grad(
    int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
    const void* target_logits, const void* behaviour_logits, const int32_t* actions,
    const float* rewards, const float* discounts, const float* values,
    const float* bootstrap_value, float rho_bar, float c_bar, float lambda,
    float baseline_cost, float entropy_cost,
    float* losses, float* d_logits, float* d_values,
    float* vs, float* pg_advantages, float* lane_losses,
    void* workspace, size_t workspace_bytes, vtrace_stream_t stream);

/*
 * vtrace_targets / vtrace_loss_grad with a variant.  `variant` is a HOST
 * pointer read during the call (NULL = V-trace with the defaults above); an
 * unknown enumerator or a bad epsilon gives VTRACE_ERR_PARAM.  NONE and EPSILON
 * do not use the importance ratio: behaviour_logits must still be a valid
 * array of the declared kind, but its values do not change the outputs.
 * In vtrace_loss_grad_ex, d_logits has the element type variant->grad_dtype.
 */
vtrace_status vtrace_targets_ex(
    int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
    const void* target_logits, const void* behaviour_logits, const int32_t* actions,
    const float* rewards, const float* discounts, const float* values,
    const float* bootstrap_value, float rho_bar, float c_bar, float lambda,
    const vtrace_variant* variant, float* vs, float* pg_advantages,
    void* workspace, size_t workspace_bytes, vtrace_stream_t stream);

vtrace_status vtrace_loss_grad_ex(
    int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
    const void* target_logits, const void* behaviour_logits, const int32_t* actions,
    const float* rewards, const float* discounts, const float* values,
    const float* bootstrap_value, float rho_bar, float c_bar, float lambda,
    float baseline_cost, float entropy_cost, const vtrace_variant* variant,
    float* losses, void* d_logits, float* d_values,
    float* vs, float* pg_advantages, float* lane_losses,
    void* workspace, size_t workspace_bytes, vtrace_stream_t stream);

/*
 * vtrace_loss_grad_ex for callers that cannot allocate device memory: code
 * being captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc.  It takes no workspace and allocates nothing (no hipMalloc,
 * hipFree or allocating library call): its cross-workgroup loss partials and
 * completion counter live in a device array of the library,
 * VTRACE_STATIC_WORKSPACE_BYTES bytes on each device that runs the call, held
 * until the process ends.  B above VTRACE_STATIC_MAX_LANES gives
 * VTRACE_ERR_WORKSPACE (use vtrace_loss_grad_ex); every other argument and
 * error is as in vtrace_loss_grad_ex.
 *
 * The first call on a device asks the runtime for the array's address on that
 * device (the device current at the call) and clears its counter with a fill
 * kernel on `stream`; later calls on other streams must be ordered after that
 * first one.  Every call on a device shares the one array: calls that overlap
 * on a device (concurrent streams, threads) race and give wrong losses, so
 * order them.  There is no readable error flag: an out-of-range action still
 * gives NaN outputs as documented above.  Outputs are bit-identical to those
 * of vtrace_loss_grad_ex on the same inputs.
 */
#define VTRACE_STATIC_MAX_LANES 65536
#define VTRACE_STATIC_WORKSPACE_BYTES (256 + 24 * VTRACE_STATIC_MAX_LANES)

vtrace_status vtrace_loss_grad_static(
    int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
    const void* target_logits, const void* behaviour_logits, const int32_t* actions,
    const float* rewards, const float* discounts, const float* values,
    const float* bootstrap_value, float rho_bar, float c_bar, float lambda,
    float baseline_cost, float entropy_cost, const vtrace_variant* variant,
    float* losses, void* d_logits, float* d_values,
    float* vs, float* pg_advantages, float* lane_losses, vtrace_stream_t stream);

/*
 * Copies of the logits at the taken actions: gathered[t,b,0] = target_logits[t,b,a_t]
 * and gathered[t,b,1] = behaviour_logits[t,b,a_t], bit for bit, in the logits
 * dtype ([T,B,2]).  These are the pi(a_t|x_t) and mu(a_t|x_t) lookups of
 * Sec. 4.1 before normalisation.  Out-of-range actions give all-ones bit
 * patterns (a NaN in both dtypes).
 */
vtrace_status vtrace_gather_logits(
    int64_t T, int64_t B, int64_t A, vtrace_dtype logits_dtype,
    const void* target_logits, const void* behaviour_logits, const int32_t* actions,
    void* gathered, vtrace_stream_t stream);

/*
 * The learner's output layer fused with the V-trace losses and the gradients
 * through the layer.  Sec. 3.1: after the LSTM, the fully connected output
 * layer is applied to all time steps at once.  Here that layer maps each
 * step's hidden state to A policy logits and the baseline,
 *   o[t,b,:] = hidden[t,b,:] @ head_weight + head_bias,
 *   policy logits = o[..., 0:A],  V(x_t) = o[..., A],
 * and the call computes the losses of vtrace_loss_grad on (logits, V) and, with
 * G = [d_logits, d_values] (dL/do),
 *   d_hidden = G @ head_weight^T,
 *   d_weight = sum over (t,b) of hidden[t,b,:]^T G[t,b,:],
 *   d_bias   = sum over (t,b) of G[t,b,:].
 * The logits, the values and their gradients never reach HBM.
 *
 *   H               hidden size: 64, 128 or 256 (else VTRACE_ERR_SHAPE)
 *   A               1..31 actions (A + 1 outputs; else VTRACE_ERR_SHAPE)
 *   behaviour_dtype element type of behaviour logits (VTRACE_F32 / VTRACE_BF16);
 *                   with variant->behaviour_input == LOG_PROBS `behaviour` is
 *                   [T,B] float32 log mu(a_t|x_t) and this is not used
 *   hidden          [T,B,H] bfloat16, 16-byte aligned
 *   head_weight     [H,A+1] bfloat16 (2-byte aligned), column A is the baseline
 *   head_bias       [A+1] float32
 *   behaviour       [T,B,A] behaviour logits (element-aligned) or log-probabilities
 *   bootstrap_value [B] float32 V(x_T): a target, it receives no gradient
 *   variant         as in vtrace_loss_grad_ex (NULL = V-trace); grad_dtype is
 *                   the element type of d_hidden
 *   losses          [4] float32, as in vtrace_loss_grad
 *   d_hidden        [T,B,H] float32 or bfloat16, 16-byte aligned
 *   d_weight        [H,A+1] float32;  d_bias [A+1] float32
 *   vs, pg_advantages, lane_losses   optional, as in vtrace_loss_grad
 *   outputs         optional [T,B,A+1] float32: the layer's outputs o
 *   workspace       required, >= vtrace_head_workspace_bytes(T,B,A,H) bytes,
 *                   16-byte aligned, cleared once by vtrace_workspace_init
 * The products use bfloat16 inputs with float32 accumulation; G enters them as
 * a bfloat16 pair (high part + low part, 2^-17 relative), so d_hidden keeps
 * float32 accuracy.  d_weight, d_bias and the losses are reduced in a fixed
 * order: repeated calls give bit-identical results.  An out-of-range action
 * sets the workspace flag and makes d_weight and d_bias NaN, besides its own
 * step's outputs.
 */
size_t vtrace_head_workspace_bytes(int64_t T, int64_t B, int64_t A, int64_t H);

vtrace_status vtrace_head_loss_grad(
    int64_t T, int64_t B, int64_t A, int64_t H, vtrace_dtype behaviour_dtype,
    const void* hidden, const void* head_weight, const float* head_bias,
    const void* behaviour, const int32_t* actions, const float* rewards,
    const float* discounts, const float* bootstrap_value,
    float rho_bar, float c_bar, float lambda, float baseline_cost, float entropy_cost,
    const vtrace_variant* variant,
    float* losses, void* d_hidden, float* d_weight, float* d_bias,
    float* vs, float* pg_advantages, float* lane_losses, float* outputs,
    void* workspace, size_t workspace_bytes, vtrace_stream_t stream);

/*
 * Synchronises `stream`, then reads the workspace's sticky out-of-range-action
 * flag into *flag (host pointer; 0 = no invalid action seen since the last
 * vtrace_workspace_init).
 */
vtrace_status vtrace_error_flag(const void* workspace, int32_t* flag, vtrace_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* VTRACE_H_ */
