// Tiled V-trace kernel, templated on the action count A (instantiated for
// 2 <= A <= 20 by tiled.hip and tiled_a*.hip; A = 9 is DeepMind Lab's set,
// A = 18 the full Atari set).
//
// Work split.  A tile is LANES consecutive lanes (batch entries) for the whole
// unroll; a workgroup walks a tile's time backwards in chunks of L steps (16 by
// default; 8 or 4 for the long-run tile shapes of 64 or 128 lanes), so every
// carry of the reverse recursion stays inside the workgroup.  Within a chunk,
// thread (lane, s) handles step t = t0 + s; the L threads of one lane are an
// aligned segment of a 16-lane DPP row of a wave.  When the batch has a whole
// multiple of the tiles the chip holds workgroups at once, each resident
// workgroup walks an equal share of tiles as one continuous sequence of chunks.
//
// Data path per chunk.
//  1. For each t the chunk's logits are one contiguous run of LANES*A elements
//     (1152 bytes for 16 lanes of fp32 logits with A = 18, nine 128-byte
//     lines; 4608 bytes for 64 lanes).  Threads copy both
//     tensors' runs with 16-byte loads into LDS.  These whole-line logit loads
//     and the gradient stores are used once, so they carry the non-temporal
//     hint; the [T,B] scalars, whose 64-byte halves neighbouring workgroups
//     share in L2, do not.  The loads of chunk k+1
//     (and its per-step scalars) are issued before chunk k is computed and land
//     in registers, so their latency hides behind the arithmetic.
//  2. Each thread reads its own two rows from LDS: row maxima, exponent sums,
//     the importance ratio (float64, see device_common.hpp), rho and c.
//  3. The recursion v_t - V(x_t) = delta_t + gamma_t c_t (v_{t+1} - V(x_{t+1}))
//     (Remark 1) is an affine map per step.  A suffix scan across the row (DPP
//     row shifts) composes the chunk's maps; applying them to the carry from
//     the later chunk gives every v_t of the chunk at once.
//  4. Advantages, d_values and the gradient row follow.  Gradient rows go
//     through LDS so that the global stores are whole 16-byte vectors along the
//     contiguous [t, b0:b0+LANES, :] runs.
//
// Workgroups whose lane tile is full and whose rows are 16-byte aligned take
// the vector path above; a ragged last tile (or unaligned rows) copies element
// by element without prefetching.
#pragma once

#include <atomic>
#include <type_traits>

#include "device_common.hpp"
#include "row_stats.hpp"
#include "wave_ops.hpp"

namespace vtrace {
namespace {

constexpr int kL = 16;  // default steps per chunk


// DPP row_shr:(L-1): lane i of a 16-lane row reads lane i-L+1, so the last
// lane of every aligned L-lane segment reads the segment's first (L = 16 is
// kRowShr15).
template <int L>
constexpr int row_shr_to_last() {
  static_assert(L >= 2 && L <= 16, "segment length");
  return 0x110 + (L - 1);
}

// L steps per chunk (16, 8 or 4): the L threads of a lane are one aligned
// segment of a 16-lane DPP row.  L = 32: a lane's threads are two DPP rows of
// a wave, steps 0-15 and 16-31 of the chunk.
template <int A_, int LANES, typename In, int L>
struct Tile {
  static constexpr int A = A_;
  static constexpr int NT = LANES * L;                         // threads per workgroup
  static constexpr int SEG = LANES * A_;                       // elements per time row
  static constexpr int IN_ROW16 = SEG * int(sizeof(In)) / 16;  // 16-byte vectors per row, logits
  static constexpr int OUT_ROW16 = SEG * 4 / 16;               // 16-byte vectors per row, d_logits
  // LDS rows are padded by one 16-byte vector: without it every step of a lane
  // would read the same banks (a row is a multiple of 128 bytes).
  static constexpr int IN_PITCH16 = IN_ROW16 + 1;
  static constexpr int OUT_PITCH16 = OUT_ROW16 + 1;
  static constexpr int IN_TILE16 = L * IN_ROW16;    // vectors per tensor and chunk
  static constexpr int OUT_TILE16 = L * OUT_ROW16;
  static constexpr int IN_LDS16 = L * IN_PITCH16;   // LDS footprint per tensor
  static constexpr int OUT_LDS16 = L * OUT_PITCH16;
  // Suffix-scan stages within a DPP row: log2 L, and 4 for L = 32, whose
  // lanes span two rows joined by one cross-row step.
  static constexpr int SCAN = L >= 16 ? 4 : L == 8 ? 3 : 2;
  static constexpr int NV = (2 * IN_TILE16 + NT - 1) / NT;  // vectors per thread, both tensors
  static constexpr int NO = (OUT_TILE16 + NT - 1) / NT;     // gradient vectors per thread
  // LDS: the two logit tiles, and for the gradient kernels a separate
  // staging tile for the gradient rows, so that a chunk needs two barriers
  // (logits staged; gradients staged) instead of four.
  static constexpr int LDS16_TARGETS = 2 * IN_LDS16;
  static constexpr int LDS16_GRAD = 2 * IN_LDS16 + OUT_LDS16;
  static constexpr int IN_PITCH = IN_PITCH16 * 16 / int(sizeof(In));  // elements per LDS row
  static constexpr int OUT_PITCH = OUT_PITCH16 * 4;                    // floats per LDS row
  static_assert((SEG * int(sizeof(In))) % 16 == 0, "logit rows must be whole 16-byte vectors");
  static_assert((SEG * 4) % 16 == 0, "gradient rows must be whole 16-byte vectors");
  static_assert(NT % kWave == 0 && NT <= 1024, "bad workgroup size");
  static_assert(OUT_ROW16 % 2 == 0, "bfloat16 gradient rows must be whole 16-byte vectors");
  static_assert(L == 32 || L == 16 || L == 8 || L == 4, "steps per chunk");
};

// For 32-step chunks (two lanes per wave, each on two DPP rows): x at the
// thread of step `step` (0 or 16) of this thread's lane, i.e. at wave lane
// step or 32 + step.  Two scalar reads per 32-bit half and a select.
template <int kStep>
__device__ __forceinline__ double lane_step_f64(double x, bool upper_lane) {
  const unsigned long long u = __double_as_longlong(x);
  const int lo = static_cast<int>(u & 0xffffffffu), hi = static_cast<int>(u >> 32);
  const int lo0 = __builtin_amdgcn_readlane(lo, kStep), lo1 = __builtin_amdgcn_readlane(lo, 32 + kStep);
  const int hi0 = __builtin_amdgcn_readlane(hi, kStep), hi1 = __builtin_amdgcn_readlane(hi, 32 + kStep);
  const unsigned l = static_cast<unsigned>(upper_lane ? lo1 : lo0), h = static_cast<unsigned>(upper_lane ? hi1 : hi0);
  return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(h) << 32) | l));
}

// Per-thread state carried along the chunk walk.
struct Carry {
  double V, v, A;  // V(x_{t+1}), v_{t+1}, v_{t+1} - V(x_{t+1}) at the later chunk's first step
  double pg, base, ent;
};

// Which variant switches a kernel takes at run time: all of them (kGeneralCall),
// none (kPlainCall: plain V-trace, is_plain_vtrace), only the reward
// transform and the gradient dtype (kPlainRewards: is_plain_vtrace_any_rewards),
// or those two with behaviour log-probabilities in place of behaviour logits,
// so that no behaviour row is read (kPlainLogProbs: is_plain_vtrace_log_probs).
constexpr int kGeneralCall = 0;
constexpr int kPlainCall = 1;
constexpr int kPlainRewards = 2;
constexpr int kPlainLogProbs = 3;

// Walks one tile (kMulti false: `tile`, with the carry cy set up by the
// caller), or (kMulti true, vector tiles only) the tiles first_tile + i *
// tile_stride, i < ntiles, one after another as one loop over their chunks, so
// that the prefetch runs across tile boundaries; each lane's loss totals are
// then added to acc[3 * lane], a slot only the lane's step-0 thread touches.
template <int A_, int LANES, typename In, int L, bool kGrad, bool kPrecise, bool kVec, bool kMulti, int kPlain>
__device__ __forceinline__ void chunk_walk(const StepArgs& a, v4u* lds, int64_t first_tile,
                                           int64_t tile_stride, int64_t ntiles, Carry& cy,
                                           double* acc) {
  static_assert(kVec || !kMulti, "the multi-tile walk takes vector tiles only");
  using S = Tile<A_, LANES, In, L>;
  constexpr int NT = S::NT;
  v4u* const lds_z = lds;
  v4u* const lds_y = lds + S::IN_LDS16;
  v4u* const lds_g = lds + 2 * S::IN_LDS16;  // gradient staging (kGrad)

  const int tid = threadIdx.x;
  const int lane_local = tid / L;
  const int s = tid % L;
  const int wl = tid % kWave;  // the thread's place in its wave
  const int64_t T = a.T, B = a.B;
  const int nchunks = static_cast<int>((T + L - 1) / L);

  // Byte stride of one time row of logits.
  const int64_t in_row = B * A_ * int64_t(sizeof(In));
  // kPlain: the call is plain V-trace (q_s from v_{s+1}, behaviour logits or,
  // for kPlainLogProbs, log-probabilities), so every variant switch below is a
  // compile-time constant; kPlainCall also has rewards as given and float32
  // gradients, while the other plain kernels keep the reward transform and
  // the gradient dtype run-time switches.
  const int correction = kPlain ? kCorrVtrace : a.correction;
  const int q_estimate = kPlain ? 0 : a.q_estimate;
  const int reward_transform = kPlain == kPlainCall ? 0 : a.reward_transform;
  const bool beh_lp = kPlain == kPlainLogProbs || (!kPlain && a.behaviour_log_probs != 0);
  // No-correction and epsilon-correction never look at the behaviour policy.
  const bool no_ratio = correction == kCorrNone || correction == kCorrEpsilon;
  const bool skip_y = beh_lp || no_ratio;
  const bool grad_bf16 = kPlain != kPlainCall && a.grad_bf16 != 0;
  const int64_t gsz = grad_bf16 ? 2 : 4;  // bytes per gradient element
  const int64_t out_row = B * A_ * gsz;
  const float* const lmu_g = static_cast<const float*>(a.behaviour_logits);
  auto lane_ok_of = [&](int64_t b0) { return kMulti || b0 + lane_local < B; };  // the walk takes full tiles

  // Register prefetch (vector path): NV 16-byte vectors covering both tensors,
  // plus this thread's action, reward, discount and value, and at a tile's
  // first chunk its lane's bootstrap value.
  v4u pre[S::NV];
  int32_t p_act = 0;
  float p_r = 0.f, p_g = 0.f, p_V = 0.f, p_lmu = 0.f, p_boot = 0.f;

  // Vector-path addresses are a wave-uniform base (the chunk's row 0 at the
  // tile's first lane, in scalar registers) plus a per-thread 32-bit offset,
  // the form of the loads' and stores' scalar-base addressing; the launcher
  // takes the vector path only where L rows of every array fit 32-bit offsets.
  const uint32_t in_row32 = static_cast<uint32_t>(in_row);
  const uint32_t out_row32 = static_cast<uint32_t>(out_row);
  const uint32_t B32 = static_cast<uint32_t>(B);
  auto prefetch = [&](int64_t tile, int k) {
    const int64_t b0 = tile * LANES;
    const int64_t t0 = T - static_cast<int64_t>(k + 1) * L;
    const int neg = t0 < 0 ? static_cast<int>(-t0) : 0;  // rows before t = 0 reread row `neg`
    const int64_t row0 = t0 * B + b0;                     // may be negative: only rows >= neg are read
    const gptr<const char> zg = offset_bytes(a.target_logits, row0 * A_ * int64_t(sizeof(In)));
    const gptr<const char> yg = offset_bytes(a.behaviour_logits, row0 * A_ * int64_t(sizeof(In)));
    static_for<S::NV>([&](auto I) {
      constexpr int i = decltype(I)::value;
      // Which tensor vector i of every thread belongs to, where that is known
      // at compile time (all but the vector that straddles the two tiles).
      constexpr bool kAllZ = (i + 1) * NT <= S::IN_TILE16;
      constexpr bool kAllY = i * NT >= S::IN_TILE16;
      constexpr bool kTail = i * NT + NT > 2 * S::IN_TILE16;
      const int f = tid + i * NT;
      const bool is_y = kAllY || (!kAllZ && f >= S::IN_TILE16);
      if ((!kTail || f < 2 * S::IN_TILE16) && !(is_y && skip_y)) {
        const int g = is_y ? f - S::IN_TILE16 : f;
        int r = g / S::IN_ROW16;
        const int c = g % S::IN_ROW16;
        r = r < neg ? neg : r;
        const uint32_t off = static_cast<uint32_t>(r) * in_row32 + static_cast<uint32_t>(c) * 16u;
        pre[i] = __builtin_nontemporal_load(reinterpret_cast<gptr<const v4u>>((is_y ? yg : zg) + off));
      }
    });
    if (lane_ok_of(b0)) {
      const uint32_t off = static_cast<uint32_t>(s < neg ? neg : s) * B32 + static_cast<uint32_t>(lane_local);
      p_act = offset_elems(a.actions, row0)[off];
      p_r = offset_elems(a.rewards, row0)[off];
      p_g = offset_elems(a.discounts, row0)[off];
      p_V = offset_elems(a.values, row0)[off];
      if (beh_lp && !no_ratio) p_lmu = offset_elems(lmu_g, row0)[off];
      if (kMulti && k == 0) p_boot = a.bootstrap_value[b0 + lane_local];
    }
  };

  const double rho_bar = a.rho_bar, c_bar = a.c_bar, lam = a.lambda;
  const float ce = a.entropy_cost;

  int64_t tile = first_tile;  // advanced by the multi-tile walk only
  int k = 0;
  // Chunks to walk: a tile's, or all the tiles' (which may exceed 32 bits).
  using Count = std::conditional_t<kMulti, int64_t, int>;
  const Count total = kMulti ? static_cast<Count>(ntiles * nchunks) : static_cast<Count>(nchunks);
  if constexpr (kVec) prefetch(tile, 0);
  for (Count it = 0; it < total; ++it) {
    const int64_t b0 = tile * LANES;
    const int64_t b = b0 + lane_local;
    const bool lane_ok = kMulti || b < B;  // the multi-tile walk takes full tiles only
    const int nb = static_cast<int>(B - b0 < LANES ? B - b0 : LANES);
    if constexpr (kMulti) {
      if (k == 0) {
        // A new tile: the carry past its last step is the bootstrap value
        // (v_T = V(x_T), so v_T - V(x_T) = 0).
        cy.V = cy.v = p_boot;
        cy.A = 0.0;
      }
    }
    const int64_t t0 = T - static_cast<int64_t>(k + 1) * L;
    const int64_t t = t0 + s;
    const bool step_ok = lane_ok && t >= 0;
    const int64_t idx = t * B + b;
    // [T,B] element (t, b) as the chunk's uniform row 0 plus a 32-bit offset
    // (vector path); where step_ok, t >= 0.
    const int64_t row0 = t0 * B + b0;
    const uint32_t soff = static_cast<uint32_t>(s) * B32 + static_cast<uint32_t>(lane_local);

    // Every thread is past the previous chunk's row reads: the gradient
    // kernels passed their staging barrier after them; the targets-only
    // kernel waits here.
    if constexpr (!kGrad) __syncthreads();
    int32_t act;
    float r32, g32, V32, lmu = 0.f;
    if constexpr (kVec) {
      static_for<S::NV>([&](auto I) {
        constexpr int i = decltype(I)::value;
        const int f = tid + i * NT;
        const bool is_y = f >= S::IN_TILE16;
        if ((i * NT + NT <= 2 * S::IN_TILE16 || f < 2 * S::IN_TILE16) && !(is_y && skip_y)) {
          const int g = is_y ? f - S::IN_TILE16 : f;
          const int r = g / S::IN_ROW16, c = g % S::IN_ROW16;
          lds[(is_y ? S::IN_LDS16 : 0) + r * S::IN_PITCH16 + c] = pre[i];
        }
      });
      act = p_act;
      r32 = p_r;
      g32 = p_g;
      V32 = p_V;
      lmu = p_lmu;
      // The next chunk's loads go out before the staging barrier (their
      // registers are free once staged) with float32 logits on the long-run
      // shapes: stress step 0.730 -> 0.714 ms, bf16 gradients 0.682 -> 0.670,
      // targets-only 0.550 -> 0.537.  With bf16 logits (and the raised
      // priority below) only the kernel that reads no behaviour rows gains
      // (0.485-0.491 -> 0.466-0.468 ms, with bf16 gradients 0.453-0.455 ->
      // 0.432-0.433); the others, and the 16-step tiles, measured up to 1%
      // slower and keep them after it.
      constexpr bool kEarlyPrefetch =
          L <= 8 && (std::is_same_v<In, float> || kPlain == kPlainLogProbs);
      // The wave issues those loads at raised priority, so that the other
      // waves' arithmetic on the same SIMD does not delay them: stress step
      // 0.727-0.730 -> 0.714-0.716 ms, 16-step tiles with float32 logits and
      // bf16 logits on the long-run shapes 1-2% faster; bf16 logits on the
      // 16-step tiles measured 1% slower with it and keep normal priority.
      constexpr bool kPrioPrefetch = std::is_same_v<In, float> || L <= 8;
      auto next_prefetch = [&]() {
        if constexpr (kMulti) {
          if (it + 1 < total) {
            const bool next_tile = k + 1 == nchunks;
            prefetch(next_tile ? tile + tile_stride : tile, next_tile ? 0 : k + 1);
          }
        } else {
          if (k + 1 < nchunks) prefetch(tile, k + 1);
        }
      };
      auto issue_prefetch = [&]() {
        if constexpr (kPrioPrefetch) __builtin_amdgcn_s_setprio(2);
        next_prefetch();
        if constexpr (kPrioPrefetch) __builtin_amdgcn_s_setprio(0);
      };
      if constexpr (kEarlyPrefetch) issue_prefetch();
      __syncthreads();
      if constexpr (!kEarlyPrefetch) issue_prefetch();
    } else {
      In* lz = reinterpret_cast<In*>(lds_z);
      In* ly = reinterpret_cast<In*>(lds_y);
      for (int e = tid; e < L * S::SEG; e += NT) {
        const int rr = e / S::SEG, c = e % S::SEG;
        const int64_t te = t0 + rr;
        if (te >= 0 && c < nb * A_) {
          const int64_t off = (te * B + b0) * A_ + c;
          lz[rr * S::IN_PITCH + c] = static_cast<const In*>(a.target_logits)[off];
          if (!skip_y) ly[rr * S::IN_PITCH + c] = static_cast<const In*>(a.behaviour_logits)[off];
        }
      }
      act = 0;
      r32 = g32 = V32 = 0.f;
      if (step_ok) {
        act = a.actions[idx];
        r32 = a.rewards[idx];
        g32 = a.discounts[idx];
        V32 = a.values[idx];
        if (beh_lp && !no_ratio) lmu = lmu_g[idx];
      }
      __syncthreads();
    }
    r32 = transform_reward(r32, reward_transform);
    if (!step_ok) act = 0;  // rows that do not exist carry a harmless action

    // This thread's rows.
    const In* zr = reinterpret_cast<const In*>(lds_z) + s * S::IN_PITCH + lane_local * A_;
    const In* yr = reinterpret_cast<const In*>(lds_y) + s * S::IN_PITCH + lane_local * A_;
    const bool act_ok = act >= 0 && act < A_;
    const int act_c = act_ok ? act : 0;
    if (!act_ok) raise_error_flag(a.error_flag);
    // e_j and z_j for the gradient.  The plain loss kernels (every kPlain
    // mode) keep both in registers from the row statistics to the gradient
    // (36 VGPRs that their two waves per SIMD have), which spares each row two
    // LDS round trips; the general kernel, which needs those registers for its
    // switches, takes e_j through this thread's row of the gradient staging tile (free
    // since the previous chunk's stores, which every thread finished before
    // this chunk's logits barrier), where the gradient row later replaces
    // them, and read z_j again from the logit tile.  The targets-only kernels
    // use neither.
    static_assert(!kGrad || kPrecise, "loss kernels form their exponent sums in float64");
    constexpr bool kRowRegs = kGrad && kPlain;
    float e_reg[A_], z_reg[A_];
    float* const lo = kGrad ? reinterpret_cast<float*>(lds_g) + s * S::OUT_PITCH + lane_local * A_ : e_reg;
    float* const e_out = kGrad && !kRowRegs ? lo : e_reg;
    RowStats st = row_stats<A_, kPrecise>(zr, yr, act_c, act_ok, beh_lp, no_ratio, lmu, e_out,
                                          kRowRegs ? z_reg : nullptr);
    const StepWeights w = variant_weights(correction, clip_above(st.ratio, rho_bar),
                                          lam * clip_above(st.ratio, c_bar), lam, act_ok);

    const double r = r32, g = g32, V = V32;
    // kSeg: steps of a lane within one DPP row; sr: this thread's place there.
    constexpr int kSeg = L < 16 ? L : 16;
    const int sr = s % kSeg;
    const bool upper_lane = wl >= 32;  // L = 32: the wave's second lane
    double V16 = 0.0;                  // L = 32: V(x) at step 16 of the lane
    if constexpr (L == 32) V16 = lane_step_f64<16>(V, upper_lane);
    double V_next = dpp_f64<kRowShl1>(V);
    if (L == 32 && s == 15) V_next = V16;
    if (s == L - 1) V_next = cy.V;
    const double delta = w.rho_v * (r + g * V_next - V);

    // Suffix scan over the lane's segment.  Its last step first absorbs the
    // carry from the later chunk, so that after the scan D holds v_t - V(x_t)
    // on every thread: (G, D) composes the maps of steps s..L-1 applied to
    // that carry.  With 32 steps the scan runs in each DPP row, and the lower
    // row then composes its maps with the upper row's first step.
    double G = g * w.c_v, D = delta;
    if (s == L - 1) D = fma(G, cy.A, D);
    static_for<S::SCAN>([&](auto I) {
      constexpr int off = 1 << decltype(I)::value;
      const double Gn = dpp_f64<0x100 + off>(G);
      const double Dn = dpp_f64<0x100 + off>(D);
      if (sr + off < kSeg) {
        D = fma(G, Dn, D);
        G = G * Gn;
      }
    });
    double D16 = 0.0;  // L = 32: v - V(x) at step 16 of the lane
    if constexpr (L == 32) {
      D16 = lane_step_f64<16>(D, upper_lane);
      if (s < 16) D = fma(G, D16, D);
    }
    const double A_t = D;  // v_t - V(x_t)
    const double v_t = V + A_t;
    double v_next = dpp_f64<kRowShl1>(v_t);
    if (L == 32 && s == 15) v_next = V16 + D16;
    if (s == L - 1) v_next = cy.v;
    const double q_next = q_estimate == kQBaseline ? V_next : v_next;
    const double adv = w.rho_pg * (r + g * q_next - V);

    // The segment's first step becomes the carry of the earlier chunk, held by
    // the segment's last thread, the only one that reads it.
    if constexpr (L == 32) {
      cy.A = lane_step_f64<0>(A_t, upper_lane);
      cy.v = lane_step_f64<0>(v_t, upper_lane);
      cy.V = lane_step_f64<0>(V, upper_lane);
    } else {
      cy.A = dpp_f64<row_shr_to_last<L>()>(A_t);
      cy.v = dpp_f64<row_shr_to_last<L>()>(v_t);
      cy.V = dpp_f64<row_shr_to_last<L>()>(V);
    }

    if (step_ok) {
      if constexpr (kVec) {
        if (a.vs) offset_elems(a.vs, row0)[soff] = static_cast<float>(v_t);
        if (a.pg_adv) offset_elems(a.pg_adv, row0)[soff] = static_cast<float>(adv);
      } else {
        if (a.vs) a.vs[idx] = static_cast<float>(v_t);
        if (a.pg_adv) a.pg_adv[idx] = static_cast<float>(adv);
      }
    }

    if constexpr (kGrad) {
      // d_logits_j = adv (pi_j - 1[j=a]) + ce pi_j (log pi_j + H), where
      // log pi_j + H = z_j - K.  For j != a this is e_j (alpha + beta z_j).
      const float K = st.mz + st.log_s - st.H;
      // epsilon-correction: the policy-gradient term is -adv log(pi_a + eps),
      // whose gradient is adv pi_a/(pi_a + eps) (pi_j - 1[j=a]).
      const float pa = st.e_a * st.inv_s;
      const bool eps_mode = correction == kCorrEpsilon;
      const float pg_w = eps_mode ? pa / (pa + a.epsilon) : 1.0f;
      const float adv32 = static_cast<float>(adv) * pg_w;
      const float beta = st.inv_s * ce;
      const float alpha = st.inv_s * adv32 - beta * K;
      const float za = logit_to_float(zr[act_c]);
      const float out_a = -adv32 * st.one_minus_pa + ce * pa * (za - K);
      if (step_ok) {
        const float dv = static_cast<float>(a.baseline_cost * (V - v_t));
        if constexpr (kVec)
          offset_elems(a.d_values, row0)[soff] = dv;
        else
          a.d_values[idx] = dv;
        const double log_pa = !act_ok ? NAN : eps_mode ? log_prob_plus_eps<kPrecise>(st, a.epsilon) : st.log_pa;
        cy.pg += -adv * log_pa;
        cy.base += 0.5 * A_t * A_t;
        cy.ent += -static_cast<double>(st.H);
      }
      float out[A_];
#pragma unroll
      for (int j = 0; j < A_; ++j) out[j] = e_out[j] * fmaf(beta, kRowRegs ? z_reg[j] : logit_to_float(zr[j]), alpha);
#pragma unroll
      for (int j = 0; j < A_; ++j) lo[j] = out[j];
      lo[act_c] = act_ok ? out_a : NAN;
      __syncthreads();
      if constexpr (kVec) {
        const int neg = t0 < 0 ? static_cast<int>(-t0) : 0;
        const gptr<char> dgr = offset_bytes(a.d_logits, row0 * A_ * gsz);  // the chunk's row 0
        if (!grad_bf16) {
          // The kernel that reads no behaviour rows spends a larger share of
          // each chunk on these stores; issued at raised priority its stress
          // step took 0.528-0.530 -> 0.519-0.522 ms (the default kernel's
          // measured 0.4% slower with it).
          if constexpr (kPlain == kPlainLogProbs) __builtin_amdgcn_s_setprio(2);
          static_for<S::NO>([&](auto I) {
            constexpr int i = decltype(I)::value;
            const int f = tid + i * NT;
            if (i * NT + NT <= S::OUT_TILE16 || f < S::OUT_TILE16) {
              const int rr = f / S::OUT_ROW16, cc = f % S::OUT_ROW16;
              if (rr >= neg)
                __builtin_nontemporal_store(
                    lds_g[rr * S::OUT_PITCH16 + cc],
                    reinterpret_cast<gptr<v4u>>(dgr + (static_cast<uint32_t>(rr) * out_row32 +
                                                  static_cast<uint32_t>(cc) * 16u)));
            }
          });
          if constexpr (kPlain == kPlainLogProbs) __builtin_amdgcn_s_setprio(0);
        } else {
          // bfloat16 rows: each 16-byte store packs two 16-byte LDS vectors.
          constexpr int kRow16 = S::OUT_ROW16 / 2, kTile16 = S::OUT_TILE16 / 2;
          for (int f = tid; f < kTile16; f += NT) {
            const int rr = f / kRow16, cc = f % kRow16;
            if (rr >= neg) {
              const v4u lo = lds_g[rr * S::OUT_PITCH16 + 2 * cc];
              const v4u hi = lds_g[rr * S::OUT_PITCH16 + 2 * cc + 1];
              v4u pk;
              pk.x = pack_bf16x2(__uint_as_float(lo.x), __uint_as_float(lo.y));
              pk.y = pack_bf16x2(__uint_as_float(lo.z), __uint_as_float(lo.w));
              pk.z = pack_bf16x2(__uint_as_float(hi.x), __uint_as_float(hi.y));
              pk.w = pack_bf16x2(__uint_as_float(hi.z), __uint_as_float(hi.w));
              __builtin_nontemporal_store(pk, reinterpret_cast<gptr<v4u>>(dgr + (static_cast<uint32_t>(rr) * out_row32 +
                                                                             static_cast<uint32_t>(cc) * 16u)));
            }
          }
        }
      } else {
        const float* lf = reinterpret_cast<const float*>(lds_g);
        for (int e2 = tid; e2 < L * S::SEG; e2 += NT) {
          const int rr = e2 / S::SEG, cc = e2 % S::SEG;
          const int64_t te = t0 + rr;
          if (te >= 0 && cc < nb * A_) {
            const float x = lf[rr * S::OUT_PITCH + cc];
            const int64_t o = (te * B + b0) * A_ + cc;
            if (grad_bf16)
              static_cast<uint16_t*>(a.d_logits)[o] = to_bf16(x);
            else
              static_cast<float*>(a.d_logits)[o] = x;
          }
        }
      }
      if (kMulti && k == nchunks - 1) {
        // The tile's last chunk: this lane's totals over the row (fixed
        // butterfly order), then the workgroup's running sums.
        double lp = cy.pg, lb = cy.base, le = cy.ent;
#pragma unroll
        for (int off = L / 2; off > 0; off >>= 1) {
          lp += __shfl_xor(lp, off, L);
          lb += __shfl_xor(lb, off, L);
          le += __shfl_xor(le, off, L);
        }
        lb *= a.baseline_cost;
        le *= a.entropy_cost;
        if (s == 0 && lane_ok) {
          if (a.lane_losses) {
            a.lane_losses[3 * b + 0] = static_cast<float>(lp);
            a.lane_losses[3 * b + 1] = static_cast<float>(lb);
            a.lane_losses[3 * b + 2] = static_cast<float>(le);
          }
          acc[3 * lane_local + 0] += lp;
          acc[3 * lane_local + 1] += lb;
          acc[3 * lane_local + 2] += le;
        }
        cy.pg = cy.base = cy.ent = 0.0;
      }
    }
    if (++k == nchunks && kMulti) {
      k = 0;
      tile += tile_stride;
    }
  }
}

// Tile of a workgroup.  Below 64 lanes a tile's share of a [T,B] time row is
// under 256 bytes and neighbouring tiles share its 128-byte lines, so
// xcd_tile puts workgroups that run side by side on one XCD on neighbouring
// tiles, which then meet in that XCD's L2.  From 64 lanes on nothing is shared
// and tiles go in workgroup order, which measured 1-4% faster for the long-run
// shapes (and the XCD order 1% faster for 16-lane tiles).
template <int LANES>
__device__ __forceinline__ int64_t first_tile_of_workgroup() {
  if constexpr (LANES >= 64) return blockIdx.x;
  return xcd_tile(blockIdx.x, gridDim.x);
}

// kMulti false: one workgroup per tile, tile first_tile_of_workgroup().
//
// kMulti true: the grid is exactly the workgroups the chip holds at once and
// each walks tiles_per_wg vector tiles, first_tile_of_workgroup() + i * gridDim.x.
// When a batch has a whole multiple of that many tiles, this runs it as one
// even generation: one workgroup per tile would instead start a second wave of
// workgroups whenever a slot frees, and leave the chip partly idle at the end.
// The fp64 ratio mode with A > 18 is asked for two waves per SIMD explicitly:
// left to itself the compiler gives A = 19 two registers more than fit.
template <int A_, int LANES, typename In, int L, bool kGrad, bool kPrecise, bool kMulti, int kPlain = kGeneralCall>
__global__ __launch_bounds__(LANES* L, (kPrecise && A_ >= 18) ? 2 : 1) void tiled_kernel(
    StepArgs a, int64_t num_vec_tiles, int64_t tiles_per_wg) {
  using S = Tile<A_, LANES, In, L>;
  constexpr int NT = S::NT;
  __shared__ v4u lds[kGrad ? S::LDS16_GRAD : S::LDS16_TARGETS];
  __shared__ double red_scratch[3 * (NT / kWave)];

  const int lane_local = threadIdx.x / L;
  const int s = threadIdx.x % L;

  if constexpr (kMulti) {
    __shared__ double acc[3 * LANES];  // per-lane loss sums over the workgroup's tiles
    if (s == 0) acc[3 * lane_local + 0] = acc[3 * lane_local + 1] = acc[3 * lane_local + 2] = 0.0;
    Carry cy{0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    chunk_walk<A_, LANES, In, L, kGrad, kPrecise, true, true, kPlain>(a, lds, first_tile_of_workgroup<LANES>(),
                                                              gridDim.x, tiles_per_wg, cy, acc);
    if constexpr (kGrad) {
      double pg = 0.0, base = 0.0, ent = 0.0;
      if (s == 0) {
        pg = acc[3 * lane_local + 0];
        base = acc[3 * lane_local + 1];
        ent = acc[3 * lane_local + 2];
      }
      finish_losses<NT>(a, pg, base, ent, red_scratch);
    }
  } else {
    const int64_t tile = first_tile_of_workgroup<LANES>();
    const int64_t b = tile * LANES + lane_local;
    const bool lane_ok = b < a.B;
    const double boot = lane_ok ? static_cast<double>(a.bootstrap_value[b]) : 0.0;
    Carry cy{boot, boot, 0.0, 0.0, 0.0, 0.0};

    if (tile < num_vec_tiles)
      chunk_walk<A_, LANES, In, L, kGrad, kPrecise, true, false, kPlain>(a, lds, tile, 0, 1, cy, nullptr);
    else
      chunk_walk<A_, LANES, In, L, kGrad, kPrecise, false, false, kPlain>(a, lds, tile, 0, 1, cy, nullptr);

    if constexpr (kGrad) {
      // Per-lane totals over the row (fixed butterfly order), then the workgroup.
      double pg = cy.pg, base = cy.base, ent = cy.ent;
#pragma unroll
      for (int off = L / 2; off > 0; off >>= 1) {
        pg += __shfl_xor(pg, off, L);
        base += __shfl_xor(base, off, L);
        ent += __shfl_xor(ent, off, L);
      }
      base *= a.baseline_cost;
      ent *= a.entropy_cost;
      if (s == 0 && lane_ok && a.lane_losses) {
        a.lane_losses[3 * b + 0] = static_cast<float>(pg);
        a.lane_losses[3 * b + 1] = static_cast<float>(base);
        a.lane_losses[3 * b + 2] = static_cast<float>(ent);
      }
      if (s != 0 || !lane_ok) pg = base = ent = 0.0;
      finish_losses<NT>(a, pg, base, ent, red_scratch);
    }
  }
}

// Workgroups of the multi-tile kernel that fit on a compute unit at once,
// asked of the runtime once (0 if it cannot say).
template <int A_, int LANES, typename In, int L, bool kGrad>
int multi_workgroups_per_cu() {
  static std::atomic<int> cached{-1};
  int n = cached.load(std::memory_order_relaxed);
  if (n < 0) {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &blocks, reinterpret_cast<const void*>(tiled_kernel<A_, LANES, In, L, kGrad, false, true>),
            LANES * L, 0) != hipSuccess) {
      (void)hipGetLastError();  // not a launch error: the single-tile kernel runs instead
      blocks = 0;
    }
    n = blocks > 0 ? blocks : 0;
    cached.store(n, std::memory_order_relaxed);
  }
  return n;
}

// Workgroups of the single-tile float32-ratio kernel that fit on a compute
// unit at once, asked of the runtime once (0 if it cannot say).
template <int A_, int LANES, typename In, int L, bool kGrad>
int single_workgroups_per_cu() {
  static std::atomic<int> cached{-1};
  int n = cached.load(std::memory_order_relaxed);
  if (n < 0) {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &blocks, reinterpret_cast<const void*>(tiled_kernel<A_, LANES, In, L, kGrad, false, false>),
            LANES * L, 0) != hipSuccess) {
      (void)hipGetLastError();
      blocks = 0;
    }
    n = blocks > 0 ? blocks : 0;
    cached.store(n, std::memory_order_relaxed);
  }
  return n;
}

// Compute units of the current device (0 if the runtime cannot say).
int compute_units() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cached[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 0;
  }
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      return 0;
    }
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Launches the kernel; returns its grid size.  The multi-tile kernel runs when
// every tile is a vector tile, two or more of its workgroups fit on a CU, the
// tiles are a whole multiple (at least two) of the resident workgroups, and the
// ratio takes the float32 mode.  Elsewhere one workgroup per tile measured as
// fast or faster: a batch that is not a whole multiple would leave some
// workgroups a tile short, the float64 ratio mode has no registers to spare for
// the longer walk, and with one resident workgroup per CU (the 512-thread
// kernel of bfloat16 logits with A = 18) the multi-tile walk measured 4-10%
// slower.
template <int A_, int LANES, typename In, int L, bool kGrad, bool kPrecise, int kPlain = kGeneralCall>
int64_t launch_kernel(const StepArgs& a, hipStream_t st, int64_t tiles, int64_t vec_tiles,
                      bool allow_multi) {
  if constexpr (!kPrecise) {
    const int per_cu = allow_multi && vec_tiles == tiles ? multi_workgroups_per_cu<A_, LANES, In, L, kGrad>() : 0;
    if (per_cu >= 2) {
      const int64_t resident = static_cast<int64_t>(per_cu) * compute_units();
      if (resident > 0 && tiles >= 2 * resident && tiles % resident == 0) {
        hipLaunchKernelGGL((tiled_kernel<A_, LANES, In, L, kGrad, false, true>), dim3(static_cast<unsigned>(resident)),
                           dim3(LANES * L), 0, st, a, vec_tiles, tiles / resident);
        return resident;
      }
    }
  }
  hipLaunchKernelGGL((tiled_kernel<A_, LANES, In, L, kGrad, kPrecise, false, kPlain>),
                     dim3(static_cast<unsigned>(tiles)), dim3(LANES * L), 0, st, a, vec_tiles, int64_t(1));
  return tiles;
}

// Loss kernels always take the float64 exponent sums; a targets-only call
// takes them when its weights can amplify ratio errors.  kFastOnly: only the
// float32 mode is instantiated (the caller has checked precise_row_sums).
template <int A_, int LANES, typename In, int L, bool kGrad, bool kFastOnly, bool kPlainVariants = false>
int64_t launch_mode(const StepArgs& a, hipStream_t st, int64_t tiles, int64_t vec_tiles,
                    bool allow_multi) {
  if constexpr (kGrad) {
    if (is_plain_vtrace(a))
      return launch_kernel<A_, LANES, In, L, true, true, kPlainCall>(a, st, tiles, vec_tiles, allow_multi);
    if constexpr (kPlainVariants) {
      if (is_plain_vtrace_any_rewards(a))
        return launch_kernel<A_, LANES, In, L, true, true, kPlainRewards>(a, st, tiles, vec_tiles, allow_multi);
      if (is_plain_vtrace_log_probs(a))
        return launch_kernel<A_, LANES, In, L, true, true, kPlainLogProbs>(a, st, tiles, vec_tiles, allow_multi);
    }
    return launch_kernel<A_, LANES, In, L, true, true>(a, st, tiles, vec_tiles, allow_multi);
  } else {
    if constexpr (!kFastOnly) {
      if (precise_row_sums(a, false))
        return launch_kernel<A_, LANES, In, L, false, true>(a, st, tiles, vec_tiles, allow_multi);
    }
    return launch_kernel<A_, LANES, In, L, false, false>(a, st, tiles, vec_tiles, allow_multi);
  }
}

// kPlainVariants: loss calls that are plain V-trace but for a reward
// transform, bfloat16 gradients or behaviour log-probabilities take plain
// kernels too (instantiated for the long-run loss shapes only).
template <int A_, int LANES, typename In, int L = kL, bool kFastOnly = false, bool kPlainVariants = false>
hipError_t launch_shape(const StepArgs& a, Mode mode, hipStream_t st, int64_t* nwg, bool allow_multi) {
  if (kFastOnly && precise_row_sums(a, mode == Mode::LossGrad)) return hipErrorInvalidValue;
  if constexpr (kFastOnly) {
    if (mode == Mode::LossGrad) return hipErrorInvalidValue;  // never instantiated
  }
  const int64_t tiles = (a.B + LANES - 1) / LANES;
  // Vector path: full lane tiles whose time rows start on 16-byte boundaries.
  const int64_t in_row = a.B * A_ * int64_t(sizeof(In));
  const int64_t out_row = a.B * A_ * (a.grad_bf16 ? 2 : 4);
  const bool aligned = (in_row % 16 == 0) && (out_row % 16 == 0);
  // The vector path addresses L rows of each array from a uniform base with
  // 32-bit offsets (L rows of logits, of gradients, of [T,B] scalars).
  constexpr int64_t k4G = int64_t(1) << 32;
  const bool offsets32 = L * in_row < k4G && L * out_row < k4G && L * a.B * 4 < k4G;
  const int64_t vec_tiles = aligned && offsets32 ? a.B / LANES : 0;
  if constexpr (!kFastOnly) {
    if (mode == Mode::LossGrad) {
      *nwg = launch_mode<A_, LANES, In, L, true, false, kPlainVariants>(a, st, tiles, vec_tiles, allow_multi);
      return hipGetLastError();
    }
  }
  *nwg = launch_mode<A_, LANES, In, L, false, kFastOnly>(a, st, tiles, vec_tiles, allow_multi);
  return hipGetLastError();
}

// Tile shapes with longer contiguous runs per time row (LANES * A elements):
// at T = 1000 the same traffic streams 5-20% faster from 2304- to 9216-byte
// runs than from 1152-byte ones, provided the workgroups keep every CU busy.
template <int LANES_, int L_>
struct Shape {
  static constexpr int LANES = LANES_;
  static constexpr int L = L_;
};
constexpr int kMinWavesPerCu = 8;

// The batch fills the chip once: the tile count is a whole multiple of the CU
// count, every tile's workgroup is resident from the start, and each CU holds
// at least kMinWavesPerCu waves.
template <int A_, typename In, bool kGrad, typename Sh>
bool fills_once(int64_t B, int cus) {
  if (B % Sh::LANES != 0) return false;
  const int64_t tiles = B / Sh::LANES;
  if (tiles % cus != 0) return false;
  const int64_t per_cu = tiles / cus;
  return per_cu <= single_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kGrad>() &&
         per_cu * (Sh::LANES * Sh::L / kWave) >= kMinWavesPerCu;
}

// The multi-tile walk of this shape runs the batch as even generations.
template <int A_, typename In, bool kGrad, typename Sh>
bool walks_evenly(int64_t B, int cus) {
  if (B % Sh::LANES != 0) return false;
  const int64_t tiles = B / Sh::LANES;
  const int64_t resident = static_cast<int64_t>(multi_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kGrad>()) * cus;
  return resident >= 2 * static_cast<int64_t>(cus) && tiles >= 2 * resident && tiles % resident == 0;
}

// One workgroup per tile runs the batch as 2 to kMaxGenerations whole
// generations of resident workgroups, each CU holding at least kMinWavesPerCu
// waves.  (Measured up to four generations.)
constexpr int64_t kMaxGenerations = 4;
template <int A_, typename In, bool kGrad, typename Sh>
bool whole_generations(int64_t B, int cus) {
  if (B % Sh::LANES != 0) return false;
  const int64_t tiles = B / Sh::LANES;
  const int per_cu = single_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kGrad>();
  const int64_t resident = static_cast<int64_t>(per_cu) * cus;
  return per_cu * (Sh::LANES * Sh::L / kWave) >= kMinWavesPerCu && resident > 0 && tiles % resident == 0 &&
         tiles >= 2 * resident && tiles <= kMaxGenerations * resident;
}

enum class ShapeTest { FillsOnce, WalksEvenly, WholeGenerations };

template <int A_, typename In, bool kGrad, typename Sh>
bool shape_fits(ShapeTest test, int64_t B, int cus) {
  switch (test) {
    case ShapeTest::FillsOnce: return fills_once<A_, In, kGrad, Sh>(B, cus);
    case ShapeTest::WalksEvenly: return walks_evenly<A_, In, kGrad, Sh>(B, cus);
    case ShapeTest::WholeGenerations: return whole_generations<A_, In, kGrad, Sh>(B, cus);
  }
  return false;
}

template <int A_, typename In>
bool try_shapes(const StepArgs&, Mode, hipStream_t, int64_t*, bool, hipError_t*, int, ShapeTest) {
  return false;
}
template <int A_, typename In, typename Sh, typename... Rest>
bool try_shapes(const StepArgs& a, Mode mode, hipStream_t st, int64_t* nwg, bool allow_multi, hipError_t* err,
                int cus, ShapeTest test) {
  if (mode == Mode::LossGrad) return false;  // loss calls: launch_long_loss
  if (shape_fits<A_, In, false, Sh>(test, a.B, cus)) {
    *err = launch_shape<A_, Sh::LANES, In, Sh::L, true>(a, mode, st, nwg, allow_multi);
    return true;
  }
  return try_shapes<A_, In, Rest...>(a, mode, st, nwg, allow_multi, err, cus, test);
}

// Launches the first of Shapes (listed longest runs first) whose batch fills
// the chip once, else the first that the multi-tile walk runs as even
// generations (the choice does not depend on allow_multi, which only says
// whether the walk may run), else the first whose single-tile workgroups run
// it as a few whole generations; returns false (launching nothing) when none
// applies or the ratio needs the float64 mode (where the 16-step chunks of the
// default shapes measured as fast or faster).
template <int A_, typename In, typename... Shapes>
bool launch_long(const StepArgs& a, Mode mode, hipStream_t st, int64_t* nwg, bool allow_multi, hipError_t* err) {
  if (precise_row_sums(a, mode == Mode::LossGrad)) return false;
  const int cus = compute_units();
  if (cus <= 0) return false;
  return try_shapes<A_, In, Shapes...>(a, mode, st, nwg, allow_multi, err, cus, ShapeTest::FillsOnce) ||
         try_shapes<A_, In, Shapes...>(a, mode, st, nwg, allow_multi, err, cus, ShapeTest::WalksEvenly) ||
         try_shapes<A_, In, Shapes...>(a, mode, st, nwg, allow_multi, err, cus, ShapeTest::WholeGenerations);
}

// Workgroups of the single-tile loss kernel (plain or with variants) that fit
// on a compute unit at once, asked of the runtime once (0 if it cannot say).
template <int A_, int LANES, typename In, int L, int kPlain>
int loss_workgroups_per_cu() {
  static std::atomic<int> cached{-1};
  int n = cached.load(std::memory_order_relaxed);
  if (n < 0) {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &blocks, reinterpret_cast<const void*>(tiled_kernel<A_, LANES, In, L, true, true, false, kPlain>),
            LANES * L, 0) != hipSuccess) {
      (void)hipGetLastError();
      blocks = 0;
    }
    n = blocks > 0 ? blocks : 0;
    cached.store(n, std::memory_order_relaxed);
  }
  return n;
}

// Loss calls on the long-run shapes: the first of Shapes whose workgroups run
// the batch as 1 to kMaxGenerations whole generations of resident workgroups,
// each CU holding at least kMinWavesPerCu waves; false (launching nothing)
// when none applies.  (The loss kernels fit two workgroups of 256 threads per
// CU, so the multi-tile walk, which needs more, does not serve them.)
template <int A_, typename In>
bool launch_long_loss(const StepArgs&, hipStream_t, int64_t*, hipError_t*, int) {
  return false;
}
template <int A_, typename In, typename Sh, typename... Rest>
bool launch_long_loss(const StepArgs& a, hipStream_t st, int64_t* nwg, hipError_t* err, int cus) {
  if (a.B % Sh::LANES == 0) {
    const int64_t tiles = a.B / Sh::LANES;
    const int per_cu = is_plain_vtrace(a) ? loss_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kPlainCall>()
                       : is_plain_vtrace_any_rewards(a)
                           ? loss_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kPlainRewards>()
                       : is_plain_vtrace_log_probs(a)
                           ? loss_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kPlainLogProbs>()
                           : loss_workgroups_per_cu<A_, Sh::LANES, In, Sh::L, kGeneralCall>();
    const int64_t resident = static_cast<int64_t>(per_cu) * cus;
    if (per_cu * (Sh::LANES * Sh::L / kWave) >= kMinWavesPerCu && resident > 0 && tiles % resident == 0 &&
        tiles <= kMaxGenerations * resident) {
      *err = launch_shape<A_, Sh::LANES, In, Sh::L, false, true>(a, Mode::LossGrad, st, nwg, false);
      return true;
    }
  }
  return launch_long_loss<A_, In, Rest...>(a, st, nwg, err, cus);
}
template <int A_, typename In, typename... Shapes>
bool launch_long_loss(const StepArgs& a, hipStream_t st, int64_t* nwg, hipError_t* err) {
  const int cus = compute_units();
  if (cus <= 0) return false;
  return launch_long_loss<A_, In, Shapes...>(a, st, nwg, err, cus);
}

// Launch for action count A with 16 lanes per workgroup, fp32 or bf16 logits.
template <int A_>
hipError_t launch_shape_16(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st, int64_t* nwg,
                           bool allow_multi) {
  if (lt == LogitsType::F32) return launch_shape<A_, 16, float>(a, mode, st, nwg, allow_multi);
  return launch_shape<A_, 16, uint16_t>(a, mode, st, nwg, allow_multi);
}

}  // namespace
}  // namespace vtrace
