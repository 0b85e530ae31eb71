// Tiled V-trace kernel for the common action counts (A = 9: DeepMind Lab,
// A = 18: the full Atari set).
//
// Work split.  A workgroup owns LANES consecutive lanes (batch entries) for the
// whole unroll and walks time backwards in chunks of L = 16 steps, so every
// carry of the reverse recursion stays inside the workgroup.  Within a chunk,
// thread (lane, s) handles step t = t0 + s; the 16 threads of one lane form one
// row of a wave.
//
// Data path per chunk.
//  1. The chunk's [L, LANES, A] slabs of target and behaviour logits are, for
//     each t, one contiguous run of LANES*A elements (1152 bytes for every
//     supported shape, nine 128-byte lines).  Threads copy them with 16-byte
//     loads into LDS.  The copy of chunk k+1 is issued before chunk k is
//     computed, so its latency hides behind the arithmetic.
//  2. Each thread reads its own two rows from LDS: max, exponent sums, the
//     importance ratio (float64, see device_common.hpp), rho and c.
//  3. The recursion v_t - V(x_t) = delta_t + gamma_t c_t (v_{t+1} - V(x_{t+1}))
//     (Remark 1) is an affine map per step.  A suffix scan across the 16
//     threads of the lane's row composes the maps of the chunk; applying the
//     result to the carry from the later chunk gives every v_t at once.
//  4. Advantages, d_values and the gradient row follow.  Gradient rows go
//     through LDS so that the global stores are whole 16-byte vectors along the
//     contiguous [t, b0:b0+LANES, :] runs.
#include <utility>

#include "device_common.hpp"

namespace vtrace {
namespace {

constexpr int kL = 16;  // steps per chunk = threads per lane row

// A native 16-byte vector: plain vector loads and stores, kept in registers
// (HIP's v4u wrapper is copied through memory when carried across loops).
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// Calls f(std::integral_constant<int, i>) for i = 0..N-1, unrolled at compile
// time so that arrays indexed by i stay in registers.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int A_, int LANES, typename In>
struct Tile {
  static constexpr int A = A_;
  static constexpr int NT = LANES * kL;                          // threads per workgroup
  static constexpr int SEG = LANES * A_;                         // elements per time row
  static constexpr int IN_ROW16 = SEG * int(sizeof(In)) / 16;    // 16-byte vectors per row, logits
  static constexpr int OUT_ROW16 = SEG * 4 / 16;                 // 16-byte vectors per row, d_logits
  static constexpr int IN_TILE16 = kL * IN_ROW16;
  static constexpr int OUT_TILE16 = kL * OUT_ROW16;
  static constexpr int NV = (IN_TILE16 + NT - 1) / NT;  // prefetch vectors per thread per tensor
  static constexpr int LDS16 = (2 * IN_TILE16 > OUT_TILE16) ? 2 * IN_TILE16 : OUT_TILE16;
  static_assert((SEG * int(sizeof(In))) % 16 == 0, "logit rows must be whole 16-byte vectors");
  static_assert((SEG * 4) % 16 == 0, "gradient rows must be whole 16-byte vectors");
  static_assert(NT % kWave == 0 && NT <= 1024, "bad workgroup size");
};

template <int A_, int LANES, typename In, bool kGrad>
__global__ __launch_bounds__(LANES* kL) void tiled_kernel(StepArgs a) {
  using S = Tile<A_, LANES, In>;
  constexpr int NT = S::NT;
  __shared__ v4u lds[S::LDS16];
  __shared__ double red_scratch[3 * (NT / kWave)];
  v4u* const lds_z = lds;
  v4u* const lds_y = lds + S::IN_TILE16;

  const int tid = threadIdx.x;
  const int lane_local = tid / kL;
  const int s = tid % kL;  // step within the chunk
  const int row_base = (tid % kWave) & ~(kL - 1);
  const int64_t T = a.T, B = a.B;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * LANES;
  const int64_t b = b0 + lane_local;
  const bool lane_ok = b < B;
  const int nb = static_cast<int>(B - b0 < LANES ? B - b0 : LANES);  // lanes present in this tile
  // 16-byte copies need every [t, b0, :] run to start on a 16-byte boundary.
  const bool vec = (nb == LANES) && ((B * A_ * int64_t(sizeof(In))) % 16 == 0) &&
                   ((B * A_ * 4) % 16 == 0);
  const int nchunks = static_cast<int>((T + kL - 1) / kL);

  const char* zg = static_cast<const char*>(a.target_logits);
  const char* yg = static_cast<const char*>(a.behaviour_logits);
  const In* zg_e = static_cast<const In*>(a.target_logits);
  const In* yg_e = static_cast<const In*>(a.behaviour_logits);

  v4u pz[S::NV], py[S::NV];  // prefetched logits of the next chunk (vector path)

  auto chunk_t0 = [&](int k) -> int64_t { return T - static_cast<int64_t>(k + 1) * kL; };

  // Issues the 16-byte loads of chunk k's logits into pz/py.
#define VTRACE_PREFETCH(k_)                                                                 \
  do {                                                                                      \
    const int64_t pf_t0 = chunk_t0(k_);                                                     \
    static_for<S::NV>([&](auto I) {                                                         \
      constexpr int i = decltype(I)::value;                                                 \
      const int idx = tid + i * NT;                                                         \
      if (idx < S::IN_TILE16) {                                                             \
        const int r = idx / S::IN_ROW16, c = idx % S::IN_ROW16;                             \
        const int64_t t = pf_t0 + r;                                                        \
        if (t >= 0) {                                                                       \
          const int64_t off = (t * B + b0) * A_ * int64_t(sizeof(In)) + int64_t(c) * 16;    \
          pz[i] = *reinterpret_cast<const v4u*>(zg + off);                                \
          py[i] = *reinterpret_cast<const v4u*>(yg + off);                                \
        }                                                                                   \
      }                                                                                     \
    });                                                                                     \
  } while (0)

  // Puts chunk k's logits into LDS, laid out [s][lane][j] like global memory.
  auto commit_scalar = [&](int k) {
    // Ragged lane tile or unaligned rows: element copies of what exists.
    const int64_t t0 = chunk_t0(k);
    In* lz = reinterpret_cast<In*>(lds_z);
    In* ly = reinterpret_cast<In*>(lds_y);
    for (int e = tid; e < kL * S::SEG; e += NT) {
      const int r = e / S::SEG, c = e % S::SEG;
      const int64_t t = t0 + r;
      if (t >= 0 && c < nb * A_) {
        const int64_t off = (t * B + b0) * A_ + c;
        lz[e] = zg_e[off];
        ly[e] = yg_e[off];
      }
    }
  };

  // Writes the chunk's gradient rows from LDS to global memory.
  auto store_grads = [&](int k) {
    const int64_t t0 = chunk_t0(k);
    if (vec) {
      char* dg = reinterpret_cast<char*>(a.d_logits);
      for (int idx = tid; idx < S::OUT_TILE16; idx += NT) {
        const int r = idx / S::OUT_ROW16, c = idx % S::OUT_ROW16;
        const int64_t t = t0 + r;
        if (t >= 0) {
          const int64_t off = (t * B + b0) * A_ * 4 + int64_t(c) * 16;
          *reinterpret_cast<v4u*>(dg + off) = lds[idx];
        }
      }
    } else {
      const float* lo = reinterpret_cast<const float*>(lds);
      for (int e = tid; e < kL * S::SEG; e += NT) {
        const int r = e / S::SEG, c = e % S::SEG;
        const int64_t t = t0 + r;
        if (t >= 0 && c < nb * A_) a.d_logits[(t * B + b0) * A_ + c] = lo[e];
      }
    }
  };

  const double rho_bar = a.rho_bar, c_bar = a.c_bar, lam = a.lambda;
  const float ce = a.entropy_cost;
  const double boot = lane_ok ? static_cast<double>(a.bootstrap_value[b]) : 0.0;
  // Carries from the first step of the later chunk: V(x_{t+1}), v_{t+1}, v_{t+1} - V(x_{t+1}).
  double carry_V = boot, carry_v = boot, carry_A = 0.0;
  double acc_pg = 0.0, acc_base = 0.0, acc_ent = 0.0;

  if (vec) VTRACE_PREFETCH(0);
  for (int k = 0; k < nchunks; ++k) {
    const int64_t t = chunk_t0(k) + s;
    const bool step_ok = lane_ok && t >= 0;
    const int64_t idx = t * B + b;

    __syncthreads();  // previous chunk is done with LDS
    if (vec) {
      static_for<S::NV>([&](auto I) {
        constexpr int i = decltype(I)::value;
        const int li = tid + i * NT;
        if (li < S::IN_TILE16) {
          lds_z[li] = pz[i];
          lds_y[li] = py[i];
        }
      });
    } else {
      commit_scalar(k);
    }
    // Per-step scalars of this thread.
    int32_t act = 0;
    double r = 0.0, g = 0.0, V = 0.0;
    if (step_ok) {
      act = a.actions[idx];
      r = a.rewards[idx];
      g = a.discounts[idx];
      V = a.values[idx];
    }
    __syncthreads();
    if (vec && k + 1 < nchunks) VTRACE_PREFETCH(k + 1);

    // Own rows from LDS.
    const In* zr = reinterpret_cast<const In*>(lds_z) + (s * LANES + lane_local) * A_;
    const In* yr = reinterpret_cast<const In*>(lds_y) + (s * LANES + lane_local) * A_;
    float dz[A_], e[A_];
    float mz = -INFINITY, my = -INFINITY, za = 0.f, ya = 0.f;
#pragma unroll
    for (int j = 0; j < A_; ++j) {
      dz[j] = logit_to_float(zr[j]);
      mz = fmaxf(mz, dz[j]);
      if (j == act) za = dz[j];
    }
    double sy = 0.0;
    {
      float yv[A_];
#pragma unroll
      for (int j = 0; j < A_; ++j) {
        yv[j] = logit_to_float(yr[j]);
        my = fmaxf(my, yv[j]);
        if (j == act) ya = yv[j];
      }
#pragma unroll
      for (int j = 0; j < A_; ++j) sy += static_cast<double>(expf(yv[j] - my));
    }
    double sz = 0.0;
    float ed = 0.f, ea = 0.f;
#pragma unroll
    for (int j = 0; j < A_; ++j) {
      dz[j] -= mz;
      e[j] = expf(dz[j]);
      sz += static_cast<double>(e[j]);
      ed += e[j] * dz[j];
      if (j == act) ea = e[j];
    }

    const bool act_ok = act >= 0 && act < A_;
    if (!act_ok) raise_error_flag(a.error_flag);
    const double ratio = act_ok ? importance_ratio(za, mz, ya, my, sz, sy) : NAN;
    const double rho = clip_above(ratio, rho_bar);
    const double c = lam * clip_above(ratio, c_bar);

    // V(x_{t+1}) from the next thread of the row, or the later chunk's carry.
    double V_next = __shfl_down(V, 1, kL);
    if (s == kL - 1) V_next = carry_V;
    const double delta = rho * (r + g * V_next - V);

    // Suffix scan of the affine maps x -> delta_t + (gamma_t c_t) x over the row:
    // (G, D) composes steps t..15 of the chunk.
    double G = g * c, D = delta;
#pragma unroll
    for (int off = 1; off < kL; off <<= 1) {
      const double Gn = __shfl_down(G, off, kL);
      const double Dn = __shfl_down(D, off, kL);
      if (s + off < kL) {
        D = D + G * Dn;
        G = G * Gn;
      }
    }
    const double A_t = D + G * carry_A;  // v_t - V(x_t)
    const double v_t = V + A_t;
    double v_next = __shfl_down(v_t, 1, kL);
    if (s == kL - 1) v_next = carry_v;
    const double adv = rho * (r + g * v_next - V);

    // Carries for the earlier chunk come from the row's first thread.
    carry_A = __shfl(A_t, row_base, kWave);
    carry_v = __shfl(v_t, row_base, kWave);
    carry_V = __shfl(V, row_base, kWave);

    if (step_ok) {
      if (a.vs) a.vs[idx] = static_cast<float>(v_t);
      if (a.pg_adv) a.pg_adv[idx] = static_cast<float>(adv);
    }

    if constexpr (kGrad) {
      const float szf = static_cast<float>(sz);
      const float inv = 1.0f / szf;
      const float log_s = logf(szf);
      const float H = log_s - ed * inv;
      const float one_minus_pa = static_cast<float>((sz - static_cast<double>(ea)) / sz);
      const float adv32 = static_cast<float>(adv);
      float out[A_];
#pragma unroll
      for (int j = 0; j < A_; ++j) {
        const float p = e[j] * inv;
        const float pg_term = (j == act) ? -one_minus_pa : p;
        out[j] = adv32 * pg_term + ce * p * ((dz[j] - log_s) + H);
      }
      if (step_ok) {
        a.d_values[idx] = static_cast<float>(a.baseline_cost * (V - v_t));
        const double log_pa = act_ok ? static_cast<double>(za - mz) - static_cast<double>(log_s) : NAN;
        acc_pg += -adv * log_pa;
        acc_base += 0.5 * A_t * A_t;
        acc_ent += -static_cast<double>(H);
      }
      __syncthreads();  // all rows read: LDS now holds the gradient tile
      float* lo = reinterpret_cast<float*>(lds) + (s * LANES + lane_local) * A_;
#pragma unroll
      for (int j = 0; j < A_; ++j) lo[j] = out[j];
      __syncthreads();
      store_grads(k);
    }
  }

#undef VTRACE_PREFETCH
  if constexpr (kGrad) {
    // Per-lane totals over the row (fixed butterfly order), then the workgroup.
#pragma unroll
    for (int off = kL / 2; off > 0; off >>= 1) {
      acc_pg += __shfl_xor(acc_pg, off, kL);
      acc_base += __shfl_xor(acc_base, off, kL);
      acc_ent += __shfl_xor(acc_ent, off, kL);
    }
    acc_base *= a.baseline_cost;
    acc_ent *= a.entropy_cost;
    if (s == 0 && lane_ok && a.lane_losses) {
      a.lane_losses[3 * b + 0] = static_cast<float>(acc_pg);
      a.lane_losses[3 * b + 1] = static_cast<float>(acc_base);
      a.lane_losses[3 * b + 2] = static_cast<float>(acc_ent);
    }
    if (s != 0 || !lane_ok) acc_pg = acc_base = acc_ent = 0.0;
    finish_losses<NT>(a, acc_pg, acc_base, acc_ent, red_scratch);
  }
}

template <int A_, int LANES, typename In>
hipError_t launch_shape(const StepArgs& a, Mode mode, hipStream_t st, int64_t* nwg) {
  const int64_t blocks = (a.B + LANES - 1) / LANES;
  *nwg = blocks;
  if (mode == Mode::LossGrad)
    hipLaunchKernelGGL((tiled_kernel<A_, LANES, In, true>), dim3(static_cast<unsigned>(blocks)),
                       dim3(LANES * kL), 0, st, a);
  else
    hipLaunchKernelGGL((tiled_kernel<A_, LANES, In, false>), dim3(static_cast<unsigned>(blocks)),
                       dim3(LANES * kL), 0, st, a);
  return hipGetLastError();
}

}  // namespace

bool tiled_supported(const StepArgs& a, LogitsType) { return a.A == 9 || a.A == 18; }

// Lanes per workgroup: the smallest count whose [t, b0:b0+LANES, :] run of
// logits is 1152 bytes (nine 128-byte lines).
hipError_t launch_tiled(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st,
                        int64_t* num_workgroups) {
  if (lt == LogitsType::F32) {
    if (a.A == 18) return launch_shape<18, 16, float>(a, mode, st, num_workgroups);
    if (a.A == 9) return launch_shape<9, 32, float>(a, mode, st, num_workgroups);
  } else {
    if (a.A == 18) return launch_shape<18, 32, uint16_t>(a, mode, st, num_workgroups);
    if (a.A == 9) return launch_shape<9, 64, uint16_t>(a, mode, st, num_workgroups);
  }
  return hipErrorNotSupported;
}

}  // namespace vtrace
