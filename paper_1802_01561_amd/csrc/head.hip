// Fused output layer + V-trace kernel.
//
// The learner applies its fully connected output layer to every step of the
// unroll at once (Sec. 3.1): o = hidden @ W + bias with W: [H, A + 1], whose
// first A outputs are the policy logits and whose last is the baseline V(x_t).
// This kernel runs that layer, the V-trace targets, losses and gradients of
// Sec. 4 on its outputs, and the gradients through the layer, in one pass over
// HBM.  With G = dL/do = [d_logits, d_values]:
//   d_hidden = G W^T,   d_W = sum over (t, b) of hidden^T G,   d_bias = sum of G.
// The three products are dense contractions and run on the matrix cores
// (bfloat16 operands, float32 accumulation).
//
// Work split.  A workgroup has four waves; wave w walks one lane (batch entry)
// backwards in time in chunks of 16 steps, so the reverse recursion stays in
// the wave, and workgroups loop over groups of four consecutive lanes.  In a
// chunk the 16 steps of the wave's lane are the 16 rows of one MFMA tile; lane
// l of the wave is (s, g) = (l % 16, l / 16).
//  1. Forward, o^T = W^T hidden^T with 16x16x32 MFMAs (M: output column, N:
//     step, K: hidden unit).  In K step j, lane (s, g) supplies hidden units
//     32j + 8g .. 32j + 8g + 7 of step s's row, one 16-byte vector: the four
//     lane groups read 64 contiguous bytes of each row per instruction and the
//     next K step the rest of the 128-byte line.  The lane receives
//     o[s][4g + i] (and o[s][16 + 4g + i] when A + 1 > 16), i = 0..3.
//  2. The V-trace epilogue works in that layout.  Row statistics of a step
//     (maxima, exponent sums, the taken action's logit, the baseline) are sums
//     over the four lane groups: two xor shuffles, whose fixed order gives all
//     four groups bit-identical results.  The per-step chain and the suffix
//     scan over the 16 steps then run on each DPP row of 16 lanes; the four
//     rows compute the same values.
//  3. d_hidden^T = W G^T (K: output column).  Each lane's G values are exactly
//     the K slots it must supply, taking the forward's output order as the
//     contraction order, so G enters the MFMA where the epilogue left it.  G
//     is split into bfloat16 high and low parts (hi + lo equals G to within
//     2^-17 relative), two MFMAs, so the product keeps float32 accuracy.  The
//     M rows (hidden units) are ordered so that each store instruction of the
//     four lane groups writes 64 contiguous bytes of a row: for float32 output
//     M tile i gives lane (s, g) units 16i + 4g .. +3, for bfloat16 output M
//     tiles 2p and 2p+1 give it units 32p + 8g .. +7 (one packed vector).
//  4. d_W contracts over steps, which lie across lanes: the hidden tile and G
//     are written to LDS, and after a workgroup barrier wave w accumulates
//     rows [w H/4, (w+1) H/4) of d_W over the four lanes' tiles with 16x16x16
//     MFMAs, in registers, for the whole walk (wave 0 also d_bias, with a ones
//     operand).  A second kernel adds the workgroups' partial sums.
#include <type_traits>

#include "device_common.hpp"
#include "head.hpp"
#include "wave_ops.hpp"

namespace vtrace {
namespace {

constexpr int kL = 16;            // steps per chunk
constexpr int kHeadWaves = 4;     // lanes in flight per workgroup
constexpr int kHeadThreads = kHeadWaves * kWave;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

template <int H, int NT>
struct HeadShape {
  static constexpr int C = 16 * NT;     // output columns covered by the MFMA tiles
  static constexpr int Q = H / 4;       // hidden units each wave's d_W tiles cover
  static constexpr int KS = H / 32;     // forward K steps = 16-byte vectors per lane and row
  static constexpr int MT = H / 16;     // d_hidden M tiles
  static constexpr int MW = H / 64;     // d_W M tiles per wave
  static constexpr int KW = 4 * NT;     // K slots per lane in the d_hidden product
  // LDS row pitches in bfloat16 elements.  W^T rows are 16-byte aligned for
  // the forward's vector reads; the hidden and G rows are 8-byte aligned and
  // padded so that the four lane groups of a transposed read (rows 4 apart)
  // fall on different banks.
  static constexpr int WT_PITCH = H + 8;
  static constexpr int WP_PITCH = (NT == 2) ? 40 : 20;
  static constexpr int HL_PITCH = H + 4;
  static constexpr int GL_PITCH = C + 4;
  static_assert(H % 64 == 0 && H <= 256, "hidden size");
  static_assert(NT == 1 || NT == 2, "column tiles");
};

// K slot of column c in the d_hidden product: the order in which the forward
// product leaves a lane's outputs (columns 4g..4g+3, then 16+4g..16+4g+3).
template <int NT>
__device__ __forceinline__ int slot_of_column(int c) {
  if constexpr (NT == 1) return c;
  const int hi = c >= 16;
  const int cc = c - 16 * hi;
  return 8 * (cc / 4) + 4 * hi + (cc % 4);
}

__device__ __forceinline__ float group_sum(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}
__device__ __forceinline__ double group_sum(double v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}
__device__ __forceinline__ float group_max(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

__device__ __forceinline__ f32x4 mfma_k32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_k16(s16x4 a, s16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Global memory inside the chunk walk goes through raw buffer descriptors.
// A load at an offset beyond the descriptor's size returns zero and a store
// there is dropped, so rows before t = 0, lanes beyond B and outputs the caller
// did not ask for are masked by their offsets or an empty descriptor, with no
// branch around any memory instruction.  That keeps the count of outstanding
// memory operations the same on every path, so the compiler can wait for the
// prefetched loads alone (vmcnt(n)) rather than for every store before them.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRawBufferFlags = 0x00020000;  // raw buffer, 32-bit elements, no swizzle
constexpr uint32_t kOutOfRange = 0xFFFFF000u;  // beyond every descriptor used here

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                           kRawBufferFlags);
}
__device__ __forceinline__ float buffer_load_f32(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
template <typename BehIn>
__device__ __forceinline__ float buffer_load_logit(Rsrc r, uint32_t off) {
  if constexpr (sizeof(BehIn) == 4)
    return buffer_load_f32(r, off);
  else
    return logit_to_float(static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0)));
}
__device__ __forceinline__ void buffer_store_f32(float x, Rsrc r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), r, off, 0, 0);
}

template <int H, int NT, bool kPrecise, typename BehIn, bool kBf16Grad>
__global__ __launch_bounds__(kHeadThreads, 2) void head_kernel(HeadArgs a) {
  using S = HeadShape<H, NT>;
  constexpr int C = S::C, Q = S::Q;
  __shared__ __align__(16) uint16_t s_wt[C * S::WT_PITCH];        // W^T [C][H]
  __shared__ __align__(16) uint16_t s_wp[H * S::WP_PITCH];        // W [H][K slot]
  __shared__ __align__(16) uint16_t s_h[kHeadWaves * kL * S::HL_PITCH];  // hidden tiles
  __shared__ __align__(16) uint16_t s_ghi[kHeadWaves * kL * S::GL_PITCH];
  __shared__ __align__(16) uint16_t s_glo[kHeadWaves * kL * S::GL_PITCH];
  __shared__ double s_red[3 * kHeadWaves];
  __shared__ float s_bias[C];
  __shared__ float s_db[C];  // wave 0's running d_bias

  const int tid = threadIdx.x;
  // The wave index, stated as wave-uniform so that lane numbers and buffer
  // descriptors derived from it live in scalar registers.
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int l = tid % kWave;
  const int s = l % kL;  // step within the chunk (and row of MFMA operands)
  const int g = l / kL;  // lane group
  const int64_t T = a.T, B = a.B, A = a.A;
  const int A1 = static_cast<int>(A) + 1;

  // The layer's weights, twice: W^T for the forward, W in K-slot order for
  // d_hidden.  Columns beyond the baseline are zero.
  for (int i = tid; i < H * C; i += kHeadThreads) {
    const int h = i / C, c = i % C;
    const uint16_t v = c < A1 ? a.weight[static_cast<int64_t>(h) * A1 + c] : uint16_t(0);
    s_wt[c * S::WT_PITCH + h] = v;
    s_wp[h * S::WP_PITCH + slot_of_column<NT>(c)] = v;
  }
  if (tid < C) {
    s_bias[tid] = tid < A1 ? a.bias[tid] : 0.0f;
    s_db[tid] = 0.0f;
  }
  __syncthreads();

  const bool beh_lp = a.behaviour_log_probs != 0;
  const bool no_ratio = a.correction == kCorrNone || a.correction == kCorrEpsilon;
  const bool use_y = !beh_lp && !no_ratio;
  const double rho_bar = a.rho_bar, c_bar = a.c_bar, lam = a.lambda;
  const float ce = a.entropy_cost;
  const int nchunks = static_cast<int>((T + kL - 1) / kL);
  // Byte strides of one time row and the byte size of a chunk's 16 rows, per
  // array (the host checks that these windows fit 32-bit offsets).
  constexpr uint32_t gsz = kBf16Grad ? 2u : 4u;
  const uint32_t row_h = static_cast<uint32_t>(B * H * 2);
  const uint32_t row_d = static_cast<uint32_t>(B * H) * gsz;
  const uint32_t row_s = static_cast<uint32_t>(B * 4);
  const uint32_t row_y = static_cast<uint32_t>(B * A * sizeof(BehIn));
  const uint32_t row_o = static_cast<uint32_t>(B * A1 * 4);
  // A descriptor over a chunk's rows of a [T, B, n] array, starting at lane
  // b of the chunk's first existing row and cut at the array's end, so that
  // no offset it accepts lies outside the array.
  auto chunk_rsrc = [&](const void* arr, int64_t n, int64_t elem_bytes, int64_t brow, bool on) {
    const int64_t begin = brow * n * elem_bytes;
    int64_t bytes = static_cast<int64_t>(kL) * B * n * elem_bytes;
    const int64_t left = T * B * n * elem_bytes - begin;
    bytes = bytes < left ? bytes : left;
    return make_rsrc(static_cast<const char*>(arr) + (on ? begin : 0), on ? static_cast<uint32_t>(bytes) : 0u);
  };
  const int64_t nquads = (B + kHeadWaves - 1) / kHeadWaves;

  f32x4 acc_w[S::MW][NT];
  static_for<NT>([&](auto CT) {
    constexpr int ct = decltype(CT)::value;
    static_for<S::MW>([&](auto MI) { acc_w[decltype(MI)::value][ct] = f32x4{0.f, 0.f, 0.f, 0.f}; });
  });
  double wave_pg = 0.0, wave_base = 0.0, wave_ent = 0.0;

  for (int64_t quad = xcd_tile(blockIdx.x, gridDim.x); quad < nquads; quad += gridDim.x) {
    const int64_t b = quad * kHeadWaves + w;
    const bool lane_ok = b < B;
    const double boot = lane_ok ? static_cast<double>(a.bootstrap_value[b]) : 0.0;
    double cy_V = boot, cy_v = boot, cy_A = 0.0;
    double l_pg = 0.0, l_base = 0.0, l_ent = 0.0;
    bool bad_action = false;

    // Register prefetch of one chunk: this lane's hidden slice, behaviour
    // values and per-step scalars.
    v4u hreg[S::KS];
    float yreg[NT][4];
    int32_t p_act = 0;
    float p_r = 0.f, p_g = 0.f, p_lmu = 0.f;
    // Descriptors of a chunk start at its first existing row (wave-uniform);
    // lane s of the row group reads row t0 + s at offset rel * row stride.
    auto prefetch = [&](int k) {
      const int64_t t0 = T - static_cast<int64_t>(k + 1) * kL;
      const int64_t tb = t0 < 0 ? 0 : t0;
      const bool row_ok = t0 + s >= 0;
      const uint32_t rel = static_cast<uint32_t>(t0 + s - tb);
      const int64_t brow = tb * B + b;
      const Rsrc rh = chunk_rsrc(a.hidden, H, 2, brow, lane_ok);
      const uint32_t oh = row_ok ? rel * row_h + 16u * g : kOutOfRange;
      static_for<S::KS>([&](auto J) {
        constexpr int j = decltype(J)::value;
        hreg[j] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rh, oh + 64 * j, 0, 0));
      });
      const uint32_t os = row_ok ? rel * row_s : kOutOfRange;
      p_act = static_cast<int32_t>(
          __builtin_amdgcn_raw_buffer_load_b32(chunk_rsrc(a.actions, 1, 4, brow, lane_ok), os, 0, 0));
      p_r = buffer_load_f32(chunk_rsrc(a.rewards, 1, 4, brow, lane_ok), os);
      p_g = buffer_load_f32(chunk_rsrc(a.discounts, 1, 4, brow, lane_ok), os);
      p_lmu = buffer_load_f32(chunk_rsrc(a.behaviour, 1, 4, brow, lane_ok && beh_lp && !no_ratio), os);
      // Behaviour logits: one offset per lane, the columns in the instruction
      // offset.  Columns >= A (the tiles' padding) get an offset beyond the
      // descriptor, so they read nothing (they would be the next lane's row).
      const Rsrc ry = chunk_rsrc(a.behaviour, A, sizeof(BehIn), brow, lane_ok && use_y);
      const uint32_t oy = row_ok ? rel * row_y + 4u * g * static_cast<uint32_t>(sizeof(BehIn)) : kOutOfRange;
      static_for<NT>([&](auto CT) {
        constexpr int ct = decltype(CT)::value;
        static_for<4>([&](auto I) {
          constexpr int i = decltype(I)::value;
          const bool col_ok = 16 * ct + 4 * g + i < A;
          yreg[ct][i] = buffer_load_logit<BehIn>(ry, col_ok ? oy + (16 * ct + i) * sizeof(BehIn) : kOutOfRange);
        });
      });
    };

    prefetch(0);
    // Wait for the first chunk here, once per lane: the loop's first use of
    // the prefetched registers is then reached from the loop entry with
    // nothing outstanding, and the compiler's wait there only has to cover
    // the previous iteration's loads, not the stores issued after them.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    for (int k = 0; k < nchunks; ++k) {
      const int64_t t0 = T - static_cast<int64_t>(k + 1) * kL;
      const int64_t t = t0 + s;
      const bool step_ok = lane_ok && t >= 0;
      const int64_t tb = t0 < 0 ? 0 : t0;
      const uint32_t rel = static_cast<uint32_t>(t - tb);
      const int64_t brow = tb * B + b;

      // 1. Forward product, from the prefetched hidden slice.
      f32x4 oacc[NT];
      static_for<NT>([&](auto CT) { oacc[decltype(CT)::value] = f32x4{0.f, 0.f, 0.f, 0.f}; });
      static_for<S::KS>([&](auto J) {
        constexpr int j = decltype(J)::value;
        const bf16x8 hv = __builtin_bit_cast(bf16x8, hreg[j]);
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          const bf16x8 wv =
              *reinterpret_cast<const bf16x8*>(&s_wt[(16 * ct + s) * S::WT_PITCH + 32 * j + 8 * g]);
          oacc[ct] = mfma_k32(wv, hv, oacc[ct]);
        });
      });
      // The hidden slice goes to LDS for d_W (the previous chunk's readers
      // finished at its closing barrier).
      {
        uint16_t* hrow = s_h + (kL * w + s) * S::HL_PITCH + 8 * g;
        static_for<S::KS>([&](auto J) {
          constexpr int j = decltype(J)::value;
          reinterpret_cast<uint2*>(hrow + 32 * j)[0] = uint2{hreg[j].x, hreg[j].y};
          reinterpret_cast<uint2*>(hrow + 32 * j)[1] = uint2{hreg[j].z, hreg[j].w};
        });
      }
      int32_t act = p_act;
      float r32 = p_r, g32 = p_g;
      const float lmu = p_lmu;
      if (!step_ok) act = 0;  // rows that do not exist carry a harmless action
      const bool act_ok = act >= 0 && act < A;
      const int act_c = act_ok ? act : 0;
      bad_action = bad_action || !act_ok;
      // Behaviour-policy statistics of the step, taken before the prefetch
      // below reuses their registers: m_y = max_j y_j, s_y = sum_j exp(y_j - m_y)
      // and y_a.
      using SumT = std::conditional_t<kPrecise, double, float>;
      float my = 0.f, ya = 0.f;
      SumT sy = 0;
      if (use_y) {
        float ymax = -INFINITY, yal = 0.f;
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          for (int i = 0; i < 4; ++i) {
            const int c = 16 * ct + 4 * g + i;
            if (c < A) ymax = fmaxf(ymax, yreg[ct][i]);
            if (c == act_c) yal = yreg[ct][i];
          }
        });
        my = group_max(ymax);
        ya = group_sum(yal);
        SumT syl = 0;
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          for (int i = 0; i < 4; ++i) {
            if (16 * ct + 4 * g + i < A) {
              if constexpr (kPrecise)
                syl += exp_nonpos_f64(static_cast<double>(yreg[ct][i]) - static_cast<double>(my));
              else
                syl += exp_fast(yreg[ct][i] - my);
            }
          }
        });
        sy = group_sum(syl);
      }
      // The next chunk's loads go out at raised wave priority, ahead of the
      // other wave's matrix products on the same SIMD: 6.64-6.65 -> 6.25-6.26
      // ms at the stress shape with float32 d_hidden; with bf16 d_hidden it
      // measured 0.6% slower and keeps normal priority.
      if (k + 1 < nchunks) {
        if constexpr (!kBf16Grad) __builtin_amdgcn_s_setprio(2);
        prefetch(k + 1);
        if constexpr (!kBf16Grad) __builtin_amdgcn_s_setprio(0);
      }

      // 2. Epilogue.
      r32 = transform_reward(r32, a.reward_transform);

      float o[NT][4];
      float zmax = -INFINITY, vloc = 0.f, zaloc = 0.f;
      static_for<NT>([&](auto CT) {
        constexpr int ct = decltype(CT)::value;
        for (int i = 0; i < 4; ++i) {
          const int c = 16 * ct + 4 * g + i;
          o[ct][i] = oacc[ct][i] + s_bias[c];
          if (c < A) zmax = fmaxf(zmax, o[ct][i]);
          if (c == A) vloc = o[ct][i];
          if (c == act_c) zaloc = o[ct][i];
        }
      });
      {
        const Rsrc ro = chunk_rsrc(a.outputs, A1, 4, brow, lane_ok && a.outputs);
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          static_for<4>([&](auto I) {
            constexpr int i = decltype(I)::value;
            const int c = 16 * ct + 4 * g + i;
            buffer_store_f32(o[ct][i], ro, (step_ok && c < A1) ? rel * row_o + 4u * c : kOutOfRange);
          });
        });
      }
      const float V32 = group_sum(vloc);
      const float mz = group_max(zmax);
      const float za = group_sum(zaloc);

      float e[NT][4];
      double ratio;
      float inv_s, log_s, one_minus_pa, e_a, ed;
      if constexpr (kPrecise) {
        double szl = 0.0;
        float edl = 0.f;
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          for (int i = 0; i < 4; ++i) {
            const int c = 16 * ct + 4 * g + i;
            e[ct][i] = 0.f;
            if (c < A) {
              const double d = static_cast<double>(o[ct][i]) - static_cast<double>(mz);
              const double x = exp_nonpos_f64(d);
              szl += x;
              e[ct][i] = static_cast<float>(x);
              edl = fmaf(e[ct][i], static_cast<float>(d), edl);
            }
          }
        });
        const double sz = group_sum(szl);
        ed = group_sum(edl);
        const double inv = 1.0 / sz;
        const double dza = static_cast<double>(za) - static_cast<double>(mz);
        const double ea = exp_nonpos_f64(dza);
        if (no_ratio) {
          ratio = act_ok ? 1.0 : NAN;
        } else if (beh_lp) {
          ratio = act_ok ? exp(dza - log(sz) - static_cast<double>(lmu)) : NAN;
        } else {
          ratio = act_ok ? exp(dza - (static_cast<double>(ya) - static_cast<double>(my))) * (sy * inv) : NAN;
        }
        inv_s = static_cast<float>(inv);
        log_s = static_cast<float>(log(sz));
        one_minus_pa = static_cast<float>((sz - ea) * inv);
        e_a = static_cast<float>(ea);
      } else {
        float szl = 0.f, edl = 0.f;
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          for (int i = 0; i < 4; ++i) {
            const int c = 16 * ct + 4 * g + i;
            e[ct][i] = 0.f;
            if (c < A) {
              const float d = o[ct][i] - mz;
              e[ct][i] = exp_fast(d);
              szl += e[ct][i];
              edl = fmaf(e[ct][i], d, edl);
            }
          }
        });
        const float sz = group_sum(szl);
        ed = group_sum(edl);
        const float inv = __builtin_amdgcn_rcpf(sz);
        const float ea = exp_fast(za - mz);
        log_s = __logf(sz);
        if (no_ratio) {
          ratio = act_ok ? 1.0 : NAN;
        } else if (beh_lp) {
          ratio = act_ok ? static_cast<double>(exp_fast((za - mz) - log_s - lmu)) : NAN;
        } else {
          ratio = act_ok ? static_cast<double>(exp_fast((za - mz) - (ya - my)) * (sy * inv)) : NAN;
        }
        inv_s = inv;
        one_minus_pa = (sz - ea) * inv;
        e_a = ea;
      }
      const float Hent = log_s - ed * inv_s;  // entropy of pi at this step

      const StepWeights wts = variant_weights(a.correction, clip_above(ratio, rho_bar),
                                              lam * clip_above(ratio, c_bar), lam, act_ok);
      const double r = r32, gm = g32, V = V32;
      double V_next = dpp_f64<kRowShl1>(V);
      if (s == kL - 1) V_next = cy_V;
      const double delta = wts.rho_v * (r + gm * V_next - V);
      // Suffix scan of the affine maps v_t - V_t = delta_t + gamma_t c_t (v_{t+1} - V_{t+1})
      // (Remark 1) over the row, the later chunk's carry folded into step 15.
      double Gs = gm * wts.c_v, D = delta;
      if (s == kL - 1) D = fma(Gs, cy_A, D);
      static_for<4>([&](auto I) {
        constexpr int off = 1 << decltype(I)::value;
        const double Gn = dpp_f64<0x100 + off>(Gs);
        const double Dn = dpp_f64<0x100 + off>(D);
        if (s + off < kL) {
          D = fma(Gs, Dn, D);
          Gs = Gs * Gn;
        }
      });
      const double A_t = D;
      const double v_t = V + A_t;
      double v_next = dpp_f64<kRowShl1>(v_t);
      if (s == kL - 1) v_next = cy_v;
      const double q_next = a.q_estimate == kQBaseline ? V_next : v_next;
      const double adv = wts.rho_pg * (r + gm * q_next - V);
      cy_A = dpp_f64<kRowShr15>(A_t);
      cy_v = dpp_f64<kRowShr15>(v_t);
      cy_V = dpp_f64<kRowShr15>(V);

      {
        const uint32_t o1 = (step_ok && g == 0) ? rel * row_s : kOutOfRange;
        buffer_store_f32(static_cast<float>(v_t), chunk_rsrc(a.vs, 1, 4, brow, lane_ok && a.vs), o1);
        buffer_store_f32(static_cast<float>(adv), chunk_rsrc(a.pg_adv, 1, 4, brow, lane_ok && a.pg_adv), o1);
      }

      // G = dL/do for this step: the policy-logit gradient of the plain loss
      // (e_j (alpha + beta z_j) off the taken action), then d_values.
      const float Kz = mz + log_s - Hent;
      const float pa = e_a * inv_s;
      const bool eps_mode = a.correction == kCorrEpsilon;
      const float pg_w = eps_mode ? pa / (pa + a.epsilon) : 1.0f;
      const float adv32 = static_cast<float>(adv) * pg_w;
      const float beta = inv_s * ce;
      const float alpha = inv_s * adv32 - beta * Kz;
      const float out_a = -adv32 * one_minus_pa + ce * pa * (za - Kz);
      const float dval = static_cast<float>(a.baseline_cost * (V - v_t));
      float Gv[NT][4];
      static_for<NT>([&](auto CT) {
        constexpr int ct = decltype(CT)::value;
        for (int i = 0; i < 4; ++i) {
          const int c = 16 * ct + 4 * g + i;
          float x = 0.f;
          if (c < A) x = (c == act_c) ? (act_ok ? out_a : NAN) : e[ct][i] * fmaf(beta, o[ct][i], alpha);
          if (c == A) x = dval;
          Gv[ct][i] = step_ok ? x : 0.f;
        }
      });
      if (step_ok && g == 0) {
        // log pi(a), and for the epsilon-correction log(pi(a) + eps) as the
        // float64 log-sum of log pi(a) and log eps: pi(a) + eps rounded to
        // float32 would lose eps near pi(a) = 1 (1 + 1e-6 is 1.00000095 there).
        const double lp = static_cast<double>(za - mz) - static_cast<double>(log_s);
        double log_pa = lp;
        if (eps_mode) {
          const double le = log(static_cast<double>(a.epsilon));
          log_pa = lp >= le ? lp + log1p(exp(le - lp)) : le + log1p(exp(lp - le));
        }
        if (!act_ok) log_pa = NAN;
        l_pg += -adv * log_pa;
        l_base += 0.5 * A_t * A_t;
        l_ent += -static_cast<double>(Hent);
      }

      // 3. d_hidden = G W^T.  For float32 output M tile i gives lane (s, g)
      // units 16i + 4g .. +3 of its step's row (one 16-byte store); for
      // bfloat16, M tiles 2p and 2p+1 give it units 32p + 8g .. +7 (packed
      // into one 16-byte store).  Either way the four lane groups write 64
      // contiguous bytes of each row per instruction.
      const int grow = (kL * w + s) * S::GL_PITCH;
      const uint32_t od = step_ok ? rel * row_d : kOutOfRange;
      const Rsrc rd = chunk_rsrc(a.d_hidden, H, gsz, brow, lane_ok);
      // M row (hidden unit) that operand lane s supplies in M tile i.
      auto m_row = [&](int i) {
        return kBf16Grad ? 32 * (i / 2) + 8 * (s / 4) + 4 * (i % 2) + (s % 4) : 16 * i + s;
      };
      f32x4 prev = {0.f, 0.f, 0.f, 0.f};
      auto store_dh = [&](f32x4 acc, int i) {
        if constexpr (!kBf16Grad) {
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, acc), rd,
                                                 od + 4u * (16u * i + 4u * g), 0, 0);
        } else {
          if (i % 2 == 1) {
            const v4u pk = {pack_bf16x2(prev[0], prev[1]), pack_bf16x2(prev[2], prev[3]),
                            pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
            __builtin_amdgcn_raw_buffer_store_b128(pk, rd, od + 2u * (32u * (i / 2) + 8u * g), 0, 0);
          }
          prev = acc;
        }
      };
      if constexpr (NT == 2) {
        const f32x8 gf = {Gv[0][0], Gv[0][1], Gv[0][2], Gv[0][3],
                          Gv[1][0], Gv[1][1], Gv[1][2], Gv[1][3]};
        const bf16x8 ghi = __builtin_convertvector(gf, bf16x8);
        const bf16x8 glo = __builtin_convertvector(gf - __builtin_convertvector(ghi, f32x8), bf16x8);
        const v4u uhi = __builtin_bit_cast(v4u, ghi), ulo = __builtin_bit_cast(v4u, glo);
        reinterpret_cast<uint2*>(s_ghi + grow + 4 * g)[0] = uint2{uhi.x, uhi.y};
        reinterpret_cast<uint2*>(s_ghi + grow + 16 + 4 * g)[0] = uint2{uhi.z, uhi.w};
        reinterpret_cast<uint2*>(s_glo + grow + 4 * g)[0] = uint2{ulo.x, ulo.y};
        reinterpret_cast<uint2*>(s_glo + grow + 16 + 4 * g)[0] = uint2{ulo.z, ulo.w};
        static_for<S::MT>([&](auto I) {
          constexpr int i = decltype(I)::value;
          const bf16x8 wv = *reinterpret_cast<const bf16x8*>(&s_wp[m_row(i) * S::WP_PITCH + 8 * g]);
          f32x4 acc = mfma_k32(wv, ghi, f32x4{0.f, 0.f, 0.f, 0.f});
          acc = mfma_k32(wv, glo, acc);
          store_dh(acc, i);
        });
      } else {
        const f32x4 gf = {Gv[0][0], Gv[0][1], Gv[0][2], Gv[0][3]};
        const bf16x4 ghi = __builtin_convertvector(gf, bf16x4);
        const bf16x4 glo = __builtin_convertvector(gf - __builtin_convertvector(ghi, f32x4), bf16x4);
        const s16x4 shi = __builtin_bit_cast(s16x4, ghi), slo = __builtin_bit_cast(s16x4, glo);
        reinterpret_cast<s16x4*>(s_ghi + grow + 4 * g)[0] = shi;
        reinterpret_cast<s16x4*>(s_glo + grow + 4 * g)[0] = slo;
        static_for<S::MT>([&](auto I) {
          constexpr int i = decltype(I)::value;
          const s16x4 wv = *reinterpret_cast<const s16x4*>(&s_wp[m_row(i) * S::WP_PITCH + 4 * g]);
          f32x4 acc = mfma_k16(wv, shi, f32x4{0.f, 0.f, 0.f, 0.f});
          acc = mfma_k16(wv, slo, acc);
          store_dh(acc, i);
        });
      }

      // 4. d_W and d_bias over the four lanes' tiles of this chunk.
      __syncthreads();
      f32x4 db[NT];
      static_for<NT>([&](auto CT) { db[decltype(CT)::value] = f32x4{0.f, 0.f, 0.f, 0.f}; });
      static_for<kHeadWaves>([&](auto QI) {
        constexpr int q = decltype(QI)::value;
        s16x4 bh[NT], bl[NT];
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          for (int rr = 0; rr < 4; ++rr) {
            const int idx = (kL * q + 4 * g + rr) * S::GL_PITCH + 16 * ct + s;
            bh[ct][rr] = static_cast<short>(s_ghi[idx]);
            bl[ct][rr] = static_cast<short>(s_glo[idx]);
          }
        });
        static_for<S::MW>([&](auto MI) {
          constexpr int mi = decltype(MI)::value;
          const int hb = w * Q + 16 * mi;
          s16x4 ah;
          for (int rr = 0; rr < 4; ++rr)
            ah[rr] = static_cast<short>(s_h[(kL * q + 4 * g + rr) * S::HL_PITCH + hb + s]);
          static_for<NT>([&](auto CT) {
            constexpr int ct = decltype(CT)::value;
            acc_w[mi][ct] = mfma_k16(ah, bh[ct], acc_w[mi][ct]);
            acc_w[mi][ct] = mfma_k16(ah, bl[ct], acc_w[mi][ct]);
          });
        });
        if (w == 0) {
          const s16x4 ones = {0x3F80, 0x3F80, 0x3F80, 0x3F80};  // bfloat16 1.0
          static_for<NT>([&](auto CT) {
            constexpr int ct = decltype(CT)::value;
            db[ct] = mfma_k16(ones, bh[ct], db[ct]);
            db[ct] = mfma_k16(ones, bl[ct], db[ct]);
          });
        }
      });
      // Wave 0 adds the chunk's column sums to its running d_bias (one lane
      // per column, so the order of additions is fixed).
      if (w == 0 && g == 0) {
        static_for<NT>([&](auto CT) {
          constexpr int ct = decltype(CT)::value;
          s_db[16 * ct + s] += db[ct][0];
        });
      }
      __syncthreads();
    }

    if (bad_action) raise_error_flag(a.error_flag);

    // This lane's loss sums (lanes of group 0 hold them), in a fixed order.
#pragma unroll
    for (int off = kL / 2; off > 0; off >>= 1) {
      l_pg += __shfl_xor(l_pg, off, kL);
      l_base += __shfl_xor(l_base, off, kL);
      l_ent += __shfl_xor(l_ent, off, kL);
    }
    l_base *= a.baseline_cost;
    l_ent *= a.entropy_cost;
    if (l == 0 && lane_ok) {
      if (a.lane_losses) {
        a.lane_losses[3 * b + 0] = static_cast<float>(l_pg);
        a.lane_losses[3 * b + 1] = static_cast<float>(l_base);
        a.lane_losses[3 * b + 2] = static_cast<float>(l_ent);
      }
      wave_pg += l_pg;
      wave_base += l_base;
      wave_ent += l_ent;
    }
  }

  // Partial sums of this workgroup: d_W rows [w H/4, (w+1) H/4), d_bias, losses.
  float* part = a.grad_partials + static_cast<size_t>(blockIdx.x) * (H + 1) * C;
  static_for<S::MW>([&](auto MI) {
    constexpr int mi = decltype(MI)::value;
    static_for<NT>([&](auto CT) {
      constexpr int ct = decltype(CT)::value;
      for (int jj = 0; jj < 4; ++jj)
        part[(w * Q + 16 * mi + 4 * g + jj) * C + 16 * ct + s] = acc_w[mi][ct][jj];
    });
  });
  if (w == 0 && g == 0) {
    static_for<NT>([&](auto CT) {
      constexpr int ct = decltype(CT)::value;
      part[H * C + 16 * ct + s] = s_db[16 * ct + s];
    });
  }
  if (l == 0) {
    s_red[3 * w + 0] = wave_pg;
    s_red[3 * w + 1] = wave_base;
    s_red[3 * w + 2] = wave_ent;
  }
  __syncthreads();
  if (tid == 0) {
    double p0 = 0.0, p1 = 0.0, p2 = 0.0;
    for (int i = 0; i < kHeadWaves; ++i) {
      p0 += s_red[3 * i + 0];
      p1 += s_red[3 * i + 1];
      p2 += s_red[3 * i + 2];
    }
    double* lp = a.loss_partials + 3 * static_cast<size_t>(blockIdx.x);
    lp[0] = p0;
    lp[1] = p1;
    lp[2] = p2;
  }
}

// Adds the workgroups' partial sums in a fixed order (float64): d_W, d_bias and
// the loss totals.  Block i covers 64 outputs; each of its 16 waves sums the
// workgroups k = wave, wave + 16, ... (one coalesced 256-byte row per step),
// and the 16 wave sums are added in wave order.
constexpr int kFinishOutputs = 64;
constexpr int kFinishWaves = 16;
__global__ __launch_bounds__(kFinishWaves* kWave) void head_finish_kernel(HeadArgs a, int C, int nwg) {
  __shared__ double s_q[kFinishWaves][kFinishOutputs];
  const int64_t H = a.H;
  const int A1 = static_cast<int>(a.A) + 1;
  const int64_t n_w = H * A1;
  const int64_t n_out = n_w + A1;
  const int wv = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kFinishOutputs + lane;
  const size_t stride = static_cast<size_t>(H + 1) * C;
  size_t off = 0;
  if (i < n_w)
    off = static_cast<size_t>(i / A1) * C + static_cast<size_t>(i % A1);
  else if (i < n_out)
    off = static_cast<size_t>(H) * C + static_cast<size_t>(i - n_w);
  double sum = 0.0;
  if (i < n_out) {
    // Unrolled so that several rows' loads are in flight; the additions keep
    // their order.
#pragma unroll 8
    for (int k = wv; k < nwg; k += kFinishWaves) sum += static_cast<double>(a.grad_partials[k * stride + off]);
  }
  s_q[wv][lane] = sum;
  __syncthreads();
  if (wv == 0 && i < n_out) {
    double tot = 0.0;
    for (int q = 0; q < kFinishWaves; ++q) tot += s_q[q][lane];
    if (i < n_w)
      a.d_weight[i] = static_cast<float>(tot);
    else
      a.d_bias[i - n_w] = static_cast<float>(tot);
  }
  if (blockIdx.x == 0) {
    // Loss totals: each thread adds the workgroups k = thread, thread + 1024,
    // ..., then a fixed-order block reduction.
    __shared__ double s_red[3 * kFinishWaves];
    double p0 = 0.0, p1 = 0.0, p2 = 0.0;
    for (int k = threadIdx.x; k < nwg; k += kFinishWaves * kWave) {
      p0 += a.loss_partials[3 * k + 0];
      p1 += a.loss_partials[3 * k + 1];
      p2 += a.loss_partials[3 * k + 2];
    }
    block_sum3<kFinishWaves * kWave>(p0, p1, p2, s_red);
    if (threadIdx.x == 0) {
      a.losses[0] = static_cast<float>(p0 + p1 + p2);
      a.losses[1] = static_cast<float>(p0);
      a.losses[2] = static_cast<float>(p1);
      a.losses[3] = static_cast<float>(p2);
    }
  }
}

template <int H, int NT, typename BehIn, bool kBf16Grad>
void launch_head_grad(const HeadArgs& a, hipStream_t st, unsigned nwg) {
  if (ratio_needs_fp64(a))
    hipLaunchKernelGGL((head_kernel<H, NT, true, BehIn, kBf16Grad>), dim3(nwg), dim3(kHeadThreads), 0, st, a);
  else
    hipLaunchKernelGGL((head_kernel<H, NT, false, BehIn, kBf16Grad>), dim3(nwg), dim3(kHeadThreads), 0, st, a);
}

template <int H, int NT, typename BehIn>
void launch_head_shape(const HeadArgs& a, hipStream_t st, unsigned nwg) {
  if (a.grad_bf16)
    launch_head_grad<H, NT, BehIn, true>(a, st, nwg);
  else
    launch_head_grad<H, NT, BehIn, false>(a, st, nwg);
}

template <int H>
void launch_head_h(const HeadArgs& a, hipStream_t st, unsigned nwg) {
  const bool two = a.A + 1 > 16;
  if (a.behaviour_bf16) {
    if (two) launch_head_shape<H, 2, uint16_t>(a, st, nwg);
    else launch_head_shape<H, 1, uint16_t>(a, st, nwg);
  } else {
    if (two) launch_head_shape<H, 2, float>(a, st, nwg);
    else launch_head_shape<H, 1, float>(a, st, nwg);
  }
}

int head_columns(int64_t A) { return A + 1 > 16 ? 32 : 16; }

}  // namespace

bool head_hidden_supported(int64_t H) { return H == 64 || H == 128 || H == 256; }

int64_t head_workgroups(int64_t B) {
  const int64_t quads = (B + kHeadWaves - 1) / kHeadWaves;
  return quads < kHeadMaxWorkgroups ? quads : kHeadMaxWorkgroups;
}

namespace {
size_t head_loss_bytes(int64_t B) {
  const size_t n = 3 * sizeof(double) * static_cast<size_t>(head_workgroups(B));
  return (n + 255) / 256 * 256;
}
}  // namespace

size_t head_workspace_bytes(int64_t B, int64_t A, int64_t H) {
  return kWsHeaderBytes + head_loss_bytes(B) +
         sizeof(float) * static_cast<size_t>(head_workgroups(B)) * static_cast<size_t>(H + 1) *
             static_cast<size_t>(head_columns(A));
}

void head_attach_workspace(HeadArgs* a, void* ws) {
  char* base = static_cast<char*>(ws);
  a->error_flag = reinterpret_cast<unsigned int*>(base + kWsFlagOffset);
  a->loss_partials = reinterpret_cast<double*>(base + kWsHeaderBytes);
  a->grad_partials = reinterpret_cast<float*>(base + kWsHeaderBytes + head_loss_bytes(a->B));
}

hipError_t launch_head(const HeadArgs& a, hipStream_t st) {
  const int64_t nwg = head_workgroups(a.B);
  const unsigned n = static_cast<unsigned>(nwg);
  if (a.H == 64) launch_head_h<64>(a, st, n);
  else if (a.H == 128) launch_head_h<128>(a, st, n);
  else if (a.H == 256) launch_head_h<256>(a, st, n);
  else return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n_out = a.H * (a.A + 1) + (a.A + 1);
  const unsigned fb = static_cast<unsigned>((n_out + kFinishOutputs - 1) / kFinishOutputs);
  hipLaunchKernelGGL(head_finish_kernel, dim3(fb), dim3(kFinishWaves * kWave), 0, st, a, head_columns(a.A),
                     static_cast<int>(nwg));
  return hipGetLastError();
}

}  // namespace vtrace
