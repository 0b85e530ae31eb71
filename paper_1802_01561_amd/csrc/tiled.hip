// Tiled V-trace kernel: the instantiations for A = 9 and A = 18 and the
// choice of instantiation for every action count (the kernel itself is in
// tiled_impl.hpp).
#include "tiled_impl.hpp"

namespace vtrace {

bool tiled_supported(const StepArgs& a, LogitsType) { return a.A >= 2 && a.A <= kTiledMaxActions; }

// Lanes per workgroup: 16 (256 threads) for A = 9 keeps twice as many
// workgroups in flight for mid-sized batches (a 4096-lane batch fills all 256
// CUs), but once 32-lane tiles cover every CU, fp32 A = 9 takes 32 (1152-byte
// runs, nine 128-byte lines, as for fp32 A = 18): measured at T = 1000, 503 ->
// 436 us for 16384 lanes and 2.00 -> 1.71 ms for 65536, while 4096 lanes
// slow from 133 to 199 us (half the CUs idle).  bf16 A = 9 measured slower
// with 32 lanes at every size and keeps 16.  fp32 A = 18 uses 16 lanes (its
// rows are already 1152 bytes).  bf16 A = 18 is the mirror image of fp32
// A = 9: 32 lanes (1152-byte rows) once the tiles fill every CU twice, 16
// below that (T = 1000: 4096 lanes 252 -> 167 us and 8192 lanes 297 -> 275 us
// with 16; 16384 lanes 593 -> 558 us and 32768 lanes 1.23 -> 1.10 ms with 32),
// and 32 when the whole batch is one tile (one workgroup, whose loss sums need
// no cross-workgroup reduction).
//
// These are the shapes with 16-step chunks.  Batches of A = 9 or 18 that fill
// the chip in whole generations take the long-run shapes of tiled_long_f32.hip
// and tiled_long_bf16.hip first (32 to 128 lanes, chunks of 8 or 4 steps).
constexpr int64_t kTwoRowMinT = 512;

hipError_t launch_tiled(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st,
                        int64_t* num_workgroups, bool allow_multi, bool allow_long) {
  if (allow_long && (a.A == 9 || a.A == 18)) {
    hipError_t err = hipSuccess;
    const bool launched = lt == LogitsType::F32
                              ? launch_tiled_long_f32(a, mode, st, num_workgroups, allow_multi, &err)
                              : launch_tiled_long_bf16(a, mode, st, num_workgroups, allow_multi, &err);
    if (launched) return err;
  }
  // A = 18 batches whose 16-lane tiles give each CU at most one workgroup
  // (B <= 16 x CUs: one wave per SIMD) take 32-step chunks for long unrolls:
  // two waves per SIMD and half as many chunks one after another.  Measured
  // (loss call, fp32 logits, event-timed medians): T = 512, B = 4096 0.147 ->
  // 0.137 ms; T = 1000, B = 4096 0.267 -> 0.248 ms and B = 2048 0.228 ->
  // 0.200 ms.  Not taken for A = 9 (T = 512-768: 2-6% slower) nor for
  // shorter unrolls (T = 100-200: 2-8% slower; the 30-task batch 27.7 ->
  // 29.8 us cold), where a 32-step chunk wastes more of the last one and the
  // latency it hides is not what bounds the call.
  if (allow_long && a.A == 18 && a.T >= kTwoRowMinT) {
    const int cus = compute_units();
    if (cus > 0 && a.B <= 16 * static_cast<int64_t>(cus)) {
      if (lt == LogitsType::F32) return launch_shape<18, 16, float, 32>(a, mode, st, num_workgroups, allow_multi);
      return launch_shape<18, 16, uint16_t, 32>(a, mode, st, num_workgroups, allow_multi);
    }
  }
  if (lt == LogitsType::F32) {
    if (a.A == 18) return launch_shape<18, 16, float>(a, mode, st, num_workgroups, allow_multi);
    if (a.A == 9) {
      const int cus = compute_units();
      if (cus > 0 && a.B >= 32 * static_cast<int64_t>(cus))
        return launch_shape<9, 32, float>(a, mode, st, num_workgroups, allow_multi);
      return launch_shape<9, 16, float>(a, mode, st, num_workgroups, allow_multi);
    }
  } else {
    if (a.A == 18) {
      const int cus = compute_units();
      if (a.B <= 32 || (cus > 0 && a.B >= 64 * static_cast<int64_t>(cus)))
        return launch_shape<18, 32, uint16_t>(a, mode, st, num_workgroups, allow_multi);
      return launch_shape<18, 16, uint16_t>(a, mode, st, num_workgroups, allow_multi);
    }
    if (a.A == 9) return launch_shape<9, 16, uint16_t>(a, mode, st, num_workgroups, allow_multi);
  }
  // The other action counts, 16 lanes per workgroup (instantiated in three
  // more files, which compile in parallel).
  if (a.A >= 2 && a.A <= 8) return launch_tiled_a2_8(a, lt, mode, st, num_workgroups, allow_multi);
  if (a.A >= 10 && a.A <= 14) return launch_tiled_a10_14(a, lt, mode, st, num_workgroups, allow_multi);
  if (a.A >= 15 && a.A <= kTiledMaxActions)
    return launch_tiled_a15_20(a, lt, mode, st, num_workgroups, allow_multi);
  return hipErrorNotSupported;
}

}  // namespace vtrace
