// Long-run tile shapes for float32 logits, A = 9 and A = 18 (the kernel is in
// tiled_impl.hpp).  Event-timed medians at T = 1000 against the 16-step tiles
// (VTRACE_KERNEL=tiled_short):
//   targets-only call: A = 18, 16384 lanes 0.640 -> 0.549 ms, 32768 lanes
//   1.278 -> 1.066 ms; A = 9, 16384 lanes 0.408 -> 0.331 ms, 32768 lanes
//   0.781 -> 0.636 ms;
//   loss call (float64 row sums): A = 18, 16384 lanes 0.808 -> 0.776 ms
//   (32 x 8; 64 x 8 0.782); A = 9, 16384 lanes 0.479 -> 0.450 ms (32 x 8), 32768 lanes
//   0.924 -> 0.851 ms (64 x 4; 32 x 8 0.897, 64 x 8 0.900).
#include "tiled_impl.hpp"

namespace vtrace {

bool launch_tiled_long_f32(const StepArgs& a, Mode mode, hipStream_t st, int64_t* num_workgroups,
                           bool allow_multi, hipError_t* err) {
  // Loss calls: A = 18 32 lanes x 8 steps (2304-byte runs per time row); A = 9
  // 64 x 4 where its tiles make whole generations, else 32 x 8.
  if (mode == Mode::LossGrad) {
    if (a.A == 18) return launch_long_loss<18, float, Shape<32, 8>>(a, st, num_workgroups, err);
    return a.A == 9 && launch_long_loss<9, float, Shape<64, 4>, Shape<32, 8>>(a, st, num_workgroups, err);
  }
  if (a.A == 18)
    return launch_long<18, float, Shape<128, 4>, Shape<64, 8>, Shape<64, 4>>(a, mode, st, num_workgroups,
                                                                            allow_multi, err);
  if (a.A == 9)
    return launch_long<9, float, Shape<128, 4>, Shape<64, 8>, Shape<64, 4>>(a, mode, st, num_workgroups,
                                                                           allow_multi, err);
  return false;
}

}  // namespace vtrace
