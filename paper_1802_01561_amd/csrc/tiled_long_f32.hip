// Long-run tile shapes for float32 logits, A = 9 and A = 18 (the kernel is in
// tiled_impl.hpp).  Measured at T = 1000 against the 16-step tiles: A = 18,
// 16384 lanes 0.762 -> 0.707 ms (64 lanes x 8 steps), 32768 lanes 1.61 ->
// 1.44 ms (128 x 4), 65536 lanes 3.09 -> 2.95 ms (64 x 4, multi-tile walk);
// A = 9, 16384 lanes 0.448 -> 0.391 ms, 32768 lanes 0.867 -> 0.777 ms.
#include "tiled_impl.hpp"

namespace vtrace {

bool launch_tiled_long_f32(const StepArgs& a, Mode mode, hipStream_t st, int64_t* num_workgroups,
                           bool allow_multi, hipError_t* err) {
  // Loss calls with A = 18: 32 lanes x 8 steps (2304-byte runs per time row).
  if (mode == Mode::LossGrad) return a.A == 18 && launch_long_loss<18, float, Shape<32, 8>>(a, st, num_workgroups, err);
  if (a.A == 18)
    return launch_long<18, float, Shape<128, 4>, Shape<64, 8>, Shape<64, 4>>(a, mode, st, num_workgroups,
                                                                            allow_multi, err);
  if (a.A == 9)
    return launch_long<9, float, Shape<128, 4>, Shape<64, 8>, Shape<64, 4>>(a, mode, st, num_workgroups,
                                                                           allow_multi, err);
  return false;
}

}  // namespace vtrace
