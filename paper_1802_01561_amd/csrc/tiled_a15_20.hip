// Tiled V-trace kernel instantiations for A = 15, 16, 17, 19, 20 (16 lanes
// per workgroup, fp32 or bf16 logits); the kernel is in tiled_impl.hpp.
#include "tiled_impl.hpp"

namespace vtrace {

hipError_t launch_tiled_a15_20(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st,
                               int64_t* num_workgroups, bool allow_multi) {
  switch (a.A) {
    case 15: return launch_shape_16<15>(a, lt, mode, st, num_workgroups, allow_multi);
    case 16: return launch_shape_16<16>(a, lt, mode, st, num_workgroups, allow_multi);
    case 17: return launch_shape_16<17>(a, lt, mode, st, num_workgroups, allow_multi);
    case 19: return launch_shape_16<19>(a, lt, mode, st, num_workgroups, allow_multi);
    case 20: return launch_shape_16<20>(a, lt, mode, st, num_workgroups, allow_multi);
    default: return hipErrorNotSupported;
  }
}

}  // namespace vtrace
