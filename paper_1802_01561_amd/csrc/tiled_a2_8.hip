// Tiled V-trace kernel instantiations for A = 2, 3, 4, 5, 6, 7, 8 (16 lanes
// per workgroup, fp32 or bf16 logits); the kernel is in tiled_impl.hpp.
#include "tiled_impl.hpp"

namespace vtrace {

hipError_t launch_tiled_a2_8(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st,
                             int64_t* num_workgroups, bool allow_multi) {
  switch (a.A) {
    case 2: return launch_shape_16<2>(a, lt, mode, st, num_workgroups, allow_multi);
    case 3: return launch_shape_16<3>(a, lt, mode, st, num_workgroups, allow_multi);
    case 4: return launch_shape_16<4>(a, lt, mode, st, num_workgroups, allow_multi);
    case 5: return launch_shape_16<5>(a, lt, mode, st, num_workgroups, allow_multi);
    case 6: return launch_shape_16<6>(a, lt, mode, st, num_workgroups, allow_multi);
    case 7: return launch_shape_16<7>(a, lt, mode, st, num_workgroups, allow_multi);
    case 8: return launch_shape_16<8>(a, lt, mode, st, num_workgroups, allow_multi);
    default: return hipErrorNotSupported;
  }
}

}  // namespace vtrace
