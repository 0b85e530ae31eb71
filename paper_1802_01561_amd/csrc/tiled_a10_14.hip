// Tiled V-trace kernel instantiations for A = 10, 11, 12, 13, 14 (16 lanes
// per workgroup, fp32 or bf16 logits); the kernel is in tiled_impl.hpp.
#include "tiled_impl.hpp"

namespace vtrace {

hipError_t launch_tiled_a10_14(const StepArgs& a, LogitsType lt, Mode mode, hipStream_t st,
                               int64_t* num_workgroups, bool allow_multi) {
  switch (a.A) {
    case 10: return launch_shape_16<10>(a, lt, mode, st, num_workgroups, allow_multi);
    case 11: return launch_shape_16<11>(a, lt, mode, st, num_workgroups, allow_multi);
    case 12: return launch_shape_16<12>(a, lt, mode, st, num_workgroups, allow_multi);
    case 13: return launch_shape_16<13>(a, lt, mode, st, num_workgroups, allow_multi);
    case 14: return launch_shape_16<14>(a, lt, mode, st, num_workgroups, allow_multi);
    default: return hipErrorNotSupported;
  }
}

}  // namespace vtrace
