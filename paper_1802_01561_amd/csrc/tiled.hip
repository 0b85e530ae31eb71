// Tiled V-trace kernel (not yet enabled).
#include "device_common.hpp"

namespace vtrace {

bool tiled_supported(const StepArgs&, LogitsType) { return false; }

hipError_t launch_tiled(const StepArgs&, LogitsType, Mode, hipStream_t, int64_t*) {
  return hipErrorNotSupported;
}

}  // namespace vtrace
