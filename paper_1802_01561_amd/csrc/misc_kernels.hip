// Small kernels: the action-logit gather and the workspace clear.
#include "device_common.hpp"

namespace vtrace {
namespace {

constexpr int kThreads = 256;

// gathered[t,b,0] = target[t,b,a], gathered[t,b,1] = behaviour[t,b,a], as bit
// copies; an out-of-range action gives an all-ones pattern (a NaN).
template <typename Bits>
__global__ __launch_bounds__(kThreads) void gather_kernel(int64_t n, int64_t A,
                                                          const Bits* __restrict__ z,
                                                          const Bits* __restrict__ y,
                                                          const int32_t* __restrict__ act,
                                                          Bits* __restrict__ out) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n; i += stride) {
    const int32_t a = act[i];
    Bits gz = static_cast<Bits>(~Bits(0)), gy = static_cast<Bits>(~Bits(0));
    if (a >= 0 && a < A) {
      gz = z[i * A + a];
      gy = y[i * A + a];
    }
    out[2 * i + 0] = gz;
    out[2 * i + 1] = gy;
  }
}

// Plain vector stores, so that the clear can be captured in a HIP graph.
__global__ __launch_bounds__(kThreads) void fill_zero_kernel(uint32_t* p, size_t words) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kThreads;
  for (size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x; i < words; i += stride)
    p[i] = 0u;
}

unsigned grid_for(int64_t n) {
  int64_t g = (n + kThreads - 1) / kThreads;
  if (g > 4096) g = 4096;
  if (g < 1) g = 1;
  return static_cast<unsigned>(g);
}

}  // namespace

hipError_t launch_gather(int64_t T, int64_t B, int64_t A, LogitsType lt, const void* target,
                         const void* behaviour, const int32_t* actions, void* gathered,
                         hipStream_t s) {
  const int64_t n = T * B;
  if (lt == LogitsType::BF16) {
    hipLaunchKernelGGL(gather_kernel<uint16_t>, dim3(grid_for(n)), dim3(kThreads), 0, s, n, A,
                       static_cast<const uint16_t*>(target), static_cast<const uint16_t*>(behaviour),
                       actions, static_cast<uint16_t*>(gathered));
  } else {
    hipLaunchKernelGGL(gather_kernel<uint32_t>, dim3(grid_for(n)), dim3(kThreads), 0, s, n, A,
                       static_cast<const uint32_t*>(target), static_cast<const uint32_t*>(behaviour),
                       actions, static_cast<uint32_t*>(gathered));
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const size_t words = bytes / 4;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(static_cast<int64_t>(words))), dim3(kThreads),
                     0, s, static_cast<uint32_t*>(p), words);
  return hipGetLastError();
}

}  // namespace vtrace
