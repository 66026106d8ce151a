// Write-rate probe (a measurement tool, not part of the MoE path or its C ABI;
// built into the probe library): grid-stride 16-byte stores that fill a buffer,
// nothing read, so a launch measures what HBM sustains for writes alone.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void write_rate_kernel(u32x4* __restrict__ out, int64_t n) {
  const u32x4 v = {uint32_t(threadIdx.x), uint32_t(blockIdx.x), 0u, 0u};
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
    __builtin_nontemporal_store(v, out + i);
}

}  // namespace

// Fills bytes (a multiple of 16) of out on `blocks` workgroups of 256 threads.
// Returns 0, 1 for bad arguments (nothing launched), or the HIP error of the launch.
extern "C" int moe_probe_write(void* out, int64_t bytes, int blocks, void* stream) {
  if (out == nullptr || bytes < 16 || bytes % 16 != 0 || blocks < 1) return 1;
  hipLaunchKernelGGL(write_rate_kernel, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<u32x4*>(out), bytes / 16);
  return static_cast<int>(hipGetLastError());
}
