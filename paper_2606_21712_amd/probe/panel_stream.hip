// Weight-panel streaming probe (a measurement tool, not part of the MoE path or
// its C ABI; built into the probe library).  Persistent workgroups of eight
// wavefronts claim 256-row panels of a row-major [panels * 256, K] byte matrix
// from a counter and stream each panel through two LDS stages one 128-byte k
// column at a time (32 KB per step, direct global -> LDS loads), the way the
// grouped GEMMs read a weight tile.  With ROTATE, panel p starts at column
// (7 p) mod (K / 128) and wraps around; without it every panel starts at column
// 0, so panels streamed at the same time read the same column of their rows.
// Each lane folds one word per step into a value it stores at the end, which
// keeps the loads live.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kThreads = 512;
constexpr int kRows = 256;
constexpr int kStep = kRows * 128;        // bytes of one k column of a panel

template <bool ROTATE>
__global__ __launch_bounds__(kThreads, 1) void panel_stream_kernel(const uint8_t* __restrict__ w, int panels,
                                                                 int K, int* __restrict__ counter,
                                                                 uint32_t* __restrict__ out) {
  __shared__ __attribute__((aligned(1024))) uint8_t st[2 * kStep];
  __shared__ int s_panel;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (panels < 0) st[tid] = 0;            // never taken: keeps the DMA-filled stage reads
  const int KT = K / 128;
  uint32_t acc = 0;
  for (;;) {
    if (tid == 0) s_panel = atomicAdd(counter, 1);
    __syncthreads();
    const int p = s_panel;
    __syncthreads();
    if (p >= panels) break;               // uniform: every wavefront leaves
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(w) + int64_t(p) * kRows * K, 0, kRows * K, 0x00020000);
    // wavefront w's pass i fills the 1 KB block 8 i + w of a stage: rows 8 (8 i + w) + lane / 8
    uint32_t off[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      off[i] = uint32_t((8 * (8 * i + wave) + (lane >> 3)) * K + (lane & 7) * 16);
    const int rot = ROTATE ? int((int64_t(p) * 7) % KT) : 0;
    auto issue = [&](int stage, int j) {
      const int q = j + rot;
      const int kt = q >= KT ? q - KT : q;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, st + stage * kStep + (8 * i + wave) * 1024, 16, off[i],
                                                 kt * 128, 0, 0);
    };
    issue(0, 0);
    for (int j = 0; j < KT; ++j) {
      __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this stage's loads landed
      __syncthreads();                      // ... for every wavefront; the other stage is free
      if (j + 1 < KT) issue((j + 1) & 1, j + 1);
      acc ^= *reinterpret_cast<const uint32_t*>(st + (j & 1) * kStep + tid * 64);
    }
    __syncthreads();
  }
  out[int64_t(blockIdx.x) * kThreads + tid] = acc;
}

}  // namespace

// Streams `panels` panels of 256 rows x K bytes from w (row-major, K a multiple of
// 128, 256 K < 2^31) on `blocks` persistent workgroups of 512 threads.  counter:
// one device int that the caller zeroes before the launch (it ends at panels +
// blocks); out: blocks * 512 device words.  Returns 0, 1 for bad arguments (nothing
// launched), or the HIP error of the launch.
extern "C" int moe_probe_stream_panels(const void* w, int panels, int K, int rotate, int blocks, int* counter,
                                       uint32_t* out, void* stream) {
  if (w == nullptr || counter == nullptr || out == nullptr || panels < 1 || blocks < 1 || K < 128 ||
      K % 128 != 0 || int64_t(kRows) * K >= (int64_t(1) << 31))
    return 1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const auto* wb = static_cast<const uint8_t*>(w);
  if (rotate)
    hipLaunchKernelGGL(panel_stream_kernel<true>, dim3(blocks), dim3(kThreads), 0, s, wb, panels, K, counter, out);
  else
    hipLaunchKernelGGL(panel_stream_kernel<false>, dim3(blocks), dim3(kThreads), 0, s, wb, panels, K, counter, out);
  return static_cast<int>(hipGetLastError());
}
