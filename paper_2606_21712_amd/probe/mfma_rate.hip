// Matrix-core rate probe (a measurement tool, not part of the MoE path or its
// C ABI; built into its own library).  Each wavefront runs `iters` iterations of
// kChains independent MFMA accumulation chains with operands held in registers:
// no memory traffic besides one store per lane at the end, so the launch
// measures what the matrix cores sustain under the board's power limit.
//
// Operands: kSets operand sets, MFMA j of an iteration taking set j % kSets for
// one operand and (j + 1) % kSets for the other, so consecutive MFMAs differ in
// both.  With RANDOM, one set is redrawn per iteration from a per-lane linear
// congruential generator (x <- 1664525 x + 1013904223, the Numerical Recipes
// constants), so the operand bits keep changing as real data does; without it
// the operands stay fixed.  Values stay finite: bf16 words keep a random sign
// and mantissa with exponents 124..127; E4M3 bytes keep the exponent's top bit
// clear (no NaN encodings).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));

constexpr int kChains = 8;
constexpr int kSets = 4;
constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t lcg(uint32_t x) { return x * 1664525u + 1013904223u; }

template <bool FP8, bool RANDOM>
__global__ __launch_bounds__(kThreads) void mfma_rate_kernel(int iters, float* __restrict__ out) {
  f32x16 acc[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  uint32_t x = lcg(uint32_t(blockIdx.x) * kThreads + threadIdx.x + 1u);
  constexpr uint32_t kMask = FP8 ? 0xF7F7F7F7u : 0x81FF81FFu;   // bits kept from the generator
  constexpr uint32_t kSet = FP8 ? 0u : 0x3E003E00u;             // bits forced on
  constexpr int kWords = FP8 ? 8 : 4;                            // dwords per operand
  typedef uint32_t words __attribute__((ext_vector_type(kWords)));
  words a[kSets], b[kSets];
#pragma unroll
  for (int s = 0; s < kSets; ++s)
#pragma unroll
    for (int w = 0; w < kWords; ++w) {
      x = lcg(x);
      a[s][w] = (x & kMask) | kSet;
      x = lcg(x);
      b[s][w] = (x & kMask) | kSet;
    }
  // iterations in groups of kSets, so that the set redrawn each iteration is a
  // compile-time index (no indirect register access)
  for (int it = 0; it < iters; it += kSets) {
#pragma unroll
    for (int s = 0; s < kSets; ++s) {
      if constexpr (RANDOM) {
#pragma unroll
        for (int w = 0; w < kWords; ++w) {
          x = lcg(x);
          a[s][w] = (x & kMask) | kSet;
          b[s][w] = ((x >> 7 | x << 25) & kMask) | kSet;
        }
      }
#pragma unroll
      for (int j = 0; j < kChains; ++j) {
        if constexpr (FP8) {
          // E4M3 x E4M3, unit E8M0 scales (127 = 2^0)
          acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              __builtin_bit_cast(i32x8, a[j % kSets]), __builtin_bit_cast(i32x8, b[(j + 1) % kSets]), acc[j], 0,
              0, 0, 127, 0, 127);
        } else {
          acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[j % kSets]),
                                                           __builtin_bit_cast(bf16x8, b[(j + 1) % kSets]), acc[j],
                                                           0, 0, 0);
        }
      }
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < kChains; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) sum += acc[j][e];
  out[size_t(blockIdx.x) * kThreads + threadIdx.x] = sum;
}

}  // namespace

// Launches `blocks` workgroups of 256 threads on `stream` (a hipStream_t, null =
// default) running the probe: fp8 = 0 for v_mfma_f32_32x32x16_bf16 (32768 flop
// per instruction), 1 for v_mfma_scale_f32_32x32x64_f8f6f4 on E4M3 (131072);
// random_operands as above.  out: device float[blocks * 256], written once per
// lane.  Each wavefront issues ceil(iters / 4) * 4 * 8 MFMAs.  Returns 0, or 1 on a bad
// argument (nothing launched), or the HIP error code of the launch.
extern "C" int moe_probe_mfma_rate(int fp8, int random_operands, int blocks, int iters, float* out,
                                   void* stream) {
  if (blocks < 1 || iters < 0 || out == nullptr) return 1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<unsigned>(blocks)), block(kThreads);
  if (fp8 && random_operands)
    hipLaunchKernelGGL((mfma_rate_kernel<true, true>), grid, block, 0, s, iters, out);
  else if (fp8)
    hipLaunchKernelGGL((mfma_rate_kernel<true, false>), grid, block, 0, s, iters, out);
  else if (random_operands)
    hipLaunchKernelGGL((mfma_rate_kernel<false, true>), grid, block, 0, s, iters, out);
  else
    hipLaunchKernelGGL((mfma_rate_kernel<false, false>), grid, block, 0, s, iters, out);
  return static_cast<int>(hipGetLastError());
}
