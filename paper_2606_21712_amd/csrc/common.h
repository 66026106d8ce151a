// Device helpers shared by the gfx950 kernels of the MoE hot path.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kNumXcd = 8;      // MI355X: 8 accelerator complex dies, workgroups dealt round-robin

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// bf16 <-> fp32 as bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Two fp32 -> two bf16 packed in one 32-bit word (low half = a), rounded to
// nearest even: gfx950's v_cvt_pk_bf16_f32.  For every finite input it gives the
// same bits as the integer rounding (u + 0x7FFF + ((u >> 16) & 1)) >> 16, which
// was checked over all 2^32 - 2^24 finite fp32 patterns.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Monotone map of a finite float to uint32 (larger float -> larger integer).
// -0.0 is first folded onto +0.0 so that the two compare equal, as floats do.
__device__ __forceinline__ uint32_t orderable(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_orderable(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}

// silu(z) = z / (1 + e^-z) in fp32, the division taken as a multiplication by the
// hardware reciprocal (1 ulp).  Large negative z: e^-z = inf, rcp(inf) = 0, silu = -0.
__device__ __forceinline__ float silu(float z) { return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  uint32_t lo = __shfl_xor(uint32_t(v), mask);
  uint32_t hi = __shfl_xor(uint32_t(v >> 32), mask);
  return (uint64_t(hi) << 32) | lo;
}

// Largest e in [0, E) with pref[e] <= q, given pref[0] <= q < pref[E]
// (the expert that owns entry q of a per-expert prefix of tile counts).
__device__ __forceinline__ int find_expert(const int32_t* pref, int E, int64_t q) {
  int lo = 0, hi = E;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pref[mid] <= q) lo = mid; else hi = mid;
  }
  return lo;
}

// Exclusive scan of one int per thread over a 256-thread block; *total = sum.
// Every thread of the block must call it (it synchronizes the block).
__device__ __forceinline__ int32_t block_exclusive_scan256(int32_t v, int32_t* total) {
  __shared__ int32_t wsum[4];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  int32_t x = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int32_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) wsum[w] = x;
  __syncthreads();
  int32_t before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    before += (i < w) ? wsum[i] : 0;
    tot += wsum[i];
  }
  __syncthreads();
  *total = tot;
  return before + x - v;
}

}  // namespace moe
