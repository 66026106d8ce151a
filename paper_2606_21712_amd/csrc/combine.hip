// moe_combine: y[t] = sum_j w[t,j] * y_perm[dest_rows[t,j]] (+ y_shared[t]) on gfx950.
//
// Gather form: one wavefront per token (or per part of a token's row, for large
// batches) walks the hidden dimension in 16-byte vectors (8 bf16 or 4 fp32 per
// lane), loads the token's k expert rows, sums them in fp32 in slot order, adds
// the shared-expert row last and rounds once.
// For k = 1, 2, 4, 8 the loads of all k rows are in flight together, up to 32
// sixteen-byte loads per lane; y is stored with nontemporal stores.
// Every output element is written by exactly one lane, so there are no atomics
// and the result is deterministic.
#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

template <bool BF16>
struct Vec;

template <>
struct Vec<true> {                 // 8 bf16 in 16 bytes
  static constexpr int N = 8;
  __device__ static void unpack(const u32x4& v, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(v[i] << 16);
      f[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
    }
  }
  __device__ static u32x4 pack(const float* f) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
    return v;
  }
};

template <>
struct Vec<false> {                // 4 fp32 in 16 bytes
  static constexpr int N = 4;
  __device__ static void unpack(const u32x4& v, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(v[i]);
  }
  __device__ static u32x4 pack(const float* f) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(f[i]);
    return v;
  }
};

// KT > 0: k is KT, known at compile time, and each lane first issues the loads of
// all KT rows for UNROLL vectors (KT * UNROLL 16-byte loads in flight), then sums
// them in slot order.  KT = 0: any k <= kMaxTopK, one row's loads at a time.
template <bool BF16, int KT, int UNROLL>
__global__ __launch_bounds__(kThreads) void combine_kernel(const uint8_t* __restrict__ y_perm,
                                                          const int32_t* __restrict__ dest,
                                                          const float* __restrict__ w,
                                                          const uint8_t* __restrict__ y_shared,
                                                          int64_t T, int k, int64_t row_bytes, int splits,
                                                          uint8_t* __restrict__ y) {
  using V = Vec<BF16>;
  constexpr int KM = KT > 0 ? KT : kMaxTopK;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t gw = int64_t(blockIdx.x) * kWavesPerBlock + wv;
  const int64_t t = gw / splits;
  const int part = int(gw % splits);
  if (t >= T) return;
  if (KT > 0) k = KT;
  int32_t rows[KM];
  float wt[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    rows[j] = j < k ? dest[t * k + j] : 0;
    wt[j] = j < k ? w[t * k + j] : 0.f;
  }
  const int nall = int(row_bytes / 16);
  const int vlo = part * nall / splits;
  const int nvec = (part + 1) * nall / splits;
  for (int v0 = vlo + lane; v0 < nvec; v0 += kWave * UNROLL) {
    float acc[UNROLL][V::N];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
#pragma unroll
      for (int i = 0; i < V::N; ++i) acc[u][i] = 0.f;
    if (KT > 0) {
      u32x4 raw[KM][UNROLL];
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        const u32x4* src = reinterpret_cast<const u32x4*>(y_perm + int64_t(rows[j]) * row_bytes);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
          if (v0 + u * kWave < nvec) raw[j][u] = __builtin_nontemporal_load(src + v0 + u * kWave);
      }
#pragma unroll
      for (int j = 0; j < KM; ++j)
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
          if (v0 + u * kWave < nvec) {
            float f[V::N];
            V::unpack(raw[j][u], f);
#pragma unroll
            for (int i = 0; i < V::N; ++i) acc[u][i] = fmaf(wt[j], f[i], acc[u][i]);
          }
        }
    } else {
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        if (j < k) {
          const u32x4* src = reinterpret_cast<const u32x4*>(y_perm + int64_t(rows[j]) * row_bytes);
          u32x4 raw[UNROLL];
#pragma unroll
          for (int u = 0; u < UNROLL; ++u)
            if (v0 + u * kWave < nvec) raw[u] = __builtin_nontemporal_load(src + v0 + u * kWave);
#pragma unroll
          for (int u = 0; u < UNROLL; ++u) {
            if (v0 + u * kWave < nvec) {
              float f[V::N];
              V::unpack(raw[u], f);
#pragma unroll
              for (int i = 0; i < V::N; ++i) acc[u][i] = fmaf(wt[j], f[i], acc[u][i]);
            }
          }
        }
      }
    }
    if (y_shared != nullptr) {
      const u32x4* src = reinterpret_cast<const u32x4*>(y_shared + t * row_bytes);
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        if (v0 + u * kWave < nvec) {
          float f[V::N];
          V::unpack(__builtin_nontemporal_load(src + v0 + u * kWave), f);
#pragma unroll
          for (int i = 0; i < V::N; ++i) acc[u][i] += f[i];
        }
      }
    }
    // y is written once and not read back by this kernel: nontemporal stores keep
    // it from displacing the rows still to be read (measured 3-8% faster).
    u32x4* dst = reinterpret_cast<u32x4*>(y + t * row_bytes);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      if (v0 + u * kWave < nvec) __builtin_nontemporal_store(V::pack(acc[u]), dst + v0 + u * kWave);
  }
}

template <bool BF16>
void launch_combine_t(const uint8_t* yp, const int32_t* dest, const float* w, const uint8_t* ys, int64_t T,
                      int k, int64_t row_bytes, int splits, uint8_t* yo, unsigned blocks, hipStream_t s) {
  // 32 (k = 1, 2: 8 or 16) sixteen-byte loads in flight per lane: k rows x UNROLL vectors.
  switch (k) {
    case 1:
      MOE_LAUNCH("combine", (combine_kernel<BF16, 1, 8>), dim3(blocks), dim3(kThreads), s, yp, dest, w, ys, T,
                 k, row_bytes, splits, yo);
      break;
    case 2:
      MOE_LAUNCH("combine", (combine_kernel<BF16, 2, 8>), dim3(blocks), dim3(kThreads), s, yp, dest, w, ys, T,
                 k, row_bytes, splits, yo);
      break;
    case 4:
      MOE_LAUNCH("combine", (combine_kernel<BF16, 4, 8>), dim3(blocks), dim3(kThreads), s, yp, dest, w, ys, T,
                 k, row_bytes, splits, yo);
      break;
    case 8:
      MOE_LAUNCH("combine", (combine_kernel<BF16, 8, 2>), dim3(blocks), dim3(kThreads), s, yp, dest, w, ys, T,
                 k, row_bytes, splits, yo);
      break;
    default:
      MOE_LAUNCH("combine", (combine_kernel<BF16, 0, 2>), dim3(blocks), dim3(kThreads), s, yp, dest, w, ys, T,
                 k, row_bytes, splits, yo);
  }
}

}  // namespace

hipError_t launch_combine(const void* y_perm, const int32_t* dest, const float* w, const void* y_shared,
                          int64_t T, int k, int H, bool bf16, void* y, hipStream_t s) {
  const int64_t row_bytes = int64_t(H) * (bf16 ? 2 : 4);
  const int nvec = int(row_bytes / 16);
  // Column split: a token's row is cut into `splits` parts, one wavefront each, so
  // that large batches run enough wavefronts with a few vectors per lane each
  // (measured cold, % of 8 TB/s: memory-constrained 71 -> 76 with 2 parts,
  // Mixtral-shaped 32K tokens 75 -> 77 with 4, DeepSeek-shaped 65 -> 70 with 8);
  // small batches (fewer than 8192 tokens) keep whole rows.
  int splits = 1;
  if (T >= 8192)
    while (splits < 8 && nvec / (2 * splits) >= kWave && T * splits < (int64_t(1) << 30) &&
           (nvec / splits > 4 * kWave || T * splits < 131072))
      splits *= 2;
  const unsigned blocks = unsigned((T * splits + kWavesPerBlock - 1) / kWavesPerBlock);
  auto yp = static_cast<const uint8_t*>(y_perm);
  auto ys = static_cast<const uint8_t*>(y_shared);
  auto yo = static_cast<uint8_t*>(y);
  if (bf16)
    launch_combine_t<true>(yp, dest, w, ys, T, k, row_bytes, splits, yo, blocks, s);
  else
    launch_combine_t<false>(yp, dest, w, ys, T, k, row_bytes, splits, yo, blocks, s);
  return hipGetLastError();
}

}  // namespace moe
