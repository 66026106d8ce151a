// Internal launchers of the gfx950 kernels behind the C ABI (include/moe.h).
// Arguments are validated by the caller (moe_abi.cpp) before any launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

constexpr int kMaxTopK = 16;

// Per-kernel event timing (profiler.cpp); no-ops unless moe_profiler_start() ran.
void prof_begin(hipStream_t s, const char* name);
void prof_end(hipStream_t s);

// Launch a kernel on `stream`, bracketed by the profiler's events.
#define MOE_LAUNCH(name, kernel, grid, block, stream, ...)             \
  do {                                                                 \
    ::moe::prof_begin(stream, name);                                   \
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, __VA_ARGS__);   \
    ::moe::prof_end(stream);                                           \
  } while (0)
constexpr int kMaxExperts = 256;

void route_shape(int E, int* G, int* V);
// Router GEMM (x [T, H] . w [E, H]^T, E <= 64) fused with the gate; logits may be null.
hipError_t launch_router_topk(const uint16_t* x, const uint16_t* w, int64_t T, int E, int k, int H, int renorm,
                              float* logits, int32_t* ids, float* wts, int num_cu, hipStream_t s);
hipError_t launch_route(const float* logits, int64_t T, int E, int k, int renorm, int32_t* ids,
                        float* w, int num_cu, hipStream_t s);

hipError_t launch_permute(const int32_t* ids, const void* x, int64_t T, int E, int k, int H, int elt,
                          int32_t* counts, int32_t* offsets, int32_t* sorted_tok, int32_t* dest,
                          void* x_perm, int32_t* unit_counts, int64_t units_padded, hipStream_t s);
// Device address of the static scratch array of moe_permute_static on the current
// device (kPermuteStaticScratchBytes, tiling.h); looked up once per device.
hipError_t permute_static_scratch(void** out);

// Grouped SwiGLU FFN (bf16).  act is x_perm [R, H], or with gather != null the
// token rows x [T, H] read through gather[r] (any size: x of 2 GiB or more is
// read with 64-bit per-lane row addresses instead of one buffer resource).  Device scratch:
// mtile_prefix (E + 1 ints), queues (2 ints), h [R, F], and the down
// projection's tail-split partial slots (ffn_tail_partial_bytes); all are
// rewritten by the call before use.
hipError_t launch_ffn_bf16(const uint16_t* act, const int32_t* gather, int64_t T, const int32_t* offsets,
                           int64_t R, int E, int H, int F, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, uint16_t* y_perm, int32_t* mtile_prefix, int32_t* queues,
                           uint16_t* h, float* partial, int num_cu, hipStream_t s);
// Sums the tail-split pieces of a down projection (G workgroups, KT k steps,
// NT n-tiles of 256 over N columns) into y; a no-op launch when the plan has none.
// row_blocks: the GEMM's m-tiles follow the bf16 rule (decode_tile<true>).
hipError_t launch_tail_reduce(const float* partial, const int32_t* mtile_prefix, const int32_t* offsets, int E,
                              int NT, int G, int KT, int N, uint16_t* y, bool row_blocks, hipStream_t s);
// Per-expert m-tile prefix of the device-side offsets (one block): ceil(rows /
// bm) m-tiles per expert; zeroes the GEMMs' tile counters when queues != null.
hipError_t launch_tile_prefix(const int32_t* offsets, int E, int bm, int32_t* mtile_prefix, int32_t* queues,
                              hipStream_t s);

// MXFP8: bf16 rows -> E4M3 codes [rows_out, K] + k-step-major E8M0 scales
// [K / 128][rows_out][4]; output row r reads source row row_map[r] (or r).
hipError_t launch_quantize_mxfp8(const uint16_t* src, const int32_t* row_map, int64_t rows_out, int K,
                                 uint8_t* codes, uint8_t* scales, int num_cu, hipStream_t s);
// Grouped SwiGLU FFN on MXFP8 operands; h (MXFP8, R x F codes + scales) and the
// down projection's tail-split partial slots are device scratch.  x is the
// grouped rows [R, H], or with gather != null the token rows [T, H] read through
// gather[r] (T * H < 2^31).
hipError_t launch_ffn_mxfp8(const uint8_t* x, const uint8_t* xs, const int32_t* gather, int64_t T,
                            const int32_t* offsets, int64_t R, int E, int H, int F, const uint8_t* wg,
                            const uint8_t* wgs, const uint8_t* wu, const uint8_t* wus, const uint8_t* wd,
                            const uint8_t* wds, uint16_t* y_perm, int32_t* mtile_prefix, int32_t* queues, uint8_t* h,
                            uint8_t* hs, float* partial, int num_cu, hipStream_t s);

hipError_t launch_ffn_f32(const float* act, const int32_t* gather, const int32_t* offsets, int64_t R,
                          int E, int H, int F, const float* wg, const float* wu, const float* wd,
                          float* y_perm, int32_t* mtile_prefix, float* h, hipStream_t s);

hipError_t launch_combine(const void* y_perm, const int32_t* dest, const float* w, const void* y_shared,
                          int64_t T, int k, int H, bool bf16, void* y, hipStream_t s);

}  // namespace moe
