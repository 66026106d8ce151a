// Host-side argument validation for the C ABI in include/moe.h.
// Plain C++ with no HIP dependency, so it can be built and tested on a machine
// without a GPU (and under host sanitizers).
#pragma once
#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/moe.h"

namespace moe {

struct Check {
  moe_status status = MOE_OK;
  std::string msg;
  bool ok() const { return status == MOE_OK; }
};

// Workspace layouts (bytes).  Offsets inside the workspace are 256-byte aligned.
size_t permute_workspace_bytes(int64_t T, int32_t E, int32_t k);
size_t ffn_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F, moe_dtype dt);
// ffn workspace: [m-tile prefix (E + 1 ints) | tile queues | h [R, F] |
//                 down-projection tail-split partial slots]
size_t ffn_queue_offset(int32_t E);
size_t ffn_h_offset(int32_t E);
size_t ffn_partial_offset(int64_t R, int32_t E, int32_t F, moe_dtype dt);
// Partial slots of the down projection's tail split: 320 x 256 fp32 each, at most
// kMaxTailPieces and at most the output-tile bound; none when the k loop (F / bk
// steps) is too short to split.
size_t ffn_tail_partial_bytes(int64_t R, int32_t E, int32_t H, int32_t F, int bk);
int64_t permute_units(int64_t R);           // count-units (1024 assignments each)

constexpr int64_t kPermuteUnit = 1024;      // assignments per counting unit (one wavefront)

Check validate_route(const float* logits, int64_t T, int32_t E, int32_t k, int32_t renormalize,
                     const int32_t* ids, const float* w);
Check validate_router_topk(const void* x, const void* w, int64_t T, int32_t E, int32_t k, int32_t H,
                           int32_t renormalize, const float* logits, const int32_t* ids, const float* wts);
Check validate_permute(const int32_t* ids, const void* x, int64_t T, int32_t E, int32_t k, int32_t H,
                       int dt, const int32_t* counts, const int32_t* offsets, const int32_t* sorted_tok,
                       const int32_t* dest, const void* x_perm, const void* ws, size_t ws_bytes);
Check validate_permute_static(const int32_t* ids, const void* x, int64_t T, int32_t E, int32_t k, int32_t H,
                              int dt, const int32_t* counts, const int32_t* offsets, const int32_t* sorted_tok,
                              const int32_t* dest, const void* x_perm);
Check validate_ffn(const void* x_perm, const int32_t* offsets, int64_t R, int32_t E, int32_t H,
                   int32_t F, const void* wg, const void* wu, const void* wd, int dt,
                   const void* y_perm, const void* ws, size_t ws_bytes);
Check validate_ffn_gather(const void* x, const int32_t* sorted_tok, int64_t T, const int32_t* offsets,
                          int64_t R, int32_t E, int32_t H, int32_t F, const void* wg, const void* wu,
                          const void* wd, int dt, const void* y_perm, const void* ws, size_t ws_bytes);
// MXFP8: scales of a [rows, K] matrix; ffn workspace [prefix | queues | h codes
// [R, F] | h scales | down-projection tail-split partial slots]
size_t mxfp8_scale_bytes(int64_t rows, int32_t K);
size_t ffn_mxfp8_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F);
size_t ffn_mxfp8_h_scales_offset(int64_t R, int32_t E, int32_t F);
size_t ffn_mxfp8_partial_offset(int64_t R, int32_t E, int32_t F);
Check validate_quantize_mxfp8(const void* src, const int32_t* row_map, int64_t rows_out, int64_t rows_src,
                              int32_t K, const void* codes, const void* scales);
Check validate_ffn_mxfp8(const void* x, const void* xs, const int32_t* offsets, int64_t R, int32_t E, int32_t H,
                         int32_t F, const void* wg, const void* wgs, const void* wu, const void* wus,
                         const void* wd, const void* wds, const void* y_perm, const void* ws, size_t ws_bytes);
Check validate_ffn_mxfp8_gather(const void* x, const void* xs, const int32_t* sorted_tok, int64_t T,
                                const int32_t* offsets, int64_t R, int32_t E, int32_t H, int32_t F, const void* wg,
                                const void* wgs, const void* wu, const void* wus, const void* wd, const void* wds,
                                const void* y_perm, const void* ws, size_t ws_bytes);
Check validate_combine(const void* y_perm, const int32_t* dest, const float* w, const void* y_shared,
                       int64_t T, int32_t k, int32_t H, int dt, const void* y);

}  // namespace moe
