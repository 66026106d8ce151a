// C ABI of the MoE hot path (include/moe.h): validation, workspace carving,
// launches and error mapping.  No allocation, no synchronization.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <atomic>
#include <mutex>
#include <string>

#include "../../include/moe.h"
#include "moe_internal.h"
#include "moe_validate.h"

namespace {

thread_local std::string g_last_error;

moe_status finish(const moe::Check& c) {
  g_last_error = c.msg;
  return c.status;
}

moe_status hip_status(const char* fn, hipError_t err) {
  if (err == hipSuccess) {
    g_last_error.clear();
    return MOE_OK;
  }
  g_last_error = std::string(fn) + ": " + hipGetErrorString(err);
  return MOE_ERR_HIP;
}

std::atomic<int> g_cu_budget{0};

// Compute units the persistent grids are sized for: the budget set with
// moe_set_cu_budget, else the current device's count (cached per device).
int cu_count(hipError_t* err) {
  const int budget = g_cu_budget.load(std::memory_order_relaxed);
  if (budget > 0) {
    *err = hipSuccess;
    return budget;
  }
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return 0;
  if (dev < 0 || dev >= 64) dev = 0;
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == 0) {
    int n = 0;
    *err = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (*err != hipSuccess) return 0;
    cache[dev] = n > 0 ? n : 256;
  }
  return cache[dev];
}

hipStream_t stream_of(moe_stream s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

int moe_abi_version(void) { return MOE_ABI_VERSION; }

moe_status moe_set_cu_budget(int32_t n) {
  moe::Check c;
  if (n < 0) {
    c.status = MOE_ERR_INVALID_ARGUMENT;
    c.msg = "moe_set_cu_budget: n=" + std::to_string(n) + " is negative";
    return finish(c);
  }
  g_cu_budget.store(n, std::memory_order_relaxed);
  return finish(c);
}

const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARGUMENT: return "MOE_ERR_INVALID_ARGUMENT";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_WORKSPACE_TOO_SMALL: return "MOE_ERR_WORKSPACE_TOO_SMALL";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
    default: return "MOE_ERR_UNKNOWN_STATUS";
  }
}

const char* moe_last_error(void) { return g_last_error.c_str(); }

moe_status moe_route(const float* logits, int64_t T, int32_t E, int32_t k, int32_t renormalize,
                     int32_t* topk_ids, float* topk_weights, moe_stream stream) {
  moe::Check c = moe::validate_route(logits, T, E, k, renormalize, topk_ids, topk_weights);
  if (!c.ok() || T == 0) return finish(c);
  hipError_t err;
  const int ncu = cu_count(&err);
  if (err != hipSuccess) return hip_status("moe_route", err);
  return hip_status("moe_route",
                    moe::launch_route(logits, T, E, k, renormalize, topk_ids, topk_weights, ncu,
                                      stream_of(stream)));
}

moe_status moe_router_topk(const void* x, const void* w_router, int64_t T, int32_t E, int32_t k, int32_t H,
                           int32_t renormalize, float* logits, int32_t* topk_ids, float* topk_weights,
                           moe_stream stream) {
  moe::Check c = moe::validate_router_topk(x, w_router, T, E, k, H, renormalize, logits, topk_ids, topk_weights);
  if (!c.ok() || T == 0) return finish(c);
  hipError_t err;
  const int ncu = cu_count(&err);
  if (err != hipSuccess) return hip_status("moe_router_topk", err);
  return hip_status("moe_router_topk",
                    moe::launch_router_topk(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_router),
                                            T, E, k, H, renormalize, logits, topk_ids, topk_weights, ncu,
                                            stream_of(stream)));
}

size_t moe_permute_workspace_bytes(int64_t T, int32_t E, int32_t k) {
  return moe::permute_workspace_bytes(T, E, k);
}

moe_status moe_permute(const int32_t* topk_ids, const void* x, int64_t T, int32_t E, int32_t k,
                       int32_t H, moe_dtype dt, int32_t* expert_counts, int32_t* expert_offsets,
                       int32_t* sorted_token_ids, int32_t* dest_rows, void* x_perm, void* ws,
                       size_t ws_bytes, moe_stream stream) {
  moe::Check c = moe::validate_permute(topk_ids, x, T, E, k, H, dt, expert_counts, expert_offsets,
                                       sorted_token_ids, dest_rows, x_perm, ws, ws_bytes);
  if (!c.ok() || T == 0) return finish(c);
  const int64_t upad = (moe::permute_units(T * k) + 3) / 4 * 4;
  return hip_status("moe_permute",
                    moe::launch_permute(topk_ids, x, T, E, k, H, dt == MOE_DTYPE_F32 ? 4 : 2,
                                        expert_counts, expert_offsets, sorted_token_ids, dest_rows,
                                        x_perm, static_cast<int32_t*>(ws), upad, stream_of(stream)));
}

moe_status moe_permute_static(const int32_t* topk_ids, const void* x, int64_t T, int32_t E, int32_t k,
                              int32_t H, moe_dtype dt, int32_t* expert_counts, int32_t* expert_offsets,
                              int32_t* sorted_token_ids, int32_t* dest_rows, void* x_perm, moe_stream stream) {
  moe::Check c = moe::validate_permute_static(topk_ids, x, T, E, k, H, dt, expert_counts, expert_offsets,
                                              sorted_token_ids, dest_rows, x_perm);
  if (!c.ok() || T == 0) return finish(c);
  void* ws = nullptr;
  const hipError_t err = moe::permute_static_scratch(&ws);
  if (err != hipSuccess) return hip_status("moe_permute_static", err);
  const int64_t upad = (moe::permute_units(T * k) + 3) / 4 * 4;
  return hip_status("moe_permute_static",
                    moe::launch_permute(topk_ids, x, T, E, k, H, dt == MOE_DTYPE_F32 ? 4 : 2, expert_counts,
                                        expert_offsets, sorted_token_ids, dest_rows, x_perm,
                                        static_cast<int32_t*>(ws), upad, stream_of(stream)));
}

size_t moe_grouped_ffn_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F, moe_dtype dt) {
  return moe::ffn_workspace_bytes(R, E, H, F, dt);
}

namespace {

moe_status run_ffn(const char* fn, const void* act, const int32_t* gather, int64_t T,
                   const int32_t* expert_offsets, int64_t R, int32_t E, int32_t H, int32_t F,
                   const void* w_gate, const void* w_up, const void* w_down, moe_dtype dt, void* y_perm,
                   void* ws, moe_stream stream) {
  auto* prefix = static_cast<int32_t*>(ws);
  auto* queues = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(ws) + moe::ffn_queue_offset(E));
  void* h = static_cast<uint8_t*>(ws) + moe::ffn_h_offset(E);
  if (dt == MOE_DTYPE_F32) {
    return hip_status(fn, moe::launch_ffn_f32(static_cast<const float*>(act), gather, expert_offsets, R, E,
                                              H, F, static_cast<const float*>(w_gate),
                                              static_cast<const float*>(w_up),
                                              static_cast<const float*>(w_down), static_cast<float*>(y_perm),
                                              prefix, static_cast<float*>(h), stream_of(stream)));
  }
  hipError_t err;
  const int ncu = cu_count(&err);
  if (err != hipSuccess) return hip_status(fn, err);
  auto* partial = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + moe::ffn_partial_offset(R, E, F, dt));
  return hip_status(
      fn, moe::launch_ffn_bf16(static_cast<const uint16_t*>(act), gather, T, expert_offsets, R, E, H, F,
                               static_cast<const uint16_t*>(w_gate), static_cast<const uint16_t*>(w_up),
                               static_cast<const uint16_t*>(w_down), static_cast<uint16_t*>(y_perm), prefix,
                               queues, static_cast<uint16_t*>(h), partial, ncu, stream_of(stream)));
}

}  // namespace

moe_status moe_grouped_ffn(const void* x_perm, const int32_t* expert_offsets, int64_t R, int32_t E,
                           int32_t H, int32_t F, const void* w_gate, const void* w_up,
                           const void* w_down, moe_dtype dt, void* y_perm, void* ws,
                           size_t ws_bytes, moe_stream stream) {
  moe::Check c = moe::validate_ffn(x_perm, expert_offsets, R, E, H, F, w_gate, w_up, w_down, dt,
                                   y_perm, ws, ws_bytes);
  if (!c.ok() || R == 0) return finish(c);
  return run_ffn("moe_grouped_ffn", x_perm, nullptr, R, expert_offsets, R, E, H, F, w_gate, w_up, w_down,
                 dt, y_perm, ws, stream);
}

moe_status moe_grouped_ffn_gather(const void* x, const int32_t* sorted_token_ids,
                                  const int32_t* expert_offsets, int64_t T, int64_t R, int32_t E,
                                  int32_t H, int32_t F, const void* w_gate, const void* w_up,
                                  const void* w_down, moe_dtype dt, void* y_perm, void* ws,
                                  size_t ws_bytes, moe_stream stream) {
  moe::Check c = moe::validate_ffn_gather(x, sorted_token_ids, T, expert_offsets, R, E, H, F, w_gate,
                                          w_up, w_down, dt, y_perm, ws, ws_bytes);
  if (!c.ok() || R == 0) return finish(c);
  return run_ffn("moe_grouped_ffn_gather", x, sorted_token_ids, T, expert_offsets, R, E, H, F, w_gate,
                 w_up, w_down, dt, y_perm, ws, stream);
}

size_t moe_mxfp8_scale_bytes(int64_t rows, int32_t K) { return moe::mxfp8_scale_bytes(rows, K); }

moe_status moe_quantize_mxfp8(const void* src, const int32_t* row_map, int64_t rows_out, int64_t rows_src,
                              int32_t K, uint8_t* codes, uint8_t* scales, moe_stream stream) {
  moe::Check c = moe::validate_quantize_mxfp8(src, row_map, rows_out, rows_src, K, codes, scales);
  if (!c.ok() || rows_out == 0) return finish(c);
  hipError_t err;
  const int ncu = cu_count(&err);
  if (err != hipSuccess) return hip_status("moe_quantize_mxfp8", err);
  return hip_status("moe_quantize_mxfp8",
                    moe::launch_quantize_mxfp8(static_cast<const uint16_t*>(src), row_map, rows_out, K, codes,
                                               scales, ncu, stream_of(stream)));
}

size_t moe_grouped_ffn_mxfp8_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F) {
  return moe::ffn_mxfp8_workspace_bytes(R, E, H, F);
}

namespace {

moe_status run_ffn_mxfp8(const char* fn, const uint8_t* x_codes, const uint8_t* x_scales, const int32_t* gather,
                         int64_t T, const int32_t* expert_offsets, int64_t R, int32_t E, int32_t H, int32_t F,
                         const uint8_t* wg_codes, const uint8_t* wg_scales, const uint8_t* wu_codes,
                         const uint8_t* wu_scales, const uint8_t* wd_codes, const uint8_t* wd_scales, void* y_perm,
                         void* ws, moe_stream stream) {
  hipError_t err;
  const int ncu = cu_count(&err);
  if (err != hipSuccess) return hip_status(fn, err);
  auto* base = static_cast<uint8_t*>(ws);
  auto* prefix = reinterpret_cast<int32_t*>(base);
  auto* queues = reinterpret_cast<int32_t*>(base + moe::ffn_queue_offset(E));
  uint8_t* h = base + moe::ffn_h_offset(E);
  uint8_t* hs = base + moe::ffn_mxfp8_h_scales_offset(R, E, F);
  auto* partial = reinterpret_cast<float*>(base + moe::ffn_mxfp8_partial_offset(R, E, F));
  return hip_status(fn, moe::launch_ffn_mxfp8(x_codes, x_scales, gather, T, expert_offsets, R, E, H, F, wg_codes,
                                              wg_scales, wu_codes, wu_scales, wd_codes, wd_scales,
                                              static_cast<uint16_t*>(y_perm), prefix, queues, h, hs, partial, ncu,
                                              stream_of(stream)));
}

}  // namespace

moe_status moe_grouped_ffn_mxfp8(const uint8_t* x_codes, const uint8_t* x_scales,
                                 const int32_t* expert_offsets, int64_t R, int32_t E, int32_t H, int32_t F,
                                 const uint8_t* wg_codes, const uint8_t* wg_scales, const uint8_t* wu_codes,
                                 const uint8_t* wu_scales, const uint8_t* wd_codes, const uint8_t* wd_scales,
                                 void* y_perm, void* ws, size_t ws_bytes, moe_stream stream) {
  moe::Check c = moe::validate_ffn_mxfp8(x_codes, x_scales, expert_offsets, R, E, H, F, wg_codes, wg_scales,
                                         wu_codes, wu_scales, wd_codes, wd_scales, y_perm, ws, ws_bytes);
  if (!c.ok() || R == 0) return finish(c);
  return run_ffn_mxfp8("moe_grouped_ffn_mxfp8", x_codes, x_scales, nullptr, R, expert_offsets, R, E, H, F,
                       wg_codes, wg_scales, wu_codes, wu_scales, wd_codes, wd_scales, y_perm, ws, stream);
}

moe_status moe_grouped_ffn_mxfp8_gather(const uint8_t* x_codes, const uint8_t* x_scales,
                                        const int32_t* sorted_token_ids, const int32_t* expert_offsets, int64_t T,
                                        int64_t R, int32_t E, int32_t H, int32_t F, const uint8_t* wg_codes,
                                        const uint8_t* wg_scales, const uint8_t* wu_codes,
                                        const uint8_t* wu_scales, const uint8_t* wd_codes,
                                        const uint8_t* wd_scales, void* y_perm, void* ws, size_t ws_bytes,
                                        moe_stream stream) {
  moe::Check c = moe::validate_ffn_mxfp8_gather(x_codes, x_scales, sorted_token_ids, T, expert_offsets, R, E, H,
                                                F, wg_codes, wg_scales, wu_codes, wu_scales, wd_codes, wd_scales,
                                                y_perm, ws, ws_bytes);
  if (!c.ok() || R == 0) return finish(c);
  return run_ffn_mxfp8("moe_grouped_ffn_mxfp8_gather", x_codes, x_scales, sorted_token_ids, T, expert_offsets, R,
                       E, H, F, wg_codes, wg_scales, wu_codes, wu_scales, wd_codes, wd_scales, y_perm, ws, stream);
}

moe_status moe_combine(const void* y_perm, const int32_t* dest_rows, const float* topk_weights,
                       const void* y_shared, int64_t T, int32_t k, int32_t H, moe_dtype dt, void* y,
                       moe_stream stream) {
  moe::Check c = moe::validate_combine(y_perm, dest_rows, topk_weights, y_shared, T, k, H, dt, y);
  if (!c.ok() || T == 0) return finish(c);
  return hip_status("moe_combine",
                    moe::launch_combine(y_perm, dest_rows, topk_weights, y_shared, T, k, H,
                                        dt == MOE_DTYPE_BF16, y, stream_of(stream)));
}

}  // extern "C"
