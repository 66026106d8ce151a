// Host-side argument validation (no HIP calls); see moe_validate.h.
#include "moe_validate.h"
#include "tiling.h"

#include <climits>
#include <cstdio>

namespace moe {
namespace {

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

Check fail(moe_status s, const char* fn, const char* fmt, long long a = 0, long long b = 0) {
  char buf[256];
  char body[200];
  std::snprintf(body, sizeof body, fmt, a, b);
  std::snprintf(buf, sizeof buf, "%s: %s", fn, body);
  Check c;
  c.status = s;
  c.msg = buf;
  return c;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A required pointer: non-null and 16-byte aligned.
Check ptr(const char* fn, const char* name, const void* p) {
  Check c;
  if (p == nullptr) {
    c.status = MOE_ERR_INVALID_ARGUMENT;
    c.msg = std::string(fn) + ": " + name + " is NULL";
  } else if (!aligned16(p)) {
    c.status = MOE_ERR_INVALID_ARGUMENT;
    c.msg = std::string(fn) + ": " + name + " is not 16-byte aligned";
  }
  return c;
}

Check experts_topk(const char* fn, int32_t E, int32_t k) {
  if (E < 1) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "E=%lld must be >= 1", E);
  if (E > MOE_MAX_EXPERTS) return fail(MOE_ERR_UNSUPPORTED, fn, "E=%lld exceeds %lld", E, MOE_MAX_EXPERTS);
  if (k < 1 || k > E) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "k=%lld must be in [1, E=%lld]", k, E);
  if (k > MOE_MAX_TOPK) return fail(MOE_ERR_UNSUPPORTED, fn, "k=%lld exceeds %lld", k, MOE_MAX_TOPK);
  return Check{};
}

Check tokens(const char* fn, int64_t T, int32_t k) {
  if (T < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "T=%lld is negative", T);
  if (T > 0 && T > INT32_MAX / k)
    return fail(MOE_ERR_INVALID_ARGUMENT, fn, "T=%lld times k=%lld exceeds INT32_MAX", T, k);
  return Check{};
}

Check dim64(const char* fn, const char* name, int32_t v) {
  if (v < 64 || v % 64 != 0) {
    Check c;
    c.status = MOE_ERR_INVALID_ARGUMENT;
    char buf[160];
    std::snprintf(buf, sizeof buf, "%s: %s=%d must be a positive multiple of 64", fn, name, v);
    c.msg = buf;
    return c;
  }
  return Check{};
}

Check dtype(const char* fn, int dt) {
  if (dt != MOE_DTYPE_F32 && dt != MOE_DTYPE_BF16)
    return fail(MOE_ERR_UNSUPPORTED, fn, "unknown dtype %lld", dt);
  return Check{};
}

size_t elt(int dt) { return dt == MOE_DTYPE_F32 ? 4 : 2; }

#define MOE_TRY(expr)              \
  do {                             \
    Check _c = (expr);             \
    if (!_c.ok()) return _c;       \
  } while (0)

}  // namespace

int64_t permute_units(int64_t R) { return (R + kPermuteUnit - 1) / kPermuteUnit; }

size_t permute_workspace_bytes(int64_t T, int32_t E, int32_t k) {
  if (T <= 0 || E < 1 || k < 1) return 0;
  // one count per (unit, expert); units padded to a whole block of 4
  int64_t units = (permute_units(T * k) + 3) / 4 * 4;
  return align256(size_t(units) * size_t(E) * sizeof(int32_t));
}

size_t ffn_queue_offset(int32_t E) { return align256(size_t(E + 1) * sizeof(int32_t)); }
size_t ffn_h_offset(int32_t E) { return ffn_queue_offset(E) + 256; }

size_t ffn_partial_offset(int64_t R, int32_t E, int32_t F, moe_dtype dt) {
  return ffn_h_offset(E) + align256(size_t(R) * size_t(F) * elt(dt));
}

size_t ffn_tail_partial_bytes(int64_t R, int32_t E, int32_t H, int32_t F, int bk) {
  if (R <= 0 || E < 1 || H < 1 || F / bk < 2 * kMinPieceSteps) return 0;
  // The grid never exceeds the output-tile bound, and the pieces never exceed the grid;
  // a slot holds a tile of up to kTileRowsMax rows.
  const int64_t mtiles = (R + int64_t(E) * (kTileRows - 1)) / kTileRows;
  const int64_t tiles = mtiles * ((H + kTileCols - 1) / kTileCols);
  const int64_t slots = tiles < kMaxTailPieces ? tiles : kMaxTailPieces;
  return size_t(slots) * kTileRowsMax * kTileCols * sizeof(float);
}

size_t ffn_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F, moe_dtype dt) {
  if (R <= 0 || E < 1 || F < 1) return 0;
  const size_t partial = dt == MOE_DTYPE_BF16 ? ffn_tail_partial_bytes(R, E, H, F, 64) : 0;
  return ffn_partial_offset(R, E, F, dt) + partial;
}

Check validate_route(const float* logits, int64_t T, int32_t E, int32_t k, int32_t renormalize,
                     const int32_t* ids, const float* w) {
  const char* fn = "moe_route";
  MOE_TRY(experts_topk(fn, E, k));
  MOE_TRY(tokens(fn, T, k));
  if (renormalize != 0 && renormalize != 1)
    return fail(MOE_ERR_INVALID_ARGUMENT, fn, "renormalize=%lld must be 0 or 1", renormalize);
  if (T == 0) return Check{};
  MOE_TRY(ptr(fn, "logits", logits));
  MOE_TRY(ptr(fn, "topk_ids", ids));
  MOE_TRY(ptr(fn, "topk_weights", w));
  return Check{};
}

Check validate_router_topk(const void* x, const void* w, int64_t T, int32_t E, int32_t k, int32_t H,
                           int32_t renormalize, const float* logits, const int32_t* ids, const float* wts) {
  const char* fn = "moe_router_topk";
  MOE_TRY(experts_topk(fn, E, k));
  if (E > MOE_MAX_ROUTER_EXPERTS)
    return fail(MOE_ERR_UNSUPPORTED, fn, "E=%lld exceeds %lld for the fused router", E, MOE_MAX_ROUTER_EXPERTS);
  MOE_TRY(tokens(fn, T, k));
  MOE_TRY(dim64(fn, "H", H));
  // the router matrix is addressed with 32-bit byte offsets
  if (int64_t(E) * int64_t(H) * 2 >= (int64_t(1) << 31))
    return fail(MOE_ERR_UNSUPPORTED, fn, "E=%lld x H=%lld router matrix exceeds 2 GiB", E, H);
  if (renormalize != 0 && renormalize != 1)
    return fail(MOE_ERR_INVALID_ARGUMENT, fn, "renormalize=%lld must be 0 or 1", renormalize);
  if (T == 0) return Check{};
  MOE_TRY(ptr(fn, "x", x));
  MOE_TRY(ptr(fn, "w_router", w));
  if (logits != nullptr) MOE_TRY(ptr(fn, "logits", logits));
  MOE_TRY(ptr(fn, "topk_ids", ids));
  MOE_TRY(ptr(fn, "topk_weights", wts));
  return Check{};
}

Check validate_permute(const int32_t* ids, const void* x, int64_t T, int32_t E, int32_t k, int32_t H,
                       int dt, const int32_t* counts, const int32_t* offsets, const int32_t* sorted_tok,
                       const int32_t* dest, const void* x_perm, const void* ws, size_t ws_bytes) {
  const char* fn = "moe_permute";
  MOE_TRY(experts_topk(fn, E, k));
  MOE_TRY(tokens(fn, T, k));
  MOE_TRY(dim64(fn, "H", H));
  MOE_TRY(dtype(fn, dt));
  if (T == 0) return Check{};
  MOE_TRY(ptr(fn, "expert_counts", counts));
  MOE_TRY(ptr(fn, "expert_offsets", offsets));
  MOE_TRY(ptr(fn, "topk_ids", ids));
  MOE_TRY(ptr(fn, "sorted_token_ids", sorted_tok));
  MOE_TRY(ptr(fn, "dest_rows", dest));
  if (x_perm != nullptr) {            // x_perm NULL: only the maps are produced, x is not read
    MOE_TRY(ptr(fn, "x", x));
    MOE_TRY(ptr(fn, "x_perm", x_perm));
  }
  size_t need = permute_workspace_bytes(T, E, k);
  if (ws_bytes < need)
    return fail(MOE_ERR_WORKSPACE_TOO_SMALL, fn, "workspace %lld bytes < %lld needed",
                (long long)ws_bytes, (long long)need);
  MOE_TRY(ptr(fn, "ws", ws));
  return Check{};
}

Check validate_permute_static(const int32_t* ids, const void* x, int64_t T, int32_t E, int32_t k, int32_t H,
                              int dt, const int32_t* counts, const int32_t* offsets, const int32_t* sorted_tok,
                              const int32_t* dest, const void* x_perm) {
  const char* fn = "moe_permute_static";
  MOE_TRY(experts_topk(fn, E, k));
  MOE_TRY(tokens(fn, T, k));
  MOE_TRY(dim64(fn, "H", H));
  MOE_TRY(dtype(fn, dt));
  if (T == 0) return Check{};
  MOE_TRY(ptr(fn, "expert_counts", counts));
  MOE_TRY(ptr(fn, "expert_offsets", offsets));
  MOE_TRY(ptr(fn, "topk_ids", ids));
  MOE_TRY(ptr(fn, "sorted_token_ids", sorted_tok));
  MOE_TRY(ptr(fn, "dest_rows", dest));
  if (x_perm != nullptr) {
    MOE_TRY(ptr(fn, "x", x));
    MOE_TRY(ptr(fn, "x_perm", x_perm));
  }
  const size_t need = permute_workspace_bytes(T, E, k);
  if (need > kPermuteStaticScratchBytes)
    return fail(MOE_ERR_UNSUPPORTED, fn, "needs %lld bytes of scratch, more than the static %lld",
                (long long)need, (long long)kPermuteStaticScratchBytes);
  return Check{};
}

namespace {

// Checks shared by both grouped-FFN entry points; `act` is x_perm or x.
Check ffn_common(const char* fn, const char* act_name, const void* act, const int32_t* offsets, int64_t R,
                 int32_t E, int32_t H, int32_t F, const void* wg, const void* wu, const void* wd, int dt,
                 const void* y_perm, const void* ws, size_t ws_bytes) {
  if (E < 1) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "E=%lld must be >= 1", E);
  if (E > MOE_MAX_EXPERTS) return fail(MOE_ERR_UNSUPPORTED, fn, "E=%lld exceeds %lld", E, MOE_MAX_EXPERTS);
  if (R < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "R=%lld is negative", R);
  if (R > INT32_MAX) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "R=%lld exceeds INT32_MAX", R);
  MOE_TRY(dim64(fn, "H", H));
  MOE_TRY(dim64(fn, "F", F));
  MOE_TRY(dtype(fn, dt));
  // The GEMM kernels address one expert's weight matrix with 32-bit byte offsets.
  if (int64_t(H) * int64_t(F) * int64_t(elt(dt)) >= (int64_t(1) << 31) || H > (1 << 20) || F > (1 << 20))
    return fail(MOE_ERR_UNSUPPORTED, fn, "H=%lld x F=%lld expert matrix exceeds 2 GiB", H, F);
  if (R == 0) return Check{};
  MOE_TRY(ptr(fn, act_name, act));
  MOE_TRY(ptr(fn, "expert_offsets", offsets));
  MOE_TRY(ptr(fn, "w_gate", wg));
  MOE_TRY(ptr(fn, "w_up", wu));
  MOE_TRY(ptr(fn, "w_down", wd));
  MOE_TRY(ptr(fn, "y_perm", y_perm));
  size_t need = ffn_workspace_bytes(R, E, H, F, moe_dtype(dt));
  if (ws_bytes < need)
    return fail(MOE_ERR_WORKSPACE_TOO_SMALL, fn, "workspace %lld bytes < %lld needed",
                (long long)ws_bytes, (long long)need);
  MOE_TRY(ptr(fn, "ws", ws));
  return Check{};
}

}  // namespace

Check validate_ffn(const void* x_perm, const int32_t* offsets, int64_t R, int32_t E, int32_t H,
                   int32_t F, const void* wg, const void* wu, const void* wd, int dt,
                   const void* y_perm, const void* ws, size_t ws_bytes) {
  return ffn_common("moe_grouped_ffn", "x_perm", x_perm, offsets, R, E, H, F, wg, wu, wd, dt, y_perm, ws,
                    ws_bytes);
}

Check validate_ffn_gather(const void* x, const int32_t* sorted_tok, int64_t T, const int32_t* offsets,
                          int64_t R, int32_t E, int32_t H, int32_t F, const void* wg, const void* wu,
                          const void* wd, int dt, const void* y_perm, const void* ws, size_t ws_bytes) {
  const char* fn = "moe_grouped_ffn_gather";
  if (T < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "T=%lld is negative", T);
  if (R > 0 && T == 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "R=%lld rows but T=0 tokens", R);
  MOE_TRY(ffn_common(fn, "x", x, offsets, R, E, H, F, wg, wu, wd, dt, y_perm, ws, ws_bytes));
  if (R == 0) return Check{};
  MOE_TRY(ptr(fn, "sorted_token_ids", sorted_tok));
  return Check{};
}

namespace {

Check dim128(const char* fn, const char* name, int32_t v) {
  if (v < 128 || v % 128 != 0) {
    Check c;
    c.status = MOE_ERR_INVALID_ARGUMENT;
    char buf[160];
    std::snprintf(buf, sizeof buf, "%s: %s=%d must be a positive multiple of 128", fn, name, v);
    c.msg = buf;
    return c;
  }
  return Check{};
}

}  // namespace

size_t mxfp8_scale_bytes(int64_t rows, int32_t K) {
  if (rows <= 0 || K <= 0) return 0;
  return size_t(rows) * size_t(K) / 32;
}

size_t ffn_mxfp8_h_scales_offset(int64_t R, int32_t E, int32_t F) {
  return ffn_h_offset(E) + align256(size_t(R) * size_t(F));
}

size_t ffn_mxfp8_partial_offset(int64_t R, int32_t E, int32_t F) {
  return ffn_mxfp8_h_scales_offset(R, E, F) + align256(mxfp8_scale_bytes(R, F));
}

size_t ffn_mxfp8_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F) {
  if (R <= 0 || E < 1 || F < 1 || H < 1) return 0;
  return ffn_mxfp8_partial_offset(R, E, F) + ffn_tail_partial_bytes(R, E, H, F, 128);
}

Check validate_quantize_mxfp8(const void* src, const int32_t* row_map, int64_t rows_out, int64_t rows_src,
                              int32_t K, const void* codes, const void* scales) {
  const char* fn = "moe_quantize_mxfp8";
  if (rows_out < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "rows_out=%lld is negative", rows_out);
  if (rows_src < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "rows_src=%lld is negative", rows_src);
  MOE_TRY(dim128(fn, "K", K));
  if (row_map == nullptr && rows_out > rows_src)
    return fail(MOE_ERR_INVALID_ARGUMENT, fn, "rows_out=%lld > rows_src=%lld without a row_map", rows_out,
                rows_src);
  if (rows_out == 0) return Check{};
  if (rows_src == 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "rows_out=%lld rows from rows_src=0", rows_out);
  MOE_TRY(ptr(fn, "src", src));
  if (row_map != nullptr) MOE_TRY(ptr(fn, "row_map", row_map));
  MOE_TRY(ptr(fn, "codes", codes));
  MOE_TRY(ptr(fn, "scales", scales));
  return Check{};
}

Check validate_ffn_mxfp8(const void* x, const void* xs, const int32_t* offsets, int64_t R, int32_t E, int32_t H,
                         int32_t F, const void* wg, const void* wgs, const void* wu, const void* wus,
                         const void* wd, const void* wds, const void* y_perm, const void* ws, size_t ws_bytes) {
  const char* fn = "moe_grouped_ffn_mxfp8";
  if (E < 1) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "E=%lld must be >= 1", E);
  if (E > MOE_MAX_EXPERTS) return fail(MOE_ERR_UNSUPPORTED, fn, "E=%lld exceeds %lld", E, MOE_MAX_EXPERTS);
  if (R < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "R=%lld is negative", R);
  if (R > INT32_MAX) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "R=%lld exceeds INT32_MAX", R);
  MOE_TRY(dim128(fn, "H", H));
  MOE_TRY(dim128(fn, "F", F));
  // 32-bit byte offsets: one expert matrix, each weight scale array, and the
  // row scale arrays of x and h.
  const int64_t lim = int64_t(1) << 31;
  if (int64_t(H) * F >= lim || int64_t(E) * H * F / 32 >= lim)
    return fail(MOE_ERR_UNSUPPORTED, fn, "H=%lld x F=%lld experts exceed the 2 GiB addressing", H, F);
  if (R * int64_t(H > F ? H : F) / 32 >= lim)
    return fail(MOE_ERR_UNSUPPORTED, fn, "R=%lld rows: a row scale array reaches 2 GiB", R);
  if (R == 0) return Check{};
  MOE_TRY(ptr(fn, "x_codes", x));
  MOE_TRY(ptr(fn, "x_scales", xs));
  MOE_TRY(ptr(fn, "expert_offsets", offsets));
  MOE_TRY(ptr(fn, "wg_codes", wg));
  MOE_TRY(ptr(fn, "wg_scales", wgs));
  MOE_TRY(ptr(fn, "wu_codes", wu));
  MOE_TRY(ptr(fn, "wu_scales", wus));
  MOE_TRY(ptr(fn, "wd_codes", wd));
  MOE_TRY(ptr(fn, "wd_scales", wds));
  MOE_TRY(ptr(fn, "y_perm", y_perm));
  size_t need = ffn_mxfp8_workspace_bytes(R, E, H, F);
  if (ws_bytes < need)
    return fail(MOE_ERR_WORKSPACE_TOO_SMALL, fn, "workspace %lld bytes < %lld needed", (long long)ws_bytes,
                (long long)need);
  MOE_TRY(ptr(fn, "ws", ws));
  return Check{};
}

Check validate_ffn_mxfp8_gather(const void* x, const void* xs, const int32_t* sorted_tok, int64_t T,
                                const int32_t* offsets, int64_t R, int32_t E, int32_t H, int32_t F, const void* wg,
                                const void* wgs, const void* wu, const void* wus, const void* wd, const void* wds,
                                const void* y_perm, const void* ws, size_t ws_bytes) {
  const char* fn = "moe_grouped_ffn_mxfp8_gather";
  if (T < 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "T=%lld is negative", T);
  if (R > 0 && T == 0) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "R=%lld rows but T=0 tokens", R);
  Check c = validate_ffn_mxfp8(x, xs, offsets, R, E, H, F, wg, wgs, wu, wus, wd, wds, y_perm, ws, ws_bytes);
  if (!c.ok()) {
    // report under this entry point's name
    const std::string other = "moe_grouped_ffn_mxfp8";
    if (c.msg.compare(0, other.size(), other) == 0) c.msg = std::string(fn) + c.msg.substr(other.size());
    return c;
  }
  if (R == 0) return Check{};
  // token rows are addressed with 32-bit byte offsets
  if (T * int64_t(H) >= (int64_t(1) << 31))
    return fail(MOE_ERR_UNSUPPORTED, fn, "x codes of T=%lld rows reach 2 GiB for the gather", T);
  MOE_TRY(ptr(fn, "sorted_token_ids", sorted_tok));
  return Check{};
}

Check validate_combine(const void* y_perm, const int32_t* dest, const float* w, const void* y_shared,
                       int64_t T, int32_t k, int32_t H, int dt, const void* y) {
  const char* fn = "moe_combine";
  if (k < 1) return fail(MOE_ERR_INVALID_ARGUMENT, fn, "k=%lld must be >= 1", k);
  if (k > MOE_MAX_TOPK) return fail(MOE_ERR_UNSUPPORTED, fn, "k=%lld exceeds %lld", k, MOE_MAX_TOPK);
  MOE_TRY(tokens(fn, T, k));
  MOE_TRY(dim64(fn, "H", H));
  MOE_TRY(dtype(fn, dt));
  if (T == 0) return Check{};
  MOE_TRY(ptr(fn, "y_perm", y_perm));
  MOE_TRY(ptr(fn, "dest_rows", dest));
  MOE_TRY(ptr(fn, "topk_weights", w));
  if (y_shared != nullptr) MOE_TRY(ptr(fn, "y_shared", y_shared));
  MOE_TRY(ptr(fn, "y", y));
  return Check{};
}

}  // namespace moe
