/*
 * moe.h - C ABI of the MI355X (gfx950) MoE-layer hot path.
 *
 * One Mixture-of-Experts layer over an expert-level batch: the module the
 * paper's forward pass (Algorithm 1) runs on the hidden states COMBINEd from
 * many yielded sequences, h_out <- MoE(h, l).  The layer is the top-k
 * softmax-gated SwiGLU expert layer of the Mixtral and DeepSeek models the
 * paper evaluates (Section 6, Models); its motivation is sparse expert
 * activation with uneven expert popularity (Section 2.2, Insight 1) and the
 * large expert batch needed to saturate the GPU (Section 7, batch-size regime).
 *
 * Four calls, issued in order on one stream, make the layer:
 *   moe_route        logits -> top-k expert ids and gate weights
 *   moe_permute      ids, x -> per-expert counts, offsets, row maps, x_perm
 *   moe_grouped_ffn  x_perm -> y_perm, each expert's SwiGLU FFN on its rows
 *   moe_combine      y_perm -> y, gate-weighted sum of each token's k rows
 * A shared (always active) expert is one more moe_grouped_ffn call with E = 1
 * over x itself, whose output moe_combine adds with weight 1.
 *
 * Conventions (all calls)
 *   - Every pointer argument is a DEVICE pointer unless stated otherwise, owned
 *     by the caller.  The library never allocates, frees or synchronizes in
 *     these calls: work is enqueued on `stream` (a hipStream_t; NULL is the
 *     default stream) and the call returns.  Buffers must not overlap.
 *   - Row-major layouts.  Shapes are given as [rows, cols].
 *   - Every base pointer must be 16-byte aligned.
 *   - Validation is done on the host before anything is enqueued.  On an error
 *     nothing is written and nothing is launched; moe_last_error() then holds
 *     a message naming the argument.  T = 0 (or R = 0) returns MOE_OK and
 *     enqueues nothing; pointers may then be NULL.
 *   - Not checked (preconditions): finite logits; expert ids in [0, E) and
 *     distinct within a token (moe_route guarantees both); offsets consistent
 *     with R; buffers large enough for the stated shapes.
 *   - Device faults surface asynchronously at the caller's next synchronization.
 *   - Thread-safe; calls on different streams are independent.
 *   - Deterministic: identical inputs give bitwise-identical outputs (no atomics
 *     decide any result).
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARGUMENT = 1,    /* null pointer, bad size, misalignment */
    MOE_ERR_UNSUPPORTED = 2,         /* E > 256, k > 16, unknown dtype */
    MOE_ERR_WORKSPACE_TOO_SMALL = 3,
    MOE_ERR_HIP = 4                  /* a HIP runtime call or kernel launch failed */
} moe_status;

typedef enum {
    MOE_DTYPE_F32 = 0,               /* fp32 activations and weights, fp32 arithmetic */
    MOE_DTYPE_BF16 = 1               /* bf16 activations and weights, fp32 accumulation */
} moe_dtype;

typedef void* moe_stream;            /* hipStream_t */

#define MOE_ABI_VERSION 1
#define MOE_MAX_EXPERTS 256
#define MOE_MAX_TOPK 16
#define MOE_MAX_ROUTER_EXPERTS 64   /* moe_router_topk */

/* ABI version of the loaded library (MOE_ABI_VERSION). */
int moe_abi_version(void);

/* Static description of a status code; never NULL. */
const char* moe_status_string(int status);

/* Message of the last failed call on this host thread ("" if none).  The
 * pointer stays valid until the next call on the same thread. */
const char* moe_last_error(void);

/*
 * moe_route - top-k gating (the MoE gate the expert batch reaches; the paper's
 * Section 2.2 expert selection).
 *
 *   logits        f32 [T, E]   gating logits (the router GEMM is the caller's)
 *   topk_ids      i32 [T, k]   out: slot 0 holds the largest logit
 *   topk_weights  f32 [T, k]   out: gate weights
 *
 * Order: larger logit first; equal logits (including +0 and -0) go to the
 * lower expert id.  Selection compares the fp32 logits exactly.  Weights:
 * p_e = exp(l_e - l_max); renormalize = 1 gives p / sum over the k selected,
 * renormalize = 0 gives p / sum over all E.  exp and the division are fp32.
 * Errors: INVALID_ARGUMENT for T < 0, E < 1, k < 1, k > E, T*k > INT32_MAX,
 * renormalize not 0/1, null or misaligned pointers; UNSUPPORTED for E > 256 or
 * k > 16.
 */
moe_status moe_route(const float* logits, int64_t T, int32_t E, int32_t k, int32_t renormalize,
                     int32_t* topk_ids, float* topk_weights, moe_stream stream);

/*
 * moe_router_topk - the MoE gate with its router GEMM: logits = x . w_router^T
 * computed on the matrix cores (bf16 operands, fp32 accumulation), then the
 * selection and gate weights of moe_route on those fp32 logits (the MoE gate
 * whose batch Section 7 sizes).  The logits stay on chip unless `logits` is given.
 *
 *   x             bf16 [T, H]   hidden states
 *   w_router      bf16 [E, H]   router matrix, one K-contiguous row per expert
 *   logits        f32  [T, E]   optional out (NULL: not written)
 *   topk_ids, topk_weights      as moe_route
 *
 * Errors: as moe_route, plus INVALID_ARGUMENT for H not a positive multiple of
 * 64 and UNSUPPORTED for E > 64 (MOE_MAX_ROUTER_EXPERTS) or a router matrix of
 * 2 GiB or more.
 */
moe_status moe_router_topk(const void* x, const void* w_router, int64_t T, int32_t E, int32_t k, int32_t H,
                           int32_t renormalize, float* logits, int32_t* topk_ids, float* topk_weights,
                           moe_stream stream);

/*
 * moe_permute - group the T*k (token, slot) assignments by expert and gather
 * each assignment's hidden row (the expert-level batch built by COMBINE,
 * Section 4.2 and Algorithm 1, regrouped per expert).
 *
 *   topk_ids          i32 [T, k]      expert of each assignment (from moe_route)
 *   x                 dt  [T, H]      hidden states
 *   expert_counts     i32 [E]         out: rows per expert
 *   expert_offsets    i32 [E + 1]     out: exclusive prefix sum, offsets[E] = T*k
 *   sorted_token_ids  i32 [T*k]       out: source token of each grouped row
 *   dest_rows         i32 [T, k]      out: grouped row of assignment (t, j)
 *   x_perm            dt  [T*k, H]    out: x_perm[r] = x[sorted_token_ids[r]], or NULL:
 *                                     then only the maps are produced and x is not read
 *                                     (x may be NULL); moe_grouped_ffn_gather reads the
 *                                     rows through sorted_token_ids instead
 *   ws, ws_bytes      device scratch of at least moe_permute_workspace_bytes()
 *
 * Expert e owns rows offsets[e] .. offsets[e+1]-1, holding its tokens in
 * ascending token order (a stable counting sort).
 * Errors: as moe_route, plus INVALID_ARGUMENT for H < 64 or H % 64 != 0,
 * UNSUPPORTED for an unknown dtype, WORKSPACE_TOO_SMALL.
 */
size_t moe_permute_workspace_bytes(int64_t T, int32_t E, int32_t k);
moe_status moe_permute(const int32_t* topk_ids, const void* x, int64_t T, int32_t E, int32_t k,
                       int32_t H, moe_dtype dt, int32_t* expert_counts, int32_t* expert_offsets,
                       int32_t* sorted_token_ids, int32_t* dest_rows, void* x_perm,
                       void* ws, size_t ws_bytes, moe_stream stream);

/*
 * moe_permute_static - moe_permute for callers that cannot allocate: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * takes no workspace and allocates nothing: its scratch (per-expert counts of
 * blocks of assignments) is a static device array of
 * MOE_PERMUTE_STATIC_SCRATCH_BYTES that the library holds on every device it
 * runs on until the process ends.  Arguments, outputs and results are those of
 * moe_permute, bit for bit.
 *
 * Calls that overlap on one device (e.g. on two streams) share that array and
 * race; serialize them.  Nothing in the array needs clearing between calls.
 * Errors: as moe_permute, without WORKSPACE_TOO_SMALL; UNSUPPORTED when
 * moe_permute_workspace_bytes(T, E, k) exceeds MOE_PERMUTE_STATIC_SCRATCH_BYTES
 * (4 MiB: e.g. up to 2^24 assignments with 64 experts, 2^22 with 256); HIP when
 * the array's device address cannot be obtained.
 */
#define MOE_PERMUTE_STATIC_SCRATCH_BYTES (4u << 20)
moe_status moe_permute_static(const int32_t* topk_ids, const void* x, int64_t T, int32_t E, int32_t k,
                              int32_t H, moe_dtype dt, int32_t* expert_counts, int32_t* expert_offsets,
                              int32_t* sorted_token_ids, int32_t* dest_rows, void* x_perm, moe_stream stream);

/*
 * moe_grouped_ffn - every expert's SwiGLU FFN on its own rows, as one grouped
 * GEMM pair (the expert computation of the MoE module in Algorithm 1).
 *
 *   x_perm          dt  [R, H]     rows grouped by expert
 *   expert_offsets  i32 [E + 1]    DEVICE array; group e = rows offsets[e]..offsets[e+1]-1
 *   w_gate, w_up    dt  [E, F, H]  K-contiguous (each row is one output feature)
 *   w_down          dt  [E, H, F]  K-contiguous
 *   y_perm          dt  [R, H]     out: W_down[e] (silu(W_gate[e] x) * (W_up[e] x))
 *   ws, ws_bytes    device scratch of at least moe_grouped_ffn_workspace_bytes();
 *                   it holds the intermediate h [R, F] and (bf16) fp32 partial
 *                   sums of down-projection tiles split along k
 *
 * silu(z) = z / (1 + exp(-z)).  bf16: fp32 accumulation, h and y_perm rounded
 * to bf16 (nearest even).  f32: fp32 throughout.  Group sizes are read on the
 * device only (no host readback).  Results are deterministic for a given device
 * and compute-unit budget (moe_set_cu_budget): when the last round of
 * down-projection tiles would leave the grid mostly idle, those tiles are
 * computed in pieces along k and their fp32 partial sums added in piece order,
 * so their rounding depends on the grid size.
 * Errors: INVALID_ARGUMENT for R < 0, E < 1, H or F not a positive multiple of
 * 64, R > INT32_MAX, null or misaligned pointers; UNSUPPORTED for E > 256 or
 * an unknown dtype; WORKSPACE_TOO_SMALL.
 */
size_t moe_grouped_ffn_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F, moe_dtype dt);
moe_status moe_grouped_ffn(const void* x_perm, const int32_t* expert_offsets, int64_t R, int32_t E,
                           int32_t H, int32_t F, const void* w_gate, const void* w_up,
                           const void* w_down, moe_dtype dt, void* y_perm, void* ws,
                           size_t ws_bytes, moe_stream stream);

/*
 * moe_grouped_ffn_gather - moe_grouped_ffn reading each grouped row straight
 * from the token rows: row r of group e is x[sorted_token_ids[r]].  The same
 * result as moe_permute's x_perm followed by moe_grouped_ffn, bit for bit, but
 * the grouped copy of the activations (T*k rows) is never written or read.
 *
 *   x                 dt  [T, H]   token rows (any size)
 *   sorted_token_ids  i32 [R]      from moe_permute (R = T*k)
 *   other arguments as moe_grouped_ffn; the workspace size is
 *   moe_grouped_ffn_workspace_bytes(R, E, H, F, dt)
 *
 * Errors: as moe_grouped_ffn, plus INVALID_ARGUMENT for T < 0, R > 0 with
 * T = 0, a NULL or misaligned x or sorted_token_ids.  Token ids are not checked
 * (precondition: 0 <= id < T).
 */
moe_status moe_grouped_ffn_gather(const void* x, const int32_t* sorted_token_ids,
                                  const int32_t* expert_offsets, int64_t T, int64_t R, int32_t E,
                                  int32_t H, int32_t F, const void* w_gate, const void* w_up,
                                  const void* w_down, moe_dtype dt, void* y_perm, void* ws,
                                  size_t ws_bytes, moe_stream stream);

/*
 * MXFP8 expert GEMMs (the paper's MoE GEMMs are FP8: Section 5, the prefill
 * cost estimate with FP8 MoE GEMMs, and Section 5.6).  MXFP8 is the OCP
 * Microscaling format: E4M3 element codes (1 sign, 4 exponent bits with bias 7,
 * 3 mantissa bits; largest value 448) and one E8M0 scale 2^(s - 127) per 32
 * consecutive elements along k, which gfx950's block-scaled MFMA applies itself.
 *
 * Layout of an MXFP8 matrix with `rows` rows and K columns (K % 128 == 0):
 *   codes   u8 [rows, K]                 row-major E4M3 codes
 *   scales  u8 [K / 128][rows][4]        the scale of row r for k in
 *                                        [32 b, 32 b + 32) is the byte
 *                                        scales[((b / 4) * rows + r) * 4 + b % 4]
 * moe_mxfp8_scale_bytes(rows, K) = rows * K / 32.  An expert weight tensor
 * [E, N, K] is the matrix of E * N rows.
 */
size_t moe_mxfp8_scale_bytes(int64_t rows, int32_t K);

/*
 * moe_quantize_mxfp8 - bf16 rows to MXFP8.
 *
 *   src      bf16 [rows_src, K]
 *   row_map  i32 [rows_out] or NULL: output row r quantizes src row row_map[r]
 *            (e.g. sorted_token_ids from moe_permute gives x_perm's order);
 *            NULL requires rows_out <= rows_src and quantizes rows 0..rows_out-1
 *   codes    u8 [rows_out, K]  out;  scales  u8, moe_mxfp8_scale_bytes(rows_out, K)  out
 *
 * Per block of 32: shared exponent floor(log2(max |v|)) - 8 clamped to
 * [-127, 127] (-127 for an all-zero block); codes = v / 2^shared_exp rounded to
 * the nearest E4M3 value, ties to an even mantissa, clamped to +-448, sign bit
 * kept (-0 gives 0x80).  Inputs are finite (not checked).
 * Errors: INVALID_ARGUMENT for rows_out < 0, rows_src < 0, K not a positive
 * multiple of 128, rows_out > rows_src without a row_map, null or misaligned
 * pointers.  Row indices are not checked (precondition: 0 <= row_map[r] < rows_src).
 */
moe_status moe_quantize_mxfp8(const void* src, const int32_t* row_map, int64_t rows_out, int64_t rows_src,
                              int32_t K, uint8_t* codes, uint8_t* scales, moe_stream stream);

/*
 * moe_grouped_ffn_mxfp8 - moe_grouped_ffn with both GEMMs on MXFP8 operands.
 *
 *   x_codes, x_scales    MXFP8 [R, H]    grouped rows (moe_quantize_mxfp8 with row_map =
 *                                        sorted_token_ids)
 *   expert_offsets       i32 [E + 1]     DEVICE array, as moe_grouped_ffn
 *   wg_*, wu_*           MXFP8 [E * F, H] W_gate, W_up quantized along H
 *   wd_*                 MXFP8 [E * H, F] W_down quantized along F
 *   y_perm               bf16 [R, H]     out
 *   ws, ws_bytes         device scratch of at least moe_grouped_ffn_mxfp8_workspace_bytes();
 *                        it holds h [R, F] in MXFP8 and fp32 partial sums of
 *                        down-projection tiles split along k
 *
 * g and u accumulate in fp32 from the dequantized operands (the matrix cores
 * apply the block scales), h = silu(g) * u in fp32 is quantized to MXFP8 along F
 * as moe_quantize_mxfp8 does, and y_perm accumulates in fp32 and is rounded to
 * bf16 (nearest even).  Determinism as moe_grouped_ffn: for a given device and
 * compute-unit budget.
 * Errors: INVALID_ARGUMENT for R < 0, R > INT32_MAX, E < 1, H or F not a
 * positive multiple of 128, null or misaligned pointers; UNSUPPORTED for
 * E > 256 or when a scale array or an expert matrix reaches 2 GiB;
 * WORKSPACE_TOO_SMALL.
 */
size_t moe_grouped_ffn_mxfp8_workspace_bytes(int64_t R, int32_t E, int32_t H, int32_t F);
moe_status moe_grouped_ffn_mxfp8(const uint8_t* x_codes, const uint8_t* x_scales,
                                 const int32_t* expert_offsets, int64_t R, int32_t E, int32_t H, int32_t F,
                                 const uint8_t* wg_codes, const uint8_t* wg_scales, const uint8_t* wu_codes,
                                 const uint8_t* wu_scales, const uint8_t* wd_codes, const uint8_t* wd_scales,
                                 void* y_perm, void* ws, size_t ws_bytes, moe_stream stream);

/*
 * moe_grouped_ffn_mxfp8_gather - moe_grouped_ffn_mxfp8 reading each grouped row's
 * codes and scales straight from the token rows: row r of group e is token
 * sorted_token_ids[r] of x.  x is then quantized once per token (T rows, no
 * row_map) instead of once per assignment; the result equals quantizing with
 * row_map = sorted_token_ids and calling moe_grouped_ffn_mxfp8, bit for bit.
 *
 *   x_codes, x_scales  MXFP8 [T, H]   token rows (T * H < 2^31)
 *   sorted_token_ids   i32 [R]        from moe_permute
 *   other arguments as moe_grouped_ffn_mxfp8 (same workspace size)
 *
 * Errors: as moe_grouped_ffn_mxfp8, plus INVALID_ARGUMENT for T < 0, R > 0 with
 * T = 0, a NULL or misaligned sorted_token_ids; UNSUPPORTED when the codes of x
 * reach 2 GiB.  Token ids are not checked (precondition: 0 <= id < T).
 */
moe_status moe_grouped_ffn_mxfp8_gather(const uint8_t* x_codes, const uint8_t* x_scales,
                                        const int32_t* sorted_token_ids, const int32_t* expert_offsets, int64_t T,
                                        int64_t R, int32_t E, int32_t H, int32_t F, const uint8_t* wg_codes,
                                        const uint8_t* wg_scales, const uint8_t* wu_codes,
                                        const uint8_t* wu_scales, const uint8_t* wd_codes,
                                        const uint8_t* wd_scales, void* y_perm, void* ws, size_t ws_bytes,
                                        moe_stream stream);

/*
 * moe_combine - gate-weighted sum of each token's k expert outputs (the MoE
 * module's output h_out in Algorithm 1).
 *
 *   y_perm        dt  [T*k, H]  expert outputs in grouped order
 *   dest_rows     i32 [T, k]    grouped row of assignment (t, j) (from moe_permute)
 *   topk_weights  f32 [T, k]
 *   y_shared      dt  [T, H]    optional (NULL = none): added with weight 1
 *   y             dt  [T, H]    out: sum_j w[t,j] * y_perm[dest_rows[t,j]] (+ y_shared[t])
 *
 * The sum is formed in fp32 in slot order j = 0..k-1, the shared row added
 * last, then rounded once to dt.  Gather form: no atomics.
 * Errors: INVALID_ARGUMENT for T < 0, k < 1, k > 16 (UNSUPPORTED), H not a
 * positive multiple of 64, T*k > INT32_MAX, null or misaligned pointers.
 */
moe_status moe_combine(const void* y_perm, const int32_t* dest_rows, const float* topk_weights,
                       const void* y_shared, int64_t T, int32_t k, int32_t H, moe_dtype dt, void* y,
                       moe_stream stream);

/*
 * Per-kernel timing (a benchmarking aid, not part of the layer).
 *
 * moe_profiler_start(capacity) creates `capacity` pairs of HIP events on the
 * current device and enables recording: every kernel the library launches
 * afterwards is bracketed by one pair, recorded on its launch stream, until the
 * pool is used up or moe_profiler_stop() is called.  Creating the events is the
 * only allocation, and it happens here, not in the layer calls.  After the
 * caller synchronizes, moe_profiler_record(i, &name, &ms) returns the i-th
 * launch's kernel name (a static string) and its duration in milliseconds.
 * moe_profiler_select(name) restricts recording to launches of the kernel of
 * that name (as moe_profiler_record reports it, e.g. "ffn_gemm1_gate_up"), so
 * that timing one kernel leaves the others' launches untouched; NULL or ""
 * records every launch again.  It applies to launches made after the call.
 * Errors: INVALID_ARGUMENT for capacity < 1 or an index out of range; HIP for
 * an event failure (e.g. the record's stream has not completed).
 */
moe_status moe_profiler_start(int capacity);
moe_status moe_profiler_select(const char* name);
moe_status moe_profiler_stop(void);
int moe_profiler_count(void);
moe_status moe_profiler_record(int i, const char** name, float* ms);

/*
 * moe_set_cu_budget - compute units the library plans its persistent grids for
 * (a scheduling knob, not part of the layer).
 *
 * The grouped GEMMs, route, the fused router and the MXFP8 quantizer launch one
 * workgroup per compute unit (or a multiple of that) and share out their work
 * among them.  With n > 0 they plan for n compute units instead of the
 * device's count (values above the device's count are used as given), so a
 * caller can leave compute units to concurrent streams.  n = 0 restores the
 * device's count.  Results do not depend on it beyond fp32 rounding: how the
 * down projection's last round of tiles is split along k depends on the grid.
 * Process-wide; set it between calls, not while other host threads launch.
 * Errors: INVALID_ARGUMENT for n < 0.
 */
moe_status moe_set_cu_budget(int32_t n);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
