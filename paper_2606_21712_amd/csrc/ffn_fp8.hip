// MXFP8 expert GEMMs on gfx950: quantization to MXFP8 and the grouped SwiGLU FFN
// on MXFP8 operands with the matrix cores' block-scaled MFMA.
//
// MXFP8 (OCP Microscaling): E4M3 element codes plus one E8M0 scale (2^(s-127))
// per 32 consecutive elements along k.  A block's shared exponent is
// floor(log2(max |v|)) - 8, clamped to [-127, 127] (-127 for an all-zero block);
// each element is v / 2^shared_exp rounded to the nearest E4M3 value, ties to
// an even mantissa, clamped to +-448, sign bit kept.
//
// Layouts.  Codes are row-major [rows, K].  Scales are k-step-major: the four
// scales of row r for k in [128 kt, 128 kt + 128) are the bytes
// scales[(kt * rows + r) * 4 + 0..3], so one GEMM step finds the scales of its
// 256 tile rows in one contiguous kilobyte.
//
// v_mfma_scale_f32_32x32x64_f8f6f4 (measured on gfx950 with in-bounds probes):
// lane l holds row l % 32 and, for half h = l / 32, bytes 0-15 = k [16h, 16h+16)
// and bytes 16-31 = k [32+16h, 32+16h+16) of the instruction's 64; the k block
// [0, 32) of row i takes its scale from lane i, the block [32, 64) from lane
// i + 32, and op_sel picks the byte of the scale register (the others are
// ignored).
//
// The GEMM is the bf16 kernel's design (persistent workgroups on an atomic
// tile queue, 256 x 256 tiles, 8 wavefronts of 128 x 64, two LDS stages filled
// by direct global->LDS loads with an XOR swizzle) with 128 k per step: a
// step moves the same 64 KB of operand bytes as a bf16 step and does twice the
// flops.  GEMM-1 quantizes h to MXFP8 in its epilogue straight from the fp32
// SwiGLU values: the 32 features of one row block are one MFMA tile, held by
// lanes l and l + 32.
#include <algorithm>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));

// ----------------------------------------------------------------------------- MXFP8 encoding
// floor(log2 amax) - 8 clamped to [-127, 127]; amax >= 0 finite.  A zero or
// subnormal amax (floor(log2) <= -127) clamps to -127.
__device__ __forceinline__ int mx_shared_exp(float amax) {
  const int ef = int((__float_as_uint(amax) >> 23) & 0xFFu);
  if (ef == 0) return -127;
  const int e = ef - 127 - 8;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// 2^-se for se in [-127, 119] (always a normal float).
__device__ __forceinline__ float mx_inv_scale(int se) { return __uint_as_float(uint32_t(127 - se) << 23); }

// E4M3 codes of four values with |v| < 512, packed low byte first: the nearest
// E4M3 value, ties to an even mantissa, magnitudes above 448 saturated to 448,
// the sign bit kept (also for zero).  gfx950's v_cvt_pk_fp8_f32 converts to OCP
// E4M3 rounding to nearest even; clamping to +-448 first gives the saturation.
// For every fp32 input with |v| < 512 this yields the codes of the definition
// (binade e = max(floor(log2 |v|), -6), spacing 2^(e-3), ties to even), which
// was checked over all 2^31 such bit patterns.
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d) {
  auto sat = [](float v) { return __builtin_amdgcn_fmed3f(v, -448.0f, 448.0f); };
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(sat(a), sat(b), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(sat(c), sat(d), w, true);
  return uint32_t(w);
}

// ----------------------------------------------------------------------------- quantize rows
// A block walks whole rows (grid-stride); each thread takes 8 consecutive
// elements per pass, so the 4 threads of a 32-element block are one DPP quad
// (K % 128 == 0 keeps quads inside a row).  Output row r quantizes source row
// row_map[r] (or r).
__global__ __launch_bounds__(256) void quantize_rows_kernel(const uint16_t* __restrict__ src,
                                                           const int32_t* __restrict__ row_map,
                                                           int64_t rows_out, int K,
                                                           uint8_t* __restrict__ codes,
                                                           uint8_t* __restrict__ scales) {
  const int per_row = K / 8;
  for (int64_t r = blockIdx.x; r < rows_out; r += gridDim.x) {
    const int64_t sr = row_map != nullptr ? int64_t(row_map[r]) : r;
    const u32x4* srow = reinterpret_cast<const u32x4*>(src + sr * K);
    uint8_t* crow = codes + r * K;
    // the next pass's 16 bytes are loaded before this pass is encoded
    u32x4 nxt = {0u, 0u, 0u, 0u};
    if (int(threadIdx.x) < per_row) nxt = __builtin_nontemporal_load(srow + threadIdx.x);
    for (int c8 = threadIdx.x; c8 < per_row; c8 += blockDim.x) {
      const u32x4 raw = nxt;
      if (c8 + int(blockDim.x) < per_row) nxt = __builtin_nontemporal_load(srow + c8 + blockDim.x);
      float v[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(raw[i] << 16);
        v[2 * i + 1] = __uint_as_float(raw[i] & 0xFFFF0000u);
      }
      float amax = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
      amax = fmaxf(amax, __uint_as_float(uint32_t(
                             __builtin_amdgcn_update_dpp(0, int(__float_as_uint(amax)), 0xB1, 0xF, 0xF, false))));
      amax = fmaxf(amax, __uint_as_float(uint32_t(
                             __builtin_amdgcn_update_dpp(0, int(__float_as_uint(amax)), 0x4E, 0xF, 0xF, false))));
      const int se = mx_shared_exp(amax);
      const float inv = mx_inv_scale(se);
      u32x2 pk;
      pk[0] = e4m3_pack4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
      pk[1] = e4m3_pack4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv);
      *reinterpret_cast<u32x2*>(crow + c8 * 8) = pk;
      if ((c8 & 3) == 0) {
        const int blk = c8 / 4;                               // block index along K
        scales[(int64_t(blk / 4) * rows_out + r) * 4 + (blk & 3)] = uint8_t(se + 127);
      }
    }
  }
}

// ----------------------------------------------------------------------------- grouped GEMM
constexpr int kBM = 256;
constexpr int kBK = 128;                  // k per step (one byte per element)
constexpr int kRowBytes = kBK;
constexpr int kOpBytes = 256 * kRowBytes; // 32 KB
constexpr int kScaleBytes = 256 * 4;      // one scale dword per tile row and step
constexpr int kWScaleOff = 2 * kOpBytes;
constexpr int kXScaleOff = 2 * kOpBytes + kScaleBytes;
constexpr int kStageBytes = 2 * kOpBytes + 2 * kScaleBytes;
constexpr int kThreads = 512;             // 8 wavefronts: 2 (m) x 4 (n)
constexpr int kEpiBytes = 32 * 144;       // a wavefront's y staging region (32 rows of 128 bytes, padded)
static_assert(kBM == kTileRows, "tile shape");
static_assert(8 * kEpiBytes <= kStageBytes, "epilogue staging fits one stage");
constexpr int kWaitVm0 = 0x0F70;
constexpr int kBufFlags = 0x00020000;

struct GemmArgsF8 {
  int32_t* queue;                 // shared tile counter (TileClaim)
  int32_t* xqueue;                // 8 chunk counters (TileClaim)
  const uint8_t* act;             // [R, K] codes of the grouped rows; with a gather, [T, K] token rows
  const uint8_t* act_scales;      // [K / 128][R][4]; with a gather, [K / 128][T][4]
  const int32_t* gather;          // [R] token of each grouped row (gather only)
  const uint8_t* w0;              // [E * N, K] (GEMM-1: W_gate; GEMM-2: W_down)
  const uint8_t* w0_scales;       // [K / 128][E * N][4]
  const uint8_t* w1;              // GEMM-1: W_up
  const uint8_t* w1_scales;
  uint8_t* h_codes;               // GEMM-1 output [R, N]
  uint8_t* h_scales;              // [N / 128][R][4]
  uint16_t* y;                    // GEMM-2 output [R, N] bf16
  float* partial;                 // GEMM-2: tail-split partial slots [kMaxTailPieces][256][256] fp32
  const int32_t* offsets;
  const int32_t* mtile_prefix;
  int E, K, N, ntiles, R;
  int T;                          // token rows of act (gather only)
};

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

template <bool SWIGLU>
__device__ __forceinline__ int wave_nrow(int wn, int ni) {
  if (SWIGLU) return ni * 128 + wn * 32;
  return wn * 64 + ni * 32;
}

// GATHER: activation row r of the tile list is token row gather[r] of act (codes
// and scales), so the grouped copy is never written.
template <bool SWIGLU, bool GATHER>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_fp8_kernel(GemmArgsF8 p) {
  __shared__ __attribute__((aligned(1024))) uint8_t st0[kStageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[kStageBytes];
  __shared__ int32_t s_pref[kMaxExperts + 1];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_claim[2];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wm = wave >> 2, wn = wave & 3;
  if (p.E < 0) {                  // never taken: keeps the DMA-filled stages' reads
    st0[tid] = 0;
    st1[tid] = 0;
  }
  for (int i = tid; i <= p.E; i += kThreads) {
    s_pref[i] = p.mtile_prefix[i];
    s_off[i] = p.offsets[i];
  }
  __syncthreads();

  const int NT = p.ntiles;
  const int K = p.K;
  const int N = p.N;
  const int KT = K / kBK;
  const int64_t EN = int64_t(p.E) * N;
  // GEMM-2 splits the tiles of its last, partly filled round along k.
  const TailPlan plan = SWIGLU ? TailPlan{int64_t(s_pref[p.E]) * NT, 0, 1}
                               : tail_plan(int64_t(s_pref[p.E]) * NT, int(gridDim.x), KT);
  const int64_t total = plan.full + int64_t(plan.r) * plan.s;
  TileClaim claim(p.xqueue, p.queue, plan.full, s_pref[p.E], p.E);
  if (tid == 0) s_claim[0] = claim.next();
  __syncthreads();

  const int qrow = lane >> 3;
  const int qpos = lane & 7;
  const int rrow = lane & 31;
  const int khalf = lane >> 5;

  for (int it = 0;; ++it) {
    const int64_t L = s_claim[it & 1];
    if (L >= total) break;
    if (tid == 0) s_claim[(it + 1) & 1] = claim.next();
    // a whole tile, or piece j of a tail tile (k steps kt0..kt1, partial slot)
    int64_t Lt = L;
    int kt0 = 0, kt1 = KT, slot = -1;
    if (L >= plan.full) {
      const int q = int(L - plan.full);
      const int j = q % plan.s;
      Lt = plan.full + q / plan.s;
      kt0 = j * KT / plan.s;
      kt1 = (j + 1) * KT / plan.s;
      slot = q;
    }
    const TileCoord tc = decode_tile(Lt, s_pref, s_off, p.E, NT);
    const int e = tc.e, nt = tc.nt, row0 = tc.row0, row_stop = tc.row_stop;

    const int arows = min(kBM, row_stop - row0);
    const int n0 = SWIGLU ? nt * 128 : nt * 256;
    const int wrows = SWIGLU ? min(128, N - n0) : min(256, N - n0);
    const __amdgpu_buffer_rsrc_t ra =
        GATHER ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.act), 0, p.T * K, kBufFlags)
               : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.act) + int64_t(row0) * K, 0, arows * K,
                                                   kBufFlags);
    const int64_t wfirst = (int64_t(e) * N + n0) * K;
    const __amdgpu_buffer_rsrc_t rw0 =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.w0) + wfirst, 0, wrows * K, kBufFlags);
    const __amdgpu_buffer_rsrc_t rw1 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(SWIGLU ? p.w1 : p.w0) + wfirst, 0, wrows * K, kBufFlags);
    // Scale arrays are read whole-array bounded; rows past the tile's group or
    // past N read other rows' (finite) scales, multiplied by zero codes.
    const int64_t act_rows = GATHER ? p.T : p.R;
    const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(p.act_scales), 0, int(int64_t(KT) * act_rows * 4), kBufFlags);
    const __amdgpu_buffer_rsrc_t rsw0 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(p.w0_scales), 0, int(int64_t(KT) * EN * 4), kBufFlags);
    const __amdgpu_buffer_rsrc_t rsw1 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(SWIGLU ? p.w1_scales : p.w0_scales), 0, int(int64_t(KT) * EN * 4), kBufFlags);

    uint32_t aoff[4], woff[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (8 * i + wave) * 8 + qrow;
      const uint32_t cb = uint32_t(swz(r, qpos) * 16);
      if (GATHER) {
        // the token's row; rows past the group end get an offset beyond num_records
        const int grow = row0 + r;
        aoff[i] = grow < row_stop ? uint32_t(p.gather[grow]) * uint32_t(K) + cb : 0x80000000u;
      } else {
        aoff[i] = uint32_t(r) * uint32_t(K) + cb;
      }
      woff[i] = uint32_t(SWIGLU ? (r & 127) : r) * uint32_t(K) + cb;
    }
    // gather: waves 4-7 each load the activation scales of 64 tile rows, one dword
    // per lane (spread over four waves, so no wave issues more than its operand
    // loads plus one): the byte offset of tile row 64 (wave - 4) + lane's token in
    // step 0, or beyond the array
    uint32_t stok;
    {
      const int grow = row0 + 64 * (wave - 4) + lane;
      stok = (GATHER && wave >= 4 && grow < row_stop) ? uint32_t(p.gather[grow]) * 4u : 0x80000000u;
    }
    // scale rows: wave 0 loads the weight tile's 256 scale dwords (GEMM-1: lanes
    // 0-31 the 128 gate rows, lanes 32-63 the up rows), wave 1 the activation tile's
    // (without a gather: contiguous rows, one 16-byte load per lane)
    const uint32_t sw_lane = SWIGLU ? uint32_t((lane & 31) * 16) : uint32_t(lane * 16);

    // A stage's loads: the activation codes first (gathered rows arrive last),
    // then the weight codes, then the scales.
    // k-step order: a down-projection tile of an expert with a single m-tile and
    // rows of at most 8 KB starts at a step of its own (as in the bf16 kernel)
    const int nk = kt1 - kt0;
    const int krot = (!SWIGLU && slot < 0 && tc.mt_e == 1 && K <= 8192) ? int((Lt * 7) % nk) : 0;
    auto issue = [&](uint8_t* stage, int kt) {
      {
        const int q = kt - kt0 + krot;
        kt = kt0 + (q >= nk ? q - nk : q);
      }
      const int kb = kt * kRowBytes;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int blk = 8 * i + wave;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, stage + kOpBytes + blk * 1024, 16, aoff[i], kb, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int blk = 8 * i + wave;
        __builtin_amdgcn_raw_ptr_buffer_load_lds((SWIGLU && i >= 2) ? rw1 : rw0, stage + blk * 1024, 16,
                                                 woff[i], kb, 0, 0);
      }
      // The scale rows' base goes into the per-lane offset, which the buffer range
      // check covers: rows past the end of a scale array read as zeros.
      if (wave == 0) {
        const uint32_t voff = uint32_t((int64_t(kt) * EN + int64_t(e) * N + n0) * 4) + sw_lane;
        if (SWIGLU && lane >= 32)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsw1, stage + kWScaleOff, 16, voff, 0, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsw0, stage + kWScaleOff, 16, voff, 0, 0, 0);
      }
      if (GATHER && wave >= 4) {
        const uint32_t step_off = uint32_t(int64_t(kt) * p.T * 4);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, stage + kXScaleOff + 256 * (wave - 4), 4,
                                                 stok == 0x80000000u ? stok : stok + step_off, 0, 0, 0);
      } else if (!GATHER && wave == 1) {
        const uint32_t voff = uint32_t((int64_t(kt) * p.R + row0) * 4) + uint32_t(lane * 16);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, stage + kXScaleOff, 16, voff, 0, 0, 0);
      }
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;

    // Operand of one 32-row fragment for sub-step s (k [64 s, 64 s + 64) of the
    // step): lane half h takes the 16-byte chunks 4 s + h and 4 s + 2 + h.
    auto frag = [&](const uint8_t* base, int row, int s) {
      const u32x4 lo = *reinterpret_cast<const u32x4*>(base + row * kRowBytes + swz(row, 4 * s + khalf) * 16);
      const u32x4 hi = *reinterpret_cast<const u32x4*>(base + row * kRowBytes + swz(row, 4 * s + 2 + khalf) * 16);
      i32x8 v;
      v[0] = int(lo[0]); v[1] = int(lo[1]); v[2] = int(lo[2]); v[3] = int(lo[3]);
      v[4] = int(hi[0]); v[5] = int(hi[1]); v[6] = int(hi[2]); v[7] = int(hi[3]);
      return v;
    };
    auto compute = [&](const uint8_t* stage) {
      // scale dwords of this step, shifted so that byte 2 s is block 2 s + h
      uint32_t wsc[2], xsc[4];
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        wsc[ni] = *reinterpret_cast<const uint32_t*>(stage + kWScaleOff + (wave_nrow<SWIGLU>(wn, ni) + rrow) * 4) >>
                  (8 * khalf);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        xsc[mi] = *reinterpret_cast<const uint32_t*>(stage + kXScaleOff + (wm * 128 + mi * 32 + rrow) * 4) >>
                  (8 * khalf);
      i32x8 wf[2][2], xf[2][4];
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) wf[0][ni] = frag(stage, wave_nrow<SWIGLU>(wn, ni) + rrow, 0);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) xf[0][mi] = frag(stage + kOpBytes, wm * 128 + mi * 32 + rrow, 0);
      // Raised wave priority for the first sub-step, while the other wavefront
      // of the SIMD issues the step's loads.
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        if (s == 0) {
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) wf[1][ni] = frag(stage, wave_nrow<SWIGLU>(wn, ni) + rrow, 1);
#pragma unroll
          for (int mi = 0; mi < 4; ++mi) xf[1][mi] = frag(stage + kOpBytes, wm * 128 + mi * 32 + rrow, 1);
        }
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 2; ++ni)
            // op_sel must be a literal: byte 2 s of the shifted scale dwords
            acc[mi][ni] = s == 0 ? __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                                       wf[0][ni], xf[0][mi], acc[mi][ni], 0, 0, 0, int(wsc[ni]), 0, int(xsc[mi]))
                                 : __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                                       wf[1][ni], xf[1][mi], acc[mi][ni], 0, 0, 2, int(wsc[ni]), 2, int(xsc[mi]));
        if (s == 0) {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // one LDS read (12 for sub-step 1)
          }
          __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
          __builtin_amdgcn_s_setprio(0);
        } else {
          __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
        }
      }
    };
    const bool active = row0 + wm * 128 < row_stop;
    auto step = [&](uint8_t* cur, uint8_t* nxt, int kt) {
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 1 < kt1) issue(nxt, kt + 1);
      if (active) compute(cur);
    };

    issue(st0, kt0);
    int kt = kt0;
    for (; kt + 2 <= kt1; kt += 2) {
      step(st0, st1, kt);
      step(st1, st0, kt + 1);
    }
    if (kt < kt1) step(st0, st1, kt);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();

    // ---- epilogue: lane holds columns n + 8 blk + 4 khalf + {0..3} of row (lane % 32).
    // The results go through a private LDS region of each wavefront in st1 (free
    // after the barrier above; the next tile writes it only after its first
    // barrier): a lane's pieces of 32 different rows become whole row segments
    // (h codes: 32 bytes, y: 128 bytes).
    uint8_t* ebuf = st1 + wave * kEpiBytes;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      const int rbase = row0 + wm * 128 + mi * 32;             // first row of this 32-row block
      if (rbase >= row_stop) continue;                          // uniform across the wave
      const int row = rbase + rrow;
      if (SWIGLU) {
        // the wave's 32 features of this row: one MX block, split between lanes l and l ^ 32
        float hv[16];
        float amax = 0.f;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          hv[q] = silu(acc[mi][0][q]) * acc[mi][1][q];
          amax = fmaxf(amax, fabsf(hv[q]));
        }
        amax = fmaxf(amax, __shfl_xor(amax, 32));
        const int f0 = n0 + wn * 32;                           // block start, a multiple of 32
        const int se = mx_shared_exp(amax);
        const float inv = mx_inv_scale(se);
        // the codes of the 32 rows x 32 features go through the wavefront's LDS
        // region (rows of 48 bytes) and leave as 16-byte pieces of whole rows
#pragma unroll
        for (int blk = 0; blk < 4; ++blk) {
          const float* hb = hv + blk * 4;
          *reinterpret_cast<uint32_t*>(ebuf + rrow * 48 + blk * 8 + khalf * 4) =
              e4m3_pack4(hb[0] * inv, hb[1] * inv, hb[2] * inv, hb[3] * inv);
        }
        if (row < row_stop && f0 < N && khalf == 0) {
          const int b = f0 / 32;
          p.h_scales[(int64_t(b / 4) * p.R + row) * 4 + (b & 3)] = uint8_t(se + 127);
        }
        const int r = lane >> 1, ch = lane & 1;
        const u32x4 v = *reinterpret_cast<const u32x4*>(ebuf + r * 48 + ch * 16);
        if (rbase + r < row_stop && f0 < N)
          *reinterpret_cast<u32x4*>(p.h_codes + int64_t(rbase + r) * N + f0 + ch * 16) = v;
      } else if (row < row_stop && slot >= 0) {
        // a piece of a tail tile: fp32 partial sums in its slot, tile-local
        // [256 rows][256 columns], added in piece order by the tail reduction
        float* prow = p.partial + (int64_t(slot) * kTileRowsMax + (row - row0)) * kTileCols;
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
#pragma unroll
          for (int blk = 0; blk < 4; ++blk) {
            const int c = wn * 64 + ni * 32 + blk * 8 + khalf * 4;
            if (n0 + c < N) {
              f32x4 v;
#pragma unroll
              for (int q = 0; q < 4; ++q) v[q] = acc[mi][ni][blk * 4 + q];
              *reinterpret_cast<f32x4*>(prow + c) = v;
            }
          }
        }
      } else if (slot < 0) {
        // y: 32 rows x 64 columns, rows of 128 bytes in LDS padded to 144
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
          for (int blk = 0; blk < 4; ++blk) {
            u32x2 pk;
            pk[0] = pack_bf16x2(acc[mi][ni][blk * 4 + 0], acc[mi][ni][blk * 4 + 1]);
            pk[1] = pack_bf16x2(acc[mi][ni][blk * 4 + 2], acc[mi][ni][blk * 4 + 3]);
            *reinterpret_cast<u32x2*>(ebuf + rrow * 144 + (ni * 32 + blk * 8 + khalf * 4) * 2) = pk;
          }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = j * 8 + (lane >> 3);
          const u32x4 v = *reinterpret_cast<const u32x4*>(ebuf + r * 144 + (lane & 7) * 16);
          const int orow = rbase + r;
          const int n = n0 + wn * 64 + (lane & 7) * 8;
          if (orow < row_stop && n < N) *reinterpret_cast<u32x4*>(p.y + int64_t(orow) * N + n) = v;
        }
      }
    }
  }
}

int grid_for(int64_t upper_tiles, int num_cu) {
  const int64_t g = upper_tiles < num_cu ? upper_tiles : num_cu;
  return int(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_quantize_mxfp8(const uint16_t* src, const int32_t* row_map, int64_t rows_out, int K,
                                 uint8_t* codes, uint8_t* scales, int num_cu, hipStream_t s) {
  const int64_t blocks = std::min<int64_t>(rows_out, int64_t(num_cu) * 16);
  MOE_LAUNCH("quantize_mxfp8", quantize_rows_kernel, dim3(unsigned(std::max<int64_t>(blocks, 1))), dim3(256), s,
             src, row_map, rows_out, K, codes, scales);
  return hipGetLastError();
}

hipError_t launch_ffn_mxfp8(const uint8_t* x, const uint8_t* xs, const int32_t* gather, int64_t T,
                            const int32_t* offsets, int64_t R, int E, int H, int F, const uint8_t* wg,
                            const uint8_t* wgs, const uint8_t* wu, const uint8_t* wus, const uint8_t* wd,
                            const uint8_t* wds, uint16_t* y_perm, int32_t* mtile_prefix, int32_t* queues, uint8_t* h,
                            uint8_t* hs, float* partial, int num_cu, hipStream_t s) {
  hipError_t err = launch_tile_prefix(offsets, E, kBM, mtile_prefix, queues, s);
  if (err != hipSuccess) return err;
  const int64_t mtiles_upper = (R + int64_t(E) * (kBM - 1)) / kBM;
  GemmArgsF8 a1{queues, queues + 2, x, xs, gather, wg, wgs, wu, wus, h, hs, nullptr, nullptr, offsets, mtile_prefix,
                E, H, F, F / 128, int(R), int(T)};
  const dim3 grid1(grid_for(mtiles_upper * a1.ntiles, num_cu));
  if (gather != nullptr)
    MOE_LAUNCH("ffn_gemm1_gate_up", (grouped_gemm_fp8_kernel<true, true>), grid1, dim3(kThreads), s, a1);
  else
    MOE_LAUNCH("ffn_gemm1_gate_up", (grouped_gemm_fp8_kernel<true, false>), grid1, dim3(kThreads), s, a1);
  GemmArgsF8 a2{queues + 1, queues + 10, h, hs, nullptr, wd, wds, nullptr, nullptr, nullptr, nullptr, y_perm, partial, offsets,
                mtile_prefix, E, F, H, (H + 255) / 256, int(R), 0};
  const int grid2 = grid_for(mtiles_upper * a2.ntiles, num_cu);
  MOE_LAUNCH("ffn_gemm2_down", (grouped_gemm_fp8_kernel<false, false>), dim3(grid2), dim3(kThreads), s, a2);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_tail_reduce(partial, mtile_prefix, offsets, E, a2.ntiles, grid2, F / kBK, H, y_perm, false, s);
}

}  // namespace moe
