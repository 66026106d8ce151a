// moe_grouped_ffn: every expert's SwiGLU FFN on its own rows, on gfx950.
//
//   GEMM-1  h[r, f]  = silu(x_perm[r] . W_gate[e][f]) * (x_perm[r] . W_up[e][f])
//   GEMM-2  y[r, n]  = h[r] . W_down[e][n]
// for every row r of expert e's group.  Both operands are K-contiguous.
//
// Tile scheduling.  A tiny kernel turns the device-side offsets into a prefix
// of m-tiles per expert (no host readback) and zeroes the tile counters.  The
// GEMM kernels are persistent, one workgroup per compute unit, over the
// flattened tile list, in which an expert's tiles are contiguous, so a hot
// expert simply owns more tiles and an empty one owns none.  Inside an expert
// the order is (block of kGroupM m-tiles, group of kGroupN n-tiles, m-tile,
// n-tile), so 32 consecutive tiles share 4 activation and 8 weight panels.  The
// workgroups of each XCD (dealt round-robin, so workgroup b runs on XCD b % 8)
// claim such chunks of 32 tiles from a counter of their own, every eighth chunk
// of the list, so the 32 compute units of an XCD work on the same panels at the
// same time and share its L2; inside an XCD cheap and costly tiles balance
// dynamically.  Only as many chunks as give every XCD the same number go out
// this way; the remaining tiles (and a split tail's pieces) come from one
// shared counter, so a small problem never leaves an XCD idle while another
// holds whole chunks.  (Measured against one queue over the whole list, same
// inputs: GEMM-1 -1% to -4%, GEMM-2 -4% to -7% on the four bf16 workloads.)
//
// bf16 tile: up to 320 rows of one expert (ceil(rows / 320) m-tiles per expert,
// cut on 32-row blocks: tiling.h) x 256 weight rows x 64 k per step, 8 wavefronts (2 x 4, two per SIMD so one issues MFMAs while
// the other waits), each up to 160 x 64: five 32-row blocks of
// v_mfma_f32_32x32x16_bf16 results, of which a wavefront computes only those
// holding rows of the tile.  The last round of down-projection tiles, when the
// grid would run it mostly idle, is split along k (fp32 partials, reduced in
// piece order by tail_reduce_kernel).
// The weight tile is the MFMA A operand and the activation tile the B operand,
// so each lane ends up holding 4 consecutive output columns of one row: the
// epilogue stores 8 bytes per lane.  For GEMM-1 the weight tile holds 128
// gate rows and the 128 up rows of the same features, so silu(g) * u is formed
// in registers and only h is written.  Tiles move from HBM straight into LDS
// (global_load_lds_dwordx4, no register staging), two stages deep, with the
// 16-byte chunks of each 128-byte row XOR-swizzled so the MFMA operand reads
// are free of bank conflicts; operand fragments are double-buffered in
// registers so LDS latency hides behind the previous sub-step's MFMAs.  After
// each step's barrier a wavefront issues the next stage's weight loads, then
// (at raised wave priority) the first sub-step's MFMAs, then the activation
// loads, so the texture unit is not flooded while the MFMA stream restarts.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

// ----------------------------------------------------------------------------- tile prefix
// Tile counters: GEMM-1's and GEMM-2's queues, then 8 chunk counters of each.
constexpr int kQueueInts = 18;

// prefix[e] = sum_{e' < e} m-tiles of expert e', prefix[E] = total, with
// ceil(count / bm) m-tiles per expert.  One block of 256.
__global__ __launch_bounds__(256) void tile_prefix_kernel(const int32_t* __restrict__ offsets, int E,
                                                         int bm, int32_t* __restrict__ prefix,
                                                         int32_t* __restrict__ queues) {
  const int e = threadIdx.x;
  if (queues != nullptr && e < kQueueInts) queues[e] = 0;      // tile queues of both GEMMs
  int32_t mt = 0;
  if (e < E) {
    const int32_t c = offsets[e + 1] - offsets[e];
    mt = (c + bm - 1) / bm;
  }
  int32_t total;
  const int32_t ex = block_exclusive_scan256(mt, &total);
  if (e < E) prefix[e] = ex;
  if (e == 0) prefix[E] = total;
}

// ----------------------------------------------------------------------------- bf16 MFMA GEMM
constexpr int kBM = 256;                  // m-tile rows of the tile-count bound (ceil(c / 320) <= ceil(c / 256))
constexpr int kBMMax = kTileRowsMax;      // 320
constexpr int kBN = 256;                  // weight rows per tile (GEMM-1: 128 gate + 128 up)
constexpr int kBK = 64;                   // k per pipeline step
constexpr int kRowBytes = kBK * 2;        // one tile row in LDS: 128 bytes = 8 chunks of 16
constexpr int kWOpBytes = kBN * kRowBytes;       // weight tile: 32 KB
constexpr int kAOpBytes = kBMMax * kRowBytes;    // activation tile: 40 KB
constexpr int kStageBytes = kWOpBytes + kAOpBytes;
constexpr int kWaveRows = kBMMax / 2;     // 160 activation rows per wavefront: 5 blocks of 32
constexpr int kGemmThreads = 512;        // 8 wavefronts: 2 (m) x 4 (n), two per SIMD
constexpr int kGroups = 8;                // chunk counters per GEMM (one per XCD)
constexpr int kEpiBytes = 32 * 144;       // a wavefront's epilogue staging region (32 rows)
static_assert(8 * kEpiBytes <= kStageBytes, "epilogue staging fits one stage");
static_assert(kBM == kTileRows && kBN == kTileCols, "tile shape");

struct GemmArgs {
  int32_t* queue;                 // shared tile counter (TileClaim), zeroed by tile_prefix_kernel
  int32_t* xqueue;                // kGroups chunk counters (TileClaim), zeroed likewise
  const uint16_t* act;            // [R, K]; with a gather, the token rows [T, K]
  const int32_t* gather;          // [R] token of each grouped row (gather only)
  const uint16_t* w0;             // [E, N, K] (GEMM-1: W_gate; GEMM-2: W_down)
  const uint16_t* w1;             // [E, N, K] (GEMM-1: W_up)
  uint16_t* out;                  // [R, N]
  float* partial;                 // GEMM-2: tail-split partial slots [kMaxTailPieces][256][256] fp32
  const int32_t* offsets;         // [E + 1]
  const int32_t* mtile_prefix;    // [E + 1]
  int E, K, N, ntiles, R;
  int act_bytes;                  // bytes of act (kTokens gather only; < 2^31)
};

// First tile row of a wavefront's n-subtile ni (0..1).  GEMM-1: ni = 0 is 32
// gate features, ni = 1 the up rows of the same features.
template <bool SWIGLU>
__device__ __forceinline__ int wave_nrow(int wn, int ni) {
  if (SWIGLU) return ni * 128 + wn * 32;
  return wn * 64 + ni * 32;
}

// LDS layout of one operand tile: 256 rows x 128 bytes (64 bf16 of k), the
// sixteen-byte chunk c of row r stored at chunk position c ^ ((r >> 1) & 7).
// gfx950 serves a 16-byte-per-lane LDS read 16 lanes at a time from 64 banks;
// the 16 rows such a group touches then land on 16 distinct 16-byte slots.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// gfx9 s_waitcnt immediate with only vmcnt(0): expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVm0 = 0x0F70;
// Buffer resource word 3 for raw (unformatted, stride 0) buffer loads on gfx9.
constexpr int kBufFlags = 0x00020000;

// Where the activation rows come from.
enum Gather : int {
  kRows = 0,       // act is the grouped rows [R, K]
  kTokens = 1,     // row r is token row gather[r] of act [T, K], act < 2 GiB: one buffer
                   // resource over all of act, 32-bit row offsets
  kTokensWide = 2  // the same for act of any size: 64-bit per-lane row addresses
};

// GATHER != kRows: activation row r of the tile list is row gather[r] of act (the
// token rows themselves), so the grouped copy of the activations is never written.
template <bool SWIGLU, int GATHER>
__global__ __launch_bounds__(kGemmThreads, 1) void grouped_gemm_bf16_kernel(GemmArgs p) {
  // Two pipeline stages, each [weight tile | activation tile].  They are filled by
  // direct global->LDS loads; two distinct objects let the compiler tell them apart.
  __shared__ __attribute__((aligned(1024))) uint8_t st0[kStageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[kStageBytes];
  __shared__ int32_t s_pref[kMaxExperts + 1];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_claim[2];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wm = wave >> 2, wn = wave & 3;

  // The stages are written only by the LDS-DMA loads, which the compiler does not
  // count as stores to them; this never-taken store keeps their reads from being
  // folded away as reads of uninitialized memory.
  if (p.E < 0) {
    st0[tid] = 0;
    st1[tid] = 0;
  }
  for (int i = tid; i <= p.E; i += kGemmThreads) {
    s_pref[i] = p.mtile_prefix[i];
    s_off[i] = p.offsets[i];
  }
  __syncthreads();

  const int NT = p.ntiles;
  const int K = p.K;
  const int N = p.N;
  const int KT = K / kBK;
  // GEMM-2 splits the tiles of its last, partly filled round along k.
  const TailPlan plan = SWIGLU ? TailPlan{int64_t(s_pref[p.E]) * NT, 0, 1}
                               : tail_plan(int64_t(s_pref[p.E]) * NT, int(gridDim.x), KT);
  const int64_t total = plan.full + int64_t(plan.r) * plan.s;
  // Tiles in chunks per XCD, the rest and the tail's pieces from one shared counter (TileClaim).
  TileClaim claim(p.xqueue, p.queue, plan.full, s_pref[p.E], p.E);
  if (tid == 0) s_claim[0] = claim.next();
  __syncthreads();

  // DMA: wave w's pass i fills the 1 KB block blk = 8*i + w of an operand (its rows
  // 8*blk..8*blk+7); lane q lands at byte 16*q of the block: row 8*blk + q/8, chunk
  // position q%8.  Weights: 32 blocks (4 passes); activations: 40 blocks (5 passes).
  const int qrow = lane >> 3;
  const int qpos = lane & 7;
  // MFMA operand reads: row (lane % 32) of a 32-row block, k-chunk 2*s + lane / 32.
  const int rrow = lane & 31;
  const int khalf = lane >> 5;

  for (int it = 0;; ++it) {
    const int64_t L = s_claim[it & 1];
    if (L >= total) break;                                      // uniform: every wave leaves
    if (tid == 0) s_claim[(it + 1) & 1] = claim.next();
    // ---- decode the entry (wave-uniform values, moved to scalar registers): a
    // whole tile, or piece j of a tail tile (k steps kt0..kt1, partial slot).
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
    const TileCoord tc = decode_tile<true>(Lt, s_pref, s_off, p.E, NT);
    const int e = tc.e, nt = tc.nt, row0 = tc.row0, row_stop = tc.row_stop;
    const int arows = row_stop - row0;                           // 1 .. 320

    // ---- buffer resources: rows past the tile (activations) or past N (weights)
    // fall outside num_records and load as zeros.
    const int n0 = SWIGLU ? nt * 128 : nt * 256;
    const int wrows = SWIGLU ? min(128, N - n0) : min(256, N - n0);
    const int64_t rowb = int64_t(K) * 2;
    const __amdgpu_buffer_rsrc_t ra =
        GATHER == kTokens
            ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.act), 0, p.act_bytes, kBufFlags)
            : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.act) + int64_t(row0) * K, 0,
                                                int(arows * rowb), kBufFlags);
    const int64_t wfirst = (int64_t(e) * N + n0) * K;
    const __amdgpu_buffer_rsrc_t rw0 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(p.w0) + wfirst, 0, int(wrows * rowb), kBufFlags);
    const __amdgpu_buffer_rsrc_t rw1 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(SWIGLU ? p.w1 : p.w0) + wfirst, 0, int(wrows * rowb), kBufFlags);
    // Per-lane byte offsets of the DMA passes (constant over the k loop).
    uint32_t aoff[5], woff[4];
    const uint8_t* aptr[5];                 // kTokensWide: the lane's row address
#pragma unroll
    for (int i = 0; i < 5; ++i) {
      const int r = (8 * i + wave) * 8 + qrow;                  // activation row this lane fills
      const uint32_t cb = uint32_t(swz(r, qpos) * 16);          // its logical chunk, in bytes
      const int grow = row0 + r;
      if (GATHER == kTokens) {
        // The token's row; rows past the tile get an offset beyond num_records.
        aoff[i] = grow < row_stop ? uint32_t(p.gather[grow]) * uint32_t(rowb) + cb : 0x80000000u;
      } else if (GATHER == kTokensWide) {
        // No bounds check on these loads: a row past the tile reads the tile's first
        // token row instead, whose products land only in output rows that are
        // never stored.
        const int64_t tok = p.gather[grow < row_stop ? grow : row0];
        aptr[i] = reinterpret_cast<const uint8_t*>(p.act) + tok * rowb + cb;
        aoff[i] = 0;
      } else {
        aoff[i] = uint32_t(r) * uint32_t(rowb) + cb;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (8 * i + wave) * 8 + qrow;
      const uint32_t cb = uint32_t(swz(r, qpos) * 16);
      // GEMM-1: tile rows 0..127 are gate features n0.., rows 128..255 the same up features.
      woff[i] = uint32_t(SWIGLU ? (r & 127) : r) * uint32_t(rowb) + cb;
    }
    // The weight passes and the activation passes of a stage's loads.  Activation
    // passes whose 8 rows all lie past the tile are not issued.
    // k-step order.  A down-projection tile of an expert that has a single m-tile
    // shares its weight panel with no other tile, and with rows of at most 8 KB the
    // same k column of every weight row lands on the same HBM channels, so the
    // tiles running at one time would all ask the same channels at each step:
    // such a tile starts its k loop at a step of its own and wraps around.  (Tiles
    // that share panels keep one order, so the L2 sees their reads together.)
    const int nk = kt1 - kt0;
    const int krot = (!SWIGLU && slot < 0 && tc.mt_e == 1 && K * 2 <= 8192) ? int((Lt * 7) % nk) : 0;
    auto kphys = [&](int kt) {
      const int q = kt - kt0 + krot;
      return kt0 + (q >= nk ? q - nk : q);
    };
    auto issue_w = [&](uint8_t* stage, int kt) {
      const int kb = kphys(kt) * kRowBytes;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int blk = 8 * i + wave;
        __builtin_amdgcn_raw_ptr_buffer_load_lds((SWIGLU && i >= 2) ? rw1 : rw0, stage + blk * 1024, 16,
                                                 woff[i], kb, 0, 0);
      }
    };
    auto issue_a = [&](uint8_t* stage, int kt) {
      const int kb = kphys(kt) * kRowBytes;
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        const int blk = 8 * i + wave;
        if (blk * 8 < arows) {
          if (GATHER == kTokensWide)
            __builtin_amdgcn_global_load_lds(aptr[i] + kb, stage + kWOpBytes + blk * 1024, 16, 0, 0);
          else
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, stage + kWOpBytes + blk * 1024, 16, aoff[i], kb, 0, 0);
        }
      }
    };

    f32x16 acc[5][2];
#pragma unroll
    for (int mi = 0; mi < 5; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;

    // This wavefront's rows: wm * 160 + 32 mi + (lane % 32); NB of its five 32-row
    // blocks hold rows of the tile (0 for the second wavefront row of a short tile:
    // it still loads and synchronizes, and the other wave on its SIMD has the
    // matrix core to itself).
    const int nb = min(5, max(0, (arows - wm * kWaveRows + 31) / 32));

    // One k-loop per block count, so the fragment reads and MFMAs of a step are a
    // fixed unrolled sequence.
    auto kloop = [&](auto nb_c) {
      constexpr int NB = decltype(nb_c)::value;
      auto frags = [&](const uint8_t* stage, int s, bf16x8* wf, bf16x8* xf) {
        const int c = 2 * s + khalf;
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int row = wave_nrow<SWIGLU>(wn, ni) + rrow;
          wf[ni] = *reinterpret_cast<const bf16x8*>(stage + row * kRowBytes + swz(row, c) * 16);
        }
#pragma unroll
        for (int mi = 0; mi < NB; ++mi) {
          const int row = wm * kWaveRows + mi * 32 + rrow;
          xf[mi] = *reinterpret_cast<const bf16x8*>(stage + kWOpBytes + row * kRowBytes + swz(row, c) * 16);
        }
      };
      // MFMAs of a stage; the next stage's activation passes (ktn >= 0) are issued
      // after the first sub-step's MFMAs.
      auto compute = [&](const uint8_t* stage, uint8_t* nxt, int ktn) {
        if constexpr (NB > 0) {
          bf16x8 wf[2][2], xf[2][NB];
          frags(stage, 0, wf[0], xf[0]);
          // Raised wave priority for the first two sub-steps: right after the
          // barrier the other wavefront of the SIMD is issuing loads and fragment
          // reads, and the MFMA stream should not wait behind them.
          __builtin_amdgcn_s_setprio(1);
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            if (s < 3) frags(stage, s + 1, wf[(s + 1) & 1], xf[(s + 1) & 1]);
#pragma unroll
            for (int mi = 0; mi < NB; ++mi)
#pragma unroll
              for (int ni = 0; ni < 2; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[s & 1][ni], xf[s & 1][mi],
                                                                      acc[mi][ni], 0, 0, 0);
            // Issue order: the next sub-step's 2 + NB LDS reads spread between this
            // one's 2 NB MFMAs.
            if (s < 3) {
              constexpr int kReads = 2 + NB, kMfmas = 2 * NB;
              constexpr int kPairs = kReads < kMfmas ? kReads : kMfmas;
#pragma unroll
              for (int i = 0; i < kPairs; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
              }
              if constexpr (kMfmas > kPairs) __builtin_amdgcn_sched_group_barrier(0x008, kMfmas - kPairs, 0);
              if constexpr (kReads > kPairs) __builtin_amdgcn_sched_group_barrier(0x100, kReads - kPairs, 0);
            } else {
              __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
            }
            if (s == 0 && ktn >= 0) {
              __builtin_amdgcn_sched_barrier(0);
              issue_a(nxt, ktn);
              __builtin_amdgcn_sched_barrier(0);
            }
            if (s == 1) __builtin_amdgcn_s_setprio(0);
          }
        } else {
          if (ktn >= 0) issue_a(nxt, ktn);
        }
      };
      // One k-step: wait for this stage's loads (own lanes, then all waves via the
      // barrier, which also frees the other stage), then run the MFMAs of this one
      // while the next step's loads go out into the other stage: the weight passes
      // first, the activation passes after the first 16-k sub-step, so that the
      // eight wavefronts' loads do not all queue at the texture unit at once and
      // hold back the first MFMAs of the step.
      auto step = [&](uint8_t* cur, uint8_t* nxt, int kt) {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
        if (kt + 1 < kt1) issue_w(nxt, kt + 1);
        compute(cur, nxt, kt + 1 < kt1 ? kt + 1 : -1);
      };
      issue_w(st0, kt0);
      issue_a(st0, kt0);
      int kt = kt0;
      for (; kt + 2 <= kt1; kt += 2) {
        step(st0, st1, kt);
        step(st1, st0, kt + 1);
      }
      if (kt < kt1) step(st0, st1, kt);
    };
    switch (nb) {
      case 5: kloop(std::integral_constant<int, 5>{}); break;
      case 4: kloop(std::integral_constant<int, 4>{}); break;
      case 3: kloop(std::integral_constant<int, 3>{}); break;
      case 2: kloop(std::integral_constant<int, 2>{}); break;
      case 1: kloop(std::integral_constant<int, 1>{}); break;
      default: kloop(std::integral_constant<int, 0>{}); break;
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();              // every wave is done with both stages before the next tile

    // ---- epilogue: lane holds columns 8*blk + 4*khalf + {0..3} of row (lane % 32) of
    // each 32-column block.  bf16 results (h, or y of a whole tile) go through a
    // private LDS region of each wavefront in st1, which the next tile writes only
    // after its first barrier: a lane's 16-byte pieces of 32 different rows become
    // whole row segments (h: 64 bytes, y: 128 bytes), 16 or 8 rows per store
    // instruction.  Measured against storing the 8-byte pieces directly, same
    // inputs, one process: memory-constrained GEMM-1 -0.9%, GEMM-2 -4.3%.
    uint8_t* ebuf = st1 + wave * kEpiBytes;
#pragma unroll
    for (int mi = 0; mi < 5; ++mi) {
      const int rbase = row0 + wm * kWaveRows + mi * 32;        // first row of this 32-row block
      if (rbase >= row_stop) continue;                          // uniform across the wave
      if (SWIGLU) {
        // h = silu(g) * u: 32 rows x 32 features, rows of 64 bytes in LDS whose four
        // 16-byte chunks sit at chunk ^ ((row >> 2) & 3) (conflict-free both ways)
#pragma unroll
        for (int blk = 0; blk < 4; ++blk) {
          float hv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) hv[q] = silu(acc[mi][0][blk * 4 + q]) * acc[mi][1][blk * 4 + q];
          u32x2 pk;
          pk[0] = pack_bf16x2(hv[0], hv[1]);
          pk[1] = pack_bf16x2(hv[2], hv[3]);
          const int c = blk ^ ((rrow >> 2) & 3);
          *reinterpret_cast<u32x2*>(ebuf + rrow * 64 + c * 16 + khalf * 8) = pk;
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int r = j * 16 + (lane >> 2);
          const int c = lane & 3;
          const u32x4 v = *reinterpret_cast<const u32x4*>(ebuf + r * 64 + (c ^ ((r >> 2) & 3)) * 16);
          const int row = rbase + r;
          const int f = n0 + wn * 32 + c * 8;
          if (row < row_stop && f < N) *reinterpret_cast<u32x4*>(p.out + int64_t(row) * N + f) = v;
        }
      } else if (slot >= 0) {
        // A piece of a tail tile: fp32 partial sums in its slot, tile-local
        // [320 rows][256 columns], added in piece order by tail_reduce_kernel.
        const int row = rbase + rrow;
        if (row < row_stop) {
          float* prow = p.partial + (int64_t(slot) * kBMMax + (row - row0)) * kBN;
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
        }
      } else {
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
          const int row = rbase + r;
          const int n = n0 + wn * 64 + (lane & 7) * 8;
          if (row < row_stop && n < N) *reinterpret_cast<u32x4*>(p.out + int64_t(row) * N + n) = v;
        }
      }
    }
  }
}

// Tail tiles of a down projection: y = bf16(sum of the tile's piece partials, in
// piece order).  kTailStrips blocks per tail tile, each 256 / kTailStrips rows of
// it; blocks past the plan's r tiles exit.  G and KT are the GEMM's grid size and
// k steps, so the plan is the GEMM's own.  A thread issues the loads of all its
// pieces before adding them (latency, not bandwidth, bounds a strip).
constexpr int kTailStrips = 16;

template <bool BLOCKS>
__global__ __launch_bounds__(256) void tail_reduce_kernel(const float* __restrict__ partial,
                                                         const int32_t* __restrict__ mtile_prefix,
                                                         const int32_t* __restrict__ offsets, int E, int NT, int G,
                                                         int KT, int N, uint16_t* __restrict__ y) {
  __shared__ int32_t s_pref[kMaxExperts + 1];
  __shared__ int32_t s_off[kMaxExperts + 1];
  for (int i = threadIdx.x; i <= E; i += blockDim.x) {
    s_pref[i] = mtile_prefix[i];
    s_off[i] = offsets[i];
  }
  __syncthreads();
  const TailPlan plan = tail_plan(int64_t(s_pref[E]) * NT, G, KT);
  const int t = int(blockIdx.x) / kTailStrips;
  if (t >= plan.r) return;                                     // uniform across the block
  const TileCoord tc = decode_tile<BLOCKS>(plan.full + t, s_pref, s_off, E, NT);
  const int rows = tc.row_stop - tc.row0;
  const int n0 = tc.nt * kTileCols;
  const int cols = min(kTileCols, N - n0);
  // this block's strip: rows r0 .. r0 + 19; 8 consecutive columns per item, 32 items a row
  constexpr int kStripRows = kTileRowsMax / kTailStrips;
  const int r0 = (int(blockIdx.x) % kTailStrips) * kStripRows;
  const float* base = partial + int64_t(t) * plan.s * (kTileRowsMax * kTileCols);
  for (int i = threadIdx.x; i < kStripRows * (kTileCols / 8); i += blockDim.x) {
    const int r = r0 + i / (kTileCols / 8);
    const int c = (i % (kTileCols / 8)) * 8;
    if (r >= rows || c >= cols) continue;
    f32x4 v[kMaxTailSplit][2];
#pragma unroll
    for (int j = 0; j < kMaxTailSplit; ++j) {
      if (j < plan.s) {
        const f32x4* src = reinterpret_cast<const f32x4*>(base + (int64_t(j) * kTileRowsMax + r) * kTileCols + c);
        v[j][0] = __builtin_nontemporal_load(src);
        v[j][1] = __builtin_nontemporal_load(src + 1);
      }
    }
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxTailSplit; ++j) {
      if (j < plan.s) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[q] += v[j][0][q];
          acc[4 + q] += v[j][1][q];
        }
      }
    }
    u32x4 pk;
#pragma unroll
    for (int q = 0; q < 4; ++q) pk[q] = pack_bf16x2(acc[2 * q], acc[2 * q + 1]);
    *reinterpret_cast<u32x4*>(y + int64_t(tc.row0 + r) * N + n0 + c) = pk;
  }
}

// ----------------------------------------------------------------------------- fp32 GEMM
// Plain LDS-tiled fp32 FMA kernel for the fp32 layer: 64 x 64 outputs per
// block (GEMM-1: 64 features of both gate and up), 4 x 4 per thread.
constexpr int kFM = 64, kFN = 64, kFK = 16;

struct GemmArgsF {
  const float* act;
  const int32_t* gather;          // [R] token of each grouped row, or null
  const float* w0;
  const float* w1;
  float* out;
  const int32_t* offsets;
  const int32_t* mtile_prefix;
  int E, K, N, ntiles;
};

template <bool SWIGLU>
__global__ __launch_bounds__(256) void grouped_gemm_f32_kernel(GemmArgsF p) {
  __shared__ float sX[kFK][kFM + 4];
  __shared__ float sG[kFK][kFN + 4];
  __shared__ float sU[kFK][kFN + 4];
  __shared__ int32_t s_pref[kMaxExperts + 1];
  const int tid = threadIdx.x;
  for (int i = tid; i <= p.E; i += 256) s_pref[i] = p.mtile_prefix[i];
  __syncthreads();
  const int64_t L = blockIdx.x;
  if (L >= int64_t(s_pref[p.E]) * p.ntiles) return;           // uniform across the block
  const int e = find_expert(s_pref, p.E, L / p.ntiles);
  const int64_t local = L - int64_t(s_pref[e]) * p.ntiles;
  const int mt = int(local / p.ntiles), nt = int(local % p.ntiles);
  const int row0 = p.offsets[e] + mt * kFM;
  const int row_end = p.offsets[e + 1];
  const int n0 = nt * kFN;
  const int K = p.K, N = p.N;
  const float* wg = p.w0 + int64_t(e) * N * K;
  const float* wu = SWIGLU ? p.w1 + int64_t(e) * N * K : nullptr;
  const int tx = tid & 15, ty = tid >> 4;
  const int lrow = tid >> 2, lk = (tid & 3) * 4;               // loader: one float4 per thread
  const int64_t arow = p.gather != nullptr ? int64_t(p.gather[min(row0 + lrow, row_end - 1)])
                                           : int64_t(min(row0 + lrow, row_end - 1));
  const int64_t wrow = min(n0 + lrow, N - 1);
  float ag[4][4] = {}, au[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += kFK) {
    const float4 xa = *reinterpret_cast<const float4*>(p.act + arow * K + k0 + lk);
    const float4 ga = *reinterpret_cast<const float4*>(wg + wrow * K + k0 + lk);
    sX[lk + 0][lrow] = xa.x; sX[lk + 1][lrow] = xa.y; sX[lk + 2][lrow] = xa.z; sX[lk + 3][lrow] = xa.w;
    sG[lk + 0][lrow] = ga.x; sG[lk + 1][lrow] = ga.y; sG[lk + 2][lrow] = ga.z; sG[lk + 3][lrow] = ga.w;
    if (SWIGLU) {
      const float4 ua = *reinterpret_cast<const float4*>(wu + wrow * K + k0 + lk);
      sU[lk + 0][lrow] = ua.x; sU[lk + 1][lrow] = ua.y; sU[lk + 2][lrow] = ua.z; sU[lk + 3][lrow] = ua.w;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kFK; ++kk) {
      float a[4], g[4], u[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = sX[kk][ty * 4 + i];
        g[i] = sG[kk][tx * 4 + i];
        if (SWIGLU) u[i] = sU[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          ag[i][j] = fmaf(a[i], g[j], ag[i][j]);
          if (SWIGLU) au[i][j] = fmaf(a[i], u[j], au[i][j]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = row0 + ty * 4 + i;
    if (row >= row_end) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < N) {
        const float v = SWIGLU ? (ag[i][j] / (1.0f + expf(-ag[i][j]))) * au[i][j] : ag[i][j];
        p.out[int64_t(row) * N + n] = v;
      }
    }
  }
}

// One persistent workgroup per compute unit (fewer for small problems).
int grid_for(int64_t upper_tiles, int num_cu) {
  const int64_t g = upper_tiles < num_cu ? upper_tiles : num_cu;
  return int(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_tail_reduce(const float* partial, const int32_t* mtile_prefix, const int32_t* offsets, int E,
                              int NT, int G, int KT, int N, uint16_t* y, bool row_blocks, hipStream_t s) {
  // A split happens only with at least two pieces of kMinPieceSteps steps; then
  // r <= min(G, kMaxTailPieces) / 2 tail tiles.
  if (KT < 2 * kMinPieceSteps || G < 2) return hipSuccess;
  const int blocks = std::min(G, kMaxTailPieces) / 2 * kTailStrips;
  if (row_blocks)
    MOE_LAUNCH("ffn_tail_reduce", tail_reduce_kernel<true>, dim3(unsigned(blocks)), dim3(256), s, partial,
               mtile_prefix, offsets, E, NT, G, KT, N, y);
  else
    MOE_LAUNCH("ffn_tail_reduce", tail_reduce_kernel<false>, dim3(unsigned(blocks)), dim3(256), s, partial,
               mtile_prefix, offsets, E, NT, G, KT, N, y);
  return hipGetLastError();
}

hipError_t launch_tile_prefix(const int32_t* offsets, int E, int bm, int32_t* mtile_prefix, int32_t* queues,
                              hipStream_t s) {
  MOE_LAUNCH("ffn_tile_prefix", tile_prefix_kernel, dim3(1), dim3(256), s, offsets, E, bm, mtile_prefix, queues);
  return hipGetLastError();
}

hipError_t launch_ffn_bf16(const uint16_t* act, const int32_t* gather, int64_t T, const int32_t* offsets,
                           int64_t R, int E, int H, int F, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, uint16_t* y_perm, int32_t* mtile_prefix, int32_t* queues,
                           uint16_t* h, float* partial, int num_cu, hipStream_t s) {
  MOE_LAUNCH("ffn_tile_prefix", tile_prefix_kernel, dim3(1), dim3(256), s, offsets, E, kBMMax, mtile_prefix,
             queues);
  const int64_t mtiles_upper = (R + int64_t(E) * (kBM - 1)) / kBM;

  const int64_t act_bytes = T * H * 2;
  const bool wide = act_bytes >= (int64_t(1) << 31);
  GemmArgs a1{queues, queues + 2, act, gather, wg, wu, h, nullptr, offsets, mtile_prefix, E, H, F, (F + 127) / 128,
              int(R), wide ? 0 : int(act_bytes)};
  const dim3 grid1(grid_for(mtiles_upper * a1.ntiles, num_cu));
  if (gather != nullptr && wide)
    MOE_LAUNCH("ffn_gemm1_gate_up", (grouped_gemm_bf16_kernel<true, kTokensWide>), grid1, dim3(kGemmThreads), s,
               a1);
  else if (gather != nullptr)
    MOE_LAUNCH("ffn_gemm1_gate_up", (grouped_gemm_bf16_kernel<true, kTokens>), grid1, dim3(kGemmThreads), s, a1);
  else
    MOE_LAUNCH("ffn_gemm1_gate_up", (grouped_gemm_bf16_kernel<true, kRows>), grid1, dim3(kGemmThreads), s, a1);
  GemmArgs a2{queues + 1, queues + 2 + kGroups, h, nullptr, wd, nullptr, y_perm, partial, offsets, mtile_prefix, E,
              F, H, (H + 255) / 256, int(R), 0};
  const int grid2 = grid_for(mtiles_upper * a2.ntiles, num_cu);
  MOE_LAUNCH("ffn_gemm2_down", (grouped_gemm_bf16_kernel<false, kRows>), dim3(grid2), dim3(kGemmThreads), s,
             a2);
  const hipError_t err = launch_tail_reduce(partial, mtile_prefix, offsets, E, a2.ntiles, grid2, F / kBK, H,
                                            y_perm, true, s);
  if (err != hipSuccess) return err;
  return hipGetLastError();
}

hipError_t launch_ffn_f32(const float* act, const int32_t* gather, const int32_t* offsets, int64_t R,
                          int E, int H, int F, const float* wg, const float* wu, const float* wd,
                          float* y_perm, int32_t* mtile_prefix, float* h, hipStream_t s) {
  MOE_LAUNCH("ffn_tile_prefix", tile_prefix_kernel, dim3(1), dim3(256), s, offsets, E, kFM, mtile_prefix,
             static_cast<int32_t*>(nullptr));
  const int64_t mtiles_upper = (R + int64_t(E) * (kFM - 1)) / kFM;
  GemmArgsF a1{act, gather, wg, wu, h, offsets, mtile_prefix, E, H, F, (F + kFN - 1) / kFN};
  MOE_LAUNCH("ffn_gemm1_gate_up", grouped_gemm_f32_kernel<true>, dim3(unsigned(mtiles_upper * a1.ntiles)),
             dim3(256), s, a1);
  GemmArgsF a2{h, nullptr, wd, nullptr, y_perm, offsets, mtile_prefix, E, F, H, (H + kFN - 1) / kFN};
  MOE_LAUNCH("ffn_gemm2_down", grouped_gemm_f32_kernel<false>, dim3(unsigned(mtiles_upper * a2.ntiles)),
             dim3(256), s, a2);
  return hipGetLastError();
}

}  // namespace moe
