// Device helpers shared by the gfx950 kernels of the MoE hot path.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tiling.h"

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

// ----------------------------------------------------------------------------- tile list
// The grouped GEMMs walk one flattened list of output tiles: experts in order,
// expert e owning pref[e+1] - pref[e] m-tiles times NT n-tiles.
// Inside an expert, blocks of up to kGroupM m-tiles are swept in groups of
// kGroupN n-tiles with the m-tile varying fastest, so the tiles in flight at
// one time share a few weight and activation panels.
constexpr int kGroupN = 8;
constexpr int kGroupM = 4;

struct TileCoord {
  int e;          // expert
  int row0;       // first grouped row of the tile
  int row_stop;   // end of the tile's rows
  int nt;         // n-tile index
  int mt_e;       // the expert's m-tiles
};

// Tile L of the list; pref/off are the m-tile prefix and row offsets (E + 1
// entries, typically staged in LDS).  All lanes pass the same L.  BLOCKS (the
// bf16 GEMMs, prefix of ceil(c / kTileRowsMax) m-tiles): the expert's
// ceil(c / 32) row blocks are shared out evenly, m-tile mt holding blocks
// [mt nb / mt_e, (mt + 1) nb / mt_e), at most 10 of them (320 rows).  Otherwise
// (prefix of ceil(c / kTileRows)): kTileRows rows each, the last one shorter.
template <bool BLOCKS = false>
__device__ __forceinline__ TileCoord decode_tile(int64_t L, const int32_t* pref, const int32_t* off, int E,
                                                 int NT) {
  TileCoord t;
  t.e = __builtin_amdgcn_readfirstlane(find_expert(pref, E, L / NT));
  const int pe = __builtin_amdgcn_readfirstlane(pref[t.e]);
  const int mt_e = __builtin_amdgcn_readfirstlane(pref[t.e + 1]) - pe;
  const int64_t local = L - int64_t(pe) * NT;
  const int64_t bsz = int64_t(kGroupM) * NT;
  const int mbi = int(local / bsz);
  const int rem = int(local - int64_t(mbi) * bsz);
  const int bm = min(kGroupM, mt_e - mbi * kGroupM);
  const int ng = rem / (bm * kGroupN);
  const int rem2 = rem - ng * bm * kGroupN;
  const int mt = mbi * kGroupM + rem2 % bm;
  t.nt = ng * kGroupN + rem2 / bm;
  t.mt_e = mt_e;
  const int row_beg = __builtin_amdgcn_readfirstlane(off[t.e]);
  const int row_end = __builtin_amdgcn_readfirstlane(off[t.e + 1]);
  if (BLOCKS) {
    const int nb = (row_end - row_beg + kTileRowBlock - 1) / kTileRowBlock;
    t.row0 = row_beg + kTileRowBlock * int(int64_t(mt) * nb / mt_e);
    t.row_stop = min(row_end, row_beg + kTileRowBlock * int(int64_t(mt + 1) * nb / mt_e));
  } else {
    t.row0 = row_beg + mt * kTileRows;
    t.row_stop = mt == mt_e - 1 ? row_end : t.row0 + kTileRows;
  }
  return t;
}

// Tail split (constants in tiling.h): of n tiles on G persistent workgroups with
// KT k steps each, tiles [0, full) run whole and the r tiles after them are cut
// into s pieces each (r = 0, s = 1 when nothing is split).  The work list is the
// full tiles, then the pieces: entry full + q is piece q % s of tile
// full + q / s, k steps [j KT / s, (j + 1) KT / s) with j = q % s, and its fp32
// partial sums go to partial slot q.
struct TailPlan {
  int64_t full;
  int r;
  int s;
};

__device__ __forceinline__ TailPlan tail_plan(int64_t n, int G, int KT) {
  TailPlan t{n, 0, 1};
  if (G < 2) return t;
  const int64_t r = n % G;
  if (r == 0 || 2 * r > G) return t;
  const int pieces = min(G, kMaxTailPieces);
  const int s = int(min(int64_t(pieces) / r, int64_t(min(KT / kMinPieceSteps, kMaxTailSplit))));
  if (s < 2) return t;
  t.full = n - r;
  t.r = int(r);
  t.s = s;
  return t;
}

// Tile claims of the persistent grouped GEMMs.  Workgroup b belongs to group
// b % ng (ng = 8 with at least 8 workgroups: the XCD the workgroups are dealt to
// round-robin).  When the experts hold at least two m-tiles each on average, the
// leading full tiles of the list go out in chunks of kGroupM * kGroupN
// consecutive tiles (one block of m-tiles x n-tiles sharing their panels), as
// many chunks as make the same whole number per group: group x takes chunks x,
// x + ng, x + 2 ng, ... through a counter of its own, so an XCD's compute units
// work on the same panels together.  The rest of the full tiles (fewer than ng
// chunks' worth), then the pieces of a split tail (entries full..), go out one at
// a time from a counter shared by all, so no XCD idles while another still holds
// tiles.  Every group has at least one workgroup, so every chunk is taken.  With
// no chunk to hand out the first claim goes straight to the shared counter: the
// counters are device-scope atomics that serialize, and in a launch of one tile
// per workgroup a second dependent atomic before the first tile delays the last
// workgroup's start.  With about one m-tile per expert a chunk shares no weight
// panel, and a single queue measured faster.  Called by one thread per workgroup.
struct TileClaim {
  static constexpr int kChunk = kGroupM * kGroupN;
  int32_t* chunk_ctr;   // [ng] counters, zeroed before the launch
  int32_t* shared_ctr;  // one counter, zeroed before the launch
  int64_t chunked;      // entries [0, chunked) go out in chunks
  int ng, grp;
  bool in_shared;
  // full_tiles: entries [0, full_tiles) are whole tiles; mtiles, E: the m-tiles of
  // all experts and the number of experts.
  __device__ TileClaim(int32_t* chunks, int32_t* shared, int64_t full_tiles, int mtiles, int E)
      : chunk_ctr(chunks), shared_ctr(shared) {
    ng = int(gridDim.x) < 8 ? int(gridDim.x) : 8;
    grp = int(blockIdx.x) % ng;
    const int64_t per = int64_t(kChunk) * ng;
    chunked = mtiles >= 2 * E ? full_tiles / per * per : 0;
    in_shared = chunked == 0;
  }
  __device__ int64_t next() {
    if (!in_shared) {
      const int64_t lx = atomicAdd(chunk_ctr + grp, 1);
      const int64_t L = ((lx / kChunk) * ng + grp) * kChunk + lx % kChunk;
      if (L < chunked) return L;
      in_shared = true;
    }
    return chunked + atomicAdd(shared_ctr, 1);
  }
};

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
