// moe_permute: stable counting sort of the T*k (token, slot) assignments by
// expert, then a row gather of x into expert-grouped order, on gfx950.
//
// The assignment list (token-major, a = t*k + j) is cut into units of 1024
// consecutive assignments, one wavefront each, which loads its unit's ids (16
// per lane) up front.  Within a wavefront, the lanes holding the same expert
// find each other with log2(E) ballots over the id bits (a match mask); a
// lane's rank among equal experts is the popcount of the match mask below it,
// so the order inside an expert group is the assignment order, i.e. ascending
// token.  No atomics.  Launches:
//   count : per block of 4 units, per-expert totals               -> bc[E][blocks]
//   rank  : per expert, the totals of the blocks before this one and of all
//           blocks (read from bc: scan and rank fused); offsets = exclusive
//           scan of the totals; every assignment's row = offsets[e] + earlier
//           blocks' and units' counts + rank                     -> counts, offsets,
//                                                                   dest_rows, sorted_token_ids
//   copy  : one wavefront per token reads x[t] once and writes its k rows.
// Batches of at most 16 units run count and rank as one single-block kernel.
#include <mutex>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kUnit = 1024;                 // assignments per unit (one wavefront)
constexpr int kIters = kUnit / kWave;

// Lanes of this wavefront whose (valid) id equals mine.  ids < 2^nbits.
__device__ __forceinline__ uint64_t wave_match(int id, bool valid, int nbits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (id >> b) & 1;
    const uint64_t bb = __ballot(bit);
    m &= bit ? bb : ~bb;
  }
  return m;
}

// The unit's kIters ids of this lane, all loads issued before any is used (-1
// past the end).  Lane l holds assignments base + 64 it + l.
__device__ __forceinline__ void load_unit_ids(const int32_t* __restrict__ ids, int64_t base, int64_t R,
                                              int lane, int (&idv)[kIters]) {
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t a = base + it * kWave + lane;
    idv[it] = a < R ? __builtin_nontemporal_load(ids + a) : -1;
  }
}

// Per-expert counts of one unit into cnt (zeroed by the caller): the lanes of a
// match group add their size once, through the group's lowest lane.
__device__ __forceinline__ void count_unit(const int (&idv)[kIters], int nbits, int lane,
                                           int32_t* __restrict__ cnt) {
  const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const bool valid = idv[it] >= 0;
    const int id = valid ? idv[it] : 0;
    const uint64_t match = wave_match(id, valid, nbits);
    if (valid && (match & below) == 0ull) cnt[id] += __popcll(match);
  }
}

// Block b (units 4b .. 4b + 3) writes its per-expert totals to bc[e][b].
__global__ __launch_bounds__(kThreads) void permute_count_kernel(const int32_t* __restrict__ ids,
                                                                int64_t R, int E, int nbits,
                                                                int64_t Bpad,
                                                                int32_t* __restrict__ bc) {
  __shared__ int32_t cnt[kWavesPerBlock][kMaxExperts];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int64_t unit = int64_t(blockIdx.x) * kWavesPerBlock + w;
  int idv[kIters];
  load_unit_ids(ids, unit * kUnit, R, lane, idv);
  for (int e = lane; e < E; e += kWave) cnt[w][e] = 0;
  __syncthreads();
  count_unit(idv, nbits, lane, cnt[w]);
  __syncthreads();
  if (tid < E) {
    int32_t c = 0;
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i) c += cnt[i][tid];
    bc[int64_t(tid) * Bpad + blockIdx.x] = c;
  }
}

// Scan and rank in one pass.  Every block's per-expert total is already in bc
// (the count kernel), so a block's exclusive prefix over the blocks before it
// needs no waiting on other blocks: it sums its predecessors' totals itself (the
// aggregates a decoupled look-back reads), and the sum over all blocks gives the
// expert totals, hence the offsets.  The threads of one expert (256 / E' of them,
// E' = E rounded up to a power of two) split its row of bc, 16-byte loads of four
// blocks each, all issued before they are summed.  The block then counts its own
// four units again (ids already in registers) for the prefix inside the block.
constexpr int kRowLoads = 8;                       // 16-byte loads in flight per thread

__global__ __launch_bounds__(kThreads) void permute_rank_kernel(
    const int32_t* __restrict__ ids, int64_t R, int E, int k, int nbits, int64_t B, int64_t Bpad,
    const int32_t* __restrict__ bc, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ dest, int32_t* __restrict__ sorted_tok) {
  __shared__ int32_t s_pre[kThreads];
  __shared__ int32_t s_tot[kThreads];
  __shared__ int32_t run[kWavesPerBlock][kMaxExperts];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int64_t b0 = blockIdx.x;
  const int64_t unit = b0 * kWavesPerBlock + w;
  int idv[kIters];
  load_unit_ids(ids, unit * kUnit, R, lane, idv);
  for (int e = lane; e < E; e += kWave) run[w][e] = 0;

  // ---- per expert: totals of the blocks before this one, and of all blocks
  const int tpe = kThreads >> nbits;                 // threads per expert (nbits <= 8)
  const int e = tid / tpe, part = tid % tpe;
  int32_t pre = 0, tot = 0;
  if (e < E) {
    const u32x4* row = reinterpret_cast<const u32x4*>(bc + int64_t(e) * Bpad);
    const int64_t nvec = Bpad / 4;
    for (int64_t v0 = part; v0 < nvec; v0 += int64_t(kRowLoads) * tpe) {
      u32x4 q[kRowLoads];
#pragma unroll
      for (int j = 0; j < kRowLoads; ++j) {
        const int64_t v = v0 + int64_t(j) * tpe;
        q[j] = v < nvec ? row[v] : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int j = 0; j < kRowLoads; ++j) {
        const int64_t v = v0 + int64_t(j) * tpe;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t b = 4 * v + i;
          const int32_t c = b < B ? int32_t(q[j][i]) : 0;
          tot += c;
          pre += b < b0 ? c : 0;
        }
      }
    }
  }
  s_pre[tid] = pre;
  s_tot[tid] = tot;
  __syncthreads();
  count_unit(idv, nbits, lane, run[w]);            // this wave's own unit
  // thread e (< E) gathers its expert's partial sums; the offsets are the
  // exclusive scan of the totals over the experts
  int32_t total_e = 0, pre_e = 0;
  if (tid < E) {
    for (int i = 0; i < tpe; ++i) {
      total_e += s_tot[tid * tpe + i];
      pre_e += s_pre[tid * tpe + i];
    }
  }
  int32_t all;
  const int32_t off_e = block_exclusive_scan256(total_e, &all);   // synchronizes the block
  if (blockIdx.x == 0) {
    if (tid < E) {
      counts[tid] = total_e;
      offsets[tid] = off_e;
    }
    if (tid == 0) offsets[E] = all;
  }
  // running row of each of the block's units: offset + blocks before this one +
  // the block's own earlier units
  if (tid < E) {
    int32_t r = off_e + pre_e;
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i) {
      const int32_t c = run[i][tid];
      run[i][tid] = r;
      r += c;
    }
  }
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
  const int64_t base = unit * kUnit;
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t a = base + it * kWave + lane;
    const bool valid = idv[it] >= 0;
    const int id = valid ? idv[it] : 0;
    const uint64_t match = wave_match(id, valid, nbits);
    if (valid) {
      const int32_t r0 = run[w][id];
      const int32_t rank = __popcll(match & below);
      const int32_t row = r0 + rank;
      dest[a] = row;
      sorted_tok[row] = int32_t(uint32_t(a) / uint32_t(k));
      if (rank == 0) run[w][id] = r0 + __popcll(match);
    }
  }
}

// Small batches (at most kSmallUnits units): the three phases in one block of
// 1024 threads, one wavefront per unit, with the per-unit counts in LDS.  Same
// results as count + scan + rank.
constexpr int kSmallUnits = 16;
constexpr int kSmallThreads = kSmallUnits * kWave;

__global__ __launch_bounds__(kSmallThreads) void permute_small_kernel(
    const int32_t* __restrict__ ids, int64_t R, int E, int k, int nbits, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ dest, int32_t* __restrict__ sorted_tok) {
  __shared__ int32_t run[kSmallUnits][kMaxExperts];
  __shared__ int32_t s_wsum[4];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;                                // the unit
  const int64_t base = int64_t(w) * kUnit;
  const uint64_t below = (1ull << lane) - 1ull;
  // the unit's ids, all loaded at once and kept for the rank phase
  int idv[kIters];
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t a = base + it * kWave + lane;
    idv[it] = a < R ? ids[a] : -1;
  }
  for (int e = lane; e < E; e += kWave) run[w][e] = 0;
  __syncthreads();
  // counts per unit
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const bool valid = idv[it] >= 0;
    const int id = valid ? idv[it] : 0;
    const uint64_t match = wave_match(id, valid, nbits);
    if (valid && (match & below) == 0ull) run[w][id] += __popcll(match);
  }
  __syncthreads();
  // per expert: exclusive scan over the units, then offsets = exclusive scan of the
  // totals over the experts (threads 0..255, one expert each)
  int32_t total = 0;
  if (tid < E) {
    for (int u = 0; u < kSmallUnits; ++u) {
      const int32_t c = run[u][tid];
      run[u][tid] = total;
      total += c;
    }
    counts[tid] = total;
  }
  int32_t x = total;                                          // inclusive scan over threads 0..255
  if (tid < kMaxExperts) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const int32_t y = __shfl_up(x, d);
      if (lane >= d) x += y;
    }
    if (lane == kWave - 1) s_wsum[w] = x;
  }
  __syncthreads();
  if (tid < kMaxExperts) {
    int32_t before = 0;
    for (int i = 0; i < w; ++i) before += s_wsum[i];
    const int32_t ex = before + x - total;                   // exclusive offset of expert tid
    if (tid < E) {
      offsets[tid] = ex;
      for (int u = 0; u < kSmallUnits; ++u) run[u][tid] += ex;
    }
    if (tid == E - 1) offsets[E] = ex + total;
  }
  __syncthreads();
  // rows: the unit's running position per expert plus the rank among equal ids
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t a = base + it * kWave + lane;
    const bool valid = idv[it] >= 0;
    const int id = valid ? idv[it] : 0;
    const uint64_t match = wave_match(id, valid, nbits);
    if (valid) {
      const int32_t r0 = run[w][id];
      const int32_t rank = __popcll(match & below);
      const int32_t row = r0 + rank;
      dest[a] = row;
      sorted_tok[row] = int32_t(uint32_t(a) / uint32_t(k));
      if (rank == 0) run[w][id] = r0 + __popcll(match);
    }
  }
}

template <int UNROLL>
__global__ __launch_bounds__(kThreads) void permute_copy_kernel(const uint8_t* __restrict__ x,
                                                               int64_t T, int k, int64_t row_bytes,
                                                               const int32_t* __restrict__ dest,
                                                               uint8_t* __restrict__ x_perm) {
  const int lane = threadIdx.x & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t t = int64_t(blockIdx.x) * kWavesPerBlock + w;
  if (t >= T) return;
  int32_t rows[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) rows[j] = j < k ? dest[t * k + j] : 0;
  const int nvec = int(row_bytes / 16);
  const u32x4* src = reinterpret_cast<const u32x4*>(x + t * row_bytes);
  for (int v = lane; v < nvec; v += kWave * UNROLL) {
    u32x4 val[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      if (v + u * kWave < nvec) val[u] = __builtin_nontemporal_load(src + v + u * kWave);
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (j < k) {
        // x_perm is not read again here: nontemporal stores
        u32x4* dst = reinterpret_cast<u32x4*>(x_perm + int64_t(rows[j]) * row_bytes);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
          if (v + u * kWave < nvec) __builtin_nontemporal_store(val[u], dst + v + u * kWave);
      }
    }
  }
}

}  // namespace

hipError_t launch_permute(const int32_t* ids, const void* x, int64_t T, int E, int k, int H, int elt,
                          int32_t* counts, int32_t* offsets, int32_t* sorted_tok, int32_t* dest,
                          void* x_perm, int32_t* uc, int64_t Upad, hipStream_t s) {
  const int64_t R = T * k;
  const int64_t U = (R + kUnit - 1) / kUnit;
  int nbits = 0;
  while ((1 << nbits) < E) ++nbits;
  if (U <= kSmallUnits) {
    MOE_LAUNCH("permute_small", permute_small_kernel, dim3(1), dim3(kSmallThreads), s, ids, R, E, k, nbits,
               counts, offsets, dest, sorted_tok);
  } else {
    // per-block totals [E][Bpad] in the workspace (E * Bpad <= E * Upad ints)
    const int64_t B = Upad / kWavesPerBlock;
    const int64_t Bpad = (B + 3) / 4 * 4;
    MOE_LAUNCH("permute_count", permute_count_kernel, dim3(unsigned(B)), dim3(kThreads), s, ids, R, E, nbits,
               Bpad, uc);
    MOE_LAUNCH("permute_rank", permute_rank_kernel, dim3(unsigned(B)), dim3(kThreads), s, ids, R, E, k, nbits,
               B, Bpad, uc, counts, offsets, dest, sorted_tok);
  }
  if (x_perm == nullptr) return hipGetLastError();     // maps only: the grouped FFN gathers rows
  const int64_t row_bytes = int64_t(H) * elt;
  const unsigned copy_blocks = unsigned((T + kWavesPerBlock - 1) / kWavesPerBlock);
  MOE_LAUNCH("permute_copy", permute_copy_kernel<8>, dim3(copy_blocks), dim3(kThreads), s,
             static_cast<const uint8_t*>(x), T, k, row_bytes, dest, static_cast<uint8_t*>(x_perm));
  return hipGetLastError();
}

// ----------------------------------------------------------------------------- static scratch
// moe_permute_static: the per-block counts live in this file-scope device array
// instead of a caller workspace, so the call allocates nothing.  Every device the
// library runs on holds its own copy for the life of the process.  In host code
// the name `scratch` is only a stand-in for the symbol, not a device address: the
// address comes from hipGetSymbolAddress, taken once per device (with that device
// current) and cached.  Nothing in it has to start at zero (the count kernel
// writes every count the rank kernel reads); calls that overlap on one device
// share the array and race.
static __device__ __align__(256) uint8_t scratch[kPermuteStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t permute_static_scratch(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace moe
