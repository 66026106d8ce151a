// moe_permute: stable counting sort of the T*k (token, slot) assignments by
// expert, then a row gather of x into expert-grouped order, on gfx950.
//
// The assignment list (token-major, a = t*k + j) is cut into units of 1024
// consecutive assignments, one wavefront each.  Within a wavefront, the lanes
// holding the same expert find each other with 8 ballots over the id bits (a
// match mask); a lane's rank among equal experts is the popcount of the match
// mask below it, so the order inside an expert group is the assignment order,
// i.e. ascending token.  Four kernels, no atomics (batches of at most 16 units
// run the first three as one single-block kernel):
//   count : per-unit, per-expert counts                      -> uc[E][units]
//   scan  : per expert, exclusive scan over units; totals    -> uc, counts
//   rank  : offsets = exclusive scan of counts; every assignment's row
//           = offsets[e] + uc[e][unit] + running count + rank -> dest_rows, sorted_token_ids
//   copy  : one wavefront per token reads x[t] once and writes its k rows.
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

__global__ __launch_bounds__(kThreads) void permute_count_kernel(const int32_t* __restrict__ ids,
                                                                int64_t R, int E, int nbits,
                                                                int64_t Upad,
                                                                int32_t* __restrict__ uc) {
  __shared__ int32_t cnt[kWavesPerBlock][kMaxExperts];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  for (int e = lane; e < E; e += kWave) cnt[w][e] = 0;
  __syncthreads();
  const int64_t unit = int64_t(blockIdx.x) * kWavesPerBlock + w;
  const int64_t base = unit * kUnit;
  const uint64_t below = (1ull << lane) - 1ull;
  for (int it = 0; it < kIters; ++it) {
    const int64_t a = base + it * kWave + lane;
    const bool valid = a < R;
    const int id = valid ? ids[a] : 0;
    const uint64_t match = wave_match(id, valid, nbits);
    if (valid && (match & below) == 0ull) cnt[w][id] += __popcll(match);   // one leader per expert
  }
  __syncthreads();
  for (int e = lane; e < E; e += kWave) uc[int64_t(e) * Upad + unit] = cnt[w][e];
}

__global__ __launch_bounds__(kThreads) void permute_scan_kernel(int32_t* __restrict__ uc, int64_t U,
                                                               int64_t Upad,
                                                               int32_t* __restrict__ counts) {
  const int e = blockIdx.x;
  int32_t* row = uc + int64_t(e) * Upad;
  const int64_t per = (U + kThreads - 1) / kThreads;
  const int64_t lo = int64_t(threadIdx.x) * per;
  const int64_t hi = lo + per < U ? lo + per : U;
  int32_t s = 0;
  for (int64_t u = lo; u < hi; ++u) s += row[u];
  int32_t total;
  int32_t run = block_exclusive_scan256(s, &total);
  for (int64_t u = lo; u < hi; ++u) {
    const int32_t c = row[u];
    row[u] = run;
    run += c;
  }
  if (threadIdx.x == 0) counts[e] = total;
}

__global__ __launch_bounds__(kThreads) void permute_rank_kernel(
    const int32_t* __restrict__ ids, int64_t R, int E, int k, int nbits, int64_t Upad,
    const int32_t* __restrict__ uc, const int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ dest, int32_t* __restrict__ sorted_tok) {
  __shared__ int32_t s_off[kMaxExperts];
  __shared__ int32_t run[kWavesPerBlock][kMaxExperts];
  const int tid = threadIdx.x;
  const int32_t c = tid < E ? counts[tid] : 0;
  int32_t total;
  const int32_t ex = block_exclusive_scan256(c, &total);
  if (tid < E) s_off[tid] = ex;
  if (blockIdx.x == 0) {
    if (tid < E) offsets[tid] = ex;
    if (tid == 0) offsets[E] = total;
  }
  __syncthreads();
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int64_t unit = int64_t(blockIdx.x) * kWavesPerBlock + w;
  for (int e = lane; e < E; e += kWave) run[w][e] = s_off[e] + uc[int64_t(e) * Upad + unit];
  __syncthreads();
  const int64_t base = unit * kUnit;
  const uint64_t below = (1ull << lane) - 1ull;
  for (int it = 0; it < kIters; ++it) {
    const int64_t a = base + it * kWave + lane;
    const bool valid = a < R;
    const int id = valid ? ids[a] : 0;
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
        u32x4* dst = reinterpret_cast<u32x4*>(x_perm + int64_t(rows[j]) * row_bytes);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
          if (v + u * kWave < nvec) dst[v + u * kWave] = val[u];
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
    const unsigned unit_blocks = unsigned(Upad / kWavesPerBlock);
    MOE_LAUNCH("permute_count", permute_count_kernel, dim3(unit_blocks), dim3(kThreads), s, ids, R, E,
               nbits, Upad, uc);
    MOE_LAUNCH("permute_scan", permute_scan_kernel, dim3(E), dim3(kThreads), s, uc, U, Upad, counts);
    MOE_LAUNCH("permute_rank", permute_rank_kernel, dim3(unit_blocks), dim3(kThreads), s, ids, R, E, k,
               nbits, Upad, uc, counts, offsets, dest, sorted_tok);
  }
  if (x_perm == nullptr) return hipGetLastError();     // maps only: the grouped FFN gathers rows
  const int64_t row_bytes = int64_t(H) * elt;
  const unsigned copy_blocks = unsigned((T + kWavesPerBlock - 1) / kWavesPerBlock);
  MOE_LAUNCH("permute_copy", permute_copy_kernel<4>, dim3(copy_blocks), dim3(kThreads), s,
             static_cast<const uint8_t*>(x), T, k, row_bytes, dest, static_cast<uint8_t*>(x_perm));
  return hipGetLastError();
}

}  // namespace moe
