// moe_grouped_ffn: every expert's SwiGLU FFN on its own rows, on gfx950.
//
//   GEMM-1  h[r, f]  = silu(x_perm[r] . W_gate[e][f]) * (x_perm[r] . W_up[e][f])
//   GEMM-2  y[r, n]  = h[r] . W_down[e][n]
// for every row r of expert e's group.  Both operands are K-contiguous.
//
// Tile scheduling.  A tiny kernel turns the device-side offsets into a prefix
// of m-tiles per expert (no host readback).  The GEMM kernels are persistent:
// each workgroup walks a strided range of the flattened tile list, in which an
// expert's tiles are contiguous, so a hot expert simply owns more tiles and an
// empty one owns none.  Workgroups are dealt to the 8 XCDs round-robin; the
// list is cut into 8 contiguous chunks, one per XCD, so tiles that share
// weight and activation panels run on the same XCD and share its L2.  Inside
// an expert the order is (group of kGroupN n-tiles, m-tile, n-tile): the
// workgroups of one XCD sweep a few m-tiles against a few n-tiles at a time.
//
// bf16 tile: 256 rows x 256 weight rows x 64 k per step, 4 wavefronts (2 x 2),
// each a 128 x 128 block of v_mfma_f32_32x32x16_bf16 results (16 MFMA tiles).
// The weight tile is the MFMA A operand and the activation tile the B operand,
// so each lane ends up holding 4 consecutive output columns of one row: the
// epilogue stores 8 bytes per lane.  For GEMM-1 the weight tile holds 128
// gate rows and the 128 up rows of the same features, so silu(g) * u is formed
// in registers and only h is written.  Tiles are staged through LDS, double
// buffered, with the 16-byte chunks of each 128-byte row XOR-swizzled by the
// row index so the MFMA operand reads are free of bank conflicts.
#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

// ----------------------------------------------------------------------------- tile prefix
// prefix[e] = sum_{e' < e} ceil(count[e'] / bm), prefix[E] = total.  One block of 256.
__global__ __launch_bounds__(256) void tile_prefix_kernel(const int32_t* __restrict__ offsets, int E,
                                                         int bm, int32_t* __restrict__ prefix) {
  const int e = threadIdx.x;
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

// Largest e in [0, E) with pref[e] <= q, given pref[0] <= q < pref[E].
__device__ __forceinline__ int find_expert(const int32_t* pref, int E, int64_t q) {
  int lo = 0, hi = E;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pref[mid] <= q) lo = mid; else hi = mid;
  }
  return lo;
}

// ----------------------------------------------------------------------------- bf16 MFMA GEMM
constexpr int kBM = 256;                  // activation rows per tile
constexpr int kBN = 256;                  // weight rows per tile (GEMM-1: 128 gate + 128 up)
constexpr int kBK = 64;                   // k per pipeline step
constexpr int kRowBytes = kBK * 2;        // one tile row in LDS: 128 bytes = 8 chunks of 16
constexpr int kOpBytes = 256 * kRowBytes; // one operand tile: 32 KB
constexpr int kStageBytes = 2 * kOpBytes;
constexpr int kGemmThreads = 256;
constexpr int kGroupN = 8;

struct GemmArgs {
  const uint16_t* act;            // [R, K]
  const uint16_t* w0;             // [E, N, K] (GEMM-1: W_gate; GEMM-2: W_down)
  const uint16_t* w1;             // [E, N, K] (GEMM-1: W_up)
  uint16_t* out;                  // [R, N]
  const int32_t* offsets;         // [E + 1]
  const int32_t* mtile_prefix;    // [E + 1]
  int E, K, N, ntiles;
};

template <bool SWIGLU>
__device__ __forceinline__ int wave_nrow(int wn, int ni) {
  if (SWIGLU) return (ni >= 2 ? 128 : 0) + wn * 64 + (ni & 1) * 32;
  return wn * 128 + ni * 32;
}

template <bool SWIGLU>
__global__ __launch_bounds__(kGemmThreads, 1) void grouped_gemm_bf16_kernel(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kStageBytes];
  __shared__ int32_t s_pref[kMaxExperts + 1];
  __shared__ int32_t s_off[kMaxExperts + 1];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm = wave >> 1, wn = wave & 1;

  for (int i = tid; i <= p.E; i += kGemmThreads) {
    s_pref[i] = p.mtile_prefix[i];
    s_off[i] = p.offsets[i];
  }
  __syncthreads();

  const int NT = p.ntiles;
  const int K = p.K;
  const int N = p.N;
  const int64_t total = int64_t(s_pref[p.E]) * NT;
  const int xcd = blockIdx.x % kNumXcd;
  const int slot = blockIdx.x / kNumXcd;
  const int slots = gridDim.x / kNumXcd;
  const int64_t per = (total + kNumXcd - 1) / kNumXcd;
  const int64_t chunk_lo = int64_t(xcd) * per;
  const int64_t chunk_hi = chunk_lo + per < total ? chunk_lo + per : total;

  // Global -> LDS staging: pass i moves rows i*32 + (tid / 8), 16-byte chunk tid % 8.
  const int lr = tid >> 3;
  const int lc = tid & 7;
  const uint32_t lds_store = uint32_t(lr * kRowBytes + ((lc ^ (lr & 7)) << 4));
  // MFMA operand reads: row (lane % 32) of a 32-row block, chunk 2*s + lane / 32.
  const uint32_t lds_read_row = uint32_t((lane & 31) * kRowBytes);
  const int sw = lane & 7;
  const int khalf = lane >> 5;

  for (int64_t L = chunk_lo + slot; L < chunk_hi; L += slots) {
    // ---- decode the tile
    const int e = find_expert(s_pref, p.E, L / NT);
    const int mt_e = s_pref[e + 1] - s_pref[e];
    const int64_t local = L - int64_t(s_pref[e]) * NT;
    const int64_t gsize = int64_t(mt_e) * kGroupN;
    const int ng = int(local / gsize);
    const int rem = int(local - int64_t(ng) * gsize);
    const int gw = min(kGroupN, NT - ng * kGroupN);
    const int mt = rem / gw;
    const int nt = ng * kGroupN + rem % gw;
    const int row0 = s_off[e] + mt * kBM;
    const int row_end = s_off[e + 1];

    // ---- per-thread global sources (byte offsets, rows clamped into range)
    const uint8_t* abase = reinterpret_cast<const uint8_t*>(p.act) + int64_t(row0) * K * 2;
    const int64_t wexp = int64_t(e) * N * K * 2;
    const uint8_t* wbase0 = reinterpret_cast<const uint8_t*>(p.w0) + wexp;
    const uint8_t* wbase1 = reinterpret_cast<const uint8_t*>(SWIGLU ? p.w1 : p.w0) + wexp;
    const int n0 = SWIGLU ? nt * 128 : nt * 256;
    uint32_t aoff[8], woff[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = i * 32 + lr;
      const int ar = min(row0 + r, row_end - 1) - row0;
      aoff[i] = uint32_t(ar) * uint32_t(K * 2) + uint32_t(lc * 16);
      const int wr = SWIGLU ? min(n0 + (i & 3) * 32 + lr, N - 1) : min(n0 + r, N - 1);
      woff[i] = uint32_t(wr) * uint32_t(K * 2) + uint32_t(lc * 16);
    }

    f32x16 acc[4][4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;

    u32x4 ga[8], gw8[8];
    auto gload = [&](int kt) {
      const uint32_t kb = uint32_t(kt) * kRowBytes;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ga[i] = *reinterpret_cast<const u32x4*>(abase + aoff[i] + kb);
        const uint8_t* wb = (SWIGLU && i >= 4) ? wbase1 : wbase0;
        gw8[i] = *reinterpret_cast<const u32x4*>(wb + woff[i] + kb);
      }
    };
    auto lstore = [&](int buf) {
      uint8_t* sW = smem + buf * kStageBytes;
      uint8_t* sX = sW + kOpBytes;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        *reinterpret_cast<u32x4*>(sW + i * 32 * kRowBytes + lds_store) = gw8[i];
        *reinterpret_cast<u32x4*>(sX + i * 32 * kRowBytes + lds_store) = ga[i];
      }
    };

    const int KT = K / kBK;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < KT) gload(kt + 1);
      const uint8_t* sW = smem + buf * kStageBytes;
      const uint8_t* sX = sW + kOpBytes;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const uint32_t coff = uint32_t(((2 * s + khalf) ^ sw) << 4);
        bf16x8 wf[4], xf[4];
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          wf[ni] = *reinterpret_cast<const bf16x8*>(sW + wave_nrow<SWIGLU>(wn, ni) * kRowBytes +
                                                    lds_read_row + coff);
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
          xf[mi] = *reinterpret_cast<const bf16x8*>(sX + (wm * 128 + mi * 32) * kRowBytes +
                                                    lds_read_row + coff);
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 4; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ni], xf[mi], acc[mi][ni], 0, 0, 0);
      }
      if (kt + 1 < KT) lstore(buf ^ 1);
      __syncthreads();
    }

    // ---- epilogue: lane holds columns n + 8*blk + 4*khalf + {0..3} of row (lane % 32)
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      const int row = row0 + wm * 128 + mi * 32 + (lane & 31);
      if (row < row_end) {
        uint16_t* orow = p.out + int64_t(row) * N;
        if (SWIGLU) {
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) {
#pragma unroll
            for (int blk = 0; blk < 4; ++blk) {
              const int f = n0 + wn * 64 + ni * 32 + blk * 8 + khalf * 4;
              if (f < N) {
                float hv[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                  hv[q] = silu(acc[mi][ni][blk * 4 + q]) * acc[mi][ni + 2][blk * 4 + q];
                u32x2 pk;
                pk[0] = pack_bf16x2(hv[0], hv[1]);
                pk[1] = pack_bf16x2(hv[2], hv[3]);
                *reinterpret_cast<u32x2*>(orow + f) = pk;
              }
            }
          }
        } else {
#pragma unroll
          for (int ni = 0; ni < 4; ++ni) {
#pragma unroll
            for (int blk = 0; blk < 4; ++blk) {
              const int n = n0 + wn * 128 + ni * 32 + blk * 8 + khalf * 4;
              if (n < N) {
                u32x2 pk;
                pk[0] = pack_bf16x2(acc[mi][ni][blk * 4 + 0], acc[mi][ni][blk * 4 + 1]);
                pk[1] = pack_bf16x2(acc[mi][ni][blk * 4 + 2], acc[mi][ni][blk * 4 + 3]);
                *reinterpret_cast<u32x2*>(orow + n) = pk;
              }
            }
          }
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------- fp32 GEMM
// Plain LDS-tiled fp32 FMA kernel for the fp32 layer: 64 x 64 outputs per
// block (GEMM-1: 64 features of both gate and up), 4 x 4 per thread.
constexpr int kFM = 64, kFN = 64, kFK = 16;

struct GemmArgsF {
  const float* act;
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
  const int64_t arow = min(row0 + lrow, row_end - 1);
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

int grid_for(int64_t upper_tiles, int num_cu) {
  int64_t g = upper_tiles < num_cu ? upper_tiles : num_cu;
  g = (g + kNumXcd - 1) / kNumXcd * kNumXcd;     // whole XCD rounds
  if (g < kNumXcd) g = kNumXcd;
  return int(g);
}

}  // namespace

hipError_t launch_ffn_bf16(const uint16_t* x_perm, const int32_t* offsets, int64_t R, int E, int H,
                           int F, const uint16_t* wg, const uint16_t* wu, const uint16_t* wd,
                           uint16_t* y_perm, int32_t* mtile_prefix, uint16_t* h, int num_cu,
                           hipStream_t s) {
  MOE_LAUNCH("ffn_tile_prefix", tile_prefix_kernel, dim3(1), dim3(256), s, offsets, E, kBM, mtile_prefix);
  const int64_t mtiles_upper = (R + int64_t(E) * (kBM - 1)) / kBM;

  GemmArgs a1{x_perm, wg, wu, h, offsets, mtile_prefix, E, H, F, (F + 127) / 128};
  MOE_LAUNCH("ffn_gemm1_gate_up", grouped_gemm_bf16_kernel<true>,
             dim3(grid_for(mtiles_upper * a1.ntiles, num_cu)), dim3(kGemmThreads), s, a1);
  GemmArgs a2{h, wd, nullptr, y_perm, offsets, mtile_prefix, E, F, H, (H + 255) / 256};
  MOE_LAUNCH("ffn_gemm2_down", grouped_gemm_bf16_kernel<false>,
             dim3(grid_for(mtiles_upper * a2.ntiles, num_cu)), dim3(kGemmThreads), s, a2);
  return hipGetLastError();
}

hipError_t launch_ffn_f32(const float* x_perm, const int32_t* offsets, int64_t R, int E, int H, int F,
                          const float* wg, const float* wu, const float* wd, float* y_perm,
                          int32_t* mtile_prefix, float* h, hipStream_t s) {
  MOE_LAUNCH("ffn_tile_prefix", tile_prefix_kernel, dim3(1), dim3(256), s, offsets, E, kFM, mtile_prefix);
  const int64_t mtiles_upper = (R + int64_t(E) * (kFM - 1)) / kFM;
  GemmArgsF a1{x_perm, wg, wu, h, offsets, mtile_prefix, E, H, F, (F + kFN - 1) / kFN};
  MOE_LAUNCH("ffn_gemm1_gate_up", grouped_gemm_f32_kernel<true>, dim3(unsigned(mtiles_upper * a1.ntiles)),
             dim3(256), s, a1);
  GemmArgsF a2{h, wd, nullptr, y_perm, offsets, mtile_prefix, E, F, H, (H + kFN - 1) / kFN};
  MOE_LAUNCH("ffn_gemm2_down", grouped_gemm_f32_kernel<false>, dim3(unsigned(mtiles_upper * a2.ntiles)),
             dim3(256), s, a2);
  return hipGetLastError();
}

}  // namespace moe
