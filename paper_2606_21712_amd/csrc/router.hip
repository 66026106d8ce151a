// moe_router_topk: the MoE gate's router GEMM fused with top-k selection on gfx950.
//
// logits[t, e] = x[t] . w_router[e] (bf16 operands, fp32 accumulation on the
// matrix cores), then the gate of moe_route on those fp32 logits: the k largest,
// ties to the lower expert id, softmax over the selected (or all) logits.  The
// logits never leave the chip unless the caller asks for them.
//
// Three kernels, one k order (so a token's result does not depend on its batch):
// with 64 tokens per compute unit and H % 128 = 0, blocks of four wavefronts share
// the router matrix through LDS (router_lds_kernel); with fewer tokens and
// H % 128 = 0, four wavefronts split each 16-token block's k (router_splitk_kernel);
// otherwise one wavefront takes MB blocks of 16 tokens against all experts
// (router_kernel), reading the router matrix from L2.  All use
// v_mfma_f32_16x16x32_bf16 on up to four 16-expert blocks (E <= 64).  The fp32
// logits go through LDS to the selection, where 4 lanes hold one token's logits
// and each round takes a quad maximum of orderable keys, then a quad minimum of
// the expert ids holding it (DPP lane permutes).
#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kTok = 16;                  // tokens per MFMA block
constexpr int kUnroll = 4;                // k-steps of 32 whose loads are issued together

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ uint32_t quad_max(uint32_t v) {
  v = max(v, dpp<0xB1>(v));              // quad_perm [1, 0, 3, 2]
  return max(v, dpp<0x4E>(v));           // quad_perm [2, 3, 0, 1]
}
__device__ __forceinline__ uint32_t quad_min(uint32_t v) {
  v = min(v, dpp<0xB1>(v));
  return min(v, dpp<0x4E>(v));
}
__device__ __forceinline__ float quad_sum(float v) {
  v += __uint_as_float(dpp<0xB1>(__float_as_uint(v)));
  return v + __uint_as_float(dpp<0x4E>(__float_as_uint(v)));
}

// MB 16-token blocks, NB 16-expert blocks (E <= 16 NB); KMAX slots of selection state.
template <int MB, int NB, int KMAX>
__global__ __launch_bounds__(64) void router_kernel(const uint16_t* __restrict__ x,
                                                   const uint16_t* __restrict__ w, int64_t T, int E,
                                                   int k, int H, int renormalize,
                                                   float* __restrict__ logits_out,
                                                   int32_t* __restrict__ topk_ids,
                                                   float* __restrict__ topk_w) {
  constexpr int EP = 16 * NB;
  constexpr int V = EP / 4;                 // logits per lane in the selection (4 lanes per token)
  __shared__ float s_log[MB * kTok][EP + 1];

  const int lane = threadIdx.x;
  const int64_t t0 = int64_t(blockIdx.x) * (MB * kTok);
  // MFMA operand lanes: row (token or expert) lane % 16, k sub-block lane / 16 (8 values)
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  bool xv[MB];
  const bf16x8* xr[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    xv[mb] = t0 + mb * kTok + r16 < T;
    xr[mb] = reinterpret_cast<const bf16x8*>(x + (xv[mb] ? t0 + mb * kTok + r16 : 0) * H + kq * 8);
  }
  const bf16x8* wr[NB];
  bool wv[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    wv[nb] = nb * 16 + r16 < E;
    wr[nb] = reinterpret_cast<const bf16x8*>(w + int64_t(wv[nb] ? nb * 16 + r16 : 0) * H + kq * 8);
  }
  f32x4 acc[MB][NB], tot[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16x8 zero = {};
  // k order of the sum (the same in every router kernel, so a token's logits do not
  // depend on the batch it arrives in): with H % 128 = 0, four quarter sums over
  // consecutive 32-k chunks, added as ((q0 + q1) + q2) + q3; otherwise one chain.
  const int qc = (H % 128 == 0) ? H / 128 : 0;         // 32-k chunks per quarter
  auto fold = [&](int c) {                              // before chunk c
    if (qc == 0 || c == 0 || c % qc != 0) return;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        tot[mb][nb] = c == qc ? acc[mb][nb] : tot[mb][nb] + acc[mb][nb];
        acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
  };

  // k-steps of 32: operand vector index k0 / 8 (each bf16x8 covers 8 of k)
  constexpr int U = MB * NB > 8 ? 2 : kUnroll;        // keep the operands in flight in registers
  int k0 = 0;
  for (; k0 + 32 * U <= H; k0 += 32 * U) {
    bf16x8 a[U][MB], b[U][NB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        a[u][mb] = xv[mb] ? __builtin_nontemporal_load(xr[mb] + (k0 + 32 * u) / 8) : zero;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) b[u][nb] = wv[nb] ? wr[nb][(k0 + 32 * u) / 8] : zero;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      fold((k0 + 32 * u) / 32);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][mb], b[u][nb], acc[mb][nb], 0, 0, 0);
    }
  }
  for (; k0 < H; k0 += 32) {
    fold(k0 / 32);
    bf16x8 b[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) b[nb] = wv[nb] ? wr[nb][k0 / 8] : zero;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const bf16x8 a = xv[mb] ? __builtin_nontemporal_load(xr[mb] + k0 / 8) : zero;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[nb], acc[mb][nb], 0, 0, 0);
    }
  }

  if (qc != 0) {                                        // the last quarter
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = tot[mb][nb] + acc[mb][nb];
  }
  // 16 x 16 output: lane holds tokens 4 (lane / 16) + q of expert block column lane % 16
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 4; ++q) s_log[mb * kTok + 4 * kq + q][nb * 16 + r16] = acc[mb][nb][q];
  __syncthreads();

  // ---- selection, 16 tokens per pass: token tt = lane / 4 of the pass, lane g = lane % 4
  // holds experts g V .. g V + V - 1
#pragma unroll 1
  for (int pass = 0; pass < MB; ++pass) {
    const int tt = pass * kTok + (lane >> 2);
    const int g = lane & 3;
    const int64_t t = t0 + tt;
    const bool valid = t < T;
    const int e0 = g * V;
    float vals[V];
    uint32_t key[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const bool live = e0 + v < E;
      vals[v] = live ? s_log[tt][e0 + v] : 0.f;
      key[v] = live ? orderable(vals[v]) : 0u;           // 0 is below every real key
    }
    if (logits_out != nullptr && valid) {
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (e0 + v < E) logits_out[t * E + e0 + v] = vals[v];
    }
    uint32_t selk[KMAX];
    uint32_t sele[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        uint32_t m = key[0];
#pragma unroll
        for (int v = 1; v < V; ++v) m = max(m, key[v]);
        m = quad_max(m);
        uint32_t id = 0xFFFFFFFFu;
#pragma unroll
        for (int v = V - 1; v >= 0; --v) id = key[v] == m ? uint32_t(e0 + v) : id;
        id = quad_min(id);
#pragma unroll
        for (int v = 0; v < V; ++v) key[v] = uint32_t(e0 + v) == id ? 0u : key[v];
        selk[j] = m;
        sele[j] = id;
      } else {
        selk[j] = 0u;
        sele[j] = 0u;
      }
    }
    const float lmax = from_orderable(selk[0]);
    float p[KMAX];
    float denom = 0.f;
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        p[j] = expf(from_orderable(selk[j]) - lmax);
        denom += p[j];                                        // slot order
      }
    }
    if (!renormalize) {
      float s = 0.f;
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (e0 + v < E) s += expf(vals[v] - lmax);
      denom = quad_sum(s);
    }
    if (valid && g == 0) {
#pragma unroll
      for (int j = 0; j < KMAX; ++j) {
        if (j < k) {
          topk_ids[t * k + j] = int32_t(sele[j]);
          topk_w[t * k + j] = p[j] / denom;
        }
      }
    }
  }
}

// Large batches: four wavefronts per block (64 tokens), the router matrix staged
// through LDS in k-slices of SK (256 or 128) that the four share, so L2 serves it
// once per block instead of once per wavefront.  Slices are double-buffered and
// filled by direct global -> LDS loads; the 16-byte chunks of each 2 SK-byte expert
// row are stored at chunk ^ (row & 15), so the 16 expert rows an MFMA operand read
// touches land on distinct banks.  Each wavefront streams its 16 token rows into
// registers one slice ahead.  The logits for the selection reuse the slices' LDS
// once the k loop is done, which keeps a block at 2 SK x E bytes (64 KB at E = 64,
// SK = 256: two blocks per compute unit).  Selection as in router_kernel.
constexpr int kLdsWaves = 4;

template <int NB, int KMAX, int SK>
__global__ __launch_bounds__(kLdsWaves * 64) void router_lds_kernel(const uint16_t* __restrict__ x,
                                                                   const uint16_t* __restrict__ w, int64_t T,
                                                                   int E, int k, int H, int renormalize,
                                                                   float* __restrict__ logits_out,
                                                                   int32_t* __restrict__ topk_ids,
                                                                   float* __restrict__ topk_w) {
  constexpr int EP = 16 * NB;
  constexpr int V = EP / 4;
  constexpr int kSliceRowBytes = SK * 2;              // one expert row of a slice
  constexpr int kSliceSteps = SK / 32;                // MFMA k-steps per slice
  constexpr int kRowsPerDma = 1024 / kSliceRowBytes;  // expert rows per 1 KB load
  constexpr int kRowChunks = kSliceRowBytes / 16;     // 16-byte chunks per row
  constexpr int kSliceBytes = EP * kSliceRowBytes;
  // two slices; after the k loop the same bytes hold the wavefronts' logits
  __shared__ __attribute__((aligned(1024))) uint8_t ws[2 * kSliceBytes];
  static_assert(sizeof(float) * kLdsWaves * kTok * (EP + 1) <= 2 * kSliceBytes, "logits fit the slices");
  uint8_t* const ws0 = ws;
  uint8_t* const ws1 = ws + kSliceBytes;
  float (*s_log)[kTok][EP + 1] = reinterpret_cast<float (*)[kTok][EP + 1]>(ws);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (T < 0) {                                        // never taken: keeps the DMA-filled slices' reads
    ws0[tid] = 0;
    ws1[tid] = 0;
  }
  const int64_t t0 = (int64_t(blockIdx.x) * kLdsWaves + wave) * kTok;
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  const bool xv = t0 + r16 < T;
  const bf16x8* xr = reinterpret_cast<const bf16x8*>(x + (xv ? t0 + r16 : 0) * H + kq * 8);
  const bf16x8 zero = {};

  // slice DMA: 1 KB instructions of kRowsPerDma expert rows each, dealt over the
  // four wavefronts; lane q fills row kRowsPerDma i + q / kRowChunks, chunk position
  // q % kRowChunks
  const __amdgpu_buffer_rsrc_t rw =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(w), 0, int(int64_t(E) * H * 2), 0x00020000);
  constexpr int kDma = EP / kRowsPerDma;
  constexpr int kDmaPerWave = (kDma + kLdsWaves - 1) / kLdsWaves;
  // (a fixed-size array: sized by the template-dependent count, the host pass
  // drops the kernel's launch stub)
  static_assert(kDmaPerWave <= 8, "at most 64 experts");
  uint32_t woff[8];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int i = j * kLdsWaves + wave;               // instruction index
    const int row = kRowsPerDma * i + lane / kRowChunks;
    const int pos = lane % kRowChunks;
    const int chunk = pos ^ (row & 15);               // logical 16-byte chunk this lane fetches
    woff[j] = row < E ? uint32_t(row) * uint32_t(H) * 2u + uint32_t(chunk) * 16u : 0x80000000u;
  }
  auto issue_w = [&](uint8_t* slice, int s) {
    const int kb = s * kSliceRowBytes;
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j) {
      const int i = j * kLdsWaves + wave;
      if (i < kDma) __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, slice + i * 1024, 16, woff[j], kb, 0, 0);
    }
  };
  auto load_x = [&](bf16x8* a, int s) {
#pragma unroll
    for (int u = 0; u < kSliceSteps; ++u)
      a[u] = xv ? __builtin_nontemporal_load(xr + (s * SK + 32 * u) / 8) : zero;
  };

  f32x4 acc[NB], tot[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // k order as router_kernel: four quarter sums, added ((q0 + q1) + q2) + q3
  const int qc = H / 128;                             // 32-k chunks per quarter
  auto compute = [&](const uint8_t* slice, const bf16x8* a, int s) {
#pragma unroll
    for (int u = 0; u < kSliceSteps; ++u) {
      const int c = s * kSliceSteps + u;
      if (c != 0 && c % qc == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          tot[nb] = c == qc ? acc[nb] : tot[nb] + acc[nb];
          acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int row = nb * 16 + r16;
        const int chunk = 4 * u + kq;
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(slice + row * kSliceRowBytes + ((chunk ^ (row & 15)) * 16));
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u], b, acc[nb], 0, 0, 0);
      }
    }
  };

  const int S = H / SK;
  bf16x8 xa[2][kSliceSteps];
  issue_w(ws0, 0);
  load_x(xa[0], 0);
  auto step = [&](uint8_t* cur, uint8_t* nxt, const bf16x8* a_cur, bf16x8* a_nxt, int s) {
    __builtin_amdgcn_s_waitcnt(0x0F70);               // this slice's loads (and the x rows) landed
    __syncthreads();                                  // ... for every wave; the other slice is free
    if (s + 1 < S) {
      issue_w(nxt, s + 1);
      load_x(a_nxt, s + 1);
    }
    compute(cur, a_cur, s);
  };
  int s = 0;
  for (; s + 2 <= S; s += 2) {
    step(ws0, ws1, xa[0], xa[1], s);
    step(ws1, ws0, xa[1], xa[0], s + 1);
  }
  if (s < S) step(ws0, ws1, xa[0], xa[1], s);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = tot[nb] + acc[nb];   // the last quarter
  __syncthreads();                                    // every wave is done with the slices

  // 16 x 16 outputs: lane holds tokens 4 (lane / 16) + q of expert column lane % 16
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int q = 0; q < 4; ++q) s_log[wave][4 * kq + q][nb * 16 + r16] = acc[nb][q];
  __syncthreads();

  // selection: 16 tokens per wavefront, token tt = lane / 4, lane g = lane % 4 holds
  // experts g V .. g V + V - 1
  const int tt = lane >> 2;
  const int g = lane & 3;
  const int64_t t = t0 + tt;
  const bool valid = t < T;
  const int e0 = g * V;
  float vals[V];
  uint32_t key[V];
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const bool live = e0 + v < E;
    vals[v] = live ? s_log[wave][tt][e0 + v] : 0.f;
    key[v] = live ? orderable(vals[v]) : 0u;
  }
  if (logits_out != nullptr && valid) {
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (e0 + v < E) logits_out[t * E + e0 + v] = vals[v];
  }
  uint32_t selk[KMAX];
  uint32_t sele[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
      uint32_t m = key[0];
#pragma unroll
      for (int v = 1; v < V; ++v) m = max(m, key[v]);
      m = quad_max(m);
      uint32_t id = 0xFFFFFFFFu;
#pragma unroll
      for (int v = V - 1; v >= 0; --v) id = key[v] == m ? uint32_t(e0 + v) : id;
      id = quad_min(id);
#pragma unroll
      for (int v = 0; v < V; ++v) key[v] = uint32_t(e0 + v) == id ? 0u : key[v];
      selk[j] = m;
      sele[j] = id;
    } else {
      selk[j] = 0u;
      sele[j] = 0u;
    }
  }
  const float lmax = from_orderable(selk[0]);
  float p[KMAX];
  float denom = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
      p[j] = expf(from_orderable(selk[j]) - lmax);
      denom += p[j];
    }
  }
  if (!renormalize) {
    float sum = 0.f;
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (e0 + v < E) sum += expf(vals[v] - lmax);
    denom = quad_sum(sum);
  }
  if (valid && g == 0) {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        topk_ids[t * k + j] = int32_t(sele[j]);
        topk_w[t * k + j] = p[j] / denom;
      }
    }
  }
}

// Small batches (fewer than 8 sixteen-token wavefronts per compute unit): four
// wavefronts per 16 tokens, each a quarter of the k range, their fp32 partial
// logits added in wavefront order through LDS; wavefront 0 then selects.
constexpr int kSplitWaves = 4;

template <int NB, int KMAX>
__global__ __launch_bounds__(kSplitWaves * 64) void router_splitk_kernel(const uint16_t* __restrict__ x,
                                                                        const uint16_t* __restrict__ w, int64_t T,
                                                                        int E, int k, int H, int renormalize,
                                                                        float* __restrict__ logits_out,
                                                                        int32_t* __restrict__ topk_ids,
                                                                        float* __restrict__ topk_w) {
  constexpr int EP = 16 * NB;
  constexpr int V = EP / 4;
  __shared__ float s_part[kSplitWaves][kTok][EP + 1];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int64_t t0 = int64_t(blockIdx.x) * kTok;
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  const int Hq = H / kSplitWaves;                     // a multiple of 32
  const int kbase = wave * Hq;
  const bool xv = t0 + r16 < T;
  const bf16x8* xr = reinterpret_cast<const bf16x8*>(x + (xv ? t0 + r16 : 0) * H + kbase + kq * 8);
  const bf16x8* wr[NB];
  bool wv[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    wv[nb] = nb * 16 + r16 < E;
    wr[nb] = reinterpret_cast<const bf16x8*>(w + int64_t(wv[nb] ? nb * 16 + r16 : 0) * H + kbase + kq * 8);
  }
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16x8 zero = {};
  int k0 = 0;
  for (; k0 + 32 * kUnroll <= Hq; k0 += 32 * kUnroll) {
    bf16x8 a[kUnroll], b[kUnroll][NB];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      a[u] = xv ? __builtin_nontemporal_load(xr + (k0 + 32 * u) / 8) : zero;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) b[u][nb] = wv[nb] ? wr[nb][(k0 + 32 * u) / 8] : zero;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u], b[u][nb], acc[nb], 0, 0, 0);
  }
  for (; k0 < Hq; k0 += 32) {
    const bf16x8 a = xv ? __builtin_nontemporal_load(xr + k0 / 8) : zero;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const bf16x8 b = wv[nb] ? wr[nb][k0 / 8] : zero;
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[nb], 0, 0, 0);
    }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int q = 0; q < 4; ++q) s_part[wave][4 * kq + q][nb * 16 + r16] = acc[nb][q];
  __syncthreads();
  if (wave != 0) return;

  // selection: token tt = lane / 4, lane g = lane % 4 holds experts g V .. g V + V - 1
  const int tt = lane >> 2;
  const int g = lane & 3;
  const int64_t t = t0 + tt;
  const bool valid = t < T;
  const int e0 = g * V;
  float vals[V];
  uint32_t key[V];
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const bool live = e0 + v < E;
    float l = 0.f;
    if (live) {
      l = s_part[0][tt][e0 + v];
#pragma unroll
      for (int q = 1; q < kSplitWaves; ++q) l += s_part[q][tt][e0 + v];   // quarters in k order
    }
    vals[v] = l;
    key[v] = live ? orderable(l) : 0u;
  }
  if (logits_out != nullptr && valid) {
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (e0 + v < E) logits_out[t * E + e0 + v] = vals[v];
  }
  uint32_t selk[KMAX];
  uint32_t sele[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
      uint32_t m = key[0];
#pragma unroll
      for (int v = 1; v < V; ++v) m = max(m, key[v]);
      m = quad_max(m);
      uint32_t id = 0xFFFFFFFFu;
#pragma unroll
      for (int v = V - 1; v >= 0; --v) id = key[v] == m ? uint32_t(e0 + v) : id;
      id = quad_min(id);
#pragma unroll
      for (int v = 0; v < V; ++v) key[v] = uint32_t(e0 + v) == id ? 0u : key[v];
      selk[j] = m;
      sele[j] = id;
    } else {
      selk[j] = 0u;
      sele[j] = 0u;
    }
  }
  const float lmax = from_orderable(selk[0]);
  float p[KMAX];
  float denom = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
      p[j] = expf(from_orderable(selk[j]) - lmax);
      denom += p[j];
    }
  }
  if (!renormalize) {
    float sum = 0.f;
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (e0 + v < E) sum += expf(vals[v] - lmax);
    denom = quad_sum(sum);
  }
  if (valid && g == 0) {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        topk_ids[t * k + j] = int32_t(sele[j]);
        topk_w[t * k + j] = p[j] / denom;
      }
    }
  }
}

template <int NB>
hipError_t launch_splitk(const uint16_t* x, const uint16_t* w, int64_t T, int E, int k, int H, int renorm,
                         float* logits, int32_t* ids, float* wts, hipStream_t s) {
  const dim3 grid(unsigned((T + kTok - 1) / kTok));
  const dim3 block(kSplitWaves * 64);
  if (k <= 4)
    MOE_LAUNCH("router_topk", (router_splitk_kernel<NB, 4>), grid, block, s, x, w, T, E, k, H, renorm, logits,
               ids, wts);
  else if (k <= 8)
    MOE_LAUNCH("router_topk", (router_splitk_kernel<NB, 8>), grid, block, s, x, w, T, E, k, H, renorm, logits,
               ids, wts);
  else
    MOE_LAUNCH("router_topk", (router_splitk_kernel<NB, kMaxTopK>), grid, block, s, x, w, T, E, k, H, renorm,
               logits, ids, wts);
  return hipGetLastError();
}

template <int NB, int SK>
hipError_t launch_lds(const uint16_t* x, const uint16_t* w, int64_t T, int E, int k, int H, int renorm,
                      float* logits, int32_t* ids, float* wts, hipStream_t s) {
  const dim3 grid(unsigned((T + kLdsWaves * kTok - 1) / (kLdsWaves * kTok)));
  const dim3 block(kLdsWaves * 64);
  if (k <= 4)
    MOE_LAUNCH("router_topk", (router_lds_kernel<NB, 4, SK>), grid, block, s, x, w, T, E, k, H, renorm, logits, ids,
               wts);
  else if (k <= 8)
    MOE_LAUNCH("router_topk", (router_lds_kernel<NB, 8, SK>), grid, block, s, x, w, T, E, k, H, renorm, logits, ids,
               wts);
  else
    MOE_LAUNCH("router_topk", (router_lds_kernel<NB, kMaxTopK, SK>), grid, block, s, x, w, T, E, k, H, renorm, logits,
               ids, wts);
  return hipGetLastError();
}

template <int MB, int NB>
hipError_t launch_mn(const uint16_t* x, const uint16_t* w, int64_t T, int E, int k, int H, int renorm,
                     float* logits, int32_t* ids, float* wts, hipStream_t s) {
  const dim3 grid(unsigned((T + MB * kTok - 1) / (MB * kTok)));
  if (k <= 4)
    MOE_LAUNCH("router_topk", (router_kernel<MB, NB, 4>), grid, dim3(64), s, x, w, T, E, k, H, renorm, logits,
               ids, wts);
  else if (k <= 8)
    MOE_LAUNCH("router_topk", (router_kernel<MB, NB, 8>), grid, dim3(64), s, x, w, T, E, k, H, renorm, logits,
               ids, wts);
  else
    MOE_LAUNCH("router_topk", (router_kernel<MB, NB, kMaxTopK>), grid, dim3(64), s, x, w, T, E, k, H, renorm,
               logits, ids, wts);
  return hipGetLastError();
}

// Tokens per wavefront: 64 when that still gives every compute unit 8 wavefronts,
// else 32, else 16.
template <int NB>
hipError_t launch_nb(const uint16_t* x, const uint16_t* w, int64_t T, int E, int k, int H, int renorm,
                     float* logits, int32_t* ids, float* wts, int num_cu, hipStream_t s) {
  // Enough 64-token blocks for every compute unit: the LDS-staged kernel.
  // Slices of 256 k where H allows (half the barriers of 128), else of 128.
  if (H % 128 == 0 && T >= int64_t(num_cu) * kLdsWaves * kTok) {
    if (H % 256 == 0) return launch_lds<NB, 256>(x, w, T, E, k, H, renorm, logits, ids, wts, s);
    return launch_lds<NB, 128>(x, w, T, E, k, H, renorm, logits, ids, wts, s);
  }
  const int64_t waves_wanted = int64_t(num_cu) * 8;
  // Fewer than 8 sixteen-token wavefronts per compute unit: split k four ways.
  if (H % (kSplitWaves * 32) == 0 && T < waves_wanted * kTok)
    return launch_splitk<NB>(x, w, T, E, k, H, renorm, logits, ids, wts, s);
  if (T >= waves_wanted * 64) return launch_mn<4, NB>(x, w, T, E, k, H, renorm, logits, ids, wts, s);
  if (T >= waves_wanted * 32) return launch_mn<2, NB>(x, w, T, E, k, H, renorm, logits, ids, wts, s);
  return launch_mn<1, NB>(x, w, T, E, k, H, renorm, logits, ids, wts, s);
}

}  // namespace

hipError_t launch_router_topk(const uint16_t* x, const uint16_t* w, int64_t T, int E, int k, int H, int renorm,
                              float* logits, int32_t* ids, float* wts, int num_cu, hipStream_t s) {
  switch ((E + 15) / 16) {
    case 1: return launch_nb<1>(x, w, T, E, k, H, renorm, logits, ids, wts, num_cu, s);
    case 2: return launch_nb<2>(x, w, T, E, k, H, renorm, logits, ids, wts, num_cu, s);
    case 3: return launch_nb<3>(x, w, T, E, k, H, renorm, logits, ids, wts, num_cu, s);
    default: return launch_nb<4>(x, w, T, E, k, H, renorm, logits, ids, wts, num_cu, s);
  }
}

}  // namespace moe
