// moe_route: top-k gating on gfx950.
//
// Each token is handled by a segment of G lanes of one wavefront (G a power of
// two, 1..64), each lane holding V <= 8 of the token's E logits as orderable
// 32-bit keys (the unsigned order of orderable(l) is the order of l, with -0
// equal to +0).  Round j of k picks the slot-j winner: the segment maximum of the
// keys, then the segment minimum of the expert ids holding that key, so ties go
// to the lower expert id exactly as the layer's gate orders experts; the owning
// lane retires it.  Segment reductions use DPP lane permutes (quad swaps, then
// the 8- and 16-lane mirrors, which pair lanes of different halves once the
// halves agree); wider segments fall back to lane shuffles.  Gate weights are a
// softmax over the selected logits (renormalize = 1) or over all E
// (renormalize = 0), in fp32.
#include <algorithm>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kRouteThreads = 256;

// src of lane i for DPP control CTRL (quad_perm / row mirrors), inside its row.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;           // quad_perm [1, 0, 3, 2]
constexpr int kQuadXor2 = 0x4E;           // quad_perm [2, 3, 0, 1]
constexpr int kRowHalfMirror = 0x141;     // lane i <- lane 7 - i within each 8
constexpr int kRowMirror = 0x140;         // lane i <- lane 15 - i within each 16

// All-reduce over aligned segments of G lanes.
template <int G, typename Op>
__device__ __forceinline__ uint32_t seg_reduce(uint32_t v, Op op) {
  if constexpr (G >= 2) v = op(v, dpp<kQuadXor1>(v));
  if constexpr (G >= 4) v = op(v, dpp<kQuadXor2>(v));
  if constexpr (G >= 8) v = op(v, dpp<kRowHalfMirror>(v));
  if constexpr (G >= 16) v = op(v, dpp<kRowMirror>(v));
  if constexpr (G >= 32) v = op(v, uint32_t(__shfl_xor(int(v), 16)));
  if constexpr (G >= 64) v = op(v, uint32_t(__shfl_xor(int(v), 32)));
  return v;
}

// One block per group of kRouteThreads / G tokens.
template <int G, int V, bool VEC4, int KMAX>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(const float* __restrict__ logits,
                                                             int64_t T, int E, int k,
                                                             int renormalize,
                                                             int32_t* __restrict__ topk_ids,
                                                             float* __restrict__ topk_w) {
  constexpr int kTokensPerBlock = kRouteThreads / G;
  const int g = threadIdx.x & (G - 1);                       // lane inside the token's segment
  const int e0 = g * V;

  auto load = [&](int64_t t, float* vals) {
    const bool valid = t < T;                                 // the same for a whole segment
    if (VEC4) {
      // E % 4 == 0 and V % 4 == 0: every lane's slice starts 16-byte aligned.
      const f32x4* src = reinterpret_cast<const f32x4*>(logits + (valid ? t : 0) * E + e0);
#pragma unroll
      for (int v = 0; v < V; v += 4) {
        f32x4 q = {0.f, 0.f, 0.f, 0.f};
        if (valid && e0 + v < E) q = __builtin_nontemporal_load(src + v / 4);
        vals[v] = q[0]; vals[v + 1] = q[1]; vals[v + 2] = q[2]; vals[v + 3] = q[3];
      }
    } else {
#pragma unroll
      for (int v = 0; v < V; ++v)
        vals[v] = (valid && e0 + v < E) ? __builtin_nontemporal_load(logits + t * E + e0 + v) : 0.f;
    }
  };

  float cur[V];
  const int64_t t = int64_t(blockIdx.x) * kTokensPerBlock + threadIdx.x / G;
  load(t, cur);
  {
    const bool valid = t < T;

    // Key 0 is below every real key (orderable(-inf) = 0x007FFFFF): padding and
    // retired experts.
    uint32_t key[V];
#pragma unroll
    for (int v = 0; v < V; ++v) key[v] = (valid && e0 + v < E) ? orderable(cur[v]) : 0u;

    uint32_t selk[KMAX];
    uint32_t sele[KMAX];
    const auto umax = [](uint32_t a, uint32_t b) { return a > b ? a : b; };
    const auto umin = [](uint32_t a, uint32_t b) { return a < b ? a : b; };
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        uint32_t m = key[0];
#pragma unroll
        for (int v = 1; v < V; ++v) m = umax(m, key[v]);
        m = seg_reduce<G>(m, umax);
        // The lowest expert holding the maximum: lanes are in expert order and so
        // are a lane's v, so the segment minimum of each lane's first match is it.
        uint32_t id = 0xFFFFFFFFu;
#pragma unroll
        for (int v = V - 1; v >= 0; --v) id = key[v] == m ? uint32_t(e0 + v) : id;
        id = seg_reduce<G>(id, umin);
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
        denom += p[j];                                      // slot order
      }
    }
    if (!renormalize) {
      float s = 0.f;
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (valid && e0 + v < E) s += expf(cur[v] - lmax);
      const auto fadd = [](uint32_t a, uint32_t b) {
        return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
      };
      denom = __uint_as_float(seg_reduce<G>(__float_as_uint(s), fadd));
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

// One block per token group (the loop runs once): blocks past the resident
// wave start as earlier ones finish, so their loads overlap the selection rounds
// of the running ones.  (A grid of one resident wave walking the tokens with a
// register prefetch measured 12-14% slower at 131072 tokens x 64 experts and the
// same at 4096 tokens, where both are 16 blocks.)
template <int G, int V, bool VEC4, int KMAX>
hipError_t launch_k(const float* logits, int64_t T, int E, int k, int renorm, int32_t* ids, float* w,
                    hipStream_t s) {
  const int64_t per_block = kRouteThreads / G;
  const int64_t blocks = (T + per_block - 1) / per_block;
  MOE_LAUNCH("route", (route_kernel<G, V, VEC4, KMAX>), dim3(unsigned(blocks)), dim3(kRouteThreads), s,
             logits, T, E, k, renorm, ids, w);
  return hipGetLastError();
}

// The selection state in registers is sized for k <= 4, k <= 8 or k <= 16 slots.
template <int G, int V, bool VEC4>
hipError_t launch_gvk(const float* logits, int64_t T, int E, int k, int renorm, int32_t* ids, float* w,
                      int num_cu, hipStream_t s) {
  (void)num_cu;
  if (k <= 4) return launch_k<G, V, VEC4, 4>(logits, T, E, k, renorm, ids, w, s);
  if (k <= 8) return launch_k<G, V, VEC4, 8>(logits, T, E, k, renorm, ids, w, s);
  return launch_k<G, V, VEC4, kMaxTopK>(logits, T, E, k, renorm, ids, w, s);
}

template <int G, int V>
hipError_t launch_gv(const float* logits, int64_t T, int E, int k, int renorm, int32_t* ids, float* w,
                     int num_cu, hipStream_t s) {
  if constexpr ((V % 4) == 0) {
    if ((E % 4) == 0) return launch_gvk<G, V, true>(logits, T, E, k, renorm, ids, w, num_cu, s);
  }
  return launch_gvk<G, V, false>(logits, T, E, k, renorm, ids, w, num_cu, s);
}

// G > 1 only arises with V in 5..8 (E > 8 gives V = ceil(E / G) > 4).
template <int G>
hipError_t launch_g(const float* logits, int64_t T, int E, int k, int V, int renorm, int32_t* ids,
                    float* w, int num_cu, hipStream_t s) {
  switch (V) {
    case 5: return launch_gv<G, 5>(logits, T, E, k, renorm, ids, w, num_cu, s);
    case 6: return launch_gv<G, 6>(logits, T, E, k, renorm, ids, w, num_cu, s);
    case 7: return launch_gv<G, 7>(logits, T, E, k, renorm, ids, w, num_cu, s);
    default: return launch_gv<G, 8>(logits, T, E, k, renorm, ids, w, num_cu, s);
  }
}

}  // namespace

// Segment width: the smallest power of two G with G * 8 >= E; V = ceil(E / G) <= 8.
void route_shape(int E, int* G, int* V) {
  int g = 1;
  while (g * 8 < E) g <<= 1;
  *G = g;
  *V = (E + g - 1) / g;
}

hipError_t launch_route(const float* logits, int64_t T, int E, int k, int renorm, int32_t* ids,
                        float* w, int num_cu, hipStream_t s) {
  int G, V;
  route_shape(E, &G, &V);
  switch (G) {
    case 1:
      switch (V) {
        case 1: return launch_gv<1, 1>(logits, T, E, k, renorm, ids, w, num_cu, s);
        case 2: return launch_gv<1, 2>(logits, T, E, k, renorm, ids, w, num_cu, s);
        case 3: return launch_gv<1, 3>(logits, T, E, k, renorm, ids, w, num_cu, s);
        case 4: return launch_gv<1, 4>(logits, T, E, k, renorm, ids, w, num_cu, s);
        case 5: return launch_gv<1, 5>(logits, T, E, k, renorm, ids, w, num_cu, s);
        case 6: return launch_gv<1, 6>(logits, T, E, k, renorm, ids, w, num_cu, s);
        case 7: return launch_gv<1, 7>(logits, T, E, k, renorm, ids, w, num_cu, s);
        default: return launch_gv<1, 8>(logits, T, E, k, renorm, ids, w, num_cu, s);
      }
    case 2: return launch_g<2>(logits, T, E, k, V, renorm, ids, w, num_cu, s);
    case 4: return launch_g<4>(logits, T, E, k, V, renorm, ids, w, num_cu, s);
    case 8: return launch_g<8>(logits, T, E, k, V, renorm, ids, w, num_cu, s);
    case 16: return launch_g<16>(logits, T, E, k, V, renorm, ids, w, num_cu, s);
    default: return launch_g<32>(logits, T, E, k, V, renorm, ids, w, num_cu, s);
  }
}

}  // namespace moe
