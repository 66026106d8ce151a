// moe_route: top-k gating on gfx950.
//
// Each token is handled by a segment of G lanes of one wavefront (G a power of
// two, 1..64), each lane holding V <= 8 of the token's E logits.  A logit l of
// expert e becomes the 64-bit key (orderable(l) << 32) | (0xFFFFFFFF - e), so
// the integer maximum is the largest logit with ties going to the lower expert
// id, exactly as the layer's gate orders experts.  k rounds of a segment-wide
// maximum (xor shuffles inside the segment) pick the winners in slot order; the
// owning lane retires each winner.  Gate weights are a softmax over the
// selected logits (renormalize = 1) or over all E (renormalize = 0), in fp32.
#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kRouteThreads = 256;

template <int V, bool VEC4>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(const float* __restrict__ logits,
                                                             int64_t T, int E, int k, int G,
                                                             int renormalize,
                                                             int32_t* __restrict__ topk_ids,
                                                             float* __restrict__ topk_w) {
  const int g = threadIdx.x & (G - 1);                       // lane inside the token's segment
  const int64_t t = int64_t(blockIdx.x) * (kRouteThreads / G) + threadIdx.x / G;
  const bool valid = t < T;

  float vals[V];
  uint64_t keys[V];
  const int e0 = g * V;
  if (VEC4) {
    // E % 4 == 0 and V % 4 == 0: every lane's slice starts 16-byte aligned.
    const float4* src = reinterpret_cast<const float4*>(logits + (valid ? t : 0) * E + e0);
#pragma unroll
    for (int v = 0; v < V; v += 4) {
      float4 q = make_float4(0.f, 0.f, 0.f, 0.f);
      if (valid && e0 + v < E) q = src[v / 4];
      vals[v] = q.x; vals[v + 1] = q.y; vals[v + 2] = q.z; vals[v + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int v = 0; v < V; ++v)
      vals[v] = (valid && e0 + v < E) ? logits[t * E + e0 + v] : 0.f;
  }
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int e = e0 + v;
    keys[v] = (valid && e < E)
                  ? (uint64_t(orderable(vals[v])) << 32) | uint64_t(0xFFFFFFFFu - uint32_t(e))
                  : 0ull;                                   // below every real key
  }

  uint64_t sel[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) {
    if (j < k) {
      uint64_t best = keys[0];
#pragma unroll
      for (int v = 1; v < V; ++v) best = keys[v] > best ? keys[v] : best;
      for (int m = 1; m < G; m <<= 1) {
        const uint64_t o = shfl_xor_u64(best, m);
        best = o > best ? o : best;
      }
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (keys[v] == best) keys[v] = 0ull;                 // keys are unique: retire the winner
      sel[j] = best;
    } else {
      sel[j] = 0ull;
    }
  }

  const float lmax = from_orderable(uint32_t(sel[0] >> 32));
  float p[kMaxTopK];
  float denom = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) {
    if (j < k) {
      p[j] = expf(from_orderable(uint32_t(sel[j] >> 32)) - lmax);
      denom += p[j];                                        // slot order
    }
  }
  if (!renormalize) {
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (valid && e0 + v < E) s += expf(vals[v] - lmax);
    for (int m = 1; m < G; m <<= 1) s += __shfl_xor(s, m);
    denom = s;
  }
  if (valid && g == 0) {
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (j < k) {
        topk_ids[t * k + j] = int32_t(0xFFFFFFFFu - uint32_t(sel[j]));
        topk_w[t * k + j] = p[j] / denom;
      }
    }
  }
}

template <int V>
hipError_t launch_v(const float* logits, int64_t T, int E, int k, int G, int renorm, int32_t* ids,
                    float* w, hipStream_t s) {
  const int64_t per_block = kRouteThreads / G;
  const int64_t blocks = (T + per_block - 1) / per_block;
  if ((E % 4) == 0 && (V % 4) == 0)
    MOE_LAUNCH("route", (route_kernel<V, (V % 4) == 0>), dim3(unsigned(blocks)), dim3(kRouteThreads),
               s, logits, T, E, k, G, renorm, ids, w);
  else
    MOE_LAUNCH("route", (route_kernel<V, false>), dim3(unsigned(blocks)), dim3(kRouteThreads), s,
               logits, T, E, k, G, renorm, ids, w);
  return hipGetLastError();
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
                        float* w, hipStream_t s) {
  int G, V;
  route_shape(E, &G, &V);
  switch (V) {
    case 1: return launch_v<1>(logits, T, E, k, G, renorm, ids, w, s);
    case 2: return launch_v<2>(logits, T, E, k, G, renorm, ids, w, s);
    case 3: return launch_v<3>(logits, T, E, k, G, renorm, ids, w, s);
    case 4: return launch_v<4>(logits, T, E, k, G, renorm, ids, w, s);
    case 5: return launch_v<5>(logits, T, E, k, G, renorm, ids, w, s);
    case 6: return launch_v<6>(logits, T, E, k, G, renorm, ids, w, s);
    case 7: return launch_v<7>(logits, T, E, k, G, renorm, ids, w, s);
    default: return launch_v<8>(logits, T, E, k, G, renorm, ids, w, s);
  }
}

}  // namespace moe
