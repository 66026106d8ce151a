// Host-side fuzz of the C ABI's argument validation (moe_validate.cpp), built
// with the address and undefined-behaviour sanitizers by tests/test_validate_fuzz.py.
// Every entry point's checks run on edge and random sizes (negative, zero,
// just past each limit, near the int32/int64 ranges) with null, aligned and
// misaligned pointers; the sanitizers catch overflow, and the driver checks
// that accepted sizes keep the workspace layout consistent.
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "moe_validate.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next() {                       // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

const int64_t kI64[] = {-1, 0, 1, 2, 63, 64, 65, 127, 128, 1000, 4096, 16384, 65536, 131072,
                        (1ll << 31) - 1, 1ll << 31, (1ll << 31) + 1, 1ll << 40, INT64_MAX / 2};
const int32_t kI32[] = {-1, 0, 1, 2, 3, 7, 8, 16, 17, 63, 64, 65, 127, 128, 192, 256, 257, 4096,
                        7168, 14336, 1 << 20, (1 << 20) + 64, INT32_MAX};

int64_t pick64() { return (next() & 1) ? kI64[next() % (sizeof kI64 / sizeof kI64[0])] : int64_t(next() % 200000); }
int32_t pick32() { return (next() & 1) ? kI32[next() % (sizeof kI32 / sizeof kI32[0])] : int32_t(next() % 9000); }

alignas(16) unsigned char g_buf[64];
const void* pickp() {
  switch (next() % 4) {
    case 0: return nullptr;
    case 1: return g_buf + 4;           // misaligned
    default: return g_buf;
  }
}

int g_fail = 0;
void expect(bool ok, const char* what, long long a, long long b) {
  if (!ok) {
    std::fprintf(stderr, "FAIL %s (%lld, %lld)\n", what, a, b);
    ++g_fail;
  }
}

}  // namespace

int main() {
  using namespace moe;
  for (int i = 0; i < 200000; ++i) {
    const int64_t T = pick64(), R = pick64();
    const int32_t E = pick32(), k = pick32(), H = pick32(), F = pick32(), K = pick32();
    const size_t ws = (next() & 1) ? size_t(next() % (1ull << 34)) : ~size_t(0);
    const int dt = int(next() % 3);
    const int32_t* ip = static_cast<const int32_t*>(pickp());
    Check c;
    c = validate_route(static_cast<const float*>(pickp()), T, E, k, int32_t(next() % 3), ip,
                       static_cast<const float*>(pickp()));
    c = validate_router_topk(pickp(), pickp(), T, E, k, H, int32_t(next() % 3), nullptr, ip,
                             static_cast<const float*>(pickp()));
    c = validate_permute(ip, pickp(), T, E, k, H, dt, ip, ip, ip, ip, pickp(), pickp(), ws);
    c = validate_permute_static(ip, pickp(), T, E, k, H, dt, ip, ip, ip, ip, pickp());
    c = validate_ffn(pickp(), ip, R, E, H, F, pickp(), pickp(), pickp(), dt, pickp(), pickp(), ws);
    const bool ffn_ok = c.ok();
    c = validate_ffn_gather(pickp(), ip, T, ip, R, E, H, F, pickp(), pickp(), pickp(), dt, pickp(), pickp(), ws);
    c = validate_quantize_mxfp8(pickp(), (next() & 1) ? ip : nullptr, R, T, K, pickp(), pickp());
    c = validate_ffn_mxfp8(pickp(), pickp(), ip, R, E, H, F, pickp(), pickp(), pickp(), pickp(), pickp(), pickp(),
                           pickp(), pickp(), ws);
    const bool ffn8_ok = c.ok();
    c = validate_ffn_mxfp8_gather(pickp(), pickp(), ip, T, ip, R, E, H, F, pickp(), pickp(), pickp(), pickp(),
                                  pickp(), pickp(), pickp(), pickp(), ws);
    c = validate_combine(pickp(), ip, static_cast<const float*>(pickp()), pickp(), T, k, H, dt, pickp());
    (void)c;
    // accepted sizes: the workspace regions are ordered and fit the size reported
    if (ffn_ok && R > 0) {
      const moe_dtype d = moe_dtype(dt);
      const size_t need = ffn_workspace_bytes(R, E, H, F, d);
      expect(ffn_h_offset(E) <= ffn_partial_offset(R, E, F, d), "ffn h before partials", R, E);
      expect(ffn_partial_offset(R, E, F, d) <= need, "ffn partials inside", R, F);
      expect(ws >= need, "ffn accepted a short workspace", (long long)ws, (long long)need);
    }
    if (ffn8_ok && R > 0) {
      const size_t need = ffn_mxfp8_workspace_bytes(R, E, H, F);
      expect(ffn_mxfp8_h_scales_offset(R, E, F) <= ffn_mxfp8_partial_offset(R, E, F), "mxfp8 scales first", R, F);
      expect(ffn_mxfp8_partial_offset(R, E, F) <= need, "mxfp8 partials inside", R, F);
      expect(ws >= need, "mxfp8 accepted a short workspace", (long long)ws, (long long)need);
    }
    if (T >= 0 && T < (1ll << 31) && E >= 1 && E <= 256 && k >= 1 && k <= 16 && T * k < INT32_MAX) {
      const size_t pw = permute_workspace_bytes(T, E, k);
      expect(pw % 256 == 0, "permute workspace multiple of 256", T, E);
    }
  }
  if (g_fail) {
    std::fprintf(stderr, "%d failures\n", g_fail);
    return 1;
  }
  std::printf("validate_fuzz: 200000 rounds, no failures\n");
  return 0;
}
