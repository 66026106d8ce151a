"""The C-ABI library on a host without a GPU: it loads, exports every function
include/moe.h declares, and rejects bad arguments on the host before any launch.
No call here reaches a kernel: each one fails validation or is a T = 0 no-op."""
import ctypes

import pytest

import paper_2606_21712_amd as moe

INVALID, UNSUPPORTED, WS_SMALL = 1, 2, 3
P = 0x10000          # a 16-byte aligned address that is never dereferenced
S = None             # default stream


@pytest.fixture(scope="module")
def L():
    return moe.lib()


def test_exports_every_declared_symbol(L):
    names = moe.exported_symbols()
    assert {"moe_route", "moe_permute", "moe_grouped_ffn", "moe_combine", "moe_abi_version",
            "moe_status_string", "moe_last_error", "moe_permute_workspace_bytes",
            "moe_grouped_ffn_workspace_bytes"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings(L):
    assert moe.abi_version() == 1
    for s, name in [(0, b"MOE_OK"), (1, b"MOE_ERR_INVALID_ARGUMENT"), (2, b"MOE_ERR_UNSUPPORTED"),
                    (3, b"MOE_ERR_WORKSPACE_TOO_SMALL"), (4, b"MOE_ERR_HIP")]:
        assert L.moe_status_string(s) == name
    assert L.moe_status_string(99) is not None


def route(L, logits=P, T=16, E=8, k=2, renorm=1, ids=P, w=P):
    return L.moe_route(logits, T, E, k, renorm, ids, w, S)


def test_route_validation(L):
    assert route(L, k=0) == INVALID
    assert route(L, k=9) == INVALID
    assert route(L, E=0) == INVALID
    assert route(L, E=300, k=2) == UNSUPPORTED
    assert route(L, E=64, k=17) == UNSUPPORTED
    assert route(L, T=-1) == INVALID
    assert route(L, T=2**31, k=2) == INVALID                      # T*k > INT32_MAX
    assert route(L, renorm=2) == INVALID
    assert route(L, logits=None) == INVALID
    assert b"logits" in L.moe_last_error()
    assert route(L, ids=P + 8) == INVALID
    assert b"aligned" in L.moe_last_error()
    assert route(L, T=0, logits=None, ids=None, w=None) == 0       # no-op


def permute(L, ids=P, x=P, T=16, E=8, k=2, H=64, dt=1, cnt=P, off=P, st=P, dest=P, xp=P, ws=P,
            ws_bytes=1 << 20):
    return L.moe_permute(ids, x, T, E, k, H, dt, cnt, off, st, dest, xp, ws, ws_bytes, S)


def test_permute_validation(L):
    assert permute(L, H=96) == INVALID
    assert permute(L, H=0) == INVALID
    assert permute(L, dt=7) == UNSUPPORTED
    assert permute(L, k=3, E=2) == INVALID
    assert permute(L, x=None) == INVALID
    assert permute(L, ws_bytes=0) == WS_SMALL
    assert permute(L, T=0, ids=None, x=None, cnt=None, off=None, st=None, dest=None, xp=None,
                   ws=None, ws_bytes=0) == 0


def test_permute_workspace_size(L):
    # one int32 count per (unit of 1024 assignments, expert), units padded to 4
    assert L.moe_permute_workspace_bytes(0, 8, 2) == 0
    assert L.moe_permute_workspace_bytes(4096, 8, 2) == 8 * 8 * 4
    assert L.moe_permute_workspace_bytes(131072, 64, 4) == 512 * 64 * 4
    assert L.moe_permute_workspace_bytes(1, 3, 1) == 256          # 4 units x 3 experts, 256-aligned


def ffn(L, xp=P, off=P, R=100, E=8, H=128, F=256, wg=P, wu=P, wd=P, dt=1, yp=P, ws=P, ws_bytes=1 << 30):
    return L.moe_grouped_ffn(xp, off, R, E, H, F, wg, wu, wd, dt, yp, ws, ws_bytes, S)


def test_ffn_validation(L):
    assert ffn(L, H=100) == INVALID
    assert ffn(L, F=32) == INVALID
    assert ffn(L, E=0) == INVALID
    assert ffn(L, E=257) == UNSUPPORTED
    assert ffn(L, R=-5) == INVALID
    assert ffn(L, R=2**31) == INVALID
    assert ffn(L, dt=3) == UNSUPPORTED
    assert ffn(L, H=65536, F=32768) == UNSUPPORTED                 # expert matrix > 2 GiB
    assert ffn(L, wd=None) == INVALID
    assert b"w_down" in L.moe_last_error()
    need = L.moe_grouped_ffn_workspace_bytes(100, 8, 128, 256, 1)
    assert need >= 100 * 256 * 2
    assert ffn(L, ws_bytes=need - 1) == WS_SMALL
    assert ffn(L, R=0, xp=None, off=None, wg=None, wu=None, wd=None, yp=None, ws=None, ws_bytes=0) == 0
    # fp32 h is twice as large
    assert L.moe_grouped_ffn_workspace_bytes(100, 8, 128, 256, 0) > need
    # the down projection's tail split: one 320 x 256 fp32 slot per possible output
    # tile (E * 255 + R rows in 256-row tiles, times H / 256), at most 256 slots
    R, H, F = 2048, 256, 4096
    slot = 320 * 256 * 4                    # a tile of up to 320 rows x 256 columns, fp32
    tiles = (R + 8 * 255) // 256 * (H // 256)
    need = L.moe_grouped_ffn_workspace_bytes(R, 8, H, F, 1)
    assert R * F * 2 + tiles * slot <= need < R * F * 2 + (tiles + 1) * slot
    big = L.moe_grouped_ffn_workspace_bytes(1 << 20, 8, 4096, F, 1)
    assert (1 << 20) * F * 2 + 256 * slot <= big < (1 << 20) * F * 2 + 257 * slot
    # a k loop too short to cut in two pieces of 8 steps (F / 64 < 16): no slots
    assert L.moe_grouped_ffn_workspace_bytes(R, 8, H, 1024, 1) >= R * 1024 * 2 + tiles * slot
    assert L.moe_grouped_ffn_workspace_bytes(R, 8, H, 960, 1) < R * 960 * 2 + slot
    # fp32 has no tail split
    assert L.moe_grouped_ffn_workspace_bytes(R, 8, H, F, 0) < R * F * 4 + slot


def ffn_gather(L, x=P, st=P, off=P, T=50, R=100, E=8, H=128, F=256, wg=P, wu=P, wd=P, dt=1, yp=P, ws=P,
               ws_bytes=1 << 30):
    return L.moe_grouped_ffn_gather(x, st, off, T, R, E, H, F, wg, wu, wd, dt, yp, ws, ws_bytes, S)


def test_ffn_gather_validation(L):
    assert ffn_gather(L, st=None) == INVALID
    assert b"sorted_token_ids" in L.moe_last_error()
    assert ffn_gather(L, x=None) == INVALID
    assert b"x is NULL" in L.moe_last_error()
    assert ffn_gather(L, T=0) == INVALID
    assert ffn_gather(L, T=-1) == INVALID
    # x of 2 GiB or more is read with 64-bit row addresses: no size error (the short
    # workspace stops this call before any launch)
    assert ffn_gather(L, T=2**20, H=1024, ws_bytes=10) == WS_SMALL
    assert ffn_gather(L, ws_bytes=10) == WS_SMALL
    assert ffn_gather(L, R=0, T=0, x=None, st=None, off=None, wg=None, wu=None, wd=None, yp=None,
                      ws=None, ws_bytes=0) == 0


def quant(L, src=P, rm=None, rows_out=64, rows_src=64, K=256, codes=P, scales=P):
    return L.moe_quantize_mxfp8(src, rm, rows_out, rows_src, K, codes, scales, S)


def test_quantize_mxfp8_validation(L):
    assert quant(L, K=64) == INVALID                              # K % 128
    assert quant(L, K=0) == INVALID
    assert quant(L, rows_out=-1) == INVALID
    assert quant(L, rows_src=-1) == INVALID
    assert quant(L, rows_out=65) == INVALID                       # more rows than the source, no map
    assert b"row_map" in L.moe_last_error()
    assert quant(L, rows_out=65, rm=P, src=None) == INVALID       # with a map it is allowed; src checked
    assert quant(L, rows_out=5, rows_src=0, rm=P) == INVALID
    assert quant(L, scales=P + 4) == INVALID
    assert quant(L, codes=None) == INVALID
    assert quant(L, rows_out=0, src=None, codes=None, scales=None) == 0
    assert L.moe_mxfp8_scale_bytes(64, 256) == 64 * 256 // 32
    assert L.moe_mxfp8_scale_bytes(0, 256) == 0


def ffn8(L, x=P, xs=P, off=P, R=100, E=8, H=128, F=256, wg=P, wgs=P, wu=P, wus=P, wd=P, wds=P, yp=P, ws=P,
         ws_bytes=1 << 30):
    return L.moe_grouped_ffn_mxfp8(x, xs, off, R, E, H, F, wg, wgs, wu, wus, wd, wds, yp, ws, ws_bytes, S)


def test_ffn_mxfp8_validation(L):
    assert ffn8(L, H=192) == INVALID                              # H % 128
    assert ffn8(L, F=64) == INVALID
    assert ffn8(L, E=0) == INVALID
    assert ffn8(L, E=257) == UNSUPPORTED
    assert ffn8(L, R=-1) == INVALID
    assert ffn8(L, R=2**31) == INVALID
    assert ffn8(L, H=65536, F=65536) == UNSUPPORTED               # one expert matrix of 4 GiB
    assert ffn8(L, E=256, H=16384, F=16384) == UNSUPPORTED        # weight scales of 2 GiB
    assert ffn8(L, R=2**30, H=128, F=1024) == UNSUPPORTED         # h scales of 32 GiB / 32
    assert ffn8(L, wds=None) == INVALID
    assert b"wd_scales" in L.moe_last_error()
    assert ffn8(L, xs=P + 8) == INVALID
    need = L.moe_grouped_ffn_mxfp8_workspace_bytes(100, 8, 128, 256)
    assert need >= 100 * 256 + 100 * 256 // 32                   # h codes + scales
    assert need < 100 * 256 * 2                                   # k loop of 2 steps: no tail split
    assert ffn8(L, ws_bytes=need - 1) == WS_SMALL
    # k loop of 16 steps of 128: tail-split slots of 320 x 256 fp32 per possible output tile
    tiles = (100 + 8 * 255) // 256
    assert L.moe_grouped_ffn_mxfp8_workspace_bytes(100, 8, 256, 2048) >= 100 * 2048 + tiles * 320 * 256 * 4
    assert ffn8(L, R=0, x=None, xs=None, off=None, wg=None, wgs=None, wu=None, wus=None, wd=None, wds=None,
                yp=None, ws=None, ws_bytes=0) == 0


def ffn8g(L, x=P, xs=P, st=P, off=P, T=50, R=100, E=8, H=128, F=256, wg=P, wgs=P, wu=P, wus=P, wd=P, wds=P, yp=P,
          ws=P, ws_bytes=1 << 30):
    return L.moe_grouped_ffn_mxfp8_gather(x, xs, st, off, T, R, E, H, F, wg, wgs, wu, wus, wd, wds, yp, ws,
                                          ws_bytes, S)


def test_ffn_mxfp8_gather_validation(L):
    assert ffn8g(L, st=None) == INVALID
    assert b"sorted_token_ids" in L.moe_last_error()
    assert ffn8g(L, T=0) == INVALID
    assert ffn8g(L, T=-1) == INVALID
    assert ffn8g(L, H=192) == INVALID
    assert b"moe_grouped_ffn_mxfp8_gather" in L.moe_last_error()
    assert ffn8g(L, T=2**24, H=128) == UNSUPPORTED                 # token codes of 2 GiB
    assert ffn8g(L, ws_bytes=10) == WS_SMALL
    assert ffn8g(L, R=0, T=0, x=None, xs=None, st=None, off=None, wg=None, wgs=None, wu=None, wus=None, wd=None,
                 wds=None, yp=None, ws=None, ws_bytes=0) == 0


def router(L, x=P, w=P, T=100, E=8, k=2, H=128, renorm=1, logits=None, ids=P, wts=P):
    return L.moe_router_topk(x, w, T, E, k, H, renorm, logits, ids, wts, S)


def test_router_topk_validation(L):
    assert router(L, E=65) == UNSUPPORTED                          # fused router holds E <= 64
    assert router(L, E=300) == UNSUPPORTED
    assert router(L, k=9) == INVALID
    assert router(L, H=96) == INVALID
    assert router(L, E=64, k=2, H=1 << 24) == UNSUPPORTED             # 2 GiB router matrix
    assert router(L, renorm=3) == INVALID
    assert router(L, T=-1) == INVALID
    assert router(L, w=None) == INVALID
    assert b"w_router" in L.moe_last_error()
    assert router(L, logits=P + 4) == INVALID                      # optional, but aligned when given
    assert router(L, T=0, x=None, w=None, ids=None, wts=None) == 0


def test_permute_maps_only_needs_no_rows(L):
    # x_perm NULL: x may be NULL too; validation passes up to the launch.  T = 0 keeps it a no-op.
    assert permute(L, T=0, x=None, xp=None, ids=None, cnt=None, off=None, st=None, dest=None, ws=None,
                   ws_bytes=0) == 0
    assert permute(L, x=None, xp=P) == INVALID


def combine(L, yp=P, dest=P, w=P, ys=None, T=16, k=2, H=64, dt=1, y=P):
    return L.moe_combine(yp, dest, w, ys, T, k, H, dt, y, S)


def test_combine_validation(L):
    assert combine(L, k=0) == INVALID
    assert combine(L, k=17) == UNSUPPORTED
    assert combine(L, H=10) == INVALID
    assert combine(L, y=None) == INVALID
    assert combine(L, ys=P + 4) == INVALID
    assert combine(L, T=0, yp=None, dest=None, w=None, y=None) == 0


def test_cu_budget_validation(L):
    assert L.moe_set_cu_budget(-1) == INVALID
    assert b"moe_set_cu_budget" in L.moe_last_error()
    assert L.moe_set_cu_budget(7) == 0
    assert L.moe_set_cu_budget(0) == 0


def test_binding_rejects_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        moe.moe_route(torch.zeros(4, 8), 2)


def test_permute_static_validation(L):
    def call(T=16, E=8, k=2, H=64, ids=P, xp=P, ws_ok=True):
        return L.moe_permute_static(ids, P, T, E, k, H, 1, P, P, P, P, xp, S)
    assert call(H=96) == INVALID
    assert call(k=3, E=2) == INVALID
    assert call(ids=None) == INVALID
    # the static array holds 4 MiB of per-unit counts: 2^22 assignments over 256 experts fit,
    # 1024 more do not
    assert L.moe_permute_workspace_bytes((1 << 22) // 8, 256, 8) == 4 << 20
    assert call(T=(1 << 22) // 8 + 128, E=256, k=8) == UNSUPPORTED
    assert b"static" in L.moe_last_error()
    assert call(T=0, ids=None, xp=None) == 0


def test_layer_graph_rejects_a_stream():
    """LayerGraph captures on the current stream; an explicit stream is refused
    before anything runs."""
    import paper_2606_21712_amd as moe
    with pytest.raises(ValueError):
        moe.LayerGraph(object(), stream=object())
