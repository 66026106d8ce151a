"""Python binding of libmoe.so, the gfx950 MoE-layer hot path.

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  PyTorch supplies device memory and the stream; outputs that are not
passed in are allocated with ``torch.empty`` on the input's device.

The binding fails loudly when the library is missing: there is no CPU or
PyTorch fallback for any call.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

__all__ = [
    "MoEError", "lib", "LIB_PATH", "HEADER_PATH", "abi_version", "exported_symbols",
    "moe_route", "moe_router_topk", "moe_permute", "moe_permute_static", "moe_grouped_ffn", "moe_grouped_ffn_gather", "moe_combine",
    "moe_permute_workspace_bytes", "moe_grouped_ffn_workspace_bytes", "MoELayer",
    "moe_mxfp8_scale_bytes", "moe_quantize_mxfp8", "moe_grouped_ffn_mxfp8_workspace_bytes",
    "moe_grouped_ffn_mxfp8", "moe_grouped_ffn_mxfp8_gather", "MXFP8", "quantize_weights_mxfp8",
    "MoELayerMXFP8", "LayerGraph",
    "profiler_start", "profiler_select", "profiler_stop", "profiler_records", "set_cu_budget",
    "DTYPE_F32", "DTYPE_BF16",
]

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe.so")
HEADER_PATH = os.path.join(os.path.dirname(HERE), "include", "moe.h")

DTYPE_F32, DTYPE_BF16 = 0, 1
_STATUS = {0: "MOE_OK", 1: "MOE_ERR_INVALID_ARGUMENT", 2: "MOE_ERR_UNSUPPORTED",
           3: "MOE_ERR_WORKSPACE_TOO_SMALL", 4: "MOE_ERR_HIP"}


class MoEError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t

_SIGNATURES = {
    "moe_abi_version": (ctypes.c_int, []),
    "moe_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "moe_last_error": (ctypes.c_char_p, []),
    "moe_route": (ctypes.c_int, [_P, _I64, _I32, _I32, _I32, _P, _P, _P]),
    "moe_router_topk": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _P]),
    "moe_permute_workspace_bytes": (_SZ, [_I64, _I32, _I32]),
    "moe_permute": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, _I32, ctypes.c_int, _P, _P, _P, _P, _P,
                                   _P, _SZ, _P]),
    "moe_permute_static": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, _I32, ctypes.c_int, _P, _P, _P, _P, _P,
                                          _P]),
    "moe_grouped_ffn_workspace_bytes": (_SZ, [_I64, _I32, _I32, _I32, ctypes.c_int]),
    "moe_grouped_ffn": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, _I32, _P, _P, _P, ctypes.c_int, _P,
                                       _P, _SZ, _P]),
    "moe_grouped_ffn_gather": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I32, _I32, _I32, _P, _P, _P,
                                              ctypes.c_int, _P, _P, _SZ, _P]),
    "moe_combine": (ctypes.c_int, [_P, _P, _P, _P, _I64, _I32, _I32, ctypes.c_int, _P, _P]),
    "moe_mxfp8_scale_bytes": (_SZ, [_I64, _I32]),
    "moe_quantize_mxfp8": (ctypes.c_int, [_P, _P, _I64, _I64, _I32, _P, _P, _P]),
    "moe_grouped_ffn_mxfp8_workspace_bytes": (_SZ, [_I64, _I32, _I32, _I32]),
    "moe_grouped_ffn_mxfp8": (ctypes.c_int, [_P, _P, _P, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P,
                                             _P, _P, _SZ, _P]),
    "moe_grouped_ffn_mxfp8_gather": (ctypes.c_int, [_P, _P, _P, _P, _I64, _I64, _I32, _I32, _I32, _P, _P, _P, _P,
                                                    _P, _P, _P, _P, _SZ, _P]),
    "moe_profiler_start": (ctypes.c_int, [ctypes.c_int]),
    "moe_profiler_select": (ctypes.c_int, [ctypes.c_char_p]),
    "moe_set_cu_budget": (ctypes.c_int, [_I32]),
    "moe_profiler_stop": (ctypes.c_int, []),
    "moe_profiler_count": (ctypes.c_int, []),
    "moe_profiler_record": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_char_p),
                                           ctypes.POINTER(ctypes.c_float)]),
}


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def exported_symbols():
    """Function names declared in include/moe.h."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^\s*(?:[\w\*]+\s+)+\**(moe_\w+)\s*\(", text, flags=re.M)))


def abi_version() -> int:
    return lib().moe_abi_version()


def _check(status: int):
    if status != 0:
        msg = lib().moe_last_error().decode()
        raise MoEError(status, msg)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return DTYPE_F32
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("all tensors must be on the GPU")
        if t is not None and not t.is_contiguous():
            raise ValueError("all tensors must be contiguous")


# --------------------------------------------------------------------------- the four calls
def moe_route(logits, k, renormalize=1, topk_ids=None, topk_weights=None, stream=None):
    """logits f32 [T, E] -> (topk_ids i32 [T, k], topk_weights f32 [T, k])."""
    T, E = logits.shape
    if logits.dtype != torch.float32:
        raise TypeError("logits must be float32")
    if topk_ids is None:
        topk_ids = torch.empty((T, k), dtype=torch.int32, device=logits.device)
    if topk_weights is None:
        topk_weights = torch.empty((T, k), dtype=torch.float32, device=logits.device)
    _dev(logits, topk_ids, topk_weights)
    _check(lib().moe_route(_ptr(logits), T, E, k, renormalize, _ptr(topk_ids), _ptr(topk_weights),
                           _stream(stream, logits.device)))
    return topk_ids, topk_weights


def moe_router_topk(x, w_router, k, renormalize=1, logits=None, topk_ids=None, topk_weights=None, stream=None):
    """x bf16 [T, H], w_router bf16 [E, H] -> (topk_ids, topk_weights); the router
    GEMM and the gate in one kernel.  Pass logits (f32 [T, E]) to also get them."""
    T, H = x.shape
    E = w_router.shape[0]
    if x.dtype != torch.bfloat16 or w_router.dtype != torch.bfloat16:
        raise TypeError("moe_router_topk takes bf16 x and w_router")
    if topk_ids is None:
        topk_ids = torch.empty((T, k), dtype=torch.int32, device=x.device)
    if topk_weights is None:
        topk_weights = torch.empty((T, k), dtype=torch.float32, device=x.device)
    _dev(x, w_router, logits, topk_ids, topk_weights)
    _check(lib().moe_router_topk(_ptr(x), _ptr(w_router), T, E, k, H, renormalize, _ptr(logits), _ptr(topk_ids),
                                 _ptr(topk_weights), _stream(stream, x.device)))
    return topk_ids, topk_weights


def moe_permute_workspace_bytes(T, E, k) -> int:
    return lib().moe_permute_workspace_bytes(T, E, k)


def moe_permute(topk_ids, x, E, out=None, ws=None, stream=None, gather_rows=True):
    """-> dict(counts, offsets, sorted_token_ids, dest_rows, x_perm).  With
    gather_rows=False (or out["x_perm"] None) only the maps are produced."""
    T, k = topk_ids.shape
    H = x.shape[1]
    dev = x.device
    if out is None:
        out = dict(counts=torch.empty(E, dtype=torch.int32, device=dev),
                   offsets=torch.empty(E + 1, dtype=torch.int32, device=dev),
                   sorted_token_ids=torch.empty(T * k, dtype=torch.int32, device=dev),
                   dest_rows=torch.empty((T, k), dtype=torch.int32, device=dev),
                   x_perm=torch.empty((T * k, H), dtype=x.dtype, device=dev) if gather_rows else None)
    if ws is None:
        ws = torch.empty(max(1, moe_permute_workspace_bytes(T, E, k)), dtype=torch.uint8, device=dev)
    _dev(topk_ids, x, ws, *out.values())
    _check(lib().moe_permute(_ptr(topk_ids), _ptr(x), T, E, k, H, _dt(x), _ptr(out["counts"]),
                             _ptr(out["offsets"]), _ptr(out["sorted_token_ids"]), _ptr(out["dest_rows"]),
                             _ptr(out["x_perm"]), _ptr(ws), ws.numel(), _stream(stream, dev)))
    return out


def moe_permute_static(topk_ids, x, E, out=None, stream=None, gather_rows=True):
    """moe_permute with the library's static device scratch instead of a workspace
    (the call allocates nothing on the device) -> the same dict as moe_permute."""
    T, k = topk_ids.shape
    H = x.shape[1]
    dev = x.device
    if out is None:
        out = dict(counts=torch.empty(E, dtype=torch.int32, device=dev),
                   offsets=torch.empty(E + 1, dtype=torch.int32, device=dev),
                   sorted_token_ids=torch.empty(T * k, dtype=torch.int32, device=dev),
                   dest_rows=torch.empty((T, k), dtype=torch.int32, device=dev),
                   x_perm=torch.empty((T * k, H), dtype=x.dtype, device=dev) if gather_rows else None)
    _dev(topk_ids, x, *out.values())
    _check(lib().moe_permute_static(_ptr(topk_ids), _ptr(x), T, E, k, H, _dt(x), _ptr(out["counts"]),
                                    _ptr(out["offsets"]), _ptr(out["sorted_token_ids"]), _ptr(out["dest_rows"]),
                                    _ptr(out["x_perm"]), _stream(stream, dev)))
    return out


def moe_grouped_ffn_workspace_bytes(R, E, H, F, dtype) -> int:
    return lib().moe_grouped_ffn_workspace_bytes(R, E, H, F, DTYPE_F32 if dtype == torch.float32 else DTYPE_BF16)


def moe_grouped_ffn(x_perm, offsets, w_gate, w_up, w_down, y_perm=None, ws=None, stream=None):
    """x_perm [R, H], offsets i32 [E+1] (device), w_gate/w_up [E, F, H], w_down [E, H, F] -> y_perm [R, H]."""
    R, H = x_perm.shape
    E, F, _ = w_gate.shape
    dev = x_perm.device
    if y_perm is None:
        y_perm = torch.empty((R, H), dtype=x_perm.dtype, device=dev)
    if ws is None:
        ws = torch.empty(max(1, moe_grouped_ffn_workspace_bytes(R, E, H, F, x_perm.dtype)),
                         dtype=torch.uint8, device=dev)
    _dev(x_perm, offsets, w_gate, w_up, w_down, y_perm, ws)
    for w in (w_gate, w_up, w_down):
        if w.dtype != x_perm.dtype:
            raise TypeError("weights and activations must share a dtype")
    _check(lib().moe_grouped_ffn(_ptr(x_perm), _ptr(offsets), R, E, H, F, _ptr(w_gate), _ptr(w_up),
                                 _ptr(w_down), _dt(x_perm), _ptr(y_perm), _ptr(ws), ws.numel(),
                                 _stream(stream, dev)))
    return y_perm


def moe_grouped_ffn_gather(x, sorted_token_ids, offsets, w_gate, w_up, w_down, y_perm=None, ws=None,
                           stream=None):
    """Grouped FFN reading row r of the groups from x[sorted_token_ids[r]] -> y_perm [R, H]."""
    T, H = x.shape
    R = sorted_token_ids.shape[0]
    E, F, _ = w_gate.shape
    dev = x.device
    if y_perm is None:
        y_perm = torch.empty((R, H), dtype=x.dtype, device=dev)
    if ws is None:
        ws = torch.empty(max(1, moe_grouped_ffn_workspace_bytes(R, E, H, F, x.dtype)),
                         dtype=torch.uint8, device=dev)
    _dev(x, sorted_token_ids, offsets, w_gate, w_up, w_down, y_perm, ws)
    for w in (w_gate, w_up, w_down):
        if w.dtype != x.dtype:
            raise TypeError("weights and activations must share a dtype")
    _check(lib().moe_grouped_ffn_gather(_ptr(x), _ptr(sorted_token_ids), _ptr(offsets), T, R, E, H, F,
                                        _ptr(w_gate), _ptr(w_up), _ptr(w_down), _dt(x), _ptr(y_perm),
                                        _ptr(ws), ws.numel(), _stream(stream, dev)))
    return y_perm


def moe_combine(y_perm, dest_rows, topk_weights, y_shared=None, y=None, stream=None):
    """-> y [T, H] = sum_j w[t, j] y_perm[dest_rows[t, j]] (+ y_shared)."""
    T, k = dest_rows.shape
    H = y_perm.shape[1]
    dev = y_perm.device
    if y is None:
        y = torch.empty((T, H), dtype=y_perm.dtype, device=dev)
    _dev(y_perm, dest_rows, topk_weights, y_shared, y)
    _check(lib().moe_combine(_ptr(y_perm), _ptr(dest_rows), _ptr(topk_weights), _ptr(y_shared), T, k, H,
                             _dt(y_perm), _ptr(y), _stream(stream, dev)))
    return y


# --------------------------------------------------------------------------- MXFP8
class MXFP8:
    """An MXFP8 matrix of `rows` rows and K columns: E4M3 codes u8 [rows, K] and
    E8M0 scales u8 in the library's k-step-major layout (include/moe.h)."""

    def __init__(self, codes, scales):
        self.codes, self.scales = codes, scales

    @property
    def shape(self):
        return tuple(self.codes.shape)


def moe_mxfp8_scale_bytes(rows, K) -> int:
    return lib().moe_mxfp8_scale_bytes(rows, K)


def moe_quantize_mxfp8(src, row_map=None, out=None, stream=None):
    """bf16 [rows_src, K] (optionally gathered through row_map i32 [rows_out]) -> MXFP8."""
    if src.dtype != torch.bfloat16:
        raise TypeError("moe_quantize_mxfp8 takes bf16 rows")
    src2 = src.reshape(-1, src.shape[-1])
    rows_src, K = src2.shape
    rows_out = rows_src if row_map is None else row_map.shape[0]
    dev = src.device
    if out is None:
        out = MXFP8(torch.empty((rows_out, K), dtype=torch.uint8, device=dev),
                    torch.empty(max(1, moe_mxfp8_scale_bytes(rows_out, K)), dtype=torch.uint8, device=dev))
    _dev(src2, row_map, out.codes, out.scales)
    _check(lib().moe_quantize_mxfp8(_ptr(src2), _ptr(row_map), rows_out, rows_src, K, _ptr(out.codes),
                                    _ptr(out.scales), _stream(stream, dev)))
    return out


def quantize_weights_mxfp8(w, stream=None):
    """Expert weights bf16 [E, N, K] -> MXFP8 of the [E * N, K] matrix (codes viewed [E, N, K])."""
    E, N, K = w.shape
    q = moe_quantize_mxfp8(w.reshape(E * N, K), stream=stream)
    return MXFP8(q.codes.view(E, N, K), q.scales)


def moe_grouped_ffn_mxfp8_workspace_bytes(R, E, H, F) -> int:
    return lib().moe_grouped_ffn_mxfp8_workspace_bytes(R, E, H, F)


def moe_grouped_ffn_mxfp8(x, offsets, w_gate, w_up, w_down, y_perm=None, ws=None, stream=None):
    """x MXFP8 [R, H] (grouped rows), w_gate/w_up MXFP8 [E, F, H], w_down MXFP8 [E, H, F]
    -> y_perm bf16 [R, H]."""
    R, H = x.codes.shape
    E, F, _ = w_gate.codes.shape
    dev = x.codes.device
    if y_perm is None:
        y_perm = torch.empty((R, H), dtype=torch.bfloat16, device=dev)
    if ws is None:
        ws = torch.empty(max(1, moe_grouped_ffn_mxfp8_workspace_bytes(R, E, H, F)), dtype=torch.uint8, device=dev)
    _dev(x.codes, x.scales, offsets, w_gate.codes, w_gate.scales, w_up.codes, w_up.scales, w_down.codes,
         w_down.scales, y_perm, ws)
    _check(lib().moe_grouped_ffn_mxfp8(_ptr(x.codes), _ptr(x.scales), _ptr(offsets), R, E, H, F,
                                       _ptr(w_gate.codes), _ptr(w_gate.scales), _ptr(w_up.codes),
                                       _ptr(w_up.scales), _ptr(w_down.codes), _ptr(w_down.scales),
                                       _ptr(y_perm), _ptr(ws), ws.numel(), _stream(stream, dev)))
    return y_perm


def moe_grouped_ffn_mxfp8_gather(x, sorted_token_ids, offsets, w_gate, w_up, w_down, y_perm=None, ws=None,
                                 stream=None):
    """x MXFP8 [T, H] token rows, row r of the groups = token sorted_token_ids[r] -> y_perm bf16 [R, H]."""
    T, H = x.codes.shape
    R = sorted_token_ids.shape[0]
    E, F, _ = w_gate.codes.shape
    dev = x.codes.device
    if y_perm is None:
        y_perm = torch.empty((R, H), dtype=torch.bfloat16, device=dev)
    if ws is None:
        ws = torch.empty(max(1, moe_grouped_ffn_mxfp8_workspace_bytes(R, E, H, F)), dtype=torch.uint8, device=dev)
    _dev(x.codes, x.scales, sorted_token_ids, offsets, w_gate.codes, w_gate.scales, w_up.codes, w_up.scales,
         w_down.codes, w_down.scales, y_perm, ws)
    _check(lib().moe_grouped_ffn_mxfp8_gather(_ptr(x.codes), _ptr(x.scales), _ptr(sorted_token_ids),
                                              _ptr(offsets), T, R, E, H, F, _ptr(w_gate.codes),
                                              _ptr(w_gate.scales), _ptr(w_up.codes), _ptr(w_up.scales),
                                              _ptr(w_down.codes), _ptr(w_down.scales), _ptr(y_perm), _ptr(ws),
                                              ws.numel(), _stream(stream, dev)))
    return y_perm


# --------------------------------------------------------------------------- scheduling
def set_cu_budget(n: int = 0):
    """Plan the persistent grids for n compute units (0: the device's count)."""
    _check(lib().moe_set_cu_budget(n))


# --------------------------------------------------------------------------- profiler
def profiler_start(capacity: int = 4096):
    """Bracket every following kernel launch of the library with HIP events."""
    _check(lib().moe_profiler_start(capacity))


def profiler_select(name=None):
    """Record only launches of the kernel `name` (None: every launch)."""
    _check(lib().moe_profiler_select(name.encode() if name else None))


def profiler_stop():
    _check(lib().moe_profiler_stop())


def profiler_records():
    """[(kernel name, milliseconds)] of the recorded launches; call after a sync."""
    out = []
    name = ctypes.c_char_p()
    ms = ctypes.c_float()
    for i in range(lib().moe_profiler_count()):
        _check(lib().moe_profiler_record(i, ctypes.byref(name), ctypes.byref(ms)))
        out.append((name.value.decode(), ms.value))
    return out


# --------------------------------------------------------------------------- whole layer
class MoELayer:
    """Preallocated buffers for one layer shape; ``run`` issues the calls on one stream
    with no allocation and no host synchronization.

    gather=False: route, permute (with x_perm), grouped FFN, combine.
    gather=True:  route, permute (maps only), grouped FFN gathering the token rows,
                  combine -- the same output without the grouped copy of x."""

    def __init__(self, T, H, E, k, F, Fs=0, dtype=torch.bfloat16, device="cuda", gather=False):
        self.T, self.H, self.E, self.k, self.F, self.Fs = T, H, E, k, F, Fs
        self.dtype = dtype
        self.gather = gather
        dev = torch.device(device)
        R = T * k
        i32 = dict(dtype=torch.int32, device=dev)
        self.topk_ids = torch.empty((T, k), **i32)
        self.topk_weights = torch.empty((T, k), dtype=torch.float32, device=dev)
        self.perm = dict(counts=torch.empty(E, **i32), offsets=torch.empty(E + 1, **i32),
                         sorted_token_ids=torch.empty(R, **i32), dest_rows=torch.empty((T, k), **i32),
                         x_perm=None if gather else torch.empty((R, H), dtype=dtype, device=dev))
        self.ws_perm = torch.empty(max(1, moe_permute_workspace_bytes(T, E, k)), dtype=torch.uint8, device=dev)
        self.y_perm = torch.empty((R, H), dtype=dtype, device=dev)
        self.ws_ffn = torch.empty(max(1, moe_grouped_ffn_workspace_bytes(R, E, H, F, dtype)),
                                  dtype=torch.uint8, device=dev)
        self.y = torch.empty((T, H), dtype=dtype, device=dev)
        if Fs:
            self.shared_offsets = torch.tensor([0, T], **i32)
            self.y_shared = torch.empty((T, H), dtype=dtype, device=dev)
            self.ws_shared = torch.empty(max(1, moe_grouped_ffn_workspace_bytes(T, 1, H, Fs, dtype)),
                                         dtype=torch.uint8, device=dev)
        else:
            self.y_shared = None

    def run(self, x, logits, w_gate, w_up, w_down, ws_gate=None, ws_up=None, ws_down=None,
            renormalize=1, stream=None):
        moe_route(logits, self.k, renormalize, self.topk_ids, self.topk_weights, stream=stream)
        moe_permute(self.topk_ids, x, self.E, out=self.perm, ws=self.ws_perm, stream=stream)
        if self.gather:
            moe_grouped_ffn_gather(x, self.perm["sorted_token_ids"], self.perm["offsets"], w_gate, w_up,
                                   w_down, y_perm=self.y_perm, ws=self.ws_ffn, stream=stream)
        else:
            moe_grouped_ffn(self.perm["x_perm"], self.perm["offsets"], w_gate, w_up, w_down,
                            y_perm=self.y_perm, ws=self.ws_ffn, stream=stream)
        if self.Fs:
            moe_grouped_ffn(x, self.shared_offsets, ws_gate, ws_up, ws_down, y_perm=self.y_shared,
                            ws=self.ws_shared, stream=stream)
        moe_combine(self.y_perm, self.perm["dest_rows"], self.topk_weights, self.y_shared, y=self.y,
                    stream=stream)
        return self.y


class LayerGraph:
    """One layer step captured as a HIP graph: ``replay()`` launches the layer's kernels
    (route, permute, grouped FFN, combine) as one graph on the current stream, which
    takes the per-kernel launch cost off small expert batches.

    The graph holds the device addresses of the tensors given at capture and of the
    layer's own buffers: to run it on new data, copy the data into those tensors in
    place.  The library's calls neither allocate nor synchronize, and nothing in a
    layer step clears memory with a memset (the tile counters are zeroed by a kernel),
    so the whole step captures.  A first eager run on a side stream (of default
    priority) does the library's one-time set-up outside the capture."""

    def __init__(self, layer, *args, **kwargs):
        if "stream" in kwargs:
            raise ValueError("LayerGraph captures on the current stream; pass no stream")
        self.layer = layer
        # the graph reads these tensors by address: keep them alive as long as it is
        self._captured = (args, kwargs)
        self.graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            layer.run(*args, **kwargs)
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(self.graph):
            layer.run(*args, **kwargs)

    def replay(self):
        """Run the captured step on the current stream; returns the layer's y."""
        self.graph.replay()
        return self.layer.y


class MoELayerMXFP8:
    """The layer with MXFP8 expert GEMMs (bf16 x and y); with Fs > 0 an always-active
    shared expert (also MXFP8) over x, added with weight 1.  Weights are quantized once
    with quantize_weights_mxfp8.  ``run`` allocates nothing and does not synchronize.

    gather=True (default): route, permute (maps only), quantize the T token rows once,
    grouped FFN gathering the token codes, combine.
    gather=False: quantize x into grouped order (R = T*k rows) and run the grouped FFN
    on those rows -- bit for bit the same output."""

    def __init__(self, T, H, E, k, F, Fs=0, device="cuda", gather=True):
        self.T, self.H, self.E, self.k, self.F, self.Fs = T, H, E, k, F, Fs
        self.gather = gather
        dev = torch.device(device)
        R = T * k
        i32 = dict(dtype=torch.int32, device=dev)
        u8 = dict(dtype=torch.uint8, device=dev)
        self.topk_ids = torch.empty((T, k), **i32)
        self.topk_weights = torch.empty((T, k), dtype=torch.float32, device=dev)
        self.perm = dict(counts=torch.empty(E, **i32), offsets=torch.empty(E + 1, **i32),
                         sorted_token_ids=torch.empty(R, **i32), dest_rows=torch.empty((T, k), **i32),
                         x_perm=None)
        self.ws_perm = torch.empty(max(1, moe_permute_workspace_bytes(T, E, k)), **u8)
        rows = T if gather else R
        self.xq = MXFP8(torch.empty((rows, H), **u8), torch.empty(max(1, moe_mxfp8_scale_bytes(rows, H)), **u8))
        self.y_perm = torch.empty((R, H), dtype=torch.bfloat16, device=dev)
        self.ws_ffn = torch.empty(max(1, moe_grouped_ffn_mxfp8_workspace_bytes(R, E, H, F)), **u8)
        self.y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        if Fs:
            self.shared_offsets = torch.tensor([0, T], **i32)
            self.xq_tokens = self.xq if gather else MXFP8(
                torch.empty((T, H), **u8), torch.empty(max(1, moe_mxfp8_scale_bytes(T, H)), **u8))
            self.y_shared = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
            self.ws_shared = torch.empty(max(1, moe_grouped_ffn_mxfp8_workspace_bytes(T, 1, H, Fs)), **u8)
        else:
            self.y_shared = None

    def run(self, x, logits, wq_gate, wq_up, wq_down, wqs_gate=None, wqs_up=None, wqs_down=None,
            renormalize=1, stream=None):
        moe_route(logits, self.k, renormalize, self.topk_ids, self.topk_weights, stream=stream)
        moe_permute(self.topk_ids, x, self.E, out=self.perm, ws=self.ws_perm, stream=stream)
        if self.gather:
            moe_quantize_mxfp8(x, out=self.xq, stream=stream)
            moe_grouped_ffn_mxfp8_gather(self.xq, self.perm["sorted_token_ids"], self.perm["offsets"], wq_gate,
                                         wq_up, wq_down, y_perm=self.y_perm, ws=self.ws_ffn, stream=stream)
        else:
            moe_quantize_mxfp8(x, row_map=self.perm["sorted_token_ids"], out=self.xq, stream=stream)
            moe_grouped_ffn_mxfp8(self.xq, self.perm["offsets"], wq_gate, wq_up, wq_down, y_perm=self.y_perm,
                                  ws=self.ws_ffn, stream=stream)
        if self.Fs:
            if not self.gather:
                moe_quantize_mxfp8(x, out=self.xq_tokens, stream=stream)
            moe_grouped_ffn_mxfp8(self.xq_tokens, self.shared_offsets, wqs_gate, wqs_up, wqs_down,
                                  y_perm=self.y_shared, ws=self.ws_shared, stream=stream)
        moe_combine(self.y_perm, self.perm["dest_rows"], self.topk_weights, self.y_shared, y=self.y,
                    stream=stream)
        return self.y
