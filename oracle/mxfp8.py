"""MXFP8 quantization and the MoE layer with MXFP8 expert GEMMs, in fp64.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke entry point and the
benchmark's CPU-baseline leg may import this module; the product path never
imports, calls or links it, and it shares no code with that path (numpy only).

Why this exists.  The paper's MoE GEMMs are third-party FP8 kernels (Section 5,
the coroutine-overhead estimate that prices DeepSeek-R1's prefill with FP8 MoE
GEMMs, and Section 5.6, Implementation Details).  The paper does not fix an FP8
recipe.  This oracle takes the OCP Microscaling (MX) format MXFP8, which is
what the gfx950 matrix cores consume natively:

  element : FP8 E4M3 -- 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits;
            no infinities; S.1111.111 is NaN; largest finite value 448
            (S.1111.110); exponent field 0 holds subnormals m/8 * 2^-6.
  scale   : E8M0 -- an 8-bit biased exponent, value 2^(s - 127), one per block
            of 32 consecutive elements along the contraction (k) dimension.
  quantize a block V_0..V_31 (the MX conversion with a shared exponent):
            shared_exp = floor(log2(max_i |V_i|)) - 8 (8 = E4M3's largest
            normal exponent), clamped to [-127, 127]; an all-zero block takes
            -127.  Each element is V_i / 2^shared_exp rounded to the nearest
            E4M3 value, ties to an even mantissa, and clamped to +-448 (a
            scaled block maximum lies in [256, 512), so only values above 448
            saturate).  The sign bit is the input's sign bit (-0 -> 0x80).

The layer (`layer_mxfp8`) is the bf16 layer of moe_oracle with the two expert
GEMMs on MXFP8 operands: x, W_gate and W_up quantized along H; h =
silu(g) * u computed exactly from the dequantized operands and quantized along
F; W_down quantized along F; routing, grouping and combine as in moe_oracle;
an always-active shared expert, when given, is the same FFN on every token
(`dense_mxfp8`), added with weight 1.
Every product and sum is fp64 on the dequantized values; the only roundings are
the three quantizations.
"""
from __future__ import annotations

import numpy as np

from . import moe_oracle as _bf

BLOCK = 32                 # elements per E8M0 scale
E4M3_MAX = 448.0
E4M3_EMAX = 8              # exponent of the largest normal E4M3 value (2^8 * 1.75 = 448)
E4M3_EMIN = -6             # exponent of the smallest normal value
SCALE_BIAS = 127


# --------------------------------------------------------------------------- E4M3
def e4m3_decode(codes) -> np.ndarray:
    """E4M3 code bytes -> float64 values (NaN for S.1111.111)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** E4M3_EMIN, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & ((c & 7) == 7), np.nan, mag)
    return sign * mag


def e4m3_encode(v) -> np.ndarray:
    """float64 values (finite) -> E4M3 codes: nearest value, ties to an even
    mantissa, magnitudes above 448 clamped to 448, sign bit kept."""
    v = np.asarray(v, dtype=np.float64)
    if not np.isfinite(v).all():
        raise ValueError("e4m3_encode: non-finite input")
    neg = np.signbit(v)
    a = np.abs(v)
    # spacing of E4M3 values around a: 2^(e - 3) in binade e >= -6, 2^-9 below
    _, ex = np.frexp(a)                      # a = f * 2^ex, f in [0.5, 1)
    e = np.where(a > 0, ex - 1, E4M3_EMIN)
    e = np.maximum(e, E4M3_EMIN)
    quantum = np.exp2(e - 3.0)
    r = np.rint(a / quantum)                 # exact division; rint rounds half to even
    val = np.minimum(r * quantum, E4M3_MAX)
    # bits of val: exponent field 0 for val < 2^-6 (mantissa = val / 2^-9), else
    # (floor(log2 val) + 7, mantissa)
    _, vex = np.frexp(val)
    ve = np.where(val > 0, vex - 1, E4M3_EMIN - 1)
    sub = val < 2.0 ** E4M3_EMIN
    mant_sub = np.rint(val / 2.0 ** -9)
    mant_norm = np.rint(val / np.exp2(ve) * 8.0 - 8.0)
    code = np.where(sub, mant_sub, (ve + 7) * 8 + mant_norm).astype(np.int64)
    return (code | np.where(neg, 0x80, 0)).astype(np.uint8)


# --------------------------------------------------------------------------- MX blocks
def shared_exponent(block_amax) -> np.ndarray:
    """floor(log2(amax)) - 8, clamped to [-127, 127]; -127 for an all-zero block."""
    amax = np.asarray(block_amax, dtype=np.float64)
    _, ex = np.frexp(amax)
    e = np.where(amax > 0, ex - 1 - E4M3_EMAX, -SCALE_BIAS)
    return np.clip(e, -SCALE_BIAS, SCALE_BIAS).astype(np.int64)


def quantize_mxfp8(a):
    """Quantize along the last axis in blocks of 32.

    a : [..., K] values (bf16 bit patterns as uint16, or float), K % 32 == 0.
    Returns (codes uint8 [..., K], scales uint8 [..., K / 32]) with
    scales = shared_exp + 127 (E8M0)."""
    x = _bf._f64(a)
    K = x.shape[-1]
    if K % BLOCK:
        raise ValueError("quantize_mxfp8: K must be a multiple of 32")
    blocks = x.reshape(x.shape[:-1] + (K // BLOCK, BLOCK))
    se = shared_exponent(np.abs(blocks).max(axis=-1))
    scaled = blocks / np.exp2(se.astype(np.float64))[..., None]
    codes = e4m3_encode(scaled).reshape(x.shape)
    return codes, (se + SCALE_BIAS).astype(np.uint8)


def dequantize_mxfp8(codes, scales) -> np.ndarray:
    """codes [..., K], scales [..., K / 32] -> float64 values."""
    vals = e4m3_decode(codes)
    K = vals.shape[-1]
    s = np.exp2(np.asarray(scales, dtype=np.float64) - SCALE_BIAS)
    return (vals.reshape(vals.shape[:-1] + (K // BLOCK, BLOCK)) * s[..., None]).reshape(vals.shape)


def roundtrip(a) -> np.ndarray:
    """The MXFP8 image of a: dequantize(quantize(a))."""
    return dequantize_mxfp8(*quantize_mxfp8(a))


# --------------------------------------------------------------------------- layer
def quantize_weights(w):
    """Expert matrices [E, N, K] (K-contiguous rows): MXFP8 along K."""
    return quantize_mxfp8(w)


def dense_mxfp8(x, w_gate, w_up, w_down):
    """One expert's MXFP8 SwiGLU FFN on every row of x (the always-active shared
    expert): Q(h) . Q(W_down)^T with h = silu(Q(x) . Q(W_gate)^T) * (Q(x) . Q(W_up)^T)."""
    xd = roundtrip(x)
    g = xd @ roundtrip(w_gate).T
    u = xd @ roundtrip(w_up).T
    h = _bf._silu(g) * u
    return roundtrip(h) @ roundtrip(w_down).T, h


def layer_mxfp8(x, logits, k, w_gate, w_up, w_down, renormalize=1, ws_gate=None, ws_up=None, ws_down=None):
    """The MoE layer with MXFP8 expert GEMMs; returns every intermediate.

    x [T, H] and the expert weights are bf16 bit patterns (or floats).  Route,
    permute and combine are moe_oracle's.  For the rows r of expert e:
      g = Q(x_perm[r]) . Q(W_gate[e])^T,  u = Q(x_perm[r]) . Q(W_up[e])^T,
      h = silu(g) * u (exact),  y_perm[r] = Q(h) . Q(W_down[e])^T,
    where Q is the MXFP8 image along the contraction dimension."""
    E = np.asarray(w_gate).shape[0]
    ids, w = _bf.route(logits, k, renormalize)
    counts, offsets, dest, sorted_tok, _ = _bf.permute(ids, x, E)
    xq_codes, xq_scales = quantize_mxfp8(x)
    xd = dequantize_mxfp8(xq_codes, xq_scales)
    gd = roundtrip(w_gate)
    ud = roundtrip(w_up)
    dd = roundtrip(w_down)
    R = sorted_tok.size
    H = xd.shape[1]
    F = gd.shape[1]
    h = np.zeros((R, F))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        xr = xd[sorted_tok[lo:hi]]
        h[lo:hi] = _bf._silu(xr @ gd[e].T) * (xr @ ud[e].T)
    h_codes, h_scales = quantize_mxfp8(h)
    hd = dequantize_mxfp8(h_codes, h_scales)
    y_perm = np.zeros((R, H))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            y_perm[lo:hi] = hd[lo:hi] @ dd[e].T
    y_shared = h_shared = None
    if ws_gate is not None:
        y_shared, h_shared = dense_mxfp8(x, ws_gate[0], ws_up[0], ws_down[0])
    y = _bf.combine(y_perm, dest, w, y_shared)
    return dict(ids=ids, w=w, counts=counts, offsets=offsets, dest_rows=dest,
                sorted_token_ids=sorted_tok, x_codes=xq_codes, x_scales=xq_scales,
                h=h, h_codes=h_codes, h_scales=h_scales, y_perm=y_perm, y_shared=y_shared,
                h_shared=h_shared, y=y)
