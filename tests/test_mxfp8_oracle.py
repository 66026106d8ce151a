"""Pins of the MXFP8 oracle (oracle/mxfp8.py), CPU only.

Nothing here retypes the oracle's formulas: E4M3 encoding is checked against a
brute-force nearest-value search over all 256 codes, decoding against the
format's stated constants and its monotone spacing, the shared exponent against
its defining interval, and the layer against exact special cases and the bf16
oracle.  Each planted mistake at the bottom must fail at least one pin."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import moe_oracle, mxfp8

FINITE = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)


def brute_encode(v, decode):
    """Nearest finite E4M3 value by exhaustive search; ties go to the even mantissa;
    magnitudes beyond 448 clamp to 448; the sign bit follows the input."""
    vals = decode(FINITE)
    out = np.empty(len(v), dtype=np.uint8)
    for i, x in enumerate(np.asarray(v, dtype=np.float64)):
        cand = FINITE[(np.signbit(vals) == np.signbit(x))]
        cv = decode(cand)
        a = min(abs(x), 448.0)
        d = np.abs(np.abs(cv) - a)
        best = cand[d == d.min()]
        if len(best) > 1:
            best = best[(best & 1) == 0]
        out[i] = best[0]
    return out


# --------------------------------------------------------------------------- decode
def check_decode(decode):
    v = decode(np.arange(256, dtype=np.uint8))
    # constants stated by the format
    assert v[0x7E] == 448.0 and v[0xFE] == -448.0
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF])
    assert np.isnan(v).sum() == 2
    assert v[0x08] == 2.0 ** -6 and v[0x01] == 2.0 ** -9 and v[0x07] == 7 * 2.0 ** -9
    assert v[0x38] == 1.0 and v[0x00] == 0.0 and np.signbit(v[0x80])
    # positive codes are strictly increasing and negative codes mirror them
    pos = v[:0x7F]
    assert (np.diff(pos) > 0).all()
    assert np.array_equal(v[0x80:0xFF], -pos)
    # codes 8g .. 8g+7 share one spacing d_g (the step into the next group too);
    # subnormals (g = 0) are spaced like the first normal binade, and the spacing
    # doubles from one normal binade to the next
    steps = np.diff(pos)                                  # steps[c] = pos[c + 1] - pos[c]
    d = [steps[8 * g] for g in range(16)]
    for g in range(16):
        seg = steps[8 * g: min(8 * g + 8, len(steps))]
        assert (seg == d[g]).all()
    assert d[0] == d[1] == 2.0 ** -9
    assert all(d[g + 1] == 2 * d[g] for g in range(1, 15))


def test_decode():
    check_decode(mxfp8.e4m3_decode)


# --------------------------------------------------------------------------- encode
def encode_cases(rng):
    vals = mxfp8.e4m3_decode(FINITE)
    pos = np.sort(vals[vals > 0])
    mids = (pos[:-1] + pos[1:]) / 2                       # exact midpoints: ties
    near = np.concatenate([mids * (1 + 1e-12), mids * (1 - 1e-12)])
    rnd = rng.standard_normal(3000) * np.exp2(rng.integers(-12, 10, 3000))
    edge = np.array([0.0, -0.0, 448.0, 449.0, 463.9, 464.0, 464.1, 479.9, 480.0, 511.9, 1e6,
                     2.0 ** -10, 2.0 ** -10 * 1.0000001, 3 * 2.0 ** -11, 2.0 ** -12, 2.0 ** -9,
                     2.0 ** -6 - 2.0 ** -10, 2.0 ** -6 - 2.0 ** -11])
    allv = np.concatenate([pos, mids, near, rnd, edge])
    return np.concatenate([allv, -allv])


def check_encode(encode, decode):
    rng = np.random.default_rng(3)
    v = encode_cases(rng)
    assert np.array_equal(encode(v), brute_encode(v, decode))
    # every representable value encodes to itself
    assert np.array_equal(encode(decode(FINITE)), FINITE)


def test_encode_matches_brute_force():
    check_encode(mxfp8.e4m3_encode, mxfp8.e4m3_decode)


# --------------------------------------------------------------------------- MX blocks
def check_quantize(quantize, dequantize):
    rng = np.random.default_rng(4)
    rows = [rng.standard_normal(64) * 2.0 ** rng.integers(-20, 20) for _ in range(200)]
    rows += [np.zeros(64), np.full(64, 2.0 ** -140), np.array([2.0 ** 100] + [0.0] * 63),
             np.concatenate([np.full(32, 1.0), np.full(32, -3.0)])]
    a = np.stack(rows)
    codes, scales = quantize(a)
    assert codes.dtype == np.uint8 and scales.dtype == np.uint8 and scales.shape == (a.shape[0], 2)
    blocks = a.reshape(a.shape[0], 2, 32)
    amax = np.abs(blocks).max(axis=-1)
    se = scales.astype(np.int64) - 127
    # the defining interval: 2^(se + 8) <= amax < 2^(se + 9), unless clamped or zero
    live = (amax > 0) & (se > -127)
    assert (np.exp2(se[live] + 8.0) <= amax[live]).all() and (amax[live] < np.exp2(se[live] + 9.0)).all()
    assert (se[amax == 0] == -127).all()
    # error bound: half a spacing of the element's E4M3 binade, or clamped to 448
    d = dequantize(codes, scales).reshape(blocks.shape)
    scaled = blocks / np.exp2(se)[..., None]
    _, ex = np.frexp(np.abs(scaled))
    spacing = np.exp2(np.maximum(ex - 1, -6) - 3.0) * np.exp2(se)[..., None]
    sat = np.abs(scaled) > 448
    ok = np.abs(d - blocks) <= spacing / 2 + 0.0
    assert (ok | sat).all()
    assert (np.abs(d[sat]) == (448.0 * np.exp2(se)[..., None] * np.ones_like(d))[sat]).all()
    # hand-worked blocks: max 1.0 -> exponent 0 - 8, byte 119, 1.0 -> 256 (code 0x78)
    c, s = quantize(np.concatenate([[1.0, -0.5, 0.25], np.zeros(29)])[None])
    assert s[0, 0] == 119 and c[0, 0] == 0x78 and c[0, 1] == 0xF0 and c[0, 2] == 0x68
    # max 3.0: floor(log2 3) = 1 -> exponent -7 (byte 120); 3.0 -> 384 = 1.5 * 2^8 (0x7C);
    # 0.1 -> 12.8 -> 13 = 1.625 * 2^3 (exponent field 10, mantissa 5: 0x55)
    c, s = quantize(np.concatenate([[3.0, 0.1], np.zeros(30)])[None])
    assert s[0, 0] == 120 and c[0, 0] == 0x7C and c[0, 1] == 0x55


def test_quantize_blocks():
    check_quantize(mxfp8.quantize_mxfp8, mxfp8.dequantize_mxfp8)


def test_quantize_reads_bf16_bits():
    """bf16 bit patterns are upcast exactly before quantizing."""
    import moegen
    rng = np.random.default_rng(5)
    a = rng.standard_normal((4, 64)).astype(np.float32)
    b = moegen.round_bf16(a)
    c1, s1 = mxfp8.quantize_mxfp8(b)
    c2, s2 = mxfp8.quantize_mxfp8(moegen.as_f64(b))
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)


# --------------------------------------------------------------------------- layer
def small_inputs(rng, T=40, H=64, E=4, k=2, F=96, exact=False):
    """Random layer inputs; exact=True draws every value from {-2, -1, -0.5, 0.5, 1, 2}
    times one power of two per block, so that MXFP8 holds them exactly."""
    def draw(shape):
        if exact:
            v = rng.choice([-2.0, -1.0, -0.5, 0.5, 1.0, 2.0], size=shape)
            return v
        return rng.standard_normal(shape) * 0.5
    x = draw((T, H))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    wg = draw((E, F, H)) / 8
    wu = draw((E, F, H)) / 8
    wd = draw((E, H, F)) / 8
    return x, logits, k, wg, wu, wd


def check_layer_exact_inputs(layer_fn):
    """MXFP8-exact x and weights: g and u are the exact products, so the layer's h
    is the bf16 oracle's h, and y_perm is Q(h) times W_down."""
    rng = np.random.default_rng(6)
    x, logits, k, wg, wu, wd = small_inputs(rng, exact=True)
    assert np.array_equal(mxfp8.roundtrip(x), x) and np.array_equal(mxfp8.roundtrip(wd), wd)
    out = layer_fn(x, logits, k, wg, wu, wd)
    ref = moe_oracle.layer(x, logits, k, wg, wu, wd)
    xp = ref["x_perm"]
    off = ref["offsets"]
    for e in range(wg.shape[0]):
        lo, hi = int(off[e]), int(off[e + 1])
        if hi == lo:
            continue
        g = xp[lo:hi] @ wg[e].T
        u = xp[lo:hi] @ wu[e].T
        h = g / (1 + np.exp(-g)) * u
        assert np.allclose(out["h"][lo:hi], h, rtol=1e-13, atol=1e-13)
        hq = mxfp8.roundtrip(h)
        assert np.allclose(out["y_perm"][lo:hi], hq @ wd[e].T, rtol=1e-13, atol=1e-13)
    assert np.array_equal(out["ids"], ref["ids"]) and np.array_equal(out["dest_rows"], ref["dest_rows"])


def check_layer_identical_experts(layer_fn):
    """Identical experts and renormalised weights: y is the dense MXFP8 FFN of every
    token whatever the routing."""
    rng = np.random.default_rng(7)
    x, logits, k, wg, wu, wd = small_inputs(rng)
    wg[:] = wg[0]
    wu[:] = wu[0]
    wd[:] = wd[0]
    out = layer_fn(x, logits, k, wg, wu, wd)
    xd = mxfp8.roundtrip(x)
    g = xd @ mxfp8.roundtrip(wg[0]).T
    u = xd @ mxfp8.roundtrip(wu[0]).T
    h = mxfp8.roundtrip(g / (1 + np.exp(-g)) * u)
    assert np.allclose(out["y"], h @ mxfp8.roundtrip(wd[0]).T, rtol=1e-12, atol=1e-12)


def check_layer_scaling(layer_fn):
    """W_down scaled by 2^5 scales y by exactly 2^5 (E8M0 scales absorb powers of two)."""
    rng = np.random.default_rng(8)
    x, logits, k, wg, wu, wd = small_inputs(rng)
    a = layer_fn(x, logits, k, wg, wu, wd)["y"]
    b = layer_fn(x, logits, k, wg, wu, wd * 32.0)["y"]
    assert np.array_equal(b, a * 32.0)


def check_layer_close_to_bf16(layer_fn):
    """MXFP8 keeps 3 mantissa bits: the layer stays within a few percent of the
    unquantized layer on Gaussian data."""
    rng = np.random.default_rng(9)
    x, logits, k, wg, wu, wd = small_inputs(rng, T=64, H=128, F=128)
    a = layer_fn(x, logits, k, wg, wu, wd)["y"]
    b = moe_oracle.layer(x, logits, k, wg, wu, wd)["y"]
    rel = np.abs(a - b).max() / np.abs(b).max()
    assert 1e-4 < rel < 0.1


def check_layer_single_expert_and_shared(layer_fn):
    """E = 1, k = 1: every token goes to expert 0 with weight 1, so the layer is the
    dense MXFP8 FFN; a shared expert adds its own dense MXFP8 FFN."""
    rng = np.random.default_rng(10)
    x, logits, _, wg, wu, wd = small_inputs(rng, E=1)
    out = layer_fn(x, logits[:, :1], 1, wg, wu, wd)
    dense, _ = mxfp8.dense_mxfp8(x, wg[0], wu[0], wd[0])
    assert np.allclose(out["y"], dense, rtol=1e-12, atol=1e-12)
    _, _, _, sg, su, sd = small_inputs(rng, E=1)
    out2 = layer_fn(x, logits[:, :1], 1, wg, wu, wd, 1, sg, su, sd)
    shared, _ = mxfp8.dense_mxfp8(x, sg[0], su[0], sd[0])
    assert np.allclose(out2["y"], dense + shared, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("check", [check_layer_exact_inputs, check_layer_identical_experts,
                                   check_layer_scaling, check_layer_close_to_bf16,
                                   check_layer_single_expert_and_shared])
def test_layer(check):
    check(mxfp8.layer_mxfp8)


# --------------------------------------------------------------------------- planted mistakes
def _mut_encode_ties_away(v):
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    _, ex = np.frexp(a)
    e = np.maximum(np.where(a > 0, ex - 1, -6), -6)
    q = np.exp2(e - 3.0)
    r = np.floor(a / q + 0.5)                                 # ties away from zero
    return mxfp8.e4m3_encode(np.sign(v) * np.minimum(r * q, 448.0) + np.where(np.signbit(v), -0.0, 0.0))


def _mut_encode_no_saturation(v):
    v = np.asarray(v, dtype=np.float64)
    out = mxfp8.e4m3_encode(v)
    big = np.abs(v) >= 464
    out[big] = (out[big] & 0x80) | 0x7F                         # overflow to NaN
    return out


def _mut_decode_bias8(c):
    return mxfp8.e4m3_decode(c) / 2.0


def _mut_quantize_exp_minus7(a):
    x = moe_oracle._f64(a)
    blocks = x.reshape(x.shape[:-1] + (-1, 32))
    se = np.clip(mxfp8.shared_exponent(np.abs(blocks).max(axis=-1)) + 1, -127, 127)
    codes = mxfp8.e4m3_encode(blocks / np.exp2(se)[..., None]).reshape(x.shape)
    return codes, (se + 127).astype(np.uint8)


def _mut_quantize_block16(a):
    x = moe_oracle._f64(a)
    b16 = x.reshape(x.shape[:-1] + (-1, 16))
    se16 = mxfp8.shared_exponent(np.abs(b16).max(axis=-1))
    codes = mxfp8.e4m3_encode(b16 / np.exp2(se16)[..., None]).reshape(x.shape)
    return codes, (se16[..., ::2] + 127).astype(np.uint8)


def _mut_dequantize_bias126(codes, scales):
    return mxfp8.dequantize_mxfp8(codes, scales) * 2.0


def _mut_layer_h_unquantized(x, logits, k, wg, wu, wd, renormalize=1):
    out = mxfp8.layer_mxfp8(x, logits, k, wg, wu, wd, renormalize)
    E = wg.shape[0]
    off, st = out["offsets"], out["sorted_token_ids"]
    dd = mxfp8.roundtrip(wd)
    y_perm = np.zeros_like(out["y_perm"])
    for e in range(E):
        lo, hi = int(off[e]), int(off[e + 1])
        if hi > lo:
            y_perm[lo:hi] = out["h"][lo:hi] @ dd[e].T
    out["y_perm"] = y_perm
    out["y"] = moe_oracle.combine(y_perm, out["dest_rows"], out["w"])
    return out


def _mut_layer_wd_unquantized(x, logits, k, wg, wu, wd, renormalize=1):
    out = mxfp8.layer_mxfp8(x, logits, k, wg, wu, wd, renormalize)
    E = wg.shape[0]
    off = out["offsets"]
    hd = mxfp8.roundtrip(out["h"])
    y_perm = np.zeros_like(out["y_perm"])
    for e in range(E):
        lo, hi = int(off[e]), int(off[e + 1])
        if hi > lo:
            y_perm[lo:hi] = hd[lo:hi] @ moe_oracle._f64(wd[e]).T
    out["y_perm"] = y_perm
    out["y"] = moe_oracle.combine(y_perm, out["dest_rows"], out["w"])
    return out


MUTANTS = [
    ("encode ties away from zero", lambda: check_encode(_mut_encode_ties_away, mxfp8.e4m3_decode)),
    ("encode overflows to NaN", lambda: check_encode(_mut_encode_no_saturation, mxfp8.e4m3_decode)),
    ("decode with exponent bias 8", lambda: check_decode(_mut_decode_bias8)),
    ("shared exponent floor(log2 amax) - 7", lambda: check_quantize(_mut_quantize_exp_minus7,
                                                                      mxfp8.dequantize_mxfp8)),
    ("blocks of 16", lambda: check_quantize(_mut_quantize_block16, mxfp8.dequantize_mxfp8)),
    ("scale bias 126", lambda: check_quantize(mxfp8.quantize_mxfp8, _mut_dequantize_bias126)),
    ("h not quantized", lambda: check_layer_exact_inputs(_mut_layer_h_unquantized)),
    ("W_down not quantized", lambda: check_layer_identical_experts(_mut_layer_wd_unquantized)),
]


@pytest.mark.parametrize("name,run", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, run):
    with pytest.raises(AssertionError):
        run()
