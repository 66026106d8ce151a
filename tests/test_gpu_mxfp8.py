"""GPU parity of the MXFP8 path (moe_quantize_mxfp8, moe_grouped_ffn_mxfp8) against
the fp64 MXFP8 oracle (oracle/mxfp8.py), through the C ABI.

Quantization of given bf16 rows is bit-exact (codes and scales), on rows built
to hit every rounding case.  In the layer, h is quantized from values the two
sides compute differently (fp32 on the GPU, exact in the oracle), and where a
value or a block maximum straddles a rounding boundary both results are
correct: so the unique results are compared bit-exactly (routing, grouping, the
x and weight codes), the kernel's h is checked to be a valid quantization of the
exact h, and y_perm and y are checked against the fp64 continuation from the
kernel's own h."""
import numpy as np
import pytest
import torch

import moegen
from oracle import mxfp8
import paper_2606_21712_amd as moe
from tests.gpu_util import f64, log, rel_max_err, to_dev, to_host

pytestmark = pytest.mark.gpu



def scales_rowmajor(scales, rows, K):
    """The library's k-step-major scale bytes [K / 128][rows][4] -> [rows, K / 32]."""
    s = np.asarray(scales)[: rows * K // 32].reshape(K // 128, rows, 4)
    return s.transpose(1, 0, 2).reshape(rows, K // 32)


def special_rows(K, rng):
    """bf16 rows whose blocks hit ties, saturation, zeros, subnormals and -0."""
    rows = []
    # block max 1.0 (shared exponent -8): scaled values are the integers k, so odd
    # integers in [16, 32) and k + 0.5 in [8, 16) are exact ties
    r = np.zeros(K, dtype=np.float32)
    r[0::32] = 1.0
    vals = np.concatenate([np.arange(1, 32) / 256.0, (np.arange(16, 31) + 0.5) / 256.0])
    for i in range(K):
        if i % 32:
            r[i] = vals[(i * 7) % len(vals)] * (-1 if i % 3 == 0 else 1)
    rows.append(r)
    # saturation: block max 1.875 -> 480 clamps to 448; 1.8125 -> 464, a tie between 448 and 480
    r = np.full(K, 1.8125, dtype=np.float32)
    r[0::32] = 1.875
    r[5::32] = -1.8125
    rows.append(r)
    rows.append(np.zeros(K, dtype=np.float32))                              # all-zero blocks
    rows.append(np.full(K, 2.0 ** -130, dtype=np.float32))                  # bf16 subnormals
    r = np.full(K, -0.0, dtype=np.float32)
    r[1::32] = 3.0
    rows.append(r)                                                          # -0 next to a value
    r = (rng.standard_normal(K) * np.exp2(rng.integers(-40, 40, K))).astype(np.float32)
    rows.append(r)                                                          # wild dynamic range
    return np.stack(rows)


@pytest.mark.parametrize("rows,K", [(37, 128), (300, 384), (1000, 4096)])
def test_quantize_bitexact(rows, K):
    rng = np.random.default_rng(rows + K)
    a = (rng.standard_normal((rows, K)) * np.exp2(rng.integers(-8, 8, (rows, 1)))).astype(np.float32)
    a[: 6] = special_rows(K, rng)
    xb = moegen.round_bf16(a)
    log(f"[gpu] quantize_mxfp8 rows={rows} K={K}")
    q = moe.moe_quantize_mxfp8(to_dev(xb))
    torch.cuda.synchronize()
    ref_c, ref_s = mxfp8.quantize_mxfp8(xb)
    got_c = to_host(q.codes)
    got_s = scales_rowmajor(to_host(q.scales), rows, K)
    assert np.array_equal(got_s, ref_s)
    assert np.array_equal(got_c, ref_c)


def test_quantize_row_map():
    rng = np.random.default_rng(11)
    src = moegen.round_bf16(rng.standard_normal((50, 256)).astype(np.float32))
    row_map = rng.integers(0, 50, 173).astype(np.int32)                     # repeats, any order
    log("[gpu] quantize_mxfp8 with a row map")
    q = moe.moe_quantize_mxfp8(to_dev(src), row_map=to_dev(row_map))
    torch.cuda.synchronize()
    ref_c, ref_s = mxfp8.quantize_mxfp8(src[row_map])
    assert np.array_equal(to_host(q.codes), ref_c)
    assert np.array_equal(scales_rowmajor(to_host(q.scales), 173, 256), ref_s)


# Several m-tiles per group with ragged tails, a half-full down-projection n-tile
# (H % 256 = 128), empty experts, pinned tiny groups.
CASES = {
    "f8_mixtral_small": moegen.MoEConfig("f8_mixtral_small", T=1500, H=384, E=8, k=2, F=384, seed=31),
    "f8_memc_small": moegen.MoEConfig("f8_memc_small", T=3000, H=256, E=32, k=4, F=256, seed=32,
                                      routing="lognormal", pinned_small=(1, 17, 31)),
    "f8_deepseek_small": moegen.MoEConfig("f8_deepseek_small", T=512, H=512, E=64, k=8, F=128, Fs=256,
                                          seed=33),
    "f8_uniform": moegen.MoEConfig("f8_uniform", T=300, H=128, E=8, k=3, F=256, seed=34, routing="uniform"),
}


def _random_cases(n=4, seed=2027):
    """Seeded random shapes within the MXFP8 limits (H, F multiples of 128)."""
    rng = np.random.default_rng(seed)
    out = {}
    for i in range(n):
        E = int(rng.choice([1, 3, 5, 8, 16, 64]))
        k = int(rng.integers(1, min(E, 8) + 1))
        T = int(rng.integers(1, 1500))
        H = 128 * int(rng.integers(1, 6))
        F = 128 * int(rng.integers(1, 5))
        Fs = int(rng.choice([0, 256]))
        out[f"f8_rand{i}"] = moegen.MoEConfig(f"f8_rand{i}", T=T, H=H, E=E, k=k, F=F, Fs=Fs, seed=40 + i)
    return out


CASES.update(_random_cases())

# Accumulation error of the block-scaled fp8 MFMA, as a fraction of sum_k |a_k b_k|:
# measured on gfx950 at 1.26e-4 for K = 512 random E4M3 codes over their whole
# range with random scales (far coarser than fp32's 6e-8 per addition: the matrix
# core adds the fp8 products at reduced internal precision).  The bound takes twice that.
ACC = 2.0 ** -12


def h_deviation_bound(xd, gd, ud, offsets):
    """Per element of h, how far the kernel's fp32 h may lie from the exact one: the
    accumulation bound on g and u propagated through silu(g) * u (|silu'| <= 1.1),
    plus 2^-14 |h| for evaluating silu(g) * u in fp32 (exp, reciprocal and two
    products, each within a few ulp; the rounding of exp's argument -g log2(e)
    adds up to |g| ulp, and |g| stays far below 2^9 here)."""
    R = xd.shape[0]
    F = gd.shape[1]
    h = np.zeros((R, F))
    dh = np.zeros((R, F))
    for e in range(gd.shape[0]):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        xr = xd[lo:hi]
        g, u = xr @ gd[e].T, xr @ ud[e].T
        dg = ACC * (np.abs(xr) @ np.abs(gd[e]).T)
        du = ACC * (np.abs(xr) @ np.abs(ud[e]).T)
        silu = g / (1 + np.exp(-g))
        h[lo:hi] = silu * u
        assert np.abs(g).max() < 2.0 ** 9
        dh[lo:hi] = 1.1 * np.abs(u) * dg + np.abs(silu) * du + 1.1 * dg * du + 2.0 ** -14 * np.abs(silu * u)
    return h, dh


def check_valid_quantization(codes, scales, h, dh):
    """codes/scales are a correct MXFP8 quantization of some h' with |h' - h| <= dh: the
    shared exponent is the exact h's unless the block maximum is within reach of a
    power of two, and every element is within half an E4M3 spacing (at the chosen
    scale) plus dh, or saturated."""
    R, F = h.shape
    blocks = h.reshape(R, F // 32, 32)
    dblk = dh.reshape(R, F // 32, 32)
    amax = np.abs(blocks).max(axis=-1)
    se_or = mxfp8.shared_exponent(amax)
    se = scales.astype(np.int64) - 127
    differ = se != se_or
    if differ.any():
        edge = np.exp2(np.maximum(se, se_or)[differ] + 8.0)
        assert (np.abs(amax[differ] - edge) <= dblk.max(axis=-1)[differ]).all()
        assert (np.abs(se - se_or)[differ] == 1).all()
    v = mxfp8.e4m3_decode(codes.reshape(R, F // 32, 32)) * np.exp2(se)[..., None]
    scaled = np.abs(blocks) / np.exp2(se)[..., None]
    _, ex = np.frexp(scaled)
    half = 0.5 * np.exp2(np.maximum(ex - 1, -6) - 3.0) * np.exp2(se)[..., None]
    sat = np.abs(blocks) + dblk > 448 * np.exp2(se)[..., None]
    ok = np.abs(v - blocks) <= half + dblk
    ok |= sat & (np.abs(v) == 448.0 * np.exp2(se)[..., None])
    assert ok.all(), int((~ok).sum())
    return differ.sum(), (codes != mxfp8.quantize_mxfp8(h)[0]).sum()


def check_ffn(xd, offsets, w_gate, w_up, w_down, ws, y_perm, label):
    """One MXFP8 grouped FFN of the kernel against the exact one: xd are the dequantized
    input rows in grouped order, ws the call's workspace (holding the kernel's h)."""
    E = w_gate.shape[0]
    R, F = xd.shape[0], w_gate.shape[1]
    h_ex, dh = h_deviation_bound(xd, mxfp8.roundtrip(w_gate), mxfp8.roundtrip(w_up), offsets)
    ws_host = to_host(ws)
    h_off = ((E + 1) * 4 + 255) // 256 * 256 + 256
    hs_off = h_off + (R * F + 255) // 256 * 256
    hc = ws_host[h_off: h_off + R * F].reshape(R, F)
    hs = scales_rowmajor(ws_host[hs_off: hs_off + R * F // 32], R, F)
    flips_s, flips_c = check_valid_quantization(hc, hs, h_ex, dh)
    log(f"[gpu]   {label} h: {flips_s} block scales and {flips_c} of {hc.size} codes differ from the exact h's")
    # y_perm against the fp64 product of the kernel's own h: the accumulation bound,
    # then bf16 rounding of the output (8 significant bits: 2^-8 relative)
    hd = mxfp8.dequantize_mxfp8(hc, hs)
    dd = mxfp8.roundtrip(w_down)
    yp = f64(to_host(y_perm))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            yr = hd[lo:hi] @ dd[e].T
            acc = ACC * (np.abs(hd[lo:hi]) @ np.abs(dd[e]).T)
            bound = 2.0 ** -8 * (np.abs(yr) + acc) + acc + 1e-30
            assert (np.abs(yp[lo:hi] - yr) <= bound).all(), (label, e, hi - lo)
    return yp


def run_mxfp8_layer(c, I, gather=True):
    wq = [moe.quantize_weights_mxfp8(to_dev(w)) for w in (I.w_gate, I.w_up, I.w_down)]
    wqs = [moe.quantize_weights_mxfp8(to_dev(w)) for w in (I.ws_gate, I.ws_up, I.ws_down)] if c.Fs \
        else [None, None, None]
    layer = moe.MoELayerMXFP8(c.T, c.H, c.E, c.k, c.F, c.Fs, gather=gather)
    layer.run(to_dev(I.x), to_dev(I.logits), *wq, *wqs)
    torch.cuda.synchronize()
    return layer, wq


@pytest.mark.parametrize("name", list(CASES))
def test_layer_mxfp8(name):
    """Unique results bit-exact (routing, grouping, x and weight codes); h checked as a
    valid quantization of the exact h within the accumulation bound; y_perm against the
    fp64 product of the kernel's own h with the quantized W_down (accumulation bound
    plus bf16 rounding, per element); y against the combine of those results."""
    c = CASES[name]
    I = moegen.make_inputs(c)
    log(f"[gpu] mxfp8 layer {name} T={c.T} H={c.H} E={c.E} k={c.k} F={c.F} Fs={c.Fs}")
    layer, wq = run_mxfp8_layer(c, I)
    sh = (I.ws_gate, I.ws_up, I.ws_down) if c.Fs else (None, None, None)
    ref = mxfp8.layer_mxfp8(I.x, I.logits, c.k, I.w_gate, I.w_up, I.w_down, 1, *sh)
    assert np.array_equal(to_host(layer.topk_ids), ref["ids"])
    assert np.array_equal(to_host(layer.perm["offsets"]), ref["offsets"])
    assert np.array_equal(to_host(layer.perm["dest_rows"]), ref["dest_rows"])
    st = ref["sorted_token_ids"]
    # the token rows are quantized once, in token order
    assert np.array_equal(to_host(layer.xq.codes), ref["x_codes"])
    assert np.array_equal(scales_rowmajor(to_host(layer.xq.scales), c.T, c.H), ref["x_scales"])
    for wt, w in zip(wq, (I.w_gate, I.w_up, I.w_down)):
        wc, wsc = mxfp8.quantize_mxfp8(w)
        rows = w.shape[0] * w.shape[1]
        assert np.array_equal(to_host(wt.codes), wc)
        assert np.array_equal(scales_rowmajor(to_host(wt.scales), rows, w.shape[2]),
                              wsc.reshape(rows, w.shape[2] // 32))
    xd = mxfp8.dequantize_mxfp8(ref["x_codes"], ref["x_scales"])
    yp = check_ffn(xd[st], ref["offsets"], I.w_gate, I.w_up, I.w_down, layer.ws_ffn, layer.y_perm, "routed")
    ys = None
    if c.Fs:
        ys = check_ffn(xd, np.array([0, c.T]), I.ws_gate, I.ws_up, I.ws_down, layer.ws_shared, layer.y_shared,
                       "shared")
    y_ref = mxfp8._bf.combine(yp, ref["dest_rows"], ref["w"], ys)
    err = rel_max_err(f64(to_host(layer.y)), y_ref)
    log(f"[gpu]   y rel max err {err:.2e} (against the combine of the kernel's expert outputs)")
    assert err <= 2.0 ** -8
    # and the whole layer stays close to the oracle's own (few flips, each small)
    assert rel_max_err(f64(to_host(layer.y)), ref["y"]) <= 0.1


def test_mxfp8_down_projection_tail_split():
    """MXFP8 down projection with its last round of tiles cut along k (planned for fewer
    compute units): h is untouched (GEMM-1 never splits), y_perm outside the tail
    keeps its bits and the tail moves only by reassociation; y_perm still meets the
    per-element bound against the kernel's own h."""
    from tests.gpu_util import split_budgets
    from tests.test_gpu_parity import check_tail_split
    c = moegen.MoEConfig("f8_tail_split", T=2048, H=512, E=8, k=2, F=4096, seed=35)
    I = moegen.make_inputs(c)
    ref = mxfp8.layer_mxfp8(I.x, I.logits, c.k, I.w_gate, I.w_up, I.w_down, 1)
    picks, plain = split_budgets(ref["offsets"], c.H, c.F // 128, 0)
    assert len(picks) >= 2 and plain is not None, (picks, plain)
    try:
        log(f"[gpu] mxfp8 tail split reference: budget {plain}, no split")
        moe.set_cu_budget(plain)
        base, _ = run_mxfp8_layer(c, I)
        h_base = to_host(base.ws_ffn)
        y_base = to_host(base.y_perm)
        xd = mxfp8.dequantize_mxfp8(ref["x_codes"], ref["x_scales"])[ref["sorted_token_ids"]]
        for b, r, s in picks:
            log(f"[gpu] mxfp8 tail split: budget {b}, {r} tail tiles in {s} pieces")
            moe.set_cu_budget(b)
            g, _ = run_mxfp8_layer(c, I)
            hb = c.T * c.k * c.F
            h_off = ((c.E + 1) * 4 + 255) // 256 * 256 + 256
            assert np.array_equal(to_host(g.ws_ffn)[h_off:h_off + hb], h_base[h_off:h_off + hb])
            check_tail_split(to_host(g.y_perm), y_base, r, f"budget {b}")
            check_ffn(xd, ref["offsets"], I.w_gate, I.w_up, I.w_down, g.ws_ffn, g.y_perm, f"budget {b}")
    finally:
        moe.set_cu_budget(0)


def test_layer_mxfp8_gather_equals_grouped_copy():
    """Gathering the token codes in GEMM-1 gives the same bits as quantizing x into
    grouped order first."""
    c = CASES["f8_memc_small"]
    I = moegen.make_inputs(c)
    log("[gpu] mxfp8 gather vs grouped copy")
    a, _ = run_mxfp8_layer(c, I, gather=True)
    b, _ = run_mxfp8_layer(c, I, gather=False)
    assert np.array_equal(to_host(a.y_perm), to_host(b.y_perm))
    assert np.array_equal(to_host(a.y), to_host(b.y))
