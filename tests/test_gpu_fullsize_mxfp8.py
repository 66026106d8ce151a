"""GPU parity of the MXFP8 layer at the workloads' full sizes, in the configuration
`bench.py --mxfp8` times (gather path: the token rows quantized once, GEMM-1
gathering their codes; the down projection's tail split at the device's grid).

Routing and grouping are compared bit-exactly on every token.  The rest is
checked on samples the oracle computes directly from the format: for every
expert group its first, middle and last rows and one random row of each of its
256-row m-tiles (the MXFP8 GEMMs cut an expert's rows into m-tiles of 256 from
its first row), on which
  * the x codes and scales of the row's token equal the oracle's quantization;
  * four 32-feature blocks of the kernel's h are a valid MXFP8 quantization of
    the exact h (from the oracle's x and weight codes) within the accumulation
    bound (the bar of test_gpu_mxfp8);
  * eight outputs of y_perm equal the fp64 product of the kernel's own h row with
    the oracle's quantization of that W_down row, within the accumulation bound
    plus bf16 rounding;
and the final y of a token sample touching every expert equals the combine of the
kernel's own expert outputs within bf16 rounding."""
import numpy as np
import pytest
import torch

import moegen
from oracle import mxfp8
import paper_2606_21712_amd as moe
from tests.gpu_util import f64, log, to_dev, to_host, weight_tol
from tests.test_gpu_mxfp8 import ACC, check_valid_quantization

pytestmark = pytest.mark.gpu


def _silu(z):
    return z / (1.0 + np.exp(-z))


def _ws_offsets(E, R, F):
    """Byte offsets of the h codes and h scales in the MXFP8 FFN workspace."""
    h_off = ((E + 1) * 4 + 255) // 256 * 256 + 256
    return h_off, h_off + (R * F + 255) // 256 * 256


def _h_row(ws, E, R, F, r):
    """Row r of the kernel's h: codes [F] and scales [F / 32] (from the k-step-major layout)."""
    h_off, hs_off = _ws_offsets(E, R, F)
    codes = ws[h_off + r * F: h_off + (r + 1) * F]
    b = np.arange(F // 32)
    scales = ws[hs_off + ((b // 4) * R + r) * 4 + (b % 4)]
    return codes, scales


def _check_rows(label, rows_tok, rows_r, e_of, xq_host, x_rows_bf16, wg, wu, wd, ws, E, R, H, F, y_rows, rng):
    """The sampled-row checks of one grouped FFN (routed or shared)."""
    n_flip = 0
    for i, (t, r) in enumerate(zip(rows_tok, rows_r)):
        t, r, e = int(t), int(r), e_of[i]
        # x codes of the token, bit-exact
        xc, xs = mxfp8.quantize_mxfp8(x_rows_bf16[i][None, :])
        assert np.array_equal(xq_host[0][t], xc[0]), (label, t)
        assert np.array_equal(xq_host[1][t], xs[0]), (label, t)
        xd = mxfp8.dequantize_mxfp8(xc, xs)[0]
        # four h blocks: valid quantization of the exact h
        hc, hsc = _h_row(ws, E, R, F, r)
        for b in rng.choice(F // 32, size=min(4, F // 32), replace=False):
            f = slice(32 * b, 32 * b + 32)
            gd = mxfp8.roundtrip(wg[e, f])
            ud = mxfp8.roundtrip(wu[e, f])
            g, u = gd @ xd, ud @ xd
            dg, du = ACC * (np.abs(gd) @ np.abs(xd)), ACC * (np.abs(ud) @ np.abs(xd))
            h = _silu(g) * u
            dh = 1.1 * np.abs(u) * dg + np.abs(_silu(g)) * du + 1.1 * dg * du + 2.0 ** -14 * np.abs(h)
            fs, fc = check_valid_quantization(hc[f][None, :], hsc[b:b + 1][None, :], h[None, :], dh[None, :])
            n_flip += fc
        # eight y_perm outputs against the kernel's own h row
        hd = mxfp8.dequantize_mxfp8(hc[None, :], hsc[None, :])[0]
        for n in rng.choice(H, size=8, replace=False):
            dd = mxfp8.roundtrip(wd[e, n][None, :])[0]
            y_ex = float(hd @ dd)
            acc = ACC * float(np.abs(hd) @ np.abs(dd))
            bound = 2.0 ** -8 * (abs(y_ex) + acc) + acc + 1e-30
            assert abs(y_rows[i, n] - y_ex) <= bound, (label, r, n, y_rows[i, n], y_ex, bound)
    return n_flip


@pytest.mark.parametrize("name", ["mixtral4k", "mixtral32k_zipf", "deepseek", "memconstrained"])
def test_full_size_layer_mxfp8(name):
    cfg = moegen.CONFIGS[name]
    log(f"[gpu] full-size mxfp8 {name}: generating T={cfg.T} H={cfg.H} E={cfg.E} k={cfg.k} F={cfg.F} Fs={cfg.Fs}")
    I = moegen.make_inputs(cfg)
    wq = [moe.quantize_weights_mxfp8(to_dev(w)) for w in (I.w_gate, I.w_up, I.w_down)]
    wqs = [moe.quantize_weights_mxfp8(to_dev(w)) for w in (I.ws_gate, I.ws_up, I.ws_down)] if cfg.Fs \
        else [None, None, None]
    layer = moe.MoELayerMXFP8(cfg.T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs)
    log(f"[gpu] full-size mxfp8 {name}: running the layer")
    layer.run(to_dev(I.x), to_dev(I.logits), *wq, *wqs, renormalize=cfg.renormalize)
    torch.cuda.synchronize()
    del wq, wqs

    # routing and grouping, every token, bit-exact
    ids_g, w_g = to_host(layer.topk_ids), to_host(layer.topk_weights)
    ids_o, w_o = mxfp8._bf.route(I.logits, cfg.k, cfg.renormalize)
    assert np.array_equal(ids_g, ids_o)
    assert np.abs(w_g - w_o).max() <= weight_tol(cfg.k, cfg.E)
    counts, offsets, dest, stok, _ = mxfp8._bf.permute(ids_o, np.zeros((cfg.T, 1), np.uint8), cfg.E)
    assert np.array_equal(to_host(layer.perm["offsets"]), offsets)
    assert np.array_equal(to_host(layer.perm["dest_rows"]), dest)
    assert np.array_equal(to_host(layer.perm["sorted_token_ids"]), stok)

    rng = np.random.default_rng(cfg.seed)
    R, T, H, F, E = cfg.R, cfg.T, cfg.H, cfg.F, cfg.E
    rows, e_of = [], []
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            pick = {lo, (lo + hi) // 2, hi - 1}
            pick.update(int(rng.integers(m0, min(hi, m0 + 256))) for m0 in range(lo, hi, 256))
            for r in sorted(pick):
                rows.append(r)
                e_of.append(e)
    rows = np.array(rows)
    toks = stok[rows]
    sel_t = torch.from_numpy(toks.astype(np.int64)).cuda()
    codes_t = to_host(layer.xq.codes[sel_t])
    # the token rows' scales, from the k-step-major layout [H / 128][T][4]
    sc = to_host(layer.xq.scales)
    b = np.arange(H // 32)
    xq_host = ({int(t): codes_t[i] for i, t in enumerate(toks)},
               {int(t): sc[((b // 4) * T + int(t)) * 4 + (b % 4)] for t in toks})
    ws = to_host(layer.ws_ffn)
    y_rows = f64(to_host(layer.y_perm[torch.from_numpy(rows.astype(np.int64)).cuda()]))
    log(f"[gpu] full-size mxfp8 {name}: checking {rows.size} grouped rows")
    flips = _check_rows("routed", toks, rows, e_of, xq_host, I.x[toks], I.w_gate, I.w_up, I.w_down, ws,
                        E, R, H, F, y_rows, rng)
    log(f"[gpu]   {flips} sampled h codes differ from the exact h's quantization (all within the bound)")

    # shared expert: the token rows themselves through one dense MXFP8 FFN
    sample = rng.choice(T, size=min(T, 24), replace=False)
    if cfg.Fs:
        wss = to_host(layer.ws_shared)
        ys = f64(to_host(layer.y_shared[torch.from_numpy(sample.astype(np.int64)).cuda()]))
        xq_s = ({int(t): to_host(layer.xq.codes[int(t)]) for t in sample},
                {int(t): sc[((b // 4) * T + int(t)) * 4 + (b % 4)] for t in sample})
        _check_rows("shared", [int(t) for t in sample], sample, [0] * sample.size, xq_s, I.x[sample],
                    I.ws_gate, I.ws_up, I.ws_down, wss, 1, T, H, cfg.Fs, ys, rng)

    # y on a token sample touching every expert: the combine of the kernel's own rows
    tok_s = set(sample.tolist())
    for e in range(E):
        hit = np.nonzero((ids_o == e).any(axis=1))[0]
        if hit.size:
            tok_s.add(int(hit[rng.integers(hit.size)]))
    tok_s = np.array(sorted(tok_s))
    dr = dest[tok_s]
    yp = f64(to_host(layer.y_perm[torch.from_numpy(dr.reshape(-1).astype(np.int64)).cuda()])).reshape(
        tok_s.size, cfg.k, H)
    wts = w_g[tok_s][:, :, None].astype(np.float64)
    y_ref = (wts * yp).sum(axis=1)
    scale = (wts * np.abs(yp)).sum(axis=1)
    if cfg.Fs:
        ysh = f64(to_host(layer.y_shared[torch.from_numpy(tok_s.astype(np.int64)).cuda()]))
        y_ref += ysh
        scale += np.abs(ysh)
    y_g = f64(to_host(layer.y[torch.from_numpy(tok_s.astype(np.int64)).cuda()]))
    # fp32 sums of at most k + 1 terms (k 2^-24 of the terms' magnitudes), then one
    # bf16 rounding (2^-8 relative)
    assert (np.abs(y_g - y_ref) <= 2.0 ** -8 * np.abs(y_ref) + 2.0 ** -20 * scale + 1e-30).all()
    log(f"[gpu] full-size mxfp8 {name}: y on {tok_s.size} tokens matches the combine of the expert outputs")
