"""GPU parity at the workloads' full sizes, in the configuration bench.py times.

Routing and permutation are compared bit-exactly on every token.  The FFN and
the layer output are compared on samples the oracle computes row by row: for
every expert group its first, middle and last rows of y_perm (so the 1-, 17- and
31-row groups of the memory-constrained workload are all covered) and one random
row of every 64-row window of the group, each row in full, so every n-tile of
every m-tile is checked: an expert of more than one m-tile has m-tiles of 160 to
320 rows, each holding at least one whole window.  Then the final y of a token sample that touches every expert.
Bars as in test_gpu_parity."""
import numpy as np
import pytest
import torch

import moegen
import oracle
import paper_2606_21712_amd as moe
from tests.gpu_util import f64, log, rel_max_err, to_dev, to_host, weight_tol

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def _sample_tokens(ids, E, n_extra, rng):
    """A token sample that contains, for every expert, at least one token routed to it."""
    toks = set()
    for e in range(E):
        hit = np.nonzero((ids == e).any(axis=1))[0]
        if hit.size:
            toks.add(int(hit[rng.integers(hit.size)]))
    toks.update(rng.choice(ids.shape[0], size=n_extra, replace=False).tolist())
    return np.array(sorted(toks))


@pytest.mark.parametrize("name", ["mixtral4k", "mixtral32k_zipf", "deepseek", "memconstrained"])
def test_full_size_layer(name):
    cfg = moegen.CONFIGS[name]
    log(f"[gpu] full-size {name}: generating T={cfg.T} H={cfg.H} E={cfg.E} k={cfg.k} F={cfg.F} Fs={cfg.Fs}")
    I = moegen.make_inputs(cfg)
    shared_dev = (to_dev(I.ws_gate), to_dev(I.ws_up), to_dev(I.ws_down)) if cfg.Fs else (None, None, None)
    layer = moe.MoELayer(cfg.T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs)
    log(f"[gpu] full-size {name}: running the layer")
    layer.run(to_dev(I.x), to_dev(I.logits), to_dev(I.w_gate), to_dev(I.w_up), to_dev(I.w_down),
              *shared_dev, renormalize=cfg.renormalize)
    torch.cuda.synchronize()

    # routing and permutation, every token, bit-exact
    ids_g, w_g = to_host(layer.topk_ids), to_host(layer.topk_weights)
    ids_o, w_o = oracle.route(I.logits, cfg.k, cfg.renormalize)
    assert np.array_equal(ids_g, ids_o)
    assert np.abs(w_g - w_o).max() <= weight_tol(cfg.k, cfg.E)
    counts, offsets, dest, stok, _ = oracle.permute(ids_o, np.zeros((cfg.T, 1), np.uint8), cfg.E)
    assert np.array_equal(to_host(layer.perm["counts"]), counts)
    assert np.array_equal(to_host(layer.perm["offsets"]), offsets)
    assert np.array_equal(to_host(layer.perm["dest_rows"]), dest)
    assert np.array_equal(to_host(layer.perm["sorted_token_ids"]), stok)
    if I.target_counts is not None:
        assert np.array_equal(counts, I.target_counts)

    # x_perm on sampled rows, y_perm per group on first / middle / last rows
    rows = []
    rng_rows = np.random.default_rng(cfg.seed + 100)
    for e in range(cfg.E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            pick = {lo, (lo + hi) // 2, hi - 1}
            for m0 in range(lo, hi, 64):
                pick.add(int(rng_rows.integers(m0, min(hi, m0 + 64))))
            rows += sorted(pick)
    rows = np.array(rows)
    xp = to_host(layer.perm["x_perm"][torch.from_numpy(rows).cuda()])
    assert np.array_equal(xp, I.x[stok[rows]])
    yp = f64(to_host(layer.y_perm[torch.from_numpy(rows).cuda()]))
    log(f"[gpu] full-size {name}: oracle on {rows.size} y_perm rows")
    for e in range(cfg.E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        sel = (rows >= lo) & (rows < hi)
        if sel.any():
            ref = oracle.ffn_rows(I.x[stok[rows[sel]]], e, I.w_gate, I.w_up, I.w_down)
            err = rel_max_err(yp[sel], ref)
            assert err <= BF16_TOL, (e, hi - lo, err)

    # final y on a token sample touching every expert
    rng = np.random.default_rng(cfg.seed)
    toks = _sample_tokens(ids_o, cfg.E, 32, rng)
    log(f"[gpu] full-size {name}: oracle on {toks.size} tokens")
    sh = (I.ws_gate, I.ws_up, I.ws_down) if cfg.Fs else (None, None, None)
    _, _, y_ref, _ = oracle.token_outputs(toks, I.x, I.logits, cfg.k, I.w_gate, I.w_up, I.w_down,
                                          cfg.renormalize, *sh)
    y_g = f64(to_host(layer.y[torch.from_numpy(toks).cuda()]))
    err = rel_max_err(y_g, y_ref)
    log(f"[gpu] full-size {name}: max|dy|/max|y| = {err:.3e}")
    assert err <= BF16_TOL

    # the gather-fused grouped FFN reproduces the same layer bit for bit
    log(f"[gpu] full-size {name}: gather-fused path")
    y_first, yp_first = layer.y.clone(), layer.y_perm.clone()
    del layer
    g = moe.MoELayer(cfg.T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs, gather=True)
    g.run(to_dev(I.x), to_dev(I.logits), to_dev(I.w_gate), to_dev(I.w_up), to_dev(I.w_down),
          *shared_dev, renormalize=cfg.renormalize)
    torch.cuda.synchronize()
    assert torch.equal(g.y_perm, yp_first)
    assert torch.equal(g.y, y_first)
