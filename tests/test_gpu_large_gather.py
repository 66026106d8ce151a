"""The gather-fused grouped FFN with token rows of 2 GiB or more.

GEMM-1 of the default path reads each grouped row straight from x through
sorted_token_ids.  Below 2 GiB one buffer resource with 32-bit row offsets spans
x; from 2 GiB on, the loads take 64-bit per-lane row addresses.  Here x is
2.18 GB (266240 tokens x 4096 hidden, bf16), so the rows of the last ~5900
tokens start beyond byte 2^31.  Routing and grouping are bit-exact on every
token; y_perm equals the x_perm path bit for bit; the oracle checks one random
row of every 64-row window of every expert group (every m-tile holds one) and the rows of the last
tokens, each in full, against the bar of the bf16 layer."""
import numpy as np
import pytest
import torch

import moegen
import oracle
import paper_2606_21712_amd as moe
from tests.gpu_util import f64, log, rel_max_err, to_dev, to_host

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def test_gather_beyond_2gib():
    T, H, E, k, F = 266240, 4096, 8, 2, 128
    assert T * H * 2 >= 2 ** 31
    cfg = moegen.MoEConfig("large_gather", T=T, H=H, E=E, k=k, F=F, seed=31)
    log(f"[gpu] large gather: generating T={T} H={H} E={E} k={k} F={F} (x = {T * H * 2 / 2**30:.2f} GiB)")
    I = moegen.make_inputs(cfg)
    x = to_dev(I.x)
    wg, wu, wd = to_dev(I.w_gate), to_dev(I.w_up), to_dev(I.w_down)
    log("[gpu] large gather: route, permute (with x_perm), both grouped FFN paths")
    ids, w = moe.moe_route(to_dev(I.logits), k)
    perm = moe.moe_permute(ids, x, E)
    y_gather = moe.moe_grouped_ffn_gather(x, perm["sorted_token_ids"], perm["offsets"], wg, wu, wd)
    y_rows = moe.moe_grouped_ffn(perm["x_perm"], perm["offsets"], wg, wu, wd)
    torch.cuda.synchronize()
    assert torch.equal(y_gather.view(torch.int16), y_rows.view(torch.int16))
    del y_rows, perm["x_perm"]

    ids_o, _ = oracle.route(I.logits, k)
    assert np.array_equal(to_host(ids), ids_o)
    _, offsets, _, stok, _ = oracle.permute(ids_o, np.zeros((T, 1), np.uint8), E)
    assert np.array_equal(to_host(perm["offsets"]), offsets)
    assert np.array_equal(to_host(perm["sorted_token_ids"]), stok)

    rng = np.random.default_rng(5)
    rows = set()
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        for m0 in range(lo, hi, 64):                          # every m-tile holds a whole window
            rows.add(int(rng.integers(m0, min(hi, m0 + 64))))
    far = np.nonzero(stok >= T - 64)[0]                 # rows of the last tokens: offsets past 2^31
    rows.update(far.tolist())
    rows = np.array(sorted(rows))
    assert (stok[rows].astype(np.int64) * H * 2 >= 2 ** 31).any()
    yp = f64(to_host(y_gather[torch.from_numpy(rows).cuda()]))
    log(f"[gpu] large gather: oracle on {rows.size} y_perm rows")
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        sel = (rows >= lo) & (rows < hi)
        if sel.any():
            ref = oracle.ffn_rows(I.x[stok[rows[sel]]], e, I.w_gate, I.w_up, I.w_down)
            err = rel_max_err(yp[sel], ref)
            assert err <= BF16_TOL, (e, hi - lo, err)
