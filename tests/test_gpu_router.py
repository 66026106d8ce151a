"""GPU parity of moe_router_topk (router GEMM + gate) against the fp64 oracle.

The gate decides integers (expert ids) from floating-point logits, so the
decision is checked in the kernel's own precision: the kernel's logits must lie
within the matrix cores' accumulation bound of the exact x . w_router, and its
ids and weights must be exactly the oracle's routing of those same logits.
Tokens whose exact top-k margins exceed twice the bound must also match the
oracle's routing of the exact logits; integer-valued operands make the logits
exact and full of ties, and then every token must match."""
import numpy as np
import pytest
import torch

import moegen
import oracle
import paper_2606_21712_amd as moe
from tests.gpu_util import log, to_dev, to_host, weight_tol

pytestmark = pytest.mark.gpu

# bf16 MFMA accumulation error, as a fraction of sum_h |x_h w_h|: measured at 1.0e-7
# for K = 1024 on gfx950 (fp32-accurate); the bound allows for K up to 7168 and more.
ACC = 2.0 ** -18


def run(x, w, k, renorm=1):
    T, H = x.shape
    E = w.shape[0]
    logits = torch.empty((T, E), dtype=torch.float32, device="cuda")
    ids, wt = moe.moe_router_topk(to_dev(x), to_dev(w), k, renorm, logits=logits)
    torch.cuda.synchronize()
    return to_host(logits), to_host(ids), to_host(wt)


def check(x, w, k, renorm=1, exact_ties=False):
    lg, ids, wt = run(x, w, k, renorm)
    return check_outputs(x, w, k, renorm, lg, ids, wt, exact_ties)


def check_outputs(x, w, k, renorm, lg, ids, wt, exact_ties=False):
    """The kernel's logits, ids and weights for the token rows x (all of them, or a
    sample: each token is checked on its own) against the oracle."""
    exact = oracle.router_logits(x, w)
    bound = ACC * (np.abs(oracle.moe_oracle._f64(x)) @ np.abs(oracle.moe_oracle._f64(w)).T) + 1e-30
    assert (np.abs(lg.astype(np.float64) - exact) <= bound).all()
    # the decision, in the kernel's precision: exactly the gate on the kernel's logits
    o_ids, o_w = oracle.route(lg, k, renorm)
    assert np.array_equal(ids, o_ids)
    assert np.abs(wt - o_w).max() <= weight_tol(k, w.shape[0])
    # against the exact logits: every token whose margins clear twice the bound
    e_ids, _ = oracle.route(exact, k, renorm)
    srt = -np.sort(-exact, axis=1)
    gaps = np.abs(np.diff(srt[:, : min(k + 1, exact.shape[1])], axis=1))
    safe = (gaps > 2 * bound.max(axis=1, keepdims=True)).all(axis=1)
    if exact_ties:
        safe[:] = True
    assert np.array_equal(ids[safe], e_ids[safe])
    return safe.mean()


# With H % 128 != 0 the per-wavefront kernel runs: T >= 65536 and >= 131072 give a
# wavefront 32 and 64 tokens (on 256 compute units).  H % 128 == 0 with T >= 16384
# runs the LDS-staged kernel (k-slices of 256 where H % 256 == 0, else of 128): 1
# to 4 expert blocks, 4, 8 and 16 selection slots, ragged last block of 64 tokens;
# below 16384 tokens the split-k kernel.
@pytest.mark.parametrize("T,E,k,H", [(1000, 8, 2, 256), (333, 64, 8, 448), (77, 3, 3, 64), (500, 40, 6, 4096),
                                     (129, 16, 4, 192), (257, 33, 16, 320), (5, 64, 1, 128),
                                     (70001, 20, 3, 64), (140007, 64, 4, 192), (40003, 64, 4, 128),
                                     (16384, 8, 2, 768), (20000, 64, 8, 256), (17000, 40, 4, 512),
                                     (33333, 20, 16, 1024), (20011, 48, 8, 384), (16391, 61, 8, 1152)])
def test_router_random(T, E, k, H):
    rng = np.random.default_rng(T + E + H)
    x = moegen.round_bf16(rng.standard_normal((T, H)).astype(np.float32))
    w = moegen.round_bf16((rng.standard_normal((E, H)) * 0.04).astype(np.float32))
    for renorm in (1, 0):
        log(f"[gpu] router T={T} E={E} k={k} H={H} renorm={renorm}")
        frac = check(x, w, k, renorm)
        assert frac > 0.95


def test_router_exact_ties():
    """Small-integer operands: fp32 accumulation is exact, ties abound, and every token
    must match the oracle (ties to the lower expert id)."""
    rng = np.random.default_rng(44)
    T, E, k, H = 300, 24, 5, 192
    x = moegen.round_bf16(rng.integers(-2, 3, (T, H)).astype(np.float32))
    w = moegen.round_bf16(rng.integers(-1, 2, (E, H)).astype(np.float32))
    log("[gpu] router with exact, tied logits")
    lg, ids, _ = run(x, w, k)
    assert np.array_equal(lg.astype(np.float64), oracle.router_logits(x, w))
    check(x, w, k, exact_ties=True)


@pytest.mark.parametrize("name", ["mixtral4k", "deepseek"])
def test_router_workload(name):
    """The Mixtral- and DeepSeek-shaped layers with the generator's router matrix."""
    I = moegen.make_inputs(name, with_weights=False)
    c = I.cfg
    log(f"[gpu] router {name} T={c.T} H={c.H} E={c.E} k={c.k}")
    frac = check(I.x, I.extra["w_router"], c.k)
    log(f"[gpu]   {frac:.4f} of the tokens checked against the exact logits' routing")
    assert frac > 0.95          # 64 experts, top-8: ~97% of tokens clear twice the bound


@pytest.mark.parametrize("H,sizes", [(640, (100, 600, 1100, 2100)), (1024, (100, 300)), (192, (100, 600, 1100, 2100))])
def test_router_batch_size_invariant(H, sizes):
    """The same tokens routed in batches of different sizes get bitwise-identical
    logits, ids and weights: every kernel variant (k split four ways for small
    batches, LDS-staged router matrix, 16 / 32 / 64 tokens per wavefront) adds the
    products in the same k order.  A budget of 4 compute units puts the variants'
    switch points at small T: with H = 640 the sizes run split-k, then the
    LDS-staged kernel with k-slices of 128; with H = 1024 split-k, then the
    LDS-staged kernel with slices of 256; H = 192 (H % 128 != 0) runs one k chain in
    the per-wavefront kernel at 16, 16, 32 and 64 tokens per wavefront."""
    rng = np.random.default_rng(H)
    E, k = 64, 4
    x = moegen.round_bf16(rng.standard_normal((max(sizes), H)).astype(np.float32))
    w = moegen.round_bf16((rng.standard_normal((E, H)) * 0.04).astype(np.float32))
    n = min(sizes)
    moe.set_cu_budget(4)
    try:
        ref = None
        for T in sizes:
            log(f"[gpu] router batch-size invariance H={H} T={T}")
            lg, ids, wt = run(x[:T], w, k)
            got = (lg[:n], ids[:n], wt[:n])
            if ref is None:
                ref = got
            else:
                for a, b in zip(got, ref):
                    assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                                          b.view(np.uint32) if b.dtype == np.float32 else b), (H, T)
    finally:
        moe.set_cu_budget(0)


def test_router_fullsize_memconstrained():
    """The memory-constrained workload's router at full size (131072 tokens, H 4096,
    64 experts, top-4: the LDS-staged kernel with k-slices of 256 on every compute
    unit), checked on 4096 sampled tokens and the last 64 (the ragged end)."""
    I = moegen.make_inputs("memconstrained", with_weights=False)
    c = I.cfg
    w = I.extra["w_router"]
    log(f"[gpu] router full size memconstrained T={c.T} H={c.H} E={c.E} k={c.k}")
    lg, ids, wt = run(I.x, w, c.k)
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([rng.choice(c.T, 4096, replace=False), np.arange(c.T - 64, c.T)]))
    frac = check_outputs(I.x[rows], w, c.k, 1, lg[rows], ids[rows], wt[rows])
    log(f"[gpu]   {frac:.4f} of the sampled tokens checked against the exact logits' routing")
    assert frac > 0.9
