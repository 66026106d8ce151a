"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Bars (bf16 layers): routing and permutation bit-exact; gate weights within
weight_tol; y_perm per expert group and y within 2e-2 * max|oracle|.  fp32
layer: 1e-4 * max|oracle| (fp32 accumulation over K <= 512 rounds at ~1e-6).
Inputs are the seeded generator's; expected values come only from oracle/."""
import numpy as np
import pytest
import torch

import moegen
import oracle
import paper_2606_21712_amd as moe
from tests.gpu_util import f64, log, rel_max_err, split_budgets, to_dev, to_host, weight_tol

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4


def small(name, **kw):
    return moegen.MoEConfig(name, **kw)


# Reduced shapes of the five workloads: several 256-row m-tiles per expert with a
# ragged tail, ragged feature (F % 128) and hidden (H % 256) tails.
CASES = {
    "tiny_f32": moegen.CONFIGS["tiny"],
    "mixtral_small": small("mixtral_small", T=1500, H=576, E=8, k=2, F=320, seed=11),
    "zipf_small": small("zipf_small", T=2048, H=256, E=8, k=2, F=256, seed=12, routing="zipf"),
    "deepseek_small": small("deepseek_small", T=512, H=448, E=64, k=8, F=192, Fs=192, seed=13),
    "memc_small": small("memc_small", T=4096, H=256, E=64, k=4, F=256, seed=14, routing="lognormal",
                        pinned_small=(1, 17, 31)),
    "uniform_router": small("uniform_router", T=300, H=128, E=8, k=3, F=128, seed=15, routing="uniform"),
    "k1": small("k1", T=700, H=128, E=6, k=1, F=192, seed=16),
    "k_eq_E": small("k_eq_E", T=260, H=64, E=4, k=4, F=64, seed=17),
    "T1": small("T1", T=1, H=64, E=8, k=2, F=64, seed=18),
    "H64_f32": small("H64_f32", T=333, H=64, E=5, k=2, F=64, seed=19, dtype="f32"),
    # the largest expert count: most groups empty or a few rows
    "e256_small": small("e256_small", T=300, H=128, E=256, k=8, F=192, seed=23),
    # few down-projection tiles and a long k (224 steps of 64)
    "longk_small": small("longk_small", T=1024, H=256, E=8, k=2, F=4096, seed=20),
}


_INPUTS = {}


def inputs(name):
    if name not in _INPUTS:
        _INPUTS[name] = moegen.make_inputs(CASES[name])
    return _INPUTS[name]


def run_layer(I, renormalize=1, gather=False):
    c = I.cfg
    dt = torch.float32 if c.dtype == "f32" else torch.bfloat16
    layer = moe.MoELayer(c.T, c.H, c.E, c.k, c.F, c.Fs, dtype=dt, gather=gather)
    shared = (to_dev(I.ws_gate), to_dev(I.ws_up), to_dev(I.ws_down)) if c.Fs else (None, None, None)
    layer.run(to_dev(I.x), to_dev(I.logits), to_dev(I.w_gate), to_dev(I.w_up), to_dev(I.w_down),
              *shared, renormalize=renormalize)
    torch.cuda.synchronize()
    out = dict(ids=to_host(layer.topk_ids), w=to_host(layer.topk_weights),
               y_perm=to_host(layer.y_perm), y=to_host(layer.y))
    out.update({k: to_host(v) for k, v in layer.perm.items() if v is not None})
    if c.Fs:
        out["y_shared"] = to_host(layer.y_shared)
    return out


def oracle_layer(I, renormalize=1):
    c = I.cfg
    sh = (I.ws_gate, I.ws_up, I.ws_down) if c.Fs else (None, None, None)
    return oracle.layer(I.x, I.logits, c.k, I.w_gate, I.w_up, I.w_down, renormalize, *sh)


def _random_cases(n=8, seed=2026):
    """Seeded random shapes within the ABI's limits (H, F multiples of 64): odd
    expert counts, k from 1 to min(E, 8), every routing generator, an optional
    shared expert."""
    rng = np.random.default_rng(seed)
    out = {}
    for i in range(n):
        E = int(rng.choice([1, 2, 3, 5, 8, 13, 32, 64]))
        k = int(rng.integers(1, min(E, 8) + 1))
        T = int(rng.integers(1, 2500))
        H = 64 * int(rng.integers(1, 13))
        F = 64 * int(rng.integers(1, 9))
        Fs = int(rng.choice([0, 0, 128]))
        # the exact-count generators need every count <= T: skewed loads only for k <= 2
        skew = str(rng.choice(["router", "zipf", "lognormal"]))
        routing = skew if E >= 4 and k <= 2 and T * k >= 4 * E else "router"
        out[f"rand{i}"] = small(f"rand{i}", T=T, H=H, E=E, k=k, F=F, Fs=Fs, seed=100 + i, routing=routing)
    return out


RANDOM_CASES = _random_cases()
CASES.update(RANDOM_CASES)


@pytest.mark.parametrize("name", list(CASES))
def test_layer_parity(name):
    I = inputs(name)
    c = I.cfg
    # the random shapes alternate between the grouped-copy and the gather path
    gather = name in RANDOM_CASES and int(name[4:]) % 2 == 1
    log(f"[gpu] layer parity {name}: T={c.T} H={c.H} E={c.E} k={c.k} F={c.F} Fs={c.Fs} {c.dtype} "
        f"routing={c.routing} gather={gather}")
    g = run_layer(I, gather=gather)
    o = oracle_layer(I)
    # routing and permutation: bit-exact
    assert np.array_equal(g["ids"], o["ids"])
    assert np.abs(g["w"] - o["w"]).max() <= weight_tol(c.k, c.E)
    for key in ("counts", "offsets", "dest_rows", "sorted_token_ids"):
        assert np.array_equal(g[key], o[key]), key
    if not gather:
        assert np.array_equal(g["x_perm"], o["x_perm"])
    tol = F32_TOL if c.dtype == "f32" else BF16_TOL
    # y_perm, per expert group (an error confined to a tiny group must not hide)
    yp = f64(g["y_perm"])
    for e in range(c.E):
        lo, hi = o["offsets"][e], o["offsets"][e + 1]
        if hi > lo:
            err = rel_max_err(yp[lo:hi], o["y_perm"][lo:hi])
            assert err <= tol, (e, hi - lo, err)
    if c.Fs:
        assert rel_max_err(f64(g["y_shared"]), o["y_shared"]) <= tol
    err = rel_max_err(f64(g["y"]), o["y"])
    log(f"[gpu]   max|dy|/max|y| = {err:.3e}")
    assert err <= tol


# Group sizes around the m-tile edges: an expert's last m-tile holds up to 320 rows
# (256 + 64), so 257..320 rows make one tile, 321 two, 576 two (256 + 320), 577
# three; plus 1, 64, 65 and an empty expert.
EDGE_COUNTS = [256, 257, 300, 320, 321, 512, 576, 577, 1, 64, 65, 0]


def edge_count_inputs(H=256, F=320, seed=22):
    """k = 1 inputs whose routing gives exactly EDGE_COUNTS rows per expert: each
    token's logit for its expert is 8 above the others (router noise is ~0.3)."""
    E = len(EDGE_COUNTS)
    T = sum(EDGE_COUNTS)
    I = moegen.make_inputs(small("edge_counts", T=T, H=H, E=E, k=1, F=F, seed=seed))
    rng = np.random.default_rng(seed)
    expert = rng.permutation(np.repeat(np.arange(E), EDGE_COUNTS))
    logits = I.logits.copy()
    logits[np.arange(T), expert] += np.float32(8.0)
    I.logits = logits
    return I, expert


def test_last_m_tile_extra_rows():
    """Groups whose sizes sit on the m-tile edges (including the 320-row last tile)
    against the oracle, through the copy and the gather paths (bitwise equal)."""
    I, expert = edge_count_inputs()
    c = I.cfg
    log(f"[gpu] edge group sizes {EDGE_COUNTS}: T={c.T} H={c.H} F={c.F}")
    o = oracle_layer(I)
    assert np.array_equal(o["counts"], np.array(EDGE_COUNTS))
    assert np.array_equal(o["ids"][:, 0], expert)
    g = run_layer(I)
    b = run_layer(I, gather=True)
    assert np.array_equal(g["ids"], o["ids"])
    assert np.array_equal(g["offsets"], o["offsets"])
    yp = f64(g["y_perm"])
    for e in range(c.E):
        lo, hi = o["offsets"][e], o["offsets"][e + 1]
        if hi > lo:
            err = rel_max_err(yp[lo:hi], o["y_perm"][lo:hi])
            assert err <= BF16_TOL, (e, hi - lo, err)
    assert rel_max_err(f64(g["y"]), o["y"]) <= BF16_TOL
    assert np.array_equal(g["y_perm"], b["y_perm"])
    assert np.array_equal(g["y"], b["y"])


def check_tail_split(y_split, y_whole, r, label):
    """A run whose down projection cut r tail tiles along k against one that ran every
    tile whole: at most r tiles' elements differ, each by fp32 reassociation of the
    pieces' partial sums plus one bf16 rounding (2^-7 relative, and 2^-16 of the
    largest output for values that cancel)."""
    a, b = f64(y_split), f64(y_whole)
    n_diff = int((y_split != y_whole).sum())
    log(f"[gpu]   {label}: {n_diff} elements differ from the unsplit run (limit {r * 256 * 256})")
    assert n_diff <= r * 256 * 256
    assert (np.abs(a - b) <= 2.0 ** -7 * np.abs(b) + 2.0 ** -16 * np.abs(b).max()).all()


def test_down_projection_tail_split():
    """The last, partly filled round of down-projection tiles cut along k, reached at a
    small size by planning the grid for fewer compute units: tiles outside the tail
    keep their bits, tail tiles move only by reassociation, y_perm stays within the
    oracle bar per expert group."""
    c = small("tail_split", T=2048, H=512, E=8, k=2, F=2048, seed=21)
    I = moegen.make_inputs(c)
    o = oracle_layer(I)
    picks, plain = split_budgets(o["offsets"], c.H, c.F // 64, 64)
    assert len(picks) >= 2 and plain is not None, (picks, plain)
    try:
        log(f"[gpu] tail split reference: budget {plain}, no split")
        moe.set_cu_budget(plain)
        base = run_layer(I)
        for b, r, s in picks:
            log(f"[gpu] tail split: budget {b}, {r} tail tiles in {s} pieces")
            moe.set_cu_budget(b)
            g = run_layer(I)
            check_tail_split(g["y_perm"], base["y_perm"], r, f"budget {b}")
            yp = f64(g["y_perm"])
            for e in range(c.E):
                lo, hi = o["offsets"][e], o["offsets"][e + 1]
                if hi > lo:
                    assert rel_max_err(yp[lo:hi], o["y_perm"][lo:hi]) <= BF16_TOL, (b, e)
            assert rel_max_err(f64(g["y"]), o["y"]) <= BF16_TOL
    finally:
        moe.set_cu_budget(0)


@pytest.mark.parametrize("name", ["tiny_f32", "mixtral_small", "zipf_small", "deepseek_small", "memc_small",
                                  "uniform_router", "T1", "longk_small", "H64_f32"])
def test_gather_path_matches_grouped_path(name):
    """moe_grouped_ffn_gather gives bit-for-bit the y_perm of moe_grouped_ffn on x_perm,
    and the layer output stays within the oracle bar."""
    I = inputs(name)
    c = I.cfg
    log(f"[gpu] gather path {name}")
    a = run_layer(I)
    b = run_layer(I, gather=True)
    assert np.array_equal(a["y_perm"], b["y_perm"])
    assert np.array_equal(a["y"], b["y"])
    o = oracle_layer(I)
    assert rel_max_err(f64(b["y"]), o["y"]) <= (F32_TOL if c.dtype == "f32" else BF16_TOL)


@pytest.mark.parametrize("name", ["mixtral_small", "deepseek_small"])
def test_route_without_renormalize(name):
    I = inputs(name)
    c = I.cfg
    log(f"[gpu] route renormalize=0 {name}")
    ids, w = moe.moe_route(to_dev(I.logits), c.k, 0)
    torch.cuda.synchronize()
    oi, ow = oracle.route(I.logits, c.k, 0)
    assert np.array_equal(to_host(ids), oi)
    assert np.abs(to_host(w) - ow).max() <= weight_tol(c.k, c.E)


def test_route_ties_and_signed_zero():
    """Integer-valued logits force ties (lower id wins); -0.0 equals +0.0."""
    rng = np.random.default_rng(5)
    # segment widths 1, 2, 4, 8, 16, 32 lanes per token; odd and even values per lane
    for (T, E, k) in [(1000, 8, 2), (513, 64, 8), (77, 256, 16), (64, 3, 3), (200, 100, 7),
                      (300, 16, 4), (300, 32, 5), (150, 129, 9), (90, 40, 6)]:
        logits = rng.integers(-2, 3, size=(T, E)).astype(np.float32)
        logits[::7, 0] = -0.0
        logits[::5, 1] = 0.0
        log(f"[gpu] route ties T={T} E={E} k={k}")
        for renorm in (0, 1):
            ids, w = moe.moe_route(to_dev(logits), k, renorm)
            torch.cuda.synchronize()
            oi, ow = oracle.route(logits, k, renorm)
            assert np.array_equal(to_host(ids), oi)
            assert np.abs(to_host(w) - ow).max() <= weight_tol(k, E)


# T * k up to 16 units of 1024 assignments runs the single-block permute, more
# the count / scan / rank kernels: both sides of the boundary, E up to 256.
@pytest.mark.parametrize("T,E,k", [(3000, 256, 5), (3277, 256, 5), (16384, 16, 1), (16385, 16, 1),
                                   (20000, 8, 2)])
def test_permute_direct(T, E, k):
    """Permute on random distinct expert sets per token against the oracle, bit-exact."""
    rng = np.random.default_rng(6 + T)
    H = 128
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    x = moegen.round_bf16(rng.standard_normal((T, H)).astype(np.float32))
    log(f"[gpu] permute E={E} T={T} k={k} ({(T * k + 1023) // 1024} units)")
    out = moe.moe_permute(to_dev(ids), to_dev(x), E)
    torch.cuda.synchronize()
    oc, oo, od, os_, oxp = oracle.permute(ids, x, E)
    assert np.array_equal(to_host(out["counts"]), oc)
    assert np.array_equal(to_host(out["offsets"]), oo)
    assert np.array_equal(to_host(out["dest_rows"]), od)
    assert np.array_equal(to_host(out["sorted_token_ids"]), os_)
    assert np.array_equal(to_host(out["x_perm"]), oxp)


def test_combine_direct():
    """Combine alone on random y_perm / weights / shared rows, bf16 and fp32.  Per
    element, |gpu - oracle| <= 2^-8 * (sum_j |w_j y_j| + |y_s|): one bf16 rounding
    (2^-9) plus fp32 summation of at most 17 terms (fp32 output: far inside)."""
    rng = np.random.default_rng(7)
    # k = 1, 2, 4, 8 take the kernels with every row's loads in flight, other k the
    # generic one; H = 4160 needs two passes of the widest unroll, with a ragged tail.
    # Batches of 8192 tokens and more cut each row into parts of one wavefront each:
    # 4 parts of 112 vectors (H = 3584, a ragged pass per lane), 8 parts (H = 8192),
    # 4 parts in fp32 (H = 1024).
    for (T, k, H, shared, bf16) in [(999, 4, 192, True, True), (64, 16, 64, False, True),
                                    (1, 1, 128, True, True), (77, 8, 576, True, True),
                                    (50, 2, 4160, False, True), (33, 1, 1024, True, True),
                                    (41, 3, 320, True, True), (90, 8, 704, True, False),
                                    (37, 2, 4160, True, False), (20, 5, 64, False, False),
                                    (8192, 4, 3584, True, True), (8192, 2, 8192, False, True),
                                    (9000, 1, 1024, True, False)]:
        R = T * k
        cast = moegen.round_bf16 if bf16 else (lambda a: a)
        yp = cast(rng.standard_normal((R, H)).astype(np.float32))
        dest = rng.permutation(R).reshape(T, k).astype(np.int32)
        w = rng.random((T, k)).astype(np.float32)
        ys = cast(rng.standard_normal((T, H)).astype(np.float32)) if shared else None
        log(f"[gpu] combine T={T} k={k} H={H} shared={shared} bf16={bf16}")
        y = moe.moe_combine(to_dev(yp), to_dev(dest), to_dev(w), None if ys is None else to_dev(ys))
        torch.cuda.synchronize()
        ref = oracle.combine(yp, dest, w, ys)
        mag = np.zeros((T, H))
        for j in range(k):
            mag += np.abs(w[:, j:j + 1].astype(np.float64) * f64(yp)[dest[:, j]])
        if ys is not None:
            mag += np.abs(f64(ys))
        assert (np.abs(f64(to_host(y)) - ref) <= 2.0 ** -8 * mag + 1e-30).all()


def test_zero_tokens_is_a_noop():
    log("[gpu] T=0")
    e = torch.empty(0, 8, device="cuda")
    ids, w = moe.moe_route(e, 2)
    assert ids.shape == (0, 2)
    torch.cuda.synchronize()


def test_deterministic():
    I = inputs("memc_small")
    log("[gpu] determinism memc_small x2")
    a = run_layer(I)
    b = run_layer(I)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
