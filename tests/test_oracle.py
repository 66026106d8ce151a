"""The oracle against its pins, and every pin against a planted mistake in the oracle.

The planted mistakes are made on the CPU in copies of oracle functions; the
oracle module itself is never modified."""
import math

import numpy as np
import pytest

import oracle
from oracle import moe_oracle as O
from tests import pins


@pytest.fixture
def rng():
    return np.random.default_rng(1234)


# --------------------------------------------------------------------------- the oracle passes
def test_route_brute_force(rng):
    pins.check_route_brute(oracle.route, rng)


def test_route_matches_scipy_softmax(rng):
    pins.check_route_library(oracle.route, rng)


def test_route_invariants(rng):
    pins.check_route_invariants(oracle.route, rng)


def test_route_uniform_router():
    pins.check_route_uniform(oracle.route)


def test_route_signed_zero():
    pins.check_route_signed_zero(oracle.route)


def test_route_rejects_bad_input():
    with pytest.raises(ValueError):
        oracle.route(np.zeros((2, 3), np.float32), 4)
    with pytest.raises(ValueError):
        oracle.route(np.array([[np.nan, 0.0]], np.float32), 1)


def test_permute_brute_force(rng):
    pins.check_permute_brute(oracle.permute, rng)


def test_permute_invariants(rng):
    pins.check_permute_invariants(oracle.permute, rng)


def test_permute_special_cases():
    pins.check_permute_special(oracle.permute)


def test_ffn_brute_force(rng):
    pins.check_ffn_brute(oracle.swiglu_ffn, rng)


def test_ffn_silu_closed_form():
    pins.check_ffn_silu_values(oracle.dense_swiglu)


def test_layer_identical_experts(rng):
    pins.check_layer_identical_experts(oracle.layer, oracle.dense_swiglu, rng)


def test_layer_metamorphic(rng):
    pins.check_layer_metamorphic(oracle.layer, rng)


def test_combine(rng):
    pins.check_combine(oracle.combine, rng)


def test_hand_worked_layer():
    pins.check_hand_worked(oracle.layer)


def test_token_outputs_match_layer(rng):
    """The sampled-token path gives the same y as the whole-layer path."""
    T, H, F, E, k, Fs = 50, 8, 6, 5, 2, 3
    x = rng.standard_normal((T, H))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    wg, wu, wd = rng.standard_normal((E, F, H)), rng.standard_normal((E, F, H)), rng.standard_normal((E, H, F))
    sg, su, sd = rng.standard_normal((1, Fs, H)), rng.standard_normal((1, Fs, H)), rng.standard_normal((1, H, Fs))
    full = oracle.layer(x, logits, k, wg, wu, wd, 1, sg, su, sd)
    toks = np.array([0, 7, 7, 49, 13])
    ids, w, y, per = oracle.token_outputs(toks, x, logits, k, wg, wu, wd, 1, sg, su, sd)
    assert np.array_equal(ids, full["ids"][toks])
    assert np.allclose(y, full["y"][toks], rtol=1e-13, atol=1e-13)
    for i, t in enumerate(toks):
        for j in range(k):
            assert np.allclose(per[i, j], full["y_perm"][full["dest_rows"][t, j]], rtol=1e-13, atol=1e-13)


def test_bf16_inputs_are_upcast_exactly():
    bits = np.array([0x3F80, 0xBFC0, 0x0001, 0x7F7F], dtype=np.uint16)   # 1, -1.5, min subnormal, max
    v = O._f64(bits)
    assert v[0] == 1.0 and v[1] == -1.5 and v[2] == 2.0 ** -133
    assert v[3] == 255.0 * 2.0 ** 120                  # 0x7F7F: exponent 254, mantissa 127/128


# --------------------------------------------------------------------------- planted mistakes
def _route_ties_to_higher_id(logits, k, renormalize=1):
    L = O._f64(logits)
    T, E = L.shape
    order = np.lexsort((-np.broadcast_to(np.arange(E), (T, E)), -L), axis=1)
    ids = order[:, :k]
    sel = np.take_along_axis(L, ids, 1)
    p = np.exp(sel - sel[:, :1])
    den = p.sum(1, keepdims=True) if renormalize else np.exp(L - sel[:, :1]).sum(1, keepdims=True)
    return ids.astype(np.int32), p / den


def _route_no_renormalize(logits, k, renormalize=1):
    return O.route(logits, k, 0)


def _route_softmax_sign(logits, k, renormalize=1):
    ids, _ = O.route(logits, k, renormalize)
    L = O._f64(logits)
    sel = np.take_along_axis(L, ids.astype(np.int64), 1)
    p = np.exp(-(sel - sel[:, :1]))                    # wrong sign in the exponent
    den = p.sum(1, keepdims=True) if renormalize else np.exp(-(L - sel[:, :1])).sum(1, keepdims=True)
    return ids, p / den


def _route_ascending(logits, k, renormalize=1):
    ids, w = O.route(logits, k, renormalize)
    return ids[:, ::-1].copy(), w[:, ::-1].copy()       # slots in the wrong order


def _permute_unstable(ids, x, E):
    counts, offsets, dest, stok, xp = O.permute(ids, x, E)
    T, k = np.asarray(ids).shape
    flat = np.asarray(ids).reshape(-1)
    order = np.argsort(-np.arange(flat.size), kind="stable")
    order = order[np.argsort(flat[order], kind="stable")]       # descending tokens in a group
    stok = order // k
    dest = np.empty(flat.size, np.int64)
    dest[order] = np.arange(flat.size)
    return counts, offsets, dest.reshape(T, k).astype(np.int32), stok.astype(np.int32), np.asarray(x)[stok]


def _permute_inclusive_offsets(ids, x, E):
    counts, offsets, dest, stok, xp = O.permute(ids, x, E)
    return counts, np.concatenate([np.cumsum(counts), [offsets[-1]]]).astype(np.int32), dest, stok, xp


def _dense_swiglu_swapped(x, wg, wu, wd):
    return O.dense_swiglu(x, wu, wg, wd)                 # gate and up exchanged


def _dense_swiglu_sigmoid(x, wg, wu, wd):
    X = O._f64(x)
    g = X @ O._f64(wg).T
    u = X @ O._f64(wu).T
    return (1.0 / (1.0 + np.exp(-g)) * u) @ O._f64(wd).T   # sigmoid instead of silu


def _dense_swiglu_transposed_down(x, wg, wu, wd):
    X = O._f64(x)
    a = O._silu(X @ O._f64(wg).T) * (X @ O._f64(wu).T)
    wd = O._f64(wd)
    return a @ wd.reshape(wd.shape[1], wd.shape[0])      # wrong reading of W_down's layout


def _swiglu_ffn_from(dense):
    def f(x_perm, offsets, wg, wu, wd):
        offsets = np.asarray(offsets, np.int64)
        y = np.zeros((int(offsets[-1]), wd.shape[1]))
        for e in range(len(offsets) - 1):
            lo, hi = offsets[e], offsets[e + 1]
            if hi > lo:
                y[lo:hi] = dense(x_perm[lo:hi], wg[e], wu[e], wd[e])
        return y
    return f


def _swiglu_ffn_off_by_one(x_perm, offsets, wg, wu, wd):
    offsets = np.asarray(offsets, np.int64)
    y = np.zeros((int(offsets[-1]), wd.shape[1]))
    for e in range(len(offsets) - 1):
        lo, hi = offsets[e], offsets[e + 1]
        if hi > lo:
            y[lo:hi] = O.dense_swiglu(x_perm[lo:hi], wg[min(e + 1, len(wg) - 1)], wu[e], wd[e])
    return y


def _combine_dropped_weight(y_perm, dest, w, y_shared=None):
    return O.combine(y_perm, dest, np.ones_like(np.asarray(w)), y_shared)


def _combine_last_slot_dropped(y_perm, dest, w, y_shared=None):
    dest = np.asarray(dest)
    w = np.asarray(w, np.float64).copy()
    if dest.shape[1] > 1:
        w[:, -1] = 0
    return O.combine(y_perm, dest, w, y_shared)


def _layer_with(route=None, permute=None, dense=None, combine=None):
    route = route or O.route
    permute = permute or O.permute
    dense = dense or O.dense_swiglu
    combine = combine or O.combine

    def layer(x, logits, k, wg, wu, wd, renormalize=1, sg=None, su=None, sd=None):
        E = wg.shape[0]
        ids, w = route(logits, k, renormalize)
        counts, offsets, dest, stok, xp = permute(ids, x, E)
        yp = _swiglu_ffn_from(dense)(xp, offsets, wg, wu, wd)
        return dict(ids=ids, w=w, y=combine(yp, dest, w), y_perm=yp)
    return layer


MUTANTS = [
    ("route ties to higher id", lambda r: pins.check_route_brute(_route_ties_to_higher_id, r)),
    ("route ties to higher id (uniform)", lambda r: pins.check_route_uniform(_route_ties_to_higher_id)),
    ("route ignores renormalize", lambda r: pins.check_route_library(_route_no_renormalize, r)),
    ("route softmax sign", lambda r: pins.check_route_brute(_route_softmax_sign, r)),
    ("route slot order", lambda r: pins.check_route_invariants(_route_ascending, r)),
    ("permute unstable", lambda r: pins.check_permute_brute(_permute_unstable, r)),
    ("permute unstable (invariants)", lambda r: pins.check_permute_invariants(_permute_unstable, r)),
    ("permute inclusive offsets", lambda r: pins.check_permute_brute(_permute_inclusive_offsets, r)),
    ("ffn gate/up swapped", lambda r: pins.check_ffn_brute(_swiglu_ffn_from(_dense_swiglu_swapped), r)),
    ("ffn sigmoid not silu", lambda r: pins.check_ffn_silu_values(_dense_swiglu_sigmoid)),
    ("ffn W_down transposed", lambda r: pins.check_ffn_brute(_swiglu_ffn_from(_dense_swiglu_transposed_down), r)),
    ("ffn wrong expert", lambda r: pins.check_ffn_brute(_swiglu_ffn_off_by_one, r)),
    ("combine drops weight", lambda r: pins.check_combine(_combine_dropped_weight, r)),
    ("combine drops last slot", lambda r: pins.check_combine(_combine_last_slot_dropped, r)),
    ("layer gate/up swapped (hand-worked)", lambda r: pins.check_hand_worked(_layer_with(dense=_dense_swiglu_swapped))),
    ("layer drops weight (identical experts)",
     lambda r: pins.check_layer_identical_experts(_layer_with(combine=_combine_dropped_weight), O.dense_swiglu, r)),
    ("layer sigmoid (metamorphic)", lambda r: pins.check_hand_worked(_layer_with(dense=_dense_swiglu_sigmoid))),
]


@pytest.mark.parametrize("name,check", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pin_catches_planted_mistake(name, check):
    with pytest.raises(AssertionError):
        check(np.random.default_rng(99))


def test_router_logits_brute_force():
    """The router GEMM against explicit loops on a tiny shape, and router_topk against
    routing the brute-force logits."""
    rng = np.random.default_rng(21)
    T, H, E, k = 7, 12, 5, 2
    x = rng.standard_normal((T, H))
    w = rng.standard_normal((E, H))
    brute = np.zeros((T, E))
    for t in range(T):
        for e in range(E):
            acc = 0.0
            for h in range(H):
                acc += x[t, h] * w[e, h]
            brute[t, e] = acc
    assert np.allclose(oracle.router_logits(x, w), brute, rtol=1e-14, atol=1e-14)
    ids, wt = oracle.router_topk(x, w, k)
    ids2, wt2 = oracle.route(brute, k)
    assert np.array_equal(ids, ids2) and np.allclose(wt, wt2, rtol=1e-14)
