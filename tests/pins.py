"""Pins for the fp64 oracle: checks fixed by mathematics, not by the oracle itself.

Each ``check_*`` takes the implementation under test as arguments and raises
AssertionError on a mismatch.  tests/test_oracle.py runs them on the oracle
(they must pass) and on deliberately broken copies of it (they must fail), so
every pin is shown to catch a plausible mistake.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import scipy.special


# --------------------------------------------------------------------------- route
def _beats(l, a, b):
    """Expert a is ranked before expert b: larger logit, or equal logit and lower id."""
    return l[a] > l[b] or (l[a] == l[b] and a < b)


def brute_topk(l, k):
    """Brute force over all C(E, k) subsets: the unique subset whose every member beats
    every non-member; slots ordered by how many members beat each member."""
    E = len(l)
    found = []
    for S in itertools.combinations(range(E), k):
        rest = [e for e in range(E) if e not in S]
        if all(_beats(l, a, b) for a in S for b in rest):
            found.append(S)
    assert len(found) == 1
    S = found[0]
    return sorted(S, key=lambda a: sum(_beats(l, b, a) for b in S))


def check_route_brute(route, rng):
    """Integer logits force ties; compare ids with brute force and weights with the
    softmax definition written with math.exp."""
    for _ in range(40):
        T = int(rng.integers(1, 9))
        E = int(rng.integers(1, 7))
        k = int(rng.integers(1, E + 1))
        logits = rng.integers(-2, 3, size=(T, E)).astype(np.float32)
        for renorm in (0, 1):
            ids, w = route(logits, k, renorm)
            for t in range(T):
                l = [float(v) for v in logits[t]]
                want = brute_topk(l, k)
                assert list(ids[t]) == want, (logits[t], k, ids[t], want)
                ex = [math.exp(v) for v in l]
                den = sum(ex[e] for e in want) if renorm else sum(ex)
                for j, e in enumerate(want):
                    assert abs(w[t, j] - ex[e] / den) <= 1e-12


def check_route_library(route, rng):
    """Weights against scipy's softmax: over all E logits (renormalize=0) and over the
    selected logits (renormalize=1); k=E reduces both to the full softmax."""
    for (T, E, k) in [(64, 8, 2), (32, 64, 8), (16, 5, 5), (8, 1, 1), (40, 256, 16)]:
        logits = (rng.standard_normal((T, E)) * 3).astype(np.float32)
        full = scipy.special.softmax(logits.astype(np.float64), axis=1)
        ids, w0 = route(logits, k, 0)
        np.testing.assert_allclose(w0, np.take_along_axis(full, ids.astype(np.int64), 1),
                                   rtol=1e-12, atol=0)
        ids1, w1 = route(logits, k, 1)
        assert (ids1 == ids).all()
        sel = np.take_along_axis(logits.astype(np.float64), ids.astype(np.int64), 1)
        np.testing.assert_allclose(w1, scipy.special.softmax(sel, axis=1), rtol=1e-12, atol=0)
        if k == E:
            np.testing.assert_allclose(w1, np.take_along_axis(full, ids.astype(np.int64), 1),
                                       rtol=1e-12)
        # the selected ids are the argsort of -logits (distinct values: no ties)
        assert (ids[:, 0] == np.argmax(logits, axis=1)).all()
        assert set(map(tuple, np.sort(ids, 1))) == set(
            map(tuple, np.sort(np.argsort(-logits.astype(np.float64), axis=1, kind="stable")[:, :k], 1)))


def check_route_invariants(route, rng):
    """Distinct ids, weights >= 0, non-increasing in the slot, renormalized sum = 1."""
    logits = (rng.standard_normal((500, 16)) * 2).astype(np.float32)
    for k in (1, 3, 16):
        ids, w = route(logits, k, 1)
        assert all(len(set(r)) == k for r in ids.tolist())
        assert (w >= 0).all()
        assert (np.diff(w, axis=1) <= 0).all()
        assert np.abs(w.sum(1) - 1).max() <= 1e-12
        if k == 1:
            assert (w == 1).all()


def check_route_uniform(route):
    """All logits equal: every token picks experts 0..k-1 with weight 1/k."""
    for E, k in [(8, 2), (64, 8), (5, 5), (3, 1)]:
        logits = np.full((7, E), 0.25, dtype=np.float32)
        ids, w = route(logits, k, 1)
        assert (ids == np.arange(k)).all()
        assert np.abs(w - 1.0 / k).max() <= 1e-15
        ids0, w0 = route(logits, k, 0)
        assert (ids0 == np.arange(k)).all()
        assert np.abs(w0 - 1.0 / E).max() <= 1e-15


def check_route_signed_zero(route):
    """-0.0 and +0.0 are equal logits: the tie goes to the lower id."""
    logits = np.array([[-0.0, 0.0, -1.0], [0.0, -0.0, -1.0]], dtype=np.float32)
    ids, _ = route(logits, 1, 1)
    assert ids[:, 0].tolist() == [0, 0]


# --------------------------------------------------------------------------- permute
def brute_permute(ids, E, k):
    """Pure-Python double loop: walk experts in order, tokens in order."""
    T = len(ids)
    counts = [0] * E
    dest = [[-1] * k for _ in range(T)]
    sorted_tok = []
    for e in range(E):
        for t in range(T):
            for j in range(k):
                if ids[t][j] == e:
                    dest[t][j] = len(sorted_tok)
                    sorted_tok.append(t)
                    counts[e] += 1
    offsets = [0]
    for c in counts:
        offsets.append(offsets[-1] + c)
    return counts, offsets, dest, sorted_tok


def _random_ids(rng, T, E, k):
    return np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) if T else \
        np.zeros((0, k), np.int32)


def check_permute_brute(permute, rng):
    for (T, E, k) in [(1, 1, 1), (5, 3, 2), (17, 6, 3), (30, 4, 4), (0, 3, 1), (40, 8, 1)]:
        ids = _random_ids(rng, T, E, k)
        x = rng.standard_normal((T, 3))
        counts, offsets, dest, stok, xp = permute(ids, x, E)
        bc, bo, bd, bs = brute_permute(ids.tolist(), E, k)
        assert list(counts) == bc and list(offsets) == bo
        assert np.asarray(dest).tolist() == bd and list(stok) == bs
        assert np.array_equal(xp, x[np.asarray(bs, dtype=np.int64)])


def check_permute_invariants(permute, rng):
    T, E, k = 300, 16, 4
    ids = _random_ids(rng, T, E, k)
    x = rng.standard_normal((T, 2))
    counts, offsets, dest, stok, xp = permute(ids, x, E)
    R = T * k
    assert counts.sum() == R
    assert offsets[0] == 0 and (np.diff(offsets) == counts).all() and offsets[-1] == R
    assert sorted(dest.ravel().tolist()) == list(range(R))             # bijection onto [0, R)
    for t in range(T):
        for j in range(k):
            e = ids[t, j]
            r = dest[t, j]
            assert stok[r] == t
            assert offsets[e] <= r < offsets[e + 1]
    for e in range(E):
        grp = stok[offsets[e]:offsets[e + 1]]
        assert (np.diff(grp) > 0).all()                                 # ascending tokens
    assert np.array_equal(xp, x[stok])
    # library routine: a stable argsort of the flattened ids
    assert np.array_equal(stok, np.argsort(ids.ravel(), kind="stable") // k)


def check_permute_special(permute):
    T, E, k = 12, 6, 3
    ids = np.tile(np.arange(k, dtype=np.int32), (T, 1))                # uniform router
    counts, offsets, dest, stok, _ = permute(ids, np.zeros((T, 1)), E)
    assert list(counts) == [T] * k + [0] * (E - k)
    assert list(stok) == list(range(T)) * k
    # balanced: token t -> experts (t + j) mod E gives R/E rows per expert
    T, E, k = 16, 8, 4
    ids = ((np.arange(T)[:, None] + np.arange(k)[None, :]) % E).astype(np.int32)
    counts, offsets, _, _, _ = permute(ids, np.zeros((T, 1)), E)
    assert list(counts) == [T * k // E] * E
    assert list(offsets) == [e * T * k // E for e in range(E + 1)]


# --------------------------------------------------------------------------- ffn
def _silu_scalar(z):
    return z / (1.0 + math.exp(-z))


def brute_ffn_row(x, wg, wu, wd):
    """Explicit loops: y_h = sum_f wd[h][f] * silu(sum_i wg[f][i] x_i) * (sum_i wu[f][i] x_i)."""
    H = len(x)
    F = len(wg)
    a = []
    for f in range(F):
        g = sum(wg[f][i] * x[i] for i in range(H))
        u = sum(wu[f][i] * x[i] for i in range(H))
        a.append(_silu_scalar(g) * u)
    return [sum(wd[h][f] * a[f] for f in range(F)) for h in range(H)]


def check_ffn_brute(swiglu_ffn, rng):
    E, H, F = 3, 5, 4
    counts = [2, 0, 3]
    offsets = np.concatenate([[0], np.cumsum(counts)])
    R = offsets[-1]
    xp = rng.standard_normal((R, H))
    wg, wu = rng.standard_normal((E, F, H)), rng.standard_normal((E, F, H))
    wd = rng.standard_normal((E, H, F))
    y = swiglu_ffn(xp, offsets, wg, wu, wd)
    for e in range(E):
        for r in range(offsets[e], offsets[e + 1]):
            want = brute_ffn_row(xp[r].tolist(), wg[e].tolist(), wu[e].tolist(), wd[e].tolist())
            assert np.allclose(y[r], want, rtol=1e-12, atol=1e-12)


def check_ffn_silu_values(dense_swiglu):
    """H = F = 1 reduces the FFN to c * silu(a x) * (b x); closed-form silu values."""
    for a, want in [(0.0, 0.0), (1.0, 1.0 / (1.0 + math.exp(-1.0))), (-2.0, -2.0 / (1.0 + math.exp(2.0))),
                    (math.log(3.0), 0.75 * math.log(3.0))]:
        y = dense_swiglu(np.array([[1.0]]), np.array([[a]]), np.array([[2.0]]), np.array([[3.0]]))
        assert abs(y[0, 0] - 6.0 * want) <= 1e-14


def check_layer_identical_experts(layer, dense_swiglu, rng):
    """Identical experts: with renormalized weights summing to 1, y is the dense SwiGLU
    of x for any routing."""
    T, H, F, E, k = 40, 8, 6, 5, 3
    x = rng.standard_normal((T, H))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    g, u, d = rng.standard_normal((F, H)), rng.standard_normal((F, H)), rng.standard_normal((H, F))
    out = layer(x, logits, k, np.stack([g] * E), np.stack([u] * E), np.stack([d] * E), 1)
    want = np.array([brute_ffn_row(x[t].tolist(), g.tolist(), u.tolist(), d.tolist()) for t in range(T)])
    assert np.allclose(out["y"], want, rtol=1e-11, atol=1e-12)
    # E = 1, k = 1: the layer is one dense FFN
    out1 = layer(x, logits[:, :1], 1, g[None], u[None], d[None], 1)
    assert np.allclose(out1["y"], want, rtol=1e-11, atol=1e-12)


def check_layer_metamorphic(layer, rng):
    """x = 0 gives y = 0; scaling W_down by c scales y by c; permuting tokens permutes y."""
    T, H, F, E, k = 24, 6, 4, 4, 2
    x = rng.standard_normal((T, H))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    wg, wu, wd = rng.standard_normal((E, F, H)), rng.standard_normal((E, F, H)), rng.standard_normal((E, H, F))
    y = layer(x, logits, k, wg, wu, wd)["y"]
    assert np.abs(layer(np.zeros_like(x), logits, k, wg, wu, wd)["y"]).max() == 0
    assert np.allclose(layer(x, logits, k, wg, wu, 2.5 * wd)["y"], 2.5 * y, rtol=1e-12, atol=1e-14)
    p = rng.permutation(T)
    assert np.allclose(layer(x[p], logits[p], k, wg, wu, wd)["y"], y[p], rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------- combine
def check_combine(combine, rng):
    T, k, H, R = 9, 3, 4, 27
    y_perm = rng.standard_normal((R, H))
    dest = rng.permutation(R).reshape(T, k)
    w = rng.random((T, k))
    y = combine(y_perm, dest, w)
    scat = np.zeros((T, H))
    for j in range(k):                       # scatter-add form, same slot order
        np.add.at(scat, np.arange(T), w[:, j:j + 1] * y_perm[dest[:, j]])
    assert np.array_equal(y, scat)
    y1 = combine(y_perm, dest[:, :1], np.ones((T, 1)))
    assert np.array_equal(y1, y_perm[dest[:, 0]])
    ys = rng.standard_normal((T, H))
    assert np.allclose(combine(y_perm, dest, w, ys), y + ys, rtol=1e-15, atol=1e-15)


def check_hand_worked(layer):
    """A layer small enough to evaluate by hand (H = F = 1, E = 3, k = 2, x = 1).

    logits (0, ln 3, ln 2): the top-2 experts are 1 then 2 with renormalized weights
    3/5 and 2/5 (6/... without renormalization: 3/6 and 2/6).  Expert e computes
    c_e * silu(a_e x) * (b_e x):
      expert 1: a = ln 3, b = 2, c = 1:  silu(ln 3) = ln 3 / (1 + 1/3) = 0.75 ln 3,
                so its output is 1.5 ln 3;
      expert 2: a = 0, so silu(0) = 0 and its output is 0.
    y = 3/5 * 1.5 ln 3 = 0.9 ln 3 (renormalized), 3/6 * 1.5 ln 3 = 0.75 ln 3 (not).
    The logits are fp32, so ln 3 and ln 2 carry a relative rounding of about 6e-8,
    hence the 1e-6 bound."""
    x = np.array([[1.0]])
    logits = np.array([[0.0, math.log(3.0), math.log(2.0)]], dtype=np.float32)
    wg = np.array([[[0.7]], [[math.log(3.0)]], [[0.0]]])
    wu = np.array([[[1.0]], [[2.0]], [[5.0]]])
    wd = np.array([[[1.0]], [[1.0]], [[4.0]]])
    out = layer(x, logits, 2, wg, wu, wd, 1)
    assert out["ids"].tolist() == [[1, 2]]
    assert abs(out["w"][0, 0] - 0.6) <= 1e-6 and abs(out["w"][0, 1] - 0.4) <= 1e-6
    assert abs(out["y"][0, 0] - 0.9 * math.log(3.0)) <= 1e-6
    out0 = layer(x, logits, 2, wg, wu, wd, 0)
    assert abs(out0["w"][0, 0] - 0.5) <= 1e-6 and abs(out0["w"][0, 1] - 1.0 / 3.0) <= 1e-6
    assert abs(out0["y"][0, 0] - 0.75 * math.log(3.0)) <= 1e-6
