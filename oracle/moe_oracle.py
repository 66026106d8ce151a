"""Plain, slow, fp64 CPU oracle of one Mixture-of-Experts layer over an expert batch.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke entry point and the
benchmark's CPU-baseline leg may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and the
oracle shares no code with that path: it uses numpy only.

What is computed.  The paper's forward pass (Algorithm 1) runs the MoE module
on the hidden states COMBINEd from many yielded sequences, h_out <- MoE(h, l),
and motivates the large combined batch by sparse expert activation with uneven
expert popularity (Section 2.2, Insight 1).  The paper does not write the MoE
layer out; this oracle takes the standard top-k softmax-gated SwiGLU expert
layer of the Mixtral and DeepSeek models it evaluates (Section 6, Models):

  route    : per token, the k experts with the largest logits (ties to the lower
             expert id, slots in descending order); gate weights are a softmax
             over the k selected logits (renormalize=1) or the slice of the full
             softmax over all E logits (renormalize=0).
  permute  : per-expert counts, exclusive-prefix offsets, and a stable grouping
             in which expert e's rows hold its tokens in ascending token order.
  ffn      : y = W_down (silu(W_gate x) * (W_up x)), silu(z) = z / (1 + e^-z),
             no biases, per expert group.
  combine  : y[t] = sum_j w[t, j] * y_perm[dest_rows[t, j]]  (+ shared expert).

Every value is computed in float64 from the exact input bits (bf16 inputs are
upcast exactly), with no intermediate rounding.  Each function is pinned by the
tests in tests/test_oracle.py (brute force, closed forms, invariants, special
cases) rather than by values printed in the paper, which gives none for the
MoE layer.
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    """Exact float64 view of a float32 array or a bf16 bit-pattern (uint16) array."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# --------------------------------------------------------------------------- route
def route(logits, k: int, renormalize: int = 1):
    """Top-k expert selection and gate weights for every token.

    logits : [T, E] float (fp32 on the GPU side; upcast exactly here).
    Returns ids int32 [T, k] (slot 0 = largest logit) and w float64 [T, k].

    Order: larger logit first; equal logits go to the lower expert id.  The
    selection is made on the logits themselves (softmax is monotone, so this is
    the same set as selecting on probabilities, without ties created by
    rounding exp).  Weights: p_e = exp(l_e - m) with m the largest logit;
    w_j = p_{ids_j} / sum_{j'<k} p_{ids_j'} when renormalizing, otherwise
    w_j = p_{ids_j} / sum_{e<E} p_e.
    """
    L = _f64(logits)
    T, E = L.shape
    if not (1 <= k <= E):
        raise ValueError("k must be in [1, E]")
    if not np.isfinite(L).all():
        raise ValueError("logits must be finite")
    expert = np.broadcast_to(np.arange(E), (T, E))
    order = np.lexsort((expert, -L), axis=1)          # primary -logit, secondary expert id
    ids = order[:, :k]
    sel = np.take_along_axis(L, ids, axis=1)
    m = sel[:, :1]
    p_sel = np.exp(sel - m)
    if renormalize:
        denom = np.zeros((T, 1))
        for j in range(k):                              # summed in slot order
            denom[:, 0] += p_sel[:, j]
    else:
        denom = np.exp(L - m).sum(axis=1, keepdims=True)
    return ids.astype(np.int32), p_sel / denom


def router_logits(x, w_router):
    """The MoE gate's router GEMM: logits[t, e] = x[t] . w_router[e] in fp64 from the
    exact input bits (x [T, H], w_router [E, H]; the step before the gate in
    Section 7's MoE-gate batch)."""
    return _f64(x) @ _f64(w_router).T


def router_topk(x, w_router, k: int, renormalize: int = 1):
    """Router GEMM followed by the gate: route(router_logits(x, w_router))."""
    return route(router_logits(x, w_router), k, renormalize)


# --------------------------------------------------------------------------- permute
def permute(ids, x, E: int):
    """Group the T*k (token, slot) assignments by expert.

    Returns counts [E], offsets [E+1], dest_rows [T, k], sorted_token_ids [T*k]
    (all int32) and x_perm [T*k, H] (same dtype as x: a pure row copy).

    Expert e's rows are offsets[e] .. offsets[e+1]-1 and hold, in ascending
    token order, the tokens routed to e.  A stable sort of the flattened
    assignment list by expert id gives exactly that order, because a token's k
    experts are distinct and flattened order is token-major.
    """
    ids = np.asarray(ids)
    T, k = ids.shape
    flat = ids.reshape(-1).astype(np.int64)
    if flat.size and (flat.min() < 0 or flat.max() >= E):
        raise ValueError("expert id out of range")
    order = np.argsort(flat, kind="stable")
    counts = np.bincount(flat, minlength=E)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    sorted_token_ids = order // k
    dest = np.empty(T * k, dtype=np.int64)
    dest[order] = np.arange(T * k)
    x = np.asarray(x)
    x_perm = x[sorted_token_ids]
    return (counts.astype(np.int32), offsets.astype(np.int32), dest.reshape(T, k).astype(np.int32),
            sorted_token_ids.astype(np.int32), x_perm)


# --------------------------------------------------------------------------- ffn
def _silu(z):
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def dense_swiglu(x, w_gate, w_up, w_down):
    """One expert's SwiGLU FFN on rows x [n, H]: W_down (silu(W_gate x) * (W_up x)).

    w_gate, w_up : [F, H]; w_down : [H, F].  fp64, no intermediate rounding."""
    X = _f64(x)
    g = X @ _f64(w_gate).T
    u = X @ _f64(w_up).T
    return (_silu(g) * u) @ _f64(w_down).T


def swiglu_ffn(x_perm, offsets, w_gate, w_up, w_down):
    """Grouped SwiGLU FFN: rows offsets[e]..offsets[e+1]-1 of x_perm go through expert e.

    w_gate, w_up : [E, F, H]; w_down : [E, H, F].  Returns y_perm float64 [R, H]."""
    offsets = np.asarray(offsets, dtype=np.int64)
    E = offsets.size - 1
    R = int(offsets[-1])
    H = w_down.shape[1]
    y = np.zeros((R, H))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            y[lo:hi] = dense_swiglu(x_perm[lo:hi], w_gate[e], w_up[e], w_down[e])
    return y


def ffn_rows(x_rows, e: int, w_gate, w_up, w_down):
    """Expert e's SwiGLU FFN on an arbitrary set of rows (used for sampled checks)."""
    return dense_swiglu(x_rows, w_gate[e], w_up[e], w_down[e])


# --------------------------------------------------------------------------- combine
def combine(y_perm, dest_rows, w, y_shared=None):
    """y[t] = sum_j w[t, j] * y_perm[dest_rows[t, j]]  (+ y_shared[t]), fp64, slots in order."""
    Y = _f64(y_perm)
    dest_rows = np.asarray(dest_rows, dtype=np.int64)
    w = np.asarray(w, dtype=np.float64)
    T, k = dest_rows.shape
    y = np.zeros((T, Y.shape[1]))
    for j in range(k):
        y += w[:, j:j + 1] * Y[dest_rows[:, j]]
    if y_shared is not None:
        y += _f64(y_shared)
    return y


# --------------------------------------------------------------------------- whole layer
def layer(x, logits, k, w_gate, w_up, w_down, renormalize=1, ws_gate=None, ws_up=None,
          ws_down=None):
    """The whole MoE layer; returns a dict of every intermediate and the output y."""
    E = w_gate.shape[0]
    ids, w = route(logits, k, renormalize)
    counts, offsets, dest, sorted_tok, x_perm = permute(ids, x, E)
    y_perm = swiglu_ffn(x_perm, offsets, w_gate, w_up, w_down)
    y_shared = None
    if ws_gate is not None:
        y_shared = dense_swiglu(x, ws_gate[0], ws_up[0], ws_down[0])
    y = combine(y_perm, dest, w, y_shared)
    return dict(ids=ids, w=w, counts=counts, offsets=offsets, dest_rows=dest,
                sorted_token_ids=sorted_tok, x_perm=x_perm, y_perm=y_perm,
                y_shared=y_shared, y=y)


def token_outputs(tokens, x, logits, k, w_gate, w_up, w_down, renormalize=1,
                  ws_gate=None, ws_up=None, ws_down=None):
    """The layer output y[t] for a subset of tokens only (sampled checks at full size).

    Routing is per token, so a token's output needs only its own logits, its
    experts' weights and its own hidden row.  Each expert's weights are upcast
    once for all sampled rows that use it.  Returns (ids, w, y_rows [n, H],
    per-assignment expert outputs [n, k, H])."""
    tokens = np.asarray(tokens, dtype=np.int64)
    ids, w = route(np.asarray(logits)[tokens], k, renormalize)
    xs = np.asarray(x)[tokens]
    n = tokens.size
    H = w_down.shape[1]
    per = np.zeros((n, k, H))
    for e in np.unique(ids):
        sel_t, sel_j = np.nonzero(ids == e)
        per[sel_t, sel_j] = ffn_rows(xs[sel_t], int(e), w_gate, w_up, w_down)
    y = np.zeros((n, H))
    for j in range(k):
        y += w[:, j:j + 1] * per[:, j]
    if ws_gate is not None:
        y += dense_swiglu(xs, ws_gate[0], ws_up[0], ws_down[0])
    return ids, w, y, per
