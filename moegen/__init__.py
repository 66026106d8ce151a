"""Seeded synthetic inputs for the MoE-layer hot path.

This module is shared by the fp64 oracle and the HIP path.  It draws random
numbers and builds routing logits; it holds none of the layer's arithmetic
(no top-k, no softmax, no grouping, no FFN, no combine).

Workload shapes follow the layers the paper evaluates (Mixtral-8x7B/8x22B and
DeepSeek-R1 class models, Section "Evaluation", Models paragraph; hidden size
7168 from the overhead discussion).  The paper's datasets and weights are not
used: every value here is synthetic.

Conventions
-----------
* bf16 tensors are carried on the host as ``uint16`` bit patterns; fp32 tensors
  as ``float32``.  ``as_f64`` upcasts either exactly.
* "N(0, s)" means mean 0, standard deviation s.
* Weights are stored K-contiguous: ``w_gate, w_up : [E, F, H]``,
  ``w_down : [E, H, F]``.
* Every tensor is drawn in fixed chunks, each from its own child of
  ``SeedSequence(seed)``, so the values do not depend on the thread count.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

__all__ = [
    "MoEConfig", "CONFIGS", "Inputs", "make_inputs", "round_bf16", "as_f64",
    "zipf_counts", "lognormal_counts", "exact_count_assignment", "router_matrix", "margin_logits", "cap_counts",
]

_CHUNK = 1 << 22          # elements per independently seeded chunk
_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@dataclass(frozen=True)
class MoEConfig:
    """One MoE layer workload.

    routing: "router"    logits = x . W_r  (W_r ~ N(0, router_std))
             "zipf"      exact per-expert counts c_r ~ r^-zipf_s, then margin logits
             "lognormal" exact per-expert counts from lognormal(0, sigma), with the
                         smallest experts pinned to ``pinned_small`` rows
             "uniform"   all logits equal (every token ties on every expert)
    """
    name: str
    T: int
    H: int
    E: int
    k: int
    F: int
    Fs: int = 0                 # shared-expert FFN dim (0 = none)
    dtype: str = "bf16"         # "bf16" or "f32"
    seed: int = 0
    routing: str = "router"
    router_std: float = 0.02
    zipf_s: float = 1.2
    lognormal_sigma: float = 1.0
    pinned_small: tuple = ()
    margin: float = 20.0
    renormalize: int = 1

    @property
    def R(self) -> int:
        return self.T * self.k

    def flops(self) -> int:
        """Algorithmic flops of the grouped SwiGLU FFN (+ shared expert)."""
        return 6 * self.H * self.F * self.R + 6 * self.H * self.Fs * self.T

    def scaled(self, **kw) -> "MoEConfig":
        return replace(self, **kw)


# The five workloads: a tiny fp32 layer, a Mixtral-shaped layer with near-uniform
# routing, the same shape with Zipf-skewed expert load, one GPU's share of a
# DeepSeek-style fine-grained layer with a shared expert, and a large
# memory-constrained expert batch with lognormal expert loads.
CONFIGS = {
    "tiny": MoEConfig("tiny", T=256, H=256, E=8, k=2, F=512, dtype="f32", seed=0),
    "mixtral4k": MoEConfig("mixtral4k", T=4096, H=4096, E=8, k=2, F=14336, seed=1),
    "mixtral32k_zipf": MoEConfig("mixtral32k_zipf", T=32768, H=4096, E=8, k=2, F=14336,
                                 seed=2, routing="zipf"),
    "deepseek": MoEConfig("deepseek", T=16384, H=7168, E=64, k=8, F=2048, Fs=2048, seed=3),
    "memconstrained": MoEConfig("memconstrained", T=131072, H=4096, E=64, k=4, F=4096,
                                seed=4, routing="lognormal", pinned_small=(1, 17, 31)),
}


# --------------------------------------------------------------------------- numerics helpers
def round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even.  Finite inputs only."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).copy()
    lsb = (u >> 16) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    return (u >> 16).astype(np.uint16)


def as_f64(a: np.ndarray) -> np.ndarray:
    """Exact upcast of a float32 array or a bf16 bit-pattern (uint16) array to float64."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


def as_f32(a: np.ndarray) -> np.ndarray:
    """Exact upcast of bf16 bit patterns (uint16) to float32; float32 passes through."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32)
    return np.asarray(a, dtype=np.float32)


# --------------------------------------------------------------------------- seeded drawing
def _normal(seq: np.random.SeedSequence, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std) of the given shape, drawn in fixed chunks with spawned seeds; bf16 or f32."""
    n = int(np.prod(shape))
    out32 = np.empty(n, dtype=np.float32)
    nchunks = max(1, -(-n // _CHUNK))
    kids = seq.spawn(nchunks)

    def work(i):
        lo, hi = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        g = np.random.default_rng(kids[i])
        g.standard_normal(out=out32[lo:hi], dtype=np.float32)
        if std != 1.0:
            out32[lo:hi] *= np.float32(std)
        if dtype == "bf16":
            return round_bf16(out32[lo:hi])
        return None

    if nchunks == 1:
        parts = [work(0)]
    else:
        with ThreadPoolExecutor(_THREADS) as ex:
            parts = list(ex.map(work, range(nchunks)))
    if dtype == "bf16":
        return np.concatenate(parts).reshape(shape)
    return out32.reshape(shape)


def largest_remainder(weights: np.ndarray, total: int) -> np.ndarray:
    """Integer counts proportional to ``weights`` summing exactly to ``total``."""
    w = np.asarray(weights, dtype=np.float64)
    q = w / w.sum() * total
    base = np.floor(q).astype(np.int64)
    rem = int(total - base.sum())
    frac = q - base
    order = np.lexsort((np.arange(len(w)), -frac))   # largest remainder, ties to lower index
    base[order[:rem]] += 1
    return base


def zipf_counts(E: int, R: int, s: float) -> np.ndarray:
    """Counts c_r proportional to r^-s (r = 1..E), largest first, summing to R."""
    return largest_remainder(np.arange(1, E + 1, dtype=np.float64) ** (-s), R)


def lognormal_counts(rng: np.random.Generator, E: int, R: int, sigma: float,
                     pinned_small=()) -> np.ndarray:
    """Counts from E lognormal(0, sigma) draws; the len(pinned_small) smallest draws
    are pinned to the given row counts and the rest share the remaining rows."""
    d = rng.lognormal(0.0, sigma, size=E)
    counts = np.zeros(E, dtype=np.int64)
    p = len(pinned_small)
    if p:
        small = np.argsort(d, kind="stable")[:p]
        counts[small] = np.asarray(sorted(pinned_small), dtype=np.int64)
        rest = np.setdiff1d(np.arange(E), small)
        counts[rest] = largest_remainder(d[rest], R - int(counts.sum()))
    else:
        counts[:] = largest_remainder(d, R)
    return counts


def cap_counts(counts: np.ndarray, cap: int) -> np.ndarray:
    """Counts with none above cap and the same sum: the excess of the capped experts
    goes, largest expert first, to the others up to the cap (needed when a batch is
    too small for its largest expert, which can hold at most one row per token)."""
    c = np.asarray(counts, dtype=np.int64).copy()
    assert c.sum() <= cap * c.size
    excess = int(np.maximum(c - cap, 0).sum())
    c = np.minimum(c, cap)
    for e in np.argsort(-c, kind="stable"):
        if excess == 0:
            break
        add = min(cap - int(c[e]), excess)
        c[e] += add
        excess -= add
    return c


def exact_count_assignment(counts: np.ndarray, T: int, k: int, rng: np.random.Generator):
    """Assign experts to tokens so expert e receives exactly counts[e] tokens and every
    token receives k distinct experts.

    Expert labels, each repeated counts[e] times in descending-count order, fill
    positions p = 0..T*k-1; position p goes to token p mod T.  A run of length
    c_e <= T never wraps onto the same token, so each token's k labels are distinct.
    Tokens and expert labels are then shuffled with ``rng``.
    Returns ``chosen [T, k]`` (unordered expert sets) and the relabelling map.
    """
    counts = np.asarray(counts, dtype=np.int64)
    E = counts.size
    assert counts.sum() == T * k and counts.max() <= T and counts.min() >= 0
    order = np.argsort(-counts, kind="stable")
    labels = np.repeat(order, counts[order])            # length T*k
    chosen = labels.reshape(k, T).T.copy()              # chosen[t, j] = labels[j*T + t]
    tok_perm = rng.permutation(T)
    relabel = rng.permutation(E)
    chosen = relabel[chosen[tok_perm]]
    return chosen.astype(np.int32), relabel


# --------------------------------------------------------------------------- the input bundle
@dataclass
class Inputs:
    cfg: MoEConfig
    x: np.ndarray               # [T, H]  uint16 (bf16 bits) or float32
    logits: np.ndarray          # [T, E]  float32
    w_gate: np.ndarray          # [E, F, H]
    w_up: np.ndarray            # [E, F, H]
    w_down: np.ndarray          # [E, H, F]
    ws_gate: np.ndarray | None = None   # [1, Fs, H]
    ws_up: np.ndarray | None = None     # [1, Fs, H]
    ws_down: np.ndarray | None = None   # [1, H, Fs]
    chosen: np.ndarray | None = None    # [T, k] constructed expert sets (zipf/lognormal)
    target_counts: np.ndarray | None = None
    extra: dict = field(default_factory=dict)


def _router_logits(x: np.ndarray, w_r: np.ndarray, bias: np.ndarray | None) -> np.ndarray:
    """fp32(x . W_r (+ bias)), accumulated in fp64 on the host, in token chunks."""
    T = x.shape[0]
    out = np.empty((T, w_r.shape[1]), dtype=np.float32)
    wr = w_r.astype(np.float64)
    step = 8192
    for lo in range(0, T, step):
        hi = min(T, lo + step)
        acc = as_f64(x[lo:hi]) @ wr
        if bias is not None:
            acc += bias[lo:hi]
        out[lo:hi] = acc.astype(np.float32)
    return out


def router_matrix(cfg: MoEConfig) -> np.ndarray:
    """The router matrix W_r [H, E] fp32 of the workload's seed (the same draw as
    make_inputs)."""
    s_r = np.random.SeedSequence(cfg.seed).spawn(9)[1]
    return _normal(s_r, (cfg.H, cfg.E), cfg.router_std, "f32")


def margin_logits(x: np.ndarray, w_r: np.ndarray, chosen: np.ndarray, margin: float) -> np.ndarray:
    """fp32(x . W_r + margin on each token's chosen experts): logits whose top-k is
    exactly the chosen set when the margin exceeds the spread of x . W_r."""
    mark = np.zeros((x.shape[0], w_r.shape[1]), dtype=np.float64)
    np.put_along_axis(mark, np.asarray(chosen, dtype=np.int64), margin, axis=1)
    return _router_logits(x, w_r, mark)


def make_inputs(cfg: MoEConfig | str, seed: int | None = None, with_weights: bool = True) -> Inputs:
    """Build the seeded inputs of one workload.  Draw order (one spawned child each):
    x, W_r, W_gate, W_up, W_down, Ws_gate, Ws_up, Ws_down, routing."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    if seed is not None:
        cfg = cfg.scaled(seed=seed)
    T, H, E, k, F, Fs = cfg.T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs
    assert 1 <= k <= E
    root = np.random.SeedSequence(cfg.seed)
    s_x, s_r, s_g, s_u, s_d, s_sg, s_su, s_sd, s_route = root.spawn(9)
    dt = cfg.dtype

    x = _normal(s_x, (T, H), 1.0, dt)
    w_r = _normal(s_r, (H, E), cfg.router_std, "f32")
    if with_weights:
        w_gate = _normal(s_g, (E, F, H), 1.0 / np.sqrt(H), dt)
        w_up = _normal(s_u, (E, F, H), 1.0 / np.sqrt(H), dt)
        w_down = _normal(s_d, (E, H, F), 1.0 / np.sqrt(F), dt)
    else:
        w_gate = w_up = w_down = None
    ws = (None, None, None)
    if Fs and with_weights:
        ws = (_normal(s_sg, (1, Fs, H), 1.0 / np.sqrt(H), dt),
              _normal(s_su, (1, Fs, H), 1.0 / np.sqrt(H), dt),
              _normal(s_sd, (1, H, Fs), 1.0 / np.sqrt(Fs), dt))

    rng = np.random.default_rng(s_route)
    chosen = None
    target = None
    if cfg.routing == "router":
        logits = _router_logits(x, w_r, None)
    elif cfg.routing == "uniform":
        logits = np.zeros((T, E), dtype=np.float32)
    elif cfg.routing in ("zipf", "lognormal"):
        if cfg.routing == "zipf":
            target = zipf_counts(E, T * k, cfg.zipf_s)
        else:
            target = lognormal_counts(rng, E, T * k, cfg.lognormal_sigma, cfg.pinned_small)
        chosen, _ = exact_count_assignment(target, T, k, rng)
        mark = np.zeros((T, E), dtype=np.float64)
        np.put_along_axis(mark, chosen.astype(np.int64), cfg.margin, axis=1)
        logits = _router_logits(x, w_r, mark)
        # The construction must leave every chosen logit above every other one.
        sel = np.take_along_axis(logits, chosen.astype(np.int64), axis=1)
        masked = np.where(mark > 0, -np.inf, logits)
        assert (sel.min(axis=1) > masked.max(axis=1)).all(), "routing margin too small"
        if cfg.routing == "zipf":
            # map target counts (listed by rank) onto the relabelled experts
            target = np.bincount(chosen.ravel(), minlength=E)
        else:
            target = np.bincount(chosen.ravel(), minlength=E)
    else:
        raise ValueError(f"unknown routing {cfg.routing!r}")

    extra = {}
    if dt == "bf16":
        # the router matrix as a bf16 [E, H] tensor (K-contiguous rows, like the
        # expert weights), for the path that computes the logits itself
        extra["w_router"] = round_bf16(np.ascontiguousarray(w_r.T))
    return Inputs(cfg, x, logits, w_gate, w_up, w_down, *ws, chosen=chosen,
                  target_counts=target, extra=extra)
