"""Helpers for the GPU parity tests: move generator outputs to the device and
compare against the oracle.  Nothing here computes any part of the layer."""
from __future__ import annotations

import sys

import numpy as np
import torch


def log(msg: str):
    """Name the case before each GPU step (flushed, so it survives a crash)."""
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dev="cuda") -> torch.Tensor:
    """Host array -> device tensor; uint16 arrays are bf16 bit patterns."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(a).to(dev)


def to_host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> host array; bf16 comes back as uint16 bit patterns."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def weight_tol(k: int, E: int) -> float:
    """Bound on |w_gpu - w_oracle| for gate weights in [0, 1] computed in fp32.

    Each p_j = exp(l_j - l_max) carries at most ~2 ulp (fp32 subtraction rounding
    amplified by |l_j - l_max| is bounded by the exp's own error for the selected
    logits), the fp32 sum of n terms adds at most n half-ulps of the sum and the
    division one more: relative error <= (n + 4) * 2^-24 with n = k (renormalized)
    or n = 8 + log2(E) (tree sum over all experts).  Weights are <= 1, so this
    is also an absolute bound."""
    n = max(k, 8 + int(np.ceil(np.log2(max(E, 2)))))
    return (n + 4) * 2.0 ** -23


def rel_max_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    """max |gpu - ref| / max |ref| (the layer's parity bound is on this ratio)."""
    scale = np.abs(ref).max()
    if scale == 0:
        return float(np.abs(gpu).max())
    return float(np.abs(gpu - ref).max() / scale)


# The grouped GEMMs' tail split (the down projection's last, partly filled round
# of 256 x 256 output tiles cut along k), restated for choosing test cases:
# n tiles on G persistent workgroups with KT k steps each.
MAX_TAIL_PIECES, MAX_TAIL_SPLIT, MIN_PIECE_STEPS = 256, 8, 8


def tail_plan(n: int, G: int, KT: int):
    """(full, r, s): tiles [0, full) whole, the r after them in s pieces each."""
    if G < 2:
        return n, 0, 1
    r = n % G
    if r == 0 or 2 * r > G:
        return n, 0, 1
    s = min(min(G, MAX_TAIL_PIECES) // r, KT // MIN_PIECE_STEPS, MAX_TAIL_SPLIT)
    if s < 2:
        return n, 0, 1
    return n - r, r, s


def mtiles(counts, extra: int) -> np.ndarray:
    """m-tiles per expert: 256-row tiles, the last taking up to 256 + extra rows."""
    c = np.asarray(counts, dtype=np.int64)
    rest = np.maximum(c - extra, 0)
    return np.where(c == 0, 0, np.maximum(1, (rest + 255) // 256))


def down_tiles(offsets: np.ndarray, H: int, extra: int) -> tuple[int, int]:
    """(actual, upper bound) of the down projection's output tiles (256 columns;
    extra = 64 for the bf16 GEMMs, whose last m-tile of an expert takes up to 320
    rows, 0 for the MXFP8 ones)."""
    counts = np.diff(np.asarray(offsets, dtype=np.int64))
    nt = (H + 255) // 256
    actual = int(mtiles(counts, extra).sum()) * nt
    upper = (int(counts.sum()) + len(counts) * 255) // 256 * nt
    return actual, upper


def split_budgets(offsets: np.ndarray, H: int, KT: int, extra: int, want: int = 3):
    """Compute-unit budgets under which the down projection splits its tail, with
    distinct (r, s); plus one under which it does not (None if there is none)."""
    n, upper = down_tiles(offsets, H, extra)
    cands, seen, plain = [], set(), None
    for b in range(2, upper + 1):
        full, r, s = tail_plan(n, min(b, upper), KT)
        if r == 0:
            plain = b if plain is None else plain
        elif (r, s) not in seen:
            seen.add((r, s))
            cands.append((b, r, s))
    # spread over the range: the smallest, the largest and evenly between
    if len(cands) > want:
        cands = [cands[round(i * (len(cands) - 1) / (want - 1))] for i in range(want)]
    return cands, plain
