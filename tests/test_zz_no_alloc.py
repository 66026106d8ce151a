"""moe_permute_static (the permute entry point that allocates nothing: its
scratch is a static device array) against moe_permute through the C ABI.

Two calls in a row on the same array, the second on a smaller batch, each
compared bit for bit with moe_permute on a caller workspace (maps and x_perm);
both sides of the single-block boundary (at most 16 units of 1024 assignments)
are covered, and the larger call leaves counts in the array that the smaller
one must not see."""
import numpy as np
import pytest
import torch

import moegen
import paper_2606_21712_amd as moe
from gpu_util import log, to_dev

pytestmark = pytest.mark.gpu

KEYS = ("counts", "offsets", "sorted_token_ids", "dest_rows", "x_perm")


def _case(T, E, k, H, seed):
    # lognormal expert loads (two experts pinned to 1 and 3 rows) on the larger batch,
    # router logits on the others
    kw = dict(routing="lognormal", pinned_small=(1, 3)) if E >= 64 else {}
    cfg = moegen.MoEConfig("no_alloc", T=T, H=H, E=E, k=k, F=64, seed=seed, **kw)
    I = moegen.make_inputs(cfg, with_weights=False)
    x, logits = to_dev(I.x), to_dev(I.logits)
    ids, _ = moe.moe_route(logits, k)
    return ids, x


@pytest.mark.parametrize("sizes", [((40000, 64, 4, 128), (3000, 16, 2, 64)),
                                   ((9000, 8, 2, 256), (700, 8, 2, 256))])
def test_static_scratch_matches_workspace_path(sizes):
    for i, (T, E, k, H) in enumerate(sizes):
        log(f"no_alloc call {i}: T={T} E={E} k={k} H={H}")
        ids, x = _case(T, E, k, H, seed=100 + i)
        ref = moe.moe_permute(ids, x, E)
        got = moe.moe_permute_static(ids, x, E)
        torch.cuda.synchronize()
        for key in KEYS:
            assert torch.equal(got[key].view(torch.int16) if got[key].dtype == torch.bfloat16 else got[key],
                               ref[key].view(torch.int16) if ref[key].dtype == torch.bfloat16 else ref[key]), \
                f"call {i}: {key} differs"
        # maps only (x_perm NULL)
        got2 = moe.moe_permute_static(ids, x, E, gather_rows=False)
        torch.cuda.synchronize()
        for key in KEYS[:4]:
            assert torch.equal(got2[key], ref[key]), f"call {i} (maps only): {key} differs"


def test_static_scratch_rejects_sizes_beyond_the_array():
    # 2^22 assignments over 256 experts need exactly the 4 MiB array; one more unit does not fit
    T, E, k = (1 << 22) // 8 + 1024, 256, 8
    ids = torch.zeros((T, k), dtype=torch.int32, device="cuda")
    x = torch.zeros((T, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(moe.MoEError) as ei:
        moe.moe_permute_static(ids, x, E, gather_rows=False)
    assert ei.value.status == 2 and b"static" in moe.lib().moe_last_error()
