"""The measurement probe library (libmoe_probe.so, built beside libmoe.so; not part
of the MoE path): it loads, exports its entry point, rejects bad arguments on the
host, and on the GPU its four variants run to completion with finite results."""
import ctypes
import os

import pytest

import paper_2606_21712_amd as moe

PATH = os.path.join(os.path.dirname(moe.__file__), "libmoe_probe.so")


def _lib():
    lib = ctypes.CDLL(PATH)
    fn = lib.moe_probe_mfma_rate
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    return fn


def test_probe_library_exports_its_entry_point():
    assert os.path.exists(PATH), "libmoe_probe.so is not built (run __graft_entry__.build())"
    fn = _lib()
    # host-side argument checks: nothing is launched
    assert fn(0, 0, 0, 4, ctypes.c_void_p(16), None) == 1        # no workgroups
    assert fn(0, 0, 1, -4, ctypes.c_void_p(16), None) == 1       # negative iterations
    assert fn(0, 0, 1, 4, None, None) == 1                        # no output buffer


@pytest.mark.gpu
def test_probe_variants_run():
    import torch
    fn = _lib()
    blocks = 256
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    for fp8 in (0, 1):
        for rnd in (0, 1):
            out.fill_(float("nan"))
            assert fn(fp8, rnd, blocks, 64, out.data_ptr(), stream) == 0
            torch.cuda.synchronize()
            assert bool(torch.isfinite(out).all()), (fp8, rnd)
            assert float(out.abs().sum()) > 0.0, (fp8, rnd)
