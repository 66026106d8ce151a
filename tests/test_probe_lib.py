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


def _stream():
    fn = ctypes.CDLL(PATH).moe_probe_stream_panels
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p]
    return fn


def test_stream_probe_rejects_bad_arguments():
    fn = _stream()
    p = ctypes.c_void_p(16)
    assert fn(None, 1, 4096, 0, 1, p, p, None) == 1           # no matrix
    assert fn(p, 0, 4096, 0, 1, p, p, None) == 1              # no panels
    assert fn(p, 1, 4000, 0, 1, p, p, None) == 1              # K not a multiple of 128
    assert fn(p, 1, 1 << 23, 0, 1, p, p, None) == 1           # a panel past 2^31 bytes
    assert fn(p, 1, 4096, 0, 0, p, p, None) == 1              # no workgroups
    assert fn(p, 1, 4096, 0, 1, None, p, None) == 1           # no counter


@pytest.mark.gpu
def test_stream_probe_runs():
    """Both orders run to completion: every panel claimed once, then one failed
    claim per workgroup."""
    import torch
    fn = _stream()
    K, panels, blocks = 4096, 24, 16
    w = torch.ones(panels * 256 * K, dtype=torch.uint8, device="cuda")
    ctr = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty(blocks * 512, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    for rot in (0, 1):
        ctr.zero_()
        assert fn(w.data_ptr(), panels, K, rot, blocks, ctr.data_ptr(), out.data_ptr(), stream) == 0
        torch.cuda.synchronize()
        assert int(ctr.item()) == panels + blocks


def test_write_probe_rejects_bad_arguments():
    fn = ctypes.CDLL(PATH).moe_probe_write
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p]
    p = ctypes.c_void_p(16)
    assert fn(None, 1024, 1, None) == 1                       # no buffer
    assert fn(p, 1000, 1, None) == 1                          # not a multiple of 16
    assert fn(p, 1024, 0, None) == 1                          # no workgroups


@pytest.mark.gpu
def test_write_probe_fills_the_buffer():
    import torch
    fn = ctypes.CDLL(PATH).moe_probe_write
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p]
    buf = torch.full((1 << 20,), -1, dtype=torch.int32, device="cuda")
    assert fn(buf.data_ptr(), buf.numel() * 4, 64, torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    v = buf.view(-1, 4).cpu()
    assert bool((v[:, 2] == 0).all()) and bool((v[:, 3] == 0).all())   # every 16-byte slot written
