"""The allocation-free conv entry point (fs_conv_bf16_device_noalloc):
split-K partial sums in the library's static device array instead of a
buffer it allocates.  Its outputs equal fs_test_conv's (same kernels, tile
and split rule) bit for bit, on consecutive calls whose second is smaller
(the array keeps the first call's contents), and shapes whose partial sums
would not fit are refused."""
import ctypes

import numpy as np
import pytest

from paper_2003_01538_amd import flexserve as fsb

pytestmark = pytest.mark.gpu


def _run(B, H, W, Cin, Cout, k, s, p, relu, with_res, seed):
    import torch
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((B, H, W, Cin), generator=g).to(torch.bfloat16)
    w = (torch.randn((Cout, k, k, Cin), generator=g) * (2.0 / (k * k * Cin)) ** 0.5).to(torch.bfloat16)
    b = torch.randn(Cout, generator=g) * 0.1
    Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    r = torch.randn((B, Ho, Wo, Cout), generator=g).to(torch.bfloat16) if with_res else None
    ref = fsb.fs_test_conv(x.float().numpy(), w.float().numpy(), b.numpy(),
                           None if r is None else r.float().numpy(), s, p, relu, fsb.FS_BF16)
    dx, dw, db = x.cuda(), w.cuda(), b.cuda()
    dr = None if r is None else r.cuda()
    out = torch.full((B, Ho, Wo, Cout), float("nan"), dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    lib = fsb.load()
    st = lib.fs_conv_bf16_device_noalloc(
        ctypes.c_void_p(dx.data_ptr()), B, H, W, Cin, ctypes.c_void_p(dw.data_ptr()),
        ctypes.cast(ctypes.c_void_p(db.data_ptr()), ctypes.POINTER(ctypes.c_float)),
        None if dr is None else ctypes.c_void_p(dr.data_ptr()), Cout, k, k, s, p, relu,
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == fsb.FS_OK, lib.fs_last_error(None)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), (B, H, Cin, Cout, np.abs(got - ref).max())


def test_noalloc_conv_equals_fs_test_conv_on_consecutive_calls():
    _run(4, 14, 14, 256, 512, 3, 2, 1, 1, False, 1)   # split K in 4: partial sums in the static array
    _run(2, 14, 14, 256, 512, 3, 2, 1, 1, False, 2)   # smaller, right after
    _run(3, 9, 11, 128, 256, 3, 1, 1, 1, True, 3)     # ragged tiles, residual
    _run(2, 7, 7, 512, 512, 3, 1, 1, 1, True, 4)      # streamed-weight halo kernel (no partial sums)
    _run(1, 7, 7, 512, 512, 1, 1, 0, 0, False, 5)


def test_noalloc_conv_refuses_what_does_not_fit():
    import torch
    lib = fsb.load()
    x = torch.zeros((5, 16, 16, 256), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((1216, 3, 3, 256), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(1216, device="cuda")
    y = torch.empty((5, 16, 16, 1216), dtype=torch.bfloat16, device="cuda")
    fp = ctypes.cast(ctypes.c_void_p(b.data_ptr()), ctypes.POINTER(ctypes.c_float))
    # split K in 4 over 20 x 19 tiles: 24.9 MB of partial sums > 16 MiB
    st = lib.fs_conv_bf16_device_noalloc(ctypes.c_void_p(x.data_ptr()), 5, 16, 16, 256, ctypes.c_void_p(w.data_ptr()),
                                         fp, None, 1216, 3, 3, 1, 1, 1, ctypes.c_void_p(y.data_ptr()), None)
    assert st == fsb.FS_ERR_UNSUPPORTED and b"scratch" in lib.fs_last_error(None)
    st = lib.fs_conv_bf16_device_noalloc(None, 5, 16, 16, 256, ctypes.c_void_p(w.data_ptr()), fp, None, 1216, 3, 3,
                                         1, 1, 1, ctypes.c_void_p(y.data_ptr()), None)
    assert st == fsb.FS_ERR_INVALID
    st = lib.fs_conv_bf16_device_noalloc(ctypes.c_void_p(x.data_ptr()), 5, 16, 16, 96, ctypes.c_void_p(w.data_ptr()),
                                         fp, None, 1216, 3, 3, 1, 1, 1, ctypes.c_void_p(y.data_ptr()), None)
    assert st == fsb.FS_ERR_UNSUPPORTED  # Cin not a multiple of 64
    torch.cuda.synchronize()
