"""Host-side behaviour of the C ABI that needs no GPU: the library loads,
exports every symbol the header declares, and rejects invalid calls with
the documented status before any device work.  Without a device, a valid
create reports FS_ERR_DEVICE instead of crashing."""
import os
import re
import subprocess

import numpy as np
import pytest

import workloads as wl
from paper_2003_01538_amd import flexserve as fsb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flexserve.h")


def header_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(fs_\w+)\s*\(", txt)))


def test_header_declares_the_boundary():
    names = header_functions()
    for n in ("fs_ensemble_create", "fs_infer", "fs_infer_device", "fs_destroy", "fs_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = fsb.load()
    out = subprocess.run(["nm", "-D", "--defined-only", fsb.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (fs_\w+)", out))
    declared = set(header_functions())
    assert declared <= exported, declared - exported
    assert {n for n, _, _ in fsb.SIGNATURES} == declared
    for n in declared:
        assert hasattr(lib, n)


def _tiny_desc(**kw):
    models = [wl.build_model("tiny", 1), wl.build_model("tiny", 2)]
    for k, v in kw.pop("mutate", {}).items():
        models[k[0]][k[1]].update(v)
    args = dict(out_hw=(32, 32), mean=wl.IMAGENET_MEAN, std=wl.IMAGENET_STD, precision="fp32",
                max_batch=8)
    args.update(kw)
    return fsb.make_desc(models, **args)


def _create_status(desc):
    import ctypes
    h = ctypes.c_void_p()
    st = fsb.load().fs_ensemble_create(ctypes.byref(desc), ctypes.byref(h))
    return st, h.value, fsb.fs_last_error(None)


@pytest.mark.parametrize("combine", [fsb.FS_COMBINE_MEAN, fsb.FS_COMBINE_PLURALITY])
def test_create_valid_without_device_reports_device_error(combine):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    d, keep = _tiny_desc(combine=combine)
    st, h, msg = _create_status(d)
    assert st == fsb.FS_ERR_DEVICE and h is None and msg


@pytest.mark.parametrize("case,status", [
    (dict(max_batch=0), fsb.FS_ERR_INVALID),
    (dict(max_batch=5000), fsb.FS_ERR_INVALID),
    (dict(precision=7), fsb.FS_ERR_INVALID),
    (dict(out_hw=(0, 32)), fsb.FS_ERR_INVALID),
    (dict(std=(0.0, 1.0, 1.0)), fsb.FS_ERR_INVALID),
    (dict(mutate={(1, 4): dict(cout=11)}), fsb.FS_ERR_INVALID),          # class counts differ
    (dict(mutate={(0, 2): dict(cin=8)}), fsb.FS_ERR_INVALID),            # chain mismatch
    (dict(mutate={(0, 2): dict(src=5)}), fsb.FS_ERR_INVALID),            # forward reference
    (dict(mutate={(0, 0): dict(k=40)}), fsb.FS_ERR_INVALID),             # empty output
    (dict(mutate={(0, 2): dict(res=1)}), fsb.FS_ERR_INVALID),            # residual shape
    (dict(mutate={(0, 0): dict(cout=12), (0, 2): dict(cin=12)}), fsb.FS_ERR_UNSUPPORTED),
    (dict(mutate={(0, 4): dict(cin=31)}), fsb.FS_ERR_INVALID),           # fc fan-in
    (dict(mutate={(0, 1): dict(pad=2)}), fsb.FS_ERR_INVALID),            # pool pad >= k
    (dict(combine=fsb.FS_COMBINE_ANY), fsb.FS_ERR_INVALID),              # its class comes from fs_set_combine
    (dict(combine=9), fsb.FS_ERR_INVALID),
])
def test_create_rejects_invalid_descriptors(case, status):
    d, keep = _tiny_desc(**case)
    st, h, msg = _create_status(d)
    assert st == status, msg
    assert h is None and msg


def test_create_rejects_null_and_empty():
    import ctypes
    lib = fsb.load()
    h = ctypes.c_void_p()
    assert lib.fs_ensemble_create(None, ctypes.byref(h)) == fsb.FS_ERR_INVALID
    d = fsb.fs_ensemble_desc()
    d.num_models = 0
    assert lib.fs_ensemble_create(ctypes.byref(d), ctypes.byref(h)) == fsb.FS_ERR_INVALID
    assert "num_models" in fsb.fs_last_error(None)
    d2, keep = _tiny_desc()
    assert lib.fs_ensemble_create(ctypes.byref(d2), None) == fsb.FS_ERR_INVALID


def test_calls_on_null_handle_fail_cleanly():
    import ctypes
    lib = fsb.load()
    assert lib.fs_infer(None, None, 0, None, None, None, None, None) == fsb.FS_ERR_INVALID
    assert lib.fs_infer_device(None, None, None, 1, None, None, None, None, None, None) == fsb.FS_ERR_INVALID
    assert lib.fs_query(None, None) == fsb.FS_ERR_INVALID
    assert lib.fs_profile_enable(None, 1) == fsb.FS_ERR_INVALID
    assert lib.fs_graphs_enable(None, 1) == fsb.FS_ERR_INVALID
    assert lib.fs_set_combine(None, fsb.FS_COMBINE_PLURALITY, 0, 1) == fsb.FS_ERR_INVALID
    h = ctypes.c_void_p(1)
    assert lib.fs_ensemble_share(None, ctypes.byref(h)) == fsb.FS_ERR_INVALID and not h.value
    b = ctypes.c_void_p(1)
    assert lib.fs_batcher_create(None, 1, 100, ctypes.byref(b)) == fsb.FS_ERR_INVALID and not b.value
    nulls = (ctypes.c_void_p * 2)()
    assert lib.fs_batcher_create(nulls, 2, 100, ctypes.byref(b)) == fsb.FS_ERR_INVALID and not b.value
    assert lib.fs_batcher_create(nulls, 0, 100, ctypes.byref(b)) == fsb.FS_ERR_INVALID
    assert lib.fs_batcher_infer(None, None, 1, None, None, None, None, None) == fsb.FS_ERR_INVALID
    assert lib.fs_batcher_stats(None, None, None, None) == fsb.FS_ERR_INVALID
    assert lib.fs_batcher_last_error()
    lib.fs_batcher_destroy(None)
    lib.fs_destroy(None)


def test_test_entries_validate_before_device():
    lib = fsb.load()
    x = np.zeros((1, 4, 4, 8), np.float32)
    w = np.zeros((12, 3, 3, 8), np.float32)  # Cout not a multiple of 8
    with pytest.raises(fsb.FsError) as e:
        fsb.fs_test_conv(x, w, None, None, 1, 1, 0, fsb.FS_BF16)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    with pytest.raises(fsb.FsError) as e:
        fsb.fs_test_maxpool(np.zeros((1, 4, 4, 8), np.float32), 2, 2, 2, fsb.FS_BF16)
    assert e.value.status == fsb.FS_ERR_INVALID
    with pytest.raises(fsb.FsError) as e:
        fsb.fs_test_softmax_combine(np.zeros((1, 1, 5000), np.float32))
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    z = np.zeros((3, 2, 10), np.float32)
    for policy, pos, k, status in [(5, 0, 1, fsb.FS_ERR_INVALID),                     # unknown policy
                                   (fsb.FS_COMBINE_ANY, 10, 1, fsb.FS_ERR_INVALID),   # class out of range
                                   (fsb.FS_COMBINE_ANY, -1, 1, fsb.FS_ERR_INVALID),
                                   (fsb.FS_COMBINE_ANY, 3, 0, fsb.FS_ERR_INVALID),    # k out of 1..N
                                   (fsb.FS_COMBINE_ANY, 3, 4, fsb.FS_ERR_INVALID)]:
        with pytest.raises(fsb.FsError) as e:
            fsb.fs_test_softmax_combine_policy(z, policy, pos, k)
        assert e.value.status == status, (policy, pos, k)
    with pytest.raises(fsb.FsError) as e:
        fsb.fs_test_softmax_combine_policy(np.zeros((65, 1, 10), np.float32), fsb.FS_COMBINE_PLURALITY)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    bad = [np.zeros((0, 4, 3), np.uint8)]
    with pytest.raises(fsb.FsError) as e:
        fsb.fs_test_preprocess(bad, 8, 8, wl.IMAGENET_MEAN, wl.IMAGENET_STD, fsb.FS_F32)
    assert e.value.status == fsb.FS_ERR_INVALID
    ok = [np.zeros((4, 4, 3), np.uint8)]
    with pytest.raises(fsb.FsError) as e:  # space-to-depth needs an even size
        fsb.fs_test_preprocess(ok, 7, 8, wl.IMAGENET_MEAN, wl.IMAGENET_STD, fsb.FS_BF16, layout=1)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    assert lib.fs_conv_num_tiles(fsb.FS_BF16) >= 3 and lib.fs_conv_num_tiles(9) == 0
    assert fsb.fs_conv_tile_name(fsb.FS_BF16, 0) and fsb.fs_conv_tile_name(fsb.FS_BF16, 99) is None


@pytest.mark.parametrize("out", [1, 9, 17, 112, 224, 1000, 4096])
def test_float_reciprocal_quotient_is_exact_below_2_pow_22(out):
    # The preprocess kernel takes floor(n / d), d = 2 * out, as
    # trunc((n + 0.5) * fl(1/d)) in fp32 when n + 1 < 2^22, and the fraction
    # as (n - q d) * fl(1/d).  Every such n, in fp32 arithmetic as on the
    # device, gives the integer quotient; the fraction is within 2 ulps.
    d = 2 * out
    n = np.arange(1, (1 << 22) - 1, dtype=np.int64)
    inv = np.float32(1.0) / np.float32(d)
    q = ((n.astype(np.float32) + np.float32(0.5)) * inv).astype(np.int64)
    assert np.array_equal(q, n // d)
    frac = (n - q * d).astype(np.float32) * inv
    exact = (n % d) / d
    assert np.all(np.abs(frac.astype(np.float64) - exact) <= 2 * np.spacing(np.float32(1.0)) * np.maximum(exact, 1e-30) + 1e-12)
