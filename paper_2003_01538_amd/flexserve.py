"""Thin ctypes binding of the C ABI in include/flexserve.h.

Argument marshalling only: every step of the path runs in the HIP library
(libflexserve.so, built by ``paper_2003_01538_amd.build``).  The functions
keep the C names.  Loading fails loudly when the library is missing; there is
no fallback.

torch is imported before the library is loaded so that the process holds a
single HIP runtime (torch's), shared by torch tensors and the library; torch
serves only as device memory and stream plumbing for callers of the
device-pointer entry point.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflexserve.so")

FS_OK, FS_ERR_INVALID, FS_ERR_OOM, FS_ERR_DEVICE, FS_ERR_UNSUPPORTED, FS_ERR_INTERNAL = range(6)
FS_F32, FS_BF16 = 0, 1
FS_OP_CONV, FS_OP_MAXPOOL, FS_OP_GAP, FS_OP_FC = range(4)
FS_COMBINE_MEAN, FS_COMBINE_PLURALITY, FS_COMBINE_ANY = range(3)
STATUS_NAMES = {0: "FS_OK", 1: "FS_ERR_INVALID", 2: "FS_ERR_OOM", 3: "FS_ERR_DEVICE",
                4: "FS_ERR_UNSUPPORTED", 5: "FS_ERR_INTERNAL"}

_fp = ctypes.POINTER(ctypes.c_float)
_i32p = ctypes.POINTER(ctypes.c_int32)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_vp = ctypes.c_void_p


class fs_layer(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("src", ctypes.c_int32), ("residual_src", ctypes.c_int32),
                ("cin", ctypes.c_int32), ("cout", ctypes.c_int32), ("kh", ctypes.c_int32),
                ("kw", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("relu", ctypes.c_int32), ("flatten_nchw", ctypes.c_int32),
                ("weight", _fp), ("bias", _fp), ("bn_scale", _fp), ("bn_shift", _fp)]


class fs_model_spec(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("layers", ctypes.POINTER(fs_layer)),
                ("num_classes", ctypes.c_int32)]


class fs_preprocess(ctypes.Structure):
    _fields_ = [("out_h", ctypes.c_int32), ("out_w", ctypes.c_int32),
                ("mean", ctypes.c_float * 3), ("std", ctypes.c_float * 3)]


class fs_ensemble_desc(ctypes.Structure):
    _fields_ = [("num_models", ctypes.c_int32), ("models", ctypes.POINTER(fs_model_spec)),
                ("pre", fs_preprocess), ("precision", ctypes.c_int32), ("combine", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("device", ctypes.c_int32)]


class fs_image(ctypes.Structure):
    _fields_ = [("data", _u8p), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("row_stride", ctypes.c_int32)]


class fs_image_desc(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_uint64), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("row_stride", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class fs_info(ctypes.Structure):
    _fields_ = [("num_models", ctypes.c_int32), ("num_classes", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("precision", ctypes.c_int32),
                ("num_groups", ctypes.c_int32), ("launches_per_pass", ctypes.c_int32),
                ("weight_bytes", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
                ("flops_per_image", ctypes.c_double)]


class fs_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


class fs_launch_stat(ctypes.Structure):
    _fields_ = [("kclass", ctypes.c_char * 16), ("kernel", ctypes.c_char * 32),
                ("group", ctypes.c_int32), ("layer", ctypes.c_int32), ("M", ctypes.c_int32),
                ("N", ctypes.c_int32), ("K", ctypes.c_int32), ("Z", ctypes.c_int32),
                ("ms", ctypes.c_double), ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


# every symbol include/flexserve.h declares: (name, restype, argtypes)
SIGNATURES = [
    ("fs_ensemble_create", ctypes.c_int, [ctypes.POINTER(fs_ensemble_desc), ctypes.POINTER(_vp)]),
    ("fs_infer", ctypes.c_int, [_vp, ctypes.POINTER(fs_image), ctypes.c_int32, _fp, _fp, _i32p, _i32p, _fp]),
    ("fs_infer_device", ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp, _vp]),
    ("fs_destroy", None, [_vp]),
    ("fs_last_error", ctypes.c_char_p, [_vp]),
    ("fs_query", ctypes.c_int, [_vp, ctypes.POINTER(fs_info)]),
    ("fs_profile_enable", ctypes.c_int, [_vp, ctypes.c_int32]),
    ("fs_graphs_enable", ctypes.c_int, [_vp, ctypes.c_int32]),
    ("fs_set_combine", ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    ("fs_ensemble_share", ctypes.c_int, [_vp, ctypes.POINTER(_vp)]),
    ("fs_batcher_create", ctypes.c_int, [ctypes.POINTER(_vp), ctypes.c_int32, ctypes.c_int32,
                                         ctypes.POINTER(_vp)]),
    ("fs_batcher_infer", ctypes.c_int, [_vp, ctypes.POINTER(fs_image), ctypes.c_int32, _fp, _fp, _i32p, _i32p,
                                        _fp]),
    ("fs_batcher_stats", ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int64)]),
    ("fs_batcher_last_error", ctypes.c_char_p, []),
    ("fs_batcher_destroy", None, [_vp]),
    ("fs_profile_read", ctypes.c_int, [_vp, ctypes.POINTER(fs_kernel_stat), ctypes.c_int32, _i32p]),
    ("fs_profile_launches", ctypes.c_int, [_vp, ctypes.POINTER(fs_launch_stat), ctypes.c_int32, _i32p]),
    ("fs_infer_phases", ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_double)]),
    ("fs_tuning_log", ctypes.c_int, [_vp, ctypes.c_char_p, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]),
    ("fs_debug_capture", ctypes.c_int, [_vp, ctypes.c_int32]),
    ("fs_debug_layer", ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, _fp, ctypes.c_int64]),
    ("fs_test_preprocess", ctypes.c_int, [ctypes.POINTER(fs_image), ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_int32, _fp, _fp, ctypes.c_int32, ctypes.c_int32, _fp,
                                          ctypes.c_int32]),
    ("fs_test_conv", ctypes.c_int, [_fp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    _fp, _fp, _fp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, _fp, ctypes.c_int32]),
    ("fs_test_stem_pool", ctypes.c_int, [_fp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _fp, _fp, _fp,
                                         ctypes.c_int32]),
    ("fs_test_maxpool", ctypes.c_int, [_fp] + [ctypes.c_int32] * 8 + [_fp, ctypes.c_int32]),
    ("fs_test_gap", ctypes.c_int, [_fp] + [ctypes.c_int32] * 5 + [_fp, ctypes.c_int32]),
    ("fs_test_fc", ctypes.c_int, [_fp, ctypes.c_int32, ctypes.c_int32, _fp, _fp, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _fp, ctypes.c_int32]),
    ("fs_test_softmax_combine", ctypes.c_int, [_fp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               _fp, _fp, _i32p, _i32p, ctypes.c_int32]),
    ("fs_test_softmax_combine_policy", ctypes.c_int, [_fp] + [ctypes.c_int32] * 6 +
                                                     [_fp, _fp, _i32p, _i32p, ctypes.c_int32]),
    ("fs_bench_conv", ctypes.c_int, [ctypes.c_int32] * 15 + [ctypes.POINTER(ctypes.c_double), _i32p,
                                                         ctypes.c_int32]),
    ("fs_conv_bf16_device_noalloc", ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                   ctypes.c_int32, _vp, _fp, _vp] + [ctypes.c_int32] * 6 +
                                                  [_vp, _vp]),
    ("fs_conv_num_tiles", ctypes.c_int32, [ctypes.c_int32]),
    ("fs_conv_tile_name", ctypes.c_char_p, [ctypes.c_int32, ctypes.c_int32]),
]

_lib = None


class FsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def load(path: str = LIB_PATH):
    """Load libflexserve.so (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library not built: {path} (run python -m paper_2003_01538_amd.build)")
    try:
        import torch  # noqa: F401  -- one HIP runtime per process: torch's
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _f(a):
    return None if a is None else a.ctypes.data_as(_fp)


def _i(a):
    return None if a is None else a.ctypes.data_as(_i32p)


def _check(st, handle=None):
    if st != FS_OK:
        msg = load().fs_last_error(handle)
        raise FsError(st, msg.decode() if msg else "")


# ------------------------------------------------------------ descriptors
_OPS = {"conv": FS_OP_CONV, "maxpool": FS_OP_MAXPOOL, "gap": FS_OP_GAP, "fc": FS_OP_FC}


def make_desc(models, out_hw, mean, std, precision, max_batch, device=0, combine=FS_COMBINE_MEAN):
    """Marshal layer dictionaries (see the ``workloads`` module) into an
    fs_ensemble_desc.  Returns (desc, keepalive)."""
    keep = []
    specs = (fs_model_spec * len(models))()
    for mi, layers in enumerate(models):
        arr = (fs_layer * len(layers))()
        for i, L in enumerate(layers):
            x = arr[i]
            x.op = _OPS[L["op"]]
            x.src = L["src"]
            x.residual_src = L.get("res", -1)
            if L["op"] == "conv":
                x.cin, x.cout, x.kh, x.kw = L["cin"], L["cout"], L["k"], L["k"]
                x.stride, x.pad, x.relu = L["stride"], L["pad"], L["relu"]
            elif L["op"] == "maxpool":
                x.kh = x.kw = L["k"]
                x.stride, x.pad = L["stride"], L["pad"]
            elif L["op"] == "fc":
                x.cin, x.cout, x.relu = L["cin"], L["cout"], L["relu"]
                x.flatten_nchw = int(bool(L.get("flatten_nchw")))
            for fld, key in (("weight", "weight"), ("bias", "bias"), ("bn_scale", "bn_scale"),
                             ("bn_shift", "bn_shift")):
                v = L.get(key)
                if v is not None:
                    v = np.ascontiguousarray(v, dtype=np.float32)
                    keep.append(v)
                    setattr(x, fld, _f(v))
        keep.append(arr)
        specs[mi].num_layers = len(layers)
        specs[mi].layers = arr
        specs[mi].num_classes = layers[-1]["cout"] if layers else 0
    d = fs_ensemble_desc()
    d.num_models = len(models)
    d.models = specs
    d.pre.out_h, d.pre.out_w = out_hw
    for c in range(3):
        d.pre.mean[c] = mean[c]
        d.pre.std[c] = std[c]
    d.precision = {"fp32": FS_F32, "bf16": FS_BF16}.get(precision, precision)
    d.combine = combine
    d.max_batch = max_batch
    d.device = device
    keep.append(specs)
    return d, keep


def image_array(imgs):
    """fs_image[] over a list of uint8 HWC arrays (strided rows allowed)."""
    arr = (fs_image * len(imgs))()
    keep = []
    for i, im in enumerate(imgs):
        im = np.asarray(im)
        if im.dtype != np.uint8 or im.ndim != 3 or im.shape[2] != 3 or im.strides[2] != 1 \
                or im.strides[1] != 3:
            im = np.ascontiguousarray(im, dtype=np.uint8)
        keep.append(im)
        arr[i].data = im.ctypes.data_as(_u8p)
        arr[i].h, arr[i].w = im.shape[0], im.shape[1]
        arr[i].row_stride = im.strides[0]
    return arr, keep


# ----------------------------------------------------------------- C names
def fs_ensemble_create(desc) -> int:
    h = _vp()
    _check(load().fs_ensemble_create(ctypes.byref(desc), ctypes.byref(h)))
    return h.value


def fs_infer(handle, imgs, N, C, want_mean=True, want_top1=True, want_logits=True):
    B = len(imgs)
    probs = np.zeros((N, B, C), np.float32)
    mean = np.zeros((B, C), np.float32) if want_mean else None
    vote = np.zeros(B, np.int32)
    top1 = np.zeros((N, B), np.int32) if want_top1 else None
    logits = np.zeros((N, B, C), np.float32) if want_logits else None
    arr, keep = image_array(imgs)
    _check(load().fs_infer(handle, arr, B, _f(probs), _f(mean), _i(vote), _i(top1), _f(logits)), handle)
    return dict(probs=probs, mean=mean, vote=vote, top1=top1, logits=logits)


def fs_infer_device(handle, d_pixels, d_desc, B, d_probs, d_mean, d_vote, d_top1, d_logits, stream=0):
    """All pointers are integer device addresses (e.g. torch data_ptr())."""
    _check(load().fs_infer_device(handle, d_pixels, d_desc, B, d_probs, d_mean or None, d_vote,
                                  d_top1 or None, d_logits or None, stream or None), handle)


def fs_destroy(handle):
    load().fs_destroy(handle)


def fs_last_error(handle=None) -> str:
    m = load().fs_last_error(handle)
    return m.decode() if m else ""


def fs_query(handle) -> dict:
    info = fs_info()
    _check(load().fs_query(handle, ctypes.byref(info)), handle)
    return {k: getattr(info, k) for k, _ in fs_info._fields_}


def fs_graphs_enable(handle, enable=True):
    _check(load().fs_graphs_enable(handle, int(bool(enable))), handle)


def fs_ensemble_share(handle) -> int:
    h = _vp()
    _check(load().fs_ensemble_share(handle, ctypes.byref(h)))
    return h.value


def _check_batcher(st):
    if st != FS_OK:
        m = load().fs_batcher_last_error()
        raise FsError(st, m.decode() if m else "")


def fs_batcher_create(handles, max_wait_us=2000) -> int:
    arr = (_vp * len(handles))(*handles)
    b = _vp()
    _check_batcher(load().fs_batcher_create(arr, len(handles), int(max_wait_us), ctypes.byref(b)))
    return b.value


def fs_batcher_infer(batcher, imgs, N, C, want_mean=True, want_top1=True, want_logits=False):
    B = len(imgs)
    probs = np.zeros((N, B, C), np.float32)
    mean = np.zeros((B, C), np.float32) if want_mean else None
    vote = np.zeros(B, np.int32)
    top1 = np.zeros((N, B), np.int32) if want_top1 else None
    logits = np.zeros((N, B, C), np.float32) if want_logits else None
    arr, keep = image_array(imgs)
    _check_batcher(load().fs_batcher_infer(batcher, arr, B, _f(probs), _f(mean), _i(vote), _i(top1),
                                           _f(logits)))
    return dict(probs=probs, mean=mean, vote=vote, top1=top1, logits=logits)


def fs_batcher_stats(batcher) -> dict:
    p, r, i = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check_batcher(load().fs_batcher_stats(batcher, ctypes.byref(p), ctypes.byref(r), ctypes.byref(i)))
    return dict(passes=p.value, requests=r.value, images=i.value)


def fs_batcher_destroy(batcher):
    load().fs_batcher_destroy(batcher)


def fs_set_combine(handle, policy, positive_class=0, min_votes=1):
    _check(load().fs_set_combine(handle, int(policy), int(positive_class), int(min_votes)), handle)


def fs_profile_enable(handle, enable=True):
    _check(load().fs_profile_enable(handle, int(bool(enable))), handle)


def fs_profile_read(handle) -> dict:
    stats = (fs_kernel_stat * 16)()
    n = ctypes.c_int32()
    _check(load().fs_profile_read(handle, stats, 16, ctypes.byref(n)), handle)
    return {stats[i].name.decode(): dict(launches=stats[i].launches, total_ms=stats[i].total_ms,
                                         flops=stats[i].flops, bytes=stats[i].bytes)
            for i in range(n.value)}


def fs_profile_launches(handle, max_out=4096) -> list:
    out = (fs_launch_stat * max_out)()
    n = ctypes.c_int32()
    _check(load().fs_profile_launches(handle, out, max_out, ctypes.byref(n)), handle)
    res = []
    for i in range(n.value):
        r = out[i]
        res.append(dict(kclass=r.kclass.decode(), kernel=r.kernel.decode(), group=r.group, layer=r.layer,
                        M=r.M, N=r.N, K=r.K, Z=r.Z, ms=r.ms, flops=r.flops, bytes=r.bytes))
    return res


def fs_tuning_log(handle) -> str:
    """Every candidate timing of the tile tuner so far, one line each."""
    need = ctypes.c_int64()
    _check(load().fs_tuning_log(handle, None, 0, ctypes.byref(need)), handle)
    buf = ctypes.create_string_buffer(need.value)
    _check(load().fs_tuning_log(handle, buf, need.value, None), handle)
    return buf.value.decode()


def fs_infer_phases(handle):
    """Host-side phase times (ms) of the handle's last fs_infer."""
    ms = (ctypes.c_double * 5)()
    _check(load().fs_infer_phases(handle, ms), handle)
    return dict(zip(("stage_upload", "issue_pass", "issue_download", "sync", "copy_out"), list(ms)))


def fs_debug_capture(handle, image):
    _check(load().fs_debug_capture(handle, image), handle)


def fs_debug_layer(handle, model, layer, shape):
    """The captured output of one layer of one model (fp32 array of `shape`)."""
    out = np.empty(shape, np.float32)
    _check(load().fs_debug_layer(handle, model, layer, _f(out), out.size), handle)
    return out


def fs_test_preprocess(imgs, out_h, out_w, mean, std, precision, layout=0, device=0):
    B = len(imgs)
    shape = (B, out_h, out_w, 4) if layout == 0 else (B, out_h // 2, out_w // 2, 16)
    out = np.zeros(shape, np.float32)
    arr, keep = image_array(imgs)
    m = np.asarray(mean, np.float32)
    s = np.asarray(std, np.float32)
    _check(load().fs_test_preprocess(arr, B, out_h, out_w, _f(m), _f(s), precision, layout, _f(out), device))
    return out


def fs_test_conv(x, w, bias, res, stride, pad, relu, precision, tile=-1, device=0):
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    B, H, W, Cin = x.shape
    Cout, kh, kw, _ = w.shape
    Ho, Wo = (H + 2 * pad - kh) // stride + 1, (W + 2 * pad - kw) // stride + 1
    out = np.zeros((B, Ho, Wo, Cout), np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    r = None if res is None else np.ascontiguousarray(res, np.float32)
    _check(load().fs_test_conv(_f(x), B, H, W, Cin, _f(w), _f(b), _f(r), Cout, kh, kw, stride, pad,
                               int(relu), precision, tile, _f(out), device))
    return out


def fs_test_stem_pool(x, w, bias, device=0):
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    B, H, W, _ = x.shape
    Ho, Wo = H // 2, W // 2
    out = np.zeros((B, (Ho - 1) // 2 + 1, (Wo - 1) // 2 + 1, 64), np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    _check(load().fs_test_stem_pool(_f(x), B, H, W, _f(w), _f(b), _f(out), device))
    return out


def fs_test_maxpool(x, k, stride, pad, precision, device=0):
    x = np.ascontiguousarray(x, np.float32)
    B, H, W, C = x.shape
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    out = np.zeros((B, Ho, Wo, C), np.float32)
    _check(load().fs_test_maxpool(_f(x), B, H, W, C, k, stride, pad, precision, _f(out), device))
    return out


def fs_test_gap(x, precision, device=0):
    x = np.ascontiguousarray(x, np.float32)
    B, H, W, C = x.shape
    out = np.zeros((B, C), np.float32)
    _check(load().fs_test_gap(_f(x), B, H, W, C, precision, _f(out), device))
    return out


def fs_test_fc(x, w, bias, relu, precision, out_storage=False, device=0):
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    B, K = x.shape
    N = w.shape[0]
    out = np.zeros((B, N), np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    _check(load().fs_test_fc(_f(x), B, K, _f(w), _f(b), N, int(relu), precision, int(out_storage),
                             _f(out), device))
    return out


def fs_test_softmax_combine(logits, device=0):
    z = np.ascontiguousarray(logits, np.float32)
    N, B, C = z.shape
    probs = np.zeros_like(z)
    mean = np.zeros((B, C), np.float32)
    vote = np.zeros(B, np.int32)
    top1 = np.zeros((N, B), np.int32)
    _check(load().fs_test_softmax_combine(_f(z), N, B, C, _f(probs), _f(mean), _i(vote), _i(top1), device))
    return dict(probs=probs, mean=mean, vote=vote, top1=top1)


def fs_test_softmax_combine_policy(logits, policy, positive_class=0, min_votes=1, device=0):
    z = np.ascontiguousarray(logits, np.float32)
    N, B, C = z.shape
    probs = np.zeros_like(z)
    mean = np.zeros((B, C), np.float32)
    vote = np.zeros(B, np.int32)
    top1 = np.zeros((N, B), np.int32)
    _check(load().fs_test_softmax_combine_policy(_f(z), N, B, C, int(policy), int(positive_class),
                                                 int(min_votes), _f(probs), _f(mean), _i(vote), _i(top1),
                                                 device))
    return dict(probs=probs, mean=mean, vote=vote, top1=top1)


def fs_bench_conv(B, H, W, Cin, Cout, k, stride, pad, relu=1, residual=0, precision=FS_BF16, tile=-1,
                  Z=1, iters=20, device=0):
    """Mean time (ms) of one launch of the conv kernel on this shape, and the
    tile used."""
    ms = ctypes.c_double()
    used = ctypes.c_int32()
    _check(load().fs_bench_conv(B, H, W, Cin, Cout, k, k, stride, pad, relu, residual, precision, tile, Z,
                                iters, ctypes.byref(ms), ctypes.byref(used), device))
    return ms.value, used.value


def fs_conv_num_tiles(precision) -> int:
    return load().fs_conv_num_tiles(precision)


def fs_conv_tile_name(precision, tile) -> str:
    n = load().fs_conv_tile_name(precision, tile)
    return n.decode() if n else None


# ------------------------------------------------------------ convenience
class Ensemble:
    """An ensemble handle built from layer dictionaries."""

    def __init__(self, models, out_hw, mean, std, precision="bf16", max_batch=256, device=0,
                 combine=FS_COMBINE_MEAN):
        desc, keep = make_desc(models, out_hw, mean, std, precision, max_batch, device, combine)
        self.handle = fs_ensemble_create(desc)
        self.N = len(models)
        self.C = models[0][-1]["cout"]
        del keep  # the library copied every weight

    def infer(self, imgs, **kw):
        return fs_infer(self.handle, imgs, self.N, self.C, **kw)

    def info(self):
        return fs_query(self.handle)

    def set_combine(self, policy, positive_class=0, min_votes=1):
        fs_set_combine(self.handle, policy, positive_class, min_votes)

    def share(self):
        """A second handle on the same device weights (fs_ensemble_share)."""
        other = Ensemble.__new__(Ensemble)
        other.handle = fs_ensemble_share(self.handle)
        other.N, other.C = self.N, self.C
        return other

    def close(self):
        if self.handle:
            fs_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()


class Batcher:
    """Request coalescing over handles of one ensemble (fs_batcher_*): one
    worker per Ensemble given (the first and handles from its share())."""

    def __init__(self, ens, max_wait_us=2000):
        self.handles = list(ens) if isinstance(ens, (list, tuple)) else [ens]  # must outlive the batcher
        self.b = fs_batcher_create([h.handle for h in self.handles], max_wait_us)

    def infer(self, imgs, **kw):
        return fs_batcher_infer(self.b, imgs, self.handles[0].N, self.handles[0].C, **kw)

    def stats(self):
        return fs_batcher_stats(self.b)

    def close(self):
        if self.b:
            fs_batcher_destroy(self.b)
            self.b = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()
