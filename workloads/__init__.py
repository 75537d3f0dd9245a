"""Seeded synthetic inputs shared by the oracle side and the HIP side.

This module holds no arithmetic of the method (no resize, no convolution, no
softmax).  It only draws random numbers and writes down network *shapes*, so
that the oracle and the library can be fed byte-identical inputs:

* uint8 HWC RGB images (uniform on 0..255), possibly ragged;
* He-normal weights (fan-in, gain sqrt(2), untruncated), BN scale ~ U(0.5, 1.5)
  and shift ~ N(0, 0.1) for the ResNets, zero biases elsewhere;
* the layer lists of the tiny net, ResNet-18, ResNet-50 (v1.5) and VGG-11;
* the seeded request stream for flexible batching.

The paper asks for an ensemble of heterogeneous CNNs sharing one device
(Fig. 1 caption; Sec. 2.1 on different architectures; Sec. 2.2) and for
variable batch sizes (Sec. 2.3).  The concrete networks and seeds are the
workload recipe of this repository; the paper itself names none.

Layer dictionaries (``op`` is one of ``conv``, ``maxpool``, ``gap``, ``fc``):

* ``src``: index of the layer whose output is consumed, -1 = the shared
  transformed input batch.
* ``res``: conv only, index of the layer added as residual before the ReLU,
  or -1.
* conv: ``cin, cout, k, stride, pad, relu, weight [cout][k][k][cin] f32,
  bias [cout] or None, bn_scale/bn_shift [cout] or None``.
* maxpool: ``k, stride, pad``.
* fc: ``cin, cout, relu, weight [cout][cin] f32, bias or None, flatten_nchw``
  (True when the input is a feature map flattened in channel-major order).
"""
from __future__ import annotations

import numpy as np

IMAGENET_MEAN = (0.485, 0.456, 0.406)
IMAGENET_STD = (0.229, 0.224, 0.225)


# --------------------------------------------------------------------------
# images
# --------------------------------------------------------------------------
def images_uniform(seed: int, B: int, h: int, w: int) -> np.ndarray:
    """[B, h, w, 3] uint8, uniform on 0..255 inclusive."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(B, h, w, 3), dtype=np.uint8)


def images_ragged(seed: int, B: int, lo: int = 160, hi: int = 320):
    """List of B uint8 HWC images whose h and w are independent uniform
    integers on [lo, hi]."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(B):
        h = int(rng.integers(lo, hi + 1))
        w = int(rng.integers(lo, hi + 1))
        out.append(rng.integers(0, 256, size=(h, w, 3), dtype=np.uint8))
    return out


def request_stream(seed: int, n_requests: int = 200,
                   sizes=(1, 2, 3, 5, 7, 16, 31, 64), lo: int = 160, hi: int = 320):
    """Seeded stream of requests: each a list of ragged images.  Batch sizes
    are uniform over ``sizes``."""
    rng = np.random.default_rng(seed)
    reqs = []
    for _ in range(n_requests):
        B = int(sizes[int(rng.integers(0, len(sizes)))])
        imgs = []
        for _ in range(B):
            h = int(rng.integers(lo, hi + 1))
            w = int(rng.integers(lo, hi + 1))
            imgs.append(rng.integers(0, 256, size=(h, w, 3), dtype=np.uint8))
        reqs.append(imgs)
    return reqs


def pack_images(imgs):
    """Pack a list (or [B,h,w,3] array) of uint8 HWC images into one flat
    uint8 buffer plus a descriptor array of (offset, h, w, row_stride).
    Rows are stored densely (row_stride = 3*w)."""
    if isinstance(imgs, np.ndarray):
        imgs = [imgs[i] for i in range(imgs.shape[0])]
    offs, desc = 0, []
    for im in imgs:
        h, w, _ = im.shape
        desc.append((offs, h, w, 3 * w))
        offs += h * w * 3
    flat = np.empty(offs, dtype=np.uint8)
    for im, (o, h, w, _) in zip(imgs, desc):
        flat[o:o + h * w * 3] = np.ascontiguousarray(im).reshape(-1)
    return flat, desc


# --------------------------------------------------------------------------
# network shapes
# --------------------------------------------------------------------------
def _conv(src, cin, cout, k, stride, pad, relu, res=-1, bn=False):
    return dict(op="conv", src=src, res=res, cin=cin, cout=cout, k=k, stride=stride,
                pad=pad, relu=int(relu), bn=bn)


def tiny_layers():
    """conv3x3 3->16 p1 + ReLU, maxpool 2, conv3x3 16->32 p1 + ReLU, global
    average pool, FC 32->10."""
    return [
        _conv(-1, 3, 16, 3, 1, 1, True),
        dict(op="maxpool", src=0, k=2, stride=2, pad=0),
        _conv(1, 16, 32, 3, 1, 1, True),
        dict(op="gap", src=2),
        dict(op="fc", src=3, cin=32, cout=10, relu=0, flatten_nchw=False),
    ]


def resnet_layers(depth: int, num_classes: int = 1000):
    """ResNet-18 (basic blocks [2,2,2,2]) or ResNet-50 (bottlenecks [3,4,6,3],
    expansion 4, stride on the 3x3).  BN follows every conv and is folded."""
    L = [_conv(-1, 3, 64, 7, 2, 3, True, bn=True),
         dict(op="maxpool", src=0, k=3, stride=2, pad=1)]
    x, cin = 1, 64
    if depth == 18:
        for stage, (width, nblk) in enumerate(zip((64, 128, 256, 512), (2, 2, 2, 2))):
            for blk in range(nblk):
                s = 2 if (stage > 0 and blk == 0) else 1
                L.append(_conv(x, cin, width, 3, s, 1, True, bn=True))
                c1 = len(L) - 1
                res = x
                if s != 1 or cin != width:
                    L.append(_conv(x, cin, width, 1, s, 0, False, bn=True))
                    res = len(L) - 1
                L.append(_conv(c1, width, width, 3, 1, 1, True, res=res, bn=True))
                x, cin = len(L) - 1, width
        feat = 512
    elif depth == 50:
        for stage, (mid, nblk) in enumerate(zip((64, 128, 256, 512), (3, 4, 6, 3))):
            out = 4 * mid
            for blk in range(nblk):
                s = 2 if (stage > 0 and blk == 0) else 1
                L.append(_conv(x, cin, mid, 1, 1, 0, True, bn=True))
                a = len(L) - 1
                L.append(_conv(a, mid, mid, 3, s, 1, True, bn=True))
                b = len(L) - 1
                res = x
                if s != 1 or cin != out:
                    L.append(_conv(x, cin, out, 1, s, 0, False, bn=True))
                    res = len(L) - 1
                L.append(_conv(b, mid, out, 1, 1, 0, True, res=res, bn=True))
                x, cin = len(L) - 1, out
        feat = 2048
    else:
        raise ValueError(depth)
    L.append(dict(op="gap", src=x))
    L.append(dict(op="fc", src=len(L) - 1, cin=feat, cout=num_classes, relu=0,
                  flatten_nchw=False))
    return L


def vgg11_layers(num_classes: int = 1000):
    """VGG-11 (configuration A): conv3x3 p1 + ReLU, 2x2 max pools, no BN, then
    FC 25088->4096->4096->num_classes on the channel-major flattened map."""
    cfg = (64, "M", 128, "M", 256, 256, "M", 512, 512, "M", 512, 512, "M")
    L, x, cin = [], -1, 3
    for v in cfg:
        if v == "M":
            L.append(dict(op="maxpool", src=x, k=2, stride=2, pad=0))
        else:
            L.append(_conv(x, cin, v, 3, 1, 1, True))
            cin = v
        x = len(L) - 1
    L.append(dict(op="fc", src=x, cin=512 * 7 * 7, cout=4096, relu=1, flatten_nchw=True))
    L.append(dict(op="fc", src=len(L) - 1, cin=4096, cout=4096, relu=1, flatten_nchw=False))
    L.append(dict(op="fc", src=len(L) - 1, cin=4096, cout=num_classes, relu=0,
                  flatten_nchw=False))
    return L


ARCHS = {
    "tiny": tiny_layers,
    "resnet18": lambda: resnet_layers(18),
    "resnet50": lambda: resnet_layers(50),
    "vgg11": vgg11_layers,
}


def init_weights(layers, seed: int):
    """Fill He-normal weights (fan-in = cin*k*k for conv, cin for FC), BN
    scale/shift for layers flagged ``bn``, and zero biases, drawing from one
    generator in layer-list order: per layer W (C-order), then scale, then
    shift.  Returns a new list of dicts."""
    rng = np.random.default_rng(seed)
    out = []
    for L in layers:
        L = dict(L)
        if L["op"] == "conv":
            cin, cout, k = L["cin"], L["cout"], L["k"]
            std = np.sqrt(2.0 / (cin * k * k))
            L["weight"] = (rng.standard_normal((cout, k, k, cin)) * std).astype(np.float32)
            if L.pop("bn", False):
                L["bn_scale"] = rng.uniform(0.5, 1.5, cout).astype(np.float32)
                L["bn_shift"] = (rng.standard_normal(cout) * 0.1).astype(np.float32)
                L["bias"] = None
            else:
                L["bn_scale"] = L["bn_shift"] = None
                L["bias"] = np.zeros(cout, np.float32)
        elif L["op"] == "fc":
            std = np.sqrt(2.0 / L["cin"])
            L["weight"] = (rng.standard_normal((L["cout"], L["cin"])) * std).astype(np.float32)
            L["bias"] = np.zeros(L["cout"], np.float32)
        out.append(L)
    return out


def build_model(arch: str, seed: int):
    return init_weights(ARCHS[arch](), seed)


def num_classes(layers) -> int:
    return layers[-1]["cout"]


# --------------------------------------------------------------------------
# the five workload recipes
# --------------------------------------------------------------------------
WORKLOADS = {
    # name: (archs, precision, batch, in_h, in_w, out_h, out_w, image seed, model seeds)
    "tiny2_fp32_b4": (("tiny", "tiny"), "fp32", 4, 32, 32, 32, 32, 1000, (1001, 1002)),
    "resnet18x3_bf16_b32": (("resnet18",) * 3, "bf16", 32, 256, 256, 224, 224, 2000,
                            (2001, 2002, 2003)),
    "hetero_r18_r50_vgg11_bf16_b32": (("resnet18", "resnet50", "vgg11"), "bf16", 32,
                                      224, 224, 224, 224, 4000, (4001, 4002, 4003)),
    "resnet50x5_bf16_b256": (("resnet50",) * 5, "bf16", 256, 224, 224, 224, 224, 5000,
                             (5001, 5002, 5003, 5004, 5005)),
}
STREAM_WORKLOAD = dict(name="resnet18x3_bf16_stream200", ensemble="resnet18x3_bf16_b32",
                       seed=3000, n_requests=200, sizes=(1, 2, 3, 5, 7, 16, 31, 64),
                       lo=160, hi=320)


def workload(name: str):
    archs, prec, B, ih, iw, oh, ow, iseed, mseeds = WORKLOADS[name]
    models = [build_model(a, s) for a, s in zip(archs, mseeds)]
    return dict(name=name, archs=archs, precision=prec, batch=B, in_hw=(ih, iw),
                out_hw=(oh, ow), image_seed=iseed, models=models)


# --------------------------------------------------------------------------
# shape bookkeeping (no arithmetic of the method: only counting)
# --------------------------------------------------------------------------
def layer_shapes(layers, in_h: int, in_w: int):
    """Per layer output shape (H, W, C), or (1, 1, C) for gap/fc."""
    shapes = []
    for L in layers:
        H, W, C = (in_h, in_w, 3) if L["src"] < 0 else shapes[L["src"]]
        if L["op"] in ("conv", "maxpool"):
            k, s, p = L["k"], L["stride"], L["pad"]
            Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
            shapes.append((Ho, Wo, L["cout"] if L["op"] == "conv" else C))
        else:
            shapes.append((1, 1, L["cout"] if L["op"] == "fc" else C))
    return shapes


def count_flops_params(layers, in_h: int = 224, in_w: int = 224):
    """(multiply-accumulates per image over conv+fc, parameters with BN folded)."""
    shapes = layer_shapes(layers, in_h, in_w)
    macs = params = 0
    for L, (Ho, Wo, C) in zip(layers, shapes):
        if L["op"] == "conv":
            kk = L["k"] * L["k"] * L["cin"]
            macs += Ho * Wo * L["cout"] * kk
            params += L["cout"] * kk + L["cout"]
        elif L["op"] == "fc":
            macs += L["cin"] * L["cout"]
            params += L["cin"] * L["cout"] + L["cout"]
    return macs, params
