"""Layer-by-layer parity of whole ensembles at the full workload shapes.

The end-to-end comparison of a random bf16 network is chaotic: one bf16
rounding that lands on the other side early in the network moves late
logits by a few per cent of their spread, and the oracle's own result moves
as much when only its summation order changes.  Here every layer of every
model is checked alone instead: the GPU pass stores one image's output of
each layer (fs_debug_capture), the oracle's same layer is fed the GPU's
stored input (and stored residual), and the two outputs are compared at
the per-kernel bound -- the same bf16 inputs on both sides, so only the
order of the fp32 sums differs:
  bf16 storage: |gpu - oracle| <= 1 bf16 ulp + 2^-16 * sum|x*w| per
  output and >= 99 % of the outputs bit-identical; fp32 logits and fp32
  storage: |gpu - oracle| <= 1e-5 * sum|x*w| + 1e-6; max pool bit-exact.
A conv whose max pool or average pool runs inside its launch has no stored
output; the oracle then runs conv + pool on the stored input, and the bound
carries through the pool (|max a - max b| <= max |a - b|; an average of
bounded errors is bounded by their average, plus one rounding).  A
projection shortcut computed inside its block's last conv has no stored
output either: that conv is checked against the oracle's sum of both
reductions, from the stored block input.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from paper_2003_01538_amd import flexserve as fsb
from tests.test_gpu_kernels import ulp_bf16

pytestmark = pytest.mark.gpu
MEAN, STD = wl.IMAGENET_MEAN, wl.IMAGENET_STD


def _bound_check(g, o, tol, what, frac_exact, exact_report):
    g, o = np.asarray(g, np.float32), np.asarray(o, np.float32)
    bad = np.abs(g - o) > tol
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} outside the bound; max err {np.abs(g - o).max()}"
    exact = float(np.mean(g.view(np.uint32) == o.view(np.uint32)))
    exact_report.append((what, exact))
    assert exact >= frac_exact, f"{what}: only {exact:.4f} bit-identical"


def _fc_abs(x, w):
    return np.abs(x.astype(np.float64)) @ np.abs(w.astype(np.float64)).T


def check_layers(ens, layers, prepared, prec, imgs, image, model, out_hw, exact_report):
    """Every layer of `model` for image `image` of the pass over imgs (the
    capture must be armed and the pass run)."""
    shapes = wl.layer_shapes(layers, *out_hw)
    h = ens.handle
    x_in = fsb.fs_debug_layer(h, model, -1, (1,) + tuple(out_hw) + (3,))
    o_in = oracle.preprocess(imgs[image], out_hw[0], out_hw[1], MEAN, STD, prec)[None]
    if prec == "bf16":
        _bound_check(x_in, o_in, ulp_bf16(o_in) + 2e-6, f"model {model} input", 0.99, exact_report)
    else:
        assert np.all(np.abs(x_in - o_in) <= 1e-6 + 1e-6 * np.abs(o_in))
    stored = {}

    def get(li):
        if li < 0:
            return x_in
        if li not in stored:
            H, W, C = shapes[li]
            stored[li] = fsb.fs_debug_layer(h, model, li, (1, H, W, C))
        return stored[li]

    last = len(layers) - 1
    fused = set()  # convs whose output is never stored
    for li, L in enumerate(layers):
        what = f"model {model} layer {li} ({L['op']})"
        try:
            y = get(li)
        except fsb.FsError as e:
            assert e.status == fsb.FS_ERR_UNSUPPORTED and L["op"] == "conv", what
            fused.add(li)
            continue
        src = L["src"]
        if L["op"] == "conv" and L.get("res", -1) in fused:
            # its projection shortcut ran inside this launch: the oracle sums
            # both reductions from the stored block input
            d = L["res"]
            D = layers[d]
            o, ab = oracle.conv2d_proj(get(src), prepared[li][0], prepared[li][1], L["stride"], L["pad"],
                                       L["relu"], get(D["src"]), prepared[d][0], prepared[d][1], D["stride"], prec,
                                       want_abs=True)
            _bound_check(y, o, ulp_bf16(o) + 2.0 ** -16 * ab, what + " (with its projection shortcut)", 0.99,
                         exact_report)
        elif L["op"] == "conv":
            res = get(L["res"]) if L.get("res", -1) >= 0 else None
            o, ab = oracle.conv2d(get(src), prepared[li][0], prepared[li][1], L["stride"], L["pad"], L["relu"],
                                  res, prec, want_abs=True)
            if li == last or prec == "fp32":
                _bound_check(y, o, 1e-5 * ab + 1e-6, what, 0.0, exact_report)
            else:
                _bound_check(y, o, ulp_bf16(o) + 2.0 ** -16 * ab, what, 0.99, exact_report)
        elif L["op"] == "maxpool":
            if src in fused:  # conv + max pool in one launch: stored input of the conv
                C = layers[src]
                oc, ab = oracle.conv2d(get(C["src"]), prepared[src][0], prepared[src][1], C["stride"], C["pad"],
                                       C["relu"], None, prec, want_abs=True)
                o = oracle.maxpool(oc, L["k"], L["stride"], L["pad"])
                tol = oracle.maxpool(ulp_bf16(oc) + 2.0 ** -16 * ab, L["k"], L["stride"], L["pad"])
                _bound_check(y, o, tol, what + " (fused with its conv)", 0.99, exact_report)
            else:
                o = oracle.maxpool(get(src), L["k"], L["stride"], L["pad"])
                assert np.array_equal(y.view(np.uint32), o.view(np.uint32)), what
        elif L["op"] == "gap":
            y = y.reshape(1, -1)
            if src in fused:  # conv + average pool in one launch
                C = layers[src]
                res = get(C["res"]) if C.get("res", -1) >= 0 else None
                oc, ab = oracle.conv2d(get(C["src"]), prepared[src][0], prepared[src][1], C["stride"], C["pad"],
                                       C["relu"], res, prec, want_abs=True)
                o = oracle.gap(oc, prec)
                tc = ulp_bf16(oc) + 2.0 ** -16 * ab
                tol = ulp_bf16(o) + tc.reshape(1, -1, tc.shape[-1]).mean(axis=1)
                _bound_check(y, o, tol, what + " (fused with its conv)", 0.95, exact_report)
            else:
                o = oracle.gap(get(src), prec)
                _bound_check(y, o, ulp_bf16(o) if prec == "bf16" else 1e-6 + 1e-6 * np.abs(o), what,
                             0.99 if prec == "bf16" else 0.0, exact_report)
        elif L["op"] == "fc":
            xs = get(src)
            f = oracle.flatten_nchw(xs) if L.get("flatten_nchw") else xs.reshape(1, -1)
            out_prec = "fp32" if li == last else prec
            o = oracle.fc(f, prepared[li][0], prepared[li][1], L["relu"], out_prec)
            ab = _fc_abs(f, prepared[li][0])
            y = y.reshape(1, -1)
            if out_prec == "fp32":
                _bound_check(y, o, 1e-5 * ab + 1e-6, what, 0.0, exact_report)
            else:
                _bound_check(y, o, ulp_bf16(o) + 2.0 ** -16 * ab, what, 0.99, exact_report)
    return len(layers) - len(fused)


@pytest.mark.parametrize("wname,images", [("hetero_r18_r50_vgg11_bf16_b32", (0, 31)),
                                          ("resnet18x3_bf16_b32", (7,)),
                                          ("tiny2_fp32_b4", (3,))])
def test_every_layer_at_full_shapes(wname, images):
    w = wl.workload(wname)
    imgs = list(wl.images_uniform(w["image_seed"], w["batch"], *w["in_hw"]))
    prepared = [oracle.prepare_model(m, w["precision"]) for m in w["models"]]
    exact = []
    with fsb.Ensemble(w["models"], w["out_hw"], MEAN, STD, w["precision"], max_batch=w["batch"]) as ens:
        ref = ens.infer(imgs)
        for image in images:
            fsb.fs_debug_capture(ens.handle, image)
            g = ens.infer(imgs)  # the capture leaves the results alone
            for k in ("probs", "logits", "vote", "top1"):
                assert np.array_equal(g[k], ref[k]), k
            checked = 0
            for m, layers in enumerate(w["models"]):
                checked += check_layers(ens, layers, prepared[m], w["precision"], imgs, image, m, w["out_hw"],
                                        exact)
            assert checked >= sum(len(L) - 2 - len(oracle.projection_shortcuts(L)) for L in w["models"])
        fsb.fs_debug_capture(ens.handle, -1)
    worst = min(exact, key=lambda t: t[1])
    print(f"{wname}: {len(exact)} layer checks, lowest bit-identical fraction {worst[1]:.4f} ({worst[0]})")


def test_capture_arguments():
    w = wl.workload("tiny2_fp32_b4")
    with fsb.Ensemble(w["models"], w["out_hw"], MEAN, STD, w["precision"], max_batch=4) as ens:
        with pytest.raises(fsb.FsError) as e:
            fsb.fs_debug_layer(ens.handle, 0, 0, (1, 32, 32, 16))
        assert e.value.status == fsb.FS_ERR_INVALID  # nothing armed
        with pytest.raises(fsb.FsError):
            fsb.fs_debug_capture(ens.handle, 4)
        fsb.fs_debug_capture(ens.handle, 3)
        ens.infer(list(wl.images_uniform(1, 2, 32, 32)))  # image 3 is not in a batch of 2
        with pytest.raises(fsb.FsError) as e:
            fsb.fs_debug_layer(ens.handle, 0, 0, (1, 32, 32, 16))
        assert e.value.status == fsb.FS_ERR_UNSUPPORTED
        with pytest.raises(fsb.FsError):
            fsb.fs_debug_layer(ens.handle, 0, 0, (1, 32, 32, 8))  # wrong size
        with pytest.raises(fsb.FsError):
            fsb.fs_debug_layer(ens.handle, 2, 0, (1, 32, 32, 16))  # no such model
