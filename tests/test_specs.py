"""The network shapes fed to both sides are pinned to published counts.

Parameter counts of the torchvision models (ResNet-18 11,689,512; ResNet-50
25,557,032; VGG-11 132,863,336) minus one parameter per batch-norm channel
(scale and shift fold into one conv bias); multiply-accumulate counts of
the ResNet paper (He et al., CVPR 2016, Table 1: 1.8 G for 18 layers; the
stride-on-3x3 variant of 50 layers does 4.1 G)."""
import workloads as wl


def _bn_channels(layers):
    return sum(L["cout"] for L in layers if L["op"] == "conv" and L.get("bn"))


def test_resnet18_counts():
    L = wl.ARCHS["resnet18"]()
    macs, params = wl.count_flops_params(L)
    assert params == 11_689_512 - _bn_channels(L)
    assert round(macs / 1e9, 1) == 1.8
    assert sum(1 for x in L if x["op"] == "conv") == 20


def test_resnet50_counts():
    L = wl.ARCHS["resnet50"]()
    macs, params = wl.count_flops_params(L)
    assert params == 25_557_032 - _bn_channels(L)
    assert round(macs / 1e9, 1) == 4.1
    assert sum(1 for x in L if x["op"] == "conv") == 53


def test_vgg11_counts():
    L = wl.ARCHS["vgg11"]()
    macs, params = wl.count_flops_params(L)
    assert params == 132_863_336
    assert round(macs / 1e9, 2) == 7.61
    assert wl.layer_shapes(L, 224, 224)[-4] == (7, 7, 512)


def test_tiny_shapes():
    L = wl.ARCHS["tiny"]()
    assert wl.layer_shapes(L, 32, 32) == [(32, 32, 16), (16, 16, 16), (16, 16, 32), (1, 1, 32),
                                          (1, 1, 10)]


def test_residual_wiring_is_topological():
    for a in ("resnet18", "resnet50", "vgg11", "tiny"):
        L = wl.ARCHS[a]()
        shapes = wl.layer_shapes(L, 224, 224)
        for i, x in enumerate(L):
            assert x["src"] < i
            if x.get("res", -1) >= 0:
                assert x["res"] < i and shapes[x["res"]] == shapes[i]


def test_generators_are_seeded_and_shaped():
    a = wl.images_uniform(7, 3, 5, 6)
    assert a.shape == (3, 5, 6, 3) and a.dtype.name == "uint8"
    assert (a == wl.images_uniform(7, 3, 5, 6)).all()
    r = wl.images_ragged(3, 20)
    assert all(160 <= im.shape[0] <= 320 and 160 <= im.shape[1] <= 320 for im in r)
    flat, desc = wl.pack_images(r)
    assert flat.size == sum(im.size for im in r) and desc[1][0] == r[0].size
    reqs = wl.request_stream(3000, 10)
    assert all(len(q) in (1, 2, 3, 5, 7, 16, 31, 64) for q in reqs)
    m1, m2 = wl.build_model("tiny", 1), wl.build_model("tiny", 1)
    assert (m1[0]["weight"] == m2[0]["weight"]).all()
    r18 = wl.build_model("resnet18", 5)
    assert r18[0]["bn_scale"].min() >= 0.5 and r18[0]["bn_scale"].max() <= 1.5
