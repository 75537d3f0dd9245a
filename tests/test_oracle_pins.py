"""Pins of the CPU oracle against things other than itself: closed forms,
library routines on the CPU (scipy, numpy, torch in float64), brute force on
tiny inputs and invariants.  Each test names the definition it pins; the
paper fixes the operations only by name (Fig. 1 caption: one data
transformation shared by all models; Sec. 2.2: every model runs on it;
Sec. 2.3: per-model, per-image outputs; Sec. 2.1: combined output)."""
import ctypes
import math

import numpy as np
import pytest
import scipy.signal
import torch
import torch.nn.functional as F

import oracle
import workloads as wl

MEAN, STD = wl.IMAGENET_MEAN, wl.IMAGENET_STD
rng = np.random.default_rng(12345)


def _norm64(v, c):
    # the constants travel as fp32 through both interfaces
    return (np.float64(v) / 255.0 - np.float64(np.float32(MEAN[c]))) / np.float64(np.float32(STD[c]))


# ------------------------------------------------------------ bf16 rounding
def test_round_bf16_matches_torch_rne():
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 200000),
        # exact ties: lower 16 bits 0x8000 with even and odd upper halves
        np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00008000, 0x00018000, 0x7F7F8000],
                 dtype=np.uint32).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 1e-45, 3.4e38], np.float32),
    ]).astype(np.float32)
    a = oracle.round_bf16(x)
    b = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.isnan(oracle.round_bf16(np.array([np.nan], np.float32))[0])


# ------------------------------------------------------ resize + normalise
def test_preprocess_identity_is_exact_normalisation():
    img = rng.integers(0, 256, (7, 9, 3), dtype=np.uint8)
    out = oracle.preprocess(img, 7, 9, MEAN, STD, "fp32")
    exp = np.stack([_norm64(img[..., c], c) for c in range(3)], -1).astype(np.float32)
    assert np.array_equal(out, exp)


@pytest.mark.parametrize("hw", [(1, 1), (5, 3), (300, 171)])
def test_preprocess_constant_image(hw):
    for val in (0, 17, 255):
        img = np.full(hw + (3,), val, np.uint8)
        out = oracle.preprocess(img, 224, 224, MEAN, STD, "fp32")
        for c in range(3):
            e = np.float32(_norm64(val, c))
            assert np.all(np.abs(out[..., c] - e) <= 2 * np.spacing(np.abs(e)) + 1e-12)


def test_preprocess_exact_2x_downsample_is_box_mean():
    img = rng.integers(0, 256, (12, 16, 3), dtype=np.uint8)
    out = oracle.preprocess(img, 6, 8, MEAN, STD, "fp32")
    box = img.astype(np.float64).reshape(6, 2, 8, 2, 3).mean(axis=(1, 3))
    exp = np.stack([_norm64(box[..., c], c) for c in range(3)], -1)
    assert np.max(np.abs(out - exp)) < 1e-6


def test_preprocess_exact_2x_upsample_weights():
    img = rng.integers(0, 256, (4, 5, 3), dtype=np.uint8).astype(np.float64)
    out = oracle.preprocess(img.astype(np.uint8), 8, 10, MEAN, STD, "fp32")

    def up(a, n):  # 1-D: output j takes 0.75/0.25 of its two nearest inputs, clamped
        r = np.empty((2 * n,) + a.shape[1:])
        for j in range(2 * n):
            s = max((j + 0.5) / 2 - 0.5, 0.0)
            i0 = int(math.floor(s)); i1 = min(i0 + 1, n - 1); l = s - i0
            r[j] = (1 - l) * a[i0] + l * a[i1]
        return r
    v = up(np.swapaxes(up(img, 4), 0, 1), 5).swapaxes(0, 1)
    exp = np.stack([_norm64(v[..., c], c) for c in range(3)], -1)
    assert np.max(np.abs(out - exp)) < 1e-6
    # the interior weights are exactly 3/4 and 1/4
    assert abs(v[1, 0, 0] - (0.75 * img[0, 0, 0] + 0.25 * img[1, 0, 0])) < 1e-12
    assert v[0, 0, 0] == img[0, 0, 0]  # top edge clamps to the first row


@pytest.mark.parametrize("src,dst", [((256, 256), (224, 224)), ((160, 317), (224, 224)),
                                     ((320, 161), (224, 224)), ((33, 29), (32, 32))])
def test_preprocess_matches_torch_bilinear_fp64(src, dst):
    img = rng.integers(0, 256, src + (3,), dtype=np.uint8)
    out = oracle.preprocess(img, dst[0], dst[1], MEAN, STD, "fp32")
    t = torch.from_numpy(img.astype(np.float64)).permute(2, 0, 1)[None]
    r = F.interpolate(t, size=dst, mode="bilinear", align_corners=False, antialias=False)[0]
    r = r.permute(1, 2, 0).numpy()
    exp = np.stack([_norm64(r[..., c], c) for c in range(3)], -1)
    assert np.max(np.abs(out - exp)) < 2e-6


def test_preprocess_bf16_is_rounded_fp32():
    img = rng.integers(0, 256, (50, 70, 3), dtype=np.uint8)
    a = oracle.preprocess(img, 32, 40, MEAN, STD, "fp32")
    b = oracle.preprocess(img, 32, 40, MEAN, STD, "bf16")
    assert np.array_equal(torch.from_numpy(a).to(torch.bfloat16).float().numpy(), b)


# -------------------------------------------------------------- convolution
@pytest.mark.parametrize("stride", [1, 2, 3])
@pytest.mark.parametrize("pad", [0, 1, 2])
@pytest.mark.parametrize("k", [1, 2, 3])
def test_conv_single_channel_brute_force_vs_scipy(stride, pad, k):
    for H, W in ((5, 5), (4, 3)):
        if H + 2 * pad < k or W + 2 * pad < k:
            continue
        x = rng.standard_normal((1, H, W, 1)).astype(np.float32)
        w = rng.standard_normal((1, k, k, 1)).astype(np.float32)
        out = oracle.conv2d(x, w, None, stride, pad, relu=False)
        xp = np.pad(x[0, :, :, 0].astype(np.float64), pad)
        full = scipy.signal.correlate2d(xp, w[0, :, :, 0].astype(np.float64), mode="valid")
        exp = full[::stride, ::stride]
        assert out.shape[1:3] == exp.shape
        assert np.max(np.abs(out[0, :, :, 0] - exp)) < 1e-6


def test_conv_delta_kernels_identity_and_shift():
    x = rng.standard_normal((2, 6, 7, 5)).astype(np.float32)
    w = np.zeros((5, 3, 3, 5), np.float32)
    for c in range(5):
        w[c, 1, 1, c] = 1.0
    assert np.array_equal(oracle.conv2d(x, w, None, 1, 1, False), x)
    w2 = np.zeros_like(w)
    for c in range(5):
        w2[c, 1, 2, c] = 1.0  # picks the right neighbour: out[y, x] = in[y, x+1]
    y = oracle.conv2d(x, w2, None, 1, 1, False)
    assert np.array_equal(y[:, :, :-1], x[:, :, 1:])
    assert np.all(y[:, :, -1] == 0)


def test_conv_ones_on_constant_counts_valid_taps():
    H, W, C, c = 6, 5, 4, 1.5
    x = np.full((1, H, W, C), c, np.float32)
    w = np.ones((2, 3, 3, C), np.float32)
    y = oracle.conv2d(x, w, None, 1, 1, False)
    for oy in range(H):
        for ox in range(W):
            taps = sum(1 for ky in range(3) for kx in range(3)
                       if 0 <= oy - 1 + ky < H and 0 <= ox - 1 + kx < W)
            assert np.all(y[0, oy, ox] == c * C * taps)


@pytest.mark.parametrize("cfg", [(2, 9, 9, 3, 8, 7, 2, 3), (1, 8, 8, 16, 32, 3, 1, 1),
                                 (3, 7, 5, 12, 6, 1, 2, 0), (1, 5, 6, 8, 4, 3, 2, 1)])
def test_conv_matches_torch_fp64(cfg):
    B, H, W, Cin, Cout, k, s, p = cfg
    x = rng.standard_normal((B, H, W, Cin)).astype(np.float32)
    w = rng.standard_normal((Cout, k, k, Cin)).astype(np.float32)
    b = rng.standard_normal(Cout).astype(np.float32)
    y = oracle.conv2d(x, w, b, s, p, relu=False)
    t = F.conv2d(torch.from_numpy(x).double().permute(0, 3, 1, 2),
                 torch.from_numpy(w).double().permute(0, 3, 1, 2),
                 torch.from_numpy(b).double(), stride=s, padding=p).permute(0, 2, 3, 1).numpy()
    assert np.max(np.abs(y - t)) <= 1e-6 * max(1.0, np.abs(t).max())


@pytest.mark.parametrize("k,stride,s2,H2", [(3, 1, 2, 18), (3, 1, 2, 17), (1, 1, 1, 9), (3, 2, 2, 9), (1, 1, 2, 17)])
@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_conv_with_projection_shortcut_matches_torch_fp64(k, stride, s2, H2, prec):
    # a block's last conv (input t) plus its 1x1 / stride s2 projection of the
    # block input x2, summed before one rounding, against torch in float64
    B, Cin, C2, Cout = 2, 8, 6, 5
    pad = k // 2
    Hm = (H2 - 1) // s2 + 1  # the projection's output size
    H = (Hm - 1) * stride + k - 2 * pad  # main conv output Hm x Hm
    t = rng.standard_normal((B, H, H, Cin)).astype(np.float32)
    x2 = rng.standard_normal((B, H2, H2, C2)).astype(np.float32)
    w = rng.standard_normal((Cout, k, k, Cin)).astype(np.float32)
    w2 = rng.standard_normal((Cout, 1, 1, C2)).astype(np.float32)
    b, b2 = rng.standard_normal(Cout).astype(np.float32), rng.standard_normal(Cout).astype(np.float32)
    if prec == "bf16":
        t, x2, w, w2 = (oracle.round_bf16(v) for v in (t, x2, w, w2))
    y = oracle.conv2d_proj(t, w, b, stride, pad, 1, x2, w2, b2, s2, prec)
    T = lambda a: torch.from_numpy(a).double().permute(0, 3, 1, 2)
    ref = F.conv2d(T(t), T(w), torch.from_numpy(b).double(), stride=stride, padding=pad) + \
        F.conv2d(T(x2), T(w2), torch.from_numpy(b2).double(), stride=s2)
    ref = torch.relu(ref).permute(0, 2, 3, 1).float()
    assert y.shape == tuple(ref.shape)
    if prec == "fp32":
        assert np.max(np.abs(y - ref.numpy())) <= 1e-6 * np.abs(ref.numpy()).max()
    else:  # one rounding of the float64 sum: equal, except a float ulp away from a tie
        r = ref.bfloat16().float().numpy()
        assert np.mean(y == r) >= 0.99 and np.all(np.abs(y - r) <= 2.0 ** -7 * np.abs(r) + 1e-30)


def test_projection_with_zero_weights_is_the_plain_conv():
    t = rng.standard_normal((2, 6, 6, 8)).astype(np.float32)
    x2 = rng.standard_normal((2, 12, 12, 4)).astype(np.float32)
    w = rng.standard_normal((3, 3, 3, 8)).astype(np.float32)
    b = rng.standard_normal(3).astype(np.float32)
    y = oracle.conv2d_proj(t, w, b, 1, 1, 0, x2, np.zeros((3, 4), np.float32), None, 2, "bf16")
    assert np.array_equal(y, oracle.conv2d(t, w, b, 1, 1, 0, None, "bf16"))


def test_projection_shortcuts_of_the_served_networks():
    # ResNet-18 has a projection at the first block of stages 2-4, ResNet-50
    # at the first block of every stage (the stage-1 one changes width 64 ->
    # 256 at stride 1); each feeds the residual of its block's last conv
    for arch, n in (("resnet18", 3), ("resnet50", 4), ("vgg11", 0), ("tiny", 0)):
        layers = wl.ARCHS[arch]()
        pr = oracle.projection_shortcuts(layers)
        assert len(pr) == n, arch
        for d, c in pr.items():
            assert layers[d]["k"] == 1 and not layers[d]["relu"] and layers[c]["res"] == d and c > d
            assert layers[c]["cout"] == layers[d]["cout"]


def test_conv_residual_then_relu_order():
    x = rng.standard_normal((1, 4, 4, 3)).astype(np.float32)
    w = rng.standard_normal((3, 3, 3, 3)).astype(np.float32)
    b = rng.standard_normal(3).astype(np.float32)
    res = rng.standard_normal((1, 4, 4, 3)).astype(np.float32)
    lin = oracle.conv2d(x, w, b, 1, 1, False).astype(np.float64)
    y = oracle.conv2d(x, w, b, 1, 1, True, res=res)
    # relu is applied after the residual add
    assert np.max(np.abs(y - np.maximum(lin + res, 0))) < 1e-5
    assert (y == 0).any() and (y > 0).any()


def test_conv_linearity_and_bn_fold_equivalence():
    x = rng.standard_normal((2, 6, 6, 4)).astype(np.float32)
    w = rng.standard_normal((5, 3, 3, 4)).astype(np.float32)
    sc = rng.uniform(0.5, 1.5, 5).astype(np.float32)
    sh = (rng.standard_normal(5) * 0.1).astype(np.float32)
    wf, bf = oracle.fold_bn(w, sc, sh, None, "fp32")
    y_fold = oracle.conv2d(x, wf, bf, 2, 1, False)
    y_ref = oracle.conv2d(x, w, None, 2, 1, False).astype(np.float64) * sc + sh
    assert np.max(np.abs(y_fold - y_ref)) <= 1e-6 * np.abs(y_ref).max()
    y2 = oracle.conv2d(2 * x, w, None, 2, 1, False)
    assert np.array_equal(y2, 2 * oracle.conv2d(x, w, None, 2, 1, False))
    # bf16 fold = fp32 product then one rounding
    wb, _ = oracle.fold_bn(w, sc, sh, None, "bf16")
    prod = (w * sc[:, None, None, None]).astype(np.float32)
    assert np.array_equal(wb, torch.from_numpy(prod).to(torch.bfloat16).float().numpy())


def test_conv_storage_rounding_bf16():
    x = oracle.round_bf16(rng.standard_normal((1, 5, 5, 8)))
    w = oracle.round_bf16(rng.standard_normal((4, 3, 3, 8)))
    y32 = oracle.conv2d(x, w, None, 1, 1, True, prec="fp32")
    y16 = oracle.conv2d(x, w, None, 1, 1, True, prec="bf16")
    assert np.array_equal(oracle.round_bf16(y32), y16)


def test_conv_absacc_bounds_the_sum():
    x = rng.standard_normal((1, 5, 5, 8)).astype(np.float32)
    w = rng.standard_normal((4, 3, 3, 8)).astype(np.float32)
    y, ab = oracle.conv2d(x, w, None, 1, 1, False, want_abs=True)
    assert np.all(np.abs(y) <= ab * (1 + 1e-6))
    t = F.conv2d(torch.from_numpy(np.abs(x)).double().permute(0, 3, 1, 2),
                 torch.from_numpy(np.abs(w)).double().permute(0, 3, 1, 2), padding=1)
    assert np.max(np.abs(ab - t.permute(0, 2, 3, 1).numpy())) < 1e-4


# ------------------------------------------------------------------ pooling
def test_maxpool_known_and_padding_border():
    x = np.arange(16, dtype=np.float32).reshape(1, 4, 4, 1)
    y = oracle.maxpool(x, 2, 2, 0)
    assert y[0, :, :, 0].tolist() == [[5, 7], [13, 15]]
    neg = -np.arange(1, 17, dtype=np.float32).reshape(1, 4, 4, 1)
    y = oracle.maxpool(neg, 3, 2, 1)  # padding taps must not win (would give 0)
    assert y[0, :, :, 0].tolist() == [[-1, -2], [-5, -6]]


@pytest.mark.parametrize("k,s,p", [(3, 2, 1), (2, 2, 0)])
def test_maxpool_matches_torch(k, s, p):
    x = rng.standard_normal((2, 9, 8, 5)).astype(np.float32)
    y = oracle.maxpool(x, k, s, p)
    t = F.max_pool2d(torch.from_numpy(x).permute(0, 3, 1, 2), k, s, p).permute(0, 2, 3, 1)
    assert np.array_equal(y, t.numpy())


def test_gap_constant_and_mean():
    assert np.all(oracle.gap(np.full((2, 7, 7, 3), 0.3, np.float32)) == np.float32(0.3))
    x = rng.standard_normal((3, 7, 7, 9)).astype(np.float32)
    assert np.max(np.abs(oracle.gap(x) - x.astype(np.float64).mean(axis=(1, 2)))) < 1e-7
    assert np.array_equal(oracle.gap(x, "bf16"), oracle.round_bf16(oracle.gap(x)))


# ----------------------------------------------------------------------- FC
def test_fc_identity_and_numpy():
    x = rng.standard_normal((4, 6)).astype(np.float32)
    assert np.array_equal(oracle.fc(x, np.eye(6, dtype=np.float32), None, False), x)
    w = rng.standard_normal((5, 6)).astype(np.float32)
    b = rng.standard_normal(5).astype(np.float32)
    exp = x.astype(np.float64) @ w.astype(np.float64).T + b
    assert np.max(np.abs(oracle.fc(x, w, b, False) - exp)) < 1e-6
    assert np.array_equal(oracle.fc(x, w, b, True), np.maximum(oracle.fc(x, w, b, False), 0))


def test_flatten_nchw_matches_torch():
    x = rng.standard_normal((2, 3, 4, 5)).astype(np.float32)  # NHWC
    exp = torch.flatten(torch.from_numpy(x).permute(0, 3, 1, 2), 1).numpy()
    assert np.array_equal(oracle.flatten_nchw(x), exp)


# ------------------------------------------------------------------ softmax
def test_softmax_identities():
    p = oracle.softmax(np.array([[0.0, math.log(2.0)]], np.float32))
    assert np.allclose(p, [[1 / 3, 2 / 3]], atol=1e-7)
    z = (rng.standard_normal((50, 1000)) * 30).astype(np.float32)
    p = oracle.softmax(z)
    assert np.max(np.abs(p.astype(np.float64).sum(1) - 1)) <= 1e-6
    assert np.max(np.abs(oracle.softmax(z + 7.0) - p)) < 1e-6
    u = oracle.softmax(np.full((1, 1000), 3.25, np.float32))
    assert np.all(u == np.float32(1 / 1000))
    t = torch.softmax(torch.from_numpy(z).double(), 1).numpy()
    assert np.max(np.abs(p - t)) < 1e-7


# ------------------------------------------------------------------ combine
def test_combine_identical_models_and_ties():
    z = rng.standard_normal((1, 6, 10)).astype(np.float32)
    p = oracle.softmax(z)
    r = oracle.combine(np.repeat(p, 3, 0), np.repeat(z, 3, 0))
    assert np.max(np.abs(r["mean"] - p[0])) < 1e-7
    assert np.array_equal(r["vote"], r["top1"][0])
    assert np.array_equal(r["top1"][0], np.argmax(z[0], 1))
    # two saturated models voting for different classes tie exactly: lowest index wins
    pt = np.zeros((2, 1, 10), np.float32)
    pt[0, 0, 7] = 1.0
    pt[1, 0, 3] = 1.0
    r = oracle.combine(pt, pt)
    assert r["vote"][0] == 3 and r["top1"][:, 0].tolist() == [7, 3]
    assert oracle.argmax(np.array([1, 5, 5, 2], np.float32)) == 1


# Hand-worked combinations of top-1 lists (one column per image, one row per
# model): plurality answers, and the detection policy of Sec. 2.1 for a class
# c* and count k, worked out by reading each column.
POLICY_TOP1 = np.array([[5, 7, 4, 1, 3],
                        [5, 2, 4, 8, 3],
                        [2, 9, 9, 8, 3],
                        [6, 9, 9, 1, 3]], np.int32)
POLICY_CASES = [  # (policy, c*, k, expected per column)
    (oracle.PLURALITY, 0, 1, [5, 9, 4, 1, 3]),  # 2-1-1 / 2 nines / 4 vs 9 tie -> 4 / 1 vs 8 tie -> 1 / all 3
    (oracle.ANY, 9, 1, [0, 1, 1, 0, 0]),        # OR: one model naming 9 is enough
    (oracle.ANY, 9, 2, [0, 1, 1, 0, 0]),
    (oracle.ANY, 9, 3, [0, 0, 0, 0, 0]),
    (oracle.ANY, 3, 4, [0, 0, 0, 0, 1]),        # AND of all four models
    (oracle.ANY, 5, 2, [1, 0, 0, 0, 0]),
    (oracle.ANY, 8, 1, [0, 0, 0, 1, 0]),
]


@pytest.mark.parametrize("case", range(len(POLICY_CASES)))
def test_vote_policies_hand_worked(case):
    policy, pos, k, want = POLICY_CASES[case]
    assert oracle.vote_policy(POLICY_TOP1, 10, policy, pos, k).tolist() == want


def test_plurality_is_the_smallest_mode():
    # scipy.stats.mode returns the most frequent value, the smallest on ties
    import scipy.stats
    g = np.random.default_rng(5)
    for N, C in [(1, 10), (2, 4), (3, 5), (5, 3), (7, 1000), (16, 6)]:
        t = g.integers(0, C, size=(N, 200)).astype(np.int32)
        want = scipy.stats.mode(t, axis=0, keepdims=False).mode
        assert np.array_equal(oracle.vote_policy(t, C, oracle.PLURALITY), want), (N, C)


def test_detection_policy_properties():
    g = np.random.default_rng(6)
    N, C = 5, 4
    t = g.integers(0, C, size=(N, 300)).astype(np.int32)
    for pos in range(C):
        by_k = [oracle.vote_policy(t, C, oracle.ANY, pos, k) for k in range(1, N + 1)]
        for a, b in zip(by_k, by_k[1:]):  # asking for more models never detects more
            assert np.all(b <= a)
        plural = oracle.vote_policy(t, C, oracle.PLURALITY)
        assert np.all(by_k[0][plural == pos] == 1)  # the plurality class is named by someone
    one = t[:1]  # a single model: plurality is its top-1, detection is top-1 == c*
    assert np.array_equal(oracle.vote_policy(one, C, oracle.PLURALITY), one[0])
    assert np.array_equal(oracle.vote_policy(one, C, oracle.ANY, 2, 1), (one[0] == 2).astype(np.int32))


# -------------------------------------------------------------- whole nets
def _torch_forward(layers, x, prec):
    """Independent float64 forward with torch CPU ops, rounding to the storage
    type at the same points, used to pin the oracle's network driver."""
    def st(t):
        t = t.float().double()
        return t.bfloat16().double() if prec == "bf16" else t
    outs = []
    xt = torch.from_numpy(x).double().permute(0, 3, 1, 2)
    # a 1x1 conv without activation that only feeds one residual add is
    # that block's projection shortcut: its sum is added unrounded
    uses = {}
    for L in layers:
        uses[L["src"]] = uses.get(L["src"], 0) + 1
        if L["op"] == "conv" and L["res"] >= 0:
            uses[L["res"]] = uses.get(L["res"], 0) + 1
    proj = {L["res"] for L in layers if L["op"] == "conv" and L["res"] >= 0
            and layers[L["res"]]["op"] == "conv" and layers[L["res"]]["k"] == 1
            and not layers[L["res"]]["relu"] and layers[L["res"]]["pad"] == 0 and uses[L["res"]] == 1}
    for i, L in enumerate(layers):
        src = xt if L["src"] < 0 else outs[L["src"]]
        if L["op"] == "conv":
            w = torch.from_numpy(L["weight"]).double()
            if L.get("bn_scale") is not None:
                w = (w.float() * torch.from_numpy(L["bn_scale"])[:, None, None, None]).double()
                b = torch.from_numpy(L["bn_shift"]).double()
            else:
                b = torch.from_numpy(L["bias"]).double()
            if prec == "bf16":
                w = w.float().bfloat16().double()
            y = F.conv2d(src, w.permute(0, 3, 1, 2), b, stride=L["stride"], padding=L["pad"])
            if L["res"] >= 0:
                y = y + outs[L["res"]]
            if i in proj:
                outs.append(y)  # unrounded: summed into the block's last conv
                continue
            y = st(torch.relu(y) if L["relu"] else y)
        elif L["op"] == "maxpool":
            y = F.max_pool2d(src, L["k"], L["stride"], L["pad"])
        elif L["op"] == "gap":
            y = st(src.mean(dim=(2, 3), keepdim=True))
        else:
            f = torch.flatten(src, 1)  # channel-major flatten of an NCHW tensor
            w = torch.from_numpy(L["weight"]).double()
            if prec == "bf16":
                w = w.float().bfloat16().double()
            y = f @ w.T + torch.from_numpy(L["bias"]).double()
            y = torch.relu(y) if L["relu"] else y
            y = y.float().double() if i == len(layers) - 1 else st(y)
            y = y[:, :, None, None]
        outs.append(y)
    return outs[-1][:, :, 0, 0].numpy()


@pytest.mark.parametrize("arch,hw,prec", [("tiny", 32, "fp32"), ("resnet18", 64, "fp32"),
                                          ("resnet50", 64, "fp32"), ("vgg11", 32, "fp32"),
                                          ("resnet18", 64, "bf16")])
def test_network_driver_matches_torch_fp64(arch, hw, prec):
    layers = wl.build_model(arch, 77)
    if arch == "vgg11":  # a 32x32 input leaves a 1x1 map: shrink fc1 to match
        layers[-3] = dict(layers[-3], cin=512,
                          weight=layers[-3]["weight"][:, :512].copy())
    imgs = wl.images_uniform(5, 2, hw, hw)
    x = oracle.preprocess_batch(imgs, hw, hw, MEAN, STD, prec)
    z = oracle.forward_model(layers, x, prec)
    t = _torch_forward(layers, x, prec)
    scale = np.abs(t).max()
    if prec == "fp32":
        assert np.max(np.abs(z - t)) <= 1e-5 * scale
    else:  # storage rounding makes the comparison chaotic: a loose scale-free check
        assert np.max(np.abs(z - t)) <= 3e-2 * np.std(t)


def test_vgg_flatten_order_in_driver():
    # a 7x7 map so fc1 reads the channel-major flatten of a genuine spatial map
    layers = [dict(op="maxpool", src=-1, k=1, stride=1, pad=0),
              dict(op="fc", src=0, cin=3 * 7 * 7, cout=4, relu=0, flatten_nchw=True,
                   weight=rng.standard_normal((4, 147)).astype(np.float32),
                   bias=np.zeros(4, np.float32))]
    x = rng.standard_normal((2, 7, 7, 3)).astype(np.float32)
    z = oracle.forward_model(layers, x, "fp32")
    exp = torch.flatten(torch.from_numpy(x).permute(0, 3, 1, 2), 1).double().numpy() @ \
        layers[1]["weight"].astype(np.float64).T
    assert np.max(np.abs(z - exp)) < 1e-5


def test_ensemble_batch_permutation_and_size_invariance():
    models = [wl.build_model("tiny", s) for s in (1001, 1002)]
    imgs = wl.images_uniform(1000, 4, 32, 32)
    r = oracle.ensemble(models, imgs, (32, 32), MEAN, STD, "fp32")
    perm = [2, 0, 3, 1]
    rp = oracle.ensemble(models, imgs[perm], (32, 32), MEAN, STD, "fp32")
    assert np.array_equal(rp["probs"], r["probs"][:, perm])
    assert np.array_equal(rp["vote"], r["vote"][perm])
    r1 = oracle.ensemble(models, imgs[1:2], (32, 32), MEAN, STD, "fp32")
    assert np.array_equal(r1["probs"][:, 0], r["probs"][:, 1])
    assert np.max(np.abs(r["probs"].astype(np.float64).sum(-1) - 1)) <= 1e-6


def test_oracle_thread_count_invariance():
    gomp = ctypes.CDLL("libgomp.so.1")
    layers = wl.build_model("resnet18", 3)
    x = oracle.preprocess_batch(wl.images_uniform(9, 2, 48, 48), 48, 48, MEAN, STD, "bf16")
    a = oracle.forward_model(layers, x, "bf16")
    gomp.omp_set_num_threads(1)
    try:
        b = oracle.forward_model(layers, x, "bf16")
    finally:
        gomp.omp_set_num_threads(8)
    assert np.array_equal(a, b)


def test_acc32_switch_is_order_noise_only():
    x = rng.standard_normal((1, 6, 6, 64)).astype(np.float32)
    w = rng.standard_normal((8, 3, 3, 64)).astype(np.float32)
    a, ab = oracle.conv2d(x, w, None, 1, 1, False, want_abs=True)
    oracle.set_acc32(True)
    try:
        b = oracle.conv2d(x, w, None, 1, 1, False)
    finally:
        oracle.set_acc32(False)
    assert not np.array_equal(a, b)
    assert np.all(np.abs(a - b) <= 576 * 2 ** -24 * ab)
