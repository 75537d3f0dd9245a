"""Per-kernel parity of the HIP path against the CPU oracle, element by
element, on the same seeded inputs (the single-kernel C entry points).

Tolerances (derived from the arithmetic of each kernel):
* fp32 storage: |gpu - oracle| <= 1e-5 * sum|x*w| + 1e-6 (an fp32 sum in
  another order against a double sum).
* bf16 storage: |gpu - oracle| <= 1 bf16 ulp of the oracle value +
  2^-16 * sum|x*w|, and at least 99% of the outputs bit-identical
  (preprocess: + 2e-6 absolute for the cancellation in v/255 - mean).
* max pool: bit-exact.  Softmax: 1e-6 absolute."""
import numpy as np
import pytest

import oracle
import workloads as wl
from paper_2003_01538_amd import flexserve as fsb

pytestmark = pytest.mark.gpu
MEAN, STD = wl.IMAGENET_MEAN, wl.IMAGENET_STD
F32, BF16 = fsb.FS_F32, fsb.FS_BF16
PREC = {F32: "fp32", BF16: "bf16"}


def ulp_bf16(x):
    x = np.abs(np.asarray(x, np.float32))
    e = np.floor(np.log2(np.maximum(x, np.float32(2.0 ** -126))))
    return np.float32(2.0) ** (e - 7)


def assert_bf16_close(g, o, absacc=None, frac_exact=0.99, what="", abs_tol=0.0):
    g, o = np.asarray(g, np.float32), np.asarray(o, np.float32)
    tol = ulp_bf16(o) + (0 if absacc is None else 2.0 ** -16 * absacc) + abs_tol
    bad = np.abs(g - o) > tol
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} outside 1 ulp + bound; max err {np.abs(g - o).max()}"
    exact = np.mean(g.view(np.uint32) == o.view(np.uint32))
    assert exact >= frac_exact, f"{what}: only {exact:.4f} bit-identical"


# ----------------------------------------------------------------- preprocess
@pytest.mark.parametrize("prec", [F32, BF16])
@pytest.mark.parametrize("case", ["identity32", "resize256to224", "ragged", "tiny_up"])
def test_preprocess_parity(gpu_lib, prec, case):
    rng = np.random.default_rng(sum(map(ord, case)))
    if case == "identity32":
        imgs, oh, ow = list(wl.images_uniform(1000, 4, 32, 32)), 32, 32
    elif case == "resize256to224":
        imgs, oh, ow = list(wl.images_uniform(2000, 3, 256, 256)), 224, 224
    elif case == "ragged":
        imgs, oh, ow = wl.images_ragged(3000, 5), 224, 224
    else:
        imgs = [rng.integers(0, 256, (1, 1, 3), dtype=np.uint8),
                rng.integers(0, 256, (3, 7, 3), dtype=np.uint8)]
        oh, ow = 17, 9
    # a strided view: rows longer than 3*w bytes
    big = rng.integers(0, 256, (40, 50, 3), dtype=np.uint8)
    imgs = list(imgs) + [big[5:37, 3:41]]
    g = fsb.fs_test_preprocess(imgs, oh, ow, MEAN, STD, prec)
    assert np.all(g[..., 3] == 0)
    for i, im in enumerate(imgs):
        o = oracle.preprocess(im, oh, ow, MEAN, STD, PREC[prec])
        if prec == F32:
            assert np.max(np.abs(g[i, ..., :3] - o)) <= 1e-5, (case, i)
        else:
            # (v/255 - mean) cancels near zero: the fp32 kernel carries an
            # absolute error of a few fp32 ulps of the operands (|x| <= 4.4)
            assert_bf16_close(g[i, ..., :3], o, frac_exact=0.99, what=f"{case}[{i}]", abs_tol=2e-6)


def test_preprocess_space_to_depth_layout(gpu_lib):
    rng = np.random.default_rng(4001)
    # ragged sizes, a square image, a strided view, a very wide image (its
    # taps gathered through the cache), tiny images, and the widest rows the
    # kernel stages in LDS (511 pixels) next to the narrowest it does not (512)
    big = rng.integers(0, 256, (300, 420, 3), dtype=np.uint8)
    imgs = (wl.images_ragged(4000, 3) + [wl.images_uniform(5, 1, 224, 224)[0]]
            + [big[7:290, 11:400], rng.integers(0, 256, (37, 1500, 3), dtype=np.uint8)]
            + [rng.integers(0, 256, (1, 1, 3), dtype=np.uint8), rng.integers(0, 256, (3, 5, 3), dtype=np.uint8),
               rng.integers(0, 256, (20, 511, 3), dtype=np.uint8), rng.integers(0, 256, (21, 512, 3), dtype=np.uint8)])
    g = fsb.fs_test_preprocess(imgs, 224, 224, MEAN, STD, BF16, layout=1)
    assert g.shape == (len(imgs), 112, 112, 16) and np.all(g[..., 12:] == 0)
    for i, im in enumerate(imgs):
        o = oracle.preprocess(im, 224, 224, MEAN, STD, "bf16")
        # channel (sy*2 + sx)*3 + c of block (Y, X) is pixel (2Y+sy, 2X+sx), channel c
        r = o.reshape(112, 2, 112, 2, 3).transpose(0, 2, 1, 3, 4).reshape(112, 112, 12)
        assert_bf16_close(g[i, ..., :12], r, frac_exact=0.99, what=f"s2d[{i}]", abs_tol=2e-6)


@pytest.mark.parametrize("layout", [0, 1])
def test_preprocess_tap_division_fallback(gpu_lib, layout):
    # Tap positions come from a float reciprocal while 2 * out * in < 2^22
    # and from integer division beyond; 224 outputs from more than 9362
    # input pixels along an axis take the integer path (rows and columns).
    rng = np.random.default_rng(4002)
    imgs = [rng.integers(0, 256, (3, 12000, 3), dtype=np.uint8), rng.integers(0, 256, (12000, 2, 3), dtype=np.uint8),
            rng.integers(0, 256, (9400, 9, 3), dtype=np.uint8), rng.integers(0, 256, (40, 60, 3), dtype=np.uint8)]
    prec = BF16
    g = fsb.fs_test_preprocess(imgs, 224, 224, MEAN, STD, prec, layout=layout)
    for i, im in enumerate(imgs):
        o = oracle.preprocess(im, 224, 224, MEAN, STD, "bf16")
        if layout == 1:
            o = o.reshape(112, 2, 112, 2, 3).transpose(0, 2, 1, 3, 4).reshape(112, 112, 12)
            got = g[i, ..., :12]
        else:
            got = g[i, ..., :3]
        assert_bf16_close(got, o, frac_exact=0.99, what=f"fallback[{layout}][{i}]", abs_tol=2e-6)


# ----------------------------------------------------------------------- conv
CONV_CASES = [
    # B, H, W, Cin, Cout, k, stride, pad, relu, residual
    (2, 32, 32, 3, 64, 7, 2, 3, 1, 0),     # ResNet stem shape (Cin padded to 4)
    (2, 20, 20, 3, 64, 3, 1, 1, 1, 0),     # VGG first conv shape
    (2, 14, 14, 64, 64, 3, 1, 1, 1, 1),    # basic block conv + residual + ReLU
    (3, 15, 13, 64, 128, 3, 2, 1, 1, 0),   # strided, ragged M
    (2, 14, 14, 64, 128, 1, 2, 0, 0, 0),   # 1x1 downsample
    (1, 7, 7, 256, 512, 3, 1, 1, 0, 1),    # deep layer, residual, no ReLU
    (2, 9, 9, 128, 256, 1, 1, 0, 1, 1),    # bottleneck expand + residual
    (1, 5, 6, 16, 32, 3, 1, 1, 1, 0),      # tiny-net second conv
    (2, 12, 56, 64, 64, 3, 1, 1, 1, 1),    # halo kernel, 4-row tiles of width 56
    (3, 10, 56, 64, 64, 3, 1, 1, 0, 0),    # halo kernel, partial last row tile, no residual / ReLU
    (2, 12, 20, 128, 128, 3, 1, 1, 1, 1),  # streamed-weight halo: tiles across rows and images, ragged M
    (3, 10, 9, 128, 256, 3, 1, 1, 0, 0),   # streamed-weight halo: two channel tiles, no residual / ReLU
    (1, 1, 1, 128, 128, 3, 1, 1, 1, 1),    # 1x1 image: every tap but the centre is padding
    (3, 2, 23, 128, 128, 3, 1, 1, 1, 0),   # streamed-weight halo, 40-block patch, tiles across images
    (1, 4, 70, 128, 128, 3, 1, 1, 1, 1),   # streamed-weight halo with its largest patch (48 blocks)
    (2, 5, 70, 128, 128, 3, 1, 1, 1, 0),   # patch too large for it: the implicit GEMM takes the layer
    (4, 64, 64, 128, 256, 3, 1, 1, 1, 1),  # streamed-weight halo, 256 tiles of 128 x 128
    (2, 9, 9, 64, 256, 1, 1, 0, 1, 1),     # bottleneck expand, one K-tile (never split): residual prefetched, ragged M
    (2, 7, 7, 512, 512, 3, 1, 1, 1, 1),    # streamed-weight halo, Cin 512: eight chunks per tile, residual
    (16, 14, 14, 512, 512, 3, 1, 1, 1, 0),  # streamed-weight halo, 100 tiles over the CUs, tiles across images
]
# cases the streamed-weight halo kernel (3x3/1, Cin and Cout multiples of 128) fits
HS_CASES = (5, 10, 11, 12, 13, 14, 16, 18, 19)


def _conv_inputs(case, prec, seed):
    B, H, W, Cin, Cout, k, s, p, relu, has_res = case
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, H, W, Cin)).astype(np.float32)
    w = (rng.standard_normal((Cout, k, k, Cin)) * np.sqrt(2.0 / (Cin * k * k))).astype(np.float32)
    b = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    r = rng.standard_normal((B, Ho, Wo, Cout)).astype(np.float32) if has_res else None
    if prec == BF16:
        x, w = oracle.round_bf16(x), oracle.round_bf16(w)
        r = None if r is None else oracle.round_bf16(r)
    return x, w, b, r


def _tiles_for(prec, Cin):
    out = []
    for t in range(fsb.fs_conv_num_tiles(prec)):
        name = fsb.fs_conv_tile_name(prec, t)
        vec = int(name.rsplit("_v", 1)[1])
        cin_p = 4 if Cin == 3 else Cin
        if cin_p % vec == 0:
            out.append(t)
    return out


@pytest.mark.parametrize("prec", [BF16, F32])
@pytest.mark.parametrize("ci", range(len(CONV_CASES)))
def test_conv_parity_every_tile(gpu_lib, prec, ci):
    case = CONV_CASES[ci]
    B, H, W, Cin, Cout, k, s, p, relu, has_res = case
    x, w, b, r = _conv_inputs(case, prec, 100 + ci)
    o, ab = oracle.conv2d(x, w, b, s, p, relu, r, PREC[prec], want_abs=True)
    tiles = _tiles_for(prec, Cin)
    assert tiles
    ran, ran_names = 0, []
    dma_out = {}  # the LDS-DMA family: every tile sums each output in the same order
    hs_out = {}   # the streamed-weight halo family (weights through LDS or in registers): likewise
    for t in tiles + [-1]:
        try:
            g = fsb.fs_test_conv(x, w, b, r, s, p, relu, prec, tile=t)
        except fsb.FsError as e:  # a tile that does not fit this shape (e.g. LDS-DMA needs Cin % 64 == 0)
            assert e.status == fsb.FS_ERR_UNSUPPORTED and t >= 0
            continue
        ran += 1
        ran_names.append(fsb.fs_conv_tile_name(prec, t) if t >= 0 else "auto")
        if t >= 0 and "dma" in ran_names[-1]:
            dma_out[ran_names[-1]] = g
        if t >= 0 and ("hs_" in ran_names[-1] or "hr_" in ran_names[-1]):
            hs_out[ran_names[-1]] = g
        if prec == BF16:
            assert_bf16_close(g, o, ab, what=f"case {ci} tile {t}")
        else:
            assert np.all(np.abs(g - o) <= 1e-5 * ab + 1e-6), f"case {ci} tile {t}: {np.abs(g - o).max()}"
    assert ran >= 2
    if prec == BF16 and Cin % 64 == 0:  # the LDS-DMA kernels ran on this shape
        assert ran >= 2 + sum(1 for t in tiles if "dma" in fsb.fs_conv_tile_name(prec, t))
    for fam in (dma_out, hs_out):  # so a tile choice never changes a result: identical bits across a family
        if fam:
            first_name, first = next(iter(fam.items()))
            for name, g in fam.items():
                assert np.array_equal(g.view(np.uint32), first.view(np.uint32)), \
                    f"case {ci}: {name} differs from {first_name}"
    if prec == BF16 and k == 3 and s == 1 and Cin == 64 and Cout % 64 == 0 and W == 56:  # and the halo kernel
        assert any("halo" in n for n in ran_names), ran_names
    if prec == BF16:  # the streamed-weight halo kernel exactly where it fits
        assert any("hs_" in n for n in ran_names) == (ci in HS_CASES), ran_names


def _tile_index(name_part):
    return next(t for t in range(fsb.fs_conv_num_tiles(BF16)) if name_part in fsb.fs_conv_tile_name(BF16, t))


def test_halo_kernel_bits_equal_implicit_gemm_for_one_chunk(gpu_lib):
    # With Cin = 64 the halo kernel sums each output over the taps in the
    # implicit GEMM's K order with the same MFMA sequence: identical bits.
    x, w, b, r = _conv_inputs(CONV_CASES[8], BF16, 17)  # 12 x 56, Cin 64, residual
    g_halo = fsb.fs_test_conv(x, w, b, r, 1, 1, 1, BF16, tile=_tile_index("halo_4x56"))
    g_dma = fsb.fs_test_conv(x, w, b, r, 1, 1, 1, BF16, tile=_tile_index("dma2_128x64"))
    assert np.array_equal(g_halo.view(np.uint32), g_dma.view(np.uint32))


def test_conv_repeat_is_bit_identical(gpu_lib):
    x, w, b, r = _conv_inputs(CONV_CASES[2], BF16, 7)
    g0 = fsb.fs_test_conv(x, w, b, r, 1, 1, 1, BF16)
    for _ in range(5):
        assert np.array_equal(fsb.fs_test_conv(x, w, b, r, 1, 1, 1, BF16), g0)


@pytest.mark.parametrize("kind", ["halo", "hs", "hs_large", "stem"])
def test_persistent_kernels_repeat_bit_identical(gpu_lib, kind):
    # The persistent kernels wait on fixed vector-memory counts; if the
    # compiler drops or merges any of the loads and stores those counts
    # assume, a step can start before its operands have landed and results
    # vary from run to run.  Identical inputs must give identical bits, at a
    # batch where each workgroup walks only two or three tiles (first steps
    # weigh most); "hs_large" has 256 tiles of 128 x 128.
    rng = np.random.default_rng(11)
    if kind == "stem":
        x = oracle.round_bf16(rng.standard_normal((16, 224, 224, 3)).astype(np.float32))
        w = oracle.round_bf16((rng.standard_normal((64, 7, 7, 3)) * np.sqrt(2.0 / 147)).astype(np.float32))
        b = (rng.standard_normal(64) * 0.1).astype(np.float32)
        run = lambda: fsb.fs_test_stem_pool(x, w, b)
    else:
        B, H, Ci, Co = {"halo": (16, 56, 64, 64), "hs": (16, 7, 512, 512), "hs_large": (4, 64, 128, 256)}[kind]
        x = oracle.round_bf16(rng.standard_normal((B, H, H, Ci)).astype(np.float32))
        w = oracle.round_bf16((rng.standard_normal((Co, 3, 3, Ci)) * np.sqrt(2.0 / (9 * Ci))).astype(np.float32))
        b = (rng.standard_normal(Co) * 0.1).astype(np.float32)
        r = oracle.round_bf16(rng.standard_normal((B, H, H, Co)).astype(np.float32))
        t = _tile_index("halo_4x56" if kind == "halo" else "hs_128x128")
        run = lambda: fsb.fs_test_conv(x, w, b, r, 1, 1, 1, BF16, tile=t)
    g0 = run()
    for i in range(12):
        assert np.array_equal(run().view(np.uint32), g0.view(np.uint32)), i


@pytest.mark.parametrize("B,H,W", [(2, 32, 32), (1, 224, 224), (3, 30, 20), (1, 2, 6)])
def test_stem_conv_maxpool_fused(gpu_lib, B, H, W):
    # the fused stem equals the conv and the max pool run separately, bit for
    # bit (same sums, and max commutes with the bf16 rounding), and the oracle
    rng = np.random.default_rng(H * 1000 + W)
    x = oracle.round_bf16(rng.standard_normal((B, H, W, 3)).astype(np.float32))
    w = oracle.round_bf16((rng.standard_normal((64, 7, 7, 3)) * np.sqrt(2.0 / 147)).astype(np.float32))
    b = (rng.standard_normal(64) * 0.1).astype(np.float32)
    g = fsb.fs_test_stem_pool(x, w, b)
    sep = fsb.fs_test_maxpool(fsb.fs_test_conv(x, w, b, None, 2, 3, 1, BF16), 3, 2, 1, BF16)
    assert g.shape == sep.shape
    assert np.array_equal(g.view(np.uint32), sep.view(np.uint32))
    c, ab = oracle.conv2d(x, w, b, 2, 3, 1, None, "bf16", want_abs=True)
    o = oracle.maxpool(c, 3, 2, 1)
    abp = oracle.maxpool(ab, 3, 2, 1)  # a bound for whichever window element won
    assert_bf16_close(g, o, abp, frac_exact=0.99, what=f"stem {B}x{H}x{W}")


# -------------------------------------------------------------------- pooling
@pytest.mark.parametrize("prec", [BF16, F32])
@pytest.mark.parametrize("k,s,p,hw", [(3, 2, 1, (17, 16)), (2, 2, 0, (16, 14)), (3, 2, 1, (112, 112)),
                                      (3, 1, 1, (9, 5))])
def test_maxpool_bit_exact(gpu_lib, prec, k, s, p, hw):
    rng = np.random.default_rng(k * 10 + hw[0])
    x = rng.standard_normal((2,) + hw + (64,)).astype(np.float32)
    if prec == BF16:
        x = oracle.round_bf16(x)
    g = fsb.fs_test_maxpool(x, k, s, p, prec)
    assert np.array_equal(g, oracle.maxpool(x, k, s, p))


@pytest.mark.parametrize("prec", [BF16, F32])
@pytest.mark.parametrize("shape", [(3, 7, 7, 512), (2, 7, 7, 2048), (4, 16, 16, 32)])
def test_gap_parity(gpu_lib, prec, shape):
    rng = np.random.default_rng(shape[-1])
    x = np.abs(rng.standard_normal(shape)).astype(np.float32)
    if prec == BF16:
        x = oracle.round_bf16(x)
    g = fsb.fs_test_gap(x, prec)
    o = oracle.gap(x, PREC[prec])
    if prec == BF16:
        assert_bf16_close(g, o, frac_exact=0.99, what="gap")
    else:
        assert np.max(np.abs(g - o)) <= 1e-6 * np.abs(o).max()


# ------------------------------------------------------------------------- fc
@pytest.mark.parametrize("prec", [BF16, F32])
@pytest.mark.parametrize("B,K,N,relu,out_storage", [
    (32, 512, 1000, 0, 0),     # ResNet-18 head
    (5, 2048, 1000, 0, 0),     # ResNet-50 head, ragged batch
    (3, 25088, 64, 1, 1),      # VGG fc1 fan-in (split-K), hidden output
    (70, 4096, 96, 1, 1),      # more than 64 images
    (32, 4096, 4096, 1, 1),    # VGG fc2: weight-streaming kernel, split-K over 64-feature tiles
    (17, 1088, 200, 0, 0),     # weight-streaming kernel: a split ending inside a 256-wide chunk, ragged B and N
    (4, 32, 10, 0, 0),         # tiny head
    (1, 512, 1000, 0, 0),
])
def test_fc_parity(gpu_lib, prec, B, K, N, relu, out_storage):
    rng = np.random.default_rng(B * 7 + K)
    x = rng.standard_normal((B, K)).astype(np.float32)
    w = (rng.standard_normal((N, K)) * np.sqrt(2.0 / K)).astype(np.float32)
    b = (rng.standard_normal(N) * 0.1).astype(np.float32)
    if prec == BF16:
        x, w = oracle.round_bf16(x), oracle.round_bf16(w)
    st = "bf16" if (prec == BF16 and out_storage) else "fp32"
    o = oracle.fc(x, w, b, relu, st)
    ab = np.abs(x).astype(np.float64) @ np.abs(w).astype(np.float64).T
    g = fsb.fs_test_fc(x, w, b, relu, prec, out_storage)
    if st == "bf16":
        assert_bf16_close(g, o, ab, what="fc")
    else:
        assert np.all(np.abs(g - o) <= 1e-5 * ab + 1e-6), np.abs(g - o).max()


# -------------------------------------------------------- softmax + combine
@pytest.mark.parametrize("N,B,C,scale", [(3, 32, 1000, 80.0), (5, 7, 1000, 3.0), (2, 4, 10, 2.0),
                                         (1, 3, 4096, 1.0), (4, 2, 257, 0.0), (8, 5, 1000, 40.0),
                                         (7, 3, 129, 1.0)])
def test_softmax_combine_parity(gpu_lib, N, B, C, scale):
    rng = np.random.default_rng(N * 100 + C)
    z = (rng.standard_normal((N, B, C)) * scale).astype(np.float32)
    g = fsb.fs_test_softmax_combine(z)
    p = oracle.softmax(z)
    o = oracle.combine(p, z)
    assert np.max(np.abs(g["probs"] - p)) <= 1e-6
    assert np.max(np.abs(g["mean"] - o["mean"])) <= 1e-6
    assert np.array_equal(g["top1"], o["top1"])  # logits are exact inputs: same argmax
    S = o["S"]
    for b in range(B):
        top2 = np.sort(S[b])[-2:] if C > 1 else S[b]
        if C == 1 or top2[1] - top2[0] > 2 * N * 1e-6:
            assert g["vote"][b] == o["vote"][b]
        else:
            assert S[b, g["vote"][b]] >= S[b].max() - 2 * N * 1e-6


@pytest.mark.parametrize("N,C", [(1, 7), (3, 4), (4, 1000), (3, 2000), (6, 5), (9, 1000)])
def test_combine_policies_match_the_oracle(gpu_lib, N, C):
    # few classes make equal vote counts common; (3, 2000), (6, 5), (9, 1000)
    # run the one-model-at-a-time kernel, the others the side-by-side one
    B = 64
    rng = np.random.default_rng(N * 7 + C)
    z = rng.standard_normal((N, B, C)).astype(np.float32)
    z[:, :4] = np.round(z[:, :4])  # exact logit ties: top-1 is the smallest maximising class
    o = oracle.combine(oracle.softmax(z), z)
    ref = fsb.fs_test_softmax_combine(z)
    cases = [(fsb.FS_COMBINE_PLURALITY, 0, 1)] + [(fsb.FS_COMBINE_ANY, c, k) for c in (0, C // 2, C - 1)
                                                  for k in sorted({1, (N + 1) // 2, N})]
    for policy, pos, k in cases:
        g = fsb.fs_test_softmax_combine_policy(z, policy, pos, k)
        assert np.array_equal(g["top1"], o["top1"])
        want = oracle.vote_policy(o["top1"], C, policy, pos, k)
        assert np.array_equal(g["vote"], want), (policy, pos, k)
        # probabilities, mean and top-1 do not depend on the policy
        for key in ("probs", "mean", "top1"):
            assert np.array_equal(g[key], ref[key]), key


def test_softmax_combine_exact_ties_take_lowest_index(gpu_lib):
    z = np.full((2, 3, 50), -1e4, np.float32)
    z[0, :, 31] = 0.0   # model 0 saturates on 31
    z[1, :, 12] = 0.0   # model 1 saturates on 12: S ties at 1.0
    z[0, 1, 5] = 0.0    # model 0, image 1: exact logit tie 5 vs 31
    g = fsb.fs_test_softmax_combine(z)
    # image 1: model 0 splits 0.5/0.5 over 5 and 31, so S[12] = 1 still wins
    assert g["vote"].tolist() == [12, 12, 12]
    assert g["top1"][0].tolist() == [31, 5, 31] and g["top1"][1].tolist() == [12, 12, 12]
