"""Host-side check of the float-reciprocal quotient the conv and preprocess
kernels use for pixel, row and filter-tap indices: with inv the correctly
rounded fp32 reciprocal of d, truncating (n + 0.5) * inv in fp32 gives
floor(n / d) for every 0 <= n < 2^22.  numpy's float32 division and
multiplication round like the GPU's IEEE fp32 operations, so the kernels'
expression is evaluated here exactly as the device evaluates it."""
import numpy as np

LIMIT = 1 << 22
# divisors of the served shapes: output planes and widths (224 input, stride
# 2 stem and pools), channel counts of a K-tile's filter tap, filter widths
SHAPE_DIVISORS = [12544, 3136, 784, 196, 49, 112, 56, 28, 14, 7, 16, 64, 128, 256, 512, 1024, 2048, 1, 3, 4,
                  448, 896, 2 * 224, 2 * 112, 2 * 1000, 2 * 320, 2 * 160]


def fdiv(n, d, half=0.5):
    inv = np.float32(1.0) / np.float32(d)
    return ((n.astype(np.float32) + np.float32(half)) * inv).astype(np.int64)


def boundary_dividends(d):
    """Every n = q d and n = q d + d - 1 below the limit: the dividends whose
    quotient lies nearest an integer from above and from below."""
    q = np.arange(0, (LIMIT - 1) // d + 1, dtype=np.int64)
    n = np.concatenate([q * d, q * d + d - 1])
    return n[n < LIMIT]


def test_every_dividend_for_the_shape_divisors():
    n = np.arange(LIMIT, dtype=np.int64)
    for d in SHAPE_DIVISORS:
        assert np.array_equal(fdiv(n, d), n // d), d


def test_quotient_boundaries_for_every_divisor_up_to_4096_and_large_ones():
    rng = np.random.default_rng(7)
    divisors = list(range(1, 4097)) + [int(x) for x in rng.integers(4097, LIMIT, 300)] + [LIMIT - 1]
    for d in divisors:
        n = boundary_dividends(d)
        assert np.array_equal(fdiv(n, d), n // d), d


def test_the_half_offset_is_needed():
    # without the 0.5 a reciprocal rounded down puts exact multiples just
    # below their quotient: the check above would catch that form
    bad = 0
    for d in range(1, 4097):
        n = boundary_dividends(d)
        bad += int(np.count_nonzero(fdiv(n, d, half=0.0) != n // d))
    assert bad > 0
