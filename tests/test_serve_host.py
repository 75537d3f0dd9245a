"""Request decoding and response shape of the HTTP front end (no device)."""
import base64
import io

import numpy as np
import pytest

from paper_2003_01538_amd import serve


def _png(a):
    from PIL import Image
    buf = io.BytesIO()
    Image.fromarray(a).save(buf, format="PNG")
    return base64.b64encode(buf.getvalue()).decode()


def test_decode_png_and_raw_arrays():
    rng = np.random.default_rng(0)
    a = rng.integers(0, 256, size=(17, 23, 3), dtype=np.uint8)
    b = rng.integers(0, 256, size=(5, 9, 3), dtype=np.uint8)
    imgs = serve.decode_images({"images": [_png(a)],
                                "arrays": [{"shape": [5, 9, 3], "data": base64.b64encode(b.tobytes()).decode()}]})
    assert len(imgs) == 2
    assert np.array_equal(imgs[0], a) and np.array_equal(imgs[1], b)
    gray = serve.decode_images({"images": [_png(a[:, :, 0].copy())]})[0]  # converted to RGB
    assert gray.shape == (17, 23, 3) and np.array_equal(gray[:, :, 2], a[:, :, 0])


@pytest.mark.parametrize("body", [
    {},                                                            # no images
    [],                                                            # not an object
    {"images": ["not base64!"]},
    {"images": [base64.b64encode(b"not an image").decode()]},
    {"arrays": [{"shape": [2, 2, 3], "data": base64.b64encode(b"123").decode()}]},  # size mismatch
    {"arrays": [{"shape": [2, 2, 4], "data": base64.b64encode(bytes(16)).decode()}]},  # not RGB
    {"arrays": [{"data": ""}]},                                    # no shape
])
def test_decode_rejects_bad_requests(body):
    with pytest.raises(serve.BadRequest):
        serve.decode_images(body)


def test_result_format():
    res = {"top1": np.array([[3, 1], [3, 7], [0, 1]], np.int32), "vote": np.array([3, 1], np.int32)}
    out = serve.format_result(res, "plurality")
    assert out == {"model y_0": [3, 1], "model y_1": [3, 7], "model y_2": [0, 1], "combined": [3, 1],
                   "policy": "plurality"}
