"""Thin HTTP/JSON front end of the ensemble library.

FlexServe answers a POST of a batch of images of any size and count
(Sec. 2.3) with every model's per-image classes together with the ensemble's
combined result (Fig. 1 caption; Sec. 2.1): ``{"model y_i": [c, ...]}`` for
every model i.  Classes are integer ids: the library has no class names.

The server is the standard library's threading HTTP server.  Every request
thread hands its images to one ``fs_batcher`` over the given handles, so
concurrent clients share device passes (the role of the paper's Gunicorn
workers).  The combine policy is fixed when the server starts: one pass
serves many requests, and the policy runs on the device as part of the
pass.

Request body (JSON): ``{"images": [<base64 of an image file>, ...]}`` (any
format PIL reads, converted to RGB) or ``{"arrays": [{"shape": [h, w, 3],
"data": <base64 of the h*w*3 uint8 bytes>}, ...]}``; optionally
``"policy": "mean" | "plurality" | "any"``, which must be the server's.
Response: ``{"model y_0": [...], ..., "combined": [...], "policy": ...}``.
``GET /health`` returns the ensemble's shape.
"""
from __future__ import annotations

import base64
import io
import json
import threading
from http.server import BaseHTTPRequestHandler, ThreadingHTTPServer

import numpy as np

from . import flexserve as fsb

POLICIES = {"mean": fsb.FS_COMBINE_MEAN, "plurality": fsb.FS_COMBINE_PLURALITY, "any": fsb.FS_COMBINE_ANY}
MAX_BODY = 256 << 20


class BadRequest(ValueError):
    pass


def decode_images(body: dict) -> list:
    """The request's images as uint8 HWC RGB arrays."""
    if not isinstance(body, dict):
        raise BadRequest("the body must be a JSON object")
    out = []
    for i, item in enumerate(body.get("images", [])):
        try:
            from PIL import Image
            with Image.open(io.BytesIO(base64.b64decode(item, validate=True))) as im:
                out.append(np.asarray(im.convert("RGB"), dtype=np.uint8))
        except Exception as ex:
            raise BadRequest(f"images[{i}]: not a readable image ({ex})") from None
    for i, item in enumerate(body.get("arrays", [])):
        try:
            h, w, c = (int(v) for v in item["shape"])
            raw = base64.b64decode(item["data"], validate=True)
        except Exception as ex:
            raise BadRequest(f"arrays[{i}]: needs shape [h, w, 3] and base64 data ({ex})") from None
        if c != 3 or h < 1 or w < 1 or len(raw) != h * w * 3:
            raise BadRequest(f"arrays[{i}]: shape {item['shape']} does not match {len(raw)} bytes of RGB")
        out.append(np.frombuffer(raw, np.uint8).reshape(h, w, 3))
    if not out:
        raise BadRequest("no images or arrays in the request")
    return out


def format_result(res: dict, policy: str) -> dict:
    """Per-model class lists and the combined result, as plain JSON types."""
    top1 = res["top1"]
    out = {f"model y_{i}": top1[i].tolist() for i in range(top1.shape[0])}
    out["combined"] = res["vote"].tolist()
    out["policy"] = policy
    return out


class Server:
    """HTTP front end over handles of one ensemble (the first and handles
    from its share()); start() serves from a background thread."""

    def __init__(self, handles, host="127.0.0.1", port=0, max_wait_us=200, policy="mean",
                 positive_class=0, min_votes=1):
        if policy not in POLICIES:
            raise ValueError(f"policy must be one of {sorted(POLICIES)}")
        self.handles = list(handles)
        self.policy = policy
        for h in self.handles:
            h.set_combine(POLICIES[policy], positive_class, min_votes)
        self.batcher = fsb.Batcher(self.handles, max_wait_us=max_wait_us)
        info = self.handles[0].info()
        self.shape = {"models": info["num_models"], "classes": info["num_classes"],
                      "max_batch": info["max_batch"], "policy": policy}
        server = self

        class Handler(BaseHTTPRequestHandler):
            def log_message(self, *a):  # quiet
                pass

            def _reply(self, code, obj):
                data = json.dumps(obj).encode()
                self.send_response(code)
                self.send_header("Content-Type", "application/json")
                self.send_header("Content-Length", str(len(data)))
                self.end_headers()
                self.wfile.write(data)

            def do_GET(self):
                if self.path.rstrip("/") == "/health":
                    self._reply(200, server.shape)
                else:
                    self._reply(404, {"error": "unknown path"})

            def do_POST(self):
                if self.path.rstrip("/") != "/infer":
                    self._reply(404, {"error": "unknown path"})
                    return
                try:
                    n = int(self.headers.get("Content-Length", "0"))
                    if n <= 0 or n > MAX_BODY:
                        raise BadRequest("missing or oversized body")
                    body = json.loads(self.rfile.read(n))
                    if "policy" in body and body["policy"] != server.policy:
                        raise BadRequest(f"this server combines by {server.policy!r}")
                    imgs = decode_images(body)
                except (BadRequest, ValueError) as ex:
                    self._reply(400, {"error": str(ex)})
                    return
                try:
                    res = server.batcher.infer(imgs, want_mean=False, want_top1=True)
                except fsb.FsError as ex:
                    self._reply(400 if ex.status == fsb.FS_ERR_INVALID else 500, {"error": str(ex)})
                    return
                self._reply(200, format_result(res, server.policy))

        self.httpd = ThreadingHTTPServer((host, port), Handler)
        # handler threads are joined by server_close(), so none is inside
        # the batcher when stop() closes it
        self.httpd.daemon_threads = False
        self.httpd.block_on_close = True
        self.thread = None

    @property
    def url(self) -> str:
        host, port = self.httpd.server_address[:2]
        return f"http://{host}:{port}"

    def start(self):
        self.thread = threading.Thread(target=self.httpd.serve_forever, daemon=True)
        self.thread.start()
        return self

    def stop(self):
        self.httpd.shutdown()
        self.httpd.server_close()
        if self.thread:
            self.thread.join()
        self.batcher.close()

    def __enter__(self):
        return self.start()

    def __exit__(self, *a):
        self.stop()


def main():
    """Serve a seeded synthetic ensemble of the benchmark workloads (random
    weights: there are no trained ones here)."""
    import argparse
    import sys
    import os
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="resnet18x3_bf16_b32")
    ap.add_argument("--host", default="127.0.0.1")
    ap.add_argument("--port", type=int, default=8000)
    ap.add_argument("--handles", type=int, default=2)
    ap.add_argument("--max-wait-us", type=int, default=200)
    ap.add_argument("--policy", default="mean", choices=sorted(POLICIES))
    ap.add_argument("--positive-class", type=int, default=0)
    ap.add_argument("--min-votes", type=int, default=1)
    args = ap.parse_args()
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import workloads as wl
    w = wl.workload(args.workload)
    ens = fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                       max_batch=w["batch"])
    handles = [ens] + [ens.share() for _ in range(args.handles - 1)]
    srv = Server(handles, args.host, args.port, args.max_wait_us, args.policy, args.positive_class, args.min_votes)
    import gc
    gc.collect()
    gc.freeze()  # the models and buffers live as long as the server: no full GC passes over them
    print(f"serving {args.workload} on {srv.url} (POST /infer, GET /health)", flush=True)
    try:
        srv.httpd.serve_forever()
    except KeyboardInterrupt:
        pass
    finally:
        srv.httpd.server_close()
        srv.batcher.close()
        for h in handles:
            h.close()


if __name__ == "__main__":
    main()
