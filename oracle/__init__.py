"""CPU oracle for the ensemble-inference path (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never calls it, and the two share no code: the oracle's
arithmetic is the plain C in ``fso.c`` (double accumulation, storage rounding
at the points where the GPU path stores), driven layer by layer from Python.

What it follows in the FlexServe paper:
* one data transformation of the request's images, shared by all models
  (Fig. 1 caption; Sec. 2.2) -> ``preprocess_batch``;
* every model of the ensemble runs on that one tensor (Sec. 2.2) and the
  batch size is arbitrary (Sec. 2.3) -> ``forward_model``;
* the outputs of all models are returned together, per model and per image
  (Fig. 1 caption; Sec. 2.3), and combined (Sec. 2.1) -> ``ensemble``.
The paper fixes no arithmetic; the readings taken where it is silent are the
textbook definitions written in ``fso.c``.  Storage points follow the HIP
path's: a residual block's projection shortcut (``projection_shortcuts``) is
summed into the block's last conv before that conv's one rounding.

Parity pins for every function live in ``tests/test_oracle_pins.py``.  The
end-to-end values of the random bf16 networks have no external pin beyond the
composition of the per-layer pins: parity unpinned for those values as a whole.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fso.c")
_LIB = os.path.join(_HERE, "libfso.so")
_lib = None

F32 = np.float32
PREC = {"fp32": 0, "bf16": 1}


def build(force: bool = True) -> str:
    """Compile fso.c with gcc (no fast-math; OpenMP over outputs only)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fno-fast-math", "-ffp-contract=off",
                               "-std=c11", "-Wall", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        P, I, I64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
        L.fso_round_bf16.restype = ctypes.c_float
        L.fso_round_bf16.argtypes = [ctypes.c_float]
        L.fso_round_array.argtypes = [P, I64, I, P]
        L.fso_set_acc32.argtypes = [I]
        L.fso_preprocess.argtypes = [P, I, I, I, I, I, P, P, I, P]
        L.fso_fold_bn.argtypes = [P, I, I64, P, P, P, I, P, P]
        L.fso_conv2d.argtypes = [P, I, I, I, I, P, P, P, I, I, I, I, I, I, I, P, P]
        L.fso_conv2d_proj.argtypes = [P, I, I, I, I, P, P, P, I, I, I, P, P, I, I, I, I, I, I, I, I, P, P]
        L.fso_maxpool.argtypes = [P, I, I, I, I, I, I, I, P]
        L.fso_gap.argtypes = [P, I, I, I, I, I, P]
        L.fso_flatten_nchw.argtypes = [P, I, I, I, I, P]
        L.fso_fc.argtypes = [P, I, I, P, P, I, I, I, P]
        L.fso_softmax.argtypes = [P, I, I, P]
        L.fso_argmax.argtypes = [P, I]
        L.fso_combine.argtypes = [P, P, I, I, I, P, P, P, P]
        L.fso_vote_policy.argtypes = [P, I, I, I, I, I, I, P]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt=F32):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


# ------------------------------------------------------------- primitives
def round_bf16(x) -> np.ndarray:
    x = _c(x)
    out = np.empty_like(x)
    lib().fso_round_array(_p(x), x.size, 1, _p(out))
    return out


def set_acc32(on: bool):
    lib().fso_set_acc32(int(bool(on)))


def preprocess(img, out_h, out_w, mean, std, prec="fp32"):
    """One uint8 HWC image (h, w, 3), possibly a strided view -> [out_h, out_w, 3]."""
    img = np.asarray(img)
    h, w, _ = img.shape
    buf = np.ascontiguousarray(img, dtype=np.uint8)
    out = np.empty((out_h, out_w, 3), F32)
    m, s = _c(np.array(mean)), _c(np.array(std))
    lib().fso_preprocess(_p(buf), h, w, 3 * w, out_h, out_w, _p(m), _p(s), PREC[prec], _p(out))
    return out


def preprocess_batch(imgs, out_h, out_w, mean, std, prec="fp32"):
    """The single transformation shared by every model: [B, out_h, out_w, 3]."""
    return np.stack([preprocess(im, out_h, out_w, mean, std, prec) for im in imgs])


def fold_bn(weight, scale, shift, bias, prec="fp32"):
    w = _c(weight)
    cout = w.shape[0]
    wo, bo = np.empty_like(w), np.empty(cout, F32)
    lib().fso_fold_bn(_p(w), cout, w.size // cout, _p(_c(scale)), _p(_c(shift)),
                      _p(_c(bias)), PREC[prec], _p(wo), _p(bo))
    return wo, bo


def conv2d(x, w, bias, stride, pad, relu, res=None, prec="fp32", want_abs=False):
    """x [B,H,W,Cin], w [Cout,kh,kw,Cin] -> [B,Ho,Wo,Cout]."""
    x, w = _c(x), _c(w)
    B, H, W, Cin = x.shape
    Cout, kh, kw, _ = w.shape
    Ho, Wo = (H + 2 * pad - kh) // stride + 1, (W + 2 * pad - kw) // stride + 1
    out = np.empty((B, Ho, Wo, Cout), F32)
    ab = np.empty_like(out) if want_abs else None
    lib().fso_conv2d(_p(x), B, H, W, Cin, _p(w), _p(_c(bias)), _p(_c(res)), Cout, kh, kw,
                     stride, pad, int(relu), PREC[prec], _p(out), _p(ab))
    return (out, ab) if want_abs else out


def conv2d_proj(x, w, bias, stride, pad, relu, x2, w2, bias2, stride2, prec="fp32", want_abs=False):
    """A block's last conv with its projection shortcut summed in before the
    one rounding: x [B,H,W,Cin], w [Cout,kh,kw,Cin], x2 [B,H2,W2,C2] (the
    block input), w2 [Cout,1,1,C2] or [Cout,C2], 1x1 with stride stride2."""
    x, w, x2 = _c(x), _c(w), _c(x2)
    w2 = _c(np.asarray(w2).reshape(w.shape[0], -1))
    B, H, W, Cin = x.shape
    Cout, kh, kw, _ = w.shape
    _, H2, W2, C2 = x2.shape
    Ho, Wo = (H + 2 * pad - kh) // stride + 1, (W + 2 * pad - kw) // stride + 1
    assert w2.shape[1] == C2 and (Ho - 1) * stride2 < H2 and (Wo - 1) * stride2 < W2
    out = np.empty((B, Ho, Wo, Cout), F32)
    ab = np.empty_like(out) if want_abs else None
    lib().fso_conv2d_proj(_p(x), B, H, W, Cin, _p(w), _p(_c(bias)), _p(x2), H2, W2, C2, _p(w2), _p(_c(bias2)),
                          stride2, Cout, kh, kw, stride, pad, int(relu), PREC[prec], _p(out), _p(ab))
    return (out, ab) if want_abs else out


def projection_shortcuts(layers):
    """{projection layer index: the conv that sums it in}.  A projection
    shortcut is a 1x1 conv without activation and padding whose output is
    read only as the residual of one later conv (He et al.'s downsample
    branch); that conv takes its products into its own sum."""
    readers = {}
    for i, L in enumerate(layers):
        readers.setdefault(L["src"], []).append((i, "src"))
        if L["op"] == "conv" and L.get("res", -1) >= 0:
            readers.setdefault(L["res"], []).append((i, "res"))
    out = {}
    for d, L in enumerate(layers):
        if L["op"] != "conv" or L["k"] != 1 or L["pad"] != 0 or L["relu"]:
            continue
        r = readers.get(d, [])
        if len(r) == 1 and r[0][1] == "res" and layers[r[0][0]]["op"] == "conv":
            out[d] = r[0][0]
    return out


def maxpool(x, k, stride, pad):
    x = _c(x)
    B, H, W, C = x.shape
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    out = np.empty((B, Ho, Wo, C), F32)
    lib().fso_maxpool(_p(x), B, H, W, C, k, stride, pad, _p(out))
    return out


def gap(x, prec="fp32"):
    x = _c(x)
    B, H, W, C = x.shape
    out = np.empty((B, C), F32)
    lib().fso_gap(_p(x), B, H, W, C, PREC[prec], _p(out))
    return out


def flatten_nchw(x):
    x = _c(x)
    B, H, W, C = x.shape
    out = np.empty((B, C * H * W), F32)
    lib().fso_flatten_nchw(_p(x), B, H, W, C, _p(out))
    return out


def fc(x, w, bias, relu, prec="fp32"):
    x, w = _c(x), _c(w)
    B, K = x.shape
    N = w.shape[0]
    out = np.empty((B, N), F32)
    lib().fso_fc(_p(x), B, K, _p(w), _p(_c(bias)), N, int(relu), PREC[prec], _p(out))
    return out


def softmax(z):
    z = _c(z)
    C = z.shape[-1]
    out = np.empty_like(z)
    lib().fso_softmax(_p(z), z.size // C, C, _p(out))
    return out


def argmax(x) -> int:
    x = _c(x)
    return int(lib().fso_argmax(_p(x), x.size))


def combine(p, z=None):
    """p, z [N, B, C] -> dict(S, mean, vote [B], top1 [N, B])."""
    p = _c(p)
    N, B, C = p.shape
    S, mean = np.empty((B, C), F32), np.empty((B, C), F32)
    vote = np.empty(B, np.int32)
    top1 = np.empty((N, B), np.int32)
    zc = _c(z)
    lib().fso_combine(_p(p), _p(zc), N, B, C, _p(S), _p(mean), _p(vote),
                      _p(top1) if zc is not None else None)
    return dict(S=S, mean=mean, vote=vote, top1=top1 if zc is not None else None)


PLURALITY, ANY = 1, 2


def vote_policy(top1, C, policy, pos=0, k=1):
    """top1 [N, B] -> [B]: plurality (policy 1) or detection of class `pos`
    by at least k models (policy 2; k = 1 is the OR of Sec. 2.1)."""
    t = np.ascontiguousarray(top1, np.int32)
    N, B = t.shape
    out = np.empty(B, np.int32)
    lib().fso_vote_policy(_p(t), N, B, int(C), int(policy), int(pos), int(k), _p(out))
    return out


# ------------------------------------------------------------- networks
def prepare_model(layers, prec):
    """Fold BN into the conv weights and round the weights to the storage
    type once (the weight storage point).  Returns per-layer (w, b)."""
    out = []
    for L in layers:
        if L["op"] == "conv":
            out.append(fold_bn(L["weight"], L.get("bn_scale"), L.get("bn_shift"),
                               L.get("bias"), prec))
        elif L["op"] == "fc":
            w = _c(L["weight"])
            w = round_bf16(w) if prec == "bf16" else w
            b = _c(L["bias"]) if L.get("bias") is not None else np.zeros(L["cout"], F32)
            out.append((w, b))
        else:
            out.append(None)
    return out


def forward_model(layers, x, prec="fp32", prepared=None, keep=False):
    """Run one network on the transformed batch x [B, H, W, 3].  Returns the
    fp32 logits [B, classes] (and every layer output when keep=True)."""
    prepared = prepared or prepare_model(layers, prec)
    outs = []
    last = len(layers) - 1
    proj = projection_shortcuts(layers)
    folded = {c: d for d, c in proj.items()}
    for i, (L, wb) in enumerate(zip(layers, prepared)):
        if i in proj:  # summed into its block's last conv, never stored on its own
            outs.append(None)
            continue
        src = x if L["src"] < 0 else outs[L["src"]]
        op = L["op"]
        if op == "conv" and i in folded:
            d = folded[i]
            D = layers[d]
            x2 = x if D["src"] < 0 else outs[D["src"]]
            y = conv2d_proj(src, wb[0], wb[1], L["stride"], L["pad"], L["relu"], x2, prepared[d][0],
                            prepared[d][1], D["stride"], prec)
        elif op == "conv":
            res = outs[L["res"]] if L.get("res", -1) >= 0 else None
            y = conv2d(src, wb[0], wb[1], L["stride"], L["pad"], L["relu"], res, prec)
        elif op == "maxpool":
            y = maxpool(src, L["k"], L["stride"], L["pad"])
        elif op == "gap":
            y = gap(src, prec)
        elif op == "fc":
            f = flatten_nchw(src) if L.get("flatten_nchw") else src.reshape(src.shape[0], -1)
            y = fc(f, wb[0], wb[1], L["relu"], "fp32" if i == last else prec)
        else:
            raise ValueError(op)
        outs.append(y)
        if not keep and i > 0:
            # free outputs no later layer reads
            needed = {M["src"] for M in layers[i + 1:]} | {M.get("res", -1) for M in layers[i + 1:]}
            needed |= {layers[d]["src"] for d, c in proj.items() if c > i}
            for j in range(i + 1):
                if j not in needed and j != i:
                    outs[j] = None
    return (outs[-1], outs) if keep else outs[-1]


def ensemble(models, imgs, out_hw, mean, std, prec="fp32", prepared=None):
    """Whole path: one transformation, every model on it, softmax per model,
    combination.  Returns dict(x, logits [N,B,C], probs, S, mean, vote, top1)."""
    x = preprocess_batch(imgs, out_hw[0], out_hw[1], mean, std, prec)
    prepared = prepared or [prepare_model(m, prec) for m in models]
    logits = np.stack([forward_model(m, x, prec, pp) for m, pp in zip(models, prepared)])
    probs = softmax(logits)
    comb = combine(probs, logits)
    return dict(x=x, logits=logits, probs=probs, **comb)
