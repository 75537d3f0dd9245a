"""Benchmark of the ensemble-inference hot path on one MI355X.

One step = one device pass of the whole path over one batch already resident
in HBM: the shared resize+normalise of the batch, every model's forward pass,
the softmax per model and the ensemble combine (fs_infer_device).  The
default workload is three ResNet-18-shaped models in bf16 on a batch of 32
uint8 256x256 images resized to 224x224.

Prints ONE JSON line (rank 0, N=1):
  value = images/s of the whole ensemble = B * K / (time of K steps),
  roofline = the conv kernels (the dominant cost) measured with HIP events on
             the launch stream over the timed steps, against bf16 MFMA peak,
  cpu_baseline = the CPU oracle on this host, timed on a bounded sample.
"""
import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 (the fp32 convs run on fp32 MFMA)
DEFAULT_WORKLOAD = "resnet18x3_bf16_b32"
METRIC = "ensemble images/sec at B=32 (3xResNet-18, bf16) + MFMA util vs peak"
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    help="tiny2_fp32_b4, resnet18x3_bf16_b32 (the headline), hetero_r18_r50_vgg11_bf16_b32, "
                         "resnet50x5_bf16_b256")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="bound on the CPU-oracle sample (0 disables it)")
    ap.add_argument("--dump-launches", default="",
                    help="write the per-launch event times of one profiled step to this JSON file")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (scales the HBM byte "
                         "counters of a profiler run) and exit")
    ap.add_argument("--graphs", action="store_true",
                    help="record each step's launches once and replay them (fs_graphs_enable) instead of "
                         "launching every kernel from the host (the default, measured faster)")
    ap.add_argument("--combine", default="mean", choices=["mean", "plurality", "any"],
                    help="combine policy of vote (any: class 0 detected by at least one model)")
    ap.add_argument("--serve", action="store_true",
                    help="only time the request stream (200 requests of 1..64 ragged images, host "
                         "images in, host results out): one client, 4 clients on shared handles, "
                         "4 clients through one batcher; print one JSON line and exit")
    ap.add_argument("--max-wait-us", type=int, default=100, help="batcher wait for --serve")
    ap.add_argument("--no-e2e", action="store_true",
                    help="skip the end-to-end fs_infer timing (host images in, host results out), so that "
                         "only device-resident passes run, as in a kernel-trace profile")
    ap.add_argument("--no-profile", action="store_true",
                    help="time without the per-launch events (no roofline)")
    ap.add_argument("--batch", type=int, default=0,
                    help="images per step (default: the workload's batch); other sizes are a sweep, not the "
                         "configuration the metric is quoted on")
    ap.add_argument("--max-batch", type=int, default=0,
                    help="ensemble max_batch (default: the workload's batch); a smaller one runs each step as "
                         "ceil(B / max_batch) device passes (micro-batches)")
    ap.add_argument("--cold", action="store_true",
                    help="before every profiled step, write a 512 MiB buffer on the launch stream so that the step "
                         "starts with its inputs and weights out of the caches (the per-kernel rates are then cold "
                         "for the transformation's image reads and the weight reads)")
    ap.add_argument("--no-vendor-gemm", action="store_true",
                    help="skip timing the vendor GEMM (torch.bmm, hipBLASLt) on every conv layer's GEMM shape, "
                         "the reference column vendor_us of roofline.conv_layers")
    ap.add_argument("--tuning-log", default="",
                    help="write the tile tuner's candidate timings (fs_tuning_log) to this file")
    return ap.parse_args()


PROFILE = os.path.join(ROOT, "profiles", "conv_resnet18x3_b32.md")


def conv_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in ("conv.hip", "conv_dma.hip", "conv_hs.hip", "lds_dma.hpp"):
        with open(os.path.join(ROOT, "paper_2003_01538_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counted_traffic():
    """HBM bytes per conv launch from the committed rocprofv3 counter summary,
    or None when the conv sources changed since the counters were taken."""
    try:
        txt = open(PROFILE).read()
    except OSError:
        return None
    vals = dict(l.split(":", 1) for l in txt.splitlines() if l.startswith(("traffic_bytes", "kernel-source")))
    if vals.get("kernel-source-sha256-16", "").split()[0:1] != [conv_source_hash()]:
        return None
    return int(vals["traffic_bytes_per_conv_launch"])


def vendor_gemm_us(Z, M, N, K, reps=20):
    """Event time of torch.bmm (hipBLASLt) for Z GEMMs [M x K] x [K x N] in
    bf16: the layer's GEMM with its im2col operand already materialised, so
    only the library's GEMM is timed (a reference, never the product path)."""
    import torch
    a = torch.randn(Z, M, K, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(Z, K, N, device="cuda", dtype=torch.bfloat16).contiguous()
    c = torch.empty(Z, M, N, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        torch.bmm(a, b, out=c)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        torch.bmm(a, b, out=c)
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) / reps * 1e3


def vendor_reference(conv_layers, by_layer, peak):
    """Adds vendor_us / vendor_frac_peak to every conv layer entry."""
    import torch
    cache = {}
    for ent, rs in zip(conv_layers, (rs for _, rs in sorted(by_layer.items()))):
        M, N, K = ent["MNK"]
        Z = max(1, round(rs[0]["flops"] / (2.0 * M * N * K)))
        key = (Z, M, N, K)
        if key not in cache:
            cache[key] = vendor_gemm_us(Z, M, N, K)
        us = cache[key]
        ent["vendor_us"] = round(us, 2)
        ent["vendor_frac_peak"] = round(rs[0]["flops"] / (us * 1e-6) / 1e12 / peak, 4)
    torch.cuda.empty_cache()
    return {"what": "torch.bmm (hipBLASLt), bf16, on each conv layer's GEMM with the im2col operand materialised "
                    "(no bias, residual or pooling); reference only",
            "conv_us_per_step": round(sum(e["us"] for e in conv_layers), 1),
            "vendor_us_per_step": round(sum(e["vendor_us"] for e in conv_layers), 1)}


def omp_threads():
    try:
        return int(ctypes.CDLL("libgomp.so.1").omp_get_max_threads())
    except OSError:
        return os.cpu_count()


def _oracle_rate(w, imgs, prec, seconds):
    """Images/s of the oracle over a bounded sample of imgs (all models)."""
    import oracle
    import workloads as wl
    prepared = [oracle.prepare_model(m, prec) for m in w["models"]]
    n, t0 = 0, time.perf_counter()
    while n < len(imgs):
        oracle.ensemble(w["models"], imgs[n:n + 1], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, prec, prepared)
        n += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    return n / dt, (f"{n} of the {len(imgs)} images through all {len(w['models'])} models "
                    f"({prec} storage, double accumulation), {dt:.1f} s"), prepared


def cpu_baseline(w, imgs, seconds):
    """The oracle on this host's cores: fp32 storage (the reported value) and,
    for a bf16 workload, its bf16-storage emulation alongside; plus fp32 on
    one thread for one image."""
    import oracle
    import workloads as wl
    v, sample, prepared = _oracle_rate(w, imgs, "fp32", seconds)
    out = {"value": v, "unit": "images/s", "cores": omp_threads(), "kind": "oracle", "sample": sample}
    if w["precision"] == "bf16":
        vb, sb, _ = _oracle_rate(w, imgs, "bf16", seconds / 2)
        out["bf16_storage"] = {"value": vb, "unit": "images/s", "cores": omp_threads(), "sample": sb}
    # the same oracle on one thread, one image (its sums do not depend on the thread count)
    try:
        gomp = ctypes.CDLL("libgomp.so.1")
    except OSError:
        return out
    threads = gomp.omp_get_max_threads()
    gomp.omp_set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.ensemble(w["models"], imgs[:1], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, "fp32", prepared)
        dt1 = time.perf_counter() - t0
    finally:
        gomp.omp_set_num_threads(threads)
    out["single_thread"] = {"value": 1 / dt1, "unit": "images/s", "cores": 1,
                            "sample": f"1 image, fp32 storage, {dt1:.1f} s"}
    return out


def serve_bench(args):
    """Closed-loop request stream, end to end through fs_infer (PCIe
    included): each client sends its next request when the last returned."""
    import threading
    import torch
    import workloads as wl
    from paper_2003_01538_amd import flexserve as fsb

    torch.cuda.set_device(0)
    sw = wl.STREAM_WORKLOAD
    w = wl.workload(sw["ensemble"])
    reqs = wl.request_stream(sw["seed"], sw["n_requests"], sw["sizes"], sw["lo"], sw["hi"])
    n_img = sum(len(q) for q in reqs)
    Bm, K = max(sw["sizes"]), 4
    ens = fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                       max_batch=Bm)
    handles = [ens] + [ens.share() for _ in range(K - 1)]
    # conv tiles for every batch size a pass can see, timed before the clock
    # starts; the largest batch of the largest images first, so the pinned
    # staging buffers reach their final size here, not inside the timed loops
    warm = [np.zeros((sw["hi"], sw["hi"], 3), np.uint8)] * Bm
    for h in handles:
        for b in [Bm] + list(range(1, Bm)):
            h.infer(warm[:b], want_logits=False)

    import gc
    gc.collect()
    gc.freeze()

    def run_clients(call):
        errs = []

        def client(k):
            try:
                for q in reqs[k::K]:
                    call(k, q)
            except Exception as ex:
                errs.append(ex)
        ts = [threading.Thread(target=client, args=(k,)) for k in range(K)]
        t0 = time.perf_counter()
        for t in ts:
            t.start()
        for t in ts:
            t.join()
        if errs:
            raise errs[0]
        return time.perf_counter() - t0

    def pct(v):
        v = np.asarray(v)
        return {"p50": round(float(np.percentile(v, 50)), 3), "p99": round(float(np.percentile(v, 99)), 3)}

    lat = []
    t0 = time.perf_counter()
    for q in reqs:
        t1 = time.perf_counter()
        ens.infer(q, want_logits=False)
        lat.append((time.perf_counter() - t1) * 1e3)
    seq_s = time.perf_counter() - t0
    lat_sh = []

    def timed(fn, k, q, out):
        t1 = time.perf_counter()
        fn(k, q)
        out.append((time.perf_counter() - t1) * 1e3)
    shared_s = run_clients(lambda k, q: timed(lambda k_, q_: handles[k_].infer(q_, want_logits=False), k, q, lat_sh))
    res = {}
    for nw in (1, 2, 4):  # one batcher worker per handle, all warmed above
        with fsb.Batcher(handles[:nw], max_wait_us=args.max_wait_us) as bt:
            lat_b = []
            t = run_clients(lambda k, q: timed(lambda k_, q_: bt.infer(q_, want_logits=False), k, q, lat_b))
            res[nw] = dict(images_per_s=round(n_img / t, 1), passes=bt.stats()["passes"], request_ms=pct(lat_b))
    for h in handles:
        h.close()
    print(json.dumps({
        "metric": "request-stream images/s (end to end, host images in, host results out)",
        "unit": "images/s", "higher_is_better": True, "data": "synthetic: seeded uint8 noise images",
        "config": {"workload": sw["name"], "requests": len(reqs), "images": n_img,
                   "batch_sizes": list(sw["sizes"]), "image_hw": [sw["lo"], sw["hi"]], "max_batch": Bm},
        "one_client": round(n_img / seq_s, 1),
        "one_client_request_ms": pct(lat),
        "clients_4_shared_handles": round(n_img / shared_s, 1),
        "clients_4_shared_handles_request_ms": pct(lat_sh),
        "clients_4_batcher": {f"workers_{k}": v for k, v in res.items()},
        "batcher_max_wait_us": args.max_wait_us,
    }))


def main():
    args = parse()
    if args.serve:
        serve_bench(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported "
              "(every box has one GPU; the multi-GPU design is documented, not built)", file=sys.stderr)
        sys.exit(2)
    import torch
    import workloads as wl
    from paper_2003_01538_amd import flexserve as fsb

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": n, "launches": 5}))
        return
    w = wl.workload(args.workload)
    B = args.batch or w["batch"]
    imgs = list(wl.images_uniform(w["image_seed"], B, *w["in_hw"]))
    Bm = min(args.max_batch or B, B)
    ens = fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                       max_batch=Bm)
    if args.graphs:
        fsb.fs_graphs_enable(ens.handle, True)
    if args.combine != "mean":
        policy = {"plurality": fsb.FS_COMBINE_PLURALITY, "any": fsb.FS_COMBINE_ANY}[args.combine]
        fsb.fs_set_combine(ens.handle, policy, 0, 1)
    info = ens.info()
    N, C = info["num_models"], info["num_classes"]
    peak = PEAK_BF16_TFLOPS if w["precision"] == "bf16" else PEAK_FP32_TFLOPS

    flat, desc = wl.pack_images(imgs)
    d_pix = torch.from_numpy(flat).cuda()
    d_desc = torch.tensor([[o, h | (wd << 32), rs] for o, h, wd, rs in desc], dtype=torch.int64).cuda()
    # one set of outputs per micro-batch (model-major within each)
    chunks = [(c0, min(Bm, B - c0)) for c0 in range(0, B, Bm)]
    outs = [(torch.empty((N, nb, C), dtype=torch.float32, device="cuda"),
             torch.empty((N, nb, C), dtype=torch.float32, device="cuda"),
             torch.empty((nb, C), dtype=torch.float32, device="cuda"),
             torch.empty(nb, dtype=torch.int32, device="cuda"),
             torch.empty((N, nb), dtype=torch.int32, device="cuda")) for _, nb in chunks]
    # a stream of our own: the pass runs on it, so events recorded on it
    # bracket the whole pass (stream 0 would hand the pass to the library's
    # own stream)
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()

    def step():
        for (c0, nb), (probs, logits, mean, vote, top1) in zip(chunks, outs):
            fsb.fs_infer_device(ens.handle, d_pix.data_ptr(), d_desc.data_ptr() + c0 * d_desc.stride(0) * 8, nb,
                                probs.data_ptr(), mean.data_ptr(), vote.data_ptr(), top1.data_ptr(),
                                logits.data_ptr(), stream.cuda_stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.tuning_log:
        with open(args.tuning_log, "w") as f:
            f.write(fsb.fs_tuning_log(ens.handle))
    # everything allocated so far is long-lived: keep it out of the cyclic
    # garbage collector's full passes, which otherwise land in timed calls
    import gc
    gc.collect()
    gc.freeze()

    # plain timing (no events) and event-profiled timing of the same steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    plain_s = time.perf_counter() - t0

    roof, stats = None, {}
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda") if args.cold else None
    if not args.no_profile:
        fsb.fs_profile_enable(ens.handle, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            if flush is not None:
                with torch.cuda.stream(stream):
                    flush.fill_(i & 0xff)
            step()
        torch.cuda.synchronize()
        prof_s = time.perf_counter() - t0
        stats = fsb.fs_profile_read(ens.handle)
        recs = fsb.fs_profile_launches(ens.handle, max_out=info["launches_per_pass"] * args.steps * len(chunks))
        per_step = len(recs) // args.steps  # records of one step (a split layer is one record)
        if args.dump_launches:
            with open(args.dump_launches, "w") as f:
                json.dump(recs[-per_step:], f, indent=0)
        fsb.fs_profile_enable(ens.handle, False)
        # one conv launch = one conv layer: its implicit-GEMM dispatch plus, for
        # a layer that splits K, the dispatch that sums the partial products
        conv = [r for r in recs if r["kclass"] == "conv"]
        per_launch_ms = sum(r["ms"] for r in conv) / len(conv)
        flops_per_launch = sum(r["flops"] for r in conv) / len(conv)
        achieved = flops_per_launch / (per_launch_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": counted_traffic() if w["name"] == DEFAULT_WORKLOAD else None,
                "algorithmic_bytes_per_launch": round(sum(r["bytes"] for r in conv) / len(conv)),
                "kernel": "conv layer (implicit-GEMM dispatch + split-K reduce where used), mean over the layers of a step",
                "avg_launch_us": round(per_launch_ms * 1e3, 2)}
        # per conv layer: achieved rate against the peak and against the
        # attainable min(peak, AI x HBM bandwidth), AI = algorithmic FLOP per
        # algorithmic HBM byte (the 1x1 downsamples sit far below the ridge)
        by_layer = {}
        for r in conv:
            by_layer.setdefault((r["group"], r["layer"]), []).append(r)
        conv_layers = []
        for (gi, li), rs in sorted(by_layer.items()):
            ms_l = sum(r["ms"] for r in rs) / len(rs)
            fl, by = rs[0]["flops"], rs[0]["bytes"]
            tf = fl / (ms_l * 1e-3) / 1e12
            ai = fl / by
            att = min(peak, ai * PEAK_HBM_GBS / 1e3)
            conv_layers.append({"layer": li, "kernel": rs[0]["kernel"], "MNK": [rs[0]["M"], rs[0]["N"], rs[0]["K"]],
                                "us": round(ms_l * 1e3, 2), "tflops": round(tf, 1), "ai": round(ai, 1),
                                "attainable": round(att, 1), "frac_peak": round(tf / peak, 4),
                                "frac_attainable": round(tf / att, 4)})
        if w["precision"] == "bf16" and not args.no_vendor_gemm:
            roof["vendor_gemm"] = vendor_reference(conv_layers, by_layer, peak)
        roof["conv_layers"] = conv_layers
        print(json.dumps({"profiled_ms_per_step": prof_s / args.steps * 1e3,
                          "kernels": {k: dict(v, avg_us=v["total_ms"] / v["launches"] * 1e3,
                                              share=v["total_ms"] / args.steps / (plain_s / args.steps * 1e3))
                                      for k, v in stats.items()}}), file=sys.stderr)

    # per-step spread of the device-resident pass, events on the launch stream
    spans = []
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(args.steps):
        ev0.record(stream)
        step()
        ev1.record(stream)
        ev1.synchronize()
        spans.append(ev0.elapsed_time(ev1))
    spans = np.sort(np.asarray(spans))
    # end to end: host uint8 images in, host results out (PCIe included; never the value)
    walls, phases = [], []
    for i in range(0 if args.no_e2e else max(25, args.steps) + 2):
        t0 = time.perf_counter()
        ens.infer(imgs, want_logits=False)
        if i >= 2:
            walls.append((time.perf_counter() - t0) * 1e3)
            phases.append(fsb.fs_infer_phases(ens.handle))
    order = np.argsort(walls)
    walls = np.asarray(walls)[order]
    phases = [phases[i] for i in order]

    def pct(v, qs=(("p10", 10), ("p50", 50), ("p90", 90))):
        return {q: round(float(np.percentile(v, p)), 4) for q, p in qs}

    hbm = None
    if stats and "preprocess" in stats:
        # the library counts what the transformation writes (it never sees the
        # images' sizes on the device path); add the uint8 images it reads
        stats["preprocess"]["bytes"] += float(flat.nbytes) * args.steps
    if stats:
        # memory-bound kernel classes: algorithmic bytes over their event time
        hbm = {k: {"achieved": round(v["bytes"] / (v["total_ms"] * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS,
                   "unit": "GB/s", "frac": round(v["bytes"] / (v["total_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                   "avg_us": round(v["total_ms"] / v["launches"] * 1e3, 2)}
               for k, v in stats.items() if k in ("preprocess", "maxpool", "gap", "fc", "softmax_combine")
               and v["launches"] > 0 and v["total_ms"] > 0}

    ms = plain_s / args.steps * 1e3
    out = {
        "metric": METRIC if w["name"] == DEFAULT_WORKLOAD and B == w["batch"] else
                  f"ensemble images/sec at B={B} ({'+'.join(w['archs'])}, {w['precision']}) + MFMA util vs peak",
        "value": round(B * args.steps / plain_s, 1),
        "unit": "images/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w["precision"] == "bf16" else "f32",
        "data": "synthetic: seeded uint8 noise images, He-normal random weights",
        "config": {"workload": w["name"], "models": list(w["archs"]), "batch": B, "max_batch": Bm,
                   "input_hw": list(w["in_hw"]), "transformed_hw": list(w["out_hw"]),
                   "combine": args.combine,
                   "flops_per_image": info["flops_per_image"],
                   "launches_per_step": info["launches_per_pass"]},
        "roofline": roof,
        "hbm_kernels": hbm,
        "hbm_kernels_cold": bool(args.cold),
        "device_step_ms": pct(spans),
        "end_to_end": None if args.no_e2e else {
            "images_per_s": round(B / float(np.median(walls)) * 1e3, 1),
            "ms": pct(walls, (("p10", 10), ("p50", 50), ("p90", 90), ("p99", 99))),
            "in_library_ms": pct(np.sort([sum(p.values()) for p in phases]),
                                 (("p50", 50), ("p90", 90), ("p99", 99))),
            "phases_ms_median_call": {k: round(v, 4) for k, v in phases[len(phases) // 2].items()},
            "phases_ms_slowest_call": {k: round(v, 4) for k, v in phases[-1].items()},
            "note": "fs_infer from host images to host results, PCIe included"},
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(w, imgs, args.cpu_seconds)
    ens.close()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
