#!/usr/bin/env python3
"""Throughput of the retraining hot path on one MI355X.

Headline workload: full ResNet18 retraining (every stage trainable, BatchNorm
in train mode) at 224x224x3 in bf16 with fp32 accumulation, 6 classes, on a
4000-frame synthetic drifting window (class prototypes plus noise, contrast
and brightness moving across the window) at 100%, 10 epochs of SGD with
momentum at batch 128, held-out accuracy on 400 frames after every epoch.
One step = one ekya_retrain call over the window (40,000 trained samples);
value = trained samples per second of step time, inputs resident in HBM.

Beside it, as extra keys: layer4+fc retraining on a 2000-frame window at 30%
(5 epochs, batch 64), inference img/s at 224/160/112, the 16-candidate
micro-profiler sweep on the 4000-frame window (wall time, aggregate samples/s),
and inference beside a layer3+ retraining job (the joint window).

`roofline` covers the GEMM kernel with the largest total time in one
instrumented step (HIP events around every launch on its own stream, serial
schedule); `gemm_by_kind` and `hbm_kernels` give every convolution kind's
fraction of bf16 MFMA peak and every memory-bound kernel's fraction of HBM
peak, from algorithmic flops and bytes.  `cpu_baseline` times the CPU oracle
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "retrain samples/s (fwd+bwd) ResNet18 224px bf16, % MFMA peak; infer img/s"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

FULL = dict(n_frames=4000, n_heldout=400, px=224, k=6, frac=1.0, epochs=10, batch=128, lr=0.01,
            momentum=0.9, seed=0, drift="drift")
LAYER4 = dict(n_frames=2000, n_heldout=400, px=224, k=2, frac=0.3, epochs=5, batch=64, lr=0.01,
              momentum=0.9, seed=0, drift="shift")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_digest():
    """sha256 of the sources that define the GEMM kernels."""
    import hashlib
    h = hashlib.sha256()
    for f in ("conv.hip", "common.hpp", "kernels.hpp"):
        with open(os.path.join(ROOT, "paper_2012_10557_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes recorded in profiles/traffic.json (scaled by a plain copy's
    counts), or None if they were taken on another kernel or other sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel") != kernel or t.get("kernel_source_sha256") != kernel_source_digest():
        return None
    return int(t["fetch_bytes_per_launch"] + t["write_bytes_per_launch"])


def cpu_baseline(n=64, n_heldout=8):
    """The oracle, as it stands, on a bounded sample of the headline workload:
    one SGD step of full-depth retraining on 64 frames of the 224 px drifting
    window (8 held-out frames evaluated after it), fp64 numpy."""
    from threadpoolctl import threadpool_info

    from oracle import ekya as oracle
    from synth import WindowSpec, kaiming_resnet18_weights, make_window

    w = FULL
    win = make_window(WindowSpec(n, n_heldout, w["px"], w["px"], drift=w["drift"], seed=1))
    import torch
    bf = lambda a: torch.tensor(a).to(torch.bfloat16).float().numpy()  # same bytes as the GPU reads
    w0 = kaiming_resnet18_weights(seed=0)
    t0 = time.perf_counter()
    res = oracle.retrain(w0, w["k"], bf(win["frames"]), win["labels"], bf(win["heldout_frames"]),
                         win["heldout_labels"], 1.0, 1, w["lr"], w["momentum"], n, w["seed"])
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": round(len(res.train_indices) / dt, 3), "unit": "samples/s", "cores": int(threads),
            "nproc": os.cpu_count(), "kind": "oracle",
            "sample": f"one SGD step of full-depth retraining on {n} frames of the 224 px window "
                      f"(+{n_heldout} held-out frames evaluated), fp64 numpy with BLAS on {threads} "
                      f"threads; {dt:.1f} s"}


def dev_window(spec_kw, seed):
    import torch
    from synth import WindowSpec, make_window
    win = make_window(WindowSpec(spec_kw["n_frames"], spec_kw["n_heldout"], spec_kw["px"], spec_kw["px"],
                                 drift=spec_kw["drift"], seed=seed))
    dev = torch.device("cuda:0")
    return {"fr": torch.tensor(win["frames"]).to(torch.bfloat16).to(dev),
            "lab": torch.tensor(win["labels"]).to(dev),
            "hf": torch.tensor(win["heldout_frames"]).to(torch.bfloat16).to(dev),
            "hl": torch.tensor(win["heldout_labels"]).to(dev)}


def instrumented_step(binding, ctx, step):
    """Per-kernel HIP-event timing of one step (serial schedule)."""
    binding.ekya_set_kernel_timing(ctx, True)
    step()
    stats = binding.ekya_kernel_timing(ctx)
    binding.ekya_set_kernel_timing(ctx, False)
    gemm = sorted([s for s in stats if s["flops"] > 0], key=lambda s: -s["total_ms"])
    mem = sorted([s for s in stats if s["flops"] == 0], key=lambda s: -s["total_ms"])
    for s in gemm:
        log(f"  {s['name']:34s} launches {s['launches']:5d} total {s['total_ms']:8.3f} ms "
            f"avg {s['total_ms'] / s['launches'] * 1e3:8.2f} us  "
            f"{s['flops'] / (s['total_ms'] * 1e-3) / 1e12:7.1f} TFLOP/s")
    for s in mem:
        log(f"  {s['name']:34s} launches {s['launches']:5d} total {s['total_ms']:8.3f} ms "
            f"avg {s['total_ms'] / s['launches'] * 1e3:8.2f} us  "
            f"{s['bytes'] / (s['total_ms'] * 1e-3) / 1e9:7.1f} GB/s")
    return gemm, mem


def roofline_of(gemm, mem):
    dom = gemm[0]
    avg_ms = dom["total_ms"] / dom["launches"]
    achieved = dom["flops"] / (dom["total_ms"] * 1e-3) / 1e12
    gemm_ms = sum(s["total_ms"] for s in gemm)
    gemm_flops = sum(s["flops"] for s in gemm)
    kinds = {}
    for s in gemm:
        kind = s["name"].split("<")[0]
        k = kinds.setdefault(kind, {"ms": 0.0, "flops": 0.0})
        k["ms"] += s["total_ms"]
        k["flops"] += s["flops"]
    by_kind = {kind: {"tflops": round(v["flops"] / (v["ms"] * 1e-3) / 1e12, 1),
                      "frac": round(v["flops"] / (v["ms"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                      "ms_per_step": round(v["ms"], 3)} for kind, v in kinds.items()}
    hbm = {s["name"]: {"gbs": round(s["bytes"] / (s["total_ms"] * 1e-3) / 1e9, 1),
                       "frac": round(s["bytes"] / (s["total_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                       "launches": s["launches"], "ms_per_step": round(s["total_ms"], 3)}
           for s in mem}
    mem_ms = sum(s["total_ms"] for s in mem)
    mem_bytes = sum(s["bytes"] for s in mem)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(dom["name"]),
                "algorithmic_bytes_per_launch": round(dom["bytes"] / dom["launches"]),
                "kernel": dom["name"], "launches_per_step": dom["launches"],
                "avg_launch_us": round(avg_ms * 1e3, 2),
                "flops_per_launch": dom["flops"] / dom["launches"],
                "all_gemm_tflops": round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 2),
                "all_gemm_frac": round(gemm_flops / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "gemm_ms_per_step": round(gemm_ms, 3),
                "memory_bound_ms_per_step": round(mem_ms, 3),
                "memory_bound_gbs": round(mem_bytes / (mem_ms * 1e-3) / 1e9, 1) if mem_ms else None}
    return roofline, by_kind, hbm


COPY_BYTES = 1 << 28  # calibration copy of the traffic probe


def traffic_probe(binding, torch):
    """The all-taps weight gradients of one full-depth batch -- the 3x3
    stride-1 convolutions of the step (4 at 56 px x 64 channels, 3 at 28 x 128,
    3 at 14 x 256, 3 at 7 x 512; batch 128, bf16) -- through the C-ABI op, then
    one device-to-device copy of COPY_BYTES whose counts calibrate the
    FETCH_SIZE / WRITE_SIZE counters.  Meant to run under rocprofv3 --pmc."""
    dev = torch.device("cuda:0")
    gen = torch.Generator().manual_seed(0)
    launches = 0
    for hw, c, count in ((56, 64, 4), (28, 128, 3), (14, 256, 3), (7, 512, 3)):
        x = (torch.rand(128, hw, hw, c, generator=gen) - 0.5).to(torch.bfloat16).to(dev)
        dy = (torch.rand(128, hw, hw, c, generator=gen) - 0.5).to(torch.bfloat16).to(dev)
        for _ in range(count):
            binding.ekya_op_conv2d_wgrad(x, dy, (c, c, 3, 3), 1, 1)
            launches += 1
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"probe": "traffic", "kernel": "conv_wgrad<bf16,taps9,64>", "launches": launches,
                      "copy_bytes": COPY_BYTES}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the headline workload (no layer4, inference, sweep, joint window)")
    ap.add_argument("--timing-all-steps", action="store_true",
                    help="per-kernel timing (serial schedule) on every step, so that a profiler "
                         "run of this command measures the kernels as the roofline does")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="run only the dominant kernel's launches of one batch and a calibration "
                         "copy (for rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE passes), then exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build runs the whole path on a single "
              "MI355X (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2012_10557_amd import binding
    from synth import kaiming_resnet18_weights

    if args.traffic_probe:
        traffic_probe(binding, torch)
        return
    dev = torch.device("cuda:0")
    w = FULL
    t_gen = time.perf_counter()
    d = dev_window(w, seed=0)
    log(f"generated the {w['n_frames']}-frame window in {time.perf_counter() - t_gen:.1f} s")
    w0 = torch.tensor(kaiming_resnet18_weights(seed=0)).to(dev)
    weights = torch.empty_like(w0)
    ws = binding.ekya_retrain_workspace(6, w["k"], w["n_frames"], w["px"], w["px"], w["n_heldout"],
                                        w["frac"], w["epochs"], w["lr"], w["momentum"], w["batch"])
    ctx = binding.ekya_create(0, 6, workspace_bytes=ws)
    log(f"workspace {ws / 2**30:.2f} GiB")

    def step():
        weights.copy_(w0)
        return binding.ekya_retrain(ctx, weights, w["k"], d["fr"], d["lab"], d["hf"], d["hl"],
                                    w["frac"], w["epochs"], w["lr"], w["momentum"], w["batch"],
                                    w["seed"])

    if args.timing_all_steps:
        binding.ekya_set_kernel_timing(ctx, True)
    for i in range(args.warmup):
        out = step()
        log(f"warmup {i}: epochs {[round(x * 1e3, 1) for x in out['epoch_seconds']]} ms, "
            f"acc {out['heldout_acc']}")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        out = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    samples = out["n_train"] * w["epochs"]
    value = samples / (ms * 1e-3)
    log(f"timed: {ms:.2f} ms/step, {value:.1f} samples/s, held-out acc {out['heldout_acc']}, "
        f"epochs {[round(x * 1e3, 2) for x in out['epoch_seconds']]} ms, "
        f"evaluations {[round(x * 1e3, 2) for x in out['eval_seconds']]} ms")
    flops_per_sample = 10.645e9  # forward + data gradient + weight gradient, all stages, 224 px
    whole_frac = samples * flops_per_sample / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS

    gemm, mem = instrumented_step(binding, ctx, step)
    roofline, by_kind, hbm = roofline_of(gemm, mem)
    binding.ekya_destroy(ctx)

    extras = {}
    if not args.no_extras:
        extras = run_extras(binding, torch, d, w0)

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample ...")
        cpu = cpu_baseline()
        log(f"cpu baseline: {cpu}")

    line = {"metric": METRIC, "value": round(value, 2), "unit": "samples/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded class-prototype frames with drift; random-init Kaiming weights)",
            "config": {"workload": "ResNet18 224px bf16, full retraining (all stages, BatchNorm in "
                                   "train mode), 4000-frame drifting window at 100%, 10 epochs, "
                                   "batch 128, 400 held-out",
                       "global_batch": w["batch"], "k_trainable": w["k"], "epochs": w["epochs"],
                       "train_samples_per_step": samples, "parallelism": "single GPU"},
            "heldout_acc_final": out["heldout_acc_final"],
            "step_mfma_frac": round(whole_frac, 4),
            "roofline": roofline, "gemm_by_kind": by_kind, "hbm_kernels": hbm,
            **extras, "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


def run_extras(binding, torch, d, w0):
    out = {}
    # layer4+fc retraining on a 2000-frame window at 30%
    c = LAYER4
    d2 = dev_window(c, seed=0)
    ctx = binding.ekya_create(0, 6)
    wts = w0.clone()

    def step2():
        wts.copy_(w0)
        return binding.ekya_retrain(ctx, wts, c["k"], d2["fr"], d2["lab"], d2["hf"], d2["hl"], c["frac"],
                                    c["epochs"], c["lr"], c["momentum"], c["batch"], c["seed"])
    step2()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        o2 = step2()
    torch.cuda.synchronize()
    ms2 = (time.perf_counter() - t0) * 1e3 / 3
    out["layer4_retrain"] = {"samples_per_s": round(o2["n_train"] * c["epochs"] / (ms2 * 1e-3), 1),
                             "ms_per_step": round(ms2, 3), "prefix_ms": round(o2["prefix_seconds"] * 1e3, 3),
                             "workload": "layer4+fc, 2000-frame window at 30%, 5 epochs, batch 64"}
    log(f"layer4+fc: {out['layer4_retrain']}")

    # the same job with a hidden classifier layer of 1024 neurons
    from synth import kaiming_resnet18_weights
    hctx = binding.ekya_create(0, 6, hidden=1024)
    wh0 = torch.tensor(kaiming_resnet18_weights(seed=0, hidden=1024), device=w0.device)
    wh = wh0.clone()

    def step_h():
        wh.copy_(wh0)
        return binding.ekya_retrain(hctx, wh, c["k"], d2["fr"], d2["lab"], d2["hf"], d2["hl"],
                                    c["frac"], c["epochs"], c["lr"], c["momentum"], c["batch"],
                                    c["seed"])
    step_h()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        oh = step_h()
    torch.cuda.synchronize()
    msh = (time.perf_counter() - t0) * 1e3 / 3
    out["layer4_retrain_hidden1024"] = {
        "samples_per_s": round(oh["n_train"] * c["epochs"] / (msh * 1e-3), 1),
        "ms_per_step": round(msh, 3),
        "workload": "as layer4_retrain, with a 1024-neuron hidden layer before the classifier"}
    log(f"layer4+fc, hidden 1024: {out['layer4_retrain_hidden1024']}")
    binding.ekya_destroy(hctx)
    del d2

    # inference img/s on 2000 frames of the window
    infer = {}
    sub = d["fr"][:2000].contiguous()
    for r in (224, 160, 112):
        lab = binding.ekya_infer(ctx, w0, sub, r)
        torch.cuda.synchronize()
        ti = time.perf_counter()
        for _ in range(3):
            binding.ekya_infer(ctx, w0, sub, r, labels_out=lab)
        torch.cuda.synchronize()
        infer[str(r)] = round(3 * sub.shape[0] / (time.perf_counter() - ti), 1)
    out["infer_img_per_s"] = infer
    log(f"infer img/s: {infer}")
    binding.ekya_destroy(ctx)

    # micro-profiler sweep: 16 candidates on the 4000-frame window
    cfgs = [{"k": k, "subsample_frac": f, "epochs": e, "lr": 0.01, "momentum": 0.9, "batch": 64,
             "seed": 100 + i}
            for i, (k, f, e) in enumerate((k, f, e) for k in (1, 2, 3, 6) for f in (0.05, 0.10)
                                          for e in (1, 2))]
    ctx = binding.ekya_create(0, 6)
    sweep = {}
    for mode in ("concurrent", "sequential"):
        binding.ekya_profile(ctx, w0, cfgs, d["fr"], d["lab"], d["hf"], d["hl"], 7, concurrent=(mode == "concurrent"))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res = binding.ekya_profile(ctx, w0, cfgs, d["fr"], d["lab"], d["hf"], d["hl"], 7,
                                   concurrent=(mode == "concurrent"))
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        trained = sum(r["n_train"] * c["epochs"] for r, c in zip(res, cfgs))
        sweep[mode] = {"wall_s": round(wall, 4), "samples_per_s": round(trained / wall, 1)}
    out["profile_sweep"] = dict(sweep, candidates=len(cfgs),
                                workload="16 candidates: depth {fc, layer4+, layer3+, all} x "
                                         "{5%, 10%} x {1, 2} epochs, batch 64, 4000-frame window")
    log(f"sweep: {out['profile_sweep']}")

    # joint window: inference beside a layer3+ retraining job
    ictx = binding.ekya_create(0, 6)
    inf = d["fr"][:3600].contiguous()
    s_inf, s_tr = torch.cuda.Stream(), torch.cuda.Stream()
    r3, l3 = d["fr"][:3600].contiguous(), d["lab"][:3600].contiguous()
    lab = binding.ekya_infer(ictx, w0, inf, 224, stream=s_inf)
    s_inf.synchronize()
    t0 = time.perf_counter()
    binding.ekya_infer(ictx, w0, inf, 224, labels_out=lab, stream=s_inf)
    s_inf.synchronize()
    alone = inf.shape[0] / (time.perf_counter() - t0)
    wt = w0.clone()
    torch.cuda.synchronize()
    box = {}

    def trainer():
        t = time.perf_counter()
        box["o"] = binding.ekya_retrain(ctx, wt, 3, r3, l3, d["hf"], d["hl"], 0.1, 5, 0.01, 0.9, 128, 0,
                                        stream=s_tr)
        box["t"] = time.perf_counter() - t
    th = threading.Thread(target=trainer)
    th.start()
    t0 = time.perf_counter()
    binding.ekya_infer(ictx, w0, inf, 224, labels_out=lab, stream=s_inf)
    s_inf.synchronize()
    together = inf.shape[0] / (time.perf_counter() - t0)
    th.join()
    out["joint_window"] = {"infer_224_alone_img_per_s": round(alone, 1),
                           "infer_224_beside_retrain_img_per_s": round(together, 1),
                           "retrain_wall_s": round(box["t"], 4),
                           "workload": "3600 frames at 224 px beside layer3+ retraining "
                                       "(10% of 3600 frames, 5 epochs, batch 128)"}
    log(f"joint: {out['joint_window']}")

    # the same joint window on complementary CU ranges, the GPU split in
    # steps of 0.1 (the scheduler's quantum): inference on [0, s), the
    # retraining job's streams on [s, 1); each alone on its range, then both
    def retrain_on(stream):
        t = time.perf_counter()
        binding.ekya_retrain(ctx, w0.clone(), 3, r3, l3, d["hf"], d["hl"], 0.1, 5, 0.01, 0.9, 128,
                             0, stream=stream)
        return time.perf_counter() - t

    def infer_on(stream):
        t = time.perf_counter()
        binding.ekya_infer(ictx, w0, inf, 224, labels_out=lab, stream=stream)
        stream.synchronize()
        return inf.shape[0] / (time.perf_counter() - t)

    shares = []
    for i in range(1, 10):
        s = i / 10
        si, st = binding.CuStream(0, 0.0, s), binding.CuStream(0, s, 1.0 - s)
        binding.ekya_set_cu_partition(ctx, s, 1.0 - s)
        infer_on(si)
        rate_alone = infer_on(si)
        retrain_on(st)
        wall_alone = retrain_on(st)
        box = {}
        th = threading.Thread(target=lambda: box.update(t=retrain_on(st)))
        th.start()
        rate_joint = infer_on(si)
        th.join()
        shares.append({"infer_share": s, "infer_cus": si.cu_count(), "retrain_cus": st.cu_count(),
                       "infer_img_per_s_alone": round(rate_alone, 1),
                       "infer_img_per_s_joint": round(rate_joint, 1),
                       "retrain_wall_s_alone": round(wall_alone, 4),
                       "retrain_wall_s_joint": round(box["t"], 4)})
        si.destroy()
        st.destroy()
        log(f"cu share: {shares[-1]}")
    binding.ekya_set_cu_partition(ctx, 0.0, 1.0)
    out["cu_shares"] = {"workload": out["joint_window"]["workload"], "splits": shares}

    # hot reload: one load of the model (prepared inference weights) and the
    # cost of publishing a checkpoint after every epoch of the retraining job
    model = binding.ekya_model_create(0, 6, binding.EKYA_BF16)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s_tr):
        binding.ekya_model_load(model, w0, stream=s_tr)
        e0.record(s_tr)
        for _ in range(10):
            binding.ekya_model_load(model, w0, stream=s_tr)
        e1.record(s_tr)
    s_tr.synchronize()
    load_ms = e0.elapsed_time(e1) / 10
    retrain_on(s_tr)
    plain = min(retrain_on(s_tr) for _ in range(3))
    binding.ekya_set_checkpoint(ctx, model, 1)
    published = min(retrain_on(s_tr) for _ in range(3))
    binding.ekya_set_checkpoint(ctx, None, 0)
    out["hot_reload"] = {"model_load_ms": round(load_ms, 4),
                         "retrain_wall_s": round(plain, 4),
                         "retrain_wall_s_checkpoint_every_epoch": round(published, 4),
                         "workload": "layer3+ retraining (10% of 3600 frames, 5 epochs, batch 128); "
                                     "bf16 ResNet18 weights"}
    log(f"hot reload: {out['hot_reload']}")
    binding.ekya_model_destroy(model)

    # ten streams, each with its own model, 360 frames each at 224 px in one
    # call, against the same 3600 frames through one model
    models = [binding.ekya_model_create(0, 6, binding.EKYA_BF16) for _ in range(10)]
    for m in models:
        binding.ekya_model_load(m, w0)
    counts = [360] * 10
    lab10, _ = binding.ekya_infer_models(ictx, models, inf, counts, 224)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        binding.ekya_infer_models(ictx, models, inf, counts, 224, labels_out=lab10)
    torch.cuda.synchronize()
    rate10 = 3 * inf.shape[0] / (time.perf_counter() - t0)
    out["infer_per_stream_models"] = {"img_per_s": round(rate10, 1),
                                      "single_model_img_per_s": out["joint_window"]["infer_224_alone_img_per_s"],
                                      "workload": "10 streams x 360 frames at 224 px, one model per stream"}
    log(f"per-stream models: {out['infer_per_stream_models']}")
    for m in models:
        binding.ekya_model_destroy(m)
    binding.ekya_destroy(ictx)
    binding.ekya_destroy(ctx)
    return out


if __name__ == "__main__":
    main()
