#!/usr/bin/env python3
"""Throughput of the retraining hot path on one MI355X.

Workload: ResNet18 at 224x224x3, bf16 with fp32 accumulation, 6 classes;
layer4 and fc trainable (k = 2); a 2000-frame synthetic window (class
prototypes plus noise with a per-window brightness/contrast shift) subsampled
to 30% (600 frames), 5 epochs at batch 64, held-out accuracy on 400 frames
after every epoch.  One step = one ekya_retrain call over the window: subset
draw, frozen-prefix cache build (stem..layer3 on 1000 frames), 5 epochs of
train-mode forward/backward/SGD, and the per-epoch held-out evaluation.
value = trained samples (600 x 5) per second of step time, inputs resident
in HBM.  Inference img/s of ekya_infer on the same frames at 224/160/112 is
reported beside it.

`roofline` covers the GEMM kernel with the largest total time inside one
step, timed with HIP events on the library's stream; `cpu_baseline` times
the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "retrain samples/s (fwd+bwd) ResNet18 224px bf16, % MFMA peak; infer img/s"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

WORKLOAD = dict(n_frames=2000, n_heldout=400, px=224, k=2, frac=0.3, epochs=5, batch=64,
                lr=0.01, momentum=0.9, seed=0, drift="shift")


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


def cpu_baseline(sample_frames=300, sample_heldout=60):
    """The oracle, as it stands, on a bounded sample of the same workload:
    a 300-frame window at 30% (90 training frames), 60 held-out frames,
    k = 2, 5 epochs, batch 64, 224 px (about 10-30 s on a many-core host)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import ekya as oracle
    from synth import WindowSpec, kaiming_resnet18_weights, make_window

    w = WORKLOAD
    win = make_window(WindowSpec(sample_frames, sample_heldout, w["px"], w["px"], drift=w["drift"],
                                 seed=1))
    import torch
    bf = lambda a: torch.tensor(a).to(torch.bfloat16).float().numpy()  # same bytes as the GPU reads
    w0 = kaiming_resnet18_weights(seed=0)
    t0 = time.perf_counter()
    res = oracle.retrain(w0, w["k"], bf(win["frames"]), win["labels"], bf(win["heldout_frames"]),
                         win["heldout_labels"], w["frac"], w["epochs"], w["lr"], w["momentum"],
                         w["batch"], w["seed"])
    dt = time.perf_counter() - t0
    samples = len(res.train_indices) * w["epochs"]
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": samples / dt, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{sample_frames}-frame 224px window at 30% ({len(res.train_indices)} training "
                      f"frames), {sample_heldout} held-out, k=2, 5 epochs, batch 64, fp64 numpy; "
                      f"{dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--infer-frames", type=int, default=2000)
    ap.add_argument("--no-infer", action="store_true", help="skip the inference img/s measurement")
    ap.add_argument("--timing-all-steps", action="store_true",
                    help="per-kernel timing (serial schedule) on every step, so that a profiler "
                         "run of this command measures the kernels as the roofline does")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build runs the whole path on a single "
              "MI355X (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2012_10557_amd import binding
    from synth import WindowSpec, kaiming_resnet18_weights, make_window

    w = WORKLOAD
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    win = make_window(WindowSpec(w["n_frames"], w["n_heldout"], w["px"], w["px"], drift=w["drift"],
                                 seed=0))
    log(f"generated window in {time.perf_counter() - t_gen:.1f} s")
    frames = torch.tensor(win["frames"]).to(torch.bfloat16).to(dev)
    labels = torch.tensor(win["labels"]).to(dev)
    hframes = torch.tensor(win["heldout_frames"]).to(torch.bfloat16).to(dev)
    hlabels = torch.tensor(win["heldout_labels"]).to(dev)
    w0 = torch.tensor(kaiming_resnet18_weights(seed=0)).to(dev)
    weights = torch.empty_like(w0)
    ctx = binding.ekya_create(0, 6)

    def step():
        weights.copy_(w0)
        return binding.ekya_retrain(ctx, weights, w["k"], frames, labels, hframes, hlabels, w["frac"],
                                    w["epochs"], w["lr"], w["momentum"], w["batch"], w["seed"])

    if args.timing_all_steps:
        binding.ekya_set_kernel_timing(ctx, True)
    for i in range(args.warmup):
        out = step()
        log(f"warmup {i}: {out['epoch_seconds']} acc {out['heldout_acc']}")
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
        f"prefix {out['prefix_seconds'] * 1e3:.2f} ms, epochs {[round(x * 1e3, 2) for x in out['epoch_seconds']]} ms")

    # one instrumented step: per-kernel event timing on the library's stream
    # (the weight gradients then run on the job's stream, each kernel alone)
    binding.ekya_set_kernel_timing(ctx, True)
    step()
    stats = binding.ekya_kernel_timing(ctx)
    binding.ekya_set_kernel_timing(ctx, False)
    stats.sort(key=lambda s: -s["total_ms"])
    for s in stats:
        log(f"  {s['name']:28s} launches {s['launches']:5d} total {s['total_ms']:8.3f} ms "
            f"avg {s['total_ms'] / s['launches'] * 1e3:8.2f} us  "
            f"{s['flops'] / (s['total_ms'] * 1e-3) / 1e12:7.1f} TFLOP/s")
    dom = stats[0]
    avg_ms = dom["total_ms"] / dom["launches"]
    achieved = dom["flops"] / (dom["total_ms"] * 1e-3) / 1e12
    gemm_ms = sum(s["total_ms"] for s in stats)
    gemm_flops = sum(s["flops"] for s in stats)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(dom["name"]),
                "algorithmic_bytes_per_launch": round(dom["bytes"] / dom["launches"]),
                "kernel": dom["name"], "launches_per_step": dom["launches"],
                "avg_launch_us": round(avg_ms * 1e3, 2),
                "flops_per_launch": dom["flops"] / dom["launches"],
                "all_gemm_tflops": round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 2),
                "gemm_ms_per_step": round(gemm_ms, 3)}

    # inference img/s on the same frames
    infer = {}
    nf = min(args.infer_frames, frames.shape[0])
    sub = frames[:nf].contiguous()
    for r in (() if args.no_infer else (224, 160, 112)):
        lab = binding.ekya_infer(ctx, w0, sub, r)
        torch.cuda.synchronize()
        ti = time.perf_counter()
        for _ in range(3):
            binding.ekya_infer(ctx, w0, sub, r, labels_out=lab)
        torch.cuda.synchronize()
        infer[str(r)] = round(3 * nf / (time.perf_counter() - ti), 1)
    log(f"infer img/s: {infer}")
    binding.ekya_destroy(ctx)

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample ...")
        cpu = cpu_baseline()
        log(f"cpu baseline: {cpu}")

    line = {"metric": METRIC, "value": round(value, 2), "unit": "samples/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded class-prototype frames; random-init Kaiming weights)",
            "config": {"workload": "ResNet18 224px bf16, layer4+fc retraining (k=2), 2000-frame "
                                   "window at 30% subsample, 5 epochs, batch 64, 400 held-out",
                       "global_batch": w["batch"], "k_trainable": w["k"], "epochs": w["epochs"],
                       "train_samples_per_step": samples, "parallelism": "single GPU"},
            "heldout_acc_final": out["heldout_acc_final"],
            "infer_img_per_s": infer,
            "roofline": roofline, "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
