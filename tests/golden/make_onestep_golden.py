#!/usr/bin/env python3
"""Writes stored oracle results of one SGD step of bf16-shaped retraining at
224 px at depth (section 3.1, retraining configurations: the last k stages
trainable with BatchNorm in train mode): ResNet18 with fixed-seed weights, one
batch of n drifting frames (rounded to bfloat16, the bytes the bf16 path
reads), k = 3 (layer3 and above) and k = 6 (every stage), n = 32 and n = 128
(the full-depth workload's batch).  Calls only the CPU oracle.

Stored per case: the step loss; every running statistic and the classifier
of the trainable stages after the step (complete); for every other
trainable tensor the update (w1 - w0) at 512 fixed positions (every position
for smaller tensors) together with the largest and the root-mean-square
update over the whole tensor.

    python tests/golden/make_onestep_golden.py   # writes onestep_224.json.gz
"""
import gzip
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402
import torch  # noqa: E402

from oracle import ekya  # noqa: E402
from oracle.resnet18 import STAGES, ResNet18  # noqa: E402
from synth import WindowSpec, kaiming_resnet18_weights, make_window  # noqa: E402

CASES = [dict(k=3, n=32), dict(k=3, n=128), dict(k=6, n=32), dict(k=6, n=128)]
COMMON = dict(px=224, drift="drift", window_seed=4, weights_seed=0, lr=0.01, momentum=0.9, seed=0,
              n_heldout=8, samples=512)


def bf16(a):
    return torch.tensor(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def sample_positions(name, size, count):
    """Fixed positions of a tensor: all of them, or `count` drawn without
    replacement from a generator seeded by the tensor's name."""
    if size <= count:
        return np.arange(size)
    seed = int.from_bytes(name.encode(), "little") % (2 ** 32)
    return np.sort(np.random.default_rng(seed).choice(size, count, replace=False))


def main():
    c0 = COMMON
    net = ResNet18(6)
    w0 = kaiming_resnet18_weights(seed=c0["weights_seed"])
    W0 = net.unpack(w0.astype(np.float64))
    out = {"common": c0, "cases": []}
    for case in CASES:
        k, n = case["k"], case["n"]
        t0 = time.time()
        win = make_window(WindowSpec(n, c0["n_heldout"], c0["px"], c0["px"], drift=c0["drift"],
                                     seed=c0["window_seed"]))
        res = ekya.retrain(w0, k, bf16(win["frames"]), win["labels"], bf16(win["heldout_frames"]),
                           win["heldout_labels"], 1.0, 1, c0["lr"], c0["momentum"], n, c0["seed"])
        W1 = net.unpack(res.weights)
        lo = len(STAGES) - k
        entry = {"k": k, "n": n, "loss": float(res.losses[0]), "full": {}, "sampled": {}}
        for name, _ in net.spec:
            if net.stage_of[name] < lo:
                continue
            if name.startswith("fc.") or net.is_running_stat(name):
                entry["full"][name] = [float(v) for v in W1[name].reshape(-1)]
                continue
            d = (W1[name] - W0[name]).reshape(-1)
            pos = sample_positions(name, d.size, c0["samples"])
            entry["sampled"][name] = {"pos": [int(p) for p in pos],
                                      "w1": [float(v) for v in W1[name].reshape(-1)[pos]],
                                      "max_abs_update": float(np.abs(d).max()),
                                      "rms_update": float(np.sqrt(np.mean(d * d)))}
        entry["oracle_seconds"] = round(time.time() - t0, 1)
        out["cases"].append(entry)
        print(k, n, entry["loss"], entry["oracle_seconds"], flush=True)
    with gzip.open(os.path.join(HERE, "onestep_224.json.gz"), "wt") as f:
        json.dump(out, f)


if __name__ == "__main__":
    main()
