#!/usr/bin/env python3
"""Writes the stored oracle run of a short full-depth retraining job shaped
like the full-depth workload (section 3.1, retraining configurations: every
stage trainable, BatchNorm in train mode): ResNet18 at 224 px, 256 drifting
frames at 100%, batch 128 (two SGD steps per epoch), 2 epochs, 400 held-out
frames.  Frames are rounded to bfloat16 first (the bytes the bf16 path reads).
Calls only the CPU oracle.

    python tests/golden/make_c3_golden.py   # writes retrain_224_k6.json
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402
import torch  # noqa: E402

from oracle import ekya  # noqa: E402
from synth import WindowSpec, kaiming_resnet18_weights, make_window  # noqa: E402

CASE = dict(n_frames=256, n_heldout=400, px=224, drift="drift", window_seed=5, weights_seed=0,
            k=6, frac=1.0, epochs=2, lr=0.01, momentum=0.9, batch=128, seed=3)


def bf16(a):
    return torch.tensor(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def main():
    c = CASE
    win = make_window(WindowSpec(c["n_frames"], c["n_heldout"], c["px"], c["px"], drift=c["drift"],
                                 seed=c["window_seed"]))
    w0 = kaiming_resnet18_weights(seed=c["weights_seed"])
    t0 = time.time()
    res = ekya.retrain(w0, c["k"], bf16(win["frames"]), win["labels"], bf16(win["heldout_frames"]),
                       win["heldout_labels"], c["frac"], c["epochs"], c["lr"], c["momentum"],
                       c["batch"], c["seed"])
    spe = -(-len(res.train_indices) // c["batch"])
    out = {"case": c, "n_train": len(res.train_indices), "heldout_acc": res.heldout_acc,
           "n_correct": res.n_correct,
           "epoch_loss": [float(np.mean(res.losses[e * spe:(e + 1) * spe])) for e in range(c["epochs"])],
           "step_loss": [float(x) for x in res.losses],
           "oracle_seconds": round(time.time() - t0, 1)}
    with open(os.path.join(HERE, "retrain_224_k6.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(out["heldout_acc"], out["epoch_loss"], out["oracle_seconds"])


if __name__ == "__main__":
    main()
