#!/usr/bin/env python3
"""Writes the stored oracle results of the 224 px bf16 retraining windows
(ResNet18, layer4 and fc trainable, 2000 frames at 30%, 5 epochs, batch 64,
400 held-out frames): the window with a per-window brightness/contrast shift
and pixel noise 0.3 (retrain_224_k2.json), and a harder one with noise 3.0
and a drift across the window, whose accuracy rises over the epochs without
saturating (retrain_224_k2_hard.json).  Calls only the CPU oracle; frames are
rounded to bfloat16 first (the bytes the bf16 path reads).

    python tests/golden/make_retrain_golden.py [easy|hard]
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

CASES = {
    "easy": ("retrain_224_k2.json",
             dict(n_frames=2000, n_heldout=400, px=224, drift="shift", window_seed=0, weights_seed=0,
                  k=2, frac=0.3, epochs=5, lr=0.01, momentum=0.9, batch=64, seed=0)),
    "hard": ("retrain_224_k2_hard.json",
             dict(n_frames=2000, n_heldout=400, px=224, drift="drift", window_seed=0, weights_seed=0,
                  k=2, frac=0.3, epochs=5, lr=0.01, momentum=0.9, batch=64, seed=0, noise=3.0)),
}


def bf16(a):
    return torch.tensor(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def main(which="easy"):
    fname, c = CASES[which]
    win = make_window(WindowSpec(c["n_frames"], c["n_heldout"], c["px"], c["px"], drift=c["drift"],
                                 seed=c["window_seed"], noise_std=c.get("noise", 0.3)))
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
    with open(os.path.join(HERE, fname), "w") as f:
        json.dump(out, f, indent=1)
    print(out["heldout_acc"], out["epoch_loss"], out["oracle_seconds"])


if __name__ == "__main__":
    main(sys.argv[1] if len(sys.argv) > 1 else "easy")
