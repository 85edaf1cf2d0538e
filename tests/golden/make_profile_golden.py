#!/usr/bin/env python3
"""Writes stored oracle results of the micro-profiler sweep at full size
(section 4.3, micro-profiling: short retraining runs on a small uniform
subset of the window, accuracy measured after every epoch): ResNet18 with
fixed-seed weights on a 4000-frame drifting 224 px window (frames rounded to
bfloat16, the bytes the bf16 path reads) with 400 held-out frames, one
candidate per trainable depth (fc, layer4+, layer3+, all) at 5% of the window
for one epoch, batch 64.  Calls only the CPU oracle.

Per held-out frame the file also stores, for the oracle's final weights, the
top-2 margin of the logits and their scale max_j sum_i |W_ji f_i| (f the
pooled features, W the classifier): a relative error tol in the features
moves each logit by at most tol times that scale, so labels of frames whose
margin is below twice it may differ between two runs that agree to tol.

    python tests/golden/make_profile_golden.py   # writes profile_224.json
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
from oracle.resnet18 import ResNet18  # noqa: E402
from synth import WindowSpec, kaiming_resnet18_weights, make_window  # noqa: E402

CASE = dict(n_frames=4000, n_heldout=400, px=224, drift="drift", window_seed=0, weights_seed=0,
            subsample_seed=7, batch=64, lr=0.01, momentum=0.9,
            cfgs=[dict(k=k, frac=0.05, epochs=1, seed=100 + 4 * i) for i, k in enumerate((1, 2, 3, 6))])


def bf16(a):
    return torch.tensor(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def heldout_margins(weights, hf, labels, chunk=40):
    """Top-2 logit margin and logit scale of every held-out frame (eval mode)."""
    net = ResNet18(6)
    P = net.unpack(weights)
    f = np.concatenate([net.forward(P, hf[i:i + chunk], 0, 4, train=False, tape={})
                        for i in range(0, len(hf), chunk)])
    W, b = P["fc.weight"], P["fc.bias"]
    lg = f @ W.T + b
    srt = np.sort(lg, axis=1)
    scale = (np.abs(f) @ np.abs(W).T).max(axis=1)
    return srt[:, -1] - srt[:, -2], scale, int((np.argmax(lg, axis=1) == np.asarray(labels)).sum())


def main():
    c = CASE
    win = make_window(WindowSpec(c["n_frames"], c["n_heldout"], c["px"], c["px"], drift=c["drift"],
                                 seed=c["window_seed"]))
    w0 = kaiming_resnet18_weights(seed=c["weights_seed"])
    fr, hf = bf16(win["frames"]), bf16(win["heldout_frames"])
    out = {"case": c, "results": []}
    for cfg in c["cfgs"]:
        t0 = time.time()
        r = ekya.profile(w0, [ekya.ProfileConfig(cfg["k"], cfg["frac"], cfg["epochs"], c["lr"],
                                                 c["momentum"], c["batch"], cfg["seed"])],
                         fr, win["labels"], hf, win["heldout_labels"],
                         subsample_seed=c["subsample_seed"])[0]
        spe = -(-len(r.train_indices) // c["batch"])
        margin, scale, n_correct = heldout_margins(r.weights, hf, win["heldout_labels"])
        assert n_correct == r.n_correct[-1]
        out["results"].append({"k": cfg["k"], "n_train": len(r.train_indices),
                               "heldout_acc": r.heldout_acc, "n_correct": r.n_correct,
                               "epoch_loss": [float(np.mean(r.losses[e * spe:(e + 1) * spe]))
                                              for e in range(cfg["epochs"])],
                               "step_loss": [float(x) for x in r.losses],
                               "heldout_margin": [float("%.9g" % v) for v in margin],
                               "heldout_scale": [float("%.9g" % v) for v in scale],
                               "oracle_seconds": round(time.time() - t0, 1)})
        print(out["results"][-1]["k"], out["results"][-1]["heldout_acc"],
              out["results"][-1]["epoch_loss"], out["results"][-1]["oracle_seconds"], flush=True)
    with open(os.path.join(HERE, "profile_224.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
