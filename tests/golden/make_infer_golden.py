#!/usr/bin/env python3
"""Writes the stored oracle logits of batched inference (sections 1 and 3.1,
inference configurations: frames downsized to the configured resolution and
classified): ResNet18 with fixed-seed weights on 520 drifting 224 px frames,
resized bilinearly to 224, 160 and 112.  The bf16 cases read the frames
rounded to bfloat16 (the bytes the bf16 path reads); the fp32 case at 224 the
float32 frames.  Calls only the CPU oracle.

A randomly initialised network sends every frame to one class (its pooled
features share a large mean, and the classifier row with the largest
projection on it wins everywhere), which would make label parity trivial.
Each case's stored classifier is therefore the initial one with that mean
direction removed from every row (measured on the oracle's own pooled
features of that case) and scaled so the logits spread over a few units; the
test uses it in place of the initial classifier.

Per frame the file also stores the logits' scale max_j sum_i |W_ji f_i| (f
the oracle's pooled features): a relative error e in the features moves a
logit by at most e times that, which bounds where two logits may swap.

    python tests/golden/make_infer_golden.py   # writes infer_224.json
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402
import torch  # noqa: E402

from oracle import nn  # noqa: E402
from oracle.resnet18 import ResNet18  # noqa: E402
from synth import WindowSpec, kaiming_resnet18_weights, make_frames  # noqa: E402

CASE = dict(n_frames=520, px=224, drift="drift", window_seed=31, weights_seed=2,
            cases=[["bf16", 224], ["bf16", 160], ["bf16", 112], ["f32", 224]])
CHUNK = 40  # frames per oracle call (eval mode: every frame is independent)


def frames_for(prec):
    c = CASE
    spec = WindowSpec(c["n_frames"], 0, c["px"], c["px"], drift=c["drift"], seed=c["window_seed"])
    fr, _ = make_frames(spec, c["n_frames"], 1, 2)
    if prec == "bf16":
        return torch.tensor(fr).to(torch.bfloat16).double().numpy()
    return fr.astype(np.float64)


def pooled(P, net, fr, res):
    """Eval-mode pooled features of frames resized to res (the oracle's forward, stages 0-4)."""
    out = []
    for i in range(0, len(fr), CHUNK):
        x = fr[i:i + CHUNK]
        if x.shape[1] != res:
            x = nn.resize_bilinear(x, res, res)
        out.append(net.forward(P, x, 0, 4, train=False, tape={}))
    return np.concatenate(out)


def main():
    c = CASE
    w0 = kaiming_resnet18_weights(seed=c["weights_seed"])
    net = ResNet18(6)
    P = net.unpack(w0)
    out = {"case": c, "logits": {}}
    t0 = time.time()
    feats = {}
    for prec, res in c["cases"]:
        feats[(prec, res)] = pooled(P, net, frames_for(prec), res)
        print(prec, res, "pooled", round(time.time() - t0, 1), flush=True)
    out["fc"] = {}
    out["scale"] = {}
    for (prec, res), F in feats.items():
        mu = F.mean(axis=0)
        W = P["fc.weight"] - np.outer(P["fc.weight"] @ mu, mu) / (mu @ mu)
        W *= 3.0 / np.std(F @ W.T)
        W = W.astype(np.float32).astype(np.float64)   # stored as float32 values
        b = np.zeros(6)
        out["fc"][f"{prec}_{res}"] = {"weight": [[float(v) for v in row] for row in W.astype(np.float32)],
                                      "bias": [0.0] * 6}
        lg = nn.linear(F, W, b)
        out["logits"][f"{prec}_{res}"] = [[float("%.12g" % v) for v in row] for row in lg]
        out["scale"][f"{prec}_{res}"] = [float("%.12g" % v)
                                         for v in (np.abs(F) @ np.abs(W).T).max(axis=1)]
        print(prec, res, np.bincount(np.argmax(lg, 1), minlength=6), flush=True)
    out["oracle_seconds"] = round(time.time() - t0, 1)
    with open(os.path.join(HERE, "infer_224.json"), "w") as f:
        json.dump(out, f)


if __name__ == "__main__":
    main()
