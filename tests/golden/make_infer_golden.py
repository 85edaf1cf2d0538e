#!/usr/bin/env python3
"""Writes the stored oracle logits of batched inference (sections 1 and 3.1,
inference configurations: frames downsized to the configured resolution and
classified): ResNet18 with fixed-seed weights on 520 drifting 224 px frames,
resized bilinearly to 224, 160 and 112.  The bf16 cases read the frames
rounded to bfloat16 (the bytes the bf16 path reads); the fp32 case at 224 the
float32 frames.  Calls only the CPU oracle.

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

from oracle import ekya  # noqa: E402
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


def main():
    c = CASE
    w0 = kaiming_resnet18_weights(seed=c["weights_seed"])
    out = {"case": c, "logits": {}}
    t0 = time.time()
    for prec, res in c["cases"]:
        fr = frames_for(prec)
        parts = [ekya.infer_logits(w0, fr[i:i + CHUNK], res) for i in range(0, len(fr), CHUNK)]
        lg = np.concatenate(parts)
        out["logits"][f"{prec}_{res}"] = [[float("%.12g" % v) for v in row] for row in lg]
        print(prec, res, round(time.time() - t0, 1), np.bincount(np.argmax(lg, 1), minlength=6),
              flush=True)
    out["oracle_seconds"] = round(time.time() - t0, 1)
    with open(os.path.join(HERE, "infer_224.json"), "w") as f:
        json.dump(out, f)


if __name__ == "__main__":
    main()
