"""Batched inference (sections 1 and 3.1, inference configurations) through
ekya_infer at the workload's resolutions against stored oracle logits: 520
drifting 224 px frames (two equal 260-frame chunks, so the chunk split runs),
resized to 224 (the stem reads the frames directly), 160 and 112 (resize
kernel, then the padded-input stem).  bf16: labels equal except where the
oracle's top-2 logit margin is below 2e-2 of its largest logit; fp32 at 224:
equal except below 1e-5.  The stored logits and classifier come from
tests/golden/make_infer_golden.py (oracle only)."""
import json
import os

import numpy as np
import pytest

from synth import WindowSpec, kaiming_resnet18_weights, make_frames
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "infer_224.json")
MARGIN = {"bf16": 2e-2, "f32": 1e-5}


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.fixture(scope="module")
def ctx():
    from paper_2012_10557_amd import binding
    c = binding.ekya_create(0, 6)
    yield c
    binding.ekya_destroy(c)


def _weights(g):
    w = kaiming_resnet18_weights(seed=g["case"]["weights_seed"]).copy()
    fw = np.asarray(g["fc_weight"], dtype=np.float32).reshape(-1)
    fb = np.asarray(g["fc_bias"], dtype=np.float32)
    w[len(w) - fw.size - fb.size:len(w) - fb.size] = fw
    w[len(w) - fb.size:] = fb
    return w


@pytest.mark.parametrize("prec,res", [("bf16", 224), ("bf16", 160), ("bf16", 112), ("f32", 224)])
def test_infer_labels_match_oracle(ctx, golden, prec, res):
    import torch
    from paper_2012_10557_amd import binding
    c = golden["case"]
    spec = WindowSpec(c["n_frames"], 0, c["px"], c["px"], drift=c["drift"], seed=c["window_seed"])
    frames, _ = make_frames(spec, c["n_frames"], 1, 2)
    logits = np.asarray(golden["logits"][f"{prec}_{res}"])
    ref = np.argmax(logits, axis=1)
    labels = binding.ekya_infer(ctx, torch.tensor(_weights(golden), device="cuda"),
                                to_dev(frames, prec), res)
    torch.cuda.synchronize()
    got = labels.cpu().numpy()
    srt = np.sort(logits, axis=1)
    margin = (srt[:, -1] - srt[:, -2]) / np.abs(logits).max()
    tie = margin < MARGIN[prec]
    counts = np.bincount(ref, minlength=6)
    print(f"{prec} {res}px: {int((got == ref).sum())}/{len(ref)} labels equal, {int(tie.sum())} "
          f"within the tie margin, oracle class counts {counts.tolist()}")
    assert (counts > 0).sum() >= 3, "the stored case must exercise several classes"
    assert np.all((got == ref) | tie), np.nonzero((got != ref) & ~tie)
