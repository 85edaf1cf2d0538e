"""Decisions that rounding can flip on the retraining path.

The backward pass of a ReLU routes the gradient by the sign of its input, and
a max-pool backward routes it to the window's maximum: both are
discontinuous.  Where an input lies within rounding error of zero (or two
window entries within rounding error of each other), an fp32 implementation
and the fp64 oracle may legitimately take different branches, and that one
element then moves the gradient of a whole output channel by a large
fraction.  The strict fp32 parity tests therefore require (and assert) that
the oracle's run has no such near-decision anywhere in the trainable stages;
this module measures it from the oracle's own forward tape (test
infrastructure, no library code)."""
import numpy as np

from oracle import ekya as oracle_ekya
from oracle import nn
from oracle.resnet18 import STAGES, ResNet18


def _affine(P, prefix, saved):
    xhat = saved[0]
    return P[prefix + ".weight"] * xhat + P[prefix + ".bias"]


def decision_margins(weights, k, batch_frames, n_classes=6):
    """Smallest distance to a branch point, in units of each tensor's RMS,
    over every ReLU input and every max-pool top-2 gap in stages
    lowest..4 of one train-mode forward of `batch_frames` (the first step of
    a job, from the initial weights).  Returns (min_margin, list of
    (name, margin))."""
    net = ResNet18(n_classes)
    P = net.unpack(np.asarray(weights, dtype=np.float64))
    lowest = len(STAGES) - k
    x = oracle_ekya.prefix_forward(net, P, batch_frames, lowest)
    tape: dict = {}
    net.forward(P, x, lowest, 5, train=True, tape=tape)
    out = []

    def rel(v):
        rms = float(np.sqrt(np.mean(v * v)))
        return float(np.min(np.abs(v))) / rms if rms > 0 else np.inf

    if lowest == 0:
        pre = _affine(P, "bn1", tape["bn1"])
        out.append(("bn1.relu", rel(pre)))
        a = np.maximum(pre, 0.0)
        # top-2 gap of every 3x3/2 window (padding -inf) whose maximum is > 0
        xp = np.pad(a, ((0, 0), (1, 1), (1, 1), (0, 0)), constant_values=-np.inf)
        Pq = nn.out_size(a.shape[1], 3, 2, 1)
        Qq = nn.out_size(a.shape[2], 3, 2, 1)
        vals = np.stack([xp[:, r:r + 2 * Pq:2, s:s + 2 * Qq:2, :] for r in range(3) for s in range(3)])
        srt = np.sort(vals, axis=0)
        top, second = srt[-1], srt[-2]
        gap = np.where(top > 0, top - second, np.inf)
        rms = float(np.sqrt(np.mean(a * a)))
        out.append(("maxpool.tie", float(np.min(gap)) / rms if rms > 0 else np.inf))
    for stage in range(max(lowest, 1), 5):
        for p, _, has_ds in net._block_cfg[stage - 1]:
            xin = tape[p][0]
            out.append((p + ".relu1", rel(_affine(P, p + ".bn1", tape[p + ".bn1"]))))
            sc = _affine(P, p + ".downsample.1", tape[p + ".downsample.1"]) if has_ds else xin
            out.append((p + ".relu2", rel(_affine(P, p + ".bn2", tape[p + ".bn2"]) + sc)))
    return (min(m for _, m in out) if out else np.inf), out
