"""Retraining, micro-profiling and inference as the paper defines them.

Retraining (sections 2.2 and 3.1): continue training the edge classifier on
the current window's labelled frames.  The retraining configuration fixes the
number of trainable stages k (the rest is frozen), the fraction of the
window's data used, the number of epochs, the learning rate and the batch
size.  Training is plain mini-batch SGD with momentum on the mean
cross-entropy; the paper's iCaRL modifications are not described and are not
modelled.

Micro-profiling (section 4.3): each candidate configuration trains on a
uniform random subset of the window for a few epochs and reports its held-out
accuracy after every epoch; its GPU time per epoch is what the scheduler
scales.  Accuracy-curve extrapolation is a separate later step.

Inference (sections 1 and 3.1, inference configurations): frames sampled from
the stream are downsized to the configured resolution and classified.

Frozen-prefix reuse: stages below the lowest trainable one never change, so
their eval-mode output can be computed once per frame and reused by every
epoch.  This oracle does the same (and `use_cache=False` recomputes it for
every batch, which gives bitwise the same numbers).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import nn, rng
from .resnet18 import ResNet18, STAGES


@dataclass
class RetrainResult:
    weights: np.ndarray                    # canonical flat, float64
    heldout_acc: List[float] = field(default_factory=list)   # after each epoch
    losses: List[float] = field(default_factory=list)        # per SGD step
    train_indices: List[int] = field(default_factory=list)   # the subset, in draw order
    n_correct: List[int] = field(default_factory=list)


def prefix_forward(net: ResNet18, P, frames: np.ndarray, lowest: int) -> np.ndarray:
    """Eval-mode output of stages 0..lowest-1 (the frozen prefix)."""
    x = np.asarray(frames, dtype=np.float64)
    if lowest == 0:
        return x
    return net.forward(P, x, 0, lowest - 1, train=False, tape={})


def heldout_correct(net: ResNet18, P, feats: np.ndarray, labels: np.ndarray, lowest: int) -> int:
    logits = net.forward(P, feats, lowest, 5, train=False, tape={})
    return int(np.sum(nn.argmax(logits) == labels))


def retrain(weights: np.ndarray, k: int, frames: np.ndarray, labels: np.ndarray,
            heldout_frames: np.ndarray, heldout_labels: np.ndarray,
            subsample_frac: float, epochs: int, lr: float, momentum: float = 0.9,
            batch: int = 64, seed: int = 0, shuffle_seed: Optional[int] = None,
            n_classes: int = 6, use_cache: bool = True,
            net: Optional[ResNet18] = None) -> RetrainResult:
    """Fine-tune the last k stages; returns new weights and per-epoch held-out accuracy.

    The subset uses `seed`; epoch shuffles use `shuffle_seed` (default `seed`)."""
    if shuffle_seed is None:
        shuffle_seed = seed
    net = net or ResNet18(n_classes)
    P = net.unpack(weights)
    lowest = len(STAGES) - k
    trainable = net.trainable_names(k)
    vel: Dict[str, np.ndarray] = {n: np.zeros_like(P[n]) for n in trainable}

    S = rng.training_subset(len(frames), subsample_frac, seed)
    res = RetrainResult(weights=None, train_indices=list(S))
    train_frames = np.asarray(frames)[S]
    train_labels = np.asarray(labels)[S]
    if use_cache:
        feats = prefix_forward(net, P, train_frames, lowest)
    hfeats = prefix_forward(net, P, heldout_frames, lowest)

    n = len(S)
    nb = math.ceil(n / batch)
    for e in range(epochs):
        order = rng.epoch_order(n, shuffle_seed, e)
        for b in range(nb):
            idx = order[b * batch:(b + 1) * batch]
            if use_cache:
                x = feats[idx]
            else:
                x = prefix_forward(net, P, train_frames[idx], lowest)
            tape: dict = {}
            logits = net.forward(P, x, lowest, 5, train=True, tape=tape)
            loss, dz, _ = nn.softmax_cross_entropy(logits, train_labels[idx])
            grads = net.backward(P, dz, lowest, tape)
            for name in trainable:
                P[name], vel[name] = nn.sgd_momentum(P[name], vel[name], grads[name], lr, momentum)
            res.losses.append(loss)
        c = heldout_correct(net, P, hfeats, np.asarray(heldout_labels), lowest)
        res.n_correct.append(c)
        res.heldout_acc.append(c / len(heldout_labels))
    res.weights = net.pack(P)
    return res


@dataclass
class ProfileConfig:
    k: int
    subsample_frac: float
    epochs: int
    lr: float = 0.01
    momentum: float = 0.9
    batch: int = 64
    seed: int = 0     # epoch-shuffle seed of this configuration


def profile(weights: np.ndarray, configs: List[ProfileConfig], frames, labels,
            heldout_frames, heldout_labels, subsample_seed: int = 0,
            n_classes: int = 6) -> List[RetrainResult]:
    """Micro-profile every configuration from the same starting weights.

    All configurations draw their subset from one shuffle (seed
    `subsample_seed`), so a smaller fraction's subset is a prefix of a larger
    one's; each configuration shuffles its epochs with its own seed."""
    net = ResNet18(n_classes)
    return [retrain(weights, c.k, frames, labels, heldout_frames, heldout_labels,
                    c.subsample_frac, c.epochs, c.lr, c.momentum, c.batch,
                    seed=subsample_seed, shuffle_seed=c.seed, n_classes=n_classes, net=net)
            for c in configs]


def infer(weights: np.ndarray, frames: np.ndarray, resolution: int,
          n_classes: int = 6, net: Optional[ResNet18] = None) -> np.ndarray:
    """Labels (int32) of frames resized to resolution x resolution, eval mode."""
    net = net or ResNet18(n_classes)
    P = net.unpack(weights)
    x = np.asarray(frames, dtype=np.float64)
    if x.shape[1] != resolution or x.shape[2] != resolution:
        x = nn.resize_bilinear(x, resolution, resolution)
    logits = net.forward(P, x, 0, 5, train=False, tape={})
    return nn.argmax(logits).astype(np.int32)


def infer_logits(weights: np.ndarray, frames: np.ndarray, resolution: int,
                 n_classes: int = 6) -> np.ndarray:
    net = ResNet18(n_classes)
    P = net.unpack(weights)
    x = np.asarray(frames, dtype=np.float64)
    if x.shape[1] != resolution or x.shape[2] != resolution:
        x = nn.resize_bilinear(x, resolution, resolution)
    return net.forward(P, x, 0, 5, train=False, tape={})
