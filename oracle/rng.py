"""Random draws of the method: the training subset and the epoch shuffles.

The paper's micro-profiler trains on a uniform random subset of the window's
training data (section 4.3, "Training data sampling"); plain mini-batch SGD
visits that subset in a fresh random order every epoch.  Both draws use
SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) with the generator's published
constants, and the forward form of the Fisher-Yates shuffle (Durstenfeld,
CACM 1964): for i = 0, 1, ..., pick j uniformly in [i, n) and swap a[i], a[j].
A uniform integer in [0, m) is taken as (next output) mod m.

Seeds: the subset uses start state `seed`; the shuffle of epoch e (0-based)
uses start state seed + (e + 1) * 0xD1B54A32D192ED03 (mod 2**64).
Because the subset is the first n entries of a shuffle, the subset for a
smaller fraction is a prefix of the subset for a larger one.
"""
from __future__ import annotations

import math
from typing import List

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
EPOCH_STRIDE = 0xD1B54A32D192ED03


class SplitMix64:
    def __init__(self, state: int):
        self.state = state & MASK64

    def next(self) -> int:
        self.state = (self.state + GOLDEN) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)


def partial_shuffle(n: int, count: int, state: int) -> List[int]:
    """First `count` entries of a forward Fisher-Yates shuffle of 0..n-1."""
    g = SplitMix64(state)
    a = list(range(n))
    for i in range(count):
        j = i + g.next() % (n - i)
        a[i], a[j] = a[j], a[i]
    return a[:count]


def subset_size(n_frames: int, frac: float) -> int:
    """round-half-up(frac * n), at least 1."""
    return max(1, int(math.floor(frac * n_frames + 0.5)))


def training_subset(n_frames: int, frac: float, seed: int) -> List[int]:
    return partial_shuffle(n_frames, subset_size(n_frames, frac), seed)


def epoch_order(n: int, seed: int, epoch: int) -> List[int]:
    return partial_shuffle(n, n, (seed + (epoch + 1) * EPOCH_STRIDE) & MASK64)
