"""Pins for the oracle's random draws (subset and epoch shuffles)."""
import itertools
import os
from collections import Counter

from oracle import rng

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")


def _golden_rows():
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                vals = [int(v) for v in line.split()]
                yield vals[0], vals[1:]


def test_splitmix64_published_outputs():
    rows = list(_golden_rows())
    assert len(rows) == 2
    for state, expected in rows:
        g = rng.SplitMix64(state)
        assert [g.next() for _ in expected] == expected


def test_fisher_yates_is_uniform_on_small_n():
    # Every permutation of 4 elements should be equally likely (Fisher-Yates
    # property); with 24000 draws each count is ~1000 +- 3 sigma (~95).
    counts = Counter(tuple(rng.partial_shuffle(4, 4, seed * 7919 + 1)) for seed in range(24000))
    assert set(counts) == set(itertools.permutations(range(4)))
    assert max(counts.values()) < 1000 + 150 and min(counts.values()) > 1000 - 150


def test_subset_is_without_replacement_and_prefix_nested():
    n = 4000
    big = rng.training_subset(n, 0.10, seed=3)
    small = rng.training_subset(n, 0.05, seed=3)
    assert len(big) == 400 and len(small) == 200
    assert len(set(big)) == 400 and all(0 <= i < n for i in big)
    assert big[:200] == small


def test_subset_sizes_round_half_up():
    assert rng.subset_size(2000, 0.3) == 600
    assert rng.subset_size(4000, 0.05) == 200
    assert rng.subset_size(3600, 0.10) == 360
    assert rng.subset_size(10, 0.25) == 3      # 2.5 rounds up
    assert rng.subset_size(10, 0.01) == 1      # at least one frame
    assert rng.subset_size(64, 1.0) == 64


def test_epoch_orders_are_permutations_and_differ():
    a = rng.epoch_order(600, 0, 0)
    b = rng.epoch_order(600, 0, 1)
    assert sorted(a) == list(range(600)) and sorted(b) == list(range(600))
    assert a != b


def test_first_draw_by_hand():
    # The first swap partner of a shuffle of n is (first output) mod n.
    first = rng.SplitMix64(0).next()
    assert rng.partial_shuffle(1000, 1, 0) == [first % 1000]
