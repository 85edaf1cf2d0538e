"""Pins of the thief-scheduler oracle (oracle/scheduler.py): the numbers of
the paper's worked example (Table 1 and the text around it), closed forms of
EstimateAccuracy, the invariants of Algorithm 1 (shares in whole quanta,
total conserved, never worse than the fair start) and brute force over every
allocation of small instances (the heuristic never beats the optimum and
reaches it where stealing is monotone)."""
import itertools

import pytest

from oracle import scheduler as S

T = 120.0
FULL = [S.InferConfig(cost=1.0, factor=1.0)]


def table1_window1():
    """Section 3.2's example: cameras A and B, models at 65% and 50% before
    window 1; Cfg1A 75% / 85 GPU-s, Cfg2A 70% / 65, Cfg1B 90% / 80,
    Cfg2B 85% / 50; the inference job needs one GPU to keep up."""
    A = S.Video(0.65, FULL, [S.TrainConfig(0.75, 85.0), S.TrainConfig(0.70, 65.0)])
    B = S.Video(0.50, FULL, [S.TrainConfig(0.90, 80.0), S.TrainConfig(0.85, 50.0)])
    return [A, B]


def test_inference_drops_as_in_the_worked_example():
    """Inference of A keeps 0.75 of the GPU it needs: 65% -> 49% (48.75%);
    B: 50% -> 37.5%, as the text states."""
    assert abs(S.inference_accuracy(0.65, FULL[0], 0.75) - 0.4875) < 1e-15
    assert abs(S.inference_accuracy(0.50, FULL[0], 0.75) - 0.375) < 1e-15
    assert S.inference_accuracy(0.65, FULL[0], 1.5) == 0.65


def test_estimate_accuracy_closed_form():
    """Uniform split of 3 GPUs (0.75 each job): Cfg1B retrains in 80 / 0.75 =
    106.7 s at 37.5%, then 13.3 s at 90% x 0.75 of the frames."""
    A, B = table1_window1()
    a = S.estimate_accuracy(B, B.train[0], FULL[0], 0.75, 0.75, T)
    d = 80.0 / 0.75
    assert abs(a - (d * 0.375 + (T - d) * 0.9 * 0.75) / T) < 1e-15
    # 85 GPU-s at a quarter GPU takes 340 s > 120 s: not feasible
    assert S.estimate_accuracy(A, A.train[0], FULL[0], 0.75, 0.25, T) is None
    # no retraining: the current model for the whole window
    assert abs(S.estimate_accuracy(A, None, FULL[0], 0.75, 0.75, T) - 0.4875) < 1e-15


def test_fair_allocation_spreads_quanta():
    assert S.fair_allocation(4, 12) == [3, 3, 3, 3]
    assert S.fair_allocation(4, 30) == [8, 8, 7, 7]


def _check_invariants(videos, G, delta, sched, a_min):
    q = [round(a / delta) for a in sched.alloc]
    assert all(abs(a - k * delta) < 1e-12 for a, k in zip(sched.alloc, q))
    assert sum(q) == round(G / delta) and min(q) >= 0
    ic, tc, accs, acc = S.pick_configs(videos, sched.alloc, T, a_min)
    assert (ic, tc, acc) == (sched.infer_choice, sched.train_choice, sched.accuracy)
    fair = [k * delta for k in S.fair_allocation(len(sched.alloc), round(G / delta))]
    assert sched.accuracy >= S.pick_configs(videos, fair, T, a_min)[3]


@pytest.mark.parametrize("delta", [0.75, 0.25, 0.1])
def test_worked_example_schedule(delta):
    """The thief beats the uniform schedule on the worked example and, as the
    text describes, gives video B's retraining (+35 points) more GPU than A's
    (+5 points) and picks cheaper configurations where they pay off."""
    videos = table1_window1()
    sched = S.thief_schedule(videos, 3.0, delta, T, 0.40)
    _check_invariants(videos, 3.0, delta, sched, 0.40)
    uniform = S.pick_configs(videos, [0.75] * 4, T, 0.40)[3]
    print(delta, sched.alloc, sched.train_choice, round(sched.accuracy, 4), round(uniform, 4))
    if delta < 0.75:
        assert sched.accuracy > uniform
        assert sched.alloc[3] > sched.alloc[1]


def _brute_force(videos, G, delta, a_min):
    quanta, n = round(G / delta), 2 * len(videos)
    best = -1.0
    for cut in itertools.combinations(range(quanta + n - 1), n - 1):
        parts, prev = [], -1
        for c in cut + (quanta + n - 1,):
            parts.append(c - prev - 1)
            prev = c
        best = max(best, S.pick_configs(videos, [p * delta for p in parts], T, a_min)[3])
    return best


@pytest.mark.parametrize("seed", range(4))
def test_never_better_than_exhaustive_search(seed):
    import random
    r = random.Random(seed)
    videos = []
    for _ in range(2):
        infer = [S.InferConfig(cost=c, factor=f) for c, f in ((1.0, 1.0), (0.5, 0.85), (0.25, 0.6))]
        train = [S.TrainConfig(r.uniform(0.6, 0.95), r.uniform(20, 150)) for _ in range(3)]
        videos.append(S.Video(r.uniform(0.4, 0.7), infer, train))
    sched = S.thief_schedule(videos, 2.0, 0.25, T, 0.3)
    _check_invariants(videos, 2.0, 0.25, sched, 0.3)
    opt = _brute_force(videos, 2.0, 0.25, 0.3)
    assert sched.accuracy <= opt + 1e-12


def test_reaches_the_optimum_when_stealing_is_monotone():
    """One stream, a retraining configuration that pays off more the faster
    it runs, and inference that keeps up with a quarter GPU: moving every
    spare quantum to retraining is optimal and the thief finds it."""
    v = S.Video(0.5, [S.InferConfig(cost=0.25, factor=1.0)], [S.TrainConfig(0.9, 60.0)])
    sched = S.thief_schedule([v], 2.0, 0.25, T, 0.3)
    assert abs(sched.accuracy - _brute_force([v], 2.0, 0.25, 0.3)) < 1e-15
    assert sched.alloc == [0.25, 1.75]
