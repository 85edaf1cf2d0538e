"""The scheduling layer of the library (include/ekya_sched.h; host code, no
GPU) against the oracle: NNLS, the accuracy-curve fit, the extrapolation of
a profiled candidate and the thief scheduler give the oracle's results on
the same inputs."""
import os
import random

import numpy as np
import pytest

from oracle import curve, scheduler as S

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2012_10557_amd",
                   "libekya.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libekya.so not built")


@pytest.mark.parametrize("m,n,seed", [(8, 4, 0), (20, 6, 1), (5, 8, 2), (40, 3, 3), (64, 16, 4)])
def test_nnls_matches_oracle(m, n, seed):
    from paper_2012_10557_amd import binding
    rng = np.random.default_rng(seed)
    A, b = rng.standard_normal((m, n)), rng.standard_normal(m)
    x, r = binding.ekya_nnls(A, b)
    xo, ro = curve.nnls(A, b)
    np.testing.assert_allclose(x, xo, atol=1e-10)
    assert abs(r - ro) <= 1e-10 * max(1.0, ro)


def test_nnls_rejects_bad_arguments():
    from paper_2012_10557_amd import binding
    with pytest.raises(binding.EkyaError):
        binding.ekya_nnls(np.zeros((0, 3)), np.zeros(0))
    with pytest.raises(binding.EkyaError):
        binding.ekya_nnls(np.full((2, 2), np.nan), np.zeros(2))


@pytest.mark.parametrize("seed", range(5))
def test_curve_fit_matches_oracle(seed):
    from paper_2012_10557_amd import binding
    rng = np.random.default_rng(seed)
    f = [0.05, 0.1, 0.25][seed % 3]
    xs = f * np.arange(1, 2 + seed)
    acc = np.clip(1.0 - (1.0 / (rng.uniform(2, 20) * xs + rng.uniform(1.05, 3)) + rng.uniform(0, 0.3))
                  + 0.01 * rng.standard_normal(xs.size), 0.0, 1.0)
    c = binding.ekya_fit_accuracy_curve(xs, acc)
    co = curve.fit_accuracy_curve(xs, acc)
    for x in (xs[0], 1.0, 5.0, 30.0):
        assert abs(binding.ekya_curve_accuracy(c, x) - float(co.accuracy(x))) < 1e-7
    assert abs(c.rss - co.rss) <= 1e-9 + 1e-6 * co.rss


def test_extrapolate_matches_oracle():
    from paper_2012_10557_amd import binding
    cfg = {"k": 2, "subsample_frac": 0.05, "epochs": 3, "batch": 64}
    res = {"status": 0, "n_train": 200, "heldout_acc": [0.3, 0.55, 0.62],
           "epoch_seconds": [0.0021, 0.0020, 0.0022]}
    c, acc, sec = binding.ekya_extrapolate(cfg, res, 4000, 10)
    f32 = lambda v: [float(np.float32(x)) for x in v]  # the result record holds float32
    co, acco, seco = curve.extrapolate(f32(res["heldout_acc"]), f32(res["epoch_seconds"]), 200, 4000,
                                       64, 10)
    assert abs(acc - acco) < 1e-7
    assert abs(sec - seco) < 1e-12


def _random_videos(seed, n):
    r = random.Random(seed)
    out = []
    for _ in range(n):
        infer = [(c, f) for c, f in ((1.0, 1.0), (0.5, 0.85), (0.25, 0.6))]
        train = [(r.uniform(0.55, 0.95), r.uniform(10, 200)) for _ in range(r.randint(0, 4))]
        out.append({"acc_now": r.uniform(0.3, 0.8), "infer": infer, "train": train})
    return out


@pytest.mark.parametrize("seed,n,G,delta", [(0, 2, 3.0, 0.25), (1, 3, 2.0, 0.1), (2, 4, 4.0, 0.5),
                                            (3, 10, 2.0, 0.1), (4, 1, 1.0, 0.1)])
def test_thief_schedule_matches_oracle(seed, n, G, delta):
    from paper_2012_10557_amd import binding
    vids = _random_videos(seed, n)
    got = binding.ekya_thief_schedule(vids, G, delta, 120.0, 0.35)
    ref = S.thief_schedule([S.Video(v["acc_now"], [S.InferConfig(c, f) for c, f in v["infer"]],
                                    [S.TrainConfig(a, g) for a, g in v["train"]]) for v in vids],
                           G, delta, 120.0, 0.35)
    assert got["alloc"] == ref.alloc
    assert got["infer_choice"] == ref.infer_choice and got["train_choice"] == ref.train_choice
    assert abs(got["accuracy"] - ref.accuracy) < 1e-15
    assert got["video_accuracy"] == ref.video_accuracy


def test_thief_schedule_rejects_fractional_quanta():
    from paper_2012_10557_amd import binding
    with pytest.raises(binding.EkyaError):
        binding.ekya_thief_schedule(_random_videos(0, 2), 1.0, 0.3, 120.0, 0.3)
