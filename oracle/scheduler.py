"""The thief scheduler of section 4.2 (Algorithm 1) with PickConfigs
(Algorithm 2) and EstimateAccuracy, as the paper describes them; test
infrastructure (the CPU oracle), plain Python.

Problem (section 4.1): for every video stream v in a retraining window of T
seconds on G GPUs, choose an inference configuration, a retraining
configuration (or none) and the GPU shares of the stream's inference job and
retraining job, in multiples of a quantum Delta, maximising the inference
accuracy averaged over the window and over the streams.

Readings (the paper fixes the algorithms' steps but not every model):
  * An inference configuration lambda has a cost c (the GPU share it needs to
    keep up with the live stream) and an accuracy factor q (its accuracy
    relative to the full configuration).  Run on a share I it reaches
    model accuracy x q x min(1, I / c): frames it cannot keep up with are
    not analysed (in Table 1's example 65% falls to 49% when the inference
    job keeps 0.75 of the 1 GPU it needs).  PickConfigs picks, among the
    configurations with c <= I whose accuracy acc_now x q is at least
    a_min, the most accurate one; if none qualifies, the cheapest.
  * A retraining configuration gamma has the accuracy acc_after of the model
    it produces and the GPU time g it takes on a full GPU (the micro-
    profiler's estimates).  EstimateAccuracy of gamma with a retraining share
    R: retraining lasts d = g / R; configurations with d > T are skipped;
    the inference runs the old model (acc_now) for d seconds and the new one
    for T - d, so the window's mean accuracy is
    (d acc_now + (T - d) acc_after) / T x (inference factor).  "No
    retraining" (always available) keeps acc_now for the whole window.
  * fair_allocation splits the G / Delta quanta evenly over the jobs (the
    first jobs take the remainder).
  * Ties keep the earlier choice (strict improvement is required to switch).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple


@dataclass
class InferConfig:
    cost: float    # GPU share needed to keep up with the stream
    factor: float  # accuracy relative to the full inference configuration


@dataclass
class TrainConfig:
    acc_after: float    # accuracy of the retrained model
    gpu_seconds: float  # retraining time on a whole GPU


@dataclass
class Video:
    acc_now: float
    infer: List[InferConfig]
    train: List[TrainConfig]


@dataclass
class Schedule:
    alloc: List[float]                 # per job: [infer v0, train v0, infer v1, ...]
    infer_choice: List[int]            # per video
    train_choice: List[int]            # per video, -1 = no retraining
    accuracy: float                    # mean over videos of the window accuracy
    video_accuracy: List[float] = field(default_factory=list)


def inference_accuracy(model_acc: float, cfg: InferConfig, share: float) -> float:
    keep = 1.0 if share >= cfg.cost else share / cfg.cost
    return model_acc * cfg.factor * keep


def estimate_accuracy(v: Video, train: Optional[TrainConfig], icfg: InferConfig, infer_share: float,
                      train_share: float, T: float) -> Optional[float]:
    """Mean inference accuracy over the window, or None if the retraining does
    not finish inside it."""
    if train is None:
        return inference_accuracy(v.acc_now, icfg, infer_share)
    if train_share <= 0.0:
        return None
    d = train.gpu_seconds / train_share
    if d > T:
        return None
    return (d * inference_accuracy(v.acc_now, icfg, infer_share)
            + (T - d) * inference_accuracy(train.acc_after, icfg, infer_share)) / T


def pick_configs(videos: List[Video], alloc: List[float], T: float, a_min: float
                 ) -> Tuple[List[int], List[int], List[float], float]:
    """Algorithm 2: per video the inference configuration, then the
    retraining configuration maximising the window accuracy; returns the
    choices, the per-video accuracies and their mean."""
    ichoice, tchoice, accs = [], [], []
    for vi, v in enumerate(videos):
        ishare, tshare = alloc[2 * vi], alloc[2 * vi + 1]
        pool = [i for i, c in enumerate(v.infer)
                if c.cost <= ishare + 1e-12 and v.acc_now * c.factor >= a_min]
        if pool:
            best_i = max(pool, key=lambda i: (v.infer[i].factor, -i))
        else:
            best_i = min(range(len(v.infer)), key=lambda i: (v.infer[i].cost, i))
        icfg = v.infer[best_i]
        best_acc = estimate_accuracy(v, None, icfg, ishare, tshare, T)
        best_t = -1
        for ti, tc in enumerate(v.train):
            a = estimate_accuracy(v, tc, icfg, ishare, tshare, T)
            if a is not None and a > best_acc:
                best_acc, best_t = a, ti
        ichoice.append(best_i)
        tchoice.append(best_t)
        accs.append(best_acc)
    return ichoice, tchoice, accs, sum(accs) / len(accs)


def fair_allocation(n_jobs: int, quanta: int) -> List[int]:
    """The quanta split evenly over the jobs (the first jobs take the remainder)."""
    base, extra = divmod(quanta, n_jobs)
    return [base + (1 if j < extra else 0) for j in range(n_jobs)]


def thief_schedule(videos: List[Video], G: float, delta: float, T: float, a_min: float) -> Schedule:
    """Algorithm 1: start from the fair allocation; every job in turn steals
    one quantum at a time from every other job while the window accuracy
    improves.  Allocations are counted in quanta of delta (G / delta of them)."""
    n_jobs = 2 * len(videos)
    quanta = int(round(G / delta))
    share = lambda q: [x * delta for x in q]
    best_q = fair_allocation(n_jobs, quanta)
    ic, tc, accs, best = pick_configs(videos, share(best_q), T, a_min)
    best_cfg = (ic, tc, accs)
    for thief in range(n_jobs):
        for victim in range(n_jobs):
            if thief == victim:
                continue
            temp = list(best_q)
            while True:
                temp[victim] -= 1
                temp[thief] += 1
                if temp[victim] < 0:
                    break
                ic, tc, accs, acc = pick_configs(videos, share(temp), T, a_min)
                if acc > best:
                    best_q, best, best_cfg = list(temp), acc, (ic, tc, accs)
                else:
                    break
    return Schedule(share(best_q), best_cfg[0], best_cfg[1], best, best_cfg[2])
