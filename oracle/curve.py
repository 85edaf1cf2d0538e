"""Accuracy-curve extrapolation of the micro-profiler (section 4.3): the
held-out accuracy after each epoch of a short run on a small subset is fitted
to the training-progress curve of Optimus (Peng et al., "Optimus: an efficient
dynamic resource scheduler for deep learning clusters", EuroSys 2018) with a
non-negative least-squares solver, and the fit is evaluated at the amount of
training a full retraining would do.

Test infrastructure (the CPU oracle): plain numpy, slow and direct.

Readings (the paper names the model and the solver but prints neither):
  * Optimus models the training loss after k units of training as
    l(k) = 1 / (b0 k + b1) + b2 with b0, b1, b2 >= 0.  Here the decreasing
    quantity is the held-out error e = 1 - accuracy.
  * The unit of training is one pass over the whole window's data: a run of
    E epochs on a fraction f of the window has done x = E f of them, so the
    points of a short low-fraction run and the full retraining it stands for
    (E' epochs on all the data, x = E') lie on one curve.
  * The fit is non-negative least squares in the form the model allows: for a
    given b2 below every measured error, 1 / (e - b2) = b0 x + b1 is linear in
    (b0, b1) >= 0 and is solved by NNLS; b2 itself is chosen (on a grid over
    [0, min e), refined by golden-section search) to minimise the squared
    error of the fitted curve in accuracy.  With fewer points than parameters
    many curves fit exactly; a candidate replaces the best one only if its
    squared error is smaller by more than a relative 1e-9 and an absolute
    1e-20, so such ties keep the smallest b2 tried.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Sequence

import numpy as np


def nnls(A: np.ndarray, b: np.ndarray, max_iter: int = 0):
    """min ||A x - b||_2 subject to x >= 0, by Lawson and Hanson's active-set
    method ("Solving Least Squares Problems", 1974, chapter 23): start with
    every variable held at zero; repeatedly free the held variable whose
    gradient component w = A^T (b - A x) is largest and positive, solve the
    unconstrained least-squares problem on the free set, and while that
    solution has non-positive entries move back along the segment towards it
    only as far as feasibility allows, returning the variables that hit zero
    to the held set.  Stops when no held variable has positive w.
    Returns (x, ||A x - b||)."""
    A = np.asarray(A, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    m, n = A.shape
    x = np.zeros(n)
    free = np.zeros(n, dtype=bool)
    tol = 10.0 * np.finfo(np.float64).eps * np.linalg.norm(A, 1) * max(m, n)
    max_iter = max_iter or 3 * n
    for _ in range(max_iter):
        w = A.T @ (b - A @ x)
        candidates = np.where(~free & (w > tol))[0]
        if candidates.size == 0:
            break
        free[candidates[np.argmax(w[candidates])]] = True
        while True:
            z = np.zeros(n)
            idx = np.where(free)[0]
            z[idx] = np.linalg.lstsq(A[:, idx], b, rcond=None)[0]
            if np.all(z[idx] > tol):
                x = z
                break
            neg = idx[z[idx] <= tol]
            alpha = np.min(x[neg] / (x[neg] - z[neg]))
            x = x + alpha * (z - x)
            free &= ~(x <= tol)
            x[~free] = 0.0
    return x, float(np.linalg.norm(A @ x - b))


@dataclass
class Curve:
    b0: float
    b1: float
    b2: float
    rss: float  # squared error of the fitted accuracy at the points

    def error(self, x):
        x = np.asarray(x, dtype=np.float64)
        d = self.b0 * x + self.b1
        return np.where(d > 0, 1.0 / np.where(d > 0, d, 1.0), np.inf) + self.b2

    def accuracy(self, x):
        return np.clip(1.0 - self.error(x), 0.0, 1.0)


def _better(a, b):
    """a's squared error is smaller than b's by more than a relative 1e-9 and
    an absolute 1e-20 (exact fits differ only by rounding)."""
    return a.rss < b.rss * (1.0 - 1e-9) - 1e-20


def _fit_given_b2(x, e, b2):
    """(b0, b1) >= 0 of 1 / (e - b2) = b0 x + b1 by NNLS, and the squared
    error of the resulting curve in accuracy."""
    A = np.stack([x, np.ones_like(x)], axis=1)
    (b0, b1), _ = nnls(A, 1.0 / (e - b2))
    c = Curve(float(b0), float(b1), float(b2), 0.0)
    c.rss = float(np.sum((c.error(x) - e) ** 2))
    return c


def fit_accuracy_curve(x: Sequence[float], acc: Sequence[float], grid: int = 64,
                       refine: int = 60) -> Curve:
    """Fit the Optimus curve to (training passes, held-out accuracy) points."""
    x = np.asarray(x, dtype=np.float64)
    e = 1.0 - np.asarray(acc, dtype=np.float64)
    if x.size == 0:
        raise ValueError("no points")
    emin = float(np.min(e))
    if emin <= 0.0:  # a perfect point: the curve must reach error 0 -> b2 = 0
        e = np.maximum(e, 1e-12)
        return _fit_given_b2(x, e, 0.0)
    hi = emin * (1.0 - 1e-9)
    best = None
    for i in range(grid):
        c = _fit_given_b2(x, e, hi * i / grid)
        if best is None or _better(c, best):
            best, bi = c, i
    # golden-section search on the bracket around the best grid point
    lo_b, hi_b = hi * max(bi - 1, 0) / grid, hi * min(bi + 1, grid) / grid
    g = (math.sqrt(5.0) - 1.0) / 2.0
    a, d = lo_b, hi_b
    c1, c2 = d - g * (d - a), a + g * (d - a)
    f1, f2 = _fit_given_b2(x, e, c1), _fit_given_b2(x, e, min(c2, hi))
    for _ in range(refine):
        if f1.rss <= f2.rss:
            d, c2, f2 = c2, c1, f1
            c1 = d - g * (d - a)
            f1 = _fit_given_b2(x, e, c1)
        else:
            a, c1, f1 = c1, c2, f2
            c2 = a + g * (d - a)
            f2 = _fit_given_b2(x, e, min(c2, hi))
    for c in (f1, f2):
        if _better(c, best):
            best = c
    return best


def extrapolate(epoch_acc: Sequence[float], epoch_seconds: Sequence[float], n_train: int,
                n_frames: int, batch: int, epochs_target: int):
    """From a profiled candidate (accuracy and GPU seconds after each of its
    epochs on n_train of the window's n_frames frames): the curve, the
    accuracy it predicts for epochs_target epochs on the whole window, and the
    GPU seconds of that retraining at the full GPU -- the candidate's mean
    epoch time scaled by the SGD steps of a full epoch (per-epoch cost is
    deterministic, section 4.3) and by the epochs."""
    f = n_train / n_frames
    xs = [(i + 1) * f for i in range(len(epoch_acc))]
    curve = fit_accuracy_curve(xs, epoch_acc)
    steps_sub = -(-n_train // batch)
    steps_full = -(-n_frames // batch)
    sec = float(np.mean(epoch_seconds)) * steps_full / steps_sub * epochs_target
    return curve, float(curve.accuracy(float(epochs_target))), sec
