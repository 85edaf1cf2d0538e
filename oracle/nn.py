"""Layer operations of the ResNet18 edge classifier, float64, NHWC.

The paper runs its retraining as ordinary PyTorch training (section 5,
"Ekya Implementation"), so every operation below is the textbook definition of
the matching PyTorch layer: cross-correlation with zero padding, BatchNorm with
biased batch variance and an unbiased running estimate (momentum 0.1,
eps 1e-5), max pooling with -inf padding, global average pooling, an affine
classifier, mean softmax cross-entropy, and SGD with momentum (v <- mu v + g,
w <- w - lr v; no dampening, no Nesterov, no weight decay).

Layouts: activations are [N, H, W, C]; convolution weights are [K, C, R, S]
(output channel, input channel, kernel row, kernel column); classifier weights
are [classes, features].
"""
from __future__ import annotations

import numpy as np

BN_EPS = 1e-5
BN_MOMENTUM = 0.1


def out_size(n: int, k: int, stride: int, pad: int) -> int:
    return (n + 2 * pad - k) // stride + 1


# ---------------------------------------------------------------- convolution

def _pad(x: np.ndarray, pad: int, value: float = 0.0) -> np.ndarray:
    n, h, w, c = x.shape
    xp = np.full((n, h + 2 * pad, w + 2 * pad, c), value, dtype=np.float64)
    xp[:, pad:pad + h, pad:pad + w, :] = x
    return xp


def _window(xp: np.ndarray, r: int, s: int, stride: int, p: int, q: int) -> np.ndarray:
    """xp[:, r + stride*i, s + stride*j, :] for i < p, j < q."""
    return xp[:, r:r + stride * (p - 1) + 1:stride, s:s + stride * (q - 1) + 1:stride, :]


def _tap(w: np.ndarray, r: int, s: int) -> np.ndarray:
    """The [K, C] matrix w[:, :, r, s] (contiguous, so the product runs in BLAS)."""
    return np.ascontiguousarray(w[:, :, r, s])


def _rows(a: np.ndarray) -> np.ndarray:
    """[N, P, Q, C] -> contiguous [N*P*Q, C]."""
    return np.ascontiguousarray(a).reshape(-1, a.shape[-1])


def conv2d(x: np.ndarray, w: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """y[n,p,q,k] = sum_{c,r,s} x[n, stride*p + r - pad, stride*q + s - pad, c] * w[k,c,r,s]."""
    n, h, wd, c = x.shape
    k, c2, R, S = w.shape
    assert c == c2
    P, Q = out_size(h, R, stride, pad), out_size(wd, S, stride, pad)
    xp = _pad(x, pad)
    y = np.zeros((n, P, Q, k), dtype=np.float64)
    for r in range(R):
        for s in range(S):
            y += (_rows(_window(xp, r, s, stride, P, Q)) @ _tap(w, r, s).T).reshape(y.shape)
    return y


def conv2d_dgrad(dy: np.ndarray, w: np.ndarray, x_shape, stride: int, pad: int) -> np.ndarray:
    """Gradient of `conv2d` with respect to x: every output gradient is sent back
    along the same (r, s) taps that produced it."""
    n, h, wd, c = x_shape
    _, P, Q, k = dy.shape
    R, S = w.shape[2], w.shape[3]
    dxp = np.zeros((n, h + 2 * pad, wd + 2 * pad, c), dtype=np.float64)
    for r in range(R):
        for s in range(S):
            dxp[:, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride, :] += \
                (_rows(dy) @ _tap(w, r, s)).reshape(dy.shape[:3] + (c,))
    return dxp[:, pad:pad + h, pad:pad + wd, :]


def conv2d_wgrad(x: np.ndarray, dy: np.ndarray, w_shape, stride: int, pad: int) -> np.ndarray:
    """dw[k,c,r,s] = sum_{n,p,q} dy[n,p,q,k] * x[n, stride*p + r - pad, stride*q + s - pad, c]."""
    k, c, R, S = w_shape
    _, P, Q, _ = dy.shape
    xp = _pad(x, pad)
    dy2 = _rows(dy)
    dw = np.zeros(w_shape, dtype=np.float64)
    for r in range(R):
        for s in range(S):
            dw[:, :, r, s] = dy2.T @ _rows(_window(xp, r, s, stride, P, Q))
    return dw


# ------------------------------------------------------------------ BatchNorm

def batchnorm_train(z: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float = BN_EPS):
    """Normalise with the batch mean and biased variance over (N, H, W).

    Returns (y, saved) where saved = (xhat, invstd, mean, var_biased, count)."""
    m = z.shape[0] * z.shape[1] * z.shape[2]
    mean = z.mean(axis=(0, 1, 2))
    var = ((z - mean) ** 2).mean(axis=(0, 1, 2))
    invstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mean) * invstd
    return gamma * xhat + beta, (xhat, invstd, mean, var, m)


def batchnorm_running_update(rm: np.ndarray, rv: np.ndarray, mean: np.ndarray,
                             var_biased: np.ndarray, count: int,
                             momentum: float = BN_MOMENTUM):
    """New running statistics; the variance estimate is the unbiased one."""
    var_unbiased = var_biased * count / (count - 1) if count > 1 else var_biased
    return ((1.0 - momentum) * rm + momentum * mean,
            (1.0 - momentum) * rv + momentum * var_unbiased)


def batchnorm_eval(z: np.ndarray, gamma, beta, rm, rv, eps: float = BN_EPS) -> np.ndarray:
    return (z - rm) / np.sqrt(rv + eps) * gamma + beta


def batchnorm_backward(dy: np.ndarray, saved, gamma: np.ndarray):
    """Gradients (dz, dgamma, dbeta) of batchnorm_train.

    With xhat = (z - mean) * invstd and y = gamma * xhat + beta, and m elements
    per channel: dbeta = sum dy, dgamma = sum dy * xhat, and
    dz = gamma * invstd / m * (m * dy - dbeta - xhat * dgamma)."""
    xhat, invstd, _, _, m = saved
    dbeta = dy.sum(axis=(0, 1, 2))
    dgamma = (dy * xhat).sum(axis=(0, 1, 2))
    dz = gamma * invstd / m * (m * dy - dbeta - xhat * dgamma)
    return dz, dgamma, dbeta


# ----------------------------------------------------------------------- ReLU

def relu(x: np.ndarray) -> np.ndarray:
    return np.maximum(x, 0.0)


def relu_backward(dy: np.ndarray, y: np.ndarray) -> np.ndarray:
    """ReLU'(0) = 0: gradient passes only where the output is positive."""
    return dy * (y > 0.0)


# -------------------------------------------------------------------- pooling

def maxpool(x: np.ndarray, k: int = 3, stride: int = 2, pad: int = 1):
    """Max over each k x k window of the -inf padded input.

    Returns (y, arg) where arg[n,p,q,c] = r*k + s of the first maximal element
    of the window in row-major order."""
    n, h, w, c = x.shape
    P, Q = out_size(h, k, stride, pad), out_size(w, k, stride, pad)
    xp = _pad(x, pad, value=-np.inf)
    y = np.full((n, P, Q, c), -np.inf, dtype=np.float64)
    arg = np.zeros((n, P, Q, c), dtype=np.int64)
    for r in range(k):
        for s in range(k):
            v = _window(xp, r, s, stride, P, Q)
            better = v > y
            y = np.where(better, v, y)
            arg = np.where(better, r * k + s, arg)
    return y, arg


def maxpool_backward(dy: np.ndarray, arg: np.ndarray, x_shape, k: int = 3, stride: int = 2,
                     pad: int = 1) -> np.ndarray:
    """Each output gradient goes to the input element its window picked."""
    n, h, w, c = x_shape
    _, P, Q, _ = dy.shape
    dxp = np.zeros((n, h + 2 * pad, w + 2 * pad, c), dtype=np.float64)
    for r in range(k):
        for s in range(k):
            dxp[:, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride, :] += \
                np.where(arg == r * k + s, dy, 0.0)
    return dxp[:, pad:pad + h, pad:pad + w, :]


def avgpool(x: np.ndarray) -> np.ndarray:
    return x.mean(axis=(1, 2))


def avgpool_backward(df: np.ndarray, x_shape) -> np.ndarray:
    n, h, w, c = x_shape
    return np.broadcast_to(df[:, None, None, :] / (h * w), x_shape).copy()


# ---------------------------------------------------------------- classifier

def linear(f: np.ndarray, W: np.ndarray, b: np.ndarray) -> np.ndarray:
    return f @ W.T + b


def linear_backward(dz: np.ndarray, f: np.ndarray, W: np.ndarray):
    """(df, dW, db) for z = f W^T + b."""
    return dz @ W, dz.T @ f, dz.sum(axis=0)


def softmax_cross_entropy(z: np.ndarray, y: np.ndarray):
    """Mean over the batch of logsumexp(z_i) - z_i[y_i].

    Returns (loss, dz, correct) with dz = (softmax(z) - onehot(y)) / B and
    correct = number of rows whose argmax (lowest index on ties) equals y."""
    B = z.shape[0]
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax + np.log(np.exp(z - zmax).sum(axis=1, keepdims=True))
    loss = float(np.mean(lse[:, 0] - z[np.arange(B), y]))
    p = np.exp(z - lse)
    onehot = np.zeros_like(z)
    onehot[np.arange(B), y] = 1.0
    dz = (p - onehot) / B
    correct = int(np.sum(argmax(z) == y))
    return loss, dz, correct


def argmax(z: np.ndarray) -> np.ndarray:
    """Row-wise argmax; the lowest index wins a tie."""
    return np.argmax(z, axis=1)


# ------------------------------------------------------------------ optimiser

def sgd_momentum(w: np.ndarray, v: np.ndarray, g: np.ndarray, lr: float, mu: float):
    """One SGD step with momentum (PyTorch form): v <- mu v + g; w <- w - lr v."""
    v_new = mu * v + g
    return w - lr * v_new, v_new


# ------------------------------------------------------------------- resizing

def _source_coords(n_in: int, n_out: int):
    """Half-pixel source coordinates, clamped at 0, and their two taps."""
    dst = np.arange(n_out, dtype=np.float64)
    src = (dst + 0.5) * (n_in / n_out) - 0.5
    src = np.maximum(src, 0.0)
    i0 = np.minimum(np.floor(src).astype(np.int64), n_in - 1)
    i1 = np.minimum(i0 + 1, n_in - 1)
    return i0, i1, src - i0


def resize_bilinear(x: np.ndarray, out_h: int, out_w: int) -> np.ndarray:
    """Bilinear resize with half-pixel centres (align_corners=False), no antialias."""
    r0, r1, lr_ = _source_coords(x.shape[1], out_h)
    c0, c1, lc = _source_coords(x.shape[2], out_w)
    top = x[:, r0, :, :] * (1.0 - lr_)[None, :, None, None] + x[:, r1, :, :] * lr_[None, :, None, None]
    return top[:, :, c0, :] * (1.0 - lc)[None, None, :, None] + top[:, :, c1, :] * lc[None, None, :, None]
