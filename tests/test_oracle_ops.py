"""Pins for the oracle's layer operations: brute force, closed forms, invariants,
adjoint identities and an independent library (torch CPU, float64)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import nn

RNG = np.random.default_rng(1234)


def brute_conv(x, w, stride, pad):
    n, h, wd, c = x.shape
    k, _, R, S = w.shape
    P = (h + 2 * pad - R) // stride + 1
    Q = (wd + 2 * pad - S) // stride + 1
    y = np.zeros((n, P, Q, k))
    for b in range(n):
        for p in range(P):
            for q in range(Q):
                for o in range(k):
                    acc = 0.0
                    for r in range(R):
                        for s in range(S):
                            hh, ww = stride * p + r - pad, stride * q + s - pad
                            if 0 <= hh < h and 0 <= ww < wd:
                                for ci in range(c):
                                    acc += x[b, hh, ww, ci] * w[o, ci, r, s]
                    y[b, p, q, o] = acc
    return y


CONV_CASES = [
    # (n, h, w, c, k, R, stride, pad)
    (2, 5, 7, 3, 4, 3, 1, 1),
    (1, 7, 5, 2, 3, 3, 2, 1),
    (2, 9, 9, 3, 2, 7, 2, 3),
    (1, 6, 6, 4, 5, 1, 2, 0),
    (1, 4, 4, 3, 2, 3, 1, 0),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_matches_brute_force(case):
    n, h, w, c, k, R, stride, pad = case
    x = RNG.standard_normal((n, h, w, c))
    wt = RNG.standard_normal((k, c, R, R))
    np.testing.assert_allclose(nn.conv2d(x, wt, stride, pad), brute_conv(x, wt, stride, pad),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_adjoint_identities(case):
    n, h, w, c, k, R, stride, pad = case
    x = RNG.standard_normal((n, h, w, c))
    wt = RNG.standard_normal((k, c, R, R))
    y = nn.conv2d(x, wt, stride, pad)
    dy = RNG.standard_normal(y.shape)
    lhs = np.sum(y * dy)
    dx = nn.conv2d_dgrad(dy, wt, x.shape, stride, pad)
    dw = nn.conv2d_wgrad(x, dy, wt.shape, stride, pad)
    assert abs(lhs - np.sum(x * dx)) < 1e-10 * max(1, abs(lhs))
    assert abs(lhs - np.sum(wt * dw)) < 1e-10 * max(1, abs(lhs))


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_and_grads_match_torch(case):
    n, h, w, c, k, R, stride, pad = case
    x = RNG.standard_normal((n, h, w, c))
    wt = RNG.standard_normal((k, c, R, R))
    tx = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    tw = torch.tensor(wt, requires_grad=True)
    ty = F.conv2d(tx, tw, stride=stride, padding=pad)
    dy = RNG.standard_normal(tuple(ty.permute(0, 2, 3, 1).shape))
    ty.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_allclose(nn.conv2d(x, wt, stride, pad), ty.detach().permute(0, 2, 3, 1).numpy(),
                               rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(nn.conv2d_dgrad(dy, wt, x.shape, stride, pad),
                               tx.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(nn.conv2d_wgrad(x, dy, wt.shape, stride, pad), tw.grad.numpy(),
                               rtol=1e-11, atol=1e-11)


def test_conv_1x1_is_matmul_and_delta_kernel_is_shift():
    x = RNG.standard_normal((2, 5, 6, 4))
    w1 = RNG.standard_normal((3, 4, 1, 1))
    np.testing.assert_allclose(nn.conv2d(x, w1, 1, 0), x @ w1[:, :, 0, 0].T, rtol=1e-13)
    # 3x3 kernel with a single 1 at (r, s) = (0, 2) and pad 1: y[p, q] = x[p-1, q+1]
    wd = np.zeros((4, 4, 3, 3))
    for ch in range(4):
        wd[ch, ch, 0, 2] = 1.0
    y = nn.conv2d(x, wd, 1, 1)
    expect = np.zeros_like(x)
    expect[:, 1:, :-1, :] = x[:, :-1, 1:, :]
    np.testing.assert_array_equal(y, expect)


def test_batchnorm_train_normalises():
    z = 3.0 + 2.0 * RNG.standard_normal((4, 5, 5, 6))
    y, (xhat, invstd, mean, var, m) = nn.batchnorm_train(z, np.ones(6), np.zeros(6))
    assert m == 100
    np.testing.assert_allclose(y.mean(axis=(0, 1, 2)), 0.0, atol=1e-12)
    # biased variance of the output is var / (var + eps)
    np.testing.assert_allclose(y.var(axis=(0, 1, 2)), var / (var + nn.BN_EPS), rtol=1e-12)
    g, b = RNG.standard_normal(6), RNG.standard_normal(6)
    y2, _ = nn.batchnorm_train(z, g, b)
    np.testing.assert_allclose(y2, g * y + b, rtol=1e-12, atol=1e-12)


def test_batchnorm_eval_with_unit_stats():
    z = RNG.standard_normal((2, 3, 3, 4))
    y = nn.batchnorm_eval(z, np.ones(4), np.zeros(4), np.zeros(4), np.ones(4))
    np.testing.assert_allclose(y, z / math.sqrt(1.0 + 1e-5), rtol=1e-14)


def test_batchnorm_running_update_matches_torch():
    z = RNG.standard_normal((4, 3, 5, 6)) * 2 + 1
    _, (_, _, mean, var, m) = nn.batchnorm_train(z, np.ones(6), np.zeros(6))
    rm0, rv0 = RNG.standard_normal(6), 1 + RNG.random(6)
    rm, rv = nn.batchnorm_running_update(rm0, rv0, mean, var, m)
    bn = torch.nn.BatchNorm2d(6, dtype=torch.float64)
    bn.running_mean.copy_(torch.tensor(rm0))
    bn.running_var.copy_(torch.tensor(rv0))
    bn.train()
    bn(torch.tensor(z.transpose(0, 3, 1, 2)))
    np.testing.assert_allclose(rm, bn.running_mean.numpy(), rtol=1e-13)
    np.testing.assert_allclose(rv, bn.running_var.numpy(), rtol=1e-13)


def test_batchnorm_backward_invariants_and_fd():
    z = RNG.standard_normal((3, 4, 4, 5)) * 1.5 + 0.5
    g, b = 1 + RNG.random(5), RNG.standard_normal(5)
    y, saved = nn.batchnorm_train(z, g, b)
    dy = RNG.standard_normal(y.shape)
    dz, dg, db = nn.batchnorm_backward(dy, saved, g)
    xhat, invstd, _, var, _ = saved
    np.testing.assert_allclose(dz.sum(axis=(0, 1, 2)), 0.0, atol=1e-11)
    # sum(xhat^2) = m * var / (var + eps), so sum(dz * xhat) is an eps-sized
    # multiple of dgamma rather than exactly zero
    np.testing.assert_allclose((dz * xhat).sum(axis=(0, 1, 2)),
                               g * invstd * dg * nn.BN_EPS / (var + nn.BN_EPS), rtol=1e-6, atol=1e-14)
    np.testing.assert_allclose(db, dy.sum(axis=(0, 1, 2)), rtol=1e-13)
    # constant upstream gradient: the input gradient vanishes
    dz_c, _, _ = nn.batchnorm_backward(np.ones_like(y) * 0.7, saved, g)
    np.testing.assert_allclose(dz_c, 0.0, atol=1e-12)
    # central finite differences of L = sum(y * dy)
    h = 1e-6
    for idx in [(0, 0, 0, 0), (1, 2, 3, 4), (2, 3, 1, 2)]:
        zp, zm = z.copy(), z.copy()
        zp[idx] += h
        zm[idx] -= h
        fd = (np.sum(nn.batchnorm_train(zp, g, b)[0] * dy) - np.sum(nn.batchnorm_train(zm, g, b)[0] * dy)) / (2 * h)
        assert abs(fd - dz[idx]) < 1e-6 * max(1.0, abs(fd))
    for c in range(5):
        gp, gm = g.copy(), g.copy()
        gp[c] += h
        gm[c] -= h
        fd = (np.sum(nn.batchnorm_train(z, gp, b)[0] * dy) - np.sum(nn.batchnorm_train(z, gm, b)[0] * dy)) / (2 * h)
        assert abs(fd - dg[c]) < 1e-6 * max(1.0, abs(fd))


def test_batchnorm_backward_matches_torch():
    z = RNG.standard_normal((2, 5, 3, 4)) + 0.3
    g, b = 1 + RNG.random(4), RNG.standard_normal(4)
    y, saved = nn.batchnorm_train(z, g, b)
    dy = RNG.standard_normal(y.shape)
    dz, dg, db = nn.batchnorm_backward(dy, saved, g)
    tz = torch.tensor(z.transpose(0, 3, 1, 2), requires_grad=True)
    tg = torch.tensor(g, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    ty = F.batch_norm(tz, None, None, tg, tb, training=True, eps=1e-5)
    ty.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_allclose(y, ty.detach().permute(0, 2, 3, 1).numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dz, tz.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-12)


def brute_maxpool(x):
    n, h, w, c = x.shape
    P, Q = (h + 2 - 3) // 2 + 1, (w + 2 - 3) // 2 + 1
    y = np.zeros((n, P, Q, c))
    arg = np.zeros((n, P, Q, c), dtype=int)
    for b in range(n):
        for p in range(P):
            for q in range(Q):
                for ch in range(c):
                    best, barg = -np.inf, -1
                    for r in range(3):
                        for s in range(3):
                            hh, ww = 2 * p + r - 1, 2 * q + s - 1
                            if 0 <= hh < h and 0 <= ww < w and x[b, hh, ww, ch] > best:
                                best, barg = x[b, hh, ww, ch], r * 3 + s
                    y[b, p, q, ch], arg[b, p, q, ch] = best, barg
    return y, arg


def test_maxpool_brute_force_with_ties():
    x = RNG.integers(-2, 3, size=(2, 7, 6, 3)).astype(np.float64)  # many ties
    y, arg = nn.maxpool(x)
    yb, argb = brute_maxpool(x)
    np.testing.assert_array_equal(y, yb)
    np.testing.assert_array_equal(arg, argb)
    dy = RNG.standard_normal(y.shape)
    dx = nn.maxpool_backward(dy, arg, x.shape)
    # brute-force routing
    dxb = np.zeros_like(x)
    for b, p, q, ch in np.ndindex(*y.shape):
        r, s = divmod(argb[b, p, q, ch], 3)
        dxb[b, 2 * p + r - 1, 2 * q + s - 1, ch] += dy[b, p, q, ch]
    np.testing.assert_allclose(dx, dxb, rtol=1e-14)


def test_maxpool_matches_torch_without_ties():
    x = RNG.standard_normal((2, 9, 8, 3))
    y, arg = nn.maxpool(x)
    tx = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    ty = F.max_pool2d(tx, 3, 2, 1)
    dy = RNG.standard_normal(y.shape)
    ty.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_array_equal(y, ty.detach().permute(0, 2, 3, 1).numpy())
    np.testing.assert_allclose(nn.maxpool_backward(dy, arg, x.shape), tx.grad.permute(0, 2, 3, 1).numpy(),
                               rtol=1e-14)


def test_avgpool_and_backward():
    x = RNG.standard_normal((2, 3, 5, 4))
    f = nn.avgpool(x)
    np.testing.assert_allclose(f, x.sum(axis=(1, 2)) / 15, rtol=1e-14)
    df = RNG.standard_normal(f.shape)
    dx = nn.avgpool_backward(df, x.shape)
    assert abs(np.sum(dx * x) - np.sum(df * f)) < 1e-12  # adjoint


def test_softmax_ce_closed_forms():
    z = np.zeros((5, 6))
    y = np.array([0, 1, 2, 3, 5])
    loss, dz, correct = nn.softmax_cross_entropy(z, y)
    assert abs(loss - math.log(6.0)) < 1e-15
    assert abs(math.log(6.0) - 1.791759469228055) < 1e-15
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-16)
    assert correct == 1  # all ties -> argmax 0, only the label-0 row is right
    z = RNG.standard_normal((7, 6)) * 3
    y = RNG.integers(0, 6, 7)
    l1, d1, _ = nn.softmax_cross_entropy(z, y)
    l2, d2, _ = nn.softmax_cross_entropy(z + 100.0, y)  # shift invariance
    assert abs(l1 - l2) < 1e-12
    np.testing.assert_allclose(d1, d2, atol=1e-14)
    tz = torch.tensor(z, requires_grad=True)
    tl = F.cross_entropy(tz, torch.tensor(y))
    tl.backward()
    assert abs(l1 - tl.item()) < 1e-13
    np.testing.assert_allclose(d1, tz.grad.numpy(), atol=1e-15)


def test_linear_backward_matches_fd():
    f = RNG.standard_normal((4, 5))
    W = RNG.standard_normal((3, 5))
    b = RNG.standard_normal(3)
    dz = RNG.standard_normal((4, 3))
    df, dW, db = nn.linear_backward(dz, f, W)
    h = 1e-6
    Wp, Wm = W.copy(), W.copy()
    Wp[1, 2] += h
    Wm[1, 2] -= h
    fd = (np.sum(nn.linear(f, Wp, b) * dz) - np.sum(nn.linear(f, Wm, b) * dz)) / (2 * h)
    assert abs(fd - dW[1, 2]) < 1e-8
    np.testing.assert_allclose(db, dz.sum(0))
    fp, fm = f.copy(), f.copy()
    fp[2, 4] += h
    fm[2, 4] -= h
    fd = (np.sum(nn.linear(fp, W, b) * dz) - np.sum(nn.linear(fm, W, b) * dz)) / (2 * h)
    assert abs(fd - df[2, 4]) < 1e-8


def test_sgd_two_step_closed_form_and_torch():
    w0 = RNG.standard_normal(10)
    g0, g1 = RNG.standard_normal(10), RNG.standard_normal(10)
    lr, mu = 0.01, 0.9
    w1, v1 = nn.sgd_momentum(w0, np.zeros(10), g0, lr, mu)
    w2, _ = nn.sgd_momentum(w1, v1, g1, lr, mu)
    np.testing.assert_allclose(w2, w0 - lr * g0 - lr * (mu * g0 + g1), rtol=1e-14)
    tw = torch.tensor(w0, requires_grad=True)
    opt = torch.optim.SGD([tw], lr=lr, momentum=mu)
    for g in (g0, g1):
        tw.grad = torch.tensor(g)
        opt.step()
    np.testing.assert_allclose(w2, tw.detach().numpy(), rtol=1e-14)


@pytest.mark.parametrize("shape,out", [((2, 224, 224, 3), 160), ((1, 224, 224, 3), 112),
                                       ((1, 10, 13, 2), 7), ((1, 5, 5, 1), 12)])
def test_resize_matches_torch_bilinear(shape, out):
    x = RNG.standard_normal(shape)
    y = nn.resize_bilinear(x, out, out)
    ty = F.interpolate(torch.tensor(x.transpose(0, 3, 1, 2)), size=(out, out), mode="bilinear",
                       align_corners=False, antialias=False)
    np.testing.assert_allclose(y, ty.permute(0, 2, 3, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_resize_identity_and_half():
    x = RNG.standard_normal((1, 8, 8, 2))
    np.testing.assert_allclose(nn.resize_bilinear(x, 8, 8), x, rtol=0, atol=0)
    # exact 2x downsample with half-pixel centres = mean of each 2x2 block
    y = nn.resize_bilinear(x, 4, 4)
    blocks = x.reshape(1, 4, 2, 4, 2, 2).mean(axis=(2, 4))
    np.testing.assert_allclose(y, blocks, rtol=1e-14)


def test_argmax_lowest_index_on_ties():
    z = np.array([[1.0, 3.0, 3.0], [2.0, 2.0, 2.0], [0.0, -1.0, 5.0]])
    np.testing.assert_array_equal(nn.argmax(z), [1, 0, 2])
