"""Kernel-by-kernel parity of the HIP library (through the C ABI) against the
CPU oracle, at ResNet18's layer shapes plus ragged ones that leave partial
tiles.  fp32 instantiations: per-tensor max relative error <= 1e-4; bf16:
<= 2e-2 (inputs rounded to bf16 identically on both sides)."""
import numpy as np
import pytest

from oracle import nn
from tests.gpu_util import TOL, as_np, rel_err, rounded, to_dev

pytestmark = pytest.mark.gpu

PRECS = ["f32", "bf16"]

# (N, H, W, C, K, R, stride, pad): every conv shape family of ResNet18 at
# reduced spatial size, plus odd sizes spanning several tiles with ragged tails
CONV_CASES = [
    (2, 64, 64, 3, 64, 7, 2, 3),      # stem
    (1, 37, 41, 3, 64, 7, 2, 3),      # stem, odd size
    (1, 224, 224, 3, 64, 7, 2, 3),    # stem at full width (112 output columns)
    (2, 16, 16, 64, 64, 3, 1, 1),     # layer1
    (3, 13, 11, 64, 64, 3, 1, 1),     # layer1, ragged
    (2, 16, 16, 64, 128, 3, 2, 1),    # layer2.0.conv1
    (2, 16, 16, 64, 128, 1, 2, 0),    # layer2.0.downsample
    (2, 8, 8, 128, 128, 3, 1, 1),     # layer2
    (2, 9, 9, 128, 256, 3, 2, 1),     # layer3.0.conv1, odd
    (2, 14, 14, 256, 512, 3, 2, 1),   # layer4.0.conv1
    (2, 14, 14, 256, 512, 1, 2, 0),   # layer4.0.downsample
    (2, 7, 7, 512, 512, 3, 1, 1),     # layer4
    (4, 56, 56, 64, 64, 3, 1, 1),     # layer1 at 224 px, many tiles
    (44, 14, 14, 256, 256, 3, 1, 1),  # layer3, 68 pixel tiles (ragged), split reductions,
                                      # 135 weight-gradient pixel stages
    (168, 14, 14, 256, 512, 3, 2, 1), # layer4.0.conv1, strided, 129 weight-gradient pixel stages
    (22, 56, 56, 64, 64, 3, 1, 1),    # layer1, 270 tiles of 64 x 256 (ragged)
    (84, 28, 28, 128, 128, 3, 1, 1),  # layer2, 258 tiles of 128 x 256 (ragged)
    # frozen-prefix shapes at cache-build batch sizes: more tiles than CUs
    (48, 56, 56, 64, 64, 3, 1, 1),    # layer1, 588 tiles of 64 x 256
    (60, 20, 20, 64, 64, 3, 1, 1),    # 64 -> 64: two 8 x 8 patches per block, ragged patches
    (168, 28, 28, 128, 128, 3, 1, 1), # layer2, 515 tiles of 128 x 256
    (336, 14, 14, 256, 256, 3, 1, 1), # layer3, 515 tiles of 256 x 128 (ragged)
]


def _rng(seed):
    return np.random.default_rng(seed)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_forward(prec, case):
    N, H, W, C, K, R, st, pad = case
    rs = _rng(hash(case) % 1000)
    x = rounded(rs.standard_normal((N, H, W, C)), prec)
    w = rs.standard_normal((K, C, R, R)).astype(np.float32) * np.sqrt(2.0 / (C * R * R))
    from paper_2012_10557_amd import binding
    y = binding.ekya_op_conv2d(to_dev(x, prec), to_dev(w), st, pad)
    ref = nn.conv2d(x, rounded(w, prec), st, pad)
    assert rel_err(as_np(y), ref) <= TOL[prec]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", [c for c in CONV_CASES if c[3] != 3], ids=lambda c: "x".join(map(str, c)))
def test_conv_dgrad(prec, case):
    N, H, W, C, K, R, st, pad = case
    rs = _rng(hash(case) % 1000 + 1)
    w = rs.standard_normal((K, C, R, R)).astype(np.float32) * np.sqrt(2.0 / (K * R * R))
    P, Q = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    dy = rounded(rs.standard_normal((N, P, Q, K)), prec)
    from paper_2012_10557_amd import binding
    dx = binding.ekya_op_conv2d_dgrad(to_dev(dy, prec), to_dev(w), (N, H, W, C), st, pad)
    ref = nn.conv2d_dgrad(dy, rounded(w, prec), (N, H, W, C), st, pad)
    assert rel_err(as_np(dx), ref) <= TOL[prec]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_wgrad(prec, case):
    N, H, W, C, K, R, st, pad = case
    rs = _rng(hash(case) % 1000 + 2)
    x = rounded(rs.standard_normal((N, H, W, C)), prec)
    P, Q = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    dy = rounded(rs.standard_normal((N, P, Q, K)), prec)
    from paper_2012_10557_amd import binding
    dw = binding.ekya_op_conv2d_wgrad(to_dev(x, prec), to_dev(dy, prec), (K, C, R, R), st, pad)
    ref = nn.conv2d_wgrad(x, dy, (K, C, R, R), st, pad)
    assert rel_err(as_np(dw), ref) <= TOL[prec]


def test_wgrad_is_deterministic():
    from paper_2012_10557_amd import binding
    rs = _rng(5)
    x = to_dev(rs.standard_normal((8, 28, 28, 128)), "bf16")
    dy = to_dev(rs.standard_normal((8, 28, 28, 128)), "bf16")
    a = binding.ekya_op_conv2d_wgrad(x, dy, (128, 128, 3, 3), 1, 1)
    b = binding.ekya_op_conv2d_wgrad(x, dy, (128, 128, 3, 3), 1, 1)
    assert bool((a == b).all())


BN_CASES = [(2 * 7 * 7, 512), (3 * 5 * 5, 64), (64 * 14 * 14, 256), (1000, 128), (1, 64)]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("M,C", BN_CASES)
@pytest.mark.parametrize("relu", [False, True])
def test_batchnorm_train_forward(prec, M, C, relu):
    import torch
    rs = _rng(M + C)
    z = rounded(1.5 * rs.standard_normal((M, C)) + rs.standard_normal(C), prec)
    g = (1 + 0.2 * rs.standard_normal(C)).astype(np.float32)
    b = (0.1 * rs.standard_normal(C)).astype(np.float32)
    rm0 = (0.1 * rs.standard_normal(C)).astype(np.float32)
    rv0 = (1 + rs.random(C)).astype(np.float32)
    from paper_2012_10557_amd import binding
    rm, rv = to_dev(rm0), to_dev(rv0)
    y, mean, invstd = binding.ekya_op_batchnorm_train(to_dev(z, prec), to_dev(g), to_dev(b), rm, rv,
                                                      relu=relu)
    yr, (xhat, istd, mu, var, m) = nn.batchnorm_train(z.reshape(M, 1, 1, C), g.astype(np.float64),
                                                      b.astype(np.float64))
    if relu:
        yr = nn.relu(yr)
    assert rel_err(as_np(y), yr.reshape(M, C)) <= TOL[prec]
    assert rel_err(as_np(mean), mu) <= 1e-4
    if M > 1:
        assert rel_err(as_np(invstd), istd) <= 1e-4
        erm, erv = nn.batchnorm_running_update(rm0.astype(np.float64), rv0.astype(np.float64), mu, var, m)
        assert rel_err(as_np(rm), erm) <= 1e-4
        assert rel_err(as_np(rv), erv) <= 1e-4
    torch.cuda.synchronize()


@pytest.mark.parametrize("M", [3136, 64 * 7 * 7 + 5])
def test_batchnorm_large_mean_small_spread(M):
    """Mean 2000x the standard deviation, fp32, a ragged last chunk: the
    chunk statistics must be combined without cancellation (the variance
    from sums of squares would lose every digit here)."""
    import torch
    C = 128
    rs = _rng(M + 7)
    z = rounded(40.0 + 0.02 * rs.standard_normal((M, C)), "f32")
    g = np.ones(C, np.float32)
    b = np.zeros(C, np.float32)
    from paper_2012_10557_amd import binding
    rm, rv = to_dev(np.zeros(C, np.float32)), to_dev(np.ones(C, np.float32))
    y, mean, invstd = binding.ekya_op_batchnorm_train(to_dev(z, "f32"), to_dev(g), to_dev(b), rm, rv,
                                                      relu=False)
    yr, (xhat, istd, mu, var, m) = nn.batchnorm_train(z.reshape(M, 1, 1, C), g.astype(np.float64),
                                                      b.astype(np.float64))
    assert rel_err(as_np(mean), mu) <= 1e-6
    assert rel_err(as_np(invstd), istd) <= 1e-3
    assert rel_err(as_np(y), yr.reshape(M, C)) <= 1e-3
    torch.cuda.synchronize()


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("M,C", BN_CASES[:4])
@pytest.mark.parametrize("mask", [False, True])
def test_batchnorm_backward(prec, M, C, mask):
    rs = _rng(M * 3 + C)
    z = rounded(1.5 * rs.standard_normal((M, C)) + 0.3, prec)
    dy = rounded(rs.standard_normal((M, C)), prec)
    y_mask = rounded(rs.standard_normal((M, C)), prec) if mask else None
    g = (1 + 0.2 * rs.standard_normal(C)).astype(np.float32)
    _, saved = nn.batchnorm_train(z.reshape(M, 1, 1, C), g.astype(np.float64), np.zeros(C))
    xhat, istd, mu, var, m = saved
    from paper_2012_10557_amd import binding
    dz, dg, db = binding.ekya_op_batchnorm_backward(
        to_dev(dy, prec), to_dev(y_mask, prec) if mask else None, to_dev(z, prec), to_dev(g),
        to_dev(mu.astype(np.float32)), to_dev(istd.astype(np.float32)))
    gg = dy if not mask else nn.relu_backward(dy, y_mask)
    rdz, rdg, rdb = nn.batchnorm_backward(gg.reshape(M, 1, 1, C), saved, g.astype(np.float64))
    assert rel_err(as_np(dz), rdz.reshape(M, C)) <= TOL[prec]
    assert rel_err(as_np(dg), rdg) <= 1e-4 if prec == "f32" else TOL[prec]
    assert rel_err(as_np(db), rdb) <= 1e-4 if prec == "f32" else TOL[prec]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("shape", [(2, 112, 112, 64), (3, 15, 9, 64), (1, 32, 32, 64)])
def test_maxpool_forward_backward(prec, shape):
    rs = _rng(sum(shape))
    x = rounded(rs.standard_normal(shape), prec)
    from paper_2012_10557_amd import binding
    y, arg = binding.ekya_op_maxpool(to_dev(x, prec))
    ry, rarg = nn.maxpool(x)
    np.testing.assert_array_equal(as_np(y), ry)          # max is exact
    np.testing.assert_array_equal(arg.cpu().numpy(), rarg)  # same tie rule on identical values
    dy = rounded(rs.standard_normal(ry.shape), prec)
    dx = binding.ekya_op_maxpool_backward(to_dev(dy, prec), arg, shape)
    rdx = nn.maxpool_backward(dy, rarg, shape)
    assert rel_err(as_np(dx), rdx) <= TOL[prec]


def test_maxpool_ties_pick_first_in_window():
    # integer-valued input: many exact ties
    rs = _rng(3)
    x = rs.integers(-2, 3, size=(2, 9, 10, 64)).astype(np.float64)
    from paper_2012_10557_amd import binding
    _, arg = binding.ekya_op_maxpool(to_dev(x, "bf16"))
    _, rarg = nn.maxpool(x)
    np.testing.assert_array_equal(arg.cpu().numpy(), rarg)


@pytest.mark.parametrize("prec", PRECS)
def test_avgpool_forward_backward(prec):
    rs = _rng(11)
    x = rounded(rs.standard_normal((5, 7, 7, 512)), prec)
    from paper_2012_10557_amd import binding
    f = binding.ekya_op_avgpool(to_dev(x, prec))
    assert rel_err(as_np(f), nn.avgpool(x)) <= 1e-4 if prec == "f32" else TOL[prec]
    df = rs.standard_normal((5, 512)).astype(np.float32)
    import torch
    dx = binding.ekya_op_avgpool_backward(to_dev(df), (5, 7, 7, 512),
                                          torch.float32 if prec == "f32" else torch.bfloat16)
    assert rel_err(as_np(dx), nn.avgpool_backward(df.astype(np.float64), x.shape)) <= TOL[prec]


def test_linear_softmax_ce_and_sgd():
    rs = _rng(12)
    N, I, J = 37, 512, 6
    f = rs.standard_normal((N, I)).astype(np.float32)
    W = (0.05 * rs.standard_normal((J, I))).astype(np.float32)
    b = (0.1 * rs.standard_normal(J)).astype(np.float32)
    y = rs.integers(0, J, N).astype(np.int32)
    from paper_2012_10557_amd import binding
    import torch
    z = binding.ekya_op_linear(to_dev(f), to_dev(W), to_dev(b))
    rz = nn.linear(f.astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    assert rel_err(as_np(z), rz) <= 1e-5
    out, dz = binding.ekya_op_softmax_ce(z, torch.tensor(y, device="cuda"))
    loss, rdz, correct = nn.softmax_cross_entropy(rz, y)
    o = out.cpu().numpy()
    assert abs(o[0] - loss) <= 1e-5 * max(1, abs(loss))
    assert int(o[1]) == correct and o[2] == 0
    assert rel_err(as_np(dz), rdz) <= 1e-5
    df, dW, db = binding.ekya_op_linear_backward(dz, to_dev(f), to_dev(W))
    rdf, rdW, rdb = nn.linear_backward(rdz, f.astype(np.float64), W.astype(np.float64))
    assert rel_err(as_np(dW), rdW) <= 1e-4 and rel_err(as_np(db), rdb) <= 1e-4
    assert rel_err(as_np(df), rdf) <= 1e-4
    w0 = rs.standard_normal(1001).astype(np.float32)
    v0 = rs.standard_normal(1001).astype(np.float32)
    g0 = rs.standard_normal(1001).astype(np.float32)
    w, v = to_dev(w0), to_dev(v0)
    binding.ekya_op_sgd(w, v, to_dev(g0), 0.01, 0.9)
    rw, rv = nn.sgd_momentum(w0.astype(np.float64), v0.astype(np.float64), g0.astype(np.float64), 0.01, 0.9)
    assert rel_err(as_np(w), rw) <= 1e-6 and rel_err(as_np(v), rv) <= 1e-6


def test_softmax_ce_equal_logits_is_ln_classes():
    import math
    import torch
    from paper_2012_10557_amd import binding
    z = torch.zeros(9, 6, device="cuda")
    out, dz = binding.ekya_op_softmax_ce(z, torch.arange(9, dtype=torch.int32, device="cuda") % 6)
    assert abs(out[0].item() - math.log(6)) < 1e-6
    assert abs(dz.sum(dim=1)).max().item() < 1e-7


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("r", [160, 112, 224, 57])
def test_resize(prec, r):
    rs = _rng(r)
    x = rounded(rs.standard_normal((2, 224, 224, 3)), prec)
    from paper_2012_10557_amd import binding
    y = binding.ekya_op_resize(to_dev(x, prec), r)
    assert rel_err(as_np(y), nn.resize_bilinear(x, r, r)) <= TOL[prec]
