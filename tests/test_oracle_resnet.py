"""Pins for the oracle's network and retraining loop: finite differences on a tiny
ResNet, an independent torch (CPU, float64) ResNet18 built from torch.nn
modules, and the special cases the method fixes (cache reuse is exact, frozen
stages do not move, a separable task is learned)."""
import math

import numpy as np
import pytest
import torch
import torch.nn as tnn
import torch.nn.functional as F

from oracle import ekya, nn, rng
from oracle.resnet18 import ResNet18, STAGES
from synth import WindowSpec, kaiming_resnet18_weights, make_window, resnet18_param_spec

TINY = dict(n_classes=3, widths=(4, 8, 8, 8), blocks=(1, 1, 1, 1))


def _tiny_weights(seed, hidden=0):
    rs = np.random.default_rng(seed)
    net = ResNet18(**TINY, hidden=hidden)
    flat = kaiming_resnet18_weights(seed, **TINY, hidden=hidden).astype(np.float64)
    P = net.unpack(flat)
    for name in P:  # non-trivial BN parameters and statistics
        if name.endswith(".weight") and P[name].ndim == 1:
            P[name] = 1 + 0.2 * rs.standard_normal(P[name].shape)
        elif name.endswith(".bias") and not name.startswith("fc"):
            P[name] = 0.1 * rs.standard_normal(P[name].shape)
        elif name.endswith("running_mean"):
            P[name] = 0.1 * rs.standard_normal(P[name].shape)
        elif name.endswith("running_var"):
            P[name] = 1 + 0.3 * rs.random(P[name].shape)
    return net, P


def _loss(net, P, x_prefix, labels, lowest):
    Q = {k: v.copy() for k, v in P.items()}
    logits = net.forward(Q, x_prefix, lowest, 5, train=True, tape={})
    return nn.softmax_cross_entropy(logits, labels)[0]


@pytest.mark.parametrize("hidden", [64, 1024])
def test_hidden_head_spec(hidden):
    """A hidden layer of h neurons replaces fc (512 * 6 + 6 parameters) by
    fc.0 (512 h + h) and fc.2 (6 h + 6), in torch nn.Sequential's names."""
    net = ResNet18(6, hidden=hidden)
    gen = resnet18_param_spec(6, hidden=hidden)
    assert [(n, tuple(s)) for n, s, _ in gen] == net.spec
    assert net.n_weights() == 11_189_190 - 512 * 6 - 6 + 512 * hidden + hidden + 6 * hidden + 6
    assert [n for n, _ in net.spec[-4:]] == ["fc.0.weight", "fc.0.bias", "fc.2.weight", "fc.2.bias"]
    assert all(net.stage_of[n] == 5 for n, _ in net.spec[-4:])
    w = kaiming_resnet18_weights(0, hidden=hidden)
    P = net.unpack(w)
    # torch.nn.Linear's default bounds, 1/sqrt(fan_in)
    assert np.abs(P["fc.0.weight"]).max() <= 1 / math.sqrt(512)
    assert np.abs(P["fc.2.weight"]).max() <= 1 / math.sqrt(hidden)
    assert np.abs(P["fc.2.weight"]).max() > 0.9 / math.sqrt(hidden)


def test_identity_hidden_layer_reduces_to_the_plain_classifier():
    """Pooled features are non-negative (they average ReLU outputs), so a
    hidden layer of 512 neurons with identity weights and zero bias passes
    them through unchanged: logits, loss and the output layer's gradient equal
    the plain classifier's with the same output weights, and the hidden
    layer's weight gradient is the outer product of the data gradient with
    the features."""
    rs = np.random.default_rng(3)
    f = np.maximum(rs.standard_normal((5, 512)), 0.0)
    labels = np.array([0, 3, 5, 1, 1])
    plain, mlp = ResNet18(6), ResNet18(6, hidden=512)
    W, b = 0.05 * rs.standard_normal((6, 512)), 0.1 * rs.standard_normal(6)
    P0 = {"fc.weight": W, "fc.bias": b}
    P1 = {"fc.0.weight": np.eye(512), "fc.0.bias": np.zeros(512), "fc.2.weight": W, "fc.2.bias": b}
    t0, t1 = {}, {}
    z0 = plain.stage_forward(P0, 5, f, True, t0)
    z1 = mlp.stage_forward(P1, 5, f, True, t1)
    np.testing.assert_array_equal(z0, z1)
    _, dz, _ = nn.softmax_cross_entropy(z0, labels)
    g0, g1 = plain.backward(P0, dz, 5, t0), mlp.backward(P1, dz, 5, t1)
    np.testing.assert_allclose(g1["fc.2.weight"], g0["fc.weight"], rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(g1["fc.2.bias"], g0["fc.bias"], rtol=1e-13, atol=1e-16)
    da = (dz @ W) * (f > 0)
    np.testing.assert_allclose(g1["fc.0.weight"], da.T @ f, rtol=1e-12, atol=1e-15)


def test_hidden_head_matches_torch_sequential():
    """An independent torch float64 head, nn.Sequential(Linear, ReLU, Linear),
    on pooled features: logits and every gradient."""
    rs = np.random.default_rng(4)
    f = np.maximum(rs.standard_normal((7, 512)), 0.0)
    labels = np.array([0, 1, 2, 3, 4, 5, 0])
    h = 96
    net = ResNet18(6, hidden=h)
    P = net.unpack(kaiming_resnet18_weights(2, hidden=h).astype(np.float64))
    tape = {}
    z = net.stage_forward(P, 5, f, True, tape)
    _, dz, _ = nn.softmax_cross_entropy(z, labels)
    g = net.backward(P, dz, 5, tape)
    head = tnn.Sequential(tnn.Linear(512, h), tnn.ReLU(), tnn.Linear(h, 6)).double()
    with torch.no_grad():
        head[0].weight.copy_(torch.tensor(P["fc.0.weight"]))
        head[0].bias.copy_(torch.tensor(P["fc.0.bias"]))
        head[2].weight.copy_(torch.tensor(P["fc.2.weight"]))
        head[2].bias.copy_(torch.tensor(P["fc.2.bias"]))
    zt = head(torch.tensor(f))
    F.cross_entropy(zt, torch.tensor(labels, dtype=torch.long)).backward()
    np.testing.assert_allclose(z, zt.detach().numpy(), rtol=1e-12, atol=1e-14)
    for name, t in [("fc.0.weight", head[0].weight), ("fc.0.bias", head[0].bias),
                    ("fc.2.weight", head[2].weight), ("fc.2.bias", head[2].bias)]:
        np.testing.assert_allclose(g[name], t.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_param_spec_agrees_with_generator():
    net = ResNet18(6)
    gen = resnet18_param_spec(6)
    assert [(n, tuple(s)) for n, s, _ in gen] == net.spec
    assert net.n_weights() == 11_189_190
    trainable_all = sum(int(np.prod(s)) for n, s in net.spec if not ResNet18.is_running_stat(n))
    assert trainable_all == 11_179_590


@pytest.mark.parametrize("k,hidden", [(1, 0), (2, 0), (3, 0), (6, 0), (1, 5), (2, 5), (6, 5)])
def test_tiny_resnet_gradients_match_finite_differences(k, hidden):
    net, P = _tiny_weights(7, hidden)
    rs = np.random.default_rng(11)
    x = rs.standard_normal((4, 16, 16, 3))
    labels = np.array([0, 1, 2, 1])
    lowest = len(STAGES) - k
    xp = ekya.prefix_forward(net, P, x, lowest)
    Q = {kk: v.copy() for kk, v in P.items()}
    tape = {}
    logits = net.forward(Q, xp, lowest, 5, train=True, tape=tape)
    _, dz, _ = nn.softmax_cross_entropy(logits, labels)
    grads = net.backward(Q, dz, lowest, tape)
    names = net.trainable_names(k)
    assert set(grads) == set(names)
    h = 1e-6
    checked = 0
    for name in names:
        flat = P[name].reshape(-1)
        for i in rs.choice(flat.size, size=min(3, flat.size), replace=False):
            orig = flat[i]
            flat[i] = orig + h
            lp = _loss(net, P, xp, labels, lowest)
            flat[i] = orig - h
            lm = _loss(net, P, xp, labels, lowest)
            flat[i] = orig
            fd = (lp - lm) / (2 * h)
            g = grads[name].reshape(-1)[i]
            assert abs(fd - g) <= 1e-6 * max(abs(fd), 1e-3), (name, i, fd, g)
            checked += 1
    assert checked >= len(names)


# ------------------------------------------------------ independent torch model

class _Block(tnn.Module):
    def __init__(self, cin, cout, stride):
        super().__init__()
        self.conv1 = tnn.Conv2d(cin, cout, 3, stride, 1, bias=False)
        self.bn1 = tnn.BatchNorm2d(cout)
        self.conv2 = tnn.Conv2d(cout, cout, 3, 1, 1, bias=False)
        self.bn2 = tnn.BatchNorm2d(cout)
        self.downsample = None
        if stride != 1 or cin != cout:
            self.downsample = tnn.Sequential(tnn.Conv2d(cin, cout, 1, stride, bias=False),
                                             tnn.BatchNorm2d(cout))

    def forward(self, x):
        y = F.relu(self.bn1(self.conv1(x)))
        y = self.bn2(self.conv2(y))
        return F.relu(y + (x if self.downsample is None else self.downsample(x)))


class _TorchResNet18(tnn.Module):
    def __init__(self, n_classes, widths=(64, 128, 256, 512), hidden=0):
        super().__init__()
        self.conv1 = tnn.Conv2d(3, widths[0], 7, 2, 3, bias=False)
        self.bn1 = tnn.BatchNorm2d(widths[0])
        cin = widths[0]
        for i, w in enumerate(widths):
            s = 1 if i == 0 else 2
            setattr(self, f"layer{i + 1}", tnn.Sequential(_Block(cin, w, s), _Block(w, w, 1)))
            cin = w
        if hidden:
            self.fc = tnn.Sequential(tnn.Linear(widths[-1], hidden), tnn.ReLU(),
                                     tnn.Linear(hidden, n_classes))
        else:
            self.fc = tnn.Linear(widths[-1], n_classes)

    def forward(self, x):
        x = F.max_pool2d(F.relu(self.bn1(self.conv1(x))), 3, 2, 1)
        for i in range(4):
            x = getattr(self, f"layer{i + 1}")(x)
        return self.fc(x.mean(dim=(2, 3)))


def _torch_model(flat, n_classes=6, hidden=0):
    m = _TorchResNet18(n_classes, hidden=hidden).double()
    sd = m.state_dict()
    names = [n for n in sd if not n.endswith("num_batches_tracked")]
    off = 0
    new = {}
    for n in names:
        cnt = sd[n].numel()
        new[n] = torch.tensor(np.asarray(flat[off:off + cnt], dtype=np.float64)).reshape(sd[n].shape)
        off += cnt
    assert off == flat.size
    m.load_state_dict(new, strict=False)
    return m, names


def test_whole_resnet18_matches_torch_eval_and_train_step():
    flat = kaiming_resnet18_weights(0).astype(np.float64)
    win = make_window(WindowSpec(4, 1, 64, 64, drift="shift", seed=5))
    x, y = win["frames"].astype(np.float64), win["labels"]
    net = ResNet18(6)
    # eval forward
    m, names = _torch_model(flat)
    m.eval()
    logits_t = m(torch.tensor(x.transpose(0, 3, 1, 2))).detach().numpy()
    np.testing.assert_allclose(ekya.infer_logits(flat, x, 64), logits_t, rtol=1e-9, atol=1e-10)
    # one retraining step of every stage (k = 6), train-mode BN, SGD momentum
    lr, mu = 0.05, 0.9
    res = ekya.retrain(flat.astype(np.float32), 6, x, y, x[:1], y[:1], 1.0, 1, lr, mu, batch=4,
                       seed=3)
    order = rng.epoch_order(4, 3, 0)
    S = rng.training_subset(4, 1.0, 3)
    xb = x[S][order]
    yb = y[S][order]
    m, names = _torch_model(flat.astype(np.float32).astype(np.float64))
    m.train()
    opt = torch.optim.SGD(m.parameters(), lr=lr, momentum=mu)
    loss = F.cross_entropy(m(torch.tensor(xb.transpose(0, 3, 1, 2))), torch.tensor(yb, dtype=torch.long))
    loss.backward()
    opt.step()
    assert abs(loss.item() - res.losses[0]) < 1e-10
    sd = m.state_dict()
    expect = np.concatenate([sd[n].numpy().reshape(-1) for n in names])
    np.testing.assert_allclose(res.weights, expect, rtol=1e-8, atol=1e-10)


def test_cache_reuse_is_bitwise_exact_and_frozen_stages_do_not_move():
    flat = kaiming_resnet18_weights(1)
    win = make_window(WindowSpec(24, 8, 64, 64, drift="drift", seed=2))
    args = (win["frames"], win["labels"], win["heldout_frames"], win["heldout_labels"])
    a = ekya.retrain(flat, 3, *args, 0.5, 2, 0.02, batch=5, seed=4, use_cache=True)
    b = ekya.retrain(flat, 3, *args, 0.5, 2, 0.02, batch=5, seed=4, use_cache=False)
    np.testing.assert_array_equal(a.weights, b.weights)
    assert a.losses == b.losses and a.heldout_acc == b.heldout_acc
    net = ResNet18(6)
    P0, P1 = net.unpack(flat), net.unpack(a.weights)
    lowest = len(STAGES) - 3
    for name, _ in net.spec:
        if net.stage_of[name] < lowest:
            np.testing.assert_array_equal(P0[name], P1[name])
        elif not name.endswith("num_batches_tracked"):
            assert not np.array_equal(P0[name], P1[name]), name
    # 12 frames at batch 5 -> batches of 5, 5, 2 (last partial batch kept)
    assert len(a.losses) == 2 * math.ceil(12 / 5)


def test_fc_only_first_step_is_logistic_regression_step():
    flat = kaiming_resnet18_weights(0)
    win = make_window(WindowSpec(8, 2, 64, 64, drift="none", seed=9))
    res = ekya.retrain(flat, 1, win["frames"], win["labels"], win["heldout_frames"],
                       win["heldout_labels"], 1.0, 1, 0.1, batch=8, seed=0)
    net = ResNet18(6)
    P = net.unpack(flat)
    f = ekya.prefix_forward(net, P, win["frames"].astype(np.float64), 5)  # pooled features
    W, b = P["fc.weight"], P["fc.bias"]
    z = f @ W.T + b
    p = np.exp(z - z.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    Y = np.eye(6)[win["labels"]]
    W1 = W - 0.1 * (p - Y).T @ f / 8       # one full-batch step, v = g on the first step
    np.testing.assert_allclose(net.unpack(res.weights)["fc.weight"], W1, rtol=1e-12, atol=1e-14)


@pytest.mark.slow
def test_separable_window_is_learned_fc_only():
    flat = kaiming_resnet18_weights(0)
    spec = WindowSpec(48, 48, 64, 64, drift="none", noise_std=0.0, seed=4)
    win = make_window(spec)
    res = ekya.retrain(flat, 1, win["frames"], win["labels"], win["heldout_frames"],
                       win["heldout_labels"], 1.0, 60, 0.5, batch=16, seed=0)
    assert res.heldout_acc[-1] == 1.0


def test_profile_configs_equal_individual_retrains_and_share_subset_prefix():
    flat = kaiming_resnet18_weights(0)
    win = make_window(WindowSpec(20, 6, 64, 64, drift="drift", seed=8))
    args = (win["frames"], win["labels"], win["heldout_frames"], win["heldout_labels"])
    cfgs = [ekya.ProfileConfig(1, 0.5, 2, 0.05, batch=4, seed=11),
            ekya.ProfileConfig(2, 0.25, 1, 0.01, batch=4, seed=12)]
    out = ekya.profile(flat, cfgs, *args, subsample_seed=5)
    assert out[1].train_indices == out[0].train_indices[:5]
    one = ekya.retrain(flat, 1, *args, 0.5, 2, 0.05, batch=4, seed=5, shuffle_seed=11)
    np.testing.assert_array_equal(one.weights, out[0].weights)
    assert len(out[0].heldout_acc) == 2 and len(out[1].heldout_acc) == 1
