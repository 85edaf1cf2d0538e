"""An independent re-implementation of one retraining run with torch CPU
modules, used by the GPU parity tests only to measure how far rounding alone
moves each tensor of that run from the fp64 oracle.

ReLU and max-pool backward passes route gradients by branch decisions; where
an input lies within rounding of its branch point a correct fp32 or bf16
implementation may take the other branch than the fp64 oracle, and the
gradient of that output channel moves by a large fraction (tests/margins.py).
Where a test cannot rule such decisions out, it bounds the library's error
on each tensor by a small multiple of the spread this probe shows over
several in-batch summation orders.

`bf16=True` stores every module output (activations, and through a custom
autograd function their gradients) and the conv weights used in a step in
bfloat16 (round to nearest even), with fp32 arithmetic in between, as the
library's bf16 path does; the classifier (with its hidden layer, if any),
logits, pooled features, BatchNorm statistics and master weights stay fp32."""
import numpy as np

from oracle import rng
from oracle.resnet18 import STAGES, ResNet18


def _round_fn():
    import torch

    class RoundBF16(torch.autograd.Function):
        @staticmethod
        def forward(ctx, x):
            return x.to(torch.bfloat16).to(x.dtype)

        @staticmethod
        def backward(ctx, g):
            return g.to(torch.bfloat16).to(g.dtype)

    return RoundBF16.apply


def torch_retrain(w0, k, win, frac, lr, mu, batch, seed, perm_seed=None, bf16=False, epochs=1,
                  shuffle_seed=None, hidden=0):
    """(weights, step losses): the weights (canonical flat, float64) after
    `epochs` epochs of the same retraining job, and the loss of every step;
    perm_seed permutes the samples inside every batch (the same mathematics
    with a different rounding order).  The subset uses `seed`, epoch orders
    `shuffle_seed` (default `seed`)."""
    import torch
    import torch.nn.functional as F

    from tests.test_oracle_resnet import _torch_model
    m, names = _torch_model(np.asarray(w0, dtype=np.float64), hidden=hidden)
    m = m.float()
    m.train()
    net = ResNet18(6, hidden=hidden)
    lo = len(STAGES) - k
    trainable = net.trainable_names(k)
    params = dict(m.named_parameters())
    for n, p in params.items():
        p.requires_grad_(n in trainable)
    for name, mod in m.named_modules():
        if isinstance(mod, torch.nn.BatchNorm2d) and net.stage_of[name + ".weight"] < lo:
            mod.eval()
    convs = []
    if bf16:
        rnd = _round_fn()
        for name, mod in m.named_modules():
            if name.startswith("fc"):  # the classifier computes in fp32
                continue
            if isinstance(mod, (torch.nn.Conv2d, torch.nn.BatchNorm2d, torch.nn.ReLU,
                                torch.nn.MaxPool2d)):
                mod.register_forward_hook(lambda mod, inp, out: rnd(out))
            if isinstance(mod, torch.nn.Conv2d):
                convs.append(mod.weight)
    opt = torch.optim.SGD([params[n] for n in trainable], lr=lr, momentum=mu)
    S = rng.training_subset(len(win["frames"]), frac, seed)
    prs = np.random.default_rng(perm_seed) if perm_seed is not None else None
    losses = []
    for e in range(epochs):
        order = rng.epoch_order(len(S), seed if shuffle_seed is None else shuffle_seed, e)
        x, y = win["frames"][S][order], win["labels"][S][order]
        for b0 in range(0, len(S), batch):
            xs, ys = x[b0:b0 + batch], y[b0:b0 + batch]
            if prs is not None:
                pi = prs.permutation(len(xs))
                xs, ys = xs[pi], ys[pi]
            xb = torch.tensor(np.ascontiguousarray(xs.transpose(0, 3, 1, 2)), dtype=torch.float32)
            masters = [w.data.clone() for w in convs]
            for w in convs:
                w.data = w.data.to(torch.bfloat16).float()
            opt.zero_grad()
            loss = F.cross_entropy(m(xb), torch.tensor(ys, dtype=torch.long))
            loss.backward()
            losses.append(loss.item())
            for w, mw in zip(convs, masters):
                w.data = mw
            opt.step()
    sd = m.state_dict()
    return np.concatenate([sd[n].double().numpy().reshape(-1) for n in names]), losses


def probe_spread(w0, k, win, frac, lr, mu, batch, seed, ref_weights, names, bf16=False, runs=4,
                 epochs=1):
    """Per tensor (of `names`), the largest error of the probe against
    ref_weights over `runs` in-batch orders, measured like the tests measure
    the library: max|a - b| / max|b| of the change from w0."""
    from tests.gpu_util import rel_err
    net = ResNet18(6)
    W0, R = net.unpack(np.asarray(w0, dtype=np.float64)), net.unpack(ref_weights)
    worst = {n: 0.0 for n in names}
    for ps in range(runs):
        P = net.unpack(torch_retrain(w0, k, win, frac, lr, mu, batch, seed, ps, bf16, epochs)[0])
        for n in names:
            worst[n] = max(worst[n], rel_err(P[n] - W0[n], R[n] - W0[n]))
    return worst


def probe_epoch_loss_spread(w0, k, win, frac, lr, mu, batch, seed, shuffle_seed, epochs,
                            ref_epoch_loss, runs=4):
    """Per epoch, the largest |probe - ref| of the mean training loss over
    `runs` in-batch orders (fp32)."""
    n = max(1, int(np.floor(frac * len(win["frames"]) + 0.5)))
    spe = -(-n // batch)
    worst = [0.0] * epochs
    for ps in range(runs):
        losses = torch_retrain(w0, k, win, frac, lr, mu, batch, seed, ps, False, epochs,
                               shuffle_seed)[1]
        for e in range(epochs):
            worst[e] = max(worst[e], abs(float(np.mean(losses[e * spe:(e + 1) * spe])) -
                                         ref_epoch_loss[e]))
    return worst
