"""ResNet18 edge classifier, split into the stages that retraining freezes or trains.

Topology (He et al., "Deep residual learning for image recognition", the
paper's ResNet reference; torchvision's ResNet18, whose model the paper
cites for the network's size in section 6.6):
  stem   : conv 7x7 stride 2 pad 3 (no bias), BN, ReLU, max-pool 3x3 stride 2 pad 1
  layer1..layer4 : two BasicBlocks each, widths 64/128/256/512;
           block(x) = ReLU(BN2(conv2(ReLU(BN1(conv1(x))))) + shortcut(x)),
           3x3 convs with pad 1, stride 2 on conv1 of the first block of
           layers 2-4, shortcut = BN(conv 1x1 stride 2) where the shape
           changes, identity otherwise
  pool   : global average pool (no parameters)
  fc     : affine classifier with bias; or, with `hidden` > 0 neurons in the
           last hidden layer, Linear(512, hidden), ReLU, Linear(hidden,
           classes) (torch nn.Sequential names fc.0 and fc.2)

The number of neurons in the last layer is one of the retraining
configuration's knobs (sections 3.2 and 6.1).  The output layer's width is
fixed by the classes, so the knob is read as the width of a hidden fully
connected layer between the pooled features and the classifier, trained with
the classifier (stage 5); hidden = 0 is the plain affine classifier.

Retraining "fewer layers" / "freezing more layers" (section 3.1) is read as
training the last k stages of [stem, layer1, layer2, layer3, layer4, fc]:
k = 1 trains fc, k = 2 trains layer4 and fc, ..., k = 6 trains everything.
Frozen stages always run BatchNorm in eval mode; trainable stages run it in
train mode during training and eval mode for held-out evaluation.

Canonical flat weight layout: torchvision state_dict order without
num_batches_tracked, fp32, conv weights [K, C, R, S].
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from . import nn

STAGES = ("stem", "layer1", "layer2", "layer3", "layer4", "fc")


class ResNet18:
    def __init__(self, n_classes: int = 6, widths=(64, 128, 256, 512), blocks=(2, 2, 2, 2),
                 hidden: int = 0):
        self.n_classes = n_classes
        self.hidden = hidden
        self.widths = tuple(widths)
        self.blocks = tuple(blocks)
        self.spec: List[Tuple[str, Tuple[int, ...]]] = []
        self.stage_of: Dict[str, int] = {}
        self._block_cfg: List[List[Tuple[str, int, bool]]] = []

        def add(name, shape, stage):
            self.spec.append((name, tuple(shape)))
            self.stage_of[name] = stage

        def add_bn(prefix, c, stage):
            for suffix in ("weight", "bias", "running_mean", "running_var"):
                add(f"{prefix}.{suffix}", (c,), stage)

        add("conv1.weight", (widths[0], 3, 7, 7), 0)
        add_bn("bn1", widths[0], 0)
        cin = widths[0]
        for si, (w, nb) in enumerate(zip(widths, blocks)):
            cfg = []
            for bi in range(nb):
                p = f"layer{si + 1}.{bi}"
                stride = 2 if (si > 0 and bi == 0) else 1
                has_ds = stride != 1 or cin != w
                add(p + ".conv1.weight", (w, cin, 3, 3), si + 1)
                add_bn(p + ".bn1", w, si + 1)
                add(p + ".conv2.weight", (w, w, 3, 3), si + 1)
                add_bn(p + ".bn2", w, si + 1)
                if has_ds:
                    add(p + ".downsample.0.weight", (w, cin, 1, 1), si + 1)
                    add_bn(p + ".downsample.1", w, si + 1)
                cfg.append((p, stride, has_ds))
                cin = w
            self._block_cfg.append(cfg)
        if hidden:
            add("fc.0.weight", (hidden, widths[-1]), 5)
            add("fc.0.bias", (hidden,), 5)
            add("fc.2.weight", (n_classes, hidden), 5)
            add("fc.2.bias", (n_classes,), 5)
        else:
            add("fc.weight", (n_classes, widths[-1]), 5)
            add("fc.bias", (n_classes,), 5)

    # ----------------------------------------------------------- weights
    def n_weights(self) -> int:
        return int(sum(np.prod(s) for _, s in self.spec))

    def unpack(self, flat: np.ndarray) -> Dict[str, np.ndarray]:
        out, off = {}, 0
        for name, shape in self.spec:
            n = int(np.prod(shape))
            out[name] = np.asarray(flat[off:off + n], dtype=np.float64).reshape(shape).copy()
            off += n
        assert off == flat.size, (off, flat.size)
        return out

    def pack(self, params: Dict[str, np.ndarray]) -> np.ndarray:
        return np.concatenate([params[name].reshape(-1) for name, _ in self.spec])

    @staticmethod
    def is_running_stat(name: str) -> bool:
        return name.endswith("running_mean") or name.endswith("running_var")

    def trainable_names(self, k: int) -> List[str]:
        """Parameters (not running statistics) of the last k stages."""
        lo = len(STAGES) - k
        return [n for n, _ in self.spec if self.stage_of[n] >= lo and not self.is_running_stat(n)]

    # ----------------------------------------------------------- forward
    def _bn(self, P, prefix, z, train, tape):
        g, b = P[prefix + ".weight"], P[prefix + ".bias"]
        if not train:
            return nn.batchnorm_eval(z, g, b, P[prefix + ".running_mean"], P[prefix + ".running_var"])
        y, saved = nn.batchnorm_train(z, g, b)
        _, _, mean, var, m = saved
        P[prefix + ".running_mean"], P[prefix + ".running_var"] = nn.batchnorm_running_update(
            P[prefix + ".running_mean"], P[prefix + ".running_var"], mean, var, m)
        tape[prefix] = saved
        return y

    def stage_forward(self, P, stage: int, x, train: bool, tape: dict):
        """Run one stage; for stage 4 (layer4) the global average pool follows.

        In train mode, BatchNorm running statistics in P are updated and
        everything the backward pass needs is written into `tape`."""
        if stage == 0:
            z = nn.conv2d(x, P["conv1.weight"], 2, 3)
            a = nn.relu(self._bn(P, "bn1", z, train, tape))
            y, arg = nn.maxpool(a)
            tape["stem"] = (x, a, arg)
            return y
        if stage == 5:
            tape["fc"] = x
            if not self.hidden:
                return nn.linear(x, P["fc.weight"], P["fc.bias"])
            a = nn.relu(nn.linear(x, P["fc.0.weight"], P["fc.0.bias"]))
            tape["fc.hidden"] = a
            return nn.linear(a, P["fc.2.weight"], P["fc.2.bias"])
        for prefix, stride, has_ds in self._block_cfg[stage - 1]:
            x = self._block_forward(P, prefix, x, stride, has_ds, train, tape)
        if stage == 4:
            tape["pool"] = x.shape
            x = nn.avgpool(x)
        return x

    def _block_forward(self, P, p, x, stride, has_ds, train, tape):
        a1 = nn.relu(self._bn(P, p + ".bn1", nn.conv2d(x, P[p + ".conv1.weight"], stride, 1), train, tape))
        y2 = self._bn(P, p + ".bn2", nn.conv2d(a1, P[p + ".conv2.weight"], 1, 1), train, tape)
        if has_ds:
            sc = self._bn(P, p + ".downsample.1", nn.conv2d(x, P[p + ".downsample.0.weight"], stride, 0),
                          train, tape)
        else:
            sc = x
        out = nn.relu(y2 + sc)
        tape[p] = (x, a1, out)
        return out

    def forward(self, P, x, first: int, last: int, train: bool, tape: dict):
        """Stages first..last inclusive."""
        for st in range(first, last + 1):
            x = self.stage_forward(P, st, x, train, tape)
        return x

    # ---------------------------------------------------------- backward
    def backward(self, P, dlogits, lowest: int, tape: dict) -> Dict[str, np.ndarray]:
        """Gradients of every parameter of stages lowest..5 from a train-mode tape.

        No gradient is sent into the input of stage `lowest` (it is frozen data)."""
        grads: Dict[str, np.ndarray] = {}
        if self.hidden:
            a = tape["fc.hidden"]
            da, grads["fc.2.weight"], grads["fc.2.bias"] = nn.linear_backward(dlogits, a, P["fc.2.weight"])
            df, grads["fc.0.weight"], grads["fc.0.bias"] = nn.linear_backward(
                nn.relu_backward(da, a), tape["fc"], P["fc.0.weight"])
        else:
            df, grads["fc.weight"], grads["fc.bias"] = nn.linear_backward(dlogits, tape["fc"],
                                                                          P["fc.weight"])
        if lowest == 5:
            return grads
        d = nn.avgpool_backward(df, tape["pool"])
        for stage in range(4, lowest - 1, -1):
            if stage == 0:
                self._stem_backward(P, d, tape, grads)
                break
            cfg = self._block_cfg[stage - 1]
            for bi in range(len(cfg) - 1, -1, -1):
                p, stride, has_ds = cfg[bi]
                need_dx = not (stage == lowest and bi == 0)
                d = self._block_backward(P, p, stride, has_ds, d, tape, grads, need_dx)
        return grads

    def _bn_backward(self, P, prefix, dy, tape, grads):
        dz, grads[prefix + ".weight"], grads[prefix + ".bias"] = nn.batchnorm_backward(
            dy, tape[prefix], P[prefix + ".weight"])
        return dz

    def _block_backward(self, P, p, stride, has_ds, dout, tape, grads, need_dx):
        x, a1, out = tape[p]
        g = nn.relu_backward(dout, out)
        dz2 = self._bn_backward(P, p + ".bn2", g, tape, grads)
        w2, w1 = P[p + ".conv2.weight"], P[p + ".conv1.weight"]
        grads[p + ".conv2.weight"] = nn.conv2d_wgrad(a1, dz2, w2.shape, 1, 1)
        da1 = nn.conv2d_dgrad(dz2, w2, a1.shape, 1, 1)
        dz1 = self._bn_backward(P, p + ".bn1", nn.relu_backward(da1, a1), tape, grads)
        grads[p + ".conv1.weight"] = nn.conv2d_wgrad(x, dz1, w1.shape, stride, 1)
        dx = None
        if has_ds:
            wd = P[p + ".downsample.0.weight"]
            dzd = self._bn_backward(P, p + ".downsample.1", g, tape, grads)
            grads[p + ".downsample.0.weight"] = nn.conv2d_wgrad(x, dzd, wd.shape, stride, 0)
            if need_dx:
                dx = nn.conv2d_dgrad(dzd, wd, x.shape, stride, 0)
        elif need_dx:
            dx = g
        if need_dx:
            dx = dx + nn.conv2d_dgrad(dz1, w1, x.shape, stride, 1)
        return dx

    def _stem_backward(self, P, d, tape, grads):
        x, a, arg = tape["stem"]
        da = nn.maxpool_backward(d, arg, a.shape)
        dz = self._bn_backward(P, "bn1", nn.relu_backward(da, a), tape, grads)
        grads["conv1.weight"] = nn.conv2d_wgrad(x, dz, P["conv1.weight"].shape, 2, 3)
