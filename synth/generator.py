"""Seeded synthetic video windows and initial weights.

Randomness: every draw comes from SplitMix64 (Steele, Lea and Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014), used here as a
counter-based generator: the i-th output (i >= 0) of a stream with start state
s is mix(s + (i + 1) * 0x9E3779B97F4A7C15).  Each purpose (labels, noise,
prototypes, drift, each weight tensor) gets its own start state
s = seed + tag * 0xD1B54A32D192ED03 (mod 2**64).

Frames stand in for the paper's camera windows (the evaluation setup uses
Cityscapes, Waymo and two urban video sets, none of which is available here):
  * each class c owns a prototype: a coarse G x G x 3 grid of N(0, 1) draws
    upsampled bilinearly (half-pixel centres, edge clamp) to H x W x 3;
  * a frame with label y is  a * (proto[y] + noise) + b  with per-pixel noise
    N(0, noise_std**2); (a, b) are a contrast and brightness that are fixed
    (drift="shift"), move linearly over the frame index from (a0, b0) to
    (a1, b1) (drift="drift"), or are (1, 0) (drift="none");
  * labels are i.i.d. uniform over the classes.
Normals use the Box-Muller transform of two uniforms u = (z >> 11) * 2**-53.

Weights follow torchvision's ResNet initialisation: conv weights are
Kaiming-normal in fan-out mode with ReLU gain (std = sqrt(2 / (Cout*R*S))),
BatchNorm weight 1, bias 0, running mean 0, running variance 1, and the
classifier's weight and bias uniform on +-1/sqrt(fan_in).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Tuple

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
STREAM = 0xD1B54A32D192ED03

TAG_LABELS = 1
TAG_NOISE = 2
TAG_DRIFT = 3
TAG_HELD_LABELS = 11
TAG_HELD_NOISE = 12
TAG_PROTO = 100
TAG_WEIGHTS = 1000


def _state(seed: int, tag: int) -> int:
    return (int(seed) + int(tag) * STREAM) & MASK64


def splitmix64_block(state0: int, n: int, start: int = 0) -> np.ndarray:
    """Outputs start .. start+n-1 of the SplitMix64 stream with start state `state0`."""
    i = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(state0 & MASK64) + i * np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def _uniform(state0: int, n: int, start: int = 0) -> np.ndarray:
    z = splitmix64_block(state0, n, start)
    return (z >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def _normal(state0: int, n: int, start_pair: int = 0) -> np.ndarray:
    """n standard normals; pair j uses uniforms 2j and 2j+1 of the stream."""
    npairs = (n + 1) // 2
    u = _uniform(state0, 2 * npairs, 2 * start_pair).reshape(npairs, 2)
    r = np.sqrt(-2.0 * np.log(1.0 - u[:, 0]))
    t = 2.0 * np.pi * u[:, 1]
    out = np.empty((npairs, 2), dtype=np.float64)
    out[:, 0] = r * np.cos(t)
    out[:, 1] = r * np.sin(t)
    return out.reshape(-1)[:n]


def _upsample_axis(a: np.ndarray, out: int, axis: int) -> np.ndarray:
    n = a.shape[axis]
    dst = np.arange(out, dtype=np.float64)
    src = np.maximum((dst + 0.5) * (n / out) - 0.5, 0.0)
    i0 = np.minimum(np.floor(src).astype(np.int64), n - 1)
    i1 = np.minimum(i0 + 1, n - 1)
    lam = src - i0
    a0 = np.take(a, i0, axis=axis)
    a1 = np.take(a, i1, axis=axis)
    shape = [1] * a.ndim
    shape[axis] = out
    lam = lam.reshape(shape)
    return a0 * (1.0 - lam) + a1 * lam


@dataclass
class WindowSpec:
    n_frames: int
    n_heldout: int
    H: int = 224
    W: int = 224
    n_classes: int = 6
    noise_std: float = 0.3
    drift: str = "drift"  # "none" | "shift" | "drift"
    seed: int = 0
    grid: int = 0  # 0: 7 at >= 112 px, else 4

    def grid_size(self) -> int:
        if self.grid:
            return self.grid
        return 7 if min(self.H, self.W) >= 112 else 4


def _prototypes(spec: WindowSpec) -> np.ndarray:
    g = spec.grid_size()
    protos = np.empty((spec.n_classes, spec.H, spec.W, 3), dtype=np.float64)
    for c in range(spec.n_classes):
        grid = _normal(_state(spec.seed, TAG_PROTO + c), g * g * 3).reshape(g, g, 3)
        protos[c] = _upsample_axis(_upsample_axis(grid, spec.H, 0), spec.W, 1)
    return protos


def _drift_params(spec: WindowSpec) -> Tuple[float, float, float, float]:
    u = _uniform(_state(spec.seed, TAG_DRIFT), 4)
    a0, a1 = 0.8 + 0.4 * u[0], 0.8 + 0.4 * u[1]
    b0, b1 = -0.2 + 0.4 * u[2], -0.2 + 0.4 * u[3]
    if spec.drift == "none":
        return 1.0, 1.0, 0.0, 0.0
    if spec.drift == "shift":
        return a0, a0, b0, b0
    if spec.drift == "drift":
        return a0, a1, b0, b1
    raise ValueError(f"unknown drift mode {spec.drift!r}")


def make_frames(spec: WindowSpec, n: int, label_tag: int, noise_tag: int,
                first: int = 0, count: int | None = None,
                protos: np.ndarray | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """Frames first .. first+count-1 of an n-frame sequence (float32 NHWC) and their labels."""
    if count is None:
        count = n - first
    if protos is None:
        protos = _prototypes(spec)
    a0, a1, b0, b1 = _drift_params(spec)
    labels_u = _uniform(_state(spec.seed, label_tag), count, first)
    labels = np.minimum((labels_u * spec.n_classes).astype(np.int64),
                        spec.n_classes - 1).astype(np.int32)
    npix = spec.H * spec.W * 3
    npairs = (npix + 1) // 2
    frames = np.empty((count, spec.H, spec.W, 3), dtype=np.float32)
    nstate = _state(spec.seed, noise_tag)
    for j in range(count):
        i = first + j
        t = i / (n - 1) if n > 1 else 0.0
        a = a0 + (a1 - a0) * t
        b = b0 + (b1 - b0) * t
        eps = _normal(nstate, npix, i * npairs).reshape(spec.H, spec.W, 3)
        frames[j] = a * (protos[labels[j]] + spec.noise_std * eps) + b
    return frames, labels


def make_window(spec: WindowSpec) -> dict:
    """Training window plus a held-out set drawn from the same window distribution."""
    protos = _prototypes(spec)
    frames, labels = make_frames(spec, spec.n_frames, TAG_LABELS, TAG_NOISE, protos=protos)
    hframes, hlabels = make_frames(spec, spec.n_heldout, TAG_HELD_LABELS, TAG_HELD_NOISE,
                                   protos=protos)
    return {"frames": frames, "labels": labels,
            "heldout_frames": hframes, "heldout_labels": hlabels}


def resnet18_param_spec(n_classes: int = 6, widths=(64, 128, 256, 512),
                        blocks=(2, 2, 2, 2), hidden: int = 0) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, kind) in torchvision state_dict order, without num_batches_tracked.
    hidden > 0: the classifier is Linear(512, hidden), ReLU, Linear(hidden,
    n_classes), named as an nn.Sequential (fc.0, fc.2)."""
    spec: List[Tuple[str, Tuple[int, ...], str]] = []

    def bn(prefix: str, c: int):
        spec.append((prefix + ".weight", (c,), "bn_weight"))
        spec.append((prefix + ".bias", (c,), "bn_bias"))
        spec.append((prefix + ".running_mean", (c,), "bn_mean"))
        spec.append((prefix + ".running_var", (c,), "bn_var"))

    spec.append(("conv1.weight", (widths[0], 3, 7, 7), "conv"))
    bn("bn1", widths[0])
    cin = widths[0]
    for si, (w, nb) in enumerate(zip(widths, blocks)):
        for bi in range(nb):
            p = f"layer{si + 1}.{bi}"
            stride = 2 if (si > 0 and bi == 0) else 1
            spec.append((p + ".conv1.weight", (w, cin, 3, 3), "conv"))
            bn(p + ".bn1", w)
            spec.append((p + ".conv2.weight", (w, w, 3, 3), "conv"))
            bn(p + ".bn2", w)
            if stride != 1 or cin != w:
                spec.append((p + ".downsample.0.weight", (w, cin, 1, 1), "conv"))
                bn(p + ".downsample.1", w)
            cin = w
    if hidden:
        spec.append(("fc.0.weight", (hidden, widths[-1]), "fc_weight"))
        spec.append(("fc.0.bias", (hidden,), "fc_bias"))
        spec.append(("fc.2.weight", (n_classes, hidden), "fc_weight"))
        spec.append(("fc.2.bias", (n_classes,), "fc_bias"))
    else:
        spec.append(("fc.weight", (n_classes, widths[-1]), "fc_weight"))
        spec.append(("fc.bias", (n_classes,), "fc_bias"))
    return spec


def kaiming_resnet18_weights(seed: int = 0, n_classes: int = 6, widths=(64, 128, 256, 512),
                             blocks=(2, 2, 2, 2), hidden: int = 0) -> np.ndarray:
    """Flat float32 weights in the canonical order of `resnet18_param_spec`.
    Linear layers draw weight and bias from U(-1/sqrt(fan_in), 1/sqrt(fan_in))
    (torch.nn.Linear's default), fan_in being the layer's input width."""
    parts = []
    fan_in_fc = widths[-1]
    for idx, (name, shape, kind) in enumerate(resnet18_param_spec(n_classes, widths, blocks, hidden)):
        n = int(np.prod(shape))
        st = _state(seed, TAG_WEIGHTS + idx)
        if kind == "fc_weight":
            fan_in_fc = shape[1]
        if kind == "conv":
            std = np.sqrt(2.0 / (shape[0] * shape[2] * shape[3]))
            vals = std * _normal(st, n)
        elif kind in ("fc_weight", "fc_bias"):
            bound = 1.0 / np.sqrt(fan_in_fc)
            vals = -bound + 2.0 * bound * _uniform(st, n)
        elif kind in ("bn_weight", "bn_var"):
            vals = np.ones(n)
        else:
            vals = np.zeros(n)
        parts.append(vals.astype(np.float32))
    return np.concatenate(parts)
