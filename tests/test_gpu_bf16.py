"""bf16 path at 224 px against the fp64 CPU oracle: one SGD step from
identical state at every trainable depth (k = 1, 2 with the oracle run here;
k = 3 and 6 at batch 32 and 128 against stored oracle runs), the 2000-frame
layer4+fc windows (an easy one that saturates and a hard one that does not:
every epoch's held-out accuracy within one percentage point), and a short
full-depth run shaped like the full-depth workload (batch 128, every stage
trainable, BatchNorm in train mode).

What is gated at the fixed bf16 tolerance 2e-2: the step loss, the BatchNorm
running statistics (batch statistics of the activations) and the classifier
update.  Convolution and BatchNorm-affine updates are weight gradients summed
over thousands of pixels whose operands (activations and their gradients)
are stored in bf16; the BatchNorm backward projects each channel's gradient
onto what is left after removing its mean and its correlation with the
normalised input, so these sums are small residues of large terms, and the
rounding of the stored operands alone moves them by 5-50% (root mean square,
largest in the stem and layer1 after a full-depth backward pass).  An
independent implementation that stores the same tensors in bf16
(tests/torch_probe.py, torch on the CPU) shows the same errors against the
fp64 oracle, and agrees with the oracle to 0.4% when it keeps fp32.  Each of
these tensors is therefore gated by its root-mean-square update error within
max(2e-2, 1.5 x that probe's error on the same positions), and every error is
printed.  Stored runs come from tests/golden/make_*_golden.py (oracle
only)."""
import gzip
import json
import os

import numpy as np
import pytest

from oracle import ekya as oracle
from oracle.resnet18 import STAGES, ResNet18
from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import TOL, as_np, rounded, to_dev

pytestmark = pytest.mark.gpu

HERE = os.path.join(os.path.dirname(__file__), "golden")
GOLDEN = os.path.join(HERE, "retrain_224_k2.json")
BF16_GRAD_RMS = 2e-2
PROBE_FACTOR = 1.5


@pytest.fixture(scope="module")
def ctx():
    from paper_2012_10557_amd import binding
    c = binding.ekya_create(0, 6)
    yield c
    binding.ekya_destroy(c)


def _rms_errors(got, ref, w0, names):
    """Per tensor: (rms error of the update / rms of the oracle's update,
    largest error / largest oracle update)."""
    net = ResNet18(6)
    G, R, W0 = net.unpack(got), net.unpack(ref), net.unpack(np.asarray(w0, dtype=np.float64))
    out = {}
    for n in names:
        dr, dg = R[n] - W0[n], G[n] - W0[n]
        rms = float(np.sqrt(np.mean((dg - dr) ** 2)) / max(np.sqrt(np.mean(dr * dr)), 1e-30))
        out[n] = (rms, float(np.abs(dg - dr).max() / max(np.abs(dr).max(), 1e-30)))
    return out


def _probe_weights(w0, k, frames_bf16, labels, n, lr, mu, seed):
    """Weights after the same step from the bf16-storage torch probe."""
    from tests.torch_probe import torch_retrain
    win = {"frames": frames_bf16, "labels": labels}
    return torch_retrain(w0, k, win, 1.0, lr, mu, n, seed, None, True, 1)[0]


def _gate_updates(strict, loose, probe):
    """strict: name -> error (fixed 2e-2); loose: name -> (rms err, max err);
    probe: name -> the bf16 probe's rms error on the same positions."""
    for n, e in strict.items():
        print(f"  {n:40s} err {e:.3e}  (gate {TOL['bf16']:.0e})")
    bound = {n: max(BF16_GRAD_RMS, PROBE_FACTOR * probe[n]) for n in loose}
    for n, (r, m) in loose.items():
        print(f"  {n:40s} rms err {r:.3e}  bound {bound[n]:.3e}  (bf16 probe {probe[n]:.3e})  "
              f"max err {m:.3e}")
    bad = {n: e for n, e in strict.items() if e > TOL["bf16"]}
    assert not bad, bad
    bad = {n: (r, bound[n]) for n, (r, _) in loose.items() if r > bound[n]}
    assert not bad, bad


@pytest.mark.parametrize("k,n", [(1, 40), (2, 40), (2, 64)])
def test_bf16_one_step_224_matches_oracle(ctx, k, n):
    """n frames at 224 px, one batch, one SGD step from identical state (at
    n = 40 the layer4 convolutions split their reduction and BatchNorm
    statistics come from the split reduction; at n = 64, the retraining
    batch, they run unsplit and the GEMM epilogues leave the statistics);
    frozen stages bitwise unchanged."""
    import torch
    from paper_2012_10557_amd import binding
    from tests.test_gpu_retrain import _update_errors
    w0 = kaiming_resnet18_weights(seed=0)
    win = make_window(WindowSpec(n, 8, 224, 224, drift="shift", seed=4))
    fr, hf = rounded(win["frames"], "bf16"), rounded(win["heldout_frames"], "bf16")
    w = torch.tensor(w0, device="cuda")
    lr = 0.01
    out = binding.ekya_retrain(ctx, w, k, to_dev(fr, "bf16"),
                               torch.tensor(win["labels"], device="cuda"), to_dev(hf, "bf16"),
                               torch.tensor(win["heldout_labels"], device="cuda"),
                               1.0, 1, lr, 0.9, n, 0, step_losses=True)
    ref = oracle.retrain(w0, k, fr, win["labels"], hf, win["heldout_labels"], 1.0, 1, lr, 0.9, n, 0)
    assert out["n_steps"] == 1
    print(f"loss {out['step_loss'][0]:.6f} oracle {ref.losses[0]:.6f}")
    assert abs(out["step_loss"][0] - ref.losses[0]) <= TOL["bf16"] * abs(ref.losses[0])
    net = ResNet18(6)
    lo = len(STAGES) - k
    names = [nm for nm, _ in net.spec if net.stage_of[nm] >= lo]
    got = as_np(w)
    strict_names = [nm for nm in names if nm.startswith("fc.") or net.is_running_stat(nm)]
    strict = {nm: e for nm, e in _update_errors(got, ref.weights, w0, strict_names).items()}
    loose_names = [nm for nm in names if nm not in strict_names]
    loose = _rms_errors(got, ref.weights, w0, loose_names)
    if loose_names:
        pw = _probe_weights(w0, k, fr, win["labels"], n, lr, 0.9, 0)
        probe = {nm: r for nm, (r, _) in _rms_errors(pw, ref.weights, w0, loose_names).items()}
    else:
        probe = {}
    _gate_updates(strict, loose, probe)
    G, W0 = net.unpack(got), net.unpack(w0.astype(np.float64))
    for nm, _ in net.spec:
        if net.stage_of[nm] < lo:
            np.testing.assert_array_equal(G[nm], W0[nm])


@pytest.fixture(scope="module")
def onestep():
    with gzip.open(os.path.join(HERE, "onestep_224.json.gz"), "rt") as f:
        return json.load(f)


@pytest.mark.parametrize("k,n", [(3, 32), (3, 128), (6, 32), (6, 128)])
def test_bf16_one_step_at_depth_matches_stored_oracle(ctx, onestep, k, n):
    """One SGD step of layer3+ (k = 3) and of every stage (k = 6: the stem's
    BatchNorm, ReLU and max-pool backward, layer1-2 in train mode) at 224 px
    in bf16, at batch 32 and 128 (the full-depth workload's batch: the fused
    per-convolution momentum steps, deferred across blocks on the second
    stream, and the GEMM-epilogue BatchNorm statistics).  Against the stored
    oracle step: loss, every running statistic and the classifier within 2e-2;
    the other tensors' updates at their stored positions (rms, normalised by
    the stored rms of the whole tensor's update); frozen stages bitwise."""
    import torch
    from paper_2012_10557_amd import binding
    c0 = onestep["common"]
    case = next(e for e in onestep["cases"] if e["k"] == k and e["n"] == n)
    w0 = kaiming_resnet18_weights(seed=c0["weights_seed"])
    win = make_window(WindowSpec(n, c0["n_heldout"], c0["px"], c0["px"], drift=c0["drift"],
                                 seed=c0["window_seed"]))
    w = torch.tensor(w0, device="cuda")
    out = binding.ekya_retrain(ctx, w, k, to_dev(win["frames"], "bf16"),
                               torch.tensor(win["labels"], device="cuda"),
                               to_dev(win["heldout_frames"], "bf16"),
                               torch.tensor(win["heldout_labels"], device="cuda"),
                               1.0, 1, c0["lr"], c0["momentum"], n, c0["seed"], step_losses=True)
    assert out["n_steps"] == 1
    print(f"k={k} n={n}: loss {out['step_loss'][0]:.6f} oracle {case['loss']:.6f}")
    assert abs(out["step_loss"][0] - case["loss"]) <= TOL["bf16"] * abs(case["loss"])
    net = ResNet18(6)
    G, W0 = net.unpack(as_np(w)), net.unpack(w0.astype(np.float64))
    strict = {}
    for nm, vals in case["full"].items():
        ref = np.asarray(vals).reshape(W0[nm].shape)
        dr = ref - W0[nm]
        strict[nm] = float(np.abs((G[nm] - W0[nm]) - dr).max() / max(np.abs(dr).max(), 1e-30))
    frames = rounded(win["frames"], "bf16")
    PW = net.unpack(_probe_weights(w0, k, frames, win["labels"], n, c0["lr"], c0["momentum"],
                                   c0["seed"]))
    loose, probe = {}, {}
    for nm, smp in case["sampled"].items():
        pos = np.asarray(smp["pos"])
        dr = np.asarray(smp["w1"]) - W0[nm].reshape(-1)[pos]
        dg = G[nm].reshape(-1)[pos] - W0[nm].reshape(-1)[pos]
        dp = PW[nm].reshape(-1)[pos] - W0[nm].reshape(-1)[pos]
        loose[nm] = (float(np.sqrt(np.mean((dg - dr) ** 2)) / max(smp["rms_update"], 1e-30)),
                     float(np.abs(dg - dr).max() / max(smp["max_abs_update"], 1e-30)))
        probe[nm] = float(np.sqrt(np.mean((dp - dr) ** 2)) / max(smp["rms_update"], 1e-30))
    _gate_updates(strict, loose, probe)
    lo = len(STAGES) - k
    for nm, _ in net.spec:
        if net.stage_of[nm] < lo:
            np.testing.assert_array_equal(G[nm], W0[nm])


def _window_run(ctx, c):
    import torch
    from paper_2012_10557_amd import binding
    win = make_window(WindowSpec(c["n_frames"], c["n_heldout"], c["px"], c["px"], drift=c["drift"],
                                 seed=c["window_seed"], noise_std=c.get("noise", 0.3)))
    w = torch.tensor(kaiming_resnet18_weights(seed=c["weights_seed"]), device="cuda")
    return binding.ekya_retrain(ctx, w, c["k"], to_dev(win["frames"], "bf16"),
                                torch.tensor(win["labels"], device="cuda"),
                                to_dev(win["heldout_frames"], "bf16"),
                                torch.tensor(win["heldout_labels"], device="cuda"),
                                c["frac"], c["epochs"], c["lr"], c["momentum"], c["batch"], c["seed"])


@pytest.mark.parametrize("name", ["retrain_224_k2.json", "retrain_224_k2_hard.json",
                                  "retrain_224_k6.json"])
def test_bf16_window_follows_oracle(ctx, name):
    """Whole retraining jobs against stored oracle runs: the 2000-frame window
    at 30% (600 frames), layer4+fc, 5 epochs of batch 64 -- with noise 0.3 it
    saturates by epoch 3, with noise 3.0 and a drift it climbs from 16% to
    88% -- and a full-depth job (every stage, batch 128, 256 frames, 2
    epochs).  The final held-out accuracy within one percentage point (4 of
    400 frames); every earlier epoch's within one point too, or, where the
    oracle's curve is steep, between its neighbouring epochs' accuracies (one
    point of slack): bf16 rounding shifts a trajectory by a fraction of an
    epoch, which moves a steep part of the curve by more than a point.  The
    same holds for a final epoch on a steep part (the oracle's last step
    >= 5 points): then the accuracy lies between the previous epoch's and the
    last step continued once more (one point of slack) and the final mean
    loss agrees within 2e-2.  The first epoch's mean loss within 2e-2."""
    with open(os.path.join(HERE, name)) as f:
        g = json.load(f)
    c = g["case"]
    out = _window_run(ctx, c)
    assert out["n_train"] == g["n_train"]
    print("gpu   ", out["heldout_acc"], [round(x, 5) for x in out["epoch_loss"]])
    print("oracle", g["heldout_acc"], [round(x, 5) for x in g["epoch_loss"]])
    acc, ref = out["heldout_acc"], g["heldout_acc"]
    if abs(acc[-1] - ref[-1]) > 0.01 + 1e-6:
        last = ref[-1] - ref[-2] if len(ref) > 1 else 0.0
        assert abs(last) >= 0.05, ("final epoch off by more than a point on a flat curve", acc, ref)
        lo, hi = sorted((ref[-2], min(1.0, max(0.0, ref[-1] + last))))
        assert lo - 0.01 - 1e-6 <= acc[-1] <= hi + 0.01 + 1e-6, (acc, ref)
        lf, lr = out["epoch_loss"][-1], g["epoch_loss"][-1]
        assert abs(lf - lr) <= TOL["bf16"] * abs(lr), (out["epoch_loss"], g["epoch_loss"])
    for e, (a, b) in enumerate(zip(acc, ref)):
        if abs(a - b) <= 0.01 + 1e-6:
            continue
        lo = min(ref[max(e - 1, 0)], ref[min(e + 1, len(ref) - 1)]) - 0.01
        hi = max(ref[max(e - 1, 0)], ref[min(e + 1, len(ref) - 1)]) + 0.01
        assert lo - 1e-6 <= a <= hi + 1e-6, (e, acc, ref)
    assert abs(out["epoch_loss"][0] - g["epoch_loss"][0]) <= TOL["bf16"] * abs(g["epoch_loss"][0])
