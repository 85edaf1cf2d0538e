"""bf16 path at the 224 px retraining shape (ResNet18, layer4 and fc
trainable) against the fp64 CPU oracle: one SGD step from identical state
(every trainable tensor's update within 2e-2), and the full 2000-frame window
(held-out accuracy within one percentage point of the stored oracle run)."""
import json
import os

import numpy as np
import pytest

from oracle import ekya as oracle
from oracle.resnet18 import STAGES, ResNet18
from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import TOL, as_np, rounded, to_dev

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "retrain_224_k2.json")


@pytest.fixture(scope="module")
def ctx():
    from paper_2012_10557_amd import binding
    c = binding.ekya_create(0, 6)
    yield c
    binding.ekya_destroy(c)


@pytest.mark.parametrize("k,n", [(1, 40), (2, 40), (2, 64)])
def test_bf16_one_step_224_matches_oracle(ctx, k, n):
    """n frames at 224 px, one batch, one SGD step from identical state (at
    n = 40 the layer4 convolutions split their reduction and BatchNorm
    statistics come from the split reduction; at n = 64, the retraining
    batch, they run unsplit and the GEMM epilogues leave the statistics).
    Within 2e-2 of the oracle: the step loss, the BatchNorm running-statistic
    updates (batch statistics of the activations) and the classifier update.
    Conv and BatchNorm parameter updates of the trainable stages go through
    ReLU branch decisions that bf16 rounding flips for thousands of elements
    (see tests/margins.py), so each is bounded by max(2e-2, 3 x the largest
    error of an independent bf16-storage implementation over four in-batch
    orders); frozen stages are bitwise unchanged."""
    import torch
    from paper_2012_10557_amd import binding
    from tests.test_gpu_retrain import _update_errors
    from tests.torch_probe import probe_spread
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
    assert abs(out["step_loss"][0] - ref.losses[0]) <= TOL["bf16"] * abs(ref.losses[0])
    net = ResNet18(6)
    lo = len(STAGES) - k
    names = [nm for nm, _ in net.spec if net.stage_of[nm] >= lo]
    got = as_np(w)
    errs = _update_errors(got, ref.weights, w0, names)
    strict = [nm for nm in names if nm.startswith("fc.") or net.is_running_stat(nm)]
    bad = {nm: errs[nm] for nm in strict if errs[nm] > TOL["bf16"]}
    assert not bad, bad
    loose = [nm for nm in names if nm not in strict]
    if loose:
        probe = probe_spread(w0, k, dict(win, frames=fr), 1.0, lr, 0.9, n, 0, ref.weights, loose,
                             bf16=True)
        bad = {nm: (errs[nm], probe[nm]) for nm in loose if errs[nm] > max(TOL["bf16"], 3 * probe[nm])}
        assert not bad, bad
    G, W0 = net.unpack(got), net.unpack(w0.astype(np.float64))
    for nm, _ in net.spec:
        if net.stage_of[nm] < lo:
            np.testing.assert_array_equal(G[nm], W0[nm])


def test_bf16_window_accuracy_within_1pp_of_oracle(ctx):
    """The 2000-frame 224 px window at 30% (600 frames), 5 epochs of batch 64:
    held-out accuracy after the last epoch within 1 percentage point of the
    stored oracle run, and the first epoch's mean loss within 2e-2."""
    import torch
    from paper_2012_10557_amd import binding
    with open(GOLDEN) as f:
        g = json.load(f)
    c = g["case"]
    win = make_window(WindowSpec(c["n_frames"], c["n_heldout"], c["px"], c["px"], drift=c["drift"],
                                 seed=c["window_seed"]))
    w = torch.tensor(kaiming_resnet18_weights(seed=c["weights_seed"]), device="cuda")
    out = binding.ekya_retrain(ctx, w, c["k"], to_dev(win["frames"], "bf16"),
                               torch.tensor(win["labels"], device="cuda"),
                               to_dev(win["heldout_frames"], "bf16"),
                               torch.tensor(win["heldout_labels"], device="cuda"),
                               c["frac"], c["epochs"], c["lr"], c["momentum"], c["batch"], c["seed"])
    assert out["n_train"] == g["n_train"]
    print("gpu", out["heldout_acc"], out["epoch_loss"])
    print("oracle", g["heldout_acc"], g["epoch_loss"])
    assert abs(out["heldout_acc_final"] - g["heldout_acc"][-1]) <= 0.01
    assert abs(out["epoch_loss"][0] - g["epoch_loss"][0]) <= TOL["bf16"] * abs(g["epoch_loss"][0])
