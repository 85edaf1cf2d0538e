"""Retraining-configuration variants beyond depth, fraction and epochs
(sections 3.2 and 6.1 list batch size and the number of neurons in the last
layer among the knobs), and per-stream models in batched inference:

  * a hidden classifier layer of h neurons (ekya_create_head) against the
    extended oracle: fp32 at fixed tolerance (classifier only, and through
    layer4 and the whole network on the margin-checked one-step fixtures),
    bf16 at 224 px, inference and the prepared-model path;
  * batch size as a profiler dimension: candidates that differ only in batch
    equal the corresponding retraining jobs, and fp32 classifier retraining
    at several batch sizes (one ragged) follows the oracle;
  * ekya_infer_models: ten streams, each with its own model and frame count
    (one of them empty), classified in one call, bitwise as per stream."""
import numpy as np
import pytest

from oracle import ekya as oracle
from oracle.resnet18 import STAGES, ResNet18
from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import TOL, as_np, rel_err, rounded, to_dev

pytestmark = pytest.mark.gpu


def _window(n, nh, px, drift="none", seed=0, noise=0.3):
    return make_window(WindowSpec(n, nh, px, px, drift=drift, seed=seed, noise_std=noise))


def _dev(win, prec):
    import torch
    return (to_dev(win["frames"], prec), torch.tensor(win["labels"], device="cuda"),
            to_dev(win["heldout_frames"], prec), torch.tensor(win["heldout_labels"], device="cuda"))


def _errors(net, got, ref, names):
    G, R = net.unpack(got), net.unpack(ref)
    return {n: rel_err(G[n], R[n]) for n in names}


def _frozen_unchanged(net, got, w0, k):
    lo = len(STAGES) - k
    G, W0 = net.unpack(got), net.unpack(np.asarray(w0, dtype=np.float64))
    for n, _ in net.spec:
        if net.stage_of[n] < lo:
            np.testing.assert_array_equal(G[n], W0[n])


def _ctx(hidden):
    from paper_2012_10557_amd import binding
    return binding.ekya_create(0, 6, hidden=hidden)


@pytest.mark.parametrize("hidden", [64, 1024])
def test_hidden_head_fc_only_fp32_matches_oracle(hidden):
    """64 frames at 64 px, classifier stage trainable (hidden layer and output
    layer), batch 16, two epochs: every step loss within 1e-5, both layers'
    weights within 1e-4, held-out accuracy equal, frozen stages bitwise."""
    import torch
    from paper_2012_10557_amd import binding
    net = ResNet18(6, hidden=hidden)
    w0 = kaiming_resnet18_weights(seed=0, hidden=hidden)
    assert w0.size == binding.ekya_weights_count(6, hidden)
    win = _window(64, 64, 64, seed=3)
    ctx = _ctx(hidden)
    try:
        w = torch.tensor(w0, device="cuda")
        out = binding.ekya_retrain(ctx, w, 1, *_dev(win, "f32"), 1.0, 2, 0.05, 0.9, 16, 0,
                                   step_losses=True)
        ref = oracle.retrain(w0, 1, win["frames"], win["labels"], win["heldout_frames"],
                             win["heldout_labels"], 1.0, 2, 0.05, 0.9, 16, 0, net=net)
        got = as_np(w)
        errs = _errors(net, got, ref.weights, net.trainable_names(1))
        print(f"hidden {hidden}: losses {np.round(out['step_loss'], 5).tolist()}; errors {errs}")
        np.testing.assert_allclose(out["step_loss"], ref.losses, rtol=1e-5)
        assert max(errs.values()) <= 1e-4, errs
        assert out["heldout_acc"] == pytest.approx(ref.heldout_acc, abs=1e-9)
        _frozen_unchanged(net, got, w0, 1)
    finally:
        binding.ekya_destroy(ctx)


# (px, k, window frames, fraction, batch, window seed, weights seed) of the
# margin-checked one-step fixtures of the plain network (drifting window, 8
# held-out frames, subset and shuffle seed 7): their trunk decisions (ReLU
# inputs, max-pool top-2 gaps) sit at least 1e-5 (RMS units) from their
# branch points.  The trunk weights do not depend on the head, so the same
# first batch meets the same decisions; the test re-checks them, and the
# hidden layer's own ReLU inputs.
STRICT_HIDDEN = [(64, 2, 16, 0.5, 8, 12, 1), (32, 6, 8, 0.5, 4, 1, 1)]
SEED = 7


def _update_errors(net, got, ref, w0, names):
    """Per tensor: largest error of the update beyond fp32 rounding of the
    weight itself, relative to the oracle's largest update."""
    G, R, W0 = net.unpack(got), net.unpack(ref), net.unpack(np.asarray(w0, dtype=np.float64))
    out = {}
    for n in names:
        dr = R[n] - W0[n]
        excess = np.abs((G[n] - W0[n]) - dr) - np.abs(R[n]) * 2.0 ** -23
        out[n] = float(max(excess.max(), 0.0) / max(np.abs(dr).max(), 1e-30))
    return out


@pytest.mark.parametrize("case", STRICT_HIDDEN)
def test_hidden_head_one_step_at_depth_fp32(case):
    """One SGD step through the hidden layer, the output layer and the
    trainable convolution stages: every trainable tensor within 1e-4 of the
    oracle, frozen stages bitwise."""
    import torch
    from paper_2012_10557_amd import binding
    from oracle import ekya as oracle_ekya
    from oracle import rng
    from tests.margins import decision_margins
    px, k, n, frac, batch, wseed, mseed = case
    hidden = 64
    net = ResNet18(6, hidden=hidden)
    w0 = kaiming_resnet18_weights(seed=mseed, hidden=hidden)
    win = _window(n, 8, px, drift="drift", seed=wseed)
    S = rng.training_subset(n, frac, SEED)
    first = win["frames"][S][rng.epoch_order(len(S), SEED, 0)]
    trunk_margin, _ = decision_margins(kaiming_resnet18_weights(seed=mseed), k, first)
    P = net.unpack(w0)
    lowest = len(STAGES) - k
    x = oracle_ekya.prefix_forward(net, P, first.astype(np.float64), lowest)
    f = net.forward(P, x, lowest, 4, train=True, tape={})  # the step's pooled features
    pre = f @ P["fc.0.weight"].T + P["fc.0.bias"]
    head_margin = float(np.abs(pre).min() / np.sqrt(np.mean(pre * pre)))
    assert trunk_margin >= 1e-5 and head_margin >= 1e-5, (trunk_margin, head_margin)
    ctx = _ctx(hidden)
    try:
        w = torch.tensor(w0, device="cuda")
        out = binding.ekya_retrain(ctx, w, k, *_dev(win, "f32"), frac, 1, 0.05, 0.9, batch, SEED,
                                   step_losses=True)
        ref = oracle.retrain(w0, k, win["frames"], win["labels"], win["heldout_frames"],
                             win["heldout_labels"], frac, 1, 0.05, 0.9, batch, SEED, net=net)
        assert out["n_steps"] == 1
        got = as_np(w)
        names = [nm for nm, _ in net.spec if net.stage_of[nm] >= len(STAGES) - k]
        errs = _update_errors(net, got, ref.weights, w0, names)
        worst = sorted(errs.items(), key=lambda t: -t[1])[:5]
        print(f"{case}: loss {out['step_loss'][0]:.7f} oracle {ref.losses[0]:.7f}; margins trunk "
              f"{trunk_margin:.2e} hidden layer {head_margin:.2e}; worst {worst}")
        assert abs(out["step_loss"][0] - ref.losses[0]) <= 1e-5 * abs(ref.losses[0])
        assert max(errs.values()) <= TOL["f32"], worst
        _frozen_unchanged(net, got, w0, k)
    finally:
        binding.ekya_destroy(ctx)


@pytest.mark.parametrize("k", [1, 2])
def test_hidden_head_bf16_224_one_step(k):
    """40 frames at 224 px, one step with a 256-neuron hidden layer: the loss,
    the output layer and the running statistics within 2e-2; the hidden layer
    and the layer4 updates (k = 2) within max(2e-2, 1.5 x the bf16-storage
    probe's error), every error printed."""
    import torch
    from paper_2012_10557_amd import binding
    from tests.test_gpu_bf16 import BF16_GRAD_RMS, PROBE_FACTOR
    from tests.torch_probe import torch_retrain
    hidden, n, lr = 256, 40, 0.01
    net = ResNet18(6, hidden=hidden)
    w0 = kaiming_resnet18_weights(seed=0, hidden=hidden)
    win = _window(n, 8, 224, drift="shift", seed=4)
    fr, hf = rounded(win["frames"], "bf16"), rounded(win["heldout_frames"], "bf16")
    ctx = _ctx(hidden)
    try:
        w = torch.tensor(w0, device="cuda")
        out = binding.ekya_retrain(ctx, w, k, to_dev(fr, "bf16"),
                                   torch.tensor(win["labels"], device="cuda"), to_dev(hf, "bf16"),
                                   torch.tensor(win["heldout_labels"], device="cuda"),
                                   1.0, 1, lr, 0.9, n, 0, step_losses=True)
    finally:
        binding.ekya_destroy(ctx)
    ref = oracle.retrain(w0, k, fr, win["labels"], hf, win["heldout_labels"], 1.0, 1, lr, 0.9, n, 0,
                         net=net)
    print(f"loss {out['step_loss'][0]:.6f} oracle {ref.losses[0]:.6f}")
    assert abs(out["step_loss"][0] - ref.losses[0]) <= TOL["bf16"] * abs(ref.losses[0])
    got = as_np(w)
    lo = len(STAGES) - k
    names = [nm for nm, _ in net.spec if net.stage_of[nm] >= lo]
    G, R, W0 = net.unpack(got), net.unpack(ref.weights), net.unpack(w0.astype(np.float64))
    # the hidden layer's ReLU decisions follow the bf16-rounded features, so
    # its weights are gated like the convolutions (against the probe, which
    # rounds the same features); the output layer and statistics at 2e-2
    strict = [nm for nm in names if nm.startswith("fc.2.") or net.is_running_stat(nm)]
    for nm in strict:
        dr, dg = R[nm] - W0[nm], G[nm] - W0[nm]
        e = rel_err(dg, dr) if not net.is_running_stat(nm) else rel_err(G[nm], R[nm])
        print(f"  {nm:40s} err {e:.3e}")
        assert e <= TOL["bf16"], nm
    loose = [nm for nm in names if nm not in strict]
    if loose:
        pw = torch_retrain(w0, k, {"frames": fr, "labels": win["labels"]}, 1.0, lr, 0.9, n, 0,
                           None, True, 1, hidden=hidden)[0]
        P = net.unpack(pw)
        for nm in loose:
            dr, dg, dp = R[nm] - W0[nm], G[nm] - W0[nm], P[nm] - W0[nm]
            rms = float(np.sqrt(np.mean(dr * dr))) or 1e-30
            e = float(np.sqrt(np.mean((dg - dr) ** 2))) / rms
            pe = float(np.sqrt(np.mean((dp - dr) ** 2))) / rms
            bound = max(BF16_GRAD_RMS, PROBE_FACTOR * pe)
            print(f"  {nm:40s} rms err {e:.3e} bound {bound:.3e} (probe {pe:.3e})")
            assert e <= bound, nm
    _frozen_unchanged(net, got, w0, k)


def test_hidden_head_inference_matches_oracle_and_model():
    """fp32 inference at 64 px with a hidden layer: labels equal the oracle's
    except where its top-2 logit margin is below 1e-5; a prepared model of the
    same network classifies bitwise as ekya_infer."""
    import torch
    from paper_2012_10557_amd import binding
    hidden = 128
    net = ResNet18(6, hidden=hidden)
    w0 = kaiming_resnet18_weights(seed=2, hidden=hidden)
    win = _window(96, 1, 64, seed=6)
    P = net.unpack(w0)
    z = net.forward(P, win["frames"].astype(np.float64), 0, 5, train=False, tape={})
    srt = np.sort(z, axis=1)
    margin = (srt[:, -1] - srt[:, -2]) / np.abs(z).max()
    want = np.argmax(z, axis=1)
    ctx = _ctx(hidden)
    m = binding.ekya_model_create(0, 6, binding.EKYA_FP32, hidden=hidden)
    try:
        wd = torch.tensor(w0, device="cuda")
        fr = to_dev(win["frames"])
        lab = binding.ekya_infer(ctx, wd, fr, 64)
        binding.ekya_model_load(m, wd)
        lab2, _ = binding.ekya_infer_model(ctx, m, fr, 64)
        torch.cuda.synchronize()
        got = lab.cpu().numpy()
        ok = (got == want) | (margin < 1e-5)
        print(f"labels {np.bincount(got, minlength=6)}; smallest margin {margin.min():.2e}")
        assert ok.all()
        assert torch.equal(lab, lab2)
        with pytest.raises(binding.EkyaError):  # a plain-classifier model does not fit
            plain = binding.ekya_model_create(0, 6, binding.EKYA_FP32)
            try:
                binding.ekya_model_load(plain, torch.tensor(kaiming_resnet18_weights(0),
                                                             device="cuda"))
                binding.ekya_infer_model(ctx, plain, fr, 64)
            finally:
                binding.ekya_model_destroy(plain)
    finally:
        binding.ekya_model_destroy(m)
        binding.ekya_destroy(ctx)


@pytest.mark.parametrize("batch", [3, 16, 64])
def test_batch_sizes_fc_only_fp32_match_oracle(batch):
    """Batch size as a configuration knob: 64 frames at 64 px, classifier
    retraining for two epochs at batch 3 (a ragged last batch of 1), 16 and 64
    (one step per epoch): step losses within 1e-5, weights within 1e-4."""
    import torch
    from paper_2012_10557_amd import binding
    net = ResNet18(6)
    w0 = kaiming_resnet18_weights(seed=0)
    win = _window(64, 32, 64, seed=8)
    ctx = binding.ekya_create(0, 6)
    try:
        w = torch.tensor(w0, device="cuda")
        out = binding.ekya_retrain(ctx, w, 1, *_dev(win, "f32"), 1.0, 2, 0.002, 0.9, batch, 1,
                                   step_losses=True)
    finally:
        binding.ekya_destroy(ctx)
    ref = oracle.retrain(w0, 1, win["frames"], win["labels"], win["heldout_frames"],
                         win["heldout_labels"], 1.0, 2, 0.002, 0.9, batch, 1)
    assert out["n_steps"] == 2 * -(-64 // batch)
    np.testing.assert_allclose(out["step_loss"], ref.losses, rtol=1e-5)
    errs = _errors(net, as_np(w), ref.weights, net.trainable_names(1))
    print(f"batch {batch}: {out['n_steps']} steps, errors {errs}")
    assert max(errs.values()) <= 1e-4


def test_batch_size_candidates_equal_retraining_jobs():
    """The profiler at 224 px bf16 with five candidates that differ only in
    batch size (16 .. 256; layer4 and classifier, 10% of a 2000-frame window,
    two epochs): each candidate's per-epoch accuracy and mean loss equal those
    of ekya_retrain with that batch, and its step count is ceil(200 / batch).
    Per-epoch GPU time by batch size is printed."""
    import torch
    from paper_2012_10557_amd import binding
    win = _window(2000, 400, 224, drift="drift", seed=0)
    d = _dev(win, "bf16")
    w0 = torch.tensor(kaiming_resnet18_weights(seed=0), device="cuda")
    batches = [16, 32, 64, 128, 256]
    cfgs = [dict(k=2, subsample_frac=0.1, epochs=2, lr=0.01, momentum=0.9, batch=b, seed=3)
            for b in batches]
    ctx = binding.ekya_create(0, 6)
    try:
        # the candidates' subset seed and shuffle seed equal the retraining seed
        res = binding.ekya_profile(ctx, w0, cfgs, *d, 3, concurrent=False)
        for b, r in zip(batches, res):
            w = w0.clone()
            one = binding.ekya_retrain(ctx, w, 2, d[0], d[1], d[2], d[3], 0.1, 2, 0.01, 0.9, b, 3)
            print(f"batch {b:3d}: acc {r['heldout_acc']} loss {np.round(r['epoch_loss'], 5).tolist()} "
                  f"epoch ms {[round(1e3 * s, 3) for s in r['epoch_seconds']]}")
            assert r["n_train"] == 200 and one["n_train"] == 200
            assert r["heldout_acc"] == one["heldout_acc"]
            assert r["epoch_loss"] == one["epoch_loss"]
            assert one["n_steps"] == 2 * -(-200 // b)
    finally:
        binding.ekya_destroy(ctx)


def _rotated(w, shift, bump):
    import torch
    w2 = w.clone()
    fw = w2[-(6 * 512 + 6):-6].view(6, 512)
    fb = w2[-6:]
    fw.copy_(torch.roll(fw, shift, 0))
    fb.copy_(torch.roll(fb, shift, 0) + bump)
    return w2


def test_infer_models_per_stream_weights():
    """Ten streams at 224 px bf16, each with its own model (the classifier
    rotated and shifted per stream) and its own frame count, one of them
    empty and one a single frame: labels equal ekya_infer_model per stream;
    reloading one stream's model changes only that stream's version and
    labels."""
    import torch
    from paper_2012_10557_amd import binding
    win = _window(1600, 1, 224, drift="drift", seed=9)
    fr = to_dev(win["frames"], "bf16")
    w0 = torch.tensor(kaiming_resnet18_weights(seed=0), device="cuda")
    counts = [97, 0, 360, 1, 513, 64, 200, 33, 128, 204]
    assert sum(counts) == 1600
    ctx = binding.ekya_create(0, 6)
    models = [binding.ekya_model_create(0, 6, binding.EKYA_BF16) for _ in counts]
    try:
        weights = [_rotated(w0, i % 6, 0.01 * i) for i in range(len(counts))]
        for m, w in zip(models, weights):
            binding.ekya_model_load(m, w)
        lab, ver = binding.ekya_infer_models(ctx, models, fr, counts, 224)
        torch.cuda.synchronize()
        assert ver == [1] * len(counts)
        off = 0
        for i, c in enumerate(counts):
            if c:
                ref, _ = binding.ekya_infer_model(ctx, models[i], fr[off:off + c].contiguous(), 224)
                torch.cuda.synchronize()
                assert torch.equal(lab[off:off + c], ref), i
            off += c
        print("labels per stream:", [np.bincount(lab[sum(counts[:i]):sum(counts[:i + 1])].cpu()
                                                 .numpy(), minlength=6).tolist()
                                     for i in range(len(counts)) if counts[i]])
        binding.ekya_model_load(models[4], weights[0])
        lab2, ver2 = binding.ekya_infer_models(ctx, models, fr, counts, 224)
        torch.cuda.synchronize()
        assert ver2 == [1, 1, 1, 1, 2, 1, 1, 1, 1, 1]
        s4 = slice(sum(counts[:4]), sum(counts[:5]))
        ref4, _ = binding.ekya_infer_model(ctx, models[0], fr[s4].contiguous(), 224)
        torch.cuda.synchronize()
        assert torch.equal(lab2[s4], ref4)
        keep = torch.ones(1600, dtype=torch.bool, device="cuda")
        keep[s4] = False
        assert torch.equal(lab2[keep], lab[keep])
    finally:
        for m in models:
            binding.ekya_model_destroy(m)
        binding.ekya_destroy(ctx)
