"""Model checkpointing and reloading (section 5): retrained weights are loaded
into the inference job while it keeps serving.  An ekya_model holds two
prepared slots; checked here: a loaded model exports bitwise the weights it
was loaded from and classifies bitwise as ekya_infer with them; loads issued
while inference calls are queued switch later calls to the new weights
without touching the calls already issued (each call's labels equal the
reference of the version it reports, across three loads that recycle a
slot); checkpoints published by ekya_retrain after every epoch leave the
retraining bitwise unchanged, and the last one exports the retrained
weights."""
import threading

import pytest

from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu

N_CLASSES = 6
FC = N_CLASSES * 512 + N_CLASSES


def _rotated_classes(w, shift):
    """The same network with its classifier's rows (and biases) rotated by
    `shift` classes: its labels are the first network's, rotated."""
    import torch
    w2 = w.clone()
    fw = w2[-FC:-N_CLASSES].view(N_CLASSES, 512)
    fb = w2[-N_CLASSES:]
    fw.copy_(torch.roll(fw, shift, 0))
    fb.copy_(torch.roll(fb, shift, 0) + 0.05)
    return w2


@pytest.fixture(scope="module")
def data():
    import torch
    win = make_window(WindowSpec(1200, 200, 224, 224, drift="drift", seed=5))
    return {"fr": to_dev(win["frames"], "bf16"),
            "lab": torch.tensor(win["labels"], device="cuda"),
            "hf": to_dev(win["heldout_frames"], "bf16"),
            "hl": torch.tensor(win["heldout_labels"], device="cuda"),
            "w0": torch.tensor(kaiming_resnet18_weights(seed=0), device="cuda")}


@pytest.mark.parametrize("res", [224, 112])
def test_loaded_model_equals_its_weights(data, res):
    import torch
    from paper_2012_10557_amd import binding
    d = data
    ctx = binding.ekya_create(0, N_CLASSES)
    m = binding.ekya_model_create(0, N_CLASSES, binding.EKYA_BF16)
    try:
        assert binding.ekya_model_version(m) == 0
        with pytest.raises(binding.EkyaError):
            binding.ekya_infer_model(ctx, m, d["fr"][:8].contiguous(), res)
        out = torch.empty_like(d["w0"])
        with pytest.raises(binding.EkyaError):
            binding.ekya_model_export(m, out)
        w2 = _rotated_classes(d["w0"], 2)
        for k, w in enumerate([d["w0"], w2, d["w0"]]):
            assert binding.ekya_model_load(m, w) == k + 1
            assert binding.ekya_model_export(m, out) == k + 1
            lab, v = binding.ekya_infer_model(ctx, m, d["fr"], res)
            ref = binding.ekya_infer(ctx, w, d["fr"], res)
            torch.cuda.synchronize()
            assert v == k + 1
            assert torch.equal(out, w)
            assert torch.equal(lab, ref)
    finally:
        binding.ekya_model_destroy(m)
        binding.ekya_destroy(ctx)


def test_fp32_model_matches_fp32_inference():
    import torch
    from paper_2012_10557_amd import binding
    win = make_window(WindowSpec(96, 1, 64, 64, drift="none", seed=3))
    fr = to_dev(win["frames"])
    w = torch.tensor(kaiming_resnet18_weights(seed=1), device="cuda")
    ctx = binding.ekya_create(0, N_CLASSES)
    m = binding.ekya_model_create(0, N_CLASSES, binding.EKYA_FP32)
    try:
        binding.ekya_model_load(m, w)
        lab, _ = binding.ekya_infer_model(ctx, m, fr, 64)
        ref = binding.ekya_infer(ctx, w, fr, 64)
        torch.cuda.synchronize()
        assert torch.equal(lab, ref)
    finally:
        binding.ekya_model_destroy(m)
        binding.ekya_destroy(ctx)


def test_reload_while_inference_is_queued(data):
    """24 inference calls of 100 frames are issued back to back on one stream;
    three loads (w1, w2, then w1 again, which overwrites the slot of the first
    load) are issued from a second thread on another stream in between.
    Every call's labels equal ekya_infer's for the version it reports, the
    versions never decrease, and the last calls run on the last load."""
    import torch
    from paper_2012_10557_amd import binding
    d = data
    w1, w2 = d["w0"], _rotated_classes(d["w0"], 3)
    chunks = [d["fr"][i * 50:i * 50 + 100].contiguous() for i in range(24)]
    ctx = binding.ekya_create(0, N_CLASSES)
    rctx = binding.ekya_create(0, N_CLASSES)
    m = binding.ekya_model_create(0, N_CLASSES, binding.EKYA_BF16)
    s_inf, s_load = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        refs = {}
        for tag, w in (("w1", w1), ("w2", w2)):
            refs[tag] = [binding.ekya_infer(rctx, w, c, 224) for c in chunks]
        torch.cuda.synchronize()
        version_weights = {}
        version_weights[binding.ekya_model_load(m, w1, stream=s_load)] = "w1"
        issued = threading.Event()
        go = [threading.Event() for _ in range(3)]
        results = []

        def serve():
            for i, c in enumerate(chunks):
                results.append(binding.ekya_infer_model(ctx, m, c, 224, stream=s_inf))
                if i in (5, 11, 17):
                    go[(i - 5) // 6].set()
                    issued.wait(timeout=60)
                    issued.clear()

        th = threading.Thread(target=serve)
        th.start()
        for k, (w, tag) in enumerate([(w2, "w2"), (w1, "w1"), (w2, "w2")]):
            assert go[k].wait(timeout=60)
            version_weights[binding.ekya_model_load(m, w, stream=s_load)] = tag
            issued.set()
        th.join()
        torch.cuda.synchronize()
        versions = [v for _, v in results]
        print("versions per call:", versions)
        assert versions == sorted(versions)
        assert versions[-1] == max(version_weights)
        assert len(set(versions)) == 4
        for i, (lab, v) in enumerate(results):
            assert torch.equal(lab, refs[version_weights[v]][i]), (i, v)
    finally:
        binding.ekya_model_destroy(m)
        binding.ekya_destroy(ctx)
        binding.ekya_destroy(rctx)


def test_checkpoints_during_retraining(data):
    """layer4 + classifier retraining on 50% of a 1200-frame window for 3
    epochs, publishing into a model after every epoch while a second thread
    serves inference from the model: the retraining is bitwise that of an
    unpublished run, three versions are published, the model exports the
    retrained weights, and inference on the last version equals ekya_infer
    with them."""
    import torch
    from paper_2012_10557_amd import binding
    d = data
    rctx, ictx = binding.ekya_create(0, N_CLASSES), binding.ekya_create(0, N_CLASSES)
    m = binding.ekya_model_create(0, N_CLASSES, binding.EKYA_BF16)
    s_tr, s_inf = torch.cuda.Stream(), torch.cuda.Stream()
    args = (2, d["fr"], d["lab"], d["hf"], d["hl"], 0.5, 3, 0.01, 0.9, 64, 7)
    try:
        ref_w = d["w0"].clone()
        ref = binding.ekya_retrain(rctx, ref_w, *args, stream=s_tr, step_losses=True)
        torch.cuda.synchronize()
        binding.ekya_model_load(m, d["w0"], stream=s_tr)
        binding.ekya_set_checkpoint(rctx, m, 1)
        w = d["w0"].clone()
        stop = threading.Event()
        served = []

        def serve():
            while not stop.is_set():
                lab, v = binding.ekya_infer_model(ictx, m, d["fr"][:256].contiguous(), 224,
                                                  stream=s_inf)
                s_inf.synchronize()
                served.append(v)

        th = threading.Thread(target=serve)
        th.start()
        try:
            out = binding.ekya_retrain(rctx, w, *args, stream=s_tr, step_losses=True)
        finally:
            stop.set()
            th.join()
        torch.cuda.synchronize()
        assert binding.ekya_model_version(m) == 4
        assert torch.equal(w, ref_w)
        assert out["step_loss"] == ref["step_loss"]
        assert out["heldout_acc"] == ref["heldout_acc"]
        exported = torch.empty_like(w)
        assert binding.ekya_model_export(m, exported, stream=s_inf) == 4
        lab, v = binding.ekya_infer_model(ictx, m, d["fr"], 224, stream=s_inf)
        s_inf.synchronize()
        ref_lab = binding.ekya_infer(ictx, w, d["fr"], 224, stream=s_inf)
        s_inf.synchronize()
        print(f"versions served during retraining: {sorted(set(served))} over {len(served)} calls")
        assert served == sorted(served)
        assert torch.equal(exported, w)
        assert torch.equal(lab, ref_lab)
        # stopping checkpoints leaves the model alone
        binding.ekya_set_checkpoint(rctx, None, 0)
        binding.ekya_retrain(rctx, w.clone(), *args, stream=s_tr)
        assert binding.ekya_model_version(m) == 4
        # a model of another precision is refused before any work
        m32 = binding.ekya_model_create(0, N_CLASSES, binding.EKYA_FP32)
        try:
            binding.ekya_set_checkpoint(rctx, m32, 1)
            with pytest.raises(binding.EkyaError):
                binding.ekya_retrain(rctx, w.clone(), *args, stream=s_tr)
            binding.ekya_set_checkpoint(rctx, None, 0)
        finally:
            binding.ekya_model_destroy(m32)
    finally:
        binding.ekya_model_destroy(m)
        binding.ekya_destroy(rctx)
        binding.ekya_destroy(ictx)
