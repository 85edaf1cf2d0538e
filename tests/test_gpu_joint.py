"""The joint window (sections 3.1 and 4.1: inference and retraining of a
stream share the GPU during a window): batched inference on one stream beside
a layer3+ retraining job (batch 128, 10% of a 3600-frame window, 5 epochs) in
a second context on another stream, at the same time.  Every label and every
retraining result must be bitwise those of the same calls run alone; the
inference rate alone and beside the retraining is printed."""
import threading
import time

import pytest

from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def data():
    import torch
    win = make_window(WindowSpec(3600, 400, 224, 224, drift="drift", seed=2))
    fr = to_dev(win["frames"], "bf16")
    return {"fr": fr, "lab": torch.tensor(win["labels"], device="cuda"),
            "hf": to_dev(win["heldout_frames"], "bf16"),
            "hl": torch.tensor(win["heldout_labels"], device="cuda"),
            "w0": torch.tensor(kaiming_resnet18_weights(seed=0), device="cuda"),
            # inference frames: the window seen twice, sampled at 1/2 (3600 frames)
            "inf": fr.repeat(2, 1, 1, 1)[::2].contiguous()}


@pytest.mark.parametrize("res", [224, 112])
def test_inference_beside_retraining_is_bitwise_unchanged(data, res):
    import torch
    from paper_2012_10557_amd import binding
    d = data
    ictx, rctx = binding.ekya_create(0, 6), binding.ekya_create(0, 6)
    s_inf, s_tr = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        def retrain(box):
            box["out"] = binding.ekya_retrain(rctx, box["w"], 3, d["fr"], d["lab"], d["hf"], d["hl"],
                                              0.1, 5, 0.01, 0.9, 128, 0, stream=s_tr, step_losses=True)
        # alone
        lab_ref = binding.ekya_infer(ictx, d["w0"], d["inf"], res, stream=s_inf)
        s_inf.synchronize()
        t0 = time.perf_counter()
        binding.ekya_infer(ictx, d["w0"], d["inf"], res, labels_out=lab_ref, stream=s_inf)
        s_inf.synchronize()
        alone = d["inf"].shape[0] / (time.perf_counter() - t0)
        ref = {"w": d["w0"].clone()}
        torch.cuda.synchronize()
        retrain(ref)
        torch.cuda.synchronize()
        # together
        for rep in range(2):
            box = {"w": d["w0"].clone()}
            torch.cuda.synchronize()
            th = threading.Thread(target=retrain, args=(box,))
            th.start()
            t0 = time.perf_counter()
            lab = binding.ekya_infer(ictx, d["w0"], d["inf"], res, stream=s_inf)
            s_inf.synchronize()
            together = d["inf"].shape[0] / (time.perf_counter() - t0)
            th.join()
            torch.cuda.synchronize()
            print(f"{res}px: inference {alone:.0f} img/s alone, {together:.0f} img/s beside the "
                  f"retraining job; retraining steps {box['out']['n_steps']}")
            assert torch.equal(lab, lab_ref)
            assert torch.equal(box["w"], ref["w"])
            assert box["out"]["step_loss"] == ref["out"]["step_loss"]
            assert box["out"]["heldout_acc"] == ref["out"]["heldout_acc"]
    finally:
        binding.ekya_destroy(ictx)
        binding.ekya_destroy(rctx)
