"""Error paths of the C ABI with a real context on the GPU: every argument
out of its documented range returns EKYA_ERR_INVALID_ARG and launches
nothing (weights and label outputs keep their bytes); a context created with
a fixed workspace returns EKYA_ERR_NOMEM before any launch when a call does
not fit, and runs the call when the workspace is the size the host-only
query reports."""
import numpy as np
import pytest

from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu

# (name, k, H, n_heldout, frac, epochs, batch, precision)
BAD = [("k=0", 0, 64, 8, 0.5, 1, 8, 0), ("k=7", 7, 64, 8, 0.5, 1, 8, 0),
       ("frac=0", 2, 64, 8, 0.0, 1, 8, 0), ("frac=1.5", 2, 64, 8, 1.5, 1, 8, 0),
       ("epochs=0", 2, 64, 8, 0.5, 0, 8, 0), ("epochs=65", 2, 64, 8, 0.5, 65, 8, 0),
       ("batch=0", 2, 64, 8, 0.5, 1, 0, 0), ("n_heldout=0", 2, 64, 0, 0.5, 1, 8, 0),
       ("H=31", 2, 31, 8, 0.5, 1, 8, 0), ("precision=2", 2, 64, 8, 0.5, 1, 8, 2)]


@pytest.fixture(scope="module")
def ctx():
    from paper_2012_10557_amd import binding
    c = binding.ekya_create(0, 6)
    yield c
    binding.ekya_destroy(c)


@pytest.fixture(scope="module")
def win():
    import torch
    w = make_window(WindowSpec(16, 8, 64, 64, drift="none", seed=1))
    return {"fr": to_dev(w["frames"], "f32"), "lab": torch.tensor(w["labels"], device="cuda"),
            "hf": to_dev(w["heldout_frames"], "f32"),
            "hl": torch.tensor(w["heldout_labels"], device="cuda"),
            "w0": torch.tensor(kaiming_resnet18_weights(seed=0), device="cuda")}


def _retrain_raw(ctx, w, win, k, H, nh, frac, epochs, batch, prec):
    import ctypes
    from paper_2012_10557_amd import binding
    lib = binding.load()
    opts = binding.TrainOpts(frac, epochs, 0.01, 0.9, batch, 0, prec)
    res = binding.RetrainResult()
    return lib.ekya_retrain(ctx, ctypes.c_void_p(w.data_ptr()), k, ctypes.c_void_p(win["fr"].data_ptr()),
                            ctypes.c_void_p(win["lab"].data_ptr()), 16, H, H,
                            ctypes.c_void_p(win["hf"].data_ptr()), ctypes.c_void_p(win["hl"].data_ptr()),
                            nh, ctypes.byref(opts), ctypes.byref(res), None)


@pytest.mark.parametrize("case", BAD, ids=[c[0] for c in BAD])
def test_retrain_and_profile_reject_invalid_arguments(ctx, win, case):
    import ctypes
    import torch
    from paper_2012_10557_amd import binding
    _, k, H, nh, frac, epochs, batch, prec = case
    w = win["w0"].clone()
    torch.cuda.synchronize()
    assert _retrain_raw(ctx, w, win, k, H, nh, frac, epochs, batch, prec) == binding.EKYA_ERR_INVALID_ARG
    assert binding.load().ekya_last_error(ctx)
    torch.cuda.synchronize()
    assert torch.equal(w, win["w0"])
    cfg = (binding.ProfileCfg * 1)(binding.ProfileCfg(k, frac, epochs, 0.01, 0.9, batch, 0))
    out = (binding.ProfileResult * 1)()
    st = binding.load().ekya_profile(ctx, ctypes.c_void_p(w.data_ptr()), cfg, 1,
                                     ctypes.c_void_p(win["fr"].data_ptr()),
                                     ctypes.c_void_p(win["lab"].data_ptr()), 16, H, H,
                                     ctypes.c_void_p(win["hf"].data_ptr()),
                                     ctypes.c_void_p(win["hl"].data_ptr()), nh, 0, prec, 1, out)
    assert st == binding.EKYA_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.equal(w, win["w0"])


@pytest.mark.parametrize("res,H,prec,n", [(31, 64, 0, 4), (4097, 64, 0, 4), (64, 31, 0, 4),
                                          (64, 64, 2, 4), (64, 64, 0, -1)])
def test_infer_rejects_invalid_arguments(ctx, win, res, H, prec, n):
    import ctypes
    import torch
    from paper_2012_10557_amd import binding
    lab = torch.full((16,), -7, dtype=torch.int32, device="cuda")
    st = binding.load().ekya_infer(ctx, ctypes.c_void_p(win["w0"].data_ptr()),
                                   ctypes.c_void_p(win["fr"].data_ptr()), n, H, H, res, prec,
                                   ctypes.c_void_p(lab.data_ptr()), None)
    assert st == binding.EKYA_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert bool((lab == -7).all())


def test_fixed_workspace_too_small_returns_nomem_before_any_launch(win):
    import torch
    from paper_2012_10557_amd import binding
    need = binding.ekya_retrain_workspace(6, 2, 16, 64, 64, 8, 1.0, 1, 0.01, 0.9, 8, 0, binding.EKYA_FP32)
    assert need > 0
    small = binding.ekya_create(0, 6, workspace_bytes=need // 2)
    try:
        w = win["w0"].clone()
        torch.cuda.synchronize()
        with pytest.raises(binding.EkyaError) as e:
            binding.ekya_retrain(small, w, 2, win["fr"], win["lab"], win["hf"], win["hl"], 1.0, 1, 0.01,
                                 0.9, 8, 0)
        assert e.value.status == binding.EKYA_ERR_NOMEM
        assert "too small" in str(e.value)
        torch.cuda.synchronize()
        assert torch.equal(w, win["w0"])
        lab = torch.full((16,), -7, dtype=torch.int32, device="cuda")
        with pytest.raises(binding.EkyaError) as e:
            binding.ekya_infer(small, win["w0"], win["fr"], 64, labels_out=lab)
        assert e.value.status == binding.EKYA_ERR_NOMEM
        torch.cuda.synchronize()
        assert bool((lab == -7).all())
    finally:
        binding.ekya_destroy(small)


def test_fixed_workspace_of_the_queried_size_runs_every_call_kind(win):
    """One arena sized for the largest of a retraining, a profiling and an
    inference call serves all three, call after call, and the results equal
    a context that sizes its arena itself."""
    import torch
    from paper_2012_10557_amd import binding
    cfgs = [{"k": k, "subsample_frac": 0.5, "epochs": 2, "batch": 4, "seed": 3} for k in (1, 2, 6)]
    need = max(binding.ekya_retrain_workspace(6, 6, 16, 64, 64, 8, 1.0, 2, 0.01, 0.9, 8, 0, binding.EKYA_FP32),
               binding.ekya_profile_workspace(6, cfgs, 16, 64, 64, 8, binding.EKYA_FP32),
               binding.ekya_infer_workspace(6, 48, binding.EKYA_FP32))
    fixed = binding.ekya_create(0, 6, workspace_bytes=need)
    grow = binding.ekya_create(0, 6)
    try:
        outs = []
        for c in (fixed, grow):
            w = win["w0"].clone()
            r = binding.ekya_retrain(c, w, 6, win["fr"], win["lab"], win["hf"], win["hl"], 1.0, 2, 0.01, 0.9, 8, 0)
            p = binding.ekya_profile(c, win["w0"], cfgs, win["fr"], win["lab"], win["hf"], win["hl"], 5)
            lab = binding.ekya_infer(c, w, win["hf"], 48)
            torch.cuda.synchronize()
            outs.append((r["epoch_loss"], w.clone(), [q["epoch_loss"] for q in p], lab.clone()))
        assert outs[0][0] == outs[1][0]
        assert torch.equal(outs[0][1], outs[1][1])
        assert outs[0][2] == outs[1][2]
        assert torch.equal(outs[0][3], outs[1][3])
    finally:
        binding.ekya_destroy(fixed)
        binding.ekya_destroy(grow)
