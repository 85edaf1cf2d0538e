"""Host-side checks of the C-ABI library: it loads, exports every symbol the
headers declare, validates arguments before any GPU work, and its seeded
subset / shuffle draws equal the oracle's independent implementation."""
import ctypes
import os
import re

import pytest

from oracle import rng
from oracle.resnet18 import ResNet18

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2012_10557_amd", "libekya.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libekya.so not built")


def _declared_symbols():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        with open(os.path.join(ROOT, "include", h)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(ekya_\w+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    from paper_2012_10557_amd import binding
    lib = binding.load()
    declared = _declared_symbols()
    assert len(declared) >= 20
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == set(binding.exported_symbols())


def test_weights_count_matches_oracle_layout():
    from paper_2012_10557_amd import binding
    assert binding.ekya_weights_count(6) == ResNet18(6).n_weights() == 11_189_190
    assert binding.ekya_weights_count(10) == ResNet18(10).n_weights()
    assert binding.ekya_weights_count(0) == 0


@pytest.mark.parametrize("n,frac,seed", [(2000, 0.3, 0), (4000, 0.05, 7), (4000, 0.10, 7),
                                         (64, 1.0, 0), (3600, 0.1, 123456789012345)])
def test_subset_matches_oracle(n, frac, seed):
    from paper_2012_10557_amd import binding
    assert binding.ekya_training_subset(n, frac, seed) == rng.training_subset(n, frac, seed)


@pytest.mark.parametrize("n,seed,epoch", [(600, 0, 0), (600, 0, 4), (200, 99, 1), (1, 5, 0)])
def test_epoch_order_matches_oracle(n, seed, epoch):
    from paper_2012_10557_amd import binding
    assert binding.ekya_epoch_order(n, seed, epoch) == rng.epoch_order(n, seed, epoch)


def test_invalid_arguments_rejected_before_gpu_work():
    from paper_2012_10557_amd import binding
    lib = binding.load()
    opts = binding.TrainOpts(0.3, 5, 0.01, 0.9, 64, 0, 1)
    res = binding.RetrainResult()
    st = lib.ekya_retrain(None, None, 2, None, None, 10, 224, 224, None, None, 4,
                          ctypes.byref(opts), ctypes.byref(res), None)
    assert st == binding.EKYA_ERR_INVALID_ARG
    assert b"ctx" in lib.ekya_last_error(None)
    assert lib.ekya_infer(None, None, None, 4, 224, 224, 224, 1, None, None) == binding.EKYA_ERR_INVALID_ARG
    h = ctypes.c_void_p()
    assert lib.ekya_create(ctypes.byref(h), 0, 0, 0) == binding.EKYA_ERR_INVALID_ARG
    assert lib.ekya_create(None, 0, 6, 0) == binding.EKYA_ERR_INVALID_ARG
    assert lib.ekya_training_subset(10, 0.0, 0, None, 0) == -1
    # op-level validation: channel count not a multiple of the unit
    assert lib.ekya_op_conv2d(1, ctypes.c_void_p(16), 1, 8, 8, 12, ctypes.c_void_p(16), 16, 3, 3, 1, 1,
                              ctypes.c_void_p(16), None) == binding.EKYA_ERR_INVALID_ARG
    assert lib.ekya_op_sgd(None, None, None, 4, 0.1, 0.9, None) == binding.EKYA_ERR_INVALID_ARG
    for s in range(6):
        assert lib.ekya_status_str(s)


# (name, k, n_frames, H, n_heldout, frac, epochs, batch, precision): each one
# argument out of its documented range
BAD_RETRAIN = [("k=0", 0, 400, 224, 40, 0.5, 2, 64, 1), ("k=7", 7, 400, 224, 40, 0.5, 2, 64, 1),
               ("frac=0", 2, 400, 224, 40, 0.0, 2, 64, 1), ("frac=1.5", 2, 400, 224, 40, 1.5, 2, 64, 1),
               ("epochs=0", 2, 400, 224, 40, 0.5, 0, 64, 1), ("epochs=65", 2, 400, 224, 40, 0.5, 65, 64, 1),
               ("batch=0", 2, 400, 224, 40, 0.5, 2, 0, 1), ("n_heldout=0", 2, 400, 224, 0, 0.5, 2, 64, 1),
               ("H=31", 2, 400, 31, 40, 0.5, 2, 64, 1), ("precision=2", 2, 400, 224, 40, 0.5, 2, 64, 2),
               ("n_frames=0", 2, 0, 224, 40, 0.5, 2, 64, 1)]


@pytest.mark.parametrize("case", BAD_RETRAIN, ids=[c[0] for c in BAD_RETRAIN])
def test_workspace_query_rejects_invalid_retrain(case):
    """The workspace size queries validate exactly like the calls they size
    (0 = the call would return EKYA_ERR_INVALID_ARG); host only."""
    from paper_2012_10557_amd import binding
    _, k, n, H, nh, frac, ep, b, prec = case
    assert binding.ekya_retrain_workspace(6, k, n, H, H, nh, frac, ep, 0.01, 0.9, b, 0, prec) == 0
    cfg = {"k": k, "subsample_frac": frac, "epochs": ep, "batch": b}
    assert binding.ekya_profile_workspace(6, [cfg], n, H, H, nh, prec) == 0


def test_workspace_query_sizes():
    """Sizes are positive for valid calls and grow with what they hold: the
    batch's activations, the feature cache (more frames, shallower frozen
    prefix), one job per profiler candidate; inference needs the same
    workspace for any number of frames and less at lower resolution."""
    from paper_2012_10557_amd import binding
    r = lambda k, n, b, ep=2: binding.ekya_retrain_workspace(6, k, n, 224, 224, 400, 1.0, ep, 0.01, 0.9, b)
    assert r(6, 4000, 128) > r(6, 4000, 64) > 0
    assert r(3, 4000, 128) > r(3, 2000, 128) > 0          # cache rows
    assert r(2, 2000, 64) < r(3, 2000, 64)                  # layer4 input rows are smaller
    assert r(2, 2000, 64, 10) > r(2, 2000, 64, 1)           # per-epoch orders and losses
    c = [{"k": k, "subsample_frac": f, "epochs": e, "batch": 64}
         for k in (1, 2, 3, 6) for f in (0.05, 0.1) for e in (1, 2)]
    total = binding.ekya_profile_workspace(6, c, 4000, 224, 224, 400)
    one = binding.ekya_profile_workspace(6, c[-1:], 4000, 224, 224, 400)
    assert total > one > 0
    i224 = binding.ekya_infer_workspace(6, 224)
    assert i224 > binding.ekya_infer_workspace(6, 160) > binding.ekya_infer_workspace(6, 112) > 0
    assert binding.ekya_infer_workspace(6, 31) == 0 and binding.ekya_infer_workspace(6, 224, 2) == 0
    assert binding.ekya_infer_workspace(0, 224) == 0
