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
    for h in ("ekya.h", "ekya_ops.h"):
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
    assert lib.ekya_create(ctypes.byref(h), 0, 0) == binding.EKYA_ERR_INVALID_ARG
    assert lib.ekya_create(None, 0, 6) == binding.EKYA_ERR_INVALID_ARG
    assert lib.ekya_training_subset(10, 0.0, 0, None, 0) == -1
    # op-level validation: channel count not a multiple of the unit
    assert lib.ekya_op_conv2d(1, ctypes.c_void_p(16), 1, 8, 8, 12, ctypes.c_void_p(16), 16, 3, 3, 1, 1,
                              ctypes.c_void_p(16), None) == binding.EKYA_ERR_INVALID_ARG
    assert lib.ekya_op_sgd(None, None, None, 4, 0.1, 0.9, None) == binding.EKYA_ERR_INVALID_ARG
    for s in range(6):
        assert lib.ekya_status_str(s)
