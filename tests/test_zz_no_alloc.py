"""The allocation-free BatchNorm entry point (ekya_op_batchnorm_train_noalloc,
scratch in a static device array) against ekya_op_batchnorm_train on the
same inputs: two calls in a row, the second smaller (the scratch keeps the
first call's contents), in the large-batch (partial, final, apply) and the
small-batch (partial, fold-apply) paths; outputs and running statistics
must be bitwise equal."""
import pytest

pytestmark = pytest.mark.gpu


def _inputs(M, C, prec, seed):
    import torch
    g = torch.Generator().manual_seed(seed)
    z = (torch.randn(M, C, generator=g) * 2 + 0.5).to("cuda")
    z = z.to(torch.bfloat16) if prec == "bf16" else z
    gamma = (torch.rand(C, generator=g) + 0.5).to("cuda")
    beta = torch.randn(C, generator=g).to("cuda")
    rm = torch.randn(C, generator=g).to("cuda")
    rv = (torch.rand(C, generator=g) + 0.5).to("cuda")
    return z, gamma, beta, rm, rv


@pytest.mark.parametrize("prec", ["f32", "bf16"])
def test_noalloc_batchnorm_equals_allocating_entry_point(prec):
    import torch
    from paper_2012_10557_amd import binding
    for i, (M, C, relu) in enumerate([(20000, 128, True), (3000, 64, False)]):
        z, gamma, beta, rm, rv = _inputs(M, C, prec, 11 + i)
        rm1, rv1, rm2, rv2 = rm.clone(), rv.clone(), rm.clone(), rv.clone()
        y1, m1, s1 = binding.ekya_op_batchnorm_train(z, gamma, beta, rm1, rv1, relu=relu)
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            y2, m2, s2 = binding.ekya_op_batchnorm_train_noalloc(z, gamma, beta, rm2, rv2, relu=relu,
                                                                stream=s)
        s.synchronize()
        assert torch.equal(y1, y2), (M, C)
        assert torch.equal(m1, m2) and torch.equal(s1, s2), (M, C)
        assert torch.equal(rm1, rm2) and torch.equal(rv1, rv2), (M, C)
        assert not torch.equal(rm1, rm), "running statistics were updated"


def test_noalloc_batchnorm_rejects_invalid_arguments():
    import ctypes
    from paper_2012_10557_amd import binding
    lib = binding.load()
    st = lib.ekya_op_batchnorm_train_noalloc(1, ctypes.c_void_p(16), 100, 4096, ctypes.c_void_p(16),
                                             ctypes.c_void_p(16), None, None, 0, ctypes.c_void_p(16),
                                             ctypes.c_void_p(16), ctypes.c_void_p(16), None)
    assert st == binding.EKYA_ERR_INVALID_ARG
