"""ctypes binding of libekya.so: argument marshalling only.

Every function mirrors the C entry point of the same name in include/ekya.h or
include/ekya_ops.h.  Tensors are torch tensors on the GPU (PyTorch is used for
device memory and streams); their data pointers and the current HIP stream are
handed to the library, which runs every step of the path in its own kernels.
The library must be built (python -m paper_2012_10557_amd.build); importing
this module without it raises an error.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libekya.so")

EKYA_OK = 0
EKYA_ERR_INVALID_ARG = 1
EKYA_ERR_NOMEM = 2
EKYA_ERR_HIP = 3
EKYA_ERR_NONFINITE = 4
EKYA_ERR_UNSUPPORTED = 5
EKYA_FP32 = 0
EKYA_BF16 = 1
EKYA_MAX_EPOCHS = 64


class EkyaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"ekya status {status}: {msg}")
        self.status = status


class TrainOpts(ctypes.Structure):
    _fields_ = [("subsample_frac", ctypes.c_double), ("epochs", ctypes.c_int),
                ("lr", ctypes.c_float), ("momentum", ctypes.c_float), ("batch", ctypes.c_int),
                ("seed", ctypes.c_uint64), ("precision", ctypes.c_int)]


class RetrainResult(ctypes.Structure):
    _fields_ = [("n_train", ctypes.c_int), ("n_epochs", ctypes.c_int), ("n_steps", ctypes.c_int),
                ("heldout_acc_final", ctypes.c_float),
                ("heldout_acc", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("epoch_seconds", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("eval_seconds", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("epoch_loss", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("prefix_seconds", ctypes.c_float),
                ("step_loss", ctypes.POINTER(ctypes.c_float)),
                ("step_loss_capacity", ctypes.c_int)]


class ProfileCfg(ctypes.Structure):
    _fields_ = [("k_trainable", ctypes.c_int), ("subsample_frac", ctypes.c_double),
                ("epochs", ctypes.c_int), ("lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("batch", ctypes.c_int), ("shuffle_seed", ctypes.c_uint64)]


class ProfileResult(ctypes.Structure):
    _fields_ = [("status", ctypes.c_int), ("n_train", ctypes.c_int),
                ("heldout_acc", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("epoch_seconds", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("eval_seconds", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("epoch_loss", ctypes.c_float * EKYA_MAX_EPOCHS),
                ("heldout_acc_final", ctypes.c_float)]


class Curve(ctypes.Structure):
    _fields_ = [("b0", ctypes.c_double), ("b1", ctypes.c_double), ("b2", ctypes.c_double),
                ("rss", ctypes.c_double)]


class InferCfg(ctypes.Structure):
    _fields_ = [("cost", ctypes.c_double), ("factor", ctypes.c_double)]


class TrainCfg(ctypes.Structure):
    _fields_ = [("acc_after", ctypes.c_double), ("gpu_seconds", ctypes.c_double)]


class VideoIn(ctypes.Structure):
    _fields_ = [("acc_now", ctypes.c_double), ("infer", ctypes.POINTER(InferCfg)),
                ("n_infer", ctypes.c_int), ("train", ctypes.POINTER(TrainCfg)),
                ("n_train", ctypes.c_int)]


class ScheduleOut(ctypes.Structure):
    _fields_ = [("alloc", ctypes.POINTER(ctypes.c_double)), ("infer_choice", ctypes.POINTER(ctypes.c_int)),
                ("train_choice", ctypes.POINTER(ctypes.c_int)),
                ("video_accuracy", ctypes.POINTER(ctypes.c_double)), ("accuracy", ctypes.c_double)]


_P = ctypes.c_void_p
_I = ctypes.c_int
_LL = ctypes.c_longlong
_F = ctypes.c_float

# name -> (restype, argtypes)
_SIGS = {
    "ekya_create": (_I, [ctypes.POINTER(_P), _I, _I, ctypes.c_size_t]),
    "ekya_create_head": (_I, [ctypes.POINTER(_P), _I, _I, _I, ctypes.c_size_t]),
    "ekya_weights_count_head": (ctypes.c_size_t, [_I, _I]),
    "ekya_retrain_workspace_head": (ctypes.c_size_t, [_I, _I, _I, _I, _I, _I, _I,
                                                      ctypes.POINTER(TrainOpts)]),
    "ekya_profile_workspace_head": (ctypes.c_size_t, [_I, _I, ctypes.POINTER(ProfileCfg), _I, _I,
                                                      _I, _I, _I, _I]),
    "ekya_infer_workspace_head": (ctypes.c_size_t, [_I, _I, _I, _I]),
    "ekya_model_create_head": (_I, [ctypes.POINTER(_P), _I, _I, _I, _I]),
    "ekya_destroy": (None, [_P]),
    "ekya_weights_count": (ctypes.c_size_t, [_I]),
    "ekya_status_str": (ctypes.c_char_p, [_I]),
    "ekya_last_error": (ctypes.c_char_p, [_P]),
    "ekya_retrain_workspace": (ctypes.c_size_t, [_I, _I, _I, _I, _I, _I, ctypes.POINTER(TrainOpts)]),
    "ekya_profile_workspace": (ctypes.c_size_t, [_I, ctypes.POINTER(ProfileCfg), _I, _I, _I, _I, _I,
                                                 _I]),
    "ekya_infer_workspace": (ctypes.c_size_t, [_I, _I, _I]),
    "ekya_retrain": (_I, [_P, _P, _I, _P, _P, _I, _I, _I, _P, _P, _I, ctypes.POINTER(TrainOpts),
                          ctypes.POINTER(RetrainResult), _P]),
    "ekya_profile": (_I, [_P, _P, ctypes.POINTER(ProfileCfg), _I, _P, _P, _I, _I, _I, _P, _P, _I,
                          ctypes.c_uint64, _I, _I, ctypes.POINTER(ProfileResult)]),
    "ekya_infer": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "ekya_set_kernel_timing": (_I, [_P, _I]),
    "ekya_kernel_timing": (_I, [_P, _I, ctypes.c_char_p, _I, ctypes.POINTER(_LL),
                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                ctypes.POINTER(ctypes.c_double)]),
    "ekya_training_subset": (_I, [_I, ctypes.c_double, ctypes.c_uint64, _P, _I]),
    "ekya_epoch_order": (_I, [_I, ctypes.c_uint64, _I, _P]),
    "ekya_nnls": (_I, [_P, _I, _I, _P, _P, _P]),
    "ekya_fit_accuracy_curve": (_I, [_P, _P, _I, ctypes.POINTER(Curve)]),
    "ekya_curve_accuracy": (ctypes.c_double, [ctypes.POINTER(Curve), ctypes.c_double]),
    "ekya_extrapolate": (_I, [ctypes.POINTER(ProfileCfg), ctypes.POINTER(ProfileResult), _I, _I,
                              ctypes.POINTER(Curve), ctypes.POINTER(ctypes.c_double),
                              ctypes.POINTER(ctypes.c_double)]),
    "ekya_thief_schedule": (_I, [ctypes.POINTER(VideoIn), _I, ctypes.c_double, ctypes.c_double,
                                 ctypes.c_double, ctypes.c_double, ctypes.POINTER(ScheduleOut)]),
    "ekya_partition_mask": (_I, [_I, _I, _I, ctypes.c_double, ctypes.c_double, _P, _I]),
    "ekya_stream_create": (_I, [_I, ctypes.c_double, ctypes.c_double, ctypes.POINTER(_P)]),
    "ekya_stream_destroy": (_I, [_P]),
    "ekya_stream_cu_count": (_I, [_P]),
    "ekya_set_cu_partition": (_I, [_P, ctypes.c_double, ctypes.c_double]),
    "ekya_cu_ids": (_I, [_I, _P, _P]),
    "ekya_model_create": (_I, [ctypes.POINTER(_P), _I, _I, _I]),
    "ekya_model_destroy": (None, [_P]),
    "ekya_model_load": (_I, [_P, _P, _P, ctypes.POINTER(ctypes.c_uint64)]),
    "ekya_model_export": (_I, [_P, _P, _P, ctypes.POINTER(ctypes.c_uint64)]),
    "ekya_model_version": (ctypes.c_uint64, [_P]),
    "ekya_infer_model": (_I, [_P, _P, _P, _I, _I, _I, _I, _P, _P, ctypes.POINTER(ctypes.c_uint64)]),
    "ekya_set_checkpoint": (_I, [_P, _P, _I]),
    "ekya_infer_models": (_I, [_P, _P, _I, _P, _P, _I, _I, _I, _P, _P, _P]),
    "ekya_infer_models_workspace": (ctypes.c_size_t, [_I, _I, _I, _I, _I]),
    "ekya_op_conv2d": (_I, [_I, _P, _I, _I, _I, _I, _P, _I, _I, _I, _I, _I, _P, _P]),
    "ekya_op_conv2d_dgrad": (_I, [_I, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P]),
    "ekya_op_conv2d_wgrad": (_I, [_I, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P]),
    "ekya_op_batchnorm_train": (_I, [_I, _P, _LL, _I, _P, _P, _P, _P, _I, _P, _P, _P, _P]),
    "ekya_op_batchnorm_train_noalloc": (_I, [_I, _P, _LL, _I, _P, _P, _P, _P, _I, _P, _P, _P, _P]),
    "ekya_op_batchnorm_backward": (_I, [_I, _P, _P, _P, _LL, _I, _P, _P, _P, _P, _P, _P, _P]),
    "ekya_op_maxpool": (_I, [_I, _P, _I, _I, _I, _I, _P, _P, _P]),
    "ekya_op_maxpool_backward": (_I, [_I, _P, _P, _I, _I, _I, _I, _P, _P]),
    "ekya_op_avgpool": (_I, [_I, _P, _I, _I, _I, _I, _P, _P]),
    "ekya_op_avgpool_backward": (_I, [_I, _P, _I, _I, _I, _I, _P, _P]),
    "ekya_op_linear": (_I, [_P, _P, _P, _I, _I, _I, _P, _P]),
    "ekya_op_linear_backward": (_I, [_P, _P, _P, _I, _I, _I, _P, _P, _P, _P]),
    "ekya_op_softmax_ce": (_I, [_P, _P, _I, _I, _P, _P, _P]),
    "ekya_op_sgd": (_I, [_P, _P, _P, _LL, _F, _F, _P]),
    "ekya_op_resize": (_I, [_I, _P, _I, _I, _I, _I, _P, _P]),
}

_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libekya.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with python -m paper_2012_10557_amd.build")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def exported_symbols() -> List[str]:
    return list(_SIGS)


def _check(status: int, ctx=None):
    if status != EKYA_OK:
        lib = load()
        msg = lib.ekya_last_error(ctx).decode() if lib.ekya_last_error(ctx) else ""
        raise EkyaError(status, msg or lib.ekya_status_str(status).decode())


# -------------------------------------------------------------- tensors
def _torch():
    import torch
    return torch


def _precision(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return EKYA_FP32
    if t.dtype == torch.bfloat16:
        return EKYA_BF16
    raise TypeError(f"frames must be float32 or bfloat16, got {t.dtype}")


def _dev(t, dtype=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


# ------------------------------------------------------------ context
def ekya_create(device: int = 0, n_classes: int = 6, workspace_bytes: int = 0, hidden: int = 0):
    """A context; hidden > 0 gives the network a hidden classifier layer."""
    lib = load()
    h = ctypes.c_void_p()
    if hidden:
        _check(lib.ekya_create_head(ctypes.byref(h), device, n_classes, hidden, workspace_bytes))
    else:
        _check(lib.ekya_create(ctypes.byref(h), device, n_classes, workspace_bytes))
    return h


def _profile_cfgs(cfgs: Sequence[dict]):
    arr = (ProfileCfg * len(cfgs))()
    for i, c in enumerate(cfgs):
        arr[i] = ProfileCfg(c["k"], c["subsample_frac"], c["epochs"], c.get("lr", 0.01),
                            c.get("momentum", 0.9), c.get("batch", 64), c.get("seed", 0))
    return arr


def ekya_retrain_workspace(n_classes: int, k_trainable: int, n_frames: int, H: int, W: int,
                           n_heldout: int, subsample_frac: float, epochs: int, lr: float,
                           momentum: float = 0.9, batch: int = 64, seed: int = 0,
                           precision: int = EKYA_BF16, hidden: int = 0) -> int:
    opts = TrainOpts(subsample_frac, epochs, lr, momentum, batch, seed, precision)
    return int(load().ekya_retrain_workspace_head(n_classes, hidden, k_trainable, n_frames, H, W,
                                                  n_heldout, ctypes.byref(opts)))


def ekya_profile_workspace(n_classes: int, cfgs: Sequence[dict], n_frames: int, H: int, W: int,
                           n_heldout: int, precision: int = EKYA_BF16, hidden: int = 0) -> int:
    return int(load().ekya_profile_workspace_head(n_classes, hidden, _profile_cfgs(cfgs), len(cfgs),
                                                  n_frames, H, W, n_heldout, precision))


def ekya_infer_workspace(n_classes: int, resolution: int, precision: int = EKYA_BF16,
                         hidden: int = 0) -> int:
    return int(load().ekya_infer_workspace_head(n_classes, hidden, resolution, precision))


def ekya_destroy(ctx) -> None:
    load().ekya_destroy(ctx)


def ekya_weights_count(n_classes: int = 6, hidden: int = 0) -> int:
    return int(load().ekya_weights_count_head(n_classes, hidden))


def ekya_set_kernel_timing(ctx, enable: bool) -> None:
    _check(load().ekya_set_kernel_timing(ctx, 1 if enable else 0), ctx)


def ekya_kernel_timing(ctx) -> List[dict]:
    """All timed GEMM kernels: name, launches, total_ms, flops, bytes."""
    lib = load()
    out = []
    i = 0
    while True:
        name = ctypes.create_string_buffer(256)
        n = _LL()
        ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        if lib.ekya_kernel_timing(ctx, i, name, 256, ctypes.byref(n), ctypes.byref(ms),
                                  ctypes.byref(fl), ctypes.byref(by)) != 0:
            break
        out.append({"name": name.value.decode(), "launches": n.value, "total_ms": ms.value,
                    "flops": fl.value, "bytes": by.value})
        i += 1
    return out


def ekya_training_subset(n_frames: int, subsample_frac: float, seed: int) -> List[int]:
    import numpy as np
    out = np.zeros(max(1, n_frames), dtype=np.int32)
    n = load().ekya_training_subset(n_frames, subsample_frac, seed, out.ctypes.data, out.size)
    if n < 0:
        raise ValueError("invalid subset arguments")
    return out[:n].tolist()


def ekya_epoch_order(n: int, seed: int, epoch: int) -> List[int]:
    import numpy as np
    out = np.zeros(n, dtype=np.int32)
    if load().ekya_epoch_order(n, seed, epoch, out.ctypes.data) != 0:
        raise ValueError("invalid epoch order arguments")
    return out.tolist()


def ekya_retrain(ctx, weights, k_trainable: int, frames, labels, heldout_frames, heldout_labels,
                 subsample_frac: float, epochs: int, lr: float, momentum: float = 0.9,
                 batch: int = 64, seed: int = 0, stream=None, step_losses: bool = False) -> dict:
    torch = _torch()
    lib = load()
    prec = _precision(frames)
    n, H, W, C = frames.shape
    if C != 3 or tuple(heldout_frames.shape[1:]) != (H, W, 3):
        raise ValueError("frames must be [n, H, W, 3] and held-out frames match")
    opts = TrainOpts(subsample_frac, epochs, lr, momentum, batch, seed, prec)
    res = RetrainResult()
    n_s = max(1, int(subsample_frac * n + 0.5))
    steps = epochs * -(-n_s // batch)
    buf = (ctypes.c_float * steps)() if step_losses else None
    if buf is not None:
        res.step_loss = ctypes.cast(buf, ctypes.POINTER(ctypes.c_float))
        res.step_loss_capacity = steps
    st = lib.ekya_retrain(ctx, _dev(weights, torch.float32), k_trainable, _dev(frames),
                          _dev(labels, torch.int32), n, H, W, _dev(heldout_frames, frames.dtype),
                          _dev(heldout_labels, torch.int32), heldout_frames.shape[0],
                          ctypes.byref(opts), ctypes.byref(res), _stream(stream))
    _check(st, ctx)
    ne = res.n_epochs
    out = {"n_train": res.n_train, "n_epochs": ne, "n_steps": res.n_steps,
           "heldout_acc_final": res.heldout_acc_final,
           "heldout_acc": list(res.heldout_acc[:ne]), "epoch_seconds": list(res.epoch_seconds[:ne]),
           "eval_seconds": list(res.eval_seconds[:ne]),
           "epoch_loss": list(res.epoch_loss[:ne]), "prefix_seconds": res.prefix_seconds}
    if buf is not None:
        out["step_loss"] = list(buf[:res.n_steps])
    return out


def ekya_profile(ctx, weights, cfgs: Sequence[dict], frames, labels, heldout_frames,
                 heldout_labels, subsample_seed: int = 0, concurrent: bool = True) -> List[dict]:
    torch = _torch()
    lib = load()
    prec = _precision(frames)
    n, H, W, _ = frames.shape
    arr = _profile_cfgs(cfgs)
    res = (ProfileResult * len(cfgs))()
    st = lib.ekya_profile(ctx, _dev(weights, torch.float32), arr, len(cfgs), _dev(frames),
                          _dev(labels, torch.int32), n, H, W, _dev(heldout_frames, frames.dtype),
                          _dev(heldout_labels, torch.int32), heldout_frames.shape[0],
                          subsample_seed, prec, 1 if concurrent else 0, res)
    _check(st, ctx)
    out = []
    for i, c in enumerate(cfgs):
        r = res[i]
        e = c["epochs"]
        out.append({"status": r.status, "n_train": r.n_train, "heldout_acc": list(r.heldout_acc[:e]),
                    "epoch_seconds": list(r.epoch_seconds[:e]), "eval_seconds": list(r.eval_seconds[:e]),
                    "epoch_loss": list(r.epoch_loss[:e]),
                    "heldout_acc_final": r.heldout_acc_final})
    return out


def ekya_infer(ctx, weights, frames, resolution: int, labels_out=None, stream=None):
    """Returns labels_out (int32 [n] on the GPU); asynchronous on the stream."""
    torch = _torch()
    lib = load()
    n, H, W, _ = frames.shape
    if labels_out is None:
        labels_out = torch.empty(n, dtype=torch.int32, device=frames.device)
    st = lib.ekya_infer(ctx, _dev(weights, torch.float32), _dev(frames), n, H, W, resolution,
                        _precision(frames), _dev(labels_out, torch.int32), _stream(stream))
    _check(st, ctx)
    return labels_out


# ------------------------------------------------- CU shares and hot reload
def ekya_partition_mask(n_cu: int, n_xcd: int, n_se: int, cu_begin: float, cu_share: float):
    """(CU count, mask words) of a CU range (host only); raises on invalid input."""
    import numpy as np
    words = np.zeros(max(1, (n_cu + 31) // 32), dtype=np.uint32)
    n = load().ekya_partition_mask(n_cu, n_xcd, n_se, cu_begin, cu_share, words.ctypes.data,
                                   words.size)
    if n < 0:
        raise ValueError("invalid CU range")
    return n, words


class CuStream:
    """A HIP stream restricted to a CU range; .stream is a torch ExternalStream."""

    def __init__(self, device: int, cu_begin: float, cu_share: float):
        torch = _torch()
        h = ctypes.c_void_p()
        _check(load().ekya_stream_create(device, cu_begin, cu_share, ctypes.byref(h)))
        self.handle = h
        self.stream = torch.cuda.ExternalStream(h.value, device=torch.device("cuda", device))

    @property
    def cuda_stream(self):
        return self.handle.value

    def synchronize(self):
        self.stream.synchronize()

    def cu_count(self) -> int:
        return int(load().ekya_stream_cu_count(self.handle))

    def destroy(self):
        if self.handle is not None and self.handle.value:
            self.stream.synchronize()
            _check(load().ekya_stream_destroy(self.handle))
        self.handle = None


def ekya_stream_cu_count(stream) -> int:
    return int(load().ekya_stream_cu_count(_stream(stream)))


def ekya_set_cu_partition(ctx, cu_begin: float, cu_share: float) -> None:
    _check(load().ekya_set_cu_partition(ctx, cu_begin, cu_share), ctx)


def ekya_cu_ids(n_workgroups: int, stream=None):
    """int32 view of the compute-unit id each of n one-wavefront workgroups ran on."""
    torch = _torch()
    out = torch.zeros(n_workgroups, dtype=torch.int32, device="cuda")
    _check(load().ekya_cu_ids(n_workgroups, _dev(out), _stream(stream)))
    return out


def ekya_model_create(device: int = 0, n_classes: int = 6, precision: int = EKYA_BF16,
                      hidden: int = 0):
    h = ctypes.c_void_p()
    if hidden:
        _check(load().ekya_model_create_head(ctypes.byref(h), device, n_classes, hidden, precision))
    else:
        _check(load().ekya_model_create(ctypes.byref(h), device, n_classes, precision))
    return h


def ekya_model_destroy(model) -> None:
    load().ekya_model_destroy(model)


def ekya_model_load(model, weights, stream=None) -> int:
    torch = _torch()
    v = ctypes.c_uint64()
    _check(load().ekya_model_load(model, _dev(weights, torch.float32), _stream(stream),
                                  ctypes.byref(v)))
    return int(v.value)


def ekya_model_export(model, weights_out, stream=None) -> int:
    torch = _torch()
    v = ctypes.c_uint64()
    _check(load().ekya_model_export(model, _dev(weights_out, torch.float32), _stream(stream),
                                    ctypes.byref(v)))
    return int(v.value)


def ekya_model_version(model) -> int:
    return int(load().ekya_model_version(model))


def ekya_infer_model(ctx, model, frames, resolution: int, labels_out=None, stream=None):
    """(labels_out, version of the weights used); asynchronous on the stream."""
    torch = _torch()
    n, H, W, _ = frames.shape
    if labels_out is None:
        labels_out = torch.empty(n, dtype=torch.int32, device=frames.device)
    v = ctypes.c_uint64()
    _check(load().ekya_infer_model(ctx, model, _dev(frames), n, H, W, resolution,
                                   _dev(labels_out, torch.int32), _stream(stream), ctypes.byref(v)),
           ctx)
    return labels_out, int(v.value)


def ekya_infer_models(ctx, models, frames, counts, resolution: int, labels_out=None, stream=None):
    """(labels_out, versions): frames holds counts[i] consecutive frames of
    stream i, classified with models[i]; asynchronous on the stream."""
    import numpy as np
    torch = _torch()
    n, H, W, _ = frames.shape
    if sum(counts) != n:
        raise ValueError("counts must add up to the number of frames")
    if labels_out is None:
        labels_out = torch.empty(n, dtype=torch.int32, device=frames.device)
    arr = (ctypes.c_void_p * len(models))(*[m.value for m in models])
    cnt = np.ascontiguousarray(counts, dtype=np.int32)
    ver = np.zeros(len(models), dtype=np.uint64)
    _check(load().ekya_infer_models(ctx, arr, len(models), _dev(frames), cnt.ctypes.data, H, W,
                                    resolution, _dev(labels_out, torch.int32), ver.ctypes.data,
                                    _stream(stream)), ctx)
    return labels_out, [int(v) for v in ver]


def ekya_infer_models_workspace(n_classes: int, resolution: int, n_models: int,
                                precision: int = EKYA_BF16, hidden: int = 0) -> int:
    return int(load().ekya_infer_models_workspace(n_classes, hidden, resolution, precision,
                                                  n_models))


def ekya_set_checkpoint(ctx, model, every_epochs: int = 1) -> None:
    _check(load().ekya_set_checkpoint(ctx, model, every_epochs), ctx)


# ----------------------------------------------------------------- ops
def _op(status):
    _check(status, None)


def ekya_op_conv2d(x, w, stride: int, pad: int, y=None):
    torch = _torch()
    N, H, W, C = x.shape
    K, C2, R, S = w.shape
    P, Q = (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1
    if y is None:
        y = torch.empty(N, P, Q, K, dtype=x.dtype, device=x.device)
    _op(load().ekya_op_conv2d(_precision(x), _dev(x), N, H, W, C, _dev(w, torch.float32), K, R, S,
                              stride, pad, _dev(y, x.dtype), _stream()))
    return y


def ekya_op_conv2d_dgrad(dy, w, x_shape, stride: int, pad: int):
    torch = _torch()
    N, H, W, C = x_shape
    K, _, R, S = w.shape
    dx = torch.empty(N, H, W, C, dtype=dy.dtype, device=dy.device)
    _op(load().ekya_op_conv2d_dgrad(_precision(dy), _dev(dy), _dev(w, torch.float32), N, H, W, C, K,
                                    R, S, stride, pad, _dev(dx), _stream()))
    return dx


def ekya_op_conv2d_wgrad(x, dy, w_shape, stride: int, pad: int):
    torch = _torch()
    N, H, W, C = x.shape
    K, _, R, S = w_shape
    dw = torch.empty(K, C, R, S, dtype=torch.float32, device=x.device)
    _op(load().ekya_op_conv2d_wgrad(_precision(x), _dev(x), _dev(dy, x.dtype), N, H, W, C, K, R, S,
                                    stride, pad, _dev(dw), _stream()))
    return dw


def ekya_op_batchnorm_train(z, gamma, beta, running_mean=None, running_var=None, relu=False):
    torch = _torch()
    C = z.shape[-1]
    M = z.numel() // C
    y = torch.empty_like(z)
    mean = torch.empty(C, dtype=torch.float32, device=z.device)
    invstd = torch.empty_like(mean)
    _op(load().ekya_op_batchnorm_train(_precision(z), _dev(z), M, C, _dev(gamma, torch.float32),
                                       _dev(beta, torch.float32), _dev(running_mean, torch.float32),
                                       _dev(running_var, torch.float32), int(relu), _dev(y),
                                       _dev(mean), _dev(invstd), _stream()))
    return y, mean, invstd


def ekya_op_batchnorm_train_noalloc(z, gamma, beta, running_mean=None, running_var=None,
                                    relu=False, y=None, mean=None, invstd=None, stream=None):
    """Asynchronous on the stream; outputs may be passed in (no allocation in the library)."""
    torch = _torch()
    C = z.shape[-1]
    M = z.numel() // C
    y = torch.empty_like(z) if y is None else y
    mean = torch.empty(C, dtype=torch.float32, device=z.device) if mean is None else mean
    invstd = torch.empty_like(mean) if invstd is None else invstd
    _op(load().ekya_op_batchnorm_train_noalloc(_precision(z), _dev(z), M, C, _dev(gamma, torch.float32),
                                               _dev(beta, torch.float32),
                                               _dev(running_mean, torch.float32),
                                               _dev(running_var, torch.float32), int(relu), _dev(y),
                                               _dev(mean), _dev(invstd), _stream(stream)))
    return y, mean, invstd


def ekya_op_batchnorm_backward(dy, y_relu, z, gamma, mean, invstd):
    torch = _torch()
    C = z.shape[-1]
    M = z.numel() // C
    dz = torch.empty_like(z)
    dg = torch.empty(C, dtype=torch.float32, device=z.device)
    db = torch.empty_like(dg)
    _op(load().ekya_op_batchnorm_backward(_precision(z), _dev(dy, z.dtype), _dev(y_relu, z.dtype)
                                          if y_relu is not None else None, _dev(z), M, C,
                                          _dev(gamma), _dev(mean), _dev(invstd), _dev(dz), _dev(dg),
                                          _dev(db), _stream()))
    return dz, dg, db


def ekya_op_maxpool(x):
    torch = _torch()
    N, H, W, C = x.shape
    P, Q = (H - 1) // 2 + 1, (W - 1) // 2 + 1
    y = torch.empty(N, P, Q, C, dtype=x.dtype, device=x.device)
    arg = torch.empty(N, P, Q, C, dtype=torch.uint8, device=x.device)
    _op(load().ekya_op_maxpool(_precision(x), _dev(x), N, H, W, C, _dev(y), _dev(arg), _stream()))
    return y, arg


def ekya_op_maxpool_backward(dy, arg, x_shape):
    torch = _torch()
    N, H, W, C = x_shape
    dx = torch.empty(N, H, W, C, dtype=dy.dtype, device=dy.device)
    _op(load().ekya_op_maxpool_backward(_precision(dy), _dev(dy), _dev(arg, torch.uint8), N, H, W, C,
                                        _dev(dx), _stream()))
    return dx


def ekya_op_avgpool(x):
    torch = _torch()
    N, H, W, C = x.shape
    f = torch.empty(N, C, dtype=torch.float32, device=x.device)
    _op(load().ekya_op_avgpool(_precision(x), _dev(x), N, H, W, C, _dev(f), _stream()))
    return f


def ekya_op_avgpool_backward(df, x_shape, dtype):
    torch = _torch()
    N, H, W, C = x_shape
    dx = torch.empty(N, H, W, C, dtype=dtype, device=df.device)
    _op(load().ekya_op_avgpool_backward(_precision(dx), _dev(df, torch.float32), N, H, W, C, _dev(dx),
                                        _stream()))
    return dx


def ekya_op_linear(f, W, b):
    torch = _torch()
    N, I = f.shape
    J = W.shape[0]
    z = torch.empty(N, J, dtype=torch.float32, device=f.device)
    _op(load().ekya_op_linear(_dev(f, torch.float32), _dev(W, torch.float32), _dev(b, torch.float32),
                              N, I, J, _dev(z), _stream()))
    return z


def ekya_op_linear_backward(dz, f, W):
    torch = _torch()
    N, I = f.shape
    J = W.shape[0]
    dW = torch.empty(J, I, dtype=torch.float32, device=f.device)
    db = torch.empty(J, dtype=torch.float32, device=f.device)
    df = torch.empty(N, I, dtype=torch.float32, device=f.device)
    _op(load().ekya_op_linear_backward(_dev(dz, torch.float32), _dev(f, torch.float32),
                                       _dev(W, torch.float32), N, I, J, _dev(dW), _dev(db), _dev(df),
                                       _stream()))
    return df, dW, db


def ekya_op_softmax_ce(z, labels):
    torch = _torch()
    N, J = z.shape
    dz = torch.empty_like(z)
    out = torch.empty(3, dtype=torch.float32, device=z.device)
    _op(load().ekya_op_softmax_ce(_dev(z, torch.float32), _dev(labels, torch.int32), N, J, _dev(dz),
                                  _dev(out), _stream()))
    return out, dz


def ekya_op_sgd(w, v, g, lr: float, mu: float):
    torch = _torch()
    _op(load().ekya_op_sgd(_dev(w, torch.float32), _dev(v, torch.float32), _dev(g, torch.float32),
                           w.numel(), lr, mu, _stream()))


def ekya_op_resize(frames, r: int):
    torch = _torch()
    n, H, W, _ = frames.shape
    out = torch.empty(n, r, r, 3, dtype=frames.dtype, device=frames.device)
    _op(load().ekya_op_resize(_precision(frames), _dev(frames), n, H, W, r, _dev(out), _stream()))
    return out


# ---------------------------------------------------- scheduling layer (host)
def ekya_nnls(A, b):
    """(x, ||Ax - b||) of min ||Ax - b||, x >= 0 (numpy arrays)."""
    import numpy as np
    A = np.ascontiguousarray(A, dtype=np.float64)
    b = np.ascontiguousarray(b, dtype=np.float64)
    m, n = A.shape
    x = np.zeros(n)
    r = ctypes.c_double()
    _op(load().ekya_nnls(A.ctypes.data, m, n, b.ctypes.data, x.ctypes.data, ctypes.byref(r)))
    return x, r.value


def ekya_fit_accuracy_curve(x, acc):
    import numpy as np
    x = np.ascontiguousarray(x, dtype=np.float64)
    acc = np.ascontiguousarray(acc, dtype=np.float64)
    c = Curve()
    _op(load().ekya_fit_accuracy_curve(x.ctypes.data, acc.ctypes.data, x.size, ctypes.byref(c)))
    return c


def ekya_curve_accuracy(c, x: float) -> float:
    return float(load().ekya_curve_accuracy(ctypes.byref(c), x))


def ekya_extrapolate(cfg: dict, result: dict, n_frames: int, epochs_target: int):
    """(curve, accuracy, gpu_seconds) for a candidate dict and its ekya_profile result dict."""
    pc = ProfileCfg(cfg["k"], cfg["subsample_frac"], cfg["epochs"], cfg.get("lr", 0.01),
                    cfg.get("momentum", 0.9), cfg.get("batch", 64), cfg.get("seed", 0))
    pr = ProfileResult()
    pr.status = result.get("status", 0)
    pr.n_train = result["n_train"]
    for e in range(cfg["epochs"]):
        pr.heldout_acc[e] = result["heldout_acc"][e]
        pr.epoch_seconds[e] = result["epoch_seconds"][e]
    c = Curve()
    acc, sec = ctypes.c_double(), ctypes.c_double()
    _op(load().ekya_extrapolate(ctypes.byref(pc), ctypes.byref(pr), n_frames, epochs_target,
                                ctypes.byref(c), ctypes.byref(acc), ctypes.byref(sec)))
    return c, acc.value, sec.value


def ekya_thief_schedule(videos, n_gpus: float, delta: float, window_s: float, a_min: float) -> dict:
    """videos: list of dicts {acc_now, infer: [(cost, factor)], train: [(acc_after, gpu_seconds)]}."""
    keep = []
    arr = (VideoIn * len(videos))()
    for i, v in enumerate(videos):
        inf = (InferCfg * len(v["infer"]))(*[InferCfg(c, f) for c, f in v["infer"]])
        tr = (TrainCfg * max(1, len(v["train"])))(*[TrainCfg(a, g) for a, g in v["train"]])
        keep += [inf, tr]
        arr[i] = VideoIn(v["acc_now"], inf, len(v["infer"]), tr, len(v["train"]))
    nv = len(videos)
    alloc = (ctypes.c_double * (2 * nv))()
    ic, tc = (ctypes.c_int * nv)(), (ctypes.c_int * nv)()
    va = (ctypes.c_double * nv)()
    out = ScheduleOut(alloc, ic, tc, va, 0.0)
    _op(load().ekya_thief_schedule(arr, nv, n_gpus, delta, window_s, a_min, ctypes.byref(out)))
    return {"alloc": list(alloc), "infer_choice": list(ic), "train_choice": list(tc),
            "video_accuracy": list(va), "accuracy": out.accuracy}
