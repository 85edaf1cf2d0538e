"""CU shares on the GPU (section 4.1: jobs of a window get GPU shares in steps
of Delta; section 5: a partitioning layer enforces them).  A stream made by
ekya_stream_create runs its kernels only on the CUs of its range: checked
with the hardware ids its workgroups report, with inference throughput
against the share, and with a joint window (inference on one range, a
layer3+ retraining job on the complementary range) whose results are bitwise
those of the same calls run alone on the whole GPU."""
import threading
import time

import pytest

from synth import WindowSpec, kaiming_resnet18_weights, make_window
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu


def _ids(binding, stream, n=8192):
    out = binding.ekya_cu_ids(n, stream=stream)
    stream.synchronize()
    return set(out.cpu().tolist())


def _n_xcd(ids):
    return len({i >> 10 for i in ids})


def _per_engine(ids):
    """(XCD, shader engine) -> distinct CUs that ran a workgroup."""
    out = {}
    for i in ids:
        key = (i >> 10, (i >> 4) & 7)
        out[key] = out.get(key, 0) + 1
    return out


@pytest.fixture(scope="module")
def whole():
    import torch
    from paper_2012_10557_amd import binding
    s = torch.cuda.Stream()
    ids = _ids(binding, s)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    print(f"device: {n_cu} CUs, {len(ids)} distinct CU ids on an unrestricted stream, "
          f"{_n_xcd(ids)} XCDs")
    return {"ids": ids, "n_cu": n_cu, "n_xcd": _n_xcd(ids)}


@pytest.mark.parametrize("begin,share", [(0.0, 1.0), (0.0, 0.5), (0.5, 0.5), (0.0, 0.1),
                                         (0.3, 0.7), (0.9, 0.1)])
def test_stream_runs_only_on_its_cus(whole, begin, share):
    from paper_2012_10557_amd import binding
    n_cu, n_xcd = whole["n_cu"], whole["n_xcd"]
    expect, _ = binding.ekya_partition_mask(n_cu, n_xcd, 4, begin, share)
    cs = binding.CuStream(0, begin, share)
    try:
        assert cs.cu_count() == expect
        ids = _ids(binding, cs)
        pe = _per_engine(ids)
        print(f"[{begin}, {begin + share}): mask {expect} CUs, workgroups ran on {len(ids)} CUs "
              f"of {_n_xcd(ids)} XCDs; CUs per (XCD, engine): {sorted(pe.items())}")
        assert ids <= whole["ids"]
        assert len(ids) <= expect
        assert _n_xcd(ids) == n_xcd
        assert len(ids) >= 0.9 * expect
        # the engines of every XCD differ by at most one CU (mask bits dealt
        # to XCDs, then engines, as the driver maps them)
        for x in {k[0] for k in pe}:
            c = [pe.get((x, e), 0) for e in range(4)]
            assert max(c) - min(c) <= 1, (x, c)
    finally:
        cs.destroy()


def test_complementary_ranges_use_disjoint_cus(whole):
    from paper_2012_10557_amd import binding
    a, b = binding.CuStream(0, 0.0, 0.3), binding.CuStream(0, 0.3, 0.7)
    try:
        ia, ib = _ids(binding, a), _ids(binding, b)
        print(f"30%: {len(ia)} CUs, 70%: {len(ib)} CUs, shared {len(ia & ib)}")
        assert not (ia & ib)
        assert len(ia) + len(ib) <= whole["n_cu"]
    finally:
        a.destroy()
        b.destroy()


@pytest.fixture(scope="module")
def window():
    import torch
    win = make_window(WindowSpec(3600, 400, 224, 224, drift="drift", seed=2))
    fr = to_dev(win["frames"], "bf16")
    return {"fr": fr, "lab": torch.tensor(win["labels"], device="cuda"),
            "hf": to_dev(win["heldout_frames"], "bf16"),
            "hl": torch.tensor(win["heldout_labels"], device="cuda"),
            "w0": torch.tensor(kaiming_resnet18_weights(seed=0), device="cuda"),
            "inf": fr[:2048].contiguous()}


def _rate(binding, ctx, w, frames, res, stream, reps=3):
    lab = binding.ekya_infer(ctx, w, frames, res, stream=stream)
    stream.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        binding.ekya_infer(ctx, w, frames, res, labels_out=lab, stream=stream)
    stream.synchronize()
    return reps * frames.shape[0] / (time.perf_counter() - t0), lab


def test_inference_throughput_follows_the_cu_share(window):
    """224 px bf16 inference of 2048 frames on 25%, 50%, 75% and 100% of the CUs:
    the rate grows with the share and labels are bitwise the same on every
    share (no kernel's plan depends on the CUs it gets)."""
    import torch
    from paper_2012_10557_amd import binding
    d = window
    ctx = binding.ekya_create(0, 6)
    rates, labs = {}, {}
    try:
        for share in (0.25, 0.5, 0.75, 1.0):
            cs = binding.CuStream(0, 0.0, share)
            try:
                rates[share], labs[share] = _rate(binding, ctx, d["w0"], d["inf"], 224, cs)
            finally:
                cs.destroy()
        print("inference img/s by CU share: " +
              ", ".join(f"{s:.2f}: {r:.0f} ({r / rates[1.0]:.2f} of the whole GPU)"
                        for s, r in rates.items()))
        for sh in rates:
            assert torch.equal(labs[sh], labs[1.0])
        assert rates[0.25] < rates[0.5] < rates[0.75] < 1.1 * rates[1.0]
        assert rates[0.25] < 0.6 * rates[1.0]
    finally:
        binding.ekya_destroy(ctx)


@pytest.mark.parametrize("split", [0.3, 0.5])
def test_joint_window_on_partitions_is_bitwise_unchanged(window, split):
    """Inference (3600-frame window at 224 px, every other frame) on CUs
    [0, split), layer3+ retraining (10% of the window, 5 epochs, batch 128)
    with its context's own streams on [split, 1): labels, weights, step losses
    and held-out accuracies equal those of the calls run alone."""
    import torch
    from paper_2012_10557_amd import binding
    d = window
    inf = d["fr"][::2].contiguous()
    ictx, rctx = binding.ekya_create(0, 6), binding.ekya_create(0, 6)
    s_inf, s_tr = binding.CuStream(0, 0.0, split), binding.CuStream(0, split, 1.0 - split)
    try:
        def retrain(box, stream):
            box["out"] = binding.ekya_retrain(rctx, box["w"], 3, d["fr"], d["lab"], d["hf"], d["hl"],
                                              0.1, 5, 0.01, 0.9, 128, 0, stream=stream,
                                              step_losses=True)
        # alone on the whole GPU
        ws = torch.cuda.Stream()
        lab_ref = binding.ekya_infer(ictx, d["w0"], inf, 224, stream=ws)
        ref = {"w": d["w0"].clone()}
        torch.cuda.synchronize()
        retrain(ref, ws)
        torch.cuda.synchronize()
        binding.ekya_set_cu_partition(rctx, split, 1.0 - split)
        box = {"w": d["w0"].clone()}
        torch.cuda.synchronize()
        th = threading.Thread(target=retrain, args=(box, s_tr))
        t0 = time.perf_counter()
        th.start()
        lab = binding.ekya_infer(ictx, d["w0"], inf, 224, stream=s_inf)
        s_inf.synchronize()
        t_inf = time.perf_counter() - t0
        th.join()
        t_all = time.perf_counter() - t0
        print(f"split {split}: inference {inf.shape[0] / t_inf:.0f} img/s on {s_inf.cu_count()} CUs; "
              f"retraining done after {t_all:.3f} s on {s_tr.cu_count()} CUs")
        assert torch.equal(lab, lab_ref)
        assert torch.equal(box["w"], ref["w"])
        assert box["out"]["step_loss"] == ref["out"]["step_loss"]
        assert box["out"]["heldout_acc"] == ref["out"]["heldout_acc"]
    finally:
        s_inf.destroy()
        s_tr.destroy()
        binding.ekya_destroy(ictx)
        binding.ekya_destroy(rctx)


def test_invalid_partitions_are_rejected():
    from paper_2012_10557_amd import binding
    ctx = binding.ekya_create(0, 6)
    try:
        for args in [(-0.1, 0.5), (0.5, 0.6), (0.0, 0.0), (1.0, 0.1)]:
            with pytest.raises(binding.EkyaError):
                binding.ekya_set_cu_partition(ctx, *args)
            with pytest.raises(binding.EkyaError):
                binding.CuStream(0, *args)
        binding.ekya_set_cu_partition(ctx, 0.0, 1.0)
    finally:
        binding.ekya_destroy(ctx)
