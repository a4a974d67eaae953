"""Host logic of bench.py (no GPU): the one-GPU refusal, the forward-launch
classifier used on kernel traces, compulsory bytes, the per-step FLOP count
and the guard that reports stored HBM traffic only for the sources it was
measured on."""
import argparse
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench as B  # noqa: E402
from paper_2102_06725_amd import inputs as I  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_forward_launch_classifier():
    # launch order of two sweep layers and a depthwise layer, as bench.py queues them
    names = [
        "at::native::FillFunctor",                                    # flag clear
        "nnconv::pad_channels4_vec_kernel",                           # stem padding
        "nnconv::stem_fwd4_kernel<nnconv::Half>",                     # fwd
        "nnconv::stem_wgrad4_kernel<nnconv::Half>",
        "nnconv::wgrad_reduce_vec_kernel<2, 16>",
        "nnconv::igemm_c64_kernel<nnconv::Half, 128, 64, 2, 2, 8, 1, false, false>",  # fwd
        "nnconv::transpose16_vec_kernel",
        "nnconv::igemm_c64_kernel<nnconv::Half, 128, 64, 2, 2, 8, 1, false, false>",  # dgrad
        "nnconv::wgrad_splitk_kernel<nnconv::Half, 64, 128, 2, 2, 64, 1, false>",
        "nnconv::wgrad_reduce_vec_kernel<2, 16>",
        "nnconv::dwt_fwd_kernel<nnconv::Half, 3, 1, 4, false, false>",               # fwd
        "nnconv::dwt_fwd_kernel<nnconv::Half, 3, 1, 4, false, true>",                # dgrad
        "nnconv::dwt_wgrad_kernel<nnconv::Half, 3, 1, 4>",
        "nnconv::wgrad_reduce_vec_kernel<2, 16>",
        # a register-weight halo layer: packing + GEMM in both passes
        "nnconv::pack_hring_b_kernel",                                               # fwd
        "nnconv::igemm_hring_kernel<nnconv::Half, 224, 256, 1, 4, 256, 9, 3>",       # fwd
        "nnconv::transpose16_vec_kernel<true>",
        "nnconv::pack_hring_b_kernel",
        "nnconv::igemm_hring_kernel<nnconv::Half, 224, 256, 1, 4, 256, 9, 3>",       # dgrad
        "nnconv::dgrad_border_kernel<nnconv::Half>",
        "nnconv::wgrad_splitk_kernel<nnconv::Half, 256, 256, 4, 4, 32, 2, false>",
        "nnconv::wgrad_reduce_vec_kernel<2, 16>",
    ]
    assert B.forward_calls(names) == [[2], [5], [10], [14, 15]]


def test_compulsory_bytes_by_hand():
    L = I.Layer("c1x1", 4, 64, 8, 8, 256, 1, 1)
    x, w, y = 4 * 8 * 8 * 64 * 2, 256 * 64 * 2, 4 * 8 * 8 * 256 * 2
    assert B.compulsory_bytes(L, "fwd") == x + w + y
    assert B.compulsory_bytes(L, "dgrad") == y + w + x
    assert B.compulsory_bytes(L, "wgrad") == x + y + 2 * w       # fp32 dw
    # a strided 1x1 reads only the sampled pixels of x
    S = I.Layer("proj", 2, 32, 10, 10, 64, 1, 1, 2, 0)
    assert S.p == 5 and S.q == 5
    xs = 2 * 5 * 5 * 32 * 2
    assert B.compulsory_bytes(S, "fwd") == xs + 64 * 32 * 2 + 2 * 5 * 5 * 64 * 2
    # dgrad writes the whole dx (zeros where no tap reaches)
    assert B.compulsory_bytes(S, "dgrad") == 2 * 5 * 5 * 64 * 2 + 64 * 32 * 2 + 2 * 10 * 10 * 32 * 2


def test_sweep_step_flops():
    args = argparse.Namespace(workload="sweep", dtype="f16", batch=0, layers="")
    wl, layers = B.layers_for(args)
    assert len(layers) == 53
    step = sum(L.flops() * (3 if L.dgrad else 2) for L in layers)
    # the stem counts its 3 logical channels and has no backward-data pass
    stem = [L for L in layers if not L.dgrad]
    assert len(stem) == 1 and stem[0].c_alg == 3
    assert abs(step - 6.217418145792e12) < 1e3


def test_stored_traffic_only_for_its_sources(tmp_path, monkeypatch):
    good = tmp_path / "traffic.txt"
    good.write_text("# comment: ignored\nmfma_fetch_bytes_per_launch: 100\n"
                    "mfma_write_bytes_per_launch: 23\nhbm_fetch_bytes_per_launch: 7\n"
                    "hbm_write_bytes_per_launch: 5\nsource_sha256: %s\n" % B.fwd_source_hash())
    monkeypatch.setattr(B, "TRAFFIC_FILE", str(good))
    assert B.stored_traffic("mfma") == 123.0
    assert B.stored_traffic("hbm") == 12.0
    stale = tmp_path / "stale.txt"
    stale.write_text("mfma_fetch_bytes_per_launch: 100\nmfma_write_bytes_per_launch: 23\n"
                     "source_sha256: %s\n" % ("0" * 64))
    monkeypatch.setattr(B, "TRAFFIC_FILE", str(stale))
    assert B.stored_traffic() is None
    monkeypatch.setattr(B, "TRAFFIC_FILE", str(tmp_path / "missing.txt"))
    assert B.stored_traffic() is None


@pytest.mark.parametrize("pass_", ["fwd", "dgrad", "wgrad"])
def test_roofline_bound_is_the_larger_time(pass_):
    for L, _ in I.resnet50_layers(256):
        us, bound = B.roofline_us(L, pass_)
        t_mfma = L.flops(executed=True) / (B.PEAK_F16_TFLOPS * 1e12) * 1e6
        t_hbm = B.compulsory_bytes(L, pass_) / (B.PEAK_HBM_GBS * 1e9) * 1e6
        assert us == pytest.approx(max(t_mfma, t_hbm))
        assert bound == ("mfma" if t_mfma >= t_hbm else "hbm")


def test_forward_launch_sets_partition_the_sweep():
    """The MFMA-bound and HBM-bound forward sets split the 53 layers by the
    compulsory-byte roofline: every layer in exactly one, the 3x3 layers of
    stages 3-5 MFMA-bound, the 56x56 1x1 layers and the stem HBM-bound."""
    args = argparse.Namespace(workload="sweep", dtype="f16", batch=0, layers="")
    _, layers = B.layers_for(args)
    mf, hb = B.fwd_sets(layers)
    assert sorted(mf + hb) == list(range(53)) and not set(mf) & set(hb)
    names_mf = {layers[i].name for i in mf}
    names_hb = {layers[i].name for i in hb}
    assert {"s3b1b", "s4b1b", "s5b1b", "s5b0b"} <= names_mf
    assert {"stem", "s2b0a", "s2b0c", "s2b1a", "s2b0b"} <= names_hb


def test_config1_workload_is_the_tiny_nchw_convolution():
    args = argparse.Namespace(workload="cfg1", dtype="f16", batch=0, layers="")
    wl, layers = B.layers_for(args)
    assert wl.layout == "nchw" and len(layers) == 1
    L = layers[0]
    assert (L.n, L.c, L.h, L.w, L.k, L.r, L.s, L.stride, L.pad) == (2, 16, 16, 16, 16, 3, 3, 1, 1)
    assert L.flops() == 2 * 2 * 16 * 16 * 16 * 16 * 9
