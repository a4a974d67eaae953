"""GPU parity: libnnconv (through the C ABI) against the fp64 oracle on the
same seeded, quantised inputs.  Tolerance max|err| / max|ref| <= 2e-3 for
fp16 operands and 5e-3 for bf16; integer/shape behaviour and structural
zeros exact; guard bands around every output untouched."""
import numpy as np
import pytest

import oracle.oracle as orc
from gpu_util import (TOL, Case, Guarded, full_parity, nchw_f64, oracle_conv, run_gpu,
                      stream, to_dev, to_nchw, torch)
from paper_2102_06725_amd import inputs as I
from paper_2102_06725_amd import nnconv as nc

pytestmark = pytest.mark.gpu

L = I.Layer


@pytest.fixture(scope="module", autouse=True)
def _setup(nnlib, oracle_lib):
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    orc.set_threads(min(16, max(1, orc.get_threads())))
    yield


def config1_case(dtype=I.F16):
    wl = I.workload(1, dtype)
    Lr = wl.layers[0]
    s = 1.0 / 12.0
    return Case(Lr, layout="nchw", dtype=dtype, loss_scale=1.0, x_kind="normal", dy_std=s,
                cfg=1, layer_id=0)


def test_config1_exact_recipe():
    """Config 1: 3x3 16->16 on 16x16, batch 2, NCHW fp16, x, w, dy ~ N(0,1)/12."""
    case = config1_case()
    wl = I.workload(1)
    t = I.layer_tensors(wl, 0, 1)
    # the Case draws w with the He scale; config 1 draws all three at 1/12
    got = run_gpu(case, t)
    x, w, dy = nchw_f64(case, t)
    cv = oracle_conv(case)
    for name, ref in (("y", cv.fwd(x, w)), ("dx", cv.dgrad(dy, w)), ("dw", cv.wgrad(x, dy))):
        e = orc.rel_err(to_nchw(case, name, got[name]), ref)
        print("config1", name, "rel err %.3e" % e)
        assert e <= TOL[I.F16]


SMALL = [
    ("3x3 ragged tiles", Case(L("a", 3, 64, 11, 13, 72, 3, 3, 1, 1))),
    ("3x3 stride 2", Case(L("b", 3, 32, 15, 14, 40, 3, 3, 2, 1))),
    ("1x1 stride 2", Case(L("c", 2, 64, 14, 13, 136, 1, 1, 2, 0))),
    ("1x1 C256 K64", Case(L("d", 3, 256, 7, 7, 64, 1, 1))),
    ("1x1 K512 many n-tiles", Case(L("d2", 2, 128, 5, 6, 512, 1, 1))),
    ("stem-like 7x7 s2 C3 padded to 8", Case(L("e", 2, 8, 23, 21, 64, 7, 7, 2, 3, c_logical=3),
                                            x_kind="normal")),
    # 4-channel stem pixels: partial tiles, all four channels live, bf16, and
    # an odd width (the direct kernels)
    ("stem-like C3 padded to 4", Case(L("e4", 2, 4, 24, 22, 64, 7, 7, 2, 3, c_logical=3),
                                      x_kind="normal")),
    ("stem-like C4 2x2 tiles", Case(L("e5", 3, 4, 40, 36, 64, 7, 7, 2, 3), x_kind="normal")),
    ("stem-like C3(4) bf16", Case(L("e6", 2, 4, 34, 50, 64, 7, 7, 2, 3, c_logical=3),
                                  x_kind="normal", dtype=I.BF16)),
    ("stem-like C4 odd width", Case(L("e7", 2, 4, 15, 15, 64, 7, 7, 2, 3), x_kind="normal")),
    ("stem-like C4 small odd height", Case(L("e8", 1, 4, 9, 8, 64, 7, 7, 2, 3), x_kind="normal")),
    ("stem-like C4 padding 2 (direct)", Case(L("e9", 2, 4, 12, 14, 64, 7, 7, 2, 2),
                                            x_kind="normal")),
    ("dilation 2", Case(L("f", 2, 16, 12, 12, 24, 3, 3, 1, 2, dil=2))),
    ("groups 2", Case(L("g", 2, 32, 9, 9, 48, 3, 3, 1, 1, groups=2))),
    ("5x5 stride 3 pad 2", Case(L("h", 1, 24, 17, 19, 16, 5, 5, 3, 2))),
    ("1x3 kernel", Case(L("i", 2, 16, 9, 10, 16, 1, 3, 1, 1))),
    ("3x3 NCHW ragged", Case(L("j", 3, 64, 11, 13, 72, 3, 3, 1, 1), layout="nchw")),
    ("1x1 s2 NCHW", Case(L("k", 2, 32, 9, 10, 16, 1, 1, 2, 0), layout="nchw")),
    ("3x3 bf16", Case(L("l", 3, 64, 11, 13, 72, 3, 3, 1, 1), dtype=I.BF16)),
    ("3x3 s2 bf16 NCHW", Case(L("m", 2, 32, 15, 14, 40, 3, 3, 2, 1), dtype=I.BF16, layout="nchw")),
    ("wgrad many splits", Case(L("n", 4, 64, 28, 28, 64, 3, 3, 1, 1))),
    # 3x3 64 -> 64 backward-weight in blocks of whole image rows: blocks of
    # 2 rows of 56, 8 of 14, 16 of 7 and 8 of 10 pixels; heights that leave
    # a partial last block; several blocks per workgroup
    ("row blocks W56", Case(L("rb1", 2, 64, 5, 56, 64, 3, 3, 1, 1))),
    ("row blocks W14 bf16", Case(L("rb2", 3, 64, 13, 14, 64, 3, 3, 1, 1), dtype=I.BF16)),
    ("row blocks W7", Case(L("rb3", 5, 64, 7, 7, 64, 3, 3, 1, 1))),
    ("row blocks W10 NCHW", Case(L("rb4", 2, 64, 9, 10, 64, 3, 3, 1, 1), layout="nchw")),
    ("row blocks many per split", Case(L("rb5", 300, 64, 4, 8, 64, 3, 3, 1, 1))),
    ("row blocks W12 one row", Case(L("rb6", 3, 64, 1, 12, 64, 3, 3, 1, 1))),
    ("row blocks W3", Case(L("rb7", 4, 64, 9, 3, 64, 3, 3, 1, 1))),
    ("row blocks W1 (split-K instead)", Case(L("rb8", 4, 64, 7, 1, 64, 3, 3, 1, 1))),
    ("row blocks W28 bf16 loss scale 1024", Case(L("rb9", 2, 64, 11, 28, 64, 3, 3, 1, 1),
                                                  dtype=I.BF16, loss_scale=1024.0, dy_std=1e-3)),
    ("loss scale 1024", Case(L("o", 2, 64, 14, 14, 128, 3, 3, 1, 1), loss_scale=1024.0,
                             dy_std=1e-3)),
    ("direct: C3 unpadded", Case(L("p", 2, 3, 10, 10, 16, 3, 3, 1, 1))),
    ("direct: groups Cg=4", Case(L("q", 2, 16, 8, 8, 16, 3, 3, 1, 1, groups=4))),
    ("direct: NCHW C12 bf16", Case(L("r", 2, 12, 7, 9, 20, 3, 3, 2, 1), layout="nchw",
                                   dtype=I.BF16)),
    ("3x3 s2 C64 K64 (large-tile phases)", Case(L("s2", 3, 64, 15, 13, 64, 3, 3, 2, 1))),
    ("1x1 s2 C64 K64", Case(L("s3", 2, 64, 14, 15, 64, 1, 1, 2, 0))),
    ("3x3 C128 K256 ragged M", Case(L("s4", 3, 128, 9, 11, 256, 3, 3, 1, 1))),
    ("1x1 C256 K320", Case(L("s5", 2, 256, 9, 7, 320, 1, 1))),
    ("3x3 pad 0 C64", Case(L("s6", 2, 64, 9, 8, 128, 3, 3, 1, 0))),
    ("1x1 C192 K96", Case(L("s7", 2, 192, 7, 9, 96, 1, 1))),
    ("3x3 stride 3 C64 K64 (nine phases)", Case(L("s9", 2, 64, 13, 14, 64, 3, 3, 3, 1))),
    ("1x1 stride 2 C128 K256 (zero phases)", Case(L("s10", 3, 128, 9, 10, 256, 1, 1, 2, 0))),
    ("3x3 C512 K128 (wide filter)", Case(L("s11", 2, 512, 5, 6, 128, 3, 3, 1, 1))),
    ("3x3 C256 K512 bf16", Case(L("s8", 2, 256, 6, 5, 512, 3, 3, 1, 1), dtype=I.BF16)),
    ("P = Q = 1", Case(L("s", 2, 16, 3, 3, 16, 3, 3, 1, 0))),
    ("H = W = 1, 1x1", Case(L("t", 5, 32, 1, 1, 24, 1, 1))),
    # depthwise (groups = C = K) on the vector-ALU kernels
    ("depthwise 3x3", Case(L("dw1", 3, 64, 13, 11, 64, 3, 3, 1, 1, groups=64))),
    ("depthwise 3x3 stride 2", Case(L("dw2", 2, 96, 15, 14, 96, 3, 3, 2, 1, groups=96))),
    ("depthwise 5x5 stride 2 bf16", Case(L("dw3", 2, 40, 17, 16, 40, 5, 5, 2, 2, groups=40),
                                         dtype=I.BF16)),
    ("depthwise 7x7 dilation 2", Case(L("dw4", 2, 16, 20, 19, 16, 7, 7, 1, 6, dil=2,
                                        groups=16))),
    ("depthwise 3x3 NCHW", Case(L("dw5", 2, 24, 9, 10, 24, 3, 3, 1, 1, groups=24),
                                layout="nchw")),
    ("depthwise 3x3 pad 0 C320", Case(L("dw6", 2, 320, 9, 8, 320, 3, 3, 1, 0, groups=320))),
    ("depthwise 5x5 stride 3 ragged", Case(L("dw7", 3, 8, 11, 13, 8, 5, 5, 3, 1, groups=8))),
    ("depthwise 3x3 H = W = 1", Case(L("dw8", 4, 32, 1, 1, 32, 3, 3, 1, 1, groups=32))),
    ("direct: depthwise C12", Case(L("dw9", 2, 12, 9, 9, 12, 3, 3, 1, 1, groups=12))),
    # LDS-tiled depthwise: channel blocks of 2 / 4 / 8 vectors, ragged tiles,
    # padding above R-1 (negative padding of the rotated backward-data),
    # 7x7 weights in LDS, several tiles per backward-weight split
    ("depthwise tiled C16 ragged", Case(L("dt1", 2, 16, 37, 35, 16, 3, 3, 1, 1, groups=16))),
    ("depthwise tiled C48 stride 2 odd width", Case(L("dt2", 3, 48, 23, 29, 48, 3, 3, 2, 1,
                                                      groups=48))),
    ("depthwise tiled 5x5 C144", Case(L("dt3", 2, 144, 19, 21, 144, 5, 5, 1, 2, groups=144))),
    ("depthwise tiled 7x7 C72 stride 2", Case(L("dt4", 2, 72, 25, 22, 72, 7, 7, 2, 3,
                                                groups=72))),
    ("depthwise tiled 7x7 C64", Case(L("dt5", 2, 64, 17, 18, 64, 7, 7, 1, 3, groups=64))),
    ("depthwise tiled 3x3 pad 2", Case(L("dt6", 2, 32, 10, 12, 32, 3, 3, 1, 2, groups=32))),
    ("depthwise tiled 3x3 pad 3 C24", Case(L("dt7", 1, 24, 6, 7, 24, 3, 3, 1, 3, groups=24))),
    ("depthwise tiled 5x5 stride 2 pad 0", Case(L("dt8", 6, 40, 33, 30, 40, 5, 5, 2, 0,
                                                  groups=40))),
    ("depthwise tiled 5x5 bf16", Case(L("dt9", 2, 96, 15, 17, 96, 5, 5, 1, 2, groups=96),
                                      dtype=I.BF16)),
    ("depthwise tiled many tiles per split", Case(L("dt10", 40, 8, 64, 64, 8, 3, 3, 1, 1,
                                                    groups=8))),
    ("depthwise tiled 3x3 stride 2 pad 0", Case(L("dt12", 2, 32, 17, 18, 32, 3, 3, 2, 0,
                                                  groups=32))),
    ("depthwise tiled 5x5 stride 2 pad 1 C16", Case(L("dt13", 3, 16, 21, 19, 16, 5, 5, 2, 1,
                                                      groups=16))),
    ("depthwise tiled 3x3 stride 2 pad 2 even size", Case(L("dt14", 2, 64, 16, 14, 64, 3, 3, 2,
                                                            2, groups=64))),
    ("depthwise tiled 5x5 on 7x7 (narrow tile)", Case(L("dt15", 3, 128, 7, 7, 128, 5, 5, 1, 2,
                                                        groups=128))),
    ("depthwise tiled stride 2 on 7x7 (narrow)", Case(L("dt16", 2, 64, 7, 7, 64, 3, 3, 2, 1,
                                                        groups=64))),
    ("depthwise tiled 3x3 stride 2 NCHW bf16", Case(L("dt11", 2, 56, 13, 16, 56, 3, 3, 2, 1,
                                                      groups=56), layout="nchw", dtype=I.BF16)),
    # small groups (Cg = Kg < 64) as 64-channel super-groups
    ("groups 32 x 4 channels", Case(L("sg4", 2, 128, 9, 10, 128, 3, 3, 1, 1, groups=32))),
    ("groups 32 x 8 channels stride 2", Case(L("sg8", 2, 256, 9, 8, 256, 3, 3, 2, 1,
                                                 groups=32))),
    ("groups 8 x 16 channels NCHW", Case(L("sg16", 2, 128, 7, 9, 128, 3, 3, 1, 1, groups=8),
                                         layout="nchw")),
    ("groups 4 x 32 channels bf16", Case(L("sg32", 2, 128, 6, 7, 128, 3, 3, 1, 1, groups=4),
                                         dtype=I.BF16)),
    ("groups 32 x 2 channels 1x1", Case(L("sg2", 3, 64, 5, 6, 64, 1, 1, groups=32))),
    ("groups 32 x 4 channels stride 3", Case(L("sg4s3", 2, 128, 10, 11, 128, 3, 3, 3, 1,
                                                groups=32))),
    ("depthwise 3x5 as super-groups", Case(L("sg1", 2, 64, 7, 8, 64, 3, 5, 1, 1, groups=64))),
    # stride-1 3x3 super-groups on a 56-wide image: two 256-row halo tiles
    # per group, row blocks of 2 rows for backward-weight (the last one short)
    ("groups 32 x 4 channels 56 wide", Case(L("sg4w", 1, 128, 5, 56, 128, 3, 3, 1, 1,
                                                groups=32))),
    ("groups 16 x 4 channels dilation 2", Case(L("sg4d", 2, 64, 12, 13, 64, 3, 3, 1, 2, dil=2,
                                                   groups=16))),
    # groups of exactly 64 channels: the halo tiles' group mode without the
    # block-diagonal skip (row blocks of 8 rows, the last one short)
    ("groups 2 x 64 channels", Case(L("g64", 2, 128, 11, 16, 128, 3, 3, 1, 1, groups=2))),
    ("groups 3 x 64 channels NCHW bf16", Case(L("g64b", 2, 192, 9, 12, 192, 3, 3, 1, 1,
                                                  groups=3), layout="nchw", dtype=I.BF16)),
    ("direct: depthwise 3x5", Case(L("dw10", 2, 16, 8, 9, 16, 3, 5, 1, 1, groups=16))),
]


@pytest.mark.parametrize("name,case", SMALL, ids=[s[0] for s in SMALL])
def test_small_parity(name, case):
    errs = full_parity(case)
    print(name, {k: "%.3e" % v for k, v in errs.items()})


def test_alpha_scales_forward_and_dgrad():
    case = Case(L("u", 2, 32, 9, 9, 32, 3, 3, 1, 1), alpha=0.5)
    full_parity(case, passes=("fwd", "dgrad"))


def test_deterministic():
    case = Case(L("v", 4, 64, 28, 28, 64, 3, 3, 1, 1), loss_scale=1024.0, dy_std=1e-3)
    t = case.tensors()
    a = run_gpu(case, t)
    b = run_gpu(case, t)
    for k in ("y_bits", "dx_bits", "dw_bits"):
        assert np.array_equal(a[k], b[k]), k


def test_depthwise_deterministic_and_loss_scale_invariant():
    """The depthwise kernels sum in a fixed order: two runs agree bitwise,
    and wgrad(x, S*dy)/S == wgrad(x, dy) bitwise for S = 1024."""
    base = Case(L("dwi", 4, 64, 20, 18, 64, 3, 3, 1, 1, groups=64), loss_scale=1.0,
                dy_std=1.0)
    t1 = base.tensors()
    a = run_gpu(base, t1)
    b = run_gpu(base, t1)
    for k in ("y_bits", "dx_bits", "dw_bits"):
        assert np.array_equal(a[k], b[k]), k
    dy1 = I.from_bits(t1["dy"], I.F16)
    tS = dict(t1)
    tS["dy"] = I.to_bits(dy1 * 1024.0, I.F16)
    assert np.array_equal(I.from_bits(tS["dy"], I.F16), dy1 * 1024.0)
    r1 = run_gpu(base, t1, passes=("wgrad",), inv_scale=1.0)
    rS = run_gpu(base, tS, passes=("wgrad",), inv_scale=1.0 / 1024.0)
    assert np.array_equal(r1["dw_bits"], rS["dw_bits"])


def test_grouped_deterministic_and_loss_scale_invariant():
    """Super-grouped small groups: two runs agree bitwise, and the weight
    gradient keeps the power-of-two loss-scale invariant bitwise."""
    base = Case(L("sgi", 2, 128, 14, 14, 128, 3, 3, 1, 1, groups=32), loss_scale=1.0,
                dy_std=1.0)
    t1 = base.tensors()
    a = run_gpu(base, t1)
    b = run_gpu(base, t1)
    for k in ("y_bits", "dx_bits", "dw_bits"):
        assert np.array_equal(a[k], b[k]), k
    dy1 = I.from_bits(t1["dy"], I.F16)
    tS = dict(t1)
    tS["dy"] = I.to_bits(dy1 * 1024.0, I.F16)
    r1 = run_gpu(base, t1, passes=("wgrad",), inv_scale=1.0)
    rS = run_gpu(base, tS, passes=("wgrad",), inv_scale=1.0 / 1024.0)
    assert np.array_equal(r1["dw_bits"], rS["dw_bits"])


def test_loss_scale_power_of_two_invariant():
    """wgrad(x, S*dy)/S == wgrad(x, dy) bitwise (fp32 out), and
    dgrad(S*dy) == S*dgrad(dy) bitwise where both are normal fp16 numbers."""
    base = Case(L("w", 2, 64, 14, 14, 64, 3, 3, 1, 1), loss_scale=1.0, dy_std=1.0)
    t1 = base.tensors()
    dy1 = I.from_bits(t1["dy"], I.F16)
    tS = dict(t1)
    tS["dy"] = I.to_bits(dy1 * 1024.0, I.F16)
    assert np.array_equal(I.from_bits(tS["dy"], I.F16), dy1 * 1024.0)
    r1 = run_gpu(base, t1, passes=("dgrad", "wgrad"), inv_scale=1.0)
    rS = run_gpu(base, tS, passes=("dgrad", "wgrad"), inv_scale=1.0 / 1024.0)
    assert np.array_equal(r1["dw_bits"], rS["dw_bits"])
    a, b = r1["dx"], rS["dx"]
    normal = (np.abs(a) >= 2.0 ** -14) & (np.abs(a) * 1024 < 65504)
    assert normal.mean() > 0.9
    assert np.array_equal(a[normal] * 1024.0, b[normal])


def test_overflow_flag():
    t_ = torch()
    case = Case(L("x", 2, 32, 8, 8, 32, 3, 3, 1, 1), loss_scale=1024.0, dy_std=1e-3)
    t = case.tensors()
    flag = t_.zeros(1, dtype=t_.int32, device="cuda")
    r = run_gpu(case, t, passes=("wgrad",), flag=flag)
    assert int(flag.item()) == 0 and np.all(np.isfinite(r["dw"]))
    bad = dict(t)
    dyb = bad["dy"].copy()
    dyb.reshape(-1)[12345 % dyb.size] = 0x7C00  # +inf in fp16
    bad["dy"] = dyb
    r = run_gpu(case, bad, passes=("wgrad",), flag=flag)
    assert int(flag.item()) == 1 and not np.all(np.isfinite(r["dw"]))
    # sticky: a later clean call does not clear it
    run_gpu(case, t, passes=("wgrad",), flag=flag)
    assert int(flag.item()) == 1
    # fp16 output: finite fp32 sums that overflow fp16 also raise it
    flag.zero_()
    big = dict(t)
    big["dy"] = I.to_bits(I.from_bits(t["dy"], I.F16) * 60.0, I.F16)
    r = run_gpu(case, big, passes=("wgrad",), dw_dtype=nc.NNCONV_F16, inv_scale=64.0, flag=flag)
    assert int(flag.item()) == 1 and np.isinf(r["dw"]).any()


def test_wgrad_accumulate_and_half_output():
    case = Case(L("y", 2, 32, 9, 9, 48, 3, 3, 1, 1), loss_scale=1024.0, dy_std=1e-3)
    t = case.tensors()
    x, w, dy = nchw_f64(case, t)
    cv = oracle_conv(case)
    rng = np.random.default_rng(1)
    old = rng.standard_normal((48, 3, 3, 32)).astype(np.float32)
    r = run_gpu(case, t, passes=("wgrad",), accumulate=1, dw_old=old)
    ref = cv.wgrad(x, dy, 1.0 / 1024, beta=1, dw_old=old.astype(np.float64).transpose(0, 3, 1, 2))
    assert orc.rel_err(to_nchw(case, "dw", r["dw"]), ref) <= 1e-5
    oldh = I.to_bits(old, I.F16)
    r = run_gpu(case, t, passes=("wgrad",), accumulate=1, dw_old=oldh, dw_dtype=nc.NNCONV_F16)
    ref = cv.wgrad(x, dy, 1.0 / 1024, beta=1,
                   dw_old=I.from_bits(oldh, I.F16).reshape(48, 3, 3, 32).transpose(0, 3, 1, 2))
    assert orc.rel_err(to_nchw(case, "dw", r["dw"]), ref) <= TOL[I.F16]


@pytest.mark.parametrize("dw_dtype", ["f32", "f16"])
def test_wgrad_unaligned_dw(dw_dtype):
    """dw that is only element-aligned takes per-element stores; the bits
    match the vector-store result (same summation order)."""
    case = Case(L("z", 2, 64, 10, 9, 128, 3, 3, 1, 1), loss_scale=1024.0, dy_std=1e-3)
    t = case.tensors()
    dt = nc.NNCONV_F32 if dw_dtype == "f32" else nc.NNCONV_F16
    rng = np.random.default_rng(5)
    old = rng.standard_normal(128 * 9 * 64).astype(np.float32)
    if dw_dtype == "f16":
        old = I.to_bits(old, I.F16)
    a = run_gpu(case, t, passes=("wgrad",), dw_dtype=dt, accumulate=1, dw_old=old)
    b = run_gpu(case, t, passes=("wgrad",), dw_dtype=dt, accumulate=1, dw_old=old, dw_shift=1)
    assert np.array_equal(a["dw_bits"], b["dw_bits"])
    x, w, dy = nchw_f64(case, t)
    oldf = old.astype(np.float64) if dw_dtype == "f32" else I.from_bits(old, I.F16)
    ref = oracle_conv(case).wgrad(x, dy, 1.0 / 1024, beta=1,
                                  dw_old=oldf.reshape(128, 3, 3, 64).transpose(0, 3, 1, 2))
    assert orc.rel_err(to_nchw(case, "dw", b["dw"]), ref) <= (1e-5 if dw_dtype == "f32" else TOL[I.F16])


def test_transforms_vector_path_bit_exact():
    """Sizes that take the 16-byte transpose path (multiples of 8), with
    ragged 64x64 tiles and channel padding."""
    tt = torch()
    rng = np.random.default_rng(4)
    s = stream()
    n, c, h, w, cp = 2, 72, 5, 16, 80
    src = rng.integers(0, 65535, size=(n, c, h, w), dtype=np.uint16)
    out = Guarded(n * h * w * cp)
    nc.check(nc.nnconv_nchw_to_nhwc(to_dev(src).data_ptr(), out.ptr(), n, c, h, w, cp, s))
    tt.cuda.synchronize()
    ref = np.zeros((n, h, w, cp), np.uint16)
    ref[..., :c] = src.transpose(0, 2, 3, 1)
    assert np.array_equal(out.host().reshape(n, h, w, cp), ref)
    nhwc = np.ascontiguousarray(src.transpose(0, 2, 3, 1))
    back = Guarded(n * c * h * w)
    nc.check(nc.nnconv_nhwc_to_nchw(to_dev(nhwc).data_ptr(), back.ptr(), n, c, h, w, s))
    tt.cuda.synchronize()
    assert np.array_equal(back.host().reshape(src.shape), src)


def test_transforms_bit_exact():
    tt = torch()
    rng = np.random.default_rng(3)
    s = stream()
    n, c, h, w, cp = 3, 5, 7, 9, 8
    src = rng.integers(0, 65535, size=(n, c, h, w), dtype=np.uint16)
    d_src = to_dev(src)
    out = Guarded(n * h * w * cp)
    nc.check(nc.nnconv_nchw_to_nhwc(d_src.data_ptr(), out.ptr(), n, c, h, w, cp, s))
    tt.cuda.synchronize()
    ref = np.zeros((n, h, w, cp), np.uint16)
    ref[..., :c] = src.transpose(0, 2, 3, 1)
    assert np.array_equal(out.host().reshape(n, h, w, cp), ref)
    nhwc = np.ascontiguousarray(src.transpose(0, 2, 3, 1))
    back = Guarded(n * c * h * w)
    nc.check(nc.nnconv_nhwc_to_nchw(to_dev(nhwc).data_ptr(), back.ptr(), n, c, h, w, s))
    tt.cuda.synchronize()
    assert np.array_equal(back.host().reshape(src.shape), src)
    padded = Guarded(n * h * w * cp)
    nc.check(nc.nnconv_pad_channels(to_dev(nhwc).data_ptr(), padded.ptr(), n * h * w, c, cp, s))
    tt.cuda.synchronize()
    assert np.array_equal(padded.host().reshape(n, h, w, cp), ref)
    k, cg, r, sz = 6, 5, 3, 2
    wk = rng.integers(0, 65535, size=(k, cg, r, sz), dtype=np.uint16)
    o = Guarded(k * r * sz * 8)
    nc.check(nc.nnconv_weight_kcrs_to_krsc(to_dev(wk).data_ptr(), o.ptr(), k, cg, r, sz, 8, s))
    tt.cuda.synchronize()
    refw = np.zeros((k, r, sz, 8), np.uint16)
    refw[..., :cg] = wk.transpose(0, 2, 3, 1)
    assert np.array_equal(o.host().reshape(refw.shape), refw)
    krsc = np.ascontiguousarray(wk.transpose(0, 2, 3, 1))
    o2 = Guarded(wk.size)
    nc.check(nc.nnconv_weight_krsc_to_kcrs(to_dev(krsc).data_ptr(), o2.ptr(), k, cg, r, sz, s))
    tt.cuda.synchronize()
    assert np.array_equal(o2.host().reshape(wk.shape), wk)
