"""Seeded random geometries, all three passes against the fp64 oracle.

The hand-picked parity cases pin each kernel path on shapes chosen for it;
these draw combinations nobody picked: layout, dtype, loss scale, filter
size, stride, padding, dilation, group structure and ragged image sizes,
from five families that between them reach every dispatch path (8-channel
and 64-channel implicit GEMMs with their stride phases, the direct kernels,
the tiled and gather depthwise kernels, and 64-channel super-groups), with
alpha != 1 on about a third of them.  Sizes
are capped so that the oracle takes well under a second per case."""
import dataclasses

import numpy as np
import pytest

import oracle.oracle as orc
from gpu_util import TOL, Case, full_parity, nchw_f64, oracle_conv, run_gpu, to_nchw, torch
from paper_2102_06725_amd import inputs as I
from paper_2102_06725_amd import nnconv as nc

pytestmark = pytest.mark.gpu

SEED = 2102
N_CASES = 200
MAX_MACS = 40_000_000      # per pass, keeps the fp64 oracle fast


def _draw(rng, i):
    fam = ("dense8", "dense64", "odd", "depthwise", "super")[i % 5]
    n = int(rng.integers(1, 4))
    h, w = int(rng.integers(1, 21)), int(rng.integers(1, 21))
    stride = int(rng.integers(1, 4))
    dil = int(rng.choice([1, 1, 2]))
    groups = 1
    if fam == "dense8":
        c, k = 8 * int(rng.integers(1, 13)), 8 * int(rng.integers(1, 13))
        r = s = int(rng.choice([1, 2, 3, 5]))
    elif fam == "dense64":
        c, k = 64 * int(rng.integers(1, 3)), 64 * int(rng.integers(1, 4))
        r = s = int(rng.choice([1, 3, 3, 5]))
    elif fam == "odd":
        groups = int(rng.choice([1, 1, 2, 3]))
        c = groups * int(rng.integers(1, 9))
        k = groups * int(rng.integers(1, 9))
        r, s = int(rng.integers(1, 6)), int(rng.integers(1, 6))
    elif fam == "depthwise":
        c = k = groups = 8 * int(rng.integers(1, 7))
        r = s = int(rng.choice([3, 5, 7]))
        stride = int(rng.choice([1, 2, 2, 3]))
        h, w = int(rng.integers(3, 25)), int(rng.integers(3, 25))
    else:  # super-groups: 2-32 channel groups, channels a multiple of 64
        cg = int(rng.choice([2, 4, 8, 16, 32]))
        c = k = 64 * int(rng.integers(1, 3))
        groups = c // cg
        r = s = int(rng.choice([1, 3, 3]))
    pad = int(rng.integers(0, dil * (max(r, s) - 1) + 1))
    return fam, I.Layer("rnd%d_%s" % (i, fam), n, c, h, w, k, r, s, stride, pad, dil, groups)


def _cases():
    rng = np.random.default_rng(SEED)
    rng_alpha = np.random.default_rng(SEED + 7)   # alpha of fwd / dgrad
    out = []
    i = 0
    while len(out) < N_CASES:
        fam, L = _draw(rng, i)
        i += 1
        if L.p < 1 or L.q < 1:
            continue
        if L.n * L.k * L.p * L.q * (L.c // L.groups) * L.r * L.s > MAX_MACS:
            continue
        layout = "nchw" if rng.random() < 0.3 else "nhwc"
        dtype = I.BF16 if rng.random() < 0.35 else I.F16
        scale = float(rng.choice([1.0, 128.0, 1024.0]))
        alpha = 1.0 if rng_alpha.random() < 0.7 else float(rng_alpha.choice([0.5, 2.0, 0.3, -1.0]))
        out.append(Case(L, layout=layout, dtype=dtype, loss_scale=scale, cfg=93,
                        layer_id=len(out), alpha=alpha))
    return out


CASES = _cases()


def _id(c):
    L = c.layer
    return "%s n%d c%d %dx%d k%d r%ds%d st%d p%d d%d g%d %s %s a%g" % (
        L.name, L.n, L.c, L.h, L.w, L.k, L.r, L.s, L.stride, L.pad, L.dil, L.groups, c.layout,
        c.dtype, c.alpha)


def _axis_cases(n_cases=60):
    """Geometries whose stride, padding and dilation differ between the
    height and the width axis, from the same five families: the per-axis
    index logic (stride phases and their taps, padding masks, the split-K
    pixel decode, the depthwise and direct kernels) sees each axis alone."""
    rng = np.random.default_rng(SEED + 8000)
    out = []
    i = 0
    while len(out) < n_cases:
        fam, L = _draw(rng, i)
        i += 1
        sw = int(rng.integers(1, 4))
        dw = int(rng.choice([1, 1, 2]))
        if (sw, dw) == (L.stride, L.dil):
            sw = L.stride % 3 + 1
        pw = int(rng.integers(0, dw * (L.s - 1) + 1))
        L = dataclasses.replace(L, name="ax%d_%s" % (i, fam), stride_w=sw, dil_w=dw, pad_w=pw)
        if L.p < 1 or L.q < 1:
            continue
        if L.n * L.k * L.p * L.q * (L.c // L.groups) * L.r * L.s > MAX_MACS:
            continue
        layout = "nchw" if rng.random() < 0.3 else "nhwc"
        dtype = I.BF16 if rng.random() < 0.35 else I.F16
        out.append(Case(L, layout=layout, dtype=dtype, loss_scale=float(rng.choice([1.0, 1024.0])),
                        cfg=95, layer_id=len(out)))
    return out


AX_CASES = _axis_cases()


def _axid(c):
    L = c.layer
    return "%s n%d c%d %dx%d k%d r%ds%d st%d,%d p%d,%d d%d,%d g%d %s %s" % (
        L.name, L.n, L.c, L.h, L.w, L.k, L.r, L.s, L.stride, L.s_w, L.pad, L.p_w, L.dil, L.d_w,
        L.groups, c.layout, c.dtype)


@pytest.fixture(scope="module", autouse=True)
def _setup(nnlib, oracle_lib):
    if not torch().cuda.is_available():
        pytest.skip("no GPU")
    yield


@pytest.mark.parametrize("case", CASES, ids=[_id(c) for c in CASES])
def test_random_shape_parity(case):
    print("case:", _id(case), flush=True)
    full_parity(case)


@pytest.mark.parametrize("case", AX_CASES, ids=[_axid(c) for c in AX_CASES])
def test_random_unequal_axes_parity(case):
    print("case:", _axid(case), flush=True)
    full_parity(case)


WG_CASES = CASES[::3]


@pytest.mark.parametrize("case", WG_CASES, ids=[_id(c) for c in WG_CASES])
def test_random_wgrad_output_modes(case):
    """Backward-weight with the other output modes on the same geometries:
    dw in fp32 or in the operand dtype, written (beta = 0) or added to a
    previous dw (beta = 1), against the oracle's beta*dw_old + sum/S from the
    exact values the GPU was given."""
    print("case:", _id(case), flush=True)
    L = case.layer
    cg = L.c // L.groups
    rng = np.random.default_rng(SEED + 1000 + case.layer_id)
    half = bool(rng.integers(0, 2))
    beta = int(rng.integers(0, 2))
    t = case.tensors()
    x, w, dy = nchw_f64(case, t)
    old = rng.standard_normal((L.k, cg, L.r, L.s)).astype(np.float32)   # [K][Cg][R][S]
    old_lay = old if case.layout == "nchw" else old.transpose(0, 2, 3, 1)
    if half:
        dw_old = I.to_bits(np.ascontiguousarray(old_lay), case.dtype)
        old_ref = I.from_bits(dw_old, case.dtype)
        if case.layout == "nhwc":
            old_ref = old_ref.transpose(0, 3, 1, 2)
        dw_dtype = nc.NNCONV_F16 if case.dtype == I.F16 else nc.NNCONV_BF16
    else:
        dw_old = np.ascontiguousarray(old_lay)
        old_ref = old.astype(np.float64)
        dw_dtype = nc.NNCONV_F32
    got = run_gpu(case, t, passes=("wgrad",), dw_dtype=dw_dtype, accumulate=beta,
                  dw_old=dw_old if beta else None)
    ref = oracle_conv(case).wgrad(x, dy, 1.0 / case.loss_scale, beta=beta,
                                  dw_old=old_ref if beta else None)
    g = to_nchw(case, "dw", got["dw"])
    assert np.all(np.isfinite(g))
    tol = TOL[case.dtype] if half else 1e-4
    assert orc.rel_err(g, ref) <= tol, (half, beta)


FLAG_CASES = CASES[::5]
INF_BITS = {I.F16: 0x7C00, I.BF16: 0x7F80}


@pytest.mark.parametrize("case", FLAG_CASES, ids=[_id(c) for c in FLAG_CASES])
def test_random_overflow_flag(case):
    """The overflow flag on every dispatch path: clear after a clean
    backward-weight, set when one dy element is +inf (that output channel's
    dw sums become inf or NaN, as inf * 0 is NaN)."""
    print("case:", _id(case), flush=True)
    tt = torch()
    rng = np.random.default_rng(SEED + 2000 + case.layer_id)
    dw_dtype = nc.NNCONV_F32 if rng.integers(0, 2) else (
        nc.NNCONV_F16 if case.dtype == I.F16 else nc.NNCONV_BF16)
    t = case.tensors()
    flag = tt.zeros(1, dtype=tt.int32, device="cuda")
    run_gpu(case, t, passes=("wgrad",), dw_dtype=dw_dtype, flag=flag)
    assert int(flag.item()) == 0, "flag set on finite inputs"
    bad = dict(t)
    dy = np.array(t["dy"], copy=True)
    dy.reshape(-1)[int(rng.integers(0, dy.size))] = INF_BITS[case.dtype]
    bad["dy"] = dy
    run_gpu(case, bad, passes=("wgrad",), dw_dtype=dw_dtype, flag=flag)
    assert int(flag.item()) == 1, "flag not set with an inf in dy"


NF_CASES = CASES[2::5]


def _super_group(case):
    L = case.layer
    return 1 < L.groups < L.c and L.c == L.k and L.c % 64 == 0 and (L.c // L.groups) < 64


@pytest.mark.parametrize("case", NF_CASES, ids=[_id(c) for c in NF_CASES])
def test_random_nonfinite_forward(case):
    """Where a non-finite operand reaches in the forward pass: one +inf in x,
    then one in w; the outputs that are not finite (none if the pixel is
    never read) are those of the oracle
    (which multiplies the padding zeros, 0 * inf = NaN).  Super-groups run
    64-channel blocks with zero weights between groups, which may only add
    NaNs inside the block that holds the bad value."""
    print("case:", _id(case), flush=True)
    rng = np.random.default_rng(SEED + 3000 + case.layer_id)
    t = case.tensors()
    cv = oracle_conv(case)
    for which in ("x", "w"):
        bad = dict(t)
        a = np.array(t[which], copy=True)
        a.reshape(-1)[int(rng.integers(0, a.size))] = INF_BITS[case.dtype]
        bad[which] = a
        got = run_gpu(case, bad, passes=("fwd",))
        g = to_nchw(case, "y", got["y"])
        x, w, _ = nchw_f64(case, bad)
        with np.errstate(invalid="ignore", over="ignore"):
            ref = cv.fwd(x, w)
        want, have = ~np.isfinite(ref), ~np.isfinite(g)
        # every output of the channel meets the bad weight; a strided or
        # dilated forward may never read the bad input pixel
        assert which == "x" or want.any()
        if _super_group(case):
            assert np.all(have[want]), which
        else:
            assert np.array_equal(have, want), which


@pytest.mark.parametrize("case", NF_CASES, ids=[_id(c) for c in NF_CASES])
def test_random_nonfinite_dgrad(case):
    """Backward-data with one +inf in dy, then in w: the non-finite dx are
    exactly the oracle's.  The matrix-core and depthwise kernels read dy
    zero-extended at every tap; with a non-finite weight the library
    recomputes the border pixels from the definition, so no NaN appears
    where the definition has no term with that weight.  Super-groups, whose
    zero weights between groups meet a non-finite value, only have to cover
    the oracle's non-finite dx."""
    print("case:", _id(case), flush=True)
    rng = np.random.default_rng(SEED + 4000 + case.layer_id)
    t = case.tensors()
    cv = oracle_conv(case)
    for which in ("dy", "w"):
        bad = dict(t)
        a = np.array(t[which], copy=True)
        a.reshape(-1)[int(rng.integers(0, a.size))] = INF_BITS[case.dtype]
        bad[which] = a
        got = run_gpu(case, bad, passes=("dgrad",))
        g = to_nchw(case, "dx", got["dx"])
        _, w, dy = nchw_f64(case, bad)
        with np.errstate(invalid="ignore", over="ignore"):
            ref = cv.dgrad(dy, w, alpha=case.alpha)
        want, have = ~np.isfinite(ref), ~np.isfinite(g)
        if not _super_group(case):
            assert np.array_equal(have, want), which
            # and the finite values are still the oracle's
            fin = ~want
            if fin.any():
                assert orc.rel_err(g[fin], ref[fin]) <= TOL[case.dtype], which
        else:
            assert np.all(have[want]), which


UA_CASES = CASES[4::7]


@pytest.mark.parametrize("case", UA_CASES, ids=[_id(c) for c in UA_CASES])
def test_random_unaligned_operands(case):
    """Operands one or three 16-bit elements off 16-byte alignment (inputs,
    outputs and dw) must take kernels that need no alignment and give the
    oracle's results."""
    print("case:", _id(case), flush=True)
    rng = np.random.default_rng(SEED + 5000 + case.layer_id)
    sh_in, sh_out = int(rng.choice([1, 3])), int(rng.choice([0, 1, 3]))
    t = case.tensors()
    got = run_gpu(case, t, in_shift=sh_in, out_shift=sh_out, dw_shift=1)
    x, w, dy = nchw_f64(case, t)
    cv = oracle_conv(case)
    tol = TOL[case.dtype]
    assert orc.rel_err(to_nchw(case, "y", got["y"]), cv.fwd(x, w, alpha=case.alpha)) <= tol
    assert orc.rel_err(to_nchw(case, "dx", got["dx"]), cv.dgrad(dy, w, alpha=case.alpha)) <= tol
    assert orc.rel_err(to_nchw(case, "dw", got["dw"]),
                       cv.wgrad(x, dy, 1.0 / case.loss_scale)) <= tol


def _tf_shapes():
    rng = np.random.default_rng(SEED + 6000)
    out = []
    for i in range(24):
        mult8 = i % 2 == 0          # half take the 16-byte vector kernels
        c = 8 * int(rng.integers(1, 12)) if mult8 else int(rng.integers(1, 40))
        n, h, w = int(rng.integers(1, 4)), int(rng.integers(1, 70)), int(rng.integers(1, 70))
        if mult8:
            w = 8 * ((w + 7) // 8)
        c_pad = c + int(rng.choice([0, 0, 8, 16])) if mult8 else c + int(rng.integers(0, 9))
        out.append((n, c, h, w, c_pad))
    return out


@pytest.mark.parametrize("shape", _tf_shapes(), ids=lambda s: "n%d c%d %dx%d cp%d" % s)
def test_random_transforms_bit_exact(shape):
    """Layout transforms on random sizes, both the 16-byte vector kernels
    (multiples of 8) and the element ones: NCHW -> NHWC with channel
    padding, back, channel padding alone, and KCRS <-> KRSC weights, all
    bit-exact against numpy transposes of random 16-bit patterns."""
    from gpu_util import Guarded, stream, to_dev
    tt = torch()
    n, c, h, w, cp = shape
    print("shape:", shape, flush=True)
    rng = np.random.default_rng(SEED + 6100 + c * 131 + h * 7 + w)
    s = stream()
    src = rng.integers(0, 65535, size=(n, c, h, w), dtype=np.uint16)
    ref = np.zeros((n, h, w, cp), np.uint16)
    ref[..., :c] = src.transpose(0, 2, 3, 1)
    out = Guarded(n * h * w * cp)
    nc.check(nc.nnconv_nchw_to_nhwc(to_dev(src).data_ptr(), out.ptr(), n, c, h, w, cp, s))
    nhwc = np.ascontiguousarray(src.transpose(0, 2, 3, 1))
    back = Guarded(n * c * h * w)
    nc.check(nc.nnconv_nhwc_to_nchw(to_dev(nhwc).data_ptr(), back.ptr(), n, c, h, w, s))
    padded = Guarded(n * h * w * cp)
    nc.check(nc.nnconv_pad_channels(to_dev(nhwc).data_ptr(), padded.ptr(), n * h * w, c, cp, s))
    # weights: K = n*3, Cg = c, R x S from h, w
    k, r, sz = 3 * n, 1 + h % 5, 1 + w % 4
    wk = rng.integers(0, 65535, size=(k, c, r, sz), dtype=np.uint16)
    o = Guarded(k * r * sz * cp)
    nc.check(nc.nnconv_weight_kcrs_to_krsc(to_dev(wk).data_ptr(), o.ptr(), k, c, r, sz, cp, s))
    o2 = Guarded(wk.size)
    nc.check(nc.nnconv_weight_krsc_to_kcrs(
        to_dev(np.ascontiguousarray(wk.transpose(0, 2, 3, 1))).data_ptr(), o2.ptr(), k, c, r, sz, s))
    tt.cuda.synchronize()
    assert np.array_equal(out.host().reshape(ref.shape), ref)
    assert np.array_equal(back.host().reshape(src.shape), src)
    assert np.array_equal(padded.host().reshape(ref.shape), ref)
    refw = np.zeros((k, r, sz, cp), np.uint16)
    refw[..., :c] = wk.transpose(0, 2, 3, 1)
    assert np.array_equal(o.host().reshape(refw.shape), refw)
    assert np.array_equal(o2.host().reshape(wk.shape), wk)
