"""Workload parity at full size.

Each seeded workload (the stage-1 bottleneck at batch 64, the stage
transitions at batch 128, the stem at batch 128, every distinct layer of
the 53-layer ResNet-50 sweep at batch 256, the depthwise layers of
EfficientNet-B0 at batch 128 and the grouped layers of ResNeXt-50 at batch
128) runs through the same library
calls, descriptors and therefore the same kernel launches that bench.py
times.  The oracle's single-point routines then evaluate sampled outputs:
65,536 random positions of y and of dx, every border pixel (all channels) of
the first and last image, and 2,048 random weight-gradient entries plus the
first and last filter in full.  The error is max|err| / max|ref| over the
sampled positions.  Every output element is also checked for bitwise
reproducibility across two runs.

Every distinct sweep, depthwise and grouped layer also runs at batch 3
(ragged tiles) against the full oracle, in fp16 and bf16."""
import zlib

import numpy as np
import pytest

import oracle.oracle as orc
from gpu_util import TOL, Case, full_parity, nchw_f64, oracle_conv, run_gpu, torch
from paper_2102_06725_amd import inputs as I
from paper_2102_06725_amd import nnconv as nc

pytestmark = pytest.mark.gpu

N_RANDOM = 65536
N_DW_RANDOM = 2048


@pytest.fixture(scope="module", autouse=True)
def _setup(nnlib, oracle_lib):
    t = torch()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    orc.set_threads(min(16, max(1, orc.get_threads())))
    yield


def workload_cases(cfg, dtype=I.F16):
    wl = I.workload(cfg, dtype)
    out = []
    for li, L in enumerate(wl.layers):
        out.append(("cfg%d %s" % (cfg, L.name),
                    Case(L, layout=wl.layout, dtype=dtype, loss_scale=wl.loss_scale,
                         x_kind=wl.x_kind, dy_std=wl.dy_std, cfg=cfg, layer_id=li)))
    return out


FULL_SIZE = (workload_cases(2) + workload_cases(3) + workload_cases(4) + workload_cases(5) +
             workload_cases(6) + workload_cases(7))


def border_and_random(rng, shape, n_random):
    """Flat NCHW indices: n_random random positions plus every border pixel
    (all channels) of the first and the last image."""
    n, c, h, w = shape
    total = n * c * h * w
    rand = rng.integers(0, total, size=min(n_random, total), dtype=np.int64)
    ii, jj = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    edge = (ii == 0) | (ii == h - 1) | (jj == 0) | (jj == w - 1)
    pix = (ii * w + jj)[edge]
    imgs = sorted({0, n - 1})
    border = [(b * c + ch) * h * w + pix for b in imgs for ch in range(c)]
    return np.unique(np.concatenate([rand] + border))


def pick_channel_last(flat_nhwc, idx, shape):
    """Values of a channel-last tensor at flat NCHW indices."""
    n, c, h, w = shape
    b = idx // (c * h * w)
    r = idx % (c * h * w)
    ch = r // (h * w)
    pix = r % (h * w)
    return flat_nhwc[(b * h * w + pix) * c + ch]


def sampled_rel_err(got, ref):
    scale = np.max(np.abs(ref))
    if scale == 0:
        return 0.0 if np.all(got == 0) else np.inf
    return float(np.max(np.abs(got - ref)) / scale)


@pytest.mark.parametrize("name,case", FULL_SIZE, ids=[c[0] for c in FULL_SIZE])
def test_full_size_sampled(name, case):
    L = case.layer
    t = case.tensors()
    tt = torch()
    flag = tt.zeros(1, dtype=tt.int32, device="cuda")
    passes = ("fwd", "dgrad", "wgrad") if L.dgrad else ("fwd", "wgrad")
    got = run_gpu(case, t, passes=passes, flag=flag)
    assert int(flag.item()) == 0, "overflow flag set"
    # every element, not only the sampled ones: a second run must reproduce
    # all output bits (a race between waves shows up as a few differing words)
    again = run_gpu(case, t, passes=passes, flag=flag)
    for key in ("y_bits", "dx_bits", "dw_bits"):
        if key in got:
            diff = np.count_nonzero(got[key] != again[key])
            assert diff == 0, "%s: %d elements differ between two runs" % (key, diff)
    del again
    x, w, dy = nchw_f64(case, t)
    cv = oracle_conv(case)
    cl = L.c_alg
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    tol = TOL[case.dtype]
    errs = {}

    yshape = (L.n, L.k, L.p, L.q)
    idx = border_and_random(rng, yshape, N_RANDOM)
    ref = cv.fwd_points(x, w, idx)
    g = pick_channel_last(got["y"], idx, yshape)
    assert np.all(np.isfinite(g))
    errs["fwd"] = sampled_rel_err(g, ref)

    if L.dgrad:
        xshape = (L.n, cl, L.h, L.w)
        idx = border_and_random(rng, xshape, N_RANDOM)
        ref = cv.dgrad_points(dy, w, idx)
        g = pick_channel_last(got["dx"], idx, xshape)
        assert np.all(np.isfinite(g))
        # an exactly-zero reference is an empty sum (no tap reaches the
        # position): the library must write an exact zero there too
        assert np.all(g[ref == 0] == 0), "structurally-zero dx not exactly 0"
        errs["dgrad"] = sampled_rel_err(g, ref)

    cg = L.c // L.groups
    wshape_alg = (L.k, cl // L.groups, L.r, L.s)
    per_filter = wshape_alg[1] * L.r * L.s
    total = L.k * per_filter
    idx = np.unique(np.concatenate([
        rng.integers(0, total, size=min(N_DW_RANDOM, total), dtype=np.int64),
        np.arange(per_filter, dtype=np.int64),
        np.arange(total - per_filter, total, dtype=np.int64)]))
    ref = cv.wgrad_points(x, dy, idx) / case.loss_scale
    # dw is [K][R][S][Cg] (channel-last, Cg padded for the stem)
    k = idx // per_filter
    r_ = idx % per_filter
    c = r_ // (L.r * L.s)
    rs = r_ % (L.r * L.s)
    g = got["dw"][(k * L.r * L.s + rs) * cg + c]
    assert np.all(np.isfinite(g))
    errs["wgrad"] = sampled_rel_err(g, ref)
    if cl != L.c:
        dwf = got["dw"].reshape(L.k, L.r, L.s, cg)
        assert np.all(dwf[..., cl:] == 0), "dw pad channels not exactly 0"

    print(name, {k_: "%.3e" % v for k_, v in errs.items()})
    for k_, e in errs.items():
        assert e <= tol, "%s sampled rel err %.3e > %.1e" % (k_, e, tol)


SWEEP_B3 = [("%s %s b3" % (L.name, dt),
             Case(L.with_batch(3), layout="nhwc", dtype=dt, loss_scale=1024.0,
                  x_kind="normal" if L.c_alg != L.c else "absnormal", dy_std=1e-3, cfg=5,
                  layer_id=li))
            for dt in (I.F16, I.BF16)
            for li, (L, _) in enumerate(I.resnet50_layers(3))]


SWEEP_B3 += [("%s %s b3" % (L.name, dt),
              Case(L.with_batch(3), layout="nhwc", dtype=dt, loss_scale=1024.0,
                   x_kind="absnormal", dy_std=1e-3, cfg=6, layer_id=li))
             for dt in (I.F16, I.BF16)
             for li, (L, _) in enumerate(I.efficientnet_b0_depthwise(3))]
SWEEP_B3 += [("%s %s b3" % (L.name, dt),
              Case(L.with_batch(3), layout="nhwc", dtype=dt, loss_scale=1024.0,
                   x_kind="absnormal", dy_std=1e-3, cfg=7, layer_id=li))
             for dt in (I.F16, I.BF16)
             for li, (L, _) in enumerate(I.resnext50_grouped(3))]


@pytest.mark.parametrize("name,case", SWEEP_B3, ids=[c[0] for c in SWEEP_B3])
def test_sweep_layer_batch3_full(name, case):
    passes = ("fwd", "dgrad", "wgrad") if case.layer.dgrad else ("fwd", "wgrad")
    errs = full_parity(case, passes=passes)
    print(name, {k: "%.3e" % v for k, v in errs.items()})
