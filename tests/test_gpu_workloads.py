"""Workload parity at full size.

Each seeded workload (the stage-1 bottleneck at batch 64, the stage
transitions at batch 128, the stem at batch 128, every distinct layer of
the 53-layer ResNet-50 sweep at batch 256, the depthwise layers of
EfficientNet-B0 at batch 128 and the grouped layers of ResNeXt-50 at batch
128) runs through the same library
calls, descriptors and therefore the same kernel launches that bench.py
times.  The oracle's single-point routines then evaluate sampled outputs:
65,536 random positions of y and of dx, every border pixel (all channels) of
the first and last image, and 2,048 random weight-gradient entries plus
whole filters: the first, the last and one in every block of 32 filters
(at an offset that changes from block to block), so every row block and
column of every backward-weight tile is checked.  The error is max|err| / max|ref| over the
sampled positions.  Every output element is also checked for bitwise
reproducibility across two runs.

The sweep layers run at full size in bf16 too.  Every distinct sweep,
depthwise and grouped layer also runs at batch 3 (ragged tiles) against the
full oracle, in fp16 and bf16."""
import zlib

import numpy as np
import pytest

import oracle.oracle as orc
from gpu_util import TOL, Case, full_parity, nchw_f64, oracle_conv, run_gpu, to_dev, torch
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


def bf16_cases(cfg):
    return [(name + " bf16", case) for name, case in workload_cases(cfg, I.BF16)]


# the 53-layer sweep also in bf16 at its real size: at batch 256 the picker
# sends the 14x14 layers to the 256x256 tiles, which smaller batches never
# reach
FULL_SIZE = (workload_cases(2) + workload_cases(3) + workload_cases(4) + workload_cases(5) +
             bf16_cases(5) + workload_cases(6) + workload_cases(7))


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
    # whole filters: the first, the last, and one in every block of 32
    # (the matrix-core row block of every backward-weight tile) at an offset
    # that differs from block to block, so every row block and every column
    # of every output tile has a complete row under the oracle
    rows = sorted({0, L.k - 1} | {32 * b + (7 * b + 13) % min(32, L.k)
                                  for b in range((L.k + 31) // 32)
                                  if 32 * b + (7 * b + 13) % min(32, L.k) < L.k})
    idx = np.unique(np.concatenate(
        [rng.integers(0, total, size=min(N_DW_RANDOM, total), dtype=np.int64)] +
        [np.arange(k * per_filter, (k + 1) * per_filter, dtype=np.int64) for k in rows]))
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


def test_operand_of_2_gib_takes_the_direct_path():
    """Maximum size: x of exactly 2 GiB (1 x 128 x 128 x 65536 fp16,
    channel-last) is past the byte range the fast kernels address with
    32-bit buffer offsets, so all three passes run on the direct kernels,
    which index with 64 bits.  Sampled outputs against the oracle applied to
    gathered sub-problems: a 1x1 stride-1 convolution is pointwise in space
    (y and dx at a pixel depend only on that pixel's channel column), and
    dw[k][c] depends only on input channel c and output channel k."""
    tt = torch()
    L = I.Layer("x2gib", 1, 65536, 128, 128, 8, 1, 1)
    case = Case(L, layout="nhwc", dtype=I.F16, loss_scale=1.0, x_kind="absnormal", dy_std=1.0,
                cfg=91)
    t = case.tensors()
    assert t["x"].nbytes == 2 ** 31
    d = case.desc()
    s = tt.cuda.current_stream().cuda_stream
    x, w, dy = to_dev(t["x"]), to_dev(t["w"]), to_dev(t["dy"])
    y = tt.empty(L.n * L.p * L.q * L.k, dtype=tt.int16, device="cuda")
    dx = tt.empty(L.n * L.h * L.w * L.c, dtype=tt.int16, device="cuda")
    dw = tt.empty(L.k * L.c, dtype=tt.float32, device="cuda")
    for p_, call in ((nc.NNCONV_FWD, lambda ws, nb: nc.nnconv_fwd(
                         d, x.data_ptr(), w.data_ptr(), y.data_ptr(), 1.0, ws, nb, s)),
                     (nc.NNCONV_DGRAD, lambda ws, nb: nc.nnconv_dgrad(
                         d, dy.data_ptr(), w.data_ptr(), dx.data_ptr(), 1.0, ws, nb, s)),
                     (nc.NNCONV_WGRAD, lambda ws, nb: nc.nnconv_wgrad(
                         d, x.data_ptr(), dy.data_ptr(), dw.data_ptr(), nc.NNCONV_F32, 1.0, 0,
                         None, ws, nb, s))):
        st, nb = nc.nnconv_workspace_size(d, p_)
        nc.check(st, "workspace_size")
        ws = tt.empty(max(nb, 1), dtype=tt.uint8, device="cuda")
        nc.check(call(ws.data_ptr(), nb), "pass %d" % p_)
        tt.cuda.synchronize()
        del ws
    rng = np.random.default_rng(2 ** 31)
    pix = np.unique(np.concatenate([[0, 127, 128 * 127, 128 * 128 - 1],
                                    rng.integers(0, 128 * 128, size=28)]))
    ph, pq = pix // 128, pix % 128
    wf = I.from_bits(np.ascontiguousarray(t["w"].reshape(L.k, L.c)), I.F16).reshape(L.k, L.c, 1, 1)
    tol = TOL[I.F16]

    xs = I.from_bits(np.ascontiguousarray(t["x"][0, ph, pq, :]), I.F16)          # (S, C)
    sub = orc.Conv(len(pix), L.c, 1, 1, L.k, 1, 1, (1, 1), (0, 0), (1, 1), 1)
    ref = sub.fwd(xs.reshape(len(pix), L.c, 1, 1), wf).reshape(len(pix), L.k)
    got = y.view(L.p, L.q, L.k)[tt.from_numpy(ph).cuda(), tt.from_numpy(pq).cuda()]
    got = I.from_bits(got.cpu().numpy().view(np.uint16), I.F16)
    assert sampled_rel_err(got, ref) <= tol

    dys = I.from_bits(np.ascontiguousarray(t["dy"][0, ph, pq, :]), I.F16)        # (S, K)
    ref = sub.dgrad(dys.reshape(len(pix), L.k, 1, 1), wf).reshape(len(pix), L.c)
    got = dx.view(L.h, L.w, L.c)[tt.from_numpy(ph).cuda(), tt.from_numpy(pq).cuda()]
    got = I.from_bits(got.cpu().numpy().view(np.uint16), I.F16)
    assert sampled_rel_err(got, ref) <= tol

    chans = np.unique(np.concatenate([[0, L.c - 1], rng.integers(0, L.c, size=14)]))
    dyall = I.from_bits(np.ascontiguousarray(t["dy"][0].transpose(2, 0, 1)), I.F16)  # (K, H, W)
    sub1 = orc.Conv(1, 1, L.h, L.w, L.k, 1, 1, (1, 1), (0, 0), (1, 1), 1)
    dwall = dw.view(L.k, L.c).cpu().numpy().astype(np.float64)
    for c in chans:
        xc = I.from_bits(np.ascontiguousarray(t["x"][0, :, :, c]), I.F16)
        ref = sub1.wgrad(xc.reshape(1, 1, L.h, L.w), dyall.reshape(1, L.k, L.h, L.w), 1.0)
        assert sampled_rel_err(dwall[:, c], ref.reshape(L.k)) <= tol, "channel %d" % c
