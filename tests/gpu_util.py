"""Helpers for the GPU parity tests: run one convolution geometry through
libnnconv (via the C ABI binding) and through the fp64 oracle on the same
seeded, quantised inputs, and compare.

Outputs are written between guard bands filled with a fixed byte pattern;
the bands must be untouched afterwards."""
from __future__ import annotations

import dataclasses

import numpy as np

import oracle.oracle as orc
from paper_2102_06725_amd import inputs as I
from paper_2102_06725_amd import nnconv as nc

TOL = {I.F16: 2e-3, I.BF16: 5e-3}
GUARD = 64          # guard elements on each side (keeps 16-byte alignment)
CANARY16 = 0xA5A5
CANARY32 = 0x5A5A5A5A


def torch():
    import torch as t
    return t


def to_dev(bits: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")


class Shifted:
    """16-bit input bits on the device starting `shift` elements past a
    16-byte aligned allocation (data_ptr() is the shifted address)."""

    def __init__(self, bits: np.ndarray, shift: int):
        flat = np.ascontiguousarray(bits).view(np.int16).ravel()
        host = np.zeros(flat.size + shift, np.int16)
        host[shift:] = flat
        self.buf = to_dev(host)
        self.shift = shift

    def data_ptr(self) -> int:
        return self.buf.data_ptr() + 2 * self.shift


class Guarded:
    """A device buffer of `numel` elements with guard bands on both sides."""

    def __init__(self, numel: int, fp32: bool = False, init: np.ndarray | None = None,
                 shift: int = 0):
        """`shift` elements move the start off 16-byte alignment."""
        t = torch()
        self.fp32 = fp32
        self.numel = numel
        self.lo = GUARD + shift
        if fp32:
            host = np.full(numel + 2 * GUARD + shift, CANARY32, np.uint32)
        else:
            host = np.full(numel + 2 * GUARD + shift, CANARY16, np.uint16)
        if init is not None:
            host[self.lo:self.lo + numel] = np.ascontiguousarray(init).ravel().view(host.dtype)
        self.buf = t.from_numpy(host.view(np.int32 if fp32 else np.int16)).to("cuda")
        self.view = self.buf[self.lo:self.lo + numel]

    def ptr(self) -> int:
        return self.view.data_ptr()

    def host(self) -> np.ndarray:
        h = self.buf.cpu().numpy()
        h = h.view(np.uint32 if self.fp32 else np.uint16)
        c = CANARY32 if self.fp32 else CANARY16
        assert np.all(h[:self.lo] == c) and np.all(h[self.lo + self.numel:] == c), \
            "guard band overwritten"
        return h[self.lo:self.lo + self.numel]


@dataclasses.dataclass
class Case:
    layer: I.Layer
    layout: str = "nhwc"
    dtype: str = I.F16
    loss_scale: float = 1.0
    x_kind: str = "absnormal"
    dy_std: float = 1.0
    cfg: int = 90
    layer_id: int = 0
    alpha: float = 1.0

    @property
    def workload(self):
        L = self.layer
        return I.Workload("test", (L,), self.layout, self.dtype, self.loss_scale, self.x_kind, 1.0,
                          "he", self.dy_std)

    def tensors(self):
        return I.layer_tensors(self.workload, self.layer_id, self.cfg, self.layer)

    def desc(self):
        L = self.layer
        return nc.make_desc(L.n, L.c, L.h, L.w, L.k, L.r, L.s, (L.stride, L.s_w),
                            (L.pad, L.p_w), (L.dil, L.d_w), L.groups,
                            nc.NNCONV_NCHW if self.layout == "nchw" else nc.NNCONV_NHWC,
                            nc.NNCONV_F16 if self.dtype == I.F16 else nc.NNCONV_BF16)


def nchw_f64(case: Case, t):
    """Operands as float64 in the oracle's [N][C][H][W] / [K][Cg][R][S] form,
    restricted to the logical channels (the stem's pad channels dropped).
    The 16-bit patterns are rearranged first, then converted."""
    L = case.layer
    cl = L.c_alg
    x, w, dy = t["x"], t["w"], t["dy"]
    if case.layout == "nhwc":
        x = x[..., :cl].transpose(0, 3, 1, 2)
        w = w[..., :cl // L.groups].transpose(0, 3, 1, 2)
        dy = dy.transpose(0, 3, 1, 2)
    else:
        x = x[:, :cl]
        w = w[:, :cl // L.groups]
    return (I.from_bits(np.ascontiguousarray(x), case.dtype),
            I.from_bits(np.ascontiguousarray(w), case.dtype),
            I.from_bits(np.ascontiguousarray(dy), case.dtype))


def oracle_conv(case: Case):
    L = case.layer
    return orc.Conv(L.n, L.c_alg, L.h, L.w, L.k, L.r, L.s, (L.stride, L.s_w), (L.pad, L.p_w),
                    (L.dil, L.d_w), L.groups)


def workspace(desc, pass_):
    t = torch()
    st, nb = nc.nnconv_workspace_size(desc, pass_)
    nc.check(st, "workspace_size")
    ws = t.empty(max(nb, 1) + 2 * GUARD, dtype=t.uint8, device="cuda")
    ws.fill_(0xC3)
    return ws, nb


def stream():
    return torch().cuda.current_stream().cuda_stream


def run_gpu(case: Case, t, passes=("fwd", "dgrad", "wgrad"), dw_dtype=None, inv_scale=None,
            accumulate=0, dw_old=None, flag=None, dw_shift=0, in_shift=0, out_shift=0,
            tile=None):
    """Run the requested passes on the GPU; returns dict of output bits /
    fp32 values in the case's layout.  in_shift / out_shift move x, w, dy /
    y, dx that many 16-bit elements off 16-byte alignment.  tile: force this
    implicit-GEMM tile on the forward and backward-data passes."""
    L = case.layer
    tt = torch()
    d = case.desc()
    if in_shift:
        x, w, dy = (Shifted(t["x"], in_shift), Shifted(t["w"], in_shift),
                    Shifted(t["dy"], in_shift))
    else:
        x, w, dy = to_dev(t["x"]), to_dev(t["w"]), to_dev(t["dy"])
    out = {}
    s = stream()
    if "fwd" in passes:
        y = Guarded(L.n * L.k * L.p * L.q, shift=out_shift)
        ws, nb = workspace(d, nc.NNCONV_FWD)
        if tile is None:
            st = nc.nnconv_fwd(d, x.data_ptr(), w.data_ptr(), y.ptr(), case.alpha, ws.data_ptr(),
                               nb, s)
        else:
            st = nc.nnconv_fwd_tile(d, x.data_ptr(), w.data_ptr(), y.ptr(), case.alpha,
                                    ws.data_ptr(), nb, s, tile)
        nc.check(st, "fwd")
        out["y"] = y
    if "dgrad" in passes:
        dx = Guarded(L.n * L.c * L.h * L.w, shift=out_shift)
        ws, nb = workspace(d, nc.NNCONV_DGRAD)
        if tile is None:
            st = nc.nnconv_dgrad(d, dy.data_ptr(), w.data_ptr(), dx.ptr(), case.alpha,
                                 ws.data_ptr(), nb, s)
        else:
            st = nc.nnconv_dgrad_tile(d, dy.data_ptr(), w.data_ptr(), dx.ptr(), case.alpha,
                                      ws.data_ptr(), nb, s, tile)
        nc.check(st, "dgrad")
        out["dx"] = dx
    if "wgrad" in passes:
        fp32 = dw_dtype in (None, nc.NNCONV_F32)
        dwt = Guarded(L.k * L.r * L.s * (L.c // L.groups), fp32=fp32, init=dw_old,
                      shift=dw_shift)
        ws, nb = workspace(d, nc.NNCONV_WGRAD)
        inv = (1.0 / case.loss_scale) if inv_scale is None else inv_scale
        nc.check(nc.nnconv_wgrad(d, x.data_ptr(), dy.data_ptr(), dwt.ptr(),
                                 nc.NNCONV_F32 if fp32 else dw_dtype, inv, accumulate,
                                 flag.data_ptr() if flag is not None else None, ws.data_ptr(),
                                 nb, s), "wgrad")
        out["dw"] = dwt
    tt.cuda.synchronize()
    res = {}
    for k, g in out.items():
        h = g.host()
        if g.fp32:
            res[k] = h.view(np.float32).astype(np.float64)
        else:
            res[k] = I.from_bits(h, case.dtype)
        res[k + "_bits"] = h.copy()
    return res


def shape_of(case: Case, which: str):
    L = case.layer
    nchw = case.layout == "nchw"
    cg = L.c // L.groups
    if which == "y":
        return (L.n, L.k, L.p, L.q) if nchw else (L.n, L.p, L.q, L.k)
    if which == "dx":
        return (L.n, L.c, L.h, L.w) if nchw else (L.n, L.h, L.w, L.c)
    return (L.k, cg, L.r, L.s) if nchw else (L.k, L.r, L.s, cg)


def to_nchw(case: Case, which: str, a):
    a = a.reshape(shape_of(case, which))
    if case.layout == "nhwc":
        a = a.transpose(0, 3, 1, 2)
    return a


def full_parity(case: Case, passes=("fwd", "dgrad", "wgrad"), tile=None):
    """Run every pass, compare against the full oracle.  Returns errors."""
    t = case.tensors()
    got = run_gpu(case, t, passes, tile=tile)
    x, w, dy = nchw_f64(case, t)
    cv = oracle_conv(case)
    L = case.layer
    cl = L.c_alg
    errs = {}
    tol = TOL[case.dtype]
    if "fwd" in passes:
        ref = cv.fwd(x, w, alpha=case.alpha)
        g = to_nchw(case, "y", got["y"])
        assert np.all(np.isfinite(g)), "non-finite forward output"
        errs["fwd"] = orc.rel_err(g, ref)
    if "dgrad" in passes:
        ref = cv.dgrad(dy, w, alpha=case.alpha)
        g = to_nchw(case, "dx", got["dx"])
        assert np.all(np.isfinite(g)), "non-finite dgrad output"
        if cl != L.c:
            assert not np.any(g[:, cl:]), "dgrad pad channels not zero"
            g = g[:, :cl]
        # positions no output reads must be exact zeros
        zero = ref == 0
        structural = cv.dgrad(np.ones_like(dy), np.ones_like(w)) == 0
        assert np.all(g[structural & zero] == 0), "structurally-zero dx not exactly 0"
        errs["dgrad"] = orc.rel_err(g, ref)
    if "wgrad" in passes:
        ref = cv.wgrad(x, dy, 1.0 / case.loss_scale)
        g = to_nchw(case, "dw", got["dw"])
        assert np.all(np.isfinite(g)), "non-finite wgrad output"
        if cl != L.c:
            assert np.all(g[:, cl:] == 0), "dw pad channels not exactly 0"
            g = g[:, :cl]
        errs["wgrad"] = orc.rel_err(g, ref)
    for k, e in errs.items():
        assert e <= tol, "%s rel err %.3e > %.1e for %r" % (k, e, tol, case)
    return errs
