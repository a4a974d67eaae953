"""Pins of the fp64 oracle: checks that tie it to something other than itself.

Each ``pin_*`` takes an oracle library handle and raises AssertionError when
the oracle disagrees with a fact fixed by mathematics or by an independent
library routine:

* library special cases: torch's float64 CPU conv2d and its two gradient
  helpers; scipy's 2-D cross-correlation; numpy matmul for 1x1 kernels;
* closed forms: all-ones operands give tap counts; a delta kernel is an
  exact shifted copy; hand-worked small examples (arithmetic shown inline);
* invariants: the adjoint identities tying the three passes together,
  groups as concatenation, dilation as a zero-inserted kernel, stride as
  subsampling, gather-form dgrad equal to scatter-form dgrad, power-of-two
  loss scale exactness, accumulate semantics, non-finite detection.

The same pins run against deliberately broken copies of the oracle
(``test_oracle_plants.py``) to show that each plausible mistake trips one.
"""
from __future__ import annotations

import itertools

import numpy as np

import oracle.oracle as orc

RTOL = 1e-12


def _close(a, b, rtol=RTOL, what=""):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= rtol * scale, "%s: max err %.3e (scale %.3e)" % (what, err, scale)


def _rand(rng, shape):
    return rng.standard_normal(shape)


# A fixed sweep of small geometries: (n, c, h, w, k, r, s, stride, pad, dil, g)
SWEEP = [
    (1, 1, 5, 7, 1, 3, 2, (1, 1), (0, 0), (1, 1), 1),
    (2, 3, 6, 5, 4, 3, 3, (1, 1), (1, 1), (1, 1), 1),
    (2, 4, 7, 6, 2, 2, 3, (2, 1), (1, 0), (1, 1), 2),
    (1, 2, 7, 7, 4, 3, 1, (2, 2), (2, 0), (1, 2), 2),
    (2, 4, 6, 7, 4, 3, 3, (1, 2), (1, 2), (2, 1), 4),
    (1, 3, 4, 6, 2, 1, 2, (3, 2), (0, 1), (1, 1), 1),
    (2, 2, 5, 5, 3, 2, 2, (3, 3), (2, 2), (2, 2), 1),
    (1, 4, 3, 2, 4, 3, 2, (1, 1), (1, 0), (1, 1), 2),
    (2, 1, 1, 1, 2, 1, 1, (1, 1), (0, 0), (1, 1), 1),
    (1, 2, 2, 3, 2, 3, 3, (2, 2), (1, 1), (1, 1), 1),
    (1, 4, 7, 5, 2, 2, 1, (1, 3), (0, 1), (3, 1), 1),
    (2, 3, 6, 6, 3, 3, 3, (2, 2), (1, 1), (1, 1), 3),
]


def _geoms():
    for (n, c, h, w, k, r, s, st, pd, dl, g) in SWEEP:
        yield dict(n=n, c=c, h=h, w=w, k=k, r=r, s=s, stride=st, pad=pd, dil=dl, groups=g)


def _conv(lib, gm):
    return orc.Conv(gm["n"], gm["c"], gm["h"], gm["w"], gm["k"], gm["r"], gm["s"],
                    gm["stride"], gm["pad"], gm["dil"], gm["groups"], lib=lib)


def _operands(cv, seed):
    rng = np.random.default_rng(seed)
    return _rand(rng, cv.x_shape), _rand(rng, cv.w_shape), _rand(rng, cv.y_shape)


# ---------------------------------------------------------------------------
# library special cases
# ---------------------------------------------------------------------------

def pin_torch(lib):
    """Forward, backward-data and backward-weight against torch's float64 CPU
    conv2d / grad.conv2d_input / grad.conv2d_weight."""
    import torch
    import torch.nn.functional as F
    for i, gm in enumerate(_geoms()):
        cv = _conv(lib, gm)
        x, w, dy = _operands(cv, 100 + i)
        tx, tw, tdy = (torch.from_numpy(a) for a in (x, w, dy))
        kw = dict(stride=gm["stride"], padding=gm["pad"], dilation=gm["dil"], groups=gm["groups"])
        y_ref = F.conv2d(tx, tw, **kw).numpy()
        _close(cv.fwd(x, w), y_ref, what="fwd %r" % (gm,))
        dx_ref = torch.nn.grad.conv2d_input(cv.x_shape, tw, tdy, **kw).numpy()
        _close(cv.dgrad(dy, w), dx_ref, what="dgrad %r" % (gm,))
        dw_ref = torch.nn.grad.conv2d_weight(tx, cv.w_shape, tdy, **kw).numpy()
        _close(cv.wgrad(x, dy), dw_ref, what="wgrad %r" % (gm,))


def pin_scipy_correlate(lib):
    """Single-channel, stride-1 forward = scipy.signal.correlate2d on the
    zero-padded image ('valid' mode): cross-correlation, no kernel flip."""
    from scipy.signal import correlate2d
    rng = np.random.default_rng(7)
    for (h, w, r, s, ph, pw) in [(5, 7, 3, 2, 0, 0), (6, 4, 3, 3, 1, 1), (4, 4, 2, 3, 2, 1)]:
        x = rng.standard_normal((1, 1, h, w))
        wt = rng.standard_normal((1, 1, r, s))
        cv = orc.Conv(1, 1, h, w, 1, r, s, (1, 1), (ph, pw), (1, 1), 1, lib=lib)
        xp = np.pad(x[0, 0], ((ph, ph), (pw, pw)))
        ref = correlate2d(xp, wt[0, 0], mode="valid")
        _close(cv.fwd(x, wt)[0, 0], ref, what="correlate2d")


def pin_depthwise_correlate(lib):
    """Depthwise (groups = C = K): every output channel is the single-channel
    cross-correlation of its own input channel with its own filter
    (scipy.signal.correlate2d on the zero-padded image), subsampled by the
    stride; dgrad and wgrad follow from the adjoint identities per channel."""
    from scipy.signal import correlate2d
    rng = np.random.default_rng(17)
    for (n, c, h, w, r, st, pd) in [(2, 3, 7, 6, 3, 1, 1), (1, 4, 9, 8, 5, 2, 2),
                                    (2, 2, 6, 7, 3, 2, 0)]:
        x = rng.standard_normal((n, c, h, w))
        wt = rng.standard_normal((c, 1, r, r))
        cv = orc.Conv(n, c, h, w, c, r, r, (st, st), (pd, pd), (1, 1), c, lib=lib)
        y = cv.fwd(x, wt)
        ref = np.empty_like(y)
        for b in range(n):
            for ch in range(c):
                xp = np.pad(x[b, ch], ((pd, pd), (pd, pd)))
                ref[b, ch] = correlate2d(xp, wt[ch, 0], mode="valid")[::st, ::st]
        _close(y, ref, what="depthwise correlate2d")
        dy = rng.standard_normal(y.shape)
        dx = cv.dgrad(dy, wt)
        dw = cv.wgrad(x, dy)
        for ch in range(c):
            one = orc.Conv(n, 1, h, w, 1, r, r, (st, st), (pd, pd), (1, 1), 1, lib=lib)
            _close(dx[:, ch:ch + 1], one.dgrad(dy[:, ch:ch + 1], wt[ch:ch + 1]),
                   what="depthwise dgrad per channel")
            _close(dw[ch:ch + 1], one.wgrad(x[:, ch:ch + 1], dy[:, ch:ch + 1]),
                   what="depthwise wgrad per channel")


def pin_matmul_1x1(lib):
    """1x1 kernel, stride 1, no padding: Y = W X per pixel, DX = W^T DY,
    DW = sum over pixels of DY X^T (numpy matmul)."""
    rng = np.random.default_rng(11)
    n, c, h, w, k = 2, 5, 3, 4, 6
    cv = orc.Conv(n, c, h, w, k, 1, 1, lib=lib)
    x, wt, dy = _rand(rng, cv.x_shape), _rand(rng, cv.w_shape), _rand(rng, cv.y_shape)
    W = wt[:, :, 0, 0]
    X = x.transpose(1, 0, 2, 3).reshape(c, -1)
    DY = dy.transpose(1, 0, 2, 3).reshape(k, -1)
    y_ref = (W @ X).reshape(k, n, h, w).transpose(1, 0, 2, 3)
    dx_ref = (W.T @ DY).reshape(c, n, h, w).transpose(1, 0, 2, 3)
    dw_ref = (DY @ X.T).reshape(k, c, 1, 1)
    _close(cv.fwd(x, wt), y_ref, what="1x1 fwd")
    _close(cv.dgrad(dy, wt), dx_ref, what="1x1 dgrad")
    _close(cv.wgrad(x, dy), dw_ref, what="1x1 wgrad")


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------

def pin_delta_kernel(lib):
    """W[k,c,r,s] = [k==c][r==r0][s==s0]: the forward is an exact shifted,
    strided, dilated copy y[n,c,p,q] = x[n,c,p*sh-ph+r0*dh, q*sw-pw+s0*dw]
    (zero outside), and backward-data scatters dy back to those positions."""
    rng = np.random.default_rng(3)
    for (h, w, r, s, st, pd, dl) in [(6, 7, 3, 3, (1, 1), (1, 1), (1, 1)),
                                     (7, 5, 3, 2, (2, 1), (1, 0), (1, 2)),
                                     (8, 8, 2, 3, (3, 2), (2, 1), (2, 1))]:
        c = 3
        cv = orc.Conv(2, c, h, w, c, r, s, st, pd, dl, 1, lib=lib)
        x = rng.standard_normal(cv.x_shape)
        dy = rng.standard_normal(cv.y_shape)
        for r0, s0 in itertools.product(range(r), range(s)):
            wt = np.zeros(cv.w_shape)
            for ch in range(c):
                wt[ch, ch, r0, s0] = 1.0
            y = cv.fwd(x, wt)
            dx = cv.dgrad(dy, wt)
            y_ref = np.zeros(cv.y_shape)
            dx_ref = np.zeros(cv.x_shape)
            for p in range(cv.p):
                for q in range(cv.q):
                    i = p * st[0] - pd[0] + r0 * dl[0]
                    j = q * st[1] - pd[1] + s0 * dl[1]
                    if 0 <= i < h and 0 <= j < w:
                        y_ref[:, :, p, q] = x[:, :, i, j]
                        dx_ref[:, :, i, j] += dy[:, :, p, q]
            assert np.array_equal(y, y_ref), "delta fwd not an exact copy"
            assert np.array_equal(dx, dx_ref), "delta dgrad not an exact scatter"


def _count_valid(size, out, stride, pad, dil, taps):
    """Per-axis table t[o][r] = 1 when tap r of output o lands inside the image."""
    t = np.zeros((out, taps), np.int64)
    for o in range(out):
        for r in range(taps):
            i = o * stride - pad + r * dil
            t[o, r] = 1 if 0 <= i < size else 0
    return t


def pin_ones_closed_form(lib):
    """All-ones operands: each output is a product of per-axis tap counts.
    fwd  y[n,k,p,q]   = Cg * #r(p) * #s(q)
    dgrad dx[n,c,i,j] = Kg * #(r,p hitting i) * #(s,q hitting j)
    wgrad dw[k,c,r,s] = N * #p(r) * #q(s)"""
    for gm in _geoms():
        cv = _conv(lib, gm)
        (sh, sw), (ph, pw), (dh, dw) = gm["stride"], gm["pad"], gm["dil"]
        th = _count_valid(cv.h, cv.p, sh, ph, dh, cv.r)
        tw = _count_valid(cv.w, cv.q, sw, pw, dw, cv.s)
        cg, kg = cv.c // gm["groups"], cv.k // gm["groups"]
        y = cv.fwd(np.ones(cv.x_shape), np.ones(cv.w_shape))
        y_ref = cg * np.outer(th.sum(1), tw.sum(1))
        assert np.array_equal(y, np.broadcast_to(y_ref, y.shape)), "ones fwd %r" % (gm,)
        dx = cv.dgrad(np.ones(cv.y_shape), np.ones(cv.w_shape))
        hit_h = np.zeros(cv.h)
        for p in range(cv.p):
            for r in range(cv.r):
                i = p * sh - ph + r * dh
                if 0 <= i < cv.h:
                    hit_h[i] += 1
        hit_w = np.zeros(cv.w)
        for q in range(cv.q):
            for s in range(cv.s):
                j = q * sw - pw + s * dw
                if 0 <= j < cv.w:
                    hit_w[j] += 1
        dx_ref = kg * np.outer(hit_h, hit_w)
        assert np.array_equal(dx, np.broadcast_to(dx_ref, dx.shape)), "ones dgrad %r" % (gm,)
        dwt = cv.wgrad(np.ones(cv.x_shape), np.ones(cv.y_shape))
        dw_ref = cv.n * np.outer(th.sum(0), tw.sum(0))
        assert np.array_equal(dwt, np.broadcast_to(dw_ref, dwt.shape)), "ones wgrad %r" % (gm,)


def pin_output_dims(lib):
    """P equals the number of window positions p >= 0 whose last tap
    p*stride - pad + (R-1)*dil still lies inside the padded image."""
    for h in range(1, 9):
        for r in range(1, 4):
            for st in range(1, 4):
                for pd in range(0, 3):
                    for dl in range(1, 3):
                        count = 0
                        while count * st - pd + (r - 1) * dl <= h - 1 + pd:
                            count += 1
                        try:
                            cv = orc.Conv(1, 1, h, 3, 1, r, 1, (st, 1), (pd, 0), (dl, 1), 1, lib=lib)
                            got = cv.p
                        except ValueError:
                            got = 0
                        assert got == count, ("P", h, r, st, pd, dl, got, count)


HANDWORKED_X = np.array([[1., 2., 3.], [4., 5., 6.], [7., 8., 9.]])


def pin_handworked(lib):
    """Small examples worked out by hand from the definition."""
    x = HANDWORKED_X.reshape(1, 1, 3, 3)
    # 2x2 kernel [[1,2],[0,0]], stride 1, no pad:
    #   y00 = 1*1+2*2 = 5, y01 = 1*2+2*3 = 8, y10 = 1*4+2*5 = 14, y11 = 1*5+2*6 = 17
    cv = orc.Conv(1, 1, 3, 3, 1, 2, 2, lib=lib)
    w = np.array([[1., 2.], [0., 0.]]).reshape(1, 1, 2, 2)
    assert np.array_equal(cv.fwd(x, w)[0, 0], [[5, 8], [14, 17]])
    # kernel [[1,2],[3,4]], stride 2, pad 1 -> P = Q = 2; window origin (2p-1, 2q-1):
    #   y00 = 4*x00 = 4
    #   y01 = 3*x01 + 4*x02 = 6 + 12 = 18
    #   y10 = 2*x10 + 4*x20 = 8 + 28 = 36
    #   y11 = 1*x11 + 2*x12 + 3*x21 + 4*x22 = 5 + 12 + 24 + 36 = 77
    cv = orc.Conv(1, 1, 3, 3, 1, 2, 2, (2, 2), (1, 1), lib=lib)
    w = np.array([[1., 2.], [3., 4.]]).reshape(1, 1, 2, 2)
    assert np.array_equal(cv.fwd(x, w)[0, 0], [[4, 18], [36, 77]])
    # backward-data of that layer with dy = e11: the kernel lands on x[1:3,1:3]
    dy = np.array([[0., 0.], [0., 1.]]).reshape(1, 1, 2, 2)
    assert np.array_equal(cv.dgrad(dy, w)[0, 0], [[0, 0, 0], [0, 1, 2], [0, 3, 4]])
    # ... with dy = e00: only tap (1,1) of output (0,0) is inside -> dx00 = 4
    dy = np.array([[1., 0.], [0., 0.]]).reshape(1, 1, 2, 2)
    assert np.array_equal(cv.dgrad(dy, w)[0, 0], [[4, 0, 0], [0, 0, 0], [0, 0, 0]])
    # backward-weight: dy = e11 -> dw = x[1:3,1:3]; dy = e00 -> dw = [[0,0],[0,x00]]
    dy = np.array([[0., 0.], [0., 1.]]).reshape(1, 1, 2, 2)
    assert np.array_equal(cv.wgrad(x, dy)[0, 0], [[5, 6], [8, 9]])
    dy = np.array([[1., 0.], [0., 0.]]).reshape(1, 1, 2, 2)
    assert np.array_equal(cv.wgrad(x, dy)[0, 0], [[0, 0], [0, 1]])
    # dilation 2: kernel [[1,2],[3,4]] reads x00, x02, x20, x22 -> 1 + 6 + 21 + 36 = 64
    cv = orc.Conv(1, 1, 3, 3, 1, 2, 2, (1, 1), (0, 0), (2, 2), lib=lib)
    assert np.array_equal(cv.fwd(x, w)[0, 0], [[64]])
    # two groups, 1x1: out0 = 2*in0, out1 = 3*in1
    x2 = np.array([[[1., 2.], [3., 4.]], [[5., 6.], [7., 8.]]]).reshape(1, 2, 2, 2)
    cv = orc.Conv(1, 2, 2, 2, 2, 1, 1, groups=2, lib=lib)
    w2 = np.array([2., 3.]).reshape(2, 1, 1, 1)
    assert np.array_equal(cv.fwd(x2, w2)[0], [[[2, 4], [6, 8]], [[15, 18], [21, 24]]])
    # one group, two input channels, weights (1, -1): out = in0 - in1 = -4 everywhere
    cv = orc.Conv(1, 2, 2, 2, 1, 1, 1, lib=lib)
    w3 = np.array([1., -1.]).reshape(1, 2, 1, 1)
    assert np.array_equal(cv.fwd(x2, w3)[0, 0], [[-4, -4], [-4, -4]])


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def pin_adjoint(lib):
    """<fwd(x,w), dy> = <x, dgrad(dy,w)> = <w, wgrad(x,dy)>: all three are the
    sum of x*w*dy over the same index tuples."""
    for i, gm in enumerate(_geoms()):
        cv = _conv(lib, gm)
        x, w, dy = _operands(cv, 200 + i)
        a = float(np.sum(cv.fwd(x, w) * dy))
        b = float(np.sum(x * cv.dgrad(dy, w)))
        c = float(np.sum(w * cv.wgrad(x, dy)))
        scale = float(np.sum(np.abs(cv.fwd(np.abs(x), np.abs(w)) * np.abs(dy)))) + 1.0
        assert abs(a - b) <= 1e-12 * scale, ("adjoint x", gm, a, b)
        assert abs(a - c) <= 1e-12 * scale, ("adjoint w", gm, a, c)


def pin_gather_scatter(lib):
    """Gather-form dgrad (index inversion) equals scatter-form dgrad (replay
    of the forward index tuples)."""
    for i, gm in enumerate(_geoms()):
        cv = _conv(lib, gm)
        _, w, dy = _operands(cv, 300 + i)
        _close(cv.dgrad(dy, w), cv.dgrad_scatter(dy, w), what="gather/scatter %r" % (gm,))


def pin_groups_concat(lib):
    """A g-group convolution equals g independent convolutions on channel
    slices, concatenated."""
    rng = np.random.default_rng(5)
    n, c, h, w, k, r, s, g = 2, 6, 5, 6, 4, 3, 2, 2
    cv = orc.Conv(n, c, h, w, k, r, s, (1, 2), (1, 1), (1, 1), g, lib=lib)
    x, wt, dy = _rand(rng, cv.x_shape), _rand(rng, cv.w_shape), _rand(rng, cv.y_shape)
    one = orc.Conv(n, c // g, h, w, k // g, r, s, (1, 2), (1, 1), (1, 1), 1, lib=lib)
    cs, ks = c // g, k // g
    y = cv.fwd(x, wt)
    dx = cv.dgrad(dy, wt)
    dw = cv.wgrad(x, dy)
    for j in range(g):
        xs, ws, dys = x[:, j * cs:(j + 1) * cs], wt[j * ks:(j + 1) * ks], dy[:, j * ks:(j + 1) * ks]
        _close(y[:, j * ks:(j + 1) * ks], one.fwd(xs, ws), what="groups fwd")
        _close(dx[:, j * cs:(j + 1) * cs], one.dgrad(dys, ws), what="groups dgrad")
        _close(dw[j * ks:(j + 1) * ks], one.wgrad(xs, dys), what="groups wgrad")


def pin_dilation_zero_insert(lib):
    """Dilation d equals a plain convolution with the kernel spread out by
    d-1 zeros between taps (kernel size d*(R-1)+1)."""
    rng = np.random.default_rng(9)
    n, c, h, w, k, r, s = 1, 2, 9, 8, 3, 3, 2
    dl = (2, 3)
    cv = orc.Conv(n, c, h, w, k, r, s, (1, 1), (2, 1), dl, 1, lib=lib)
    x, wt, dy = _rand(rng, cv.x_shape), _rand(rng, cv.w_shape), _rand(rng, cv.y_shape)
    re, se = dl[0] * (r - 1) + 1, dl[1] * (s - 1) + 1
    wz = np.zeros((k, c, re, se))
    wz[:, :, ::dl[0], ::dl[1]] = wt
    big = orc.Conv(n, c, h, w, k, re, se, (1, 1), (2, 1), (1, 1), 1, lib=lib)
    _close(cv.fwd(x, wt), big.fwd(x, wz), what="dilation fwd")
    _close(cv.dgrad(dy, wt), big.dgrad(dy, wz), what="dilation dgrad")
    _close(cv.wgrad(x, dy), big.wgrad(x, dy)[:, :, ::dl[0], ::dl[1]], what="dilation wgrad")


def pin_stride_subsample(lib):
    """Stride s equals the stride-1 output sampled at multiples of s."""
    rng = np.random.default_rng(13)
    n, c, h, w, k, r, s = 2, 3, 9, 8, 2, 3, 3
    st = (2, 3)
    cv = orc.Conv(n, c, h, w, k, r, s, st, (1, 1), (1, 1), 1, lib=lib)
    x, wt = _rand(rng, cv.x_shape), _rand(rng, cv.w_shape)
    one = orc.Conv(n, c, h, w, k, r, s, (1, 1), (1, 1), (1, 1), 1, lib=lib)
    _close(cv.fwd(x, wt), one.fwd(x, wt)[:, :, ::st[0], ::st[1]][:, :, :cv.p, :cv.q],
           what="stride subsample")


def pin_linearity(lib):
    """Each pass is linear in each operand."""
    gm = dict(n=2, c=4, h=6, w=5, k=4, r=3, s=2, stride=(2, 1), pad=(1, 1), dil=(1, 1), groups=2)
    cv = _conv(lib, gm)
    x, w, dy = _operands(cv, 17)
    x2, w2, dy2 = _operands(cv, 18)
    _close(cv.fwd(2 * x + x2, w), 2 * cv.fwd(x, w) + cv.fwd(x2, w), what="lin fwd")
    _close(cv.dgrad(dy, 3 * w - w2), 3 * cv.dgrad(dy, w) - cv.dgrad(dy, w2), what="lin dgrad")
    _close(cv.wgrad(x, dy + dy2), cv.wgrad(x, dy) + cv.wgrad(x, dy2), what="lin wgrad")


def pin_loss_scale(lib):
    """Loss scaling (Listing 6): dy arrives multiplied by S and the weight
    gradient is multiplied by 1/S.  For a power of two S both steps are exact
    in binary floating point, so wgrad(x, S*dy, 1/S) == wgrad(x, dy, 1)
    bitwise.  Accumulation adds the old gradient: beta=1 gives old + new."""
    gm = dict(n=2, c=3, h=5, w=6, k=2, r=3, s=3, stride=(1, 1), pad=(1, 1), dil=(1, 1), groups=1)
    cv = _conv(lib, gm)
    x, _, dy = _operands(cv, 19)
    for S in (8.0, 1024.0, 65536.0):
        assert np.array_equal(cv.wgrad(x, S * dy, 1.0 / S), cv.wgrad(x, dy, 1.0)), S
    old = np.random.default_rng(20).standard_normal(cv.w_shape)
    acc = cv.wgrad(x, dy, 0.5, beta=1, dw_old=old)
    _close(acc, old + 0.5 * cv.wgrad(x, dy, 1.0), what="beta accumulate")
    # beta = 0 ignores whatever the output held (NaN included)
    assert np.all(np.isfinite(cv.wgrad(x, dy, 1.0, beta=0)))


def pin_nonfinite(lib):
    """check_inf_or_nan_grad: any inf or NaN sets the flag."""
    a = np.zeros(100)
    assert not orc.any_nonfinite(a, lib=lib)
    for bad in (np.inf, -np.inf, np.nan):
        b = a.copy()
        b[57] = bad
        assert orc.any_nonfinite(b, lib=lib)


def pin_points(lib):
    """The sampled routines evaluate the same expression as the full ones."""
    for i, gm in enumerate(list(_geoms())[:6]):
        cv = _conv(lib, gm)
        x, w, dy = _operands(cv, 400 + i)
        y = cv.fwd(x, w, alpha=0.5)
        idx = np.arange(y.size)
        assert np.array_equal(cv.fwd_points(x, w, idx, alpha=0.5), y.ravel())
        dx = cv.dgrad(dy, w)
        assert np.array_equal(cv.dgrad_points(dy, w, np.arange(dx.size)), dx.ravel())
        dw = cv.wgrad(x, dy, 1.0)
        assert np.array_equal(cv.wgrad_points(x, dy, np.arange(dw.size)), dw.ravel())


ALL_PINS = [pin_torch, pin_scipy_correlate, pin_depthwise_correlate, pin_matmul_1x1,
            pin_delta_kernel, pin_ones_closed_form, pin_output_dims, pin_handworked, pin_adjoint,
            pin_gather_scatter, pin_groups_concat, pin_dilation_zero_insert,
            pin_stride_subsample, pin_linearity, pin_loss_scale, pin_nonfinite,
            pin_points]
