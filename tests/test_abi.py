"""C-ABI of libnnconv on the host: exported symbols, argument validation and
shape arithmetic.  Every call here fails validation (or only computes sizes)
before anything is queued, so no GPU is needed and no kernel runs."""
import ctypes
import os
import re

import pytest

from paper_2102_06725_amd import nnconv as nc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x100000  # never dereferenced: every call below fails validation first


def header_functions():
    text = open(os.path.join(ROOT, "include", "nnconv.h")).read()
    return sorted(set(re.findall(r"\b(nnconv_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_function_is_exported(nnlib):
    declared = header_functions()
    assert len(declared) >= 12
    for name in declared:
        assert hasattr(nnlib, name), name
    assert set(declared) == set(nc.EXPORTS)


def test_version_and_strings(nnlib):
    assert nc.nnconv_version() == 1
    for s in range(6):
        assert nc.status_string(s)


def good_desc(**kw):
    base = dict(n=2, c=16, h=16, w=16, k=16, r=3, s=3, stride=(1, 1), pad=(1, 1))
    base.update(kw)
    return nc.make_desc(**base)


@pytest.mark.parametrize("kw", [
    dict(n=0), dict(c=0), dict(h=-1), dict(k=0), dict(r=0),
    dict(stride=(0, 1)), dict(dil=(1, 0)), dict(pad=(-1, 0)),
    dict(groups=3), dict(groups=0), dict(c=16, k=12, groups=8),
    dict(h=2, w=2, r=5, s=5, pad=(0, 0)),        # empty output
    dict(layout=7), dict(dtype=9),
])
def test_invalid_descriptors(nnlib, kw):
    d = good_desc(**kw)
    st, _, _ = nc.nnconv_output_dims(d)
    assert st == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_fwd(d, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_dgrad(d, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_wgrad(d, FAKE, FAKE, FAKE, nc.NNCONV_F32, 1.0, 0, None, FAKE, 1 << 30,
                           None) == nc.NNCONV_ERR_INVALID_ARG


def test_fp32_operands_unsupported(nnlib):
    d = good_desc(dtype=nc.NNCONV_F32)
    assert nc.nnconv_fwd(d, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None) == nc.NNCONV_ERR_UNSUPPORTED


def test_null_and_misaligned_pointers(nnlib):
    d = good_desc(layout=nc.NNCONV_NHWC)
    assert nc.nnconv_fwd(d, None, FAKE, FAKE, 1.0, FAKE, 1 << 30, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_dgrad(d, FAKE, FAKE, None, 1.0, FAKE, 1 << 30, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_wgrad(d, FAKE, None, FAKE, nc.NNCONV_F32, 1.0, 0, None, FAKE, 1 << 30,
                           None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_fwd(d, FAKE + 1, FAKE, FAKE, 1.0, FAKE, 1 << 30, None) == nc.NNCONV_ERR_MISALIGNED
    assert nc.nnconv_wgrad(d, FAKE, FAKE, FAKE + 2, nc.NNCONV_F32, 1.0, 0, None, FAKE, 1 << 30,
                           None) == nc.NNCONV_ERR_MISALIGNED


def test_bad_wgrad_options(nnlib):
    d = good_desc(layout=nc.NNCONV_NHWC)
    assert nc.nnconv_wgrad(d, FAKE, FAKE, FAKE, nc.NNCONV_BF16, 1.0, 0, None, FAKE, 1 << 30,
                           None) == nc.NNCONV_ERR_UNSUPPORTED
    assert nc.nnconv_wgrad(d, FAKE, FAKE, FAKE, 5, 1.0, 0, None, FAKE, 1 << 30,
                           None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_wgrad(d, FAKE, FAKE, FAKE, nc.NNCONV_F32, 1.0, 2, None, FAKE, 1 << 30,
                           None) == nc.NNCONV_ERR_INVALID_ARG


@pytest.mark.parametrize("layout", [nc.NNCONV_NCHW, nc.NNCONV_NHWC])
def test_workspace_too_small(nnlib, layout):
    d = good_desc(layout=layout)
    for pass_, call in ((nc.NNCONV_FWD, lambda ws, nb: nc.nnconv_fwd(d, FAKE, FAKE, FAKE, 1.0, ws, nb, None)),
                        (nc.NNCONV_DGRAD, lambda ws, nb: nc.nnconv_dgrad(d, FAKE, FAKE, FAKE, 1.0, ws, nb, None)),
                        (nc.NNCONV_WGRAD, lambda ws, nb: nc.nnconv_wgrad(d, FAKE, FAKE, FAKE, nc.NNCONV_F32,
                                                                         1.0, 0, None, ws, nb, None))):
        st, need = nc.nnconv_workspace_size(d, pass_)
        assert st == nc.NNCONV_OK
        if need == 0:
            continue
        assert call(FAKE, need - 1) == nc.NNCONV_ERR_WORKSPACE
        assert call(None, need) == nc.NNCONV_ERR_INVALID_ARG


def test_workspace_sizes_are_deterministic_and_cover_partials(nnlib):
    d = good_desc(n=64, c=64, h=56, w=56, k=64, layout=nc.NNCONV_NHWC)
    st, f = nc.nnconv_workspace_size(d, nc.NNCONV_FWD)
    # channel-last forward: only the weights packed in fragment order for the
    # register-weight halo tiles (9 taps x 1 slice x 2 column blocks x 4 KB)
    assert st == 0 and f == 9 * 1 * 2 * 4096
    one = good_desc(n=64, c=64, h=56, w=56, k=64, r=1, s=1, pad=(0, 0), layout=nc.NNCONV_NHWC)
    assert nc.nnconv_workspace_size(one, nc.NNCONV_FWD) == (0, 0)   # 1x1: no scratch
    st, w1 = nc.nnconv_workspace_size(d, nc.NNCONV_WGRAD)
    st, w2 = nc.nnconv_workspace_size(d, nc.NNCONV_WGRAD)
    assert w1 == w2 and w1 >= 64 * 9 * 64 * 4    # at least one fp32 partial of dw
    st, dg = nc.nnconv_workspace_size(d, nc.NNCONV_DGRAD)
    assert dg >= 64 * 9 * 64 * 2                 # transposed weights
    assert nc.nnconv_workspace_size(d, 7)[0] == nc.NNCONV_ERR_INVALID_ARG


def test_output_dims_match_oracle(nnlib, oracle_lib):
    import oracle.oracle as orc
    for h in range(1, 12):
        for r in (1, 2, 3, 5, 7):
            for st in (1, 2, 3):
                for pd in (0, 1, 3):
                    for dl in (1, 2):
                        d = nc.make_desc(1, 8, h, h + 1, 8, r, r, (st, st), (pd, pd), (dl, dl))
                        s, p, q = nc.nnconv_output_dims(d)
                        try:
                            cv = orc.Conv(1, 8, h, h + 1, 8, r, r, (st, st), (pd, pd), (dl, dl), 1,
                                          lib=oracle_lib)
                        except ValueError:
                            assert s == nc.NNCONV_ERR_INVALID_ARG
                            continue
                        assert s == 0 and (p, q) == (cv.p, cv.q)


def test_transform_validation(nnlib):
    assert nc.nnconv_nchw_to_nhwc(FAKE, FAKE, 1, 3, 4, 4, 2, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_nchw_to_nhwc(None, FAKE, 1, 3, 4, 4, 8, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_pad_channels(FAKE + 1, FAKE, 10, 3, 8, None) == nc.NNCONV_ERR_MISALIGNED
    assert nc.nnconv_weight_kcrs_to_krsc(FAKE, FAKE, 4, 3, 3, 3, 2, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_weight_krsc_to_kcrs(FAKE, FAKE, 0, 3, 3, 3, None) == nc.NNCONV_ERR_INVALID_ARG
    assert nc.nnconv_nhwc_to_nchw(FAKE, None, 1, 3, 4, 4, None) == nc.NNCONV_ERR_INVALID_ARG


def test_loss_scaler_state_layout():
    assert ctypes.sizeof(nc.nnconv_loss_scaler) == 24
    assert [f for f, _ in nc.nnconv_loss_scaler._fields_] == [
        "scale", "factor", "interval", "counter", "skipped", "reserved"]


def test_loss_scaler_validation(nnlib):
    inv, mis = nc.NNCONV_ERR_INVALID_ARG, nc.NNCONV_ERR_MISALIGNED
    assert nc.nnconv_loss_scaler_init(None, 1024.0, 2.0, 2000, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE, 0.0, 2.0, 2000, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE, -1.0, 2.0, 2000, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE, float("inf"), 2.0, 2000, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE, float("nan"), 2.0, 2000, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE, 1024.0, 0.0, 2000, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE, 1024.0, 2.0, -1, None) == inv
    assert nc.nnconv_loss_scaler_init(FAKE + 2, 1024.0, 2.0, 2000, None) == mis
    assert nc.nnconv_loss_scaler_update(None, FAKE, None) == inv
    assert nc.nnconv_loss_scaler_update(FAKE, None, None) == inv
    assert nc.nnconv_loss_scaler_update(FAKE, FAKE + 1, None) == mis


def test_sgd_update_validation(nnlib):
    inv, mis = nc.NNCONV_ERR_INVALID_ARG, nc.NNCONV_ERR_MISALIGNED

    def call(count=16, master=FAKE, mom=FAKE, w16=FAKE, w16_dtype=nc.NNCONV_F16, grad=FAKE,
             state=FAKE, flag=FAKE):
        return nc.nnconv_sgd_update(count, master, mom, w16, w16_dtype, grad, state, flag,
                                    0.1, 0.9, 1e-4, None)

    assert call(count=-1) == inv
    assert call(master=None) == inv and call(mom=None) == inv and call(grad=None) == inv
    assert call(w16_dtype=nc.NNCONV_F32) == inv
    assert call(master=FAKE + 2) == mis and call(mom=FAKE + 2) == mis
    assert call(grad=FAKE + 1) == mis and call(w16=FAKE + 1) == mis
    assert call(state=FAKE + 2) == mis and call(flag=FAKE + 2) == mis
    # count 0 is a no-op that touches nothing, w16 NULL ignores w16_dtype
    assert call(count=0) == nc.NNCONV_OK
    assert call(count=0, w16=None, w16_dtype=7, state=None, flag=None) == nc.NNCONV_OK


def test_forced_tile_validation(nnlib):
    """The _tile variants refuse, before anything is queued, a negative tile,
    a value that is not a dense implicit-GEMM tile, and calls that would not
    run on that kernel."""
    inv, uns = nc.NNCONV_ERR_INVALID_ARG, nc.NNCONV_ERR_UNSUPPORTED
    dense = nc.make_desc(2, 64, 8, 8, 64, 3, 3, pad=(1, 1))
    calls = (nc.nnconv_fwd_tile, nc.nnconv_dgrad_tile)
    for f in calls:
        assert f(dense, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, -1) == inv
        for bad in (5, 16, 99):  # block-diagonal tile, out of range
            assert f(dense, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, bad) == uns
        # 16 reduction channels per tap: not the 64-channel-slice kernel
        small = nc.make_desc(2, 16, 8, 8, 16, 3, 3, pad=(1, 1))
        assert f(small, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, 2) == uns
        # depthwise and small groups have kernels of their own
        dwc = nc.make_desc(2, 64, 8, 8, 64, 3, 3, pad=(1, 1), groups=64)
        assert f(dwc, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, 2) == uns
        grp = nc.make_desc(2, 64, 8, 8, 64, 3, 3, pad=(1, 1), groups=16)
        assert f(grp, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, 2) == uns
        # operands off 16-byte alignment take the direct kernels
        assert f(dense, FAKE + 2, FAKE + 2, FAKE + 2, 1.0, FAKE, 1 << 30, None, 2) == uns
        # still the ordinary checks first
        assert f(dense, None, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, 2) == inv
    # the stem's 8-channel shape has its own forward kernel (as has the 4-channel one)
    stem = nc.make_desc(2, 8, 32, 32, 64, 7, 7, stride=(2, 2), pad=(3, 3))
    assert nc.nnconv_fwd_tile(stem, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, 2) == uns
    # backward-data with more than four stride phases
    s3 = nc.make_desc(2, 64, 9, 9, 64, 3, 3, stride=(3, 3), pad=(1, 1))
    assert nc.nnconv_dgrad_tile(s3, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, 2) == uns
    # halo tiles: stride 1 with the output the input's size, 3x3 on images up
    # to 63 pixels wide (taps spanning at most 128 raster positions)
    halo = nc.HALO_TILES
    not_same = (nc.make_desc(2, 64, 8, 8, 64, 3, 3, stride=(2, 2), pad=(1, 1)),
                nc.make_desc(2, 64, 8, 8, 64, 3, 3, pad=(0, 0)),
                nc.make_desc(2, 64, 8, 64, 64, 3, 3, pad=(1, 1)),
                nc.make_desc(2, 64, 8, 8, 64, 3, 3, pad=(1, 1), groups=2),
                nc.make_desc(2, 64, 8, 8, 32, 3, 3, pad=(1, 1)))
    for f in calls:
        for d in not_same:
            for t in halo:
                assert f(d, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, t) == uns
        # the 320-row halo tile holds taps within 64 raster positions: a 3x3
        # filter on a 32-pixel-wide image (span 66) is refused by it only
        wide = nc.make_desc(2, 64, 8, 32, 64, 3, 3, pad=(1, 1))
        assert f(wide, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None,
                 nc.NNCONV_TILE_HALO_R256x128) == uns
    # the single-slice tile takes a reduction of 64 channels: C forward, K
    # backward-data
    c128 = nc.make_desc(2, 128, 8, 8, 64, 3, 3, pad=(1, 1))
    k128 = nc.make_desc(2, 64, 8, 8, 128, 3, 3, pad=(1, 1))
    single = nc.NNCONV_TILE_HALO_R256x64S
    assert nc.nnconv_fwd_tile(c128, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, single) == uns
    assert nc.nnconv_dgrad_tile(k128, FAKE, FAKE, FAKE, 1.0, FAKE, 1 << 30, None, single) == uns


def test_noalloc_wgrad_validation(nnlib):
    """nnconv_wgrad_noalloc refuses, before anything is queued, what
    nnconv_wgrad refuses, and geometries whose workspace exceeds its scratch."""
    inv, mis = nc.NNCONV_ERR_INVALID_ARG, nc.NNCONV_ERR_MISALIGNED
    d = good_desc()
    call = nc.nnconv_wgrad_noalloc
    assert call(d, None, FAKE, FAKE, nc.NNCONV_F32, 1.0, 0, None, None) == inv
    assert call(d, FAKE, FAKE, FAKE, 5, 1.0, 0, None, None) == inv
    assert call(d, FAKE, FAKE, FAKE, nc.NNCONV_F32, 1.0, 2, None, None) == inv
    assert call(d, FAKE, FAKE, FAKE + 2, nc.NNCONV_F32, 1.0, 0, None, None) == mis
    assert call(d, FAKE, FAKE, FAKE, nc.NNCONV_F32, 1.0, 0, FAKE + 1, None) == mis
    assert call(d, FAKE, FAKE, FAKE, nc.NNCONV_BF16, 1.0, 0, None, None) == nc.NNCONV_ERR_UNSUPPORTED
    assert call(good_desc(n=0), FAKE, FAKE, FAKE, nc.NNCONV_F32, 1.0, 0, None, None) == inv
    # NCHW copies of a 56x56x256 batch-64 activation exceed the 64 MiB scratch
    big = nc.make_desc(64, 256, 56, 56, 64, 1, 1, layout=nc.NNCONV_NCHW)
    st, need = nc.nnconv_workspace_size(big, nc.NNCONV_WGRAD)
    assert st == nc.NNCONV_OK and need > nc.NNCONV_NOALLOC_WS_BYTES
    assert call(big, FAKE, FAKE, FAKE, nc.NNCONV_F32, 1.0, 0, None, None) == \
        nc.NNCONV_ERR_WORKSPACE
