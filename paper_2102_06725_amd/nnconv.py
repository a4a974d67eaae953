"""ctypes binding of libnnconv (include/nnconv.h).

The functions below carry the C names and only marshal arguments: device
pointers are Python ints (``tensor.data_ptr()``), streams are ints
(``torch.cuda.current_stream().cuda_stream``).  Every computation runs in
the HIP library; if it is missing, loading fails loudly.

``Conv2d`` is a small convenience on top: it takes torch tensors, sizes and
allocates the caller-owned workspace with torch, and raises on a non-OK
status.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libnnconv.so")

# enums (same values as nnconv.h)
NNCONV_OK = 0
NNCONV_ERR_INVALID_ARG = 1
NNCONV_ERR_UNSUPPORTED = 2
NNCONV_ERR_WORKSPACE = 3
NNCONV_ERR_MISALIGNED = 4
NNCONV_ERR_HIP = 5
NNCONV_NCHW = 0
NNCONV_NHWC = 1
NNCONV_F16 = 0
NNCONV_BF16 = 1
NNCONV_F32 = 2
NNCONV_FWD = 0
NNCONV_DGRAD = 1
NNCONV_WGRAD = 2
NNCONV_NOALLOC_WS_BYTES = 64 * 1024 * 1024
# nnconv_tile: tiles of the implicit-GEMM forward / backward-data kernel
NNCONV_TILE_256x256_8W = 0
NNCONV_TILE_128x128_2S = 1
NNCONV_TILE_128x128 = 2
NNCONV_TILE_128x64 = 3
NNCONV_TILE_256x256_16W = 4
NNCONV_TILE_256x256_RING = 6
NNCONV_TILE_256x128_RING = 7
NNCONV_TILE_256x64_RING = 8
NNCONV_TILE_HALO_256x64 = 9
NNCONV_TILE_HALO_256x128 = 10
NNCONV_TILE_HALO_256x64_2T = 11
NNCONV_TILE_HALO_R256x128 = 12
NNCONV_TILE_HALO_R128x256 = 13
NNCONV_TILE_HALO_R224x256 = 14
NNCONV_TILE_HALO_R256x64S = 15
HALO_TILES = (NNCONV_TILE_HALO_256x64, NNCONV_TILE_HALO_256x128, NNCONV_TILE_HALO_256x64_2T,
              NNCONV_TILE_HALO_R256x128, NNCONV_TILE_HALO_R128x256, NNCONV_TILE_HALO_R224x256,
              NNCONV_TILE_HALO_R256x64S)
# largest raster span of the filter taps each halo tile's buffer holds
HALO_TILE_SPAN = {NNCONV_TILE_HALO_256x64: 128, NNCONV_TILE_HALO_256x128: 128,
                  NNCONV_TILE_HALO_256x64_2T: 128, NNCONV_TILE_HALO_R256x128: 64,
                  NNCONV_TILE_HALO_R128x256: 128, NNCONV_TILE_HALO_R224x256: 32,
                  NNCONV_TILE_HALO_R256x64S: 128}
# filter taps the halo tiles with register-held weights take (3x3 only)
HALO_TILE_TAPS = {NNCONV_TILE_HALO_R256x128: 9, NNCONV_TILE_HALO_R128x256: 9,
                  NNCONV_TILE_HALO_R224x256: 9, NNCONV_TILE_HALO_R256x64S: 9}
# the pass's reduction channel count the single-slice halo tile requires
HALO_TILE_RED = {NNCONV_TILE_HALO_R256x64S: 64}
TILES = (NNCONV_TILE_256x256_8W, NNCONV_TILE_128x128_2S, NNCONV_TILE_128x128, NNCONV_TILE_128x64,
         NNCONV_TILE_256x256_16W, NNCONV_TILE_256x256_RING, NNCONV_TILE_256x128_RING,
         NNCONV_TILE_256x64_RING)

EXPORTS = ("nnconv_version", "nnconv_last_hip_error", "nnconv_status_string", "nnconv_output_dims",
           "nnconv_workspace_size", "nnconv_fwd", "nnconv_dgrad", "nnconv_fwd_tile",
           "nnconv_dgrad_tile", "nnconv_wgrad", "nnconv_wgrad_noalloc",
           "nnconv_nchw_to_nhwc", "nnconv_nhwc_to_nchw", "nnconv_pad_channels",
           "nnconv_weight_kcrs_to_krsc", "nnconv_weight_krsc_to_kcrs",
           "nnconv_loss_scaler_init", "nnconv_loss_scaler_update", "nnconv_sgd_update")


class nnconv_desc(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in
                ("n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
                 "dil_h", "dil_w", "groups", "layout", "dtype")]


class nnconv_loss_scaler(ctypes.Structure):
    """Layout of the device-resident scaler state (24 bytes)."""
    _fields_ = [("scale", ctypes.c_float), ("factor", ctypes.c_float),
                ("interval", ctypes.c_int32), ("counter", ctypes.c_int32),
                ("skipped", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class NNConvError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        extra = ""
        if status == NNCONV_ERR_HIP:
            extra = ", hipError %d" % nnconv_last_hip_error()
        super().__init__("%s: %s (status %d%s)" % (what or "libnnconv", status_string(status),
                                                   status, extra))


_lib = None

_VP = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_DESCP = ctypes.POINTER(nnconv_desc)


def load(path: str | None = None):
    """Load libnnconv.so (built in-tree by paper_2102_06725_amd.build)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise ImportError("libnnconv.so not found at %s; build it with "
                          "`python -m paper_2102_06725_amd.build`" % p)
    # torch ships its own HIP runtime whose SONAME matches the one libnnconv
    # links against.  Loading torch first makes the library bind to that same
    # runtime instance, so torch's device pointers and streams are valid in
    # it; loading libnnconv first would put a second runtime in the process.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(p)
    lib.nnconv_version.restype = _I32
    lib.nnconv_last_hip_error.restype = _I32
    lib.nnconv_status_string.argtypes = [ctypes.c_int]
    lib.nnconv_status_string.restype = ctypes.c_char_p
    lib.nnconv_output_dims.argtypes = [_DESCP, ctypes.POINTER(_I32), ctypes.POINTER(_I32)]
    lib.nnconv_workspace_size.argtypes = [_DESCP, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
    lib.nnconv_fwd.argtypes = [_DESCP, _VP, _VP, _VP, ctypes.c_float, _VP, ctypes.c_size_t, _VP]
    lib.nnconv_dgrad.argtypes = [_DESCP, _VP, _VP, _VP, ctypes.c_float, _VP, ctypes.c_size_t, _VP]
    lib.nnconv_wgrad_noalloc.argtypes = [_DESCP, _VP, _VP, _VP, _I32, ctypes.c_float, _I32,
                                         _VP, _VP]
    lib.nnconv_fwd_tile.argtypes = [_DESCP, _VP, _VP, _VP, ctypes.c_float, _VP, ctypes.c_size_t,
                                    _VP, _I32]
    lib.nnconv_dgrad_tile.argtypes = [_DESCP, _VP, _VP, _VP, ctypes.c_float, _VP,
                                      ctypes.c_size_t, _VP, _I32]
    lib.nnconv_wgrad.argtypes = [_DESCP, _VP, _VP, _VP, _I32, ctypes.c_float, _I32, _VP, _VP,
                                 ctypes.c_size_t, _VP]
    lib.nnconv_nchw_to_nhwc.argtypes = [_VP, _VP, _I32, _I32, _I32, _I32, _I32, _VP]
    lib.nnconv_nhwc_to_nchw.argtypes = [_VP, _VP, _I32, _I32, _I32, _I32, _VP]
    lib.nnconv_pad_channels.argtypes = [_VP, _VP, _I64, _I32, _I32, _VP]
    lib.nnconv_weight_kcrs_to_krsc.argtypes = [_VP, _VP, _I32, _I32, _I32, _I32, _I32, _VP]
    lib.nnconv_weight_krsc_to_kcrs.argtypes = [_VP, _VP, _I32, _I32, _I32, _I32, _VP]
    lib.nnconv_loss_scaler_init.argtypes = [_VP, ctypes.c_float, ctypes.c_float, _I32, _VP]
    lib.nnconv_loss_scaler_update.argtypes = [_VP, _VP, _VP]
    lib.nnconv_sgd_update.argtypes = [_I64, _VP, _VP, _VP, _I32, _VP, _VP, _VP, ctypes.c_float,
                                      ctypes.c_float, ctypes.c_float, _VP]
    for f in EXPORTS[3:]:
        getattr(lib, f).restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def make_desc(n, c, h, w, k, r, s, stride=(1, 1), pad=(0, 0), dil=(1, 1), groups=1,
              layout=NNCONV_NHWC, dtype=NNCONV_F16) -> nnconv_desc:
    def pair(v):
        return (v, v) if isinstance(v, int) else tuple(v)
    st, pd, dl = pair(stride), pair(pad), pair(dil)
    return nnconv_desc(n, c, h, w, k, r, s, st[0], st[1], pd[0], pd[1], dl[0], dl[1], groups,
                       layout, dtype)


# --- C entry points, same names -------------------------------------------

def nnconv_version() -> int:
    return load().nnconv_version()


def nnconv_last_hip_error() -> int:
    return load().nnconv_last_hip_error()


def status_string(status: int) -> str:
    return load().nnconv_status_string(int(status)).decode()


nnconv_status_string = status_string


def nnconv_output_dims(desc: nnconv_desc):
    p, q = _I32(), _I32()
    st = load().nnconv_output_dims(ctypes.byref(desc), ctypes.byref(p), ctypes.byref(q))
    return st, p.value, q.value


def nnconv_workspace_size(desc: nnconv_desc, pass_: int):
    b = ctypes.c_size_t()
    st = load().nnconv_workspace_size(ctypes.byref(desc), int(pass_), ctypes.byref(b))
    return st, b.value


def nnconv_fwd(desc, x, w, y, alpha, ws, ws_bytes, stream) -> int:
    return load().nnconv_fwd(ctypes.byref(desc), x, w, y, float(alpha), ws, ws_bytes, stream)


def nnconv_dgrad(desc, dy, w, dx, alpha, ws, ws_bytes, stream) -> int:
    return load().nnconv_dgrad(ctypes.byref(desc), dy, w, dx, float(alpha), ws, ws_bytes, stream)


def nnconv_fwd_tile(desc, x, w, y, alpha, ws, ws_bytes, stream, tile) -> int:
    return load().nnconv_fwd_tile(ctypes.byref(desc), x, w, y, float(alpha), ws, ws_bytes, stream,
                                  int(tile))


def nnconv_dgrad_tile(desc, dy, w, dx, alpha, ws, ws_bytes, stream, tile) -> int:
    return load().nnconv_dgrad_tile(ctypes.byref(desc), dy, w, dx, float(alpha), ws, ws_bytes,
                                    stream, int(tile))


def nnconv_wgrad(desc, x, dy, dw, dw_dtype, inv_loss_scale, accumulate, overflow_flag, ws,
                 ws_bytes, stream) -> int:
    return load().nnconv_wgrad(ctypes.byref(desc), x, dy, dw, int(dw_dtype),
                               float(inv_loss_scale), int(accumulate), overflow_flag, ws,
                               ws_bytes, stream)


def nnconv_wgrad_noalloc(desc, x, dy, dw, dw_dtype, inv_loss_scale, accumulate, overflow_flag,
                         stream) -> int:
    return load().nnconv_wgrad_noalloc(ctypes.byref(desc), x, dy, dw, int(dw_dtype),
                                       float(inv_loss_scale), int(accumulate), overflow_flag,
                                       stream)


def nnconv_nchw_to_nhwc(src, dst, n, c, h, w, c_pad, stream) -> int:
    return load().nnconv_nchw_to_nhwc(src, dst, n, c, h, w, c_pad, stream)


def nnconv_nhwc_to_nchw(src, dst, n, c, h, w, stream) -> int:
    return load().nnconv_nhwc_to_nchw(src, dst, n, c, h, w, stream)


def nnconv_pad_channels(src, dst, rows, c, c_pad, stream) -> int:
    return load().nnconv_pad_channels(src, dst, rows, c, c_pad, stream)


def nnconv_weight_kcrs_to_krsc(src, dst, k, cg, r, s, cg_pad, stream) -> int:
    return load().nnconv_weight_kcrs_to_krsc(src, dst, k, cg, r, s, cg_pad, stream)


def nnconv_weight_krsc_to_kcrs(src, dst, k, cg, r, s, stream) -> int:
    return load().nnconv_weight_krsc_to_kcrs(src, dst, k, cg, r, s, stream)


def nnconv_loss_scaler_init(state, initial_scale, factor, interval, stream) -> int:
    return load().nnconv_loss_scaler_init(state, float(initial_scale), float(factor),
                                          int(interval), stream)


def nnconv_loss_scaler_update(state, overflow_flag, stream) -> int:
    return load().nnconv_loss_scaler_update(state, overflow_flag, stream)


def nnconv_sgd_update(count, master, momentum, w16, w16_dtype, grad, state, overflow_flag, lr,
                      momentum_coef, weight_decay, stream) -> int:
    return load().nnconv_sgd_update(int(count), master, momentum, w16, int(w16_dtype), grad,
                                    state, overflow_flag, float(lr), float(momentum_coef),
                                    float(weight_decay), stream)


def check(status: int, what: str = "") -> None:
    if status != NNCONV_OK:
        raise NNConvError(status, what)


# --- torch-tensor convenience ------------------------------------------------

class Conv2d:
    """One convolution geometry bound to torch tensors on the current device.

    The workspace for each pass is a torch uint8 tensor owned by this object
    (allocated once, on first use)."""

    def __init__(self, n, c, h, w, k, r, s, stride=(1, 1), pad=(0, 0), dil=(1, 1), groups=1,
                 layout=NNCONV_NHWC, dtype=NNCONV_F16):
        self.desc = make_desc(n, c, h, w, k, r, s, stride, pad, dil, groups, layout, dtype)
        st, self.p, self.q = nnconv_output_dims(self.desc)
        check(st, "nnconv_output_dims")
        self._ws = {}

    def workspace(self, pass_: int, device=None):
        import torch
        st, nbytes = nnconv_workspace_size(self.desc, pass_)
        check(st, "nnconv_workspace_size")
        t = self._ws.get(pass_)
        if t is None or t.numel() < nbytes:
            t = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device or "cuda")
            self._ws[pass_] = t
        return t, nbytes

    @staticmethod
    def _stream(stream):
        import torch
        return stream if stream is not None else torch.cuda.current_stream().cuda_stream

    def fwd(self, x, w, y, alpha=1.0, stream=None):
        ws, nb = self.workspace(NNCONV_FWD, x.device)
        check(nnconv_fwd(self.desc, x.data_ptr(), w.data_ptr(), y.data_ptr(), alpha,
                         ws.data_ptr(), nb, self._stream(stream)), "nnconv_fwd")

    def dgrad(self, dy, w, dx, alpha=1.0, stream=None):
        ws, nb = self.workspace(NNCONV_DGRAD, dy.device)
        check(nnconv_dgrad(self.desc, dy.data_ptr(), w.data_ptr(), dx.data_ptr(), alpha,
                           ws.data_ptr(), nb, self._stream(stream)), "nnconv_dgrad")

    def wgrad(self, x, dy, dw, dw_dtype=NNCONV_F32, inv_loss_scale=1.0, accumulate=0,
              overflow_flag=None, stream=None):
        ws, nb = self.workspace(NNCONV_WGRAD, x.device)
        flag = overflow_flag.data_ptr() if overflow_flag is not None else None
        check(nnconv_wgrad(self.desc, x.data_ptr(), dy.data_ptr(), dw.data_ptr(), dw_dtype,
                           inv_loss_scale, accumulate, flag, ws.data_ptr(), nb,
                           self._stream(stream)), "nnconv_wgrad")
