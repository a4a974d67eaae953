"""Every tile of the implicit-GEMM forward / backward-data kernel, forced
through nnconv_fwd_tile / nnconv_dgrad_tile, against the full fp64 oracle
on small shapes that still span several row and column tiles with ragged
edges: padded 3x3 (one launch, all stride phases for backward-data), 1x1
stride 2 (three tapless backward-data phases of exact zeros), reductions
shorter than the slice ring and ones many times longer.  The per-shape
picker reaches some tiles only at batch 256; forcing them here puts each
under the oracle in fp16 and bf16."""
import pytest

from paper_2102_06725_amd import inputs as I
from paper_2102_06725_amd import nnconv as nc

import gpu_util as U

pytestmark = pytest.mark.gpu

SHAPES = [
    # name, n, c, h, w, k, r, s, stride, pad
    ("k3s1", 5, 64, 10, 10, 320, 3, 3, 1, 1),    # 500 rows, 5 column tiles of 64
    ("k3s2", 4, 128, 13, 11, 192, 3, 3, 2, 1),   # dgrad: 4 phases of different sizes
    ("k1s2", 3, 64, 14, 12, 128, 1, 1, 2, 0),    # dgrad: 3 tapless phases
    ("k1s1", 2, 64, 9, 15, 64, 1, 1, 1, 0),      # 2 slices of 32: fewer than the ring
    ("long", 2, 512, 5, 6, 256, 3, 3, 1, 1),     # 144 slices of 32
]


@pytest.mark.parametrize("tile", nc.TILES)
@pytest.mark.parametrize("dtype", [I.F16, I.BF16])
@pytest.mark.parametrize("shape", SHAPES, ids=[s[0] for s in SHAPES])
def test_forced_tile_parity(nnlib, oracle_lib, tile, dtype, shape):
    name, n, c, h, w, k, r, s, stride, pad = shape
    L = I.Layer(name, n, c, h, w, k, r, s, stride=stride, pad=pad)
    case = U.Case(L, dtype=dtype, loss_scale=1.0, x_kind="normal", cfg=91,
                  layer_id=tile * 10 + SHAPES.index(shape))
    print("tile %d %s %s" % (tile, dtype, name), flush=True)
    U.full_parity(case, passes=("fwd", "dgrad"), tile=tile)


# Stride-1 geometries whose output is the input's size: the halo tiles.
HALO_SHAPES = [
    # name, n, c, h, w, k, r, s, pad, dil
    ("h3", 5, 64, 10, 10, 320, 3, 3, 1, 1),      # 500 rows: a ragged second tile
    ("h3w63", 3, 128, 9, 63, 192, 3, 3, 1, 1),   # widest image: a 384-row halo
    ("h3tiny", 1, 64, 3, 4, 64, 3, 3, 1, 1),     # 12 rows, halo past both ends
    ("h1", 2, 64, 9, 15, 64, 1, 1, 0, 1),        # 1x1: the halo is the tile
    ("h5", 2, 64, 8, 12, 128, 5, 5, 2, 1),       # 25 taps
    ("hdil", 2, 128, 11, 9, 64, 3, 3, 2, 2),     # dilation 2
    ("hlong", 2, 512, 5, 6, 256, 3, 3, 1, 1),    # 8 channel slices
    ("h64", 3, 64, 20, 24, 64, 3, 3, 1, 1),      # 64 -> 64: 1440 rows, a ragged 448-row tile
    ("h64w56", 1, 64, 9, 56, 64, 3, 3, 1, 1),    # 64 -> 64 on a 56-wide image (span 114)
]


@pytest.mark.parametrize("tile", nc.HALO_TILES)
@pytest.mark.parametrize("dtype", [I.F16, I.BF16])
@pytest.mark.parametrize("shape", HALO_SHAPES, ids=[s[0] for s in HALO_SHAPES])
def test_forced_halo_tile_parity(nnlib, oracle_lib, tile, dtype, shape):
    name, n, c, h, w, k, r, s, pad, dil = shape
    L = I.Layer(name, n, c, h, w, k, r, s, stride=1, pad=pad, dil=dil)
    case = U.Case(L, dtype=dtype, loss_scale=1.0, x_kind="normal", cfg=93,
                  layer_id=tile * 10 + HALO_SHAPES.index(shape))
    print("halo tile %d %s %s" % (tile, dtype, name), flush=True)
    span = (r - 1) * dil * w + (s - 1) * dil   # raster positions between the outer taps
    taps = nc.HALO_TILE_TAPS.get(tile)
    red = nc.HALO_TILE_RED.get(tile)
    fits = span <= nc.HALO_TILE_SPAN[tile] and (taps is None or r * s == taps)
    # a halo buffer too small for the taps, a tile compiled for another tap
    # count, or (single-slice tile) a reduction other than one 64-channel
    # slice (C forward, K backward-data): refused before anything runs
    ok = {"fwd": fits and (red is None or c == red), "dgrad": fits and (red is None or k == red)}
    refused = [p for p in ("fwd", "dgrad") if not ok[p]]
    if refused:
        t = case.tensors()
        for p in refused:
            with pytest.raises(nc.NNConvError) as e:
                U.run_gpu(case, t, (p,), tile=tile)
            assert e.value.status == nc.NNCONV_ERR_UNSUPPORTED
    run = tuple(p for p in ("fwd", "dgrad") if ok[p])
    if run:
        U.full_parity(case, passes=run, tile=tile)


@pytest.mark.parametrize("tile", [nc.NNCONV_TILE_256x256_RING, nc.NNCONV_TILE_256x128_RING,
                                  nc.NNCONV_TILE_HALO_256x64, nc.NNCONV_TILE_HALO_256x128,
                                  nc.NNCONV_TILE_HALO_R256x128, nc.NNCONV_TILE_HALO_R128x256])
def test_forced_tile_nchw_and_alpha(nnlib, oracle_lib, tile):
    """NCHW calls go through the channel-last kernels via the workspace; a
    non-unit alpha scales before the single rounding."""
    L = I.Layer("nchw", 3, 64, 7, 9, 128, 3, 3, stride=1, pad=1)
    case = U.Case(L, layout="nchw", dtype=I.F16, x_kind="normal", cfg=92, layer_id=tile,
                  alpha=-0.5)
    U.full_parity(case, passes=("fwd", "dgrad"), tile=tile)
