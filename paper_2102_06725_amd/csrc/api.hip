// api.hip -- the C ABI of libnnconv: argument validation (host only, before
// anything is queued), workspace planning, and dispatch to the kernels.
#include "nnconv.h"

#include <string.h>

#include <mutex>

#include "launch.hpp"

#define NNCONV_API extern "C" __attribute__((visibility("default")))

using namespace nnconv;

namespace {

struct Geom {
    int64_t n, c, h, w, k, r, s, sh, sw, ph, pw, dh, dw, g, p, q, cg, kg;
    int layout, dtype;
    // 1: the 64x64 per-tap weight blocks are block-diagonal in 32x32 blocks
    // (super-groups of groups of at most 32 channels)
    int diag32;
};

constexpr int64_t MAX_ELEMS = int64_t(1) << 40;

nnconv_status validate(const nnconv_desc *d, Geom *G) {
    if (!d) return NNCONV_ERR_INVALID_ARG;
    if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->k < 1 || d->r < 1 || d->s < 1)
        return NNCONV_ERR_INVALID_ARG;
    if (d->stride_h < 1 || d->stride_w < 1 || d->dil_h < 1 || d->dil_w < 1 || d->pad_h < 0 ||
        d->pad_w < 0 || d->groups < 1)
        return NNCONV_ERR_INVALID_ARG;
    if (d->c % d->groups != 0 || d->k % d->groups != 0) return NNCONV_ERR_INVALID_ARG;
    if (d->layout != NNCONV_NCHW && d->layout != NNCONV_NHWC) return NNCONV_ERR_INVALID_ARG;
    if (d->dtype != NNCONV_F16 && d->dtype != NNCONV_BF16) {
        if (d->dtype == NNCONV_F32) return NNCONV_ERR_UNSUPPORTED;
        return NNCONV_ERR_INVALID_ARG;
    }
    Geom g;
    g.n = d->n; g.c = d->c; g.h = d->h; g.w = d->w; g.k = d->k; g.r = d->r; g.s = d->s;
    g.sh = d->stride_h; g.sw = d->stride_w; g.ph = d->pad_h; g.pw = d->pad_w;
    g.dh = d->dil_h; g.dw = d->dil_w; g.g = d->groups;
    const int64_t num_h = g.h + 2 * g.ph - g.dh * (g.r - 1) - 1;
    const int64_t num_w = g.w + 2 * g.pw - g.dw * (g.s - 1) - 1;
    if (num_h < 0 || num_w < 0) return NNCONV_ERR_INVALID_ARG;
    g.p = num_h / g.sh + 1;
    g.q = num_w / g.sw + 1;
    g.cg = g.c / g.g;
    g.kg = g.k / g.g;
    // guard the size products used below
    if (g.n * g.c > MAX_ELEMS / (g.h * g.w) || g.n * g.k > MAX_ELEMS / (g.p * g.q) ||
        g.k * g.cg > MAX_ELEMS / (g.r * g.s))
        return NNCONV_ERR_INVALID_ARG;
    g.layout = d->layout;
    g.dtype = d->dtype;
    g.diag32 = 0;
    *G = g;
    return NNCONV_OK;
}

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
inline bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Shape-level eligibility of the matrix-core path.
bool fast_shape(const Geom &G) {
    if (G.cg % 8 != 0 || G.kg % 8 != 0) return false;
    if (G.r * G.s > MAX_TAPS) return false;
    const int64_t lim = MAX_BUFFER_BYTES / 2;  // elements per operand
    if (G.n * G.h * G.w * G.c > lim) return false;
    if (G.n * G.p * G.q * G.k > lim) return false;
    if (G.k * G.r * G.s * G.cg > lim) return false;
    return true;
}

// Depthwise convolution on its vector-ALU kernels: one input and one output
// channel per group, 8-channel vectors, square 3x3 / 5x5 / 7x7 filters.
bool dw_shape(const Geom &G) {
    if (!(G.g == G.c && G.k == G.c && G.c % 8 == 0 && dw_supported((int)G.r, (int)G.s)))
        return false;
    const int64_t lim = MAX_BUFFER_BYTES / 2;
    return G.n * G.h * G.w * G.c <= lim && G.n * G.p * G.q * G.k <= lim;
}

// Backward-weight pixel ranges of the gather depthwise kernel: about 2048
// workgroups, at least 256 pixels per range (the LDS-tiled kernel plans its
// own splits).
int32_t dw_wgrad_splits(const Geom &G) {
    const int64_t cblocks = (G.c / 8 + 7) / 8;
    const int64_t npq = G.n * G.p * G.q;
    int64_t s = 2048 / (cblocks * G.r);
    if (s > npq / 256) s = npq / 256;
    if (s > 4096) s = 4096;
    if (s < 1) s = 1;
    return (int32_t)s;
}

// Grouped convolution with m = Cg = Kg channels per group, m < 64 dividing 64
// (ResNeXt's g = 32 layers: m = 4-32): run as super-groups of 64 channels
// with block-diagonal weights on the 64-channel-slice kernels.  For finite
// inputs the sums are the same products plus exact zeros; a non-finite input
// can turn the other groups of its super-group into NaN (0 * inf).
constexpr int64_t SUPER_GROUP = 64;

bool fast_shape(const Geom &G);

bool sg_shape(const Geom &G) {
    if (G.g < 2 || G.cg != G.kg || G.cg >= SUPER_GROUP || SUPER_GROUP % G.cg != 0 ||
        G.c % SUPER_GROUP != 0)
        return false;
    if (dw_shape(G)) return false;  // depthwise has its own kernels
    return true;
}

// The same convolution with groups of SUPER_GROUP channels.
Geom sg_geom(const Geom &G) {
    Geom S = G;
    S.g = G.c / SUPER_GROUP;
    S.cg = S.kg = SUPER_GROUP;
    S.diag32 = G.cg <= 32;  // always: the group size divides 64 and is below it
    return S;
}

// The 64-channel-slice tile for a GEMM with ncols output columns: the
// block-diagonal variant of the 64-column tile when the weights allow it.
C64Config pick_c64(int64_t m, int64_t ncols, int64_t red);
C64Config pick_c64_geom(const Geom &G, int64_t m, int64_t ncols, int64_t red) {
    const C64Config c = pick_c64(m, ncols, red);
    return (G.diag32 && ncols == SUPER_GROUP && c == C64S_128x64) ? C64D_128x64 : c;
}

// ---------------------------------------------------------------------------
// planning: workspace regions and split counts (pure functions of the shape)
// ---------------------------------------------------------------------------

// 8-channel pixels into 64 channels with the stem's filter: the patch
// kernel; 4-channel pixels too when the left padding is odd and the image
// width even.
bool stem_shape(const Geom &G) {
    if (!(G.g == 1 && G.k == 64 && G.dh == 1 && G.dw == 1 &&
          stem_fwd_supported((int)G.r, (int)G.s, (int)G.sh, (int)G.sw)))
        return false;
    return G.cg == 8 || (G.cg == 4 && G.pw % 2 == 1 && G.w % 2 == 0);
}

// Whether pass `pass` of this shape runs on the channel-last kernels: the
// implicit-GEMM shapes, and the forward and backward-weight passes of the
// 4-channel stem in channel-last layout (its backward-data and its NCHW
// calls take the direct kernels).
bool fast_pass(const Geom &G, nnconv_pass pass) {
    if (fast_shape(G)) return true;
    if (!(G.cg == 4 && stem_shape(G) && pass != NNCONV_DGRAD && G.layout == NNCONV_NHWC))
        return false;
    const int64_t lim = MAX_BUFFER_BYTES / 2;
    return G.n * G.h * G.w * G.c <= lim && G.n * G.p * G.q * G.k <= lim;
}

// Stem backward-weight: persistent workgroups (one split-K partial each).
constexpr int64_t STEM_WG_SPLITS = 256;

int device_cus();

struct WgPlan {
    bool stem;  // patch kernel (stem_shape)
    WGConfig cfg;
    int32_t splits, pix_per_split;
    int32_t rb, blocks_per_img, nblocks, blocks_per_split;  // WG_HALO: row blocks
};

// Rows per block of the row-block backward-weight kernel (wgrad_halo.hip)
// for this geometry, or 0 when it does not run it: 3x3 stride-1 "same"
// convolutions (padding 1, dilation 1) with groups of 64 input and 64 output
// channels (super-groups of smaller groups included), on images whose width
// admits blocks of whole rows of a multiple of 16 and at most 128 pixels
// (the largest such block is taken) that fits the kernel's LDS buffers.
// With more than one group the block may not be taller than the image (a
// 7x7 image would stage 16-row blocks: the 64-row tiles do better there).
int64_t wgh_rows(const Geom &G) {
    if (!(G.cg == 64 && G.kg == 64 && G.r == 3 && G.s == 3 && G.sh == 1 && G.sw == 1 &&
          G.dh == 1 && G.dw == 1 && G.ph == 1 && G.pw == 1 && G.p == G.h && G.q == G.w &&
          G.g <= 65535))
        return 0;
    int64_t rb0 = 1;
    while ((rb0 * G.w) % 16 != 0) ++rb0;  // at most 16
    if (rb0 * G.w > 128) return 0;
    const int64_t rb = rb0 * (128 / (rb0 * G.w));
    if (wgh_slots((int)rb, (int)G.w) > WGH_MAX_SLOTS) return 0;
    if (G.g > 1 && rb > G.h) return 0;
    return rb;
}

// Backward-weight tile and workgroup target, from measurements on the
// ResNet-50 layers at batch 256:
//   - 256x256 tiles and about 256 workgroups (long pixel ranges, few partial
//     tiles to write and reduce) for filters of several taps when both GEMM
//     sides are at least 256 wide;
//   - 64-row tiles when Kg <= 64, with 1024 workgroups for filters of
//     several taps and 512 for 1x1 ones (the 56x56 1x1 layers into 64
//     channels: 37 / 99 us against 41 / 111 with 1024);
//   - otherwise 128x128 tiles and 512 workgroups, single-stage for very wide
//     filters (R*S*Cg >= 4096), where more resident workgroups per CU pay
//     off.  This includes the 1x1 layers with both sides at least 256 wide,
//     which read both operands once and are bound by memory traffic: there
//     the 256x256 tiles' longer pixel ranges do not pay for the extra
//     operand streams of half as many workgroups (14x14 and 7x7 1x1 layers:
//     43 us against 49-51).
WGConfig pick_wg(int64_t kg, int64_t rscg, int64_t taps) {
    if (kg <= 64) return WG_64x128;
    if (taps > 1 && kg >= 256 && rscg >= 256 && rscg < 4096) return WG_256x256;
    return rscg >= 4096 ? WG_128x128S : WG_128x128;
}

int64_t wg_target_blocks(WGConfig cfg, int64_t taps) {
    if (cfg == WG_64x128 || cfg == WG_64x128D) return taps > 1 ? 1024 : 512;
    return cfg == WG_256x256 ? 256 : 512;
}

WgPlan plan_wgrad_fast(const Geom &G) {
    WgPlan pl = {};
    pl.stem = stem_shape(G);
    if (pl.stem) {
        const int64_t tiles = G.n * ((G.p + 15) / 16) * ((G.q + 15) / 16);
        pl.cfg = WG_128x128;
        pl.splits = (int32_t)(tiles < STEM_WG_SPLITS ? tiles : STEM_WG_SPLITS);
        if (G.cg == 4) pl.splits *= 2;  // two partials per workgroup
        pl.pix_per_split = 0;
        return pl;
    }
    pl.rb = (int32_t)wgh_rows(G);
    if (pl.rb > 0) {
        // one workgroup per CU (over all groups), consecutive row blocks each
        pl.cfg = WG_HALO;
        pl.blocks_per_img = (int32_t)((G.h + pl.rb - 1) / pl.rb);
        const int64_t nb = G.n * pl.blocks_per_img;
        const int64_t cus = device_cus();
        const int64_t per = (nb * G.g + cus - 1) / cus;
        pl.nblocks = (int32_t)nb;
        pl.blocks_per_split = (int32_t)per;
        pl.splits = (int32_t)((nb + per - 1) / per);
        pl.pix_per_split = 0;
        return pl;
    }
    const int64_t rscg = G.r * G.s * G.cg;
    pl.cfg = pick_wg(G.kg, rscg, G.r * G.s);
    if (G.diag32 && pl.cfg == WG_64x128 && G.kg == SUPER_GROUP) pl.cfg = WG_64x128D;
    static const int64_t tile_m[] = {128, 64, 256, 128, 64};
    static const int64_t tile_n[] = {128, 128, 256, 128, 128};
    const int64_t bmk = tile_m[pl.cfg], bnj = tile_n[pl.cfg];
    const int64_t tiles = G.g * ((G.kg + bmk - 1) / bmk) * ((rscg + bnj - 1) / bnj);
    const int64_t npq = G.n * G.p * G.q;
    const int64_t iters = (npq + 63) / 64;  // 64-pixel units
    const int64_t target = wg_target_blocks(pl.cfg, G.r * G.s);
    int64_t splits = (target + tiles - 1) / tiles;
    int64_t max_splits = iters / 4;  // at least 256 pixels per split
    if (max_splits < 1) max_splits = 1;
    if (splits > max_splits) splits = max_splits;
    if (splits > 1024) splits = 1024;
    if (splits < 1) splits = 1;
    const int64_t per = ((iters + splits - 1) / splits) * 64;
    pl.pix_per_split = (int32_t)per;
    pl.splits = (int32_t)((npq + per - 1) / per);
    return pl;
}

int32_t plan_wgrad_direct_splits(const Geom &G) {
    const int64_t npq = G.n * G.p * G.q;
    int64_t s = (npq + 2047) / 2048;
    if (s > 64) s = 64;
    if (s < 1) s = 1;
    return (int32_t)s;
}

struct Regions {  // byte offsets into the caller's workspace
    size_t a, b, c, d, e, f, total;
};

// Bytes of fragment-packed weights the register-weight halo tiles need for
// this geometry and pass: 3x3 filters, stride 1, output the input's size,
// 64-channel multiples, taps within the larger halo buffer's span, and one
// group or groups of 64 channels (the single-slice tile).  0 when no such
// tile can run it.
size_t hring_ws(const Geom &G, nnconv_pass pass) {
    if (!((G.g == 1 || (G.cg == 64 && G.kg == 64)) && G.sh == 1 && G.sw == 1 && G.p == G.h &&
          G.q == G.w && G.r * G.s == HRING_TAPS && G.cg % 64 == 0 && G.kg % 64 == 0 &&
          (G.r - 1) * G.dh * G.w + (G.s - 1) * G.dw <= HALO_SPAN))
        return 0;
    if (pass == NNCONV_FWD) return hring_pack_bytes(G.kg, G.cg, G.g);
    if (pass == NNCONV_DGRAD) return hring_pack_bytes(G.cg, G.kg, G.g);
    return 0;
}

Regions fast_regions(const Geom &G, nnconv_pass pass) {
    Regions R = {0, 0, 0, 0, 0, 0, 0};
    const size_t e2 = 2;
    const size_t xb = G.n * G.h * G.w * G.c * e2;
    const size_t yb = G.n * G.p * G.q * G.k * e2;
    const size_t wb = G.k * G.r * G.s * G.cg * e2;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    const bool nchw = G.layout == NNCONV_NCHW;
    if (pass == NNCONV_FWD) {
        if (nchw) {
            R.a = take(xb);  // x channel-last
            R.b = take(wb);  // w [K][R][S][Cg]
            R.c = take(yb);  // y channel-last
        }
        R.f = take(hring_ws(G, pass));  // packed weights (register-weight halo tiles)
    } else if (pass == NNCONV_DGRAD) {
        if (nchw) {
            R.a = take(yb);  // dy channel-last
            R.d = take(wb);  // w [K][R][S][Cg] (intermediate)
            R.c = take(xb);  // dx channel-last
        }
        R.b = take(wb);      // w [g][R][S][Cg][Kg]
        // non-finite flags of the weight re-layout's workgroups
        R.e = take((size_t)transpose16_blocks(G.g, G.r * G.s * G.cg, G.kg) * 4);
        R.f = take(hring_ws(G, pass));  // packed weights (register-weight halo tiles)
    } else {
        if (nchw) {
            R.a = take(xb);  // x channel-last
            R.b = take(yb);  // dy channel-last
        }
        const WgPlan pl = plan_wgrad_fast(G);
        R.c = take((size_t)pl.splits * G.k * G.r * G.s * G.cg * 4);
    }
    R.total = off;
    return R;
}

size_t direct_ws(const Geom &G, nnconv_pass pass) {
    if (pass != NNCONV_WGRAD) return 0;
    return align256((size_t)plan_wgrad_direct_splits(G) * G.k * G.r * G.s * G.cg * 4);
}

DWParams dw_params(const Geom &G, float alpha);

// Depthwise workspace: the channel-last copies for NCHW calls, fp32 split
// partials (backward-weight).
Regions dw_regions(const Geom &G, nnconv_pass pass) {
    Regions R = {0, 0, 0, 0, 0, 0, 0};
    const size_t xb = G.n * G.h * G.w * G.c * 2;
    const size_t yb = G.n * G.p * G.q * G.k * 2;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    const bool nchw = G.layout == NNCONV_NCHW;
    if (pass == NNCONV_FWD) {
        if (nchw) { R.a = take(xb); R.c = take(yb); }
    } else if (pass == NNCONV_DGRAD) {
        if (nchw) { R.a = take(yb); R.c = take(xb); }
        R.e = take((size_t)nonfinite_scan16_blocks(G.c * G.r * G.s) * 4);  // weight flags
    } else {
        if (nchw) { R.a = take(xb); R.b = take(yb); }
        R.c = take((size_t)dw_params(G, 1.0f).splits * G.c * G.r * G.s * 4);
    }
    R.total = off;
    return R;
}

// Super-group workspace: the block-diagonal weights [K][R][S][64] (forward,
// backward-data), then the super-grouped problem's own regions.
Regions sg_regions(const Geom &G, nnconv_pass pass) {
    const Geom S = sg_geom(G);
    Regions R = {0, 0, 0, 0, 0, 0, 0};
    const size_t wexp = pass == NNCONV_WGRAD ? 0 : align256(G.k * G.r * G.s * SUPER_GROUP * 2);
    const Regions in = fast_regions(S, pass);
    R.d = 0;            // expanded weights
    R.a = wexp + in.a;  // NCHW copies / dgrad weight re-layout / partials, shifted
    R.b = wexp + in.b;
    R.c = wexp + in.c;
    R.e = wexp + in.e;
    R.f = wexp + in.f;
    R.total = wexp + in.total;
    return R;
}

size_t workspace_bytes(const Geom &G, nnconv_pass pass) {
    if (sg_shape(G) && fast_shape(sg_geom(G))) {  // or the direct kernels (unaligned)
        const size_t a = sg_regions(G, pass).total, b = direct_ws(G, pass);
        return a > b ? a : b;
    }
    if (dw_shape(G)) {  // the vector kernels, or the direct ones for unaligned pointers
        const size_t a = dw_regions(G, pass).total, b = direct_ws(G, pass);
        return a > b ? a : b;
    }
    size_t d = direct_ws(G, pass);
    if (!fast_pass(G, pass)) return d;
    size_t f = fast_regions(G, pass).total;
    return f > d ? f : d;
}

DirectParams direct_params(const Geom &G, float alpha) {
    DirectParams P;
    P.n = (int32_t)G.n; P.c = (int32_t)G.c; P.h = (int32_t)G.h; P.w = (int32_t)G.w;
    P.k = (int32_t)G.k; P.r = (int32_t)G.r; P.s = (int32_t)G.s; P.p = (int32_t)G.p;
    P.q = (int32_t)G.q; P.sh = (int32_t)G.sh; P.sw = (int32_t)G.sw; P.ph = (int32_t)G.ph;
    P.pw = (int32_t)G.pw; P.dh = (int32_t)G.dh; P.dw = (int32_t)G.dw;
    P.groups = (int32_t)G.g; P.cg = (int32_t)G.cg; P.kg = (int32_t)G.kg;
    if (G.layout == NNCONV_NCHW) {
        P.xs[0] = G.c * G.h * G.w; P.xs[1] = G.h * G.w; P.xs[2] = G.w; P.xs[3] = 1;
        P.ys[0] = G.k * G.p * G.q; P.ys[1] = G.p * G.q; P.ys[2] = G.q; P.ys[3] = 1;
        P.wsd[0] = G.cg * G.r * G.s; P.wsd[1] = G.r * G.s; P.wsd[2] = G.s; P.wsd[3] = 1;
    } else {
        P.xs[0] = G.h * G.w * G.c; P.xs[1] = 1; P.xs[2] = G.w * G.c; P.xs[3] = G.c;
        P.ys[0] = G.p * G.q * G.k; P.ys[1] = 1; P.ys[2] = G.q * G.k; P.ys[3] = G.k;
        P.wsd[0] = G.r * G.s * G.cg; P.wsd[1] = 1; P.wsd[2] = G.s * G.cg; P.wsd[3] = G.cg;
    }
    P.alpha = alpha;
    return P;
}

// The same element strides for channel-last activations (the layout the
// fast kernels produce dx in, also for NCHW calls, whose dx is transposed
// afterwards), weights as the caller gave them.
DirectParams direct_params_cl(const Geom &G, float alpha) {
    DirectParams P = direct_params(G, alpha);
    P.xs[0] = G.h * G.w * G.c; P.xs[1] = 1; P.xs[2] = G.w * G.c; P.xs[3] = G.c;
    P.ys[0] = G.p * G.q * G.k; P.ys[1] = 1; P.ys[2] = G.q * G.k; P.ys[3] = G.k;
    return P;
}

// dx rows (cols) at the top / bottom (left / right) that may have filter
// taps outside dy: row i reaches p < 0 only if i < (R-1)*dil - pad, and
// p >= P only if i >= P*stride - pad.
struct Border {
    int32_t bt, bb, bl, br;
};
Border dgrad_border(const Geom &G) {
    auto ext = [](int64_t h, int64_t r, int64_t ph, int64_t dh, int64_t sh, int64_t p,
                  int32_t &lo, int32_t &hi) {
        int64_t t = (r - 1) * dh - ph;
        t = t < 0 ? 0 : (t > h ? h : t);
        int64_t b = h - (p * sh - ph);
        b = b < 0 ? 0 : (b > h - t ? h - t : b);
        lo = (int32_t)t;
        hi = (int32_t)b;
    };
    Border B;
    ext(G.h, G.r, G.ph, G.dh, G.sh, G.p, B.bt, B.bb);
    ext(G.w, G.s, G.pw, G.dw, G.sw, G.q, B.bl, B.br);
    return B;
}

thread_local int32_t last_hip_error = 0;

inline nnconv_status hip_status(hipError_t e) {
    if (e == hipSuccess) return NNCONV_OK;
    last_hip_error = (int32_t)e;
    return NNCONV_ERR_HIP;
}

#define TRY_HIP(expr)                                          \
    do {                                                       \
        hipError_t e_ = (expr);                                \
        if (e_ != hipSuccess) return hip_status(e_);           \
    } while (0)

// Launch errors are read with hipGetLastError; drop any error an unrelated
// earlier runtime call on this thread left behind so it is not blamed on us.
inline void clear_stale_error() { (void)hipGetLastError(); }

// Common part of the forward pass and of each backward-data phase.
TNParams tn_base() {
    TNParams p;
    memset(&p, 0, sizeof(p));
    return p;
}

C8Config pick_c8(int64_t ncols) { return ncols <= 64 ? C8_256x64 : C8_128x128; }

// Tile configuration for the 64-channel-slice kernel, from measurements on
// the ResNet-50 layers at batch 256 (m = GEMM rows, ncols = output channels
// per group, red = reduction length):
//   - the per-CU load path (about 64 bytes per clock) keeps the matrix
//     cores busy only with 256x256 tiles (128 flop per staged byte); they
//     win on long reductions once there are enough tiles to give most CUs
//     one (3x3 layers on 14x14 with 256 output channels, GEMM-sized
//     problems);
//   - otherwise the single-stage 128-row tiles, 3-5 per CU, hide each
//     other's load latency best; very long reductions prefer the pipelined
//     128x128 tile;
//   - a 256x256 tile run by 16 waves (four per SIMD) beats both for 256
//     output columns with long reductions on 100-256 row tiles.
constexpr int64_t MIN_BIG_TILES = 160;
constexpr int64_t BIG_RED = 2048;
constexpr int64_t LONG_RED = 4096;

C64Config pick_c64(int64_t m, int64_t ncols, int64_t red) {
    if (ncols <= 64) return C64S_128x64;
    // 256 output columns, long reductions, about 200 tiles of 256 rows (the
    // 14x14 layers at batch 256): the 16-wave 256x256 tile
    if (ncols == 256 && red >= 1024 && m > 98 * 256 && m <= 256 * 256) return C64W_256x256;
    const int64_t big_tiles = ((m + 255) / 256) * ((ncols + 255) / 256);
    if (ncols >= 256 && red >= BIG_RED && big_tiles >= MIN_BIG_TILES) return C64_256x256;
    // fewer 128x128 tiles than one round of single-stage workgroups (four
    // per CU): the pipelined tile already pays from half the long reduction
    const int64_t tiles = ((m + 127) / 128) * ((ncols + 127) / 128);
    const int64_t long_red = tiles < 4 * 256 ? LONG_RED / 2 : LONG_RED;
    return red >= long_red ? C64_128x128 : C64S_128x128;
}

// Forced-tile ids HALO_TILE0 .. HALO_TILE0 + HALO_CONFIGS - 1 select the
// halo-staged kernel (HaloConfig = id - HALO_TILE0); lower ones are
// C64Config values.
constexpr int HALO_TILE0 = 9;
constexpr int HALO_CONFIGS = HALO_R256x64S + 1;
bool halo_tile(int tile) { return tile >= HALO_TILE0 && tile < HALO_TILE0 + HALO_CONFIGS; }
// the register-weight halo configurations (packed weights in the workspace)
bool hring_cfg(int hc) { return hring_config(hc); }

// Whether the halo-staged kernel can run this shape's forward and
// backward-data passes (the geometry halo_supported() accepts, stated on the
// convolution): one group (or, on the single-slice tile, groups of 64
// channels), stride 1, output the input's size, 64-channel multiples, taps
// spanning at most HALO_SPAN raster positions.  `red` is the
// pass's reduction channel count (Cg forward, Kg backward-data), which the
// single-slice tile needs to be 64.
bool halo_geom(const Geom &G, int tile, int64_t red) {
    const HaloConfig hc = (HaloConfig)(tile - HALO_TILE0);
    const bool regw = hring_cfg(hc);
    // one group, or groups of 64 channels on the single-slice tile
    return (G.g == 1 || (hc == HALO_R256x64S && G.cg == 64 && G.kg == 64)) && G.sh == 1 &&
           G.sw == 1 && G.p == G.h && G.q == G.w && G.cg % 64 == 0 &&
           G.kg % 64 == 0 && G.r * G.s <= 32 && (!regw || G.r * G.s == HRING_TAPS) &&
           (hc != HALO_R256x64S || red == 64) &&
           (G.r - 1) * G.dh * G.w + (G.s - 1) * G.dw <= halo_cfg_span(hc);
}

// The halo-staged kernel's tile for a stride-1 "same" implicit GEMM, or -1
// for the 64-channel-slice kernel.  Measured on the ResNet-50 layers at
// batch 256 (forward and backward-data; times include the weight packing):
//   - the register-weight tiles (packed weights in the workspace, 3x3
//     filters): the single-slice 256x64 tile for a 64-channel reduction
//     into at most 64 columns (the 56x56 64-channel 3x3 layers: 82 / 86 us
//     against 101 / 102 for the 128x64 64-channel-slice tile, the packing
//     included); the 224x256 tile when the taps span at most 32 raster
//     positions, the output columns are a multiple of 256 and its tiles
//     fill between three quarters of the CUs and all of them in one round
//     (the 14x14 256-channel layers: 224 tiles, 62 / 68 us against 66 / 71
//     for the 16-wave 256x256 tile); the 256x128 tile on 7x7 images with at
//     least 512 columns (66 / 71 us against 71 / 78 for the single-buffer
//     halo tile, which those layers took before);
//   - otherwise the single-buffer 256x64 halo tile on 3x3-like filters over
//     7x7 images with at least 256 output columns, where the
//     64-channel-slice tiles stage each input pixel once per tap and per
//     64-column tile (2-3% faster than the pipelined 128x128 tile, 8-14%
//     than the single-stage ones); it ties or loses on wider images.
// A 1x1 filter has no halo to share: its tile is a plain GEMM tile, slower
// than the 64-channel-slice ones (40-60% on the 7x7 1x1 layers).
int device_cus();
int pick_halo(const TNParams &p, bool pack) {
    // groups of 64 channels (super-groups of a grouped convolution): the
    // single-slice tile or none
    if (p.groups > 1)
        return pack && p.ph[0].tap_count == HRING_TAPS && halo_cfg_supported(p, HALO_R256x64S)
                   ? HALO_R256x64S
                   : -1;
    if (p.ph[0].tap_count < 2 || !halo_supported(p)) return -1;
    if (pack && p.ph[0].tap_count == HRING_TAPS) {
        if (p.cr == 64 && p.ncols <= 64 && halo_cfg_supported(p, HALO_R256x64S))
            return HALO_R256x64S;
        const int64_t cus = device_cus();
        const int64_t t224 = ((int64_t)p.ph[0].M + 223) / 224 * ((p.ncols + 255) / 256);
        if (p.ncols % 256 == 0 && hring_supported(p, halo_cfg_span(HALO_R224x256)) &&
            t224 <= cus && 4 * t224 >= 3 * cus)
            return HALO_R224x256;
        if (p.a_w <= 7 && p.ncols >= 512 && hring_supported(p, halo_cfg_span(HALO_R256x128)))
            return HALO_R256x128;
    }
    if (p.a_w > 7 || p.ncols < 256) return -1;
    return HALO_256x64;
}

// Compute units of the current device (the persistent kernels launch one
// workgroup per CU).
int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    return cus;
}

TNPhase phase_of(int64_t m, int64_t mi, int64_t mj, int64_t oi_add, int64_t oj_add, int tap_start,
                 int tap_count) {
    TNPhase f;
    memset(&f, 0, sizeof(f));
    f.M = (int32_t)m;
    f.mi = (int32_t)mi;
    f.mj = (int32_t)mj;
    f.div_mj = make_fastdiv((uint32_t)(mj > 0 ? mj : 1));
    f.div_mi = make_fastdiv((uint32_t)(mi > 0 ? mi : 1));
    f.oi_add = (int32_t)oi_add;
    f.oj_add = (int32_t)oj_add;
    f.tap_start = tap_start;
    f.tap_count = tap_count;
    return f;
}

// Whether the 64-channel-slice kernel runs the forward / backward-data pass
// of a shape that fast_shape() accepts (the tiles a caller may force).
bool c64_fwd_shape(const Geom &G) { return !stem_shape(G) && G.cg % 64 == 0; }
bool c64_dgrad_shape(const Geom &G) { return G.kg % 64 == 0 && G.sh * G.sw <= MAX_PHASES; }

// tile: a C64Config to force on the 64-channel-slice kernel, or -1 for the
// per-shape pick.
// pack: workspace for the register-weight halo tiles' packed weights
// (hring_ws bytes), or null when the call has none.
nnconv_status fwd_fast(const Geom &G, const void *x, const void *w, void *y, float alpha,
                       hipStream_t st, int tile = -1, void *pack = nullptr) {
    if (stem_shape(G)) {
        StemParams sp;
        sp.x = x;
        sp.x_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
        sp.wt = w;
        sp.wt_bytes = (uint32_t)(G.k * G.r * G.s * G.cg * 2);
        sp.y = y;
        sp.y_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
        sp.n = (int32_t)G.n; sp.h = (int32_t)G.h; sp.w = (int32_t)G.w;
        sp.p = (int32_t)G.p; sp.q = (int32_t)G.q;
        sp.r = (int32_t)G.r; sp.s = (int32_t)G.s; sp.sh = (int32_t)G.sh; sp.sw = (int32_t)G.sw;
        sp.ph = (int32_t)G.ph; sp.pw = (int32_t)G.pw;
        sp.c = (int32_t)G.c;
        sp.alpha = alpha;
        return hip_status(launch_stem_fwd(G.dtype, sp, device_cus(), st));
    }
    TNParams p = tn_base();
    p.a = x;
    p.a_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
    p.b = w;
    p.b_bytes = (uint32_t)(G.k * G.r * G.s * G.cg * 2);
    p.out = y;
    p.o_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
    p.mi = (int32_t)G.p;
    p.mj = (int32_t)G.q;
    p.M = (int32_t)(G.n * G.p * G.q);
    p.div_mj = make_fastdiv((uint32_t)G.q);
    p.div_mi = make_fastdiv((uint32_t)G.p);
    p.a_h = (int32_t)G.h; p.a_w = (int32_t)G.w; p.a_c = (int32_t)G.c;
    p.a_cg_ofs = (int32_t)G.cg;
    p.ai_mul = (int32_t)G.sh; p.ai_add = (int32_t)-G.ph;
    p.aj_mul = (int32_t)G.sw; p.aj_add = (int32_t)-G.pw;
    p.cr = (int32_t)G.cg;
    p.div_crv = make_fastdiv((uint32_t)(G.cg / 8));
    p.ncols = (int32_t)G.kg;
    p.b_ld = (int32_t)(G.r * G.s * G.cg);
    p.b_g_ofs = (int32_t)(G.kg * G.r * G.s * G.cg);
    p.o_h = (int32_t)G.p; p.o_w = (int32_t)G.q; p.o_c = (int32_t)G.k;
    p.o_cg_ofs = (int32_t)G.kg;
    p.oi_mul = 1; p.oi_add = 0; p.oj_mul = 1; p.oj_add = 0;
    p.alpha = alpha;
    p.groups = (int32_t)G.g;
    // Tap order of the 64-channel-slice kernel: the centre tap first.  Its
    // slice reads the tile's own pixels (first touch, from HBM); the other
    // taps then read pixels already in L2 (the tile's own or its
    // neighbours', whose centre slices run at the same time on the same
    // XCD), so fewer slices wait on HBM latency.  Any order gives the same
    // sum up to fp32 rounding.
    const int ntap = (int)(G.r * G.s);
    const int t0 = G.cg % 64 == 0 ? (int)((G.r / 2) * G.s + G.s / 2) : 0;
    int t = 0;
    for (int u = 0; u < ntap; ++u, ++t) {
        const int lin = (u + t0) % ntap;
        const int r = lin / (int)G.s, s = lin % (int)G.s;
        p.taps.dh[t] = (int32_t)(r * G.dh);
        p.taps.dw[t] = (int32_t)(s * G.dw);
        p.taps.boff[t] = (int32_t)(lin * G.cg);
    }
    p.taps.n = t;
    p.k_iters = (int32_t)((int64_t(t) * G.cg + 63) / 64);
    if (G.cg % 64 == 0) {
        p.nphase = 1;
        p.ph[0] = phase_of(p.M, p.mi, p.mj, 0, 0, 0, t);
        const int hc = halo_tile(tile) ? tile - HALO_TILE0 : tile < 0 ? pick_halo(p, pack != nullptr) : -1;
        if (hc >= 0) {
            if (!halo_cfg_supported(p, (HaloConfig)hc) || (hring_cfg(hc) && !pack))
                return NNCONV_ERR_UNSUPPORTED;
            return hip_status(
                launch_igemm_halo(G.dtype, (HaloConfig)hc, p, pack, G.diag32 != 0, st));
        }
        const C64Config cfg =
            tile >= 0 ? (C64Config)tile : pick_c64_geom(G, p.M, G.kg, (int64_t)t * G.cg);
        return hip_status(launch_igemm_c64(G.dtype, cfg, p, G.ph > 0 || G.pw > 0, st));
    }
    return hip_status(launch_igemm_c8(G.dtype, pick_c8(G.kg), p, st));
}

// Backward-data as sigma_h * sigma_w independent implicit GEMMs, one per
// output phase (h mod sigma_h, w mod sigma_w): within a phase every pixel
// sees the same set of contributing taps.  wt is [g][R][S][Cg][Kg].
nnconv_status dgrad_fast(const Geom &G, const void *dy, const void *wt, void *dx, float alpha,
                         hipStream_t st, int tile = -1, void *pack = nullptr) {
    TNParams base = tn_base();
    base.a = dy;
    base.a_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
    base.b = wt;
    base.b_bytes = (uint32_t)(G.k * G.r * G.s * G.cg * 2);
    base.out = dx;
    base.o_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
    base.a_h = (int32_t)G.p; base.a_w = (int32_t)G.q; base.a_c = (int32_t)G.k;
    base.a_cg_ofs = (int32_t)G.kg;
    base.ai_mul = 1; base.ai_add = 0; base.aj_mul = 1; base.aj_add = 0;
    base.cr = (int32_t)G.kg;
    base.div_crv = make_fastdiv((uint32_t)(G.kg / 8));
    base.ncols = (int32_t)G.cg;
    base.b_ld = (int32_t)G.kg;
    base.b_g_ofs = (int32_t)(G.r * G.s * G.cg * G.kg);
    base.o_h = (int32_t)G.h; base.o_w = (int32_t)G.w; base.o_c = (int32_t)G.c;
    base.o_cg_ofs = (int32_t)G.cg;
    base.oi_mul = (int32_t)G.sh;
    base.oj_mul = (int32_t)G.sw;
    base.alpha = alpha;
    base.groups = (int32_t)G.g;
    const bool pad = !(G.r == 1 && G.s == 1 && G.ph == 0 && G.pw == 0);
    // taps of output phase (phh, phw), appended to p.taps; returns their count
    auto add_phase_taps = [&](TNParams &p, int64_t phh, int64_t phw) {
        int t = 0;
        for (int64_t r = 0; r < G.r; ++r) {
            const int64_t nh = phh + G.ph - r * G.dh;  // = sigma_h * (p - i)
            if (((nh % G.sh) + G.sh) % G.sh != 0) continue;
            for (int64_t s = 0; s < G.s; ++s) {
                const int64_t nw = phw + G.pw - s * G.dw;
                if (((nw % G.sw) + G.sw) % G.sw != 0) continue;
                const int k = p.taps.n + t;
                p.taps.dh[k] = (int32_t)(nh / G.sh);
                p.taps.dw[k] = (int32_t)(nw / G.sw);
                p.taps.boff[k] = (int32_t)((r * G.s + s) * G.cg * G.kg);
                ++t;
            }
        }
        p.taps.n += t;
        return t;
    };
    if (c64_dgrad_shape(G)) {
        // every stride phase in one launch; a phase without taps writes zeros
        TNParams p = base;
        p.taps.n = 0;
        p.nphase = 0;
        // the tile is picked for the row-weighted mean reduction of the
        // phases (a stride-2 3x3 dgrad has 1, 2, 2 and 4 taps per phase)
        int64_t rows = 0, red_rows = 0;
        for (int64_t phh = 0; phh < G.sh; ++phh) {
            for (int64_t phw = 0; phw < G.sw; ++phw) {
                const int64_t mi = phh < G.h ? (G.h - phh + G.sh - 1) / G.sh : 0;
                const int64_t mj = phw < G.w ? (G.w - phw + G.sw - 1) / G.sw : 0;
                if (mi == 0 || mj == 0) continue;
                const int start = p.taps.n;
                const int cnt = add_phase_taps(p, phh, phw);
                p.ph[p.nphase++] = phase_of(G.n * mi * mj, mi, mj, phh, phw, start, cnt);
                rows += G.n * mi * mj;
                red_rows += G.n * mi * mj * cnt * G.kg;
            }
        }
        if (p.nphase == 0) return NNCONV_OK;
        const int hc = halo_tile(tile) ? tile - HALO_TILE0 : tile < 0 ? pick_halo(p, pack != nullptr) : -1;
        if (hc >= 0) {
            if (!halo_cfg_supported(p, (HaloConfig)hc) || (hring_cfg(hc) && !pack))
                return NNCONV_ERR_UNSUPPORTED;
            return hip_status(
                launch_igemm_halo(G.dtype, (HaloConfig)hc, p, pack, G.diag32 != 0, st));
        }
        const C64Config cfg =
            tile >= 0 ? (C64Config)tile : pick_c64_geom(G, rows, G.cg, red_rows / rows);
        return hip_status(launch_igemm_c64(G.dtype, cfg, p, pad, st));
    }
    // Otherwise sigma_h * sigma_w launches, one per output phase (h mod
    // sigma_h, w mod sigma_w): within a phase every pixel sees the same set of
    // contributing taps.  wt is [g][R][S][Cg][Kg].
    for (int64_t phh = 0; phh < G.sh; ++phh) {
        for (int64_t phw = 0; phw < G.sw; ++phw) {
            const int64_t mi = phh < G.h ? (G.h - phh + G.sh - 1) / G.sh : 0;
            const int64_t mj = phw < G.w ? (G.w - phw + G.sw - 1) / G.sw : 0;
            if (mi == 0 || mj == 0) continue;
            TNParams p = base;
            p.taps.n = 0;
            const int t = add_phase_taps(p, phh, phw);
            p.mi = (int32_t)mi;
            p.mj = (int32_t)mj;
            p.M = (int32_t)(G.n * mi * mj);
            p.div_mj = make_fastdiv((uint32_t)mj);
            p.div_mi = make_fastdiv((uint32_t)mi);
            p.oi_add = (int32_t)phh;
            p.oj_add = (int32_t)phw;
            p.k_iters = (int32_t)((int64_t(t) * G.kg + 63) / 64);
            if (G.kg % 64 == 0) {
                p.nphase = 1;
                p.ph[0] = phase_of(p.M, mi, mj, phh, phw, 0, t);
                TRY_HIP(launch_igemm_c64(G.dtype, pick_c64_geom(G, p.M, G.cg, (int64_t)t * G.kg), p, pad,
                                         st));
            } else {
                TRY_HIP(launch_igemm_c8(G.dtype, pick_c8(G.cg), p, st));
            }
        }
    }
    return NNCONV_OK;
}

nnconv_status wgrad_fast(const Geom &G, const void *x, const void *dy, float *part,
                         hipStream_t st) {
    const WgPlan pl = plan_wgrad_fast(G);
    if (pl.stem) {
        StemParams sp;
        sp.x = x;
        sp.x_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
        sp.wt = nullptr;
        sp.wt_bytes = 0;
        sp.y = const_cast<void *>(dy);
        sp.y_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
        sp.n = (int32_t)G.n; sp.h = (int32_t)G.h; sp.w = (int32_t)G.w;
        sp.p = (int32_t)G.p; sp.q = (int32_t)G.q;
        sp.r = (int32_t)G.r; sp.s = (int32_t)G.s; sp.sh = (int32_t)G.sh; sp.sw = (int32_t)G.sw;
        sp.ph = (int32_t)G.ph; sp.pw = (int32_t)G.pw;
        sp.c = (int32_t)G.c;
        sp.alpha = 1.0f;
        TRY_HIP(launch_stem_wgrad(G.dtype, sp, part, pl.splits, st));
        return NNCONV_OK;
    }
    if (pl.cfg == WG_HALO) {
        WGHParams hp;
        memset(&hp, 0, sizeof(hp));
        hp.x = x;
        hp.dy = dy;
        hp.ws = part;
        hp.x_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
        hp.dy_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
        hp.h = (int32_t)G.h; hp.w = (int32_t)G.w;
        hp.c_stride = (int32_t)G.c; hp.k_stride = (int32_t)G.k;
        hp.rb = pl.rb;
        hp.blocks_per_img = pl.blocks_per_img;
        hp.nblocks = pl.nblocks;
        hp.blocks_per_split = pl.blocks_per_split;
        hp.splits = pl.splits;
        hp.groups = (int32_t)G.g;
        hp.diag32 = G.diag32;
        TRY_HIP(launch_wgrad_halo(G.dtype, hp, st));
        return NNCONV_OK;
    }
    WGParams p;
    memset(&p, 0, sizeof(p));
    p.x = x;
    p.x_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
    p.dy = dy;
    p.dy_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
    p.ws = part;
    p.h = (int32_t)G.h; p.w = (int32_t)G.w; p.c = (int32_t)G.c; p.k = (int32_t)G.k;
    p.cg = (int32_t)G.cg; p.kg = (int32_t)G.kg;
    p.p = (int32_t)G.p; p.q = (int32_t)G.q; p.npq = (int32_t)(G.n * G.p * G.q);
    p.div_q = make_fastdiv((uint32_t)G.q);
    p.div_pq = make_fastdiv((uint32_t)(G.p * G.q));
    p.div_cg = make_fastdiv((uint32_t)G.cg);
    p.div_s = make_fastdiv((uint32_t)G.s);
    p.sh = (int32_t)G.sh; p.sw = (int32_t)G.sw; p.ph = (int32_t)G.ph; p.pw = (int32_t)G.pw;
    p.dh = (int32_t)G.dh; p.dw = (int32_t)G.dw;
    p.rscg = (int32_t)(G.r * G.s * G.cg);
    p.groups = (int32_t)G.g;
    p.splits = pl.splits;
    p.pix_per_split = pl.pix_per_split;
    TRY_HIP(launch_wgrad_splitk(G.dtype, pl.cfg, p, st));
    return NNCONV_OK;
}

DWParams dw_params(const Geom &G, float alpha) {
    DWParams p;
    memset(&p, 0, sizeof(p));
    p.n = (int32_t)G.n; p.c = (int32_t)G.c; p.h = (int32_t)G.h; p.w = (int32_t)G.w;
    p.p = (int32_t)G.p; p.q = (int32_t)G.q; p.r = (int32_t)G.r; p.s = (int32_t)G.s;
    p.sh = (int32_t)G.sh; p.sw = (int32_t)G.sw; p.ph = (int32_t)G.ph; p.pw = (int32_t)G.pw;
    p.dh = (int32_t)G.dh; p.dw = (int32_t)G.dw;
    p.c8 = (int32_t)(G.c / 8);
    p.cblocks = (int32_t)((G.c / 8 + 7) / 8);
    p.x_bytes = (uint32_t)(G.n * G.h * G.w * G.c * 2);
    p.dy_bytes = (uint32_t)(G.n * G.p * G.q * G.k * 2);
    p.splits = dw_tiled(p, 2) ? dw_tiled_wgrad_splits(p) : dw_wgrad_splits(G);
    const int64_t npq = G.n * G.p * G.q;
    p.pix_per_split = (npq + p.splits - 1) / p.splits;
    p.alpha = alpha;
    return p;
}

// Depthwise passes, either layout.  Every buffer argument is caller-owned
// device memory; ws is laid out by dw_regions.
nnconv_status dw_fwd(const Geom &G, const void *x, const void *w, void *y, float alpha, char *ws,
                     hipStream_t st) {
    const Regions R = dw_regions(G, NNCONV_FWD);
    const void *xn = x;
    void *yn = y;
    if (G.layout == NNCONV_NCHW) {
        TRY_HIP(launch_transpose16(x, ws + R.a, G.n, G.c, G.h * G.w, G.c, st));
        xn = ws + R.a;
        yn = ws + R.c;
    }
    TRY_HIP(launch_depthwise(G.dtype, 0, dw_params(G, alpha), xn, w, yn, st));
    if (G.layout == NNCONV_NCHW)
        return hip_status(launch_transpose16(yn, y, G.n, G.p * G.q, G.k, G.p * G.q, st));
    return NNCONV_OK;
}

nnconv_status dw_dgrad(const Geom &G, const void *dy, const void *w, void *dx, float alpha,
                       char *ws, hipStream_t st) {
    const Regions R = dw_regions(G, NNCONV_DGRAD);
    const void *dyn = dy;
    void *dxn = dx;
    if (G.layout == NNCONV_NCHW) {
        TRY_HIP(launch_transpose16(dy, ws + R.a, G.n, G.k, G.p * G.q, G.k, st));
        dyn = ws + R.a;
        dxn = ws + R.c;
    }
    int32_t *flags = (int32_t *)(ws + R.e);
    TRY_HIP(launch_nonfinite_scan16(w, G.c * G.r * G.s, G.dtype, flags, st));
    TRY_HIP(launch_depthwise(G.dtype, 1, dw_params(G, alpha), dyn, w, dxn, st));
    // the depthwise kernels read dy zero-extended: recompute the border
    // pixels from the definition when a weight is inf or NaN
    const Border B = dgrad_border(G);
    TRY_HIP(launch_dgrad_border(G.dtype, direct_params_cl(G, alpha), dyn, w, dxn, flags,
                                (int32_t)nonfinite_scan16_blocks(G.c * G.r * G.s), B.bt, B.bb,
                                B.bl, B.br, st));
    if (G.layout == NNCONV_NCHW)
        return hip_status(launch_transpose16(dxn, dx, G.n, G.h * G.w, G.c, G.h * G.w, st));
    return NNCONV_OK;
}

nnconv_status dw_wgrad(const Geom &G, const void *x, const void *dy, void *dw, int out_code,
                       float inv_loss_scale, int accumulate, int32_t *flag, char *ws,
                       hipStream_t st) {
    const Regions R = dw_regions(G, NNCONV_WGRAD);
    const void *xn = x, *dyn = dy;
    if (G.layout == NNCONV_NCHW) {
        TRY_HIP(launch_transpose16_pair(x, ws + R.a, G.n, G.c, G.h * G.w, G.c, dy, ws + R.b, G.n,
                                        G.k, G.p * G.q, G.k, st));
        xn = ws + R.a;
        dyn = ws + R.b;
    }
    const DWParams p = dw_params(G, 1.0f);
    float *part = (float *)(ws + R.c);
    TRY_HIP(launch_depthwise(G.dtype, 2, p, xn, dyn, part, st));
    // partials are [split][C][R*S]: the [K][R][S][Cg] order with Cg = 1,
    // which is also [K][Cg][R][S]
    return hip_status(launch_wgrad_reduce(part, p.splits, G.c * G.r * G.s, dw, out_code,
                                          inv_loss_scale, accumulate, flag, 0, 1,
                                          (int32_t)(G.r * G.s), st));
}

nnconv_status sg_fwd(const Geom &G, const void *x, const void *w, void *y, float alpha,
                     char *ws, hipStream_t st) {
    const Geom S = sg_geom(G);
    const Regions R = sg_regions(G, NNCONV_FWD);
    void *wexp = ws + R.d;
    TRY_HIP(launch_expand_group_weights(w, wexp, G.k, (int32_t)(G.r * G.s), (int32_t)G.cg,
                                        (int32_t)SUPER_GROUP, G.layout == NNCONV_NCHW, st));
    void *pack = hring_ws(S, NNCONV_FWD) > 0 ? ws + R.f : nullptr;
    if (G.layout == NNCONV_NHWC) return fwd_fast(S, x, wexp, y, alpha, st, -1, pack);
    void *xt = ws + R.a, *yt = ws + R.c;
    TRY_HIP(launch_transpose16(x, xt, G.n, G.c, G.h * G.w, G.c, st));
    nnconv_status s = fwd_fast(S, xt, wexp, yt, alpha, st, -1, pack);
    if (s != NNCONV_OK) return s;
    return hip_status(launch_transpose16(yt, y, G.n, G.p * G.q, G.k, G.p * G.q, st));
}

nnconv_status sg_dgrad(const Geom &G, const void *dy, const void *w, void *dx, float alpha,
                       char *ws, hipStream_t st) {
    const Geom S = sg_geom(G);
    const Regions R = sg_regions(G, NNCONV_DGRAD);
    void *wexp = ws + R.d, *wt = ws + R.b;
    TRY_HIP(launch_expand_group_weights(w, wexp, G.k, (int32_t)(G.r * G.s), (int32_t)G.cg,
                                        (int32_t)SUPER_GROUP, G.layout == NNCONV_NCHW, st));
    // [g][Kg][R*S*Cg] -> [g][R*S*Cg][Kg] for the super-groups
    TRY_HIP(launch_transpose16(wexp, wt, S.g, S.kg, S.r * S.s * S.cg, S.kg, st));
    void *pack = hring_ws(S, NNCONV_DGRAD) > 0 ? ws + R.f : nullptr;
    if (G.layout == NNCONV_NHWC) return dgrad_fast(S, dy, wt, dx, alpha, st, -1, pack);
    void *dyt = ws + R.a, *dxt = ws + R.c;
    TRY_HIP(launch_transpose16(dy, dyt, G.n, G.k, G.p * G.q, G.k, st));
    nnconv_status s = dgrad_fast(S, dyt, wt, dxt, alpha, st, -1, pack);
    if (s != NNCONV_OK) return s;
    return hip_status(launch_transpose16(dxt, dx, G.n, G.h * G.w, G.c, G.h * G.w, st));
}

nnconv_status sg_wgrad(const Geom &G, const void *x, const void *dy, void *dw, int out_code,
                       float inv_loss_scale, int accumulate, int32_t *flag, char *ws,
                       hipStream_t st) {
    const Geom S = sg_geom(G);
    const Regions R = sg_regions(G, NNCONV_WGRAD);
    const void *xn = x, *dyn = dy;
    if (G.layout == NNCONV_NCHW) {
        void *xt = ws + R.a, *dyt = ws + R.b;
        TRY_HIP(launch_transpose16_pair(x, xt, G.n, G.c, G.h * G.w, G.c, dy, dyt, G.n, G.k,
                                        G.p * G.q, G.k, st));
        xn = xt;
        dyn = dyt;
    }
    float *part = (float *)(ws + R.c);
    nnconv_status s = wgrad_fast(S, xn, dyn, part, st);
    if (s != NNCONV_OK) return s;
    const WgPlan pl = plan_wgrad_fast(S);
    return hip_status(launch_wgrad_reduce_diag(part, pl.splits, G.k, (int32_t)(G.r * G.s),
                                               (int32_t)G.cg, (int32_t)SUPER_GROUP, dw, out_code,
                                               inv_loss_scale, accumulate, flag,
                                               G.layout == NNCONV_NCHW, st));
}

}  // namespace

// ---------------------------------------------------------------------------
// exported entry points
// ---------------------------------------------------------------------------

NNCONV_API int32_t nnconv_version(void) { return NNCONV_VERSION; }

NNCONV_API int32_t nnconv_last_hip_error(void) { return last_hip_error; }

NNCONV_API const char *nnconv_status_string(nnconv_status s) {
    switch (s) {
        case NNCONV_OK: return "ok";
        case NNCONV_ERR_INVALID_ARG: return "invalid argument";
        case NNCONV_ERR_UNSUPPORTED: return "unsupported";
        case NNCONV_ERR_WORKSPACE: return "workspace too small";
        case NNCONV_ERR_MISALIGNED: return "misaligned pointer";
        case NNCONV_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

NNCONV_API nnconv_status nnconv_output_dims(const nnconv_desc *desc, int32_t *p, int32_t *q) {
    if (!p || !q) return NNCONV_ERR_INVALID_ARG;
    Geom G;
    nnconv_status st = validate(desc, &G);
    if (st != NNCONV_OK) return st;
    *p = (int32_t)G.p;
    *q = (int32_t)G.q;
    return NNCONV_OK;
}

NNCONV_API nnconv_status nnconv_workspace_size(const nnconv_desc *desc, nnconv_pass pass,
                                               size_t *bytes) {
    if (!bytes) return NNCONV_ERR_INVALID_ARG;
    if (pass != NNCONV_FWD && pass != NNCONV_DGRAD && pass != NNCONV_WGRAD)
        return NNCONV_ERR_INVALID_ARG;
    Geom G;
    nnconv_status st = validate(desc, &G);
    if (st != NNCONV_OK) return st;
    *bytes = workspace_bytes(G, pass);
    return NNCONV_OK;
}

static nnconv_status check_ws(const Geom &G, nnconv_pass pass, const void *ws, size_t ws_bytes) {
    const size_t need = workspace_bytes(G, pass);
    if (ws_bytes < need) return NNCONV_ERR_WORKSPACE;
    if (need > 0 && !ws) return NNCONV_ERR_INVALID_ARG;
    return NNCONV_OK;
}

// Whether a forced tile can run this call: a tile of the 64-channel-slice
// kernel other than the block-diagonal one, on a dense call that takes that
// kernel with its operands as given.
bool tile_ok(int tile) {
    return (tile >= C64_256x256 && tile <= C64R_256x64 && tile != C64D_128x64) ||
           halo_tile(tile);
}

static nnconv_status fwd_impl(const nnconv_desc *desc, const void *x, const void *w, void *y,
                              float alpha, void *ws, size_t ws_bytes, void *hip_stream,
                              int tile) {
    Geom G;
    nnconv_status st = validate(desc, &G);
    if (st != NNCONV_OK) return st;
    if (!x || !w || !y) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(x, 2) || !aligned(w, 2) || !aligned(y, 2)) return NNCONV_ERR_MISALIGNED;
    if ((st = check_ws(G, NNCONV_FWD, ws, ws_bytes)) != NNCONV_OK) return st;
    hipStream_t s = (hipStream_t)hip_stream;
    if (tile >= 0) {
        const bool dense = !dw_shape(G) && !sg_shape(G) && fast_shape(G) && c64_fwd_shape(G) &&
                           aligned(x, 16) && aligned(w, 16) && aligned(y, 16) &&
                           (G.layout == NNCONV_NHWC || aligned(ws, 16)) &&
                           (!halo_tile(tile) || !hring_cfg(tile - HALO_TILE0) || aligned(ws, 16));
        if (!tile_ok(tile) || !dense || (halo_tile(tile) && !halo_geom(G, tile, G.cg)))
            return NNCONV_ERR_UNSUPPORTED;
    }
    clear_stale_error();
    if (dw_shape(G)) {
        if (!aligned(x, 16) || !aligned(w, 2) || !aligned(y, 16) || !aligned(ws, 16))
            return hip_status(launch_direct_fwd(G.dtype, direct_params(G, alpha), x, w, y, s));
        return dw_fwd(G, x, w, y, alpha, (char *)ws, s);
    }
    if (sg_shape(G) && fast_shape(sg_geom(G)) && aligned(x, 16) && aligned(y, 16) &&
        aligned(ws, 16))
        return sg_fwd(G, x, w, y, alpha, (char *)ws, s);
    const bool fast = fast_pass(G, NNCONV_FWD) && aligned(x, 16) && aligned(w, 16) && aligned(y, 16) &&
                      (G.layout == NNCONV_NHWC || aligned(ws, 16));
    if (!fast) return hip_status(launch_direct_fwd(G.dtype, direct_params(G, alpha), x, w, y, s));
    const Regions R = fast_regions(G, NNCONV_FWD);
    char *base = (char *)ws;
    void *pack = (hring_ws(G, NNCONV_FWD) > 0 && ws && aligned(ws, 16)) ? base + R.f : nullptr;
    if (G.layout == NNCONV_NHWC) return fwd_fast(G, x, w, y, alpha, s, tile, pack);
    void *xt = base + R.a, *wt = base + R.b, *yt = base + R.c;
    TRY_HIP(launch_transpose16_pair(x, xt, G.n, G.c, G.h * G.w, G.c, w, wt, G.k, G.cg, G.r * G.s,
                                    G.cg, s));
    if ((st = fwd_fast(G, xt, wt, yt, alpha, s, tile, pack)) != NNCONV_OK) return st;
    return hip_status(launch_transpose16(yt, y, G.n, G.p * G.q, G.k, G.p * G.q, s));
}

NNCONV_API nnconv_status nnconv_fwd(const nnconv_desc *desc, const void *x, const void *w, void *y,
                                    float alpha, void *ws, size_t ws_bytes, void *hip_stream) {
    return fwd_impl(desc, x, w, y, alpha, ws, ws_bytes, hip_stream, -1);
}

NNCONV_API nnconv_status nnconv_fwd_tile(const nnconv_desc *desc, const void *x, const void *w,
                                         void *y, float alpha, void *ws, size_t ws_bytes,
                                         void *hip_stream, int32_t tile) {
    if (tile < 0) return NNCONV_ERR_INVALID_ARG;
    return fwd_impl(desc, x, w, y, alpha, ws, ws_bytes, hip_stream, tile);
}

static nnconv_status dgrad_impl(const nnconv_desc *desc, const void *dy, const void *w,
                                void *dx, float alpha, void *ws, size_t ws_bytes,
                                void *hip_stream, int tile) {
    Geom G;
    nnconv_status st = validate(desc, &G);
    if (st != NNCONV_OK) return st;
    if (!dy || !w || !dx) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(dy, 2) || !aligned(w, 2) || !aligned(dx, 2)) return NNCONV_ERR_MISALIGNED;
    if ((st = check_ws(G, NNCONV_DGRAD, ws, ws_bytes)) != NNCONV_OK) return st;
    hipStream_t s = (hipStream_t)hip_stream;
    if (tile >= 0) {
        const bool dense = !dw_shape(G) && !sg_shape(G) && fast_shape(G) && c64_dgrad_shape(G) &&
                           aligned(dy, 16) && aligned(w, 16) && aligned(dx, 16) &&
                           aligned(ws, 16);
        if (!tile_ok(tile) || !dense || (halo_tile(tile) && !halo_geom(G, tile, G.kg)))
            return NNCONV_ERR_UNSUPPORTED;
    }
    clear_stale_error();
    if (dw_shape(G)) {
        if (!aligned(dy, 16) || !aligned(w, 2) || !aligned(dx, 16) || !aligned(ws, 16))
            return hip_status(
                launch_direct_dgrad(G.dtype, direct_params(G, alpha), dy, w, dx, s));
        return dw_dgrad(G, dy, w, dx, alpha, (char *)ws, s);
    }
    if (sg_shape(G) && fast_shape(sg_geom(G)) && aligned(dy, 16) && aligned(dx, 16) &&
        aligned(ws, 16))
        return sg_dgrad(G, dy, w, dx, alpha, (char *)ws, s);
    const bool fast = fast_shape(G) && aligned(dy, 16) && aligned(w, 16) && aligned(dx, 16) &&
                      aligned(ws, 16);
    if (!fast)
        return hip_status(launch_direct_dgrad(G.dtype, direct_params(G, alpha), dy, w, dx, s));
    const Regions R = fast_regions(G, NNCONV_DGRAD);
    char *base = (char *)ws;
    void *wt = base + R.b;
    const void *wkrsc = w;
    const void *dyn = dy;
    void *dxn = dx;
    if (G.layout == NNCONV_NCHW) {
        void *tmp = base + R.d;
        void *dyt = base + R.a;
        TRY_HIP(launch_transpose16_pair(w, tmp, G.k, G.cg, G.r * G.s, G.cg, dy, dyt, G.n, G.k,
                                        G.p * G.q, G.k, s));
        wkrsc = tmp;
        dyn = dyt;
        dxn = base + R.c;
    }
    // [g][Kg][R*S*Cg] -> [g][R*S*Cg][Kg], noting any inf or NaN weight
    int32_t *flags = (int32_t *)(base + R.e);
    TRY_HIP(launch_transpose16_scan(wkrsc, wt, G.g, G.kg, G.r * G.s * G.cg, G.kg, G.dtype, flags,
                                    s));
    void *pack = hring_ws(G, NNCONV_DGRAD) > 0 ? base + R.f : nullptr;
    if ((st = dgrad_fast(G, dyn, wt, dxn, alpha, s, tile, pack)) != NNCONV_OK) return st;
    // the implicit-GEMM kernels read dy zero-extended at every tap of a
    // stride phase: recompute the border pixels from the definition when a
    // weight is inf or NaN (with finite weights the kernel exits at once)
    const Border B = dgrad_border(G);
    TRY_HIP(launch_dgrad_border(G.dtype, direct_params_cl(G, alpha), dyn, w, dxn, flags,
                                (int32_t)transpose16_blocks(G.g, G.r * G.s * G.cg, G.kg), B.bt,
                                B.bb, B.bl, B.br, s));
    if (G.layout == NNCONV_NCHW)
        return hip_status(launch_transpose16(dxn, dx, G.n, G.h * G.w, G.c, G.h * G.w, s));
    return NNCONV_OK;
}

NNCONV_API nnconv_status nnconv_dgrad(const nnconv_desc *desc, const void *dy, const void *w,
                                      void *dx, float alpha, void *ws, size_t ws_bytes,
                                      void *hip_stream) {
    return dgrad_impl(desc, dy, w, dx, alpha, ws, ws_bytes, hip_stream, -1);
}

NNCONV_API nnconv_status nnconv_dgrad_tile(const nnconv_desc *desc, const void *dy,
                                           const void *w, void *dx, float alpha, void *ws,
                                           size_t ws_bytes, void *hip_stream, int32_t tile) {
    if (tile < 0) return NNCONV_ERR_INVALID_ARG;
    return dgrad_impl(desc, dy, w, dx, alpha, ws, ws_bytes, hip_stream, tile);
}

// Argument checks of the backward-weight pass that need no workspace.
static nnconv_status wgrad_check(const nnconv_desc *desc, const void *x, const void *dy,
                                 const void *dw, int32_t dw_dtype, int32_t accumulate,
                                 const int32_t *overflow_flag, Geom *G) {
    nnconv_status st = validate(desc, G);
    if (st != NNCONV_OK) return st;
    if (!x || !dy || !dw) return NNCONV_ERR_INVALID_ARG;
    if (dw_dtype != NNCONV_F32 && dw_dtype != NNCONV_F16 && dw_dtype != NNCONV_BF16)
        return NNCONV_ERR_INVALID_ARG;
    if (dw_dtype != NNCONV_F32 && dw_dtype != G->dtype) return NNCONV_ERR_UNSUPPORTED;
    if (accumulate != 0 && accumulate != 1) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(x, 2) || !aligned(dy, 2) || !aligned(dw, dw_dtype == NNCONV_F32 ? 4 : 2) ||
        (overflow_flag && !aligned(overflow_flag, 4)))
        return NNCONV_ERR_MISALIGNED;
    return NNCONV_OK;
}

// The backward-weight pass on a checked geometry with a workspace of at
// least workspace_bytes(G, NNCONV_WGRAD) bytes.
static nnconv_status wgrad_run(const Geom &G, const void *x, const void *dy, void *dw,
                               int32_t dw_dtype, float inv_loss_scale, int32_t accumulate,
                               int32_t *overflow_flag, void *ws, void *hip_stream) {
    nnconv_status st;
    hipStream_t s = (hipStream_t)hip_stream;
    clear_stale_error();
    const int out_code = dw_dtype == NNCONV_F32 ? 2 : (dw_dtype == NNCONV_F16 ? 0 : 1);
    const int64_t count = G.k * G.r * G.s * G.cg;
    const int kcrs = G.layout == NNCONV_NCHW;
    if (dw_shape(G) && aligned(x, 16) && aligned(dy, 16) && aligned(ws, 16))
        return dw_wgrad(G, x, dy, dw, out_code, inv_loss_scale, accumulate, overflow_flag,
                        (char *)ws, s);
    if (sg_shape(G) && fast_shape(sg_geom(G)) && aligned(x, 16) && aligned(dy, 16) &&
        aligned(ws, 16))
        return sg_wgrad(G, x, dy, dw, out_code, inv_loss_scale, accumulate, overflow_flag,
                        (char *)ws, s);
    const bool fast = fast_pass(G, NNCONV_WGRAD) && aligned(x, 16) && aligned(dy, 16) &&
                      aligned(ws, 16);
    if (!fast) {
        const int32_t splits = plan_wgrad_direct_splits(G);
        float *part = (float *)ws;
        TRY_HIP(launch_direct_wgrad(G.dtype, direct_params(G, 1.0f), x, dy, part, splits, s));
        return hip_status(launch_wgrad_reduce(part, splits, count, dw, out_code, inv_loss_scale,
                                              accumulate, overflow_flag, kcrs, (int32_t)G.cg,
                                              (int32_t)(G.r * G.s), s));
    }
    const Regions R = fast_regions(G, NNCONV_WGRAD);
    char *base = (char *)ws;
    const void *xn = x, *dyn = dy;
    if (G.layout == NNCONV_NCHW) {
        void *xt = base + R.a, *dyt = base + R.b;
        TRY_HIP(launch_transpose16_pair(x, xt, G.n, G.c, G.h * G.w, G.c, dy, dyt, G.n, G.k,
                                        G.p * G.q, G.k, s));
        xn = xt;
        dyn = dyt;
    }
    float *part = (float *)(base + R.c);
    if ((st = wgrad_fast(G, xn, dyn, part, s)) != NNCONV_OK) return st;
    const WgPlan pl = plan_wgrad_fast(G);
    return hip_status(launch_wgrad_reduce(part, pl.splits, count, dw, out_code, inv_loss_scale,
                                          accumulate, overflow_flag, kcrs, (int32_t)G.cg,
                                          (int32_t)(G.r * G.s), s));
}

NNCONV_API nnconv_status nnconv_wgrad(const nnconv_desc *desc, const void *x, const void *dy,
                                      void *dw, int32_t dw_dtype, float inv_loss_scale,
                                      int32_t accumulate, int32_t *overflow_flag, void *ws,
                                      size_t ws_bytes, void *hip_stream) {
    Geom G;
    nnconv_status st = wgrad_check(desc, x, dy, dw, dw_dtype, accumulate, overflow_flag, &G);
    if (st != NNCONV_OK) return st;
    if ((st = check_ws(G, NNCONV_WGRAD, ws, ws_bytes)) != NNCONV_OK) return st;
    return wgrad_run(G, x, dy, dw, dw_dtype, inv_loss_scale, accumulate, overflow_flag, ws,
                     hip_stream);
}

// ---------------------------------------------------------------------------
// backward-weight without a caller workspace
// ---------------------------------------------------------------------------

// Library-owned scratch of the allocation-free entry point: a file-scope
// device array, so each GPU the library runs on holds one copy (its
// NNCONV_NOALLOC_WS_BYTES stay allocated until the process ends).  The
// array's name is a host-side stand-in: host code uses only the device
// address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[NNCONV_NOALLOC_WS_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::once_flag scratch_once[MAX_DEVICES];
void *scratch_ptr[MAX_DEVICES];
hipError_t scratch_err[MAX_DEVICES];

// Device address of the current device's scratch copy, looked up once per
// device (with that device current) and kept.
hipError_t device_scratch(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::call_once(scratch_once[dev], [dev] {
        void *p = nullptr;
        scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        scratch_ptr[dev] = p;
    });
    if (scratch_err[dev] != hipSuccess) return scratch_err[dev];
    if (!scratch_ptr[dev]) return hipErrorInvalidSymbol;
    *out = scratch_ptr[dev];
    return hipSuccess;
}
}  // namespace

NNCONV_API nnconv_status nnconv_wgrad_noalloc(const nnconv_desc *desc, const void *x,
                                              const void *dy, void *dw, int32_t dw_dtype,
                                              float inv_loss_scale, int32_t accumulate,
                                              int32_t *overflow_flag, void *hip_stream) {
    Geom G;
    nnconv_status st = wgrad_check(desc, x, dy, dw, dw_dtype, accumulate, overflow_flag, &G);
    if (st != NNCONV_OK) return st;
    if (workspace_bytes(G, NNCONV_WGRAD) > (size_t)NNCONV_NOALLOC_WS_BYTES)
        return NNCONV_ERR_WORKSPACE;
    void *ws = nullptr;
    const hipError_t e = device_scratch(&ws);
    if (e != hipSuccess) return hip_status(e);
    return wgrad_run(G, x, dy, dw, dw_dtype, inv_loss_scale, accumulate, overflow_flag, ws,
                     hip_stream);
}

// ---------------------------------------------------------------------------
// transforms
// ---------------------------------------------------------------------------

NNCONV_API nnconv_status nnconv_nchw_to_nhwc(const void *src, void *dst, int32_t n, int32_t c,
                                             int32_t h, int32_t w, int32_t c_pad,
                                             void *hip_stream) {
    if (!src || !dst || n < 1 || c < 1 || h < 1 || w < 1 || c_pad < c)
        return NNCONV_ERR_INVALID_ARG;
    if (!aligned(src, 2) || !aligned(dst, 2)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(launch_transpose16(src, dst, n, c, (int64_t)h * w, c_pad,
                                         (hipStream_t)hip_stream));
}

NNCONV_API nnconv_status nnconv_nhwc_to_nchw(const void *src, void *dst, int32_t n, int32_t c,
                                             int32_t h, int32_t w, void *hip_stream) {
    if (!src || !dst || n < 1 || c < 1 || h < 1 || w < 1) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(src, 2) || !aligned(dst, 2)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(launch_transpose16(src, dst, n, (int64_t)h * w, c, (int64_t)h * w,
                                         (hipStream_t)hip_stream));
}

NNCONV_API nnconv_status nnconv_pad_channels(const void *src, void *dst, int64_t rows, int32_t c,
                                             int32_t c_pad, void *hip_stream) {
    if (!src || !dst || rows < 1 || c < 1 || c_pad < c) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(src, 2) || !aligned(dst, 2)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(launch_pad_channels16(src, dst, rows, c, c_pad, (hipStream_t)hip_stream));
}

NNCONV_API nnconv_status nnconv_weight_kcrs_to_krsc(const void *src, void *dst, int32_t k,
                                                    int32_t cg, int32_t r, int32_t s,
                                                    int32_t cg_pad, void *hip_stream) {
    if (!src || !dst || k < 1 || cg < 1 || r < 1 || s < 1 || cg_pad < cg)
        return NNCONV_ERR_INVALID_ARG;
    if (!aligned(src, 2) || !aligned(dst, 2)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(
        launch_transpose16(src, dst, k, cg, (int64_t)r * s, cg_pad, (hipStream_t)hip_stream));
}

NNCONV_API nnconv_status nnconv_weight_krsc_to_kcrs(const void *src, void *dst, int32_t k,
                                                    int32_t cg, int32_t r, int32_t s,
                                                    void *hip_stream) {
    if (!src || !dst || k < 1 || cg < 1 || r < 1 || s < 1) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(src, 2) || !aligned(dst, 2)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(launch_transpose16(src, dst, k, (int64_t)r * s, cg, (int64_t)r * s,
                                         (hipStream_t)hip_stream));
}

// ---------------------------------------------------------------------------
// training-step pieces: dynamic loss scaler and fp32 master-weight update
// ---------------------------------------------------------------------------

NNCONV_API nnconv_status nnconv_loss_scaler_init(nnconv_loss_scaler *state, float initial_scale,
                                                 float factor, int32_t interval,
                                                 void *hip_stream) {
    if (!state || interval < 0) return NNCONV_ERR_INVALID_ARG;
    if (!(initial_scale > 0.0f) || !(factor > 0.0f) || !__builtin_isfinite(initial_scale) ||
        !__builtin_isfinite(factor))
        return NNCONV_ERR_INVALID_ARG;
    if (!aligned(state, 4)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(
        launch_loss_scaler_init(state, initial_scale, factor, interval, (hipStream_t)hip_stream));
}

NNCONV_API nnconv_status nnconv_loss_scaler_update(nnconv_loss_scaler *state,
                                                   int32_t *overflow_flag, void *hip_stream) {
    if (!state || !overflow_flag) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(state, 4) || !aligned(overflow_flag, 4)) return NNCONV_ERR_MISALIGNED;
    clear_stale_error();
    return hip_status(launch_loss_scaler_update(state, overflow_flag, (hipStream_t)hip_stream));
}

NNCONV_API nnconv_status nnconv_sgd_update(int64_t count, float *master, float *momentum,
                                           void *w16, int32_t w16_dtype, const float *grad,
                                           const nnconv_loss_scaler *state,
                                           const int32_t *overflow_flag, float lr,
                                           float momentum_coef, float weight_decay,
                                           void *hip_stream) {
    if (count < 0 || count > MAX_ELEMS || !master || !momentum || !grad)
        return NNCONV_ERR_INVALID_ARG;
    if (w16 && w16_dtype != NNCONV_F16 && w16_dtype != NNCONV_BF16) return NNCONV_ERR_INVALID_ARG;
    if (!aligned(master, 4) || !aligned(momentum, 4) || !aligned(grad, 4) ||
        (w16 && !aligned(w16, 2)) || (state && !aligned(state, 4)) ||
        (overflow_flag && !aligned(overflow_flag, 4)))
        return NNCONV_ERR_MISALIGNED;
    if (count == 0) return NNCONV_OK;
    clear_stale_error();
    return hip_status(launch_sgd_update(count, master, momentum, w16, w16_dtype, grad, state,
                                        overflow_flag, lr, momentum_coef, weight_decay,
                                        (hipStream_t)hip_stream));
}
