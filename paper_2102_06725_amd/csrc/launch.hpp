// launch.hpp -- host-side interface between the C-ABI shim and the kernel
// translation units.  Plain structs only; every launcher queues work on the
// given stream and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "nnconv.h"

namespace nnconv {

constexpr int MAX_TAPS = 64;

// Filter taps visited by one implicit-GEMM launch.  Tap t moves the A-image
// read position by (dh[t], dw[t]) and starts at element boff[t] of a B row.
struct TapTable {
    int32_t n;
    int32_t dh[MAX_TAPS];
    int32_t dw[MAX_TAPS];
    int32_t boff[MAX_TAPS];
};

// One implicit GEMM  out[row, col] = alpha * sum_{tap, ch} A(row, tap, ch) * B[col, tap, ch]
// with channel-last operands, used for the forward pass (A = x, B = w) and
// for one stride phase of the backward-data pass (A = dy, B = w transposed
// to [R][S][Cg][Kg] per group).
//
// Row m decodes to (image n, i, j) with i < mi, j < mj.  A is read at pixel
// (i*ai_mul + ai_add + dh[t], j*aj_mul + aj_add + dw[t]) of image n (zero
// outside a_h x a_w), channels g*a_cg_ofs + ch.  B row `col` of group g
// starts at element g*b_g_ofs + col*b_ld.  The result goes to pixel
// (i*oi_mul + oi_add, j*oj_mul + oj_add) of an o_h x o_w image with o_c
// channels, channel g*o_cg_ofs + col.
// One output phase of a 64-channel-slice launch: rows m < M decode to
// (image n, i < mi, j < mj); the output pixel is (i*oi_mul + oi_add,
// j*oj_mul + oj_add); the phase uses taps [tap_start, tap_start + tap_count)
// of the tap table.  The forward pass has one phase; backward-data has one per
// stride phase, all in a single launch.
struct TNPhase {
    int32_t M, mi, mj;
    FastDiv div_mj, div_mi;
    int32_t oi_add, oj_add;
    int32_t tap_start, tap_count;
    int32_t tiles_m, block_start;  // filled by the launcher
};
constexpr int MAX_PHASES = 4;

struct TNParams {
    const void *a;
    uint32_t a_bytes;
    const void *b;
    uint32_t b_bytes;
    void *out;
    uint32_t o_bytes;     // size of the output tensor in bytes
    int32_t M;
    int32_t mi, mj;
    FastDiv div_mj, div_mi;
    int32_t a_h, a_w, a_c, a_cg_ofs;
    int32_t ai_mul, ai_add, aj_mul, aj_add;
    int32_t cr;            // reduction channels per tap (multiple of 8)
    FastDiv div_crv;       // division by cr / 8
    int32_t k_iters;       // ceil(taps * cr / 64)
    int32_t ncols;         // output columns per group (multiple of 8)
    int32_t b_ld, b_g_ofs;
    int32_t o_h, o_w, o_c, o_cg_ofs;
    int32_t oi_mul, oi_add, oj_mul, oj_add;
    float alpha;
    int32_t groups;
    int32_t tiles_m, tiles_n;  // per group; filled by the launcher
    TapTable taps;
    int32_t nphase;            // igemm_c64 only: phases in ph[]
    TNPhase ph[MAX_PHASES];
};

// Any cr (a multiple of 8): the reduction is cut into slices of 32 elements
// built from 8-channel chunks of consecutive taps (recomputes k_iters for
// its own slice depth).
enum C8Config { C8_128x128 = 0, C8_256x64 = 1, C8_256x128 = 2 };
hipError_t launch_igemm_c8(int dtype, C8Config cfg, TNParams &p, hipStream_t st);

// cr % 64 == 0: 64-channel slices of one tap (k_iters is derived from the
// taps).  pad: some (row, tap) pairs fall outside the A image and must read
// zeros.
enum C64Config { C64_256x256 = 0,   // 8 waves, 64-element slices, 2 stages
                 C64_128x128 = 1,   // 4 waves, 64-element slices, 2 stages
                 C64S_128x128 = 2,  // single stage (several workgroups per CU)
                 C64S_128x64 = 3,
                 C64W_256x256 = 4,    // 16 waves of 64x64, 2 stages
                 C64D_128x64 = 5,     // C64S_128x64 for block-diagonal 64x64 weights
                                      // (32x32 blocks): half the k-steps per wave
                 // LDS ring of 32-element slices with register-prefetched
                 // fragments (one wave per SIMD for 256x256: 128x128 per wave)
                 C64R_256x256 = 6,    // 4 waves of 128x128, 4 stages (128 KB)
                 C64R_256x128 = 7,    // 4 waves of 128x64, 3 stages (72 KB), 2 per CU
                 C64R_256x64 = 8 };   // 4 waves of 64x64, 4 stages (80 KB), 2 per CU
hipError_t launch_igemm_c64(int dtype, C64Config cfg, TNParams &p, bool pad, hipStream_t st);

// Halo staging for stride-1 "same" geometries (igemm_halo.hip): single
// phase, one group, cr % 64 == 0, A image of the output's size, at most 32
// taps whose raster shifts span at most HALO_SPAN pixels (3x3 filters with
// padding 1 on images up to 63 pixels wide).  The single-slice
// register-weight tile also takes groups of 64 reduction channels into 64
// output columns (grouped convolution run as 64-channel super-groups).
constexpr int HALO_SPAN = 128;
enum HaloConfig { HALO_256x64 = 0,      // 4 waves of 64x64
                  HALO_256x128 = 1,     // 4 waves of 128x64
                  HALO_256x64_2T = 2,   // 256x64 with the B tiles of two taps per step
                  // igemm_hring.hip: weight fragments from L2 into registers,
                  // double-buffered halo (one workgroup per CU)
                  HALO_R256x128 = 3,    // 4 waves of 128x64, taps within 64 raster positions
                  HALO_R128x256 = 4,    // 4 waves of 128x64 side by side, taps within 128
                  HALO_R224x256 = 5,    // 4 waves of 224x64 side by side, taps within 32
                  HALO_R256x64S = 6 };  // 4 waves of 64x64, single 64-channel slice
                                        // (cr == 64), three workgroups per CU
// the register-weight configurations are the ones from HALO_R256x128 on
inline bool hring_config(int cfg) { return cfg >= HALO_R256x128 && cfg <= HALO_R256x64S; }
// grouped: also accept p.groups > 1 with groups of cr reduction channels
// into ncols output columns, side by side in the A and output pixels
bool halo_supported(const TNParams &p, bool grouped = false);
// largest minus smallest raster shift of the taps of phase 0
int halo_tap_span(const TNParams &p);
// raster span of the taps the configuration's halo buffer holds
int halo_cfg_span(HaloConfig cfg);
// whether configuration cfg runs p (geometry, tap count and span)
bool halo_cfg_supported(const TNParams &p, HaloConfig cfg);
// hipErrorInvalidValue when !halo_cfg_supported(p, cfg); `pack` is used by
// the register-weight configurations only (see launch_igemm_hring).  diag32:
// the per-tap 64x64 weight blocks are block-diagonal in 32x32 blocks
// (super-groups of groups of at most 32 channels); the single-slice tile then
// skips the zero blocks, the others ignore it.
hipError_t launch_igemm_halo(int dtype, HaloConfig cfg, TNParams &p, void *pack, bool diag32,
                             hipStream_t st);
// The register-weight halo tiles (igemm_hring.hip) take 3x3 filters (9
// taps) only, HALO_R256x64S a single 64-channel slice (cr == 64) too, and
// it alone more than one group (each of 64 output columns).  They read the
// B operand packed in fragment order: `pack` is caller-provided device
// memory of hring_pack_bytes(ncols, cr, groups) bytes, which
// launch_igemm_hring fills from p.b before the GEMM.
constexpr int HRING_TAPS = 9;
bool hring_supported(const TNParams &p, int span, bool grouped = false);
size_t hring_pack_bytes(int64_t ncols, int64_t cr, int64_t groups = 1);
hipError_t launch_igemm_hring(int dtype, HaloConfig cfg, TNParams &p, void *pack, bool diag32,
                              hipStream_t st);

// Forward pass for 8-channel (16-byte) channel-last pixels, 64 output
// channels, groups 1, dilation 1 and a compiled filter size / stride (the
// stem: 7x7, stride 2).  x [n][h][w][8], wt [64][r][s][8], y [n][p][q][64].
struct StemParams {
    const void *x;
    uint32_t x_bytes;
    const void *wt;
    uint32_t wt_bytes;
    void *y;
    uint32_t y_bytes;
    int32_t n, h, w, p, q;
    int32_t r, s, sh, sw, ph, pw;
    int32_t c;                  // channels per pixel: 8, or 4 (stem4_supported)
    float alpha;
};
bool stem_fwd_supported(int r, int s, int sh, int sw);
// 4-channel pixels: the same filter with an odd left padding and an even
// image width
bool stem4_supported(const StemParams &p);
// cus: workgroups to launch at most (one per CU; the kernel loops over tiles)
hipError_t launch_stem_fwd(int dtype, const StemParams &p, int cus, hipStream_t st);
// Backward-weight partials for the same shapes: y holds dy; splits
// workgroups each write part[split][64][r*s*c] (no loss-scale step); with
// 4-channel pixels splits is even and splits / 2 workgroups write two each.
hipError_t launch_stem_wgrad(int dtype, const StemParams &p, float *part, int splits,
                             hipStream_t st);

// Backward-weight split-K partial sums:
//   ws[split][k][j] = sum over pixels of this split of dy[pix, k] * xcol[pix, j]
// with j = (r*S + s)*Cg + c (the [K][R][S][Cg] order) and channel-last x, dy.
struct WGParams {
    const void *x;
    uint32_t x_bytes;
    const void *dy;
    uint32_t dy_bytes;
    float *ws;
    int32_t h, w, c, k;         // x height/width/channels, dy channels
    int32_t cg, kg;
    int32_t p, q, npq;
    FastDiv div_q, div_pq, div_cg, div_s;
    int32_t sh, sw, ph, pw, dh, dw;
    int32_t rscg;
    int32_t groups, splits, pix_per_split;
    int32_t tiles_m, tiles_n;   // filled by the launcher
};

enum WGConfig { WG_128x128 = 0, WG_64x128 = 1, WG_256x256 = 2, WG_128x128S = 3,
                WG_64x128D = 4,  // WG_64x128 for block-diagonal super-group gradients
                WG_HALO = 5 };   // wgrad_halo.hip (3x3 stride-1 "same", 64 -> 64 channels)

// Pixel ranges of pix_per_split (a multiple of 32) pixels each.
hipError_t launch_wgrad_splitk(int dtype, WGConfig cfg, WGParams &p, hipStream_t st);

// Backward-weight of a 3x3 stride-1 convolution with padding 1 and groups of
// 64 input and 64 output channels (wgrad_halo.hip): blocks of rb whole image
// rows (rb * w a multiple of 16, at most 128 pixels, wgh_slots(rb, w) at
// most WGH_MAX_SLOTS), blocks_per_split consecutive blocks per workgroup,
// workgroup (split, group) writing rows group * 64 .. + 63 of
// ws[split][groups * 64][9 * 64] (fp32, columns (tap, c)).  diag32: the
// groups are super-groups of groups of at most 32 channels, whose gradient
// is block-diagonal in 32x32 blocks: only those blocks are computed and
// written (the rest of each row is left as it was).
constexpr int WGH_MAX_SLOTS = 3392;
// 16-byte LDS slots a block of rb rows of a w-wide image stages
int wgh_slots(int rb, int w);
struct WGHParams {
    const void *x;
    const void *dy;
    float *ws;
    uint32_t x_bytes, dy_bytes;
    int32_t h, w;                  // image size (input = output)
    int32_t c_stride, k_stride;    // channels per pixel of x and dy
    int32_t rb, blocks_per_img, nblocks, blocks_per_split, splits;
    int32_t groups;                // of 64 channels, side by side in x and dy pixels
    int32_t diag32;
};
hipError_t launch_wgrad_halo(int dtype, const WGHParams &p, hipStream_t st);

// dw[e'] = (accumulate ? dw[e'] : 0) + inv_scale * sum_{s < splits} ws[s][e]
// over e < count = K * R*S*Cg; e' = e for [K][R][S][Cg] output, or the
// matching [K][Cg][R][S] index when kcrs != 0.  Stores 1 into *flag when a
// final value is not finite.
hipError_t launch_wgrad_reduce(const float *ws, int32_t splits, int64_t count, void *dw,
                               int out_dtype, float inv_scale, int accumulate, int32_t *flag,
                               int kcrs, int32_t cg, int32_t rs, hipStream_t st);

// Direct (one thread per output) kernels for any valid geometry and either
// layout; element offsets are given by strides.
struct DirectParams {
    int32_t n, c, h, w, k, r, s, p, q;
    int32_t sh, sw, ph, pw, dh, dw, groups, cg, kg;
    int64_t xs[4];   // x strides for (n, c, h, w)
    int64_t ys[4];   // y / dy strides for (n, k, p, q)
    int64_t wsd[4];  // w strides for (k, c, r, s)
    float alpha;
};

hipError_t launch_direct_fwd(int dtype, const DirectParams &p, const void *x, const void *w,
                             void *y, hipStream_t st);
hipError_t launch_direct_dgrad(int dtype, const DirectParams &p, const void *dy, const void *w,
                               void *dx, hipStream_t st);
// Raw sums into ws[split][k][(r*S+s)*Cg + c], pixels split into `splits` ranges.
hipError_t launch_direct_wgrad(int dtype, const DirectParams &p, const void *x, const void *dy,
                               float *ws, int32_t splits, hipStream_t st);

// Grouped convolution as super-groups of sg channels (block-diagonal
// weights).  dst[k][t][c'] = w[k][c' - base][t] inside output channel k's
// own group of m channels (base = ((k % sg) / m) * m), else 0; src is
// [K][rs][m] (kcrs = 0) or [K][m][rs] (kcrs = 1).
hipError_t launch_expand_group_weights(const void *src, void *dst, int64_t k, int32_t rs, int32_t m,
                                       int32_t sg, int kcrs, hipStream_t st);
// dw[k][t][c] (c < m; [K][m][R][S] when kcrs) = (accumulate ? dw : 0) +
// inv_scale * sum_s ws[s][k][t][((k % sg) / m) * m + c]: the diagonal blocks
// of the super-group weight-gradient partials.
hipError_t launch_wgrad_reduce_diag(const float *ws, int32_t splits, int64_t k, int32_t rs,
                                    int32_t m, int32_t sg, void *dw, int out_dtype,
                                    float inv_scale, int accumulate, int32_t *flag, int kcrs,
                                    hipStream_t st);

// dst[b][cc][rr] = rr < rows ? src[b][rr][cc] : 0   for rr < dst_ld, cc < cols
hipError_t launch_transpose16(const void *src, void *dst, int64_t batch, int64_t rows,
                              int64_t cols, int64_t dst_ld, hipStream_t st);
// launch_transpose16 that also stores, per workgroup b of the
// transpose16_blocks(batch, cols, dst_ld) it launches, whether its tile of
// src held an inf or NaN of the given operand dtype into flags[b].
int64_t transpose16_blocks(int64_t batch, int64_t cols, int64_t dst_ld);
// Two independent launch_transpose16 calls in one launch (two launches
// when either cannot take the 16-byte kernel).
hipError_t launch_transpose16_pair(const void *src0, void *dst0, int64_t batch0, int64_t rows0,
                                   int64_t cols0, int64_t dst_ld0, const void *src1, void *dst1,
                                   int64_t batch1, int64_t rows1, int64_t cols1, int64_t dst_ld1,
                                   hipStream_t st);
hipError_t launch_transpose16_scan(const void *src, void *dst, int64_t batch, int64_t rows,
                                   int64_t cols, int64_t dst_ld, int dtype, int32_t *flags,
                                   hipStream_t st);
// flags[b] (b < nonfinite_scan16_blocks(count)) = whether src[2048 b ..
// 2048 b + 2047] holds an inf or NaN.
int64_t nonfinite_scan16_blocks(int64_t count);
hipError_t launch_nonfinite_scan16(const void *src, int64_t count, int dtype, int32_t *flags,
                                   hipStream_t st);
// If any of flags[0, nflags) is set: recompute dx at the border pixels (rows
// [0, bt), [H - bb, H); columns [0, bl), [W - br, W)) from the definition,
// skipping the taps outside dy.  Element strides come from p.
hipError_t launch_dgrad_border(int dtype, const DirectParams &p, const void *dy, const void *w,
                               void *dx, const int32_t *flags, int32_t nflags, int32_t bt,
                               int32_t bb, int32_t bl, int32_t br, hipStream_t st);

// dst[row][ch] = ch < c ? src[row][ch] : 0   for ch < c_pad
hipError_t launch_pad_channels16(const void *src, void *dst, int64_t rows, int32_t c,
                                 int32_t c_pad, hipStream_t st);

// Depthwise convolution (groups = C = K), channel-last, C % 8 == 0, square
// 3x3 / 5x5 / 7x7 filters (depthwise.hip).  Weights are [C][R][S] (the
// KRSC and KCRS layouts coincide for one channel per group).
struct DWParams {
    int32_t n, c, h, w, p, q, r, s;
    int32_t sh, sw, ph, pw, dh, dw;
    int32_t c8;              // c / 8
    int32_t cblocks;         // 64-channel blocks: (c8 + 7) / 8
    uint32_t x_bytes, dy_bytes;  // x and y / dy sizes (buffer range checks)
    int32_t splits;          // backward-weight pixel ranges
    int64_t pix_per_split;
    float alpha;
};
bool dw_supported(int r, int s);
// pass 0: forward (a = x, b = w, out = y); 1: backward-data (a = dy, b = w,
// out = dx); 2: backward-weight partials (a = x, b = dy,
// out = ws[split][c][r*S + s], fp32).
hipError_t launch_depthwise(int dtype, int pass, const DWParams &p, const void *a, const void *b,
                            void *out, hipStream_t st);

// LDS-tiled depthwise kernels (depthwise_tiled.hip): equal strides of 1 or 2,
// no dilation.
struct DWTParams {
    int32_t n, c, c8, cblocks;
    int32_t ih, iw, oh, ow;        // input image; output image (forward) or dy
    int32_t ph, pw;                // top / left padding of the input (may be < 0)
    int32_t tiles_h, tiles_w;
    int32_t th;                    // backward-weight: dy rows per tile
    int32_t tiles_per_split, splits;
    uint32_t in_bytes, dy_bytes;   // buffer range checks
    float alpha;
};
struct DWWgPlan {
    int32_t cbv, th, tiles_h, tiles_w, cblocks, splits, tiles_per_split;
};
bool dw_tiled(const DWParams &p, int pass);
int32_t dw_tiled_wgrad_splits(const DWParams &p);
hipError_t launch_depthwise_tiled(int dtype, int pass, const DWParams &p, const void *a,
                                  const void *b, void *out, hipStream_t st);

// Training-step pieces (update.hip).  The state type is the C ABI's.
hipError_t launch_loss_scaler_init(nnconv_loss_scaler *s, float scale, float factor,
                                   int32_t interval, hipStream_t st);
hipError_t launch_loss_scaler_update(nnconv_loss_scaler *s, int32_t *flag, hipStream_t st);
hipError_t launch_sgd_update(int64_t count, float *master, float *mom, void *w16, int w16_dtype,
                             const float *grad, const nnconv_loss_scaler *state,
                             const int32_t *flag, float lr, float mu, float wd, hipStream_t st);

}  // namespace nnconv
