/*
 * nnconv.h -- C ABI of libnnconv: mixed-precision 2-D convolution in the
 * three training passes (forward, backward-data, backward-weight) on one
 * AMD Instinct MI355X (gfx950).
 *
 * The operation is the paper's convolution call (Sec. 3.2, Listings 4-5:
 * convolution(x, base_axis=1, outmaps, kernel, ...)), trained by
 * back-propagation (Sec. 2.1) in mixed precision: half-precision storage of
 * weights, activations and gradients, products accumulated in fp32, and a
 * loss scale S that multiplies the incoming gradient and is divided out of
 * the weight gradient before the fp32 update (Sec. 3.3, Listing 6).
 *
 * Definitions (cross-correlation, symmetric zero padding):
 *   P = floor((H + 2*pad_h - dil_h*(R-1) - 1) / stride_h) + 1   (same for Q)
 *   Cg = C/groups, Kg = K/groups; output channel k reads input channels
 *   [ (k/Kg)*Cg, (k/Kg)*Cg + Cg ).
 *   forward   y[n,k,p,q]  = alpha * sum_{c<Cg,r<R,s<S} xz[n,(k/Kg)*Cg+c, p*sh-ph+r*dh, q*sw-pw+s*dw] * w[k,c,r,s]
 *   dgrad     dx = alpha * (adjoint of the forward map in x) applied to dy
 *   wgrad     dw = beta * dw + inv_loss_scale * (adjoint of the forward map in w)(x, dy)
 *   where xz is x extended by zeros.  dy is expected to carry the loss scale
 *   already (the caller scaled the loss); dgrad keeps it, wgrad removes it.
 *
 * Layouts (dense, contiguous):
 *   NNCONV_NCHW  x[N][C][H][W], y/dy[N][K][P][Q], w/dw[K][Cg][R][S]
 *   NNCONV_NHWC  x[N][H][W][C], y/dy[N][P][Q][K], w/dw[K][R][S][Cg]
 *
 * Ownership and execution:
 *   - Every buffer is a device pointer owned by the caller; the library
 *     allocates no memory (scratch comes from the caller's workspace, sized
 *     by nnconv_workspace_size) and never synchronises.
 *   - Work is queued on the caller's HIP stream (hipStream_t passed as
 *     void*; NULL means the default stream).  Calls return once queued.
 *     They queue kernel launches only (no memset, copy or event), so a
 *     sequence of calls may be captured into a HIP graph and replayed.
 *   - The library keeps no mutable global state (the one exception is the
 *     scratch array of nnconv_wgrad_noalloc, see there): calls are
 *     reentrant, and calls on different streams with disjoint buffers may
 *     run concurrently.
 *   - Fast (matrix-core) paths need 16-byte aligned pointers and Cg, Kg that
 *     are multiples of 8; other valid shapes run on slower direct kernels
 *     with identical semantics.
 *   - Depthwise convolution (groups == c == k, one channel per group, the
 *     MobileNet / EfficientNet layers trained with the paper's framework)
 *     with c a multiple of 8, a square 3x3, 5x5 or 7x7 filter and 16-byte
 *     aligned activations runs on dedicated vector-ALU kernels (R*S
 *     multiply-adds per output are too few for the matrix cores); w and dw
 *     are [K][R][S] in both layouts (one channel per filter).
 *   - Grouped convolution with m = C/groups = K/groups channels per group,
 *     m < 64 dividing 64 and c a multiple of 64 (e.g. 32 groups of 4-32
 *     channels) runs as groups of 64 channels with block-diagonal weights on
 *     the matrix-core kernels.  Results for finite inputs are those of the
 *     grouped convolution; a non-finite input value also makes the outputs
 *     of the other groups sharing its 64-channel block NaN.
 *   - Non-finite inputs: forward and backward-weight multiply the zeros of
 *     the zero-extended input at taps outside the image, as the definition
 *     reads, so an inf or NaN weight (forward) or dy (backward-weight) makes
 *     every sum it meets non-finite, padding included.  Backward-data has
 *     only the terms the adjoint definition has: where the matrix-core and
 *     depthwise kernels read dy zero-extended, a weight scan queued with
 *     the call has the border pixels recomputed from the definition when
 *     any weight is inf or NaN (small-group convolution excepted, above).
 *
 * Errors: every argument check happens on the host before anything is
 * queued.  On a non-OK status nothing is launched and no output or
 * workspace byte is touched.  No exception crosses the ABI and nothing is
 * printed.
 */
#ifndef NNCONV_H
#define NNCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NNCONV_VERSION 1

typedef enum {
    NNCONV_OK = 0,
    NNCONV_ERR_INVALID_ARG = 1,   /* bad shape, null pointer, bad enum */
    NNCONV_ERR_UNSUPPORTED = 2,   /* valid but not provided (e.g. dtype combination) */
    NNCONV_ERR_WORKSPACE = 3,     /* ws_bytes smaller than nnconv_workspace_size() */
    NNCONV_ERR_MISALIGNED = 4,    /* pointer alignment below the element size */
    NNCONV_ERR_HIP = 5            /* the HIP runtime refused a launch */
} nnconv_status;

typedef enum { NNCONV_NCHW = 0, NNCONV_NHWC = 1 } nnconv_layout;
typedef enum { NNCONV_F16 = 0, NNCONV_BF16 = 1, NNCONV_F32 = 2 } nnconv_dtype;
typedef enum { NNCONV_FWD = 0, NNCONV_DGRAD = 1, NNCONV_WGRAD = 2 } nnconv_pass;

/* Convolution geometry (the parameters of the paper's convolution call plus
 * stride, padding, dilation, groups, layout and operand type). */
typedef struct {
    int32_t n, c, h, w;          /* batch, input channels, input height, width */
    int32_t k, r, s;             /* output channels, filter height, width */
    int32_t stride_h, stride_w;  /* >= 1 */
    int32_t pad_h, pad_w;        /* >= 0, zero padding on both sides */
    int32_t dil_h, dil_w;        /* >= 1 */
    int32_t groups;              /* >= 1, divides c and k */
    int32_t layout;              /* nnconv_layout */
    int32_t dtype;               /* nnconv_dtype of x, w, y, dy, dx: F16 or BF16 */
} nnconv_desc;

/* Library version (NNCONV_VERSION). */
int32_t nnconv_version(void);

/* The hipError_t code behind the most recent NNCONV_ERR_HIP returned on the
 * calling thread (0 if there was none). */
int32_t nnconv_last_hip_error(void);

/* Static, human-readable name of a status code. */
const char *nnconv_status_string(nnconv_status status);

/* Output size (P, Q) from the floor formula above.
 * INVALID_ARG for a null argument, non-positive sizes, negative padding,
 * groups not dividing c and k, or an empty output. */
nnconv_status nnconv_output_dims(const nnconv_desc *desc, int32_t *p, int32_t *q);

/* Bytes of device workspace that nnconv_fwd / nnconv_dgrad / nnconv_wgrad
 * need for this geometry (0 is a valid answer).  Depends only on desc and
 * pass.  Workspace contents need not be initialised and are garbage after
 * the call. */
nnconv_status nnconv_workspace_size(const nnconv_desc *desc, nnconv_pass pass, size_t *bytes);

/* Forward pass (definition above): y = alpha * conv(x, w).
 * x, w, y: device pointers in desc->layout, element type desc->dtype.
 * Accumulation in fp32; y is rounded to nearest-even once, overflow gives
 * +-inf.  y must not overlap x, w or ws. */
nnconv_status nnconv_fwd(const nnconv_desc *desc, const void *x, const void *w, void *y,
                         float alpha, void *ws, size_t ws_bytes, void *hip_stream);

/* Backward-data pass: dx = alpha * (adjoint in x)(dy).  dy carries the
 * loss scale and dx keeps it.  Input positions that no output reads get an
 * exact 0.  dx must not overlap dy, w or ws. */
nnconv_status nnconv_dgrad(const nnconv_desc *desc, const void *dy, const void *w, void *dx,
                           float alpha, void *ws, size_t ws_bytes, void *hip_stream);

/* Tiles of the matrix-core implicit GEMM that runs the forward pass and the
 * backward-data pass when the reduction channels per filter tap (Cg for the
 * forward pass, Kg for backward-data) are a multiple of 64.  nnconv_fwd and
 * nnconv_dgrad pick one per shape; the _tile variants below force one, for
 * tests that must reach every tile on small shapes and for tuning.  Every
 * tile computes the same sums (the fp32 summation order may differ). */
typedef enum {
    NNCONV_TILE_256x256_8W = 0,   /* 8 waves of 128x64, 2 stages of 64-element slices */
    NNCONV_TILE_128x128_2S = 1,   /* 4 waves of 64x64, 2 stages */
    NNCONV_TILE_128x128 = 2,      /* 4 waves of 64x64, single stage */
    NNCONV_TILE_128x64 = 3,       /* 4 waves of 64x32, single stage */
    NNCONV_TILE_256x256_16W = 4,  /* 16 waves of 64x64, 2 stages */
    NNCONV_TILE_256x256_RING = 6, /* 4 waves of 128x128, ring of 4 32-element slices */
    NNCONV_TILE_256x128_RING = 7, /* 4 waves of 128x64, ring of 3 */
    NNCONV_TILE_256x64_RING = 8,  /* 4 waves of 64x64, ring of 4 */
    /* Halo staging, for stride-1 geometries whose input image has the
     * output's size and whose taps shift a pixel by at most 64 raster
     * positions (3x3 filters with padding 1 on images up to 63 pixels
     * wide; backward-data of the same at stride 1): 256-pixel tiles, each
     * 64-channel slice of the input staged once per tile for all taps. */
    NNCONV_TILE_HALO_256x64 = 9,    /* 4 waves of 64x64 */
    NNCONV_TILE_HALO_256x128 = 10,  /* 4 waves of 128x64 */
    NNCONV_TILE_HALO_256x64_2T = 11, /* 256x64, B tiles of two taps per barrier */
    /* Halo staging with the weight fragments loaded from L2 straight into
     * registers several taps ahead and the next channel slice's halo loading
     * during the current one (one workgroup per CU unless stated). */
    NNCONV_TILE_HALO_R256x128 = 12, /* 4 waves of 128x64; taps within 64 raster
                                       positions (3x3 on images up to 31 wide) */
    NNCONV_TILE_HALO_R128x256 = 13, /* 4 waves of 128x64 side by side */
    NNCONV_TILE_HALO_R224x256 = 14, /* 4 waves of 224x64 side by side; taps within
                                       32 raster positions (3x3 up to 15 wide) */
    NNCONV_TILE_HALO_R256x64S = 15  /* 4 waves of 64x64, a single 64-channel
                                       reduction slice (Cg = 64 forward, Kg = 64
                                       backward-data), two workgroups per CU */
} nnconv_tile;

/* nnconv_fwd / nnconv_dgrad with the tile forced (an nnconv_tile value).
 * Same arguments, semantics and errors, plus: INVALID_ARG for a negative
 * tile; UNSUPPORTED when the tile is not one of nnconv_tile, or when the
 * call would not run on the implicit-GEMM kernel (reduction channels per tap
 * not a multiple of 64, depthwise or small-group convolution, the stem's
 * 8- and 4-channel shapes, operands not 16-byte aligned or past 2 GiB, backward-data
 * with more than 4 stride phases), and for a halo tile on any other geometry
 * than the one it states or on grouped convolution. */
nnconv_status nnconv_fwd_tile(const nnconv_desc *desc, const void *x, const void *w, void *y,
                              float alpha, void *ws, size_t ws_bytes, void *hip_stream,
                              int32_t tile);
nnconv_status nnconv_dgrad_tile(const nnconv_desc *desc, const void *dy, const void *w, void *dx,
                                float alpha, void *ws, size_t ws_bytes, void *hip_stream,
                                int32_t tile);

/* Backward-weight pass with the loss-scale step of Sec. 3.3 / Listing 6:
 *   dw = (accumulate ? dw : 0) + inv_loss_scale * sum_{n,p,q} dy * xz
 * The batch-pixel reduction is split over the workspace in fp32 and summed
 * in a fixed order, so results are bitwise reproducible.
 * dw_dtype: NNCONV_F32 (for fp32 master weights) or desc->dtype.
 * accumulate: 0 overwrites dw (its old contents are not read), 1 adds.
 * overflow_flag: NULL or a device int32 that the caller zeroed; the call
 *   stores 1 into it when any final dw element is inf or NaN and never
 *   clears it (one flag can cover every layer of a step, as
 *   check_inf_or_nan_grad does in Listing 6). */
nnconv_status nnconv_wgrad(const nnconv_desc *desc, const void *x, const void *dy, void *dw,
                           int32_t dw_dtype, float inv_loss_scale, int32_t accumulate,
                           int32_t *overflow_flag, void *ws, size_t ws_bytes, void *hip_stream);

/* For callers that cannot allocate device memory or size a workspace --
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc: nnconv_wgrad with the workspace taken from a library-owned
 * scratch array of NNCONV_NOALLOC_WS_BYTES (64 MiB) instead of an argument.
 * Same arguments (minus ws, ws_bytes), semantics, results (bitwise equal to
 * nnconv_wgrad's) and errors, plus NNCONV_ERR_WORKSPACE, returned before
 * anything is queued, when the geometry needs more workspace than the
 * scratch holds (nnconv_workspace_size(desc, NNCONV_WGRAD) >
 * NNCONV_NOALLOC_WS_BYTES; every channel-last ResNet-50 layer at batch 256
 * fits).
 *   - The scratch is a device array of the library: every GPU the library
 *     runs on holds one copy from the first call on it (made with that GPU
 *     current, outside graph capture) until the process ends.  The call
 *     itself allocates nothing.
 *   - Every call on one GPU shares that GPU's copy, which keeps the last
 *     call's contents; nothing in it needs to start at zero.  Calls that
 *     overlap on one GPU (several streams or threads without ordering)
 *     race on it: order them on one stream. */
#define NNCONV_NOALLOC_WS_BYTES (64 * 1024 * 1024)
nnconv_status nnconv_wgrad_noalloc(const nnconv_desc *desc, const void *x, const void *dy,
                                   void *dw, int32_t dw_dtype, float inv_loss_scale,
                                   int32_t accumulate, int32_t *overflow_flag,
                                   void *hip_stream);

/* Layout transforms (pure data movement of 16-bit elements, bit exact).
 *
 * The paper's convolution call takes its channels on axis 1 (base_axis = 1
 * in Sec. 3.2, Listing 5), i.e. [N][C][H][W] activations with [K][Cg][R][S]
 * weights, stored in half precision (Sec. 3.3).  The matrix-core kernels
 * read channel-last tensors, where one 16-byte load is 8 consecutive
 * channels of a pixel; these calls move data between the two forms (the
 * NCHW entry points above use them internally through the workspace) and
 * pad the channel count of the 3-channel input image to 4 (or 8) for the
 * stem.
 * All pointers are caller-owned device memory; src and dst must not
 * overlap.  INVALID_ARG for null pointers or non-positive sizes (or a pad
 * below the channel count); MISALIGNED for pointers not 2-byte aligned.
 *
 * Activations: src[N][C][H][W] -> dst[N][H][W][c_pad], c_pad >= C; channels
 * C..c_pad-1 of dst are zero (the stem's 3 channels padded to 4). */
nnconv_status nnconv_nchw_to_nhwc(const void *src, void *dst, int32_t n, int32_t c, int32_t h,
                                  int32_t w, int32_t c_pad, void *hip_stream);

/* Activations: src[N][H][W][C] -> dst[N][C][H][W]. */
nnconv_status nnconv_nhwc_to_nchw(const void *src, void *dst, int32_t n, int32_t c, int32_t h,
                                  int32_t w, void *hip_stream);

/* Channel padding in channel-last form: src[rows][c] -> dst[rows][c_pad],
 * extra channels zero (rows = N*H*W). */
nnconv_status nnconv_pad_channels(const void *src, void *dst, int64_t rows, int32_t c,
                                  int32_t c_pad, void *hip_stream);

/* Weights: src[K][Cg][R][S] -> dst[K][R][S][cg_pad], cg_pad >= Cg, padding
 * zero. */
nnconv_status nnconv_weight_kcrs_to_krsc(const void *src, void *dst, int32_t k, int32_t cg,
                                         int32_t r, int32_t s, int32_t cg_pad, void *hip_stream);

/* Weights: src[K][R][S][Cg] -> dst[K][Cg][R][S]. */
nnconv_status nnconv_weight_krsc_to_kcrs(const void *src, void *dst, int32_t k, int32_t cg,
                                         int32_t r, int32_t s, void *hip_stream);

/* Training-step pieces after the backward passes (Sec. 3.3, Listing 6).
 *
 * A step with dynamic loss scaling, all on one stream and with no host
 * synchronisation:
 *   1. the caller seeds dy of the loss with the current scale S (it can read
 *      S from the device state below, e.g. as a 0-d tensor view);
 *   2. nnconv_wgrad for every layer with inv_loss_scale = 1, dw_dtype F32
 *      and one shared overflow flag (zeroed once, at set-up);
 *   3. nnconv_sgd_update for every parameter array, passing the state and
 *      the flag: it divides the gradient by S and does nothing at all when
 *      the flag is set;
 *   4. nnconv_loss_scaler_update once: it advances the scaler by the flag
 *      and clears the flag for the next step.
 * The order 3-before-4 matters: the update uses the scale the gradients
 * were computed with, and the scale only grows afterwards, as in the
 * listing. */

/* Device-resident dynamic loss-scaler state (24 bytes, caller-owned device
 * memory, 4-byte aligned).  Readable by the caller at any time; written
 * only by the two calls below. */
typedef struct {
    float scale;      /* current loss scale S */
    float factor;     /* growth / shrink factor (2 in the paper) */
    int32_t interval; /* clean steps between growths (2000 in the paper) */
    int32_t counter;  /* clean steps since the last growth or overflow */
    int32_t skipped;  /* steps skipped because of an inf or NaN gradient */
    int32_t reserved; /* zero */
} nnconv_loss_scaler;

/* Queues the initialisation of *state: scale = initial_scale, factor,
 * interval, counter = skipped = 0.
 * INVALID_ARG: null state, initial_scale or factor not finite and > 0,
 * interval < 0.  MISALIGNED: state not 4-byte aligned. */
nnconv_status nnconv_loss_scaler_init(nnconv_loss_scaler *state, float initial_scale,
                                      float factor, int32_t interval, void *hip_stream);

/* One step of the dynamic scaler of Listing 6, driven by *overflow_flag (a
 * device int32, nonzero = this step's gradients held an inf or a NaN):
 *   flag set:   scale /= factor; counter = 0; skipped += 1
 *   flag clear: if counter > interval { scale *= factor; counter = 0 }
 *               counter += 1
 * and then *overflow_flag = 0.  The test runs before the increment, so with
 * interval 2000 the first growth comes on the 2002nd consecutive clean step
 * and later ones every 2001 clean steps.  One thread; queue it after every
 * nnconv_sgd_update of the step.
 * INVALID_ARG: null pointer.  MISALIGNED: either pointer not 4-byte
 * aligned. */
nnconv_status nnconv_loss_scaler_update(nnconv_loss_scaler *state, int32_t *overflow_flag,
                                        void *hip_stream);

/* fp32 master-weight update (Sec. 3.3: 16-bit working weights, fp32 master
 * copy updated in fp32).  The paper names no solver; this is momentum SGD
 * with L2 weight decay, element-wise over count entries:
 *   g = grad / S + weight_decay * master      (S = state->scale, 1 if NULL)
 *   momentum = momentum_coef * momentum + g
 *   master  -= lr * momentum
 *   w16      = round-to-nearest-even(master)  (when w16 is not NULL)
 * computed in fp32 (1/S taken once, so a power-of-two S is exact).
 * master, momentum, grad: device fp32 arrays of count elements, in any
 * common element order (the nnconv_wgrad dw order of the layer's layout
 * matches the weights).  w16: NULL or device array of count elements of
 * w16_dtype (F16 or BF16), e.g. the layer's weights for the next forward.
 * overflow_flag: NULL or the step's device flag; when it is nonzero the
 * call changes nothing (the step is skipped).  The flag is only read.
 * In-place; master, momentum, grad and w16 must not overlap.  count = 0 is
 * a no-op.  16-byte aligned arrays and count % 4 == 0 take a vectorised
 * path.
 * INVALID_ARG: count < 0, null master/momentum/grad, w16_dtype not F16 or
 * BF16 when w16 is given.  MISALIGNED: fp32 arrays or state/flag not 4-byte
 * aligned, w16 not 2-byte aligned. */
nnconv_status nnconv_sgd_update(int64_t count, float *master, float *momentum, void *w16,
                                int32_t w16_dtype, const float *grad,
                                const nnconv_loss_scaler *state, const int32_t *overflow_flag,
                                float lr, float momentum_coef, float weight_decay,
                                void *hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* NNCONV_H */
