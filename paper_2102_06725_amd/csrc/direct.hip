// direct.hip -- direct convolution kernels (one thread per output element)
// for geometries the matrix-core kernels do not take: channel counts per
// group that are not multiples of 8, unaligned pointers, tensors beyond the
// 2 GiB buffer range, or more than 64 filter taps.  Same semantics as the
// fast path: fp32 accumulation, round-to-nearest-even output.  Both layouts
// are handled through element strides.  Also the 16-bit layout transforms.
#include <type_traits>

#include "launch.hpp"

namespace nnconv {

template <class T>
__device__ __forceinline__ float ld16(const void *p, int64_t i) {
    return from16<T>(((const uint16_t *)p)[i]);
}

// Exponent field of a 16-bit storage type: all ones means inf or NaN.
static uint32_t expmask16(int dtype) { return dtype == Half::id ? 0x7C00u : 0x7F80u; }

template <class T>
__global__ __launch_bounds__(256) void direct_fwd_kernel(const DirectParams P, const void *x,
                                                         const void *w, void *y) {
    const int64_t total = (int64_t)P.n * P.k * P.p * P.q;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= total) return;
    int64_t f = idx;
    const int q = (int)(f % P.q); f /= P.q;
    const int p = (int)(f % P.p); f /= P.p;
    const int k = (int)(f % P.k); f /= P.k;
    const int n = (int)f;
    const int g = k / P.kg;
    // Taps outside the image multiply the zero of the zero-extended input
    // rather than being skipped, so a non-finite weight gives a non-finite
    // output there too, as the definition does (and as the kernels whose
    // range-checked loads return zeros do).
    float acc = 0.f;
    for (int c = 0; c < P.cg; ++c) {
        const int ci = g * P.cg + c;
        for (int r = 0; r < P.r; ++r) {
            const int h = p * P.sh - P.ph + r * P.dh;
            const bool hin = h >= 0 && h < P.h;
            for (int s = 0; s < P.s; ++s) {
                const int wv = q * P.sw - P.pw + s * P.dw;
                const bool in = hin && wv >= 0 && wv < P.w;
                const float xv =
                    in ? ld16<T>(x, n * P.xs[0] + ci * P.xs[1] + h * P.xs[2] + wv * P.xs[3]) : 0.f;
                const float fv = ld16<T>(w, k * P.wsd[0] + c * P.wsd[1] + r * P.wsd[2] + s * P.wsd[3]);
                acc += xv * fv;
            }
        }
    }
    ((uint16_t *)y)[n * P.ys[0] + k * P.ys[1] + p * P.ys[2] + q * P.ys[3]] =
        (uint16_t)to16<T>(acc * P.alpha);
}

template <class T>
__global__ __launch_bounds__(256) void direct_dgrad_kernel(const DirectParams P, const void *dy,
                                                           const void *w, void *dx) {
    const int64_t total = (int64_t)P.n * P.c * P.h * P.w;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= total) return;
    int64_t f = idx;
    const int j = (int)(f % P.w); f /= P.w;
    const int i = (int)(f % P.h); f /= P.h;
    const int c = (int)(f % P.c); f /= P.c;
    const int n = (int)f;
    const int g = c / P.cg;
    const int cc = c - g * P.cg;
    float acc = 0.f;
    for (int kk = 0; kk < P.kg; ++kk) {
        const int k = g * P.kg + kk;
        for (int r = 0; r < P.r; ++r) {
            const int nump = i + P.ph - r * P.dh;
            if (nump < 0 || nump % P.sh) continue;
            const int p = nump / P.sh;
            if (p >= P.p) continue;
            for (int s = 0; s < P.s; ++s) {
                const int numq = j + P.pw - s * P.dw;
                if (numq < 0 || numq % P.sw) continue;
                const int q = numq / P.sw;
                if (q >= P.q) continue;
                const float dv = ld16<T>(dy, n * P.ys[0] + k * P.ys[1] + p * P.ys[2] + q * P.ys[3]);
                const float fv = ld16<T>(w, k * P.wsd[0] + cc * P.wsd[1] + r * P.wsd[2] + s * P.wsd[3]);
                acc += dv * fv;
            }
        }
    }
    ((uint16_t *)dx)[n * P.xs[0] + c * P.xs[1] + i * P.xs[2] + j * P.xs[3]] =
        (uint16_t)to16<T>(acc * P.alpha);
}

// ws[split][k][(r*S + s)*Cg + c] = sum over the split's pixels of dy * x
template <class T>
__global__ __launch_bounds__(256) void direct_wgrad_kernel(const DirectParams P, const void *x,
                                                           const void *dy, float *ws,
                                                           int32_t splits) {
    const int64_t rscg = (int64_t)P.r * P.s * P.cg;
    const int64_t count = (int64_t)P.k * rscg;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int split = blockIdx.y;
    if (idx >= count) return;
    const int k = (int)(idx / rscg);
    const int64_t jj = idx - (int64_t)k * rscg;
    const int tap = (int)(jj / P.cg);
    const int c = (int)(jj - (int64_t)tap * P.cg);
    const int r = tap / P.s, s = tap - (tap / P.s) * P.s;
    const int ci = (k / P.kg) * P.cg + c;
    const int64_t npq = (int64_t)P.n * P.p * P.q;
    const int64_t per = (npq + splits - 1) / splits;
    const int64_t b = split * per;
    const int64_t e = b + per < npq ? b + per : npq;
    float acc = 0.f;
    for (int64_t pix = b; pix < e; ++pix) {
        const int n = (int)(pix / ((int64_t)P.p * P.q));
        const int rm = (int)(pix - (int64_t)n * P.p * P.q);
        const int p = rm / P.q, q = rm - (rm / P.q) * P.q;
        const int h = p * P.sh - P.ph + r * P.dh;
        const int wv = q * P.sw - P.pw + s * P.dw;
        // outside the image: the zero of the zero-extended input, multiplied
        // (a non-finite dy then makes the sum non-finite, as defined)
        const bool in = h >= 0 && h < P.h && wv >= 0 && wv < P.w;
        const float xv =
            in ? ld16<T>(x, n * P.xs[0] + ci * P.xs[1] + h * P.xs[2] + wv * P.xs[3]) : 0.f;
        const float dv = ld16<T>(dy, n * P.ys[0] + k * P.ys[1] + p * P.ys[2] + q * P.ys[3]);
        acc += dv * xv;
    }
    ws[(int64_t)split * count + idx] = acc;
}

hipError_t launch_direct_fwd(int dtype, const DirectParams &p, const void *x, const void *w,
                             void *y, hipStream_t st) {
    const int64_t total = (int64_t)p.n * p.k * p.p * p.q;
    const dim3 grid((uint32_t)((total + 255) / 256));
    if (dtype == Half::id)
        hipLaunchKernelGGL(direct_fwd_kernel<Half>, grid, dim3(256), 0, st, p, x, w, y);
    else
        hipLaunchKernelGGL(direct_fwd_kernel<BFloat>, grid, dim3(256), 0, st, p, x, w, y);
    return hipGetLastError();
}

hipError_t launch_direct_dgrad(int dtype, const DirectParams &p, const void *dy, const void *w,
                               void *dx, hipStream_t st) {
    const int64_t total = (int64_t)p.n * p.c * p.h * p.w;
    const dim3 grid((uint32_t)((total + 255) / 256));
    if (dtype == Half::id)
        hipLaunchKernelGGL(direct_dgrad_kernel<Half>, grid, dim3(256), 0, st, p, dy, w, dx);
    else
        hipLaunchKernelGGL(direct_dgrad_kernel<BFloat>, grid, dim3(256), 0, st, p, dy, w, dx);
    return hipGetLastError();
}

hipError_t launch_direct_wgrad(int dtype, const DirectParams &p, const void *x, const void *dy,
                               float *ws, int32_t splits, hipStream_t st) {
    const int64_t count = (int64_t)p.k * p.r * p.s * p.cg;
    const dim3 grid((uint32_t)((count + 255) / 256), (uint32_t)splits);
    if (dtype == Half::id)
        hipLaunchKernelGGL(direct_wgrad_kernel<Half>, grid, dim3(256), 0, st, p, x, dy, ws, splits);
    else
        hipLaunchKernelGGL(direct_wgrad_kernel<BFloat>, grid, dim3(256), 0, st, p, x, dy, ws,
                           splits);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// 16-bit transforms
// ---------------------------------------------------------------------------

// dst[b][cc][rr] = rr < rows ? src[b][rr][cc] : 0, through a 64x64 LDS tile
// (reads coalesced along cc, writes coalesced along rr).
//
// SCAN: also store into flags[blockIdx.x] whether any element of the tile is
// inf or NaN (all exponent bits of expmask set).
// One 64x64 tile (index t) of a batched transpose with 2-byte accesses (any
// sizes and alignment).
template <bool SCAN>
__device__ __forceinline__ void transpose16_tile(const uint16_t *src, uint16_t *dst, int64_t rows,
                                                 int64_t cols, int64_t dst_ld, int64_t tiles_c,
                                                 int64_t tiles_r, int64_t t, uint16_t (*tile)[65],
                                                 uint32_t expmask, int32_t *flags) {
    const int64_t b = t / (tiles_c * tiles_r);
    const int64_t rem = t - b * tiles_c * tiles_r;
    const int64_t tr = rem / tiles_c, tc = rem - (rem / tiles_c) * tiles_c;
    const int64_t r0 = tr * 64, c0 = tc * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const uint16_t *s = src + b * rows * cols;
    int bad = 0;
    for (int i = ty; i < 64; i += 4) {
        const int64_t rr = r0 + i, cc = c0 + tx;
        const uint16_t v = (rr < rows && cc < cols) ? s[rr * cols + cc] : (uint16_t)0;
        tile[i][tx] = v;
        if constexpr (SCAN) bad |= (v & expmask) == expmask;
    }
    if constexpr (SCAN) {
        bad = __syncthreads_or(bad);
        if (threadIdx.x == 0) flags[t] = bad;
    } else {
        __syncthreads();
    }
    uint16_t *d = dst + b * cols * dst_ld;
    for (int i = ty; i < 64; i += 4) {
        const int64_t cc = c0 + i, rr = r0 + tx;
        if (cc < cols && rr < dst_ld) d[cc * dst_ld + rr] = tile[tx][i];
    }
}

template <bool SCAN>
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t *__restrict__ src,
                                                          uint16_t *__restrict__ dst, int64_t rows,
                                                          int64_t cols, int64_t dst_ld,
                                                          int64_t tiles_c, int64_t tiles_r,
                                                          uint32_t expmask, int32_t *flags) {
    __shared__ uint16_t tile[64][65];
    transpose16_tile<SCAN>(src, dst, rows, cols, dst_ld, tiles_c, tiles_r, blockIdx.x, tile,
                           expmask, flags);
}

// One 64x64 tile (index t) of a batched transpose, 16-byte accesses.
struct T16 {
    const uint16_t *src;
    uint16_t *dst;
    int64_t rows, cols, dst_ld, tiles_c, tiles_r;
};

template <bool SCAN>
__device__ __forceinline__ void transpose16_vec_tile(const T16 &p, int64_t t, uint16_t *tile,
                                                     uint32_t expmask, int32_t *flags) {
    const int64_t b = t / (p.tiles_c * p.tiles_r);
    const int64_t rem = t - b * p.tiles_c * p.tiles_r;
    const int64_t tr = rem / p.tiles_c, tc = rem - (rem / p.tiles_c) * p.tiles_c;
    const int64_t r0 = tr * 64, c0 = tc * 64;
    const uint16_t *s = p.src + b * p.rows * p.cols;
    int bad = 0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int id = threadIdx.x + 256 * i;
        const int row = id >> 3, cc = (id & 7) * 8;
        const int64_t rr = r0 + row, col = c0 + cc;
        u32x4 v = u32x4{};
        if (rr < p.rows && col < p.cols) v = *(const u32x4 *)(s + rr * p.cols + col);
        *(u32x4 *)(&tile[row * 64 + (((cc >> 3) ^ ((row >> 3) & 7)) << 3)]) = v;
        if constexpr (SCAN) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                bad |= ((v[e] & expmask) == expmask) | (((v[e] >> 16) & expmask) == expmask);
        }
    }
    if constexpr (SCAN) {
        bad = __syncthreads_or(bad);
        if (threadIdx.x == 0) flags[t] = bad;
    } else {
        __syncthreads();
    }
    uint16_t *d = p.dst + b * p.cols * p.dst_ld;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int id = threadIdx.x + 256 * i;
        const int oc = id >> 3, rc = (id & 7) * 8;
        const int64_t col = c0 + oc, rr = r0 + rc;
        if (col < p.cols && rr < p.dst_ld) {
            // rows rc .. rc + 7 share (r >> 3) = rc >> 3
            const int pc = (((oc >> 3) ^ ((rc >> 3) & 7)) << 3) + (oc & 7);
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                w[e] = (uint32_t)tile[(rc + 2 * e) * 64 + pc] |
                       ((uint32_t)tile[(rc + 2 * e + 1) * 64 + pc] << 16);
            *(u32x4 *)(d + col * p.dst_ld + rr) = u32x4{w[0], w[1], w[2], w[3]};
        }
    }
}

// Same transpose with 16-byte accesses on both sides (cols, dst_ld and rows
// multiples of 8, 16-byte aligned buffers): a 64x64 tile is read as 8-element
// row chunks, and each output chunk gathers 8 consecutive rows of one column
// from LDS.  The gather of a wave touches rows 8 apart, which share banks
// for any row pitch that keeps chunks 16-byte aligned, so chunk c of row r
// is stored at chunk c ^ ((r >> 3) & 7) instead of padding the rows.
template <bool SCAN>
__global__ __launch_bounds__(256) void transpose16_vec_kernel(const T16 p, uint32_t expmask,
                                                              int32_t *flags) {
    __shared__ __align__(16) uint16_t tile[64 * 64];
    transpose16_vec_tile<SCAN>(p, blockIdx.x, tile, expmask, flags);
}

// Two independent transposes in one launch (workgroups [0, n0) do the first,
// the rest the second), each with 16-byte accesses where its sizes and
// alignment allow (vec0, vec1): the layout copies on the input side of a
// channel-first call, one launch instead of two.
__global__ __launch_bounds__(256) void transpose16_pair_kernel(const T16 p0, const T16 p1,
                                                               int64_t n0, int vec0, int vec1) {
    // 16-byte aligned: the 16-byte tile path stores whole chunks
    __shared__ __align__(16) uint16_t tile[64][65];
    const int64_t t = blockIdx.x;
    const T16 &p = t < n0 ? p0 : p1;
    const int64_t u = t < n0 ? t : t - n0;
    if (t < n0 ? vec0 : vec1)
        transpose16_vec_tile<false>(p, u, &tile[0][0], 0u, nullptr);
    else
        transpose16_tile<false>(p.src, p.dst, p.rows, p.cols, p.dst_ld, p.tiles_c, p.tiles_r, u,
                                tile, 0u, nullptr);
}

// Block-diagonal super-group weights: dst[k][t][c'] (c' < sg, t < rs) is
// w[k][c' - base][t] when c' lies in output channel k's own group of m
// channels (base = ((k % sg) / m) * m), else 0.  src is [K][rs][m] (kcrs = 0)
// or [K][m][rs] (kcrs = 1).
__global__ __launch_bounds__(256) void expand_group_weights_kernel(
    const uint16_t *__restrict__ src, uint16_t *__restrict__ dst, int64_t count, int32_t rs,
    int32_t m, int32_t sg, int kcrs) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= count) return;
    const int64_t per_k = (int64_t)rs * sg;
    const int64_t k = e / per_k;
    const int64_t rem = e - k * per_k;
    const int64_t t = rem / sg;
    const int64_t cp = rem - t * sg;
    const int64_t base = ((k % sg) / m) * m;
    uint16_t v = 0;
    if (cp >= base && cp < base + m) {
        const int64_t c = cp - base;
        v = kcrs ? src[(k * m + c) * rs + t] : src[(k * rs + t) * m + c];
    }
    dst[e] = v;
}

hipError_t launch_expand_group_weights(const void *src, void *dst, int64_t k, int32_t rs, int32_t m,
                                       int32_t sg, int kcrs, hipStream_t st) {
    const int64_t count = k * rs * sg;
    if (count <= 0) return hipSuccess;
    const int64_t nb = (count + 255) / 256;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(expand_group_weights_kernel, dim3((uint32_t)nb), dim3(256), 0, st,
                       (const uint16_t *)src, (uint16_t *)dst, count, rs, m, sg, kcrs);
    return hipGetLastError();
}

int64_t transpose16_blocks(int64_t batch, int64_t cols, int64_t dst_ld) {
    return batch * ((cols + 63) / 64) * ((dst_ld + 63) / 64);
}

static T16 t16(const void *src, void *dst, int64_t rows, int64_t cols, int64_t dst_ld) {
    T16 p;
    p.src = (const uint16_t *)src;
    p.dst = (uint16_t *)dst;
    p.rows = rows;
    p.cols = cols;
    p.dst_ld = dst_ld;
    p.tiles_c = (cols + 63) / 64;
    p.tiles_r = (dst_ld + 63) / 64;
    return p;
}

static bool t16_vec(const void *src, const void *dst, int64_t rows, int64_t cols,
                    int64_t dst_ld) {
    return cols % 8 == 0 && dst_ld % 8 == 0 && rows % 8 == 0 && (uintptr_t)src % 16 == 0 &&
           (uintptr_t)dst % 16 == 0;
}

template <bool SCAN>
static hipError_t transpose16_go(const void *src, void *dst, int64_t batch, int64_t rows,
                                 int64_t cols, int64_t dst_ld, uint32_t expmask, int32_t *flags,
                                 hipStream_t st) {
    const int64_t tiles_c = (cols + 63) / 64, tiles_r = (dst_ld + 63) / 64;
    const int64_t nb = batch * tiles_c * tiles_r;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (t16_vec(src, dst, rows, cols, dst_ld))
        hipLaunchKernelGGL(transpose16_vec_kernel<SCAN>, dim3((uint32_t)nb), dim3(256), 0, st,
                           t16(src, dst, rows, cols, dst_ld), expmask, flags);
    else
        hipLaunchKernelGGL(transpose16_kernel<SCAN>, dim3((uint32_t)nb), dim3(256), 0, st,
                           (const uint16_t *)src, (uint16_t *)dst, rows, cols, dst_ld, tiles_c,
                           tiles_r, expmask, flags);
    return hipGetLastError();
}

hipError_t launch_transpose16(const void *src, void *dst, int64_t batch, int64_t rows,
                              int64_t cols, int64_t dst_ld, hipStream_t st) {
    return transpose16_go<false>(src, dst, batch, rows, cols, dst_ld, 0u, nullptr, st);
}

hipError_t launch_transpose16_pair(const void *src0, void *dst0, int64_t batch0, int64_t rows0,
                                   int64_t cols0, int64_t dst_ld0, const void *src1, void *dst1,
                                   int64_t batch1, int64_t rows1, int64_t cols1, int64_t dst_ld1,
                                   hipStream_t st) {
    const int64_t n0 = batch0 * ((cols0 + 63) / 64) * ((dst_ld0 + 63) / 64);
    const int64_t n1 = batch1 * ((cols1 + 63) / 64) * ((dst_ld1 + 63) / 64);
    if (n0 <= 0 || n1 <= 0 || n0 + n1 > 0x7FFFFFFF) {
        const hipError_t e = launch_transpose16(src0, dst0, batch0, rows0, cols0, dst_ld0, st);
        if (e != hipSuccess) return e;
        return launch_transpose16(src1, dst1, batch1, rows1, cols1, dst_ld1, st);
    }
    hipLaunchKernelGGL(transpose16_pair_kernel, dim3((uint32_t)(n0 + n1)), dim3(256), 0, st,
                       t16(src0, dst0, rows0, cols0, dst_ld0),
                       t16(src1, dst1, rows1, cols1, dst_ld1), n0,
                       (int)t16_vec(src0, dst0, rows0, cols0, dst_ld0),
                       (int)t16_vec(src1, dst1, rows1, cols1, dst_ld1));
    return hipGetLastError();
}

hipError_t launch_transpose16_scan(const void *src, void *dst, int64_t batch, int64_t rows,
                                   int64_t cols, int64_t dst_ld, int dtype, int32_t *flags,
                                   hipStream_t st) {
    return transpose16_go<true>(src, dst, batch, rows, cols, dst_ld, expmask16(dtype), flags,
                                st);
}

// flags[b] = whether any of the 16-bit elements [2048 b, 2048 b + 2048) of
// src[0, count) is inf or NaN.
__global__ __launch_bounds__(256) void nonfinite_scan16_kernel(const uint16_t *__restrict__ src,
                                                               int64_t count, uint32_t expmask,
                                                               int32_t *flags) {
    int bad = 0;
    const int64_t base = (int64_t)blockIdx.x * 2048;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int64_t e = base + u * 256 + threadIdx.x;
        if (e < count) bad |= (src[e] & expmask) == expmask;
    }
    bad = __syncthreads_or(bad);
    if (threadIdx.x == 0) flags[blockIdx.x] = bad;
}

int64_t nonfinite_scan16_blocks(int64_t count) { return (count + 2047) / 2048; }

hipError_t launch_nonfinite_scan16(const void *src, int64_t count, int dtype, int32_t *flags,
                                   hipStream_t st) {
    const int64_t nb = nonfinite_scan16_blocks(count);
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(nonfinite_scan16_kernel, dim3((uint32_t)nb), dim3(256), 0, st,
                       (const uint16_t *)src, count, expmask16(dtype), flags);
    return hipGetLastError();
}

// Backward-data border fix-up.  The matrix-core and depthwise kernels read
// dy zero-extended at every filter tap of a stride phase, so an inf or NaN
// weight meets those zeros (0 * inf = NaN) at dx pixels whose taps leave dy
// -- terms the definition does not have.  When any weight is non-finite
// (some flag set), this kernel recomputes every such border pixel from the
// definition: rows [0, bt) and [H - bb, H), and columns [0, bl) and
// [W - br, W) of the other rows, every channel, skipping the taps outside dy.
// With all flags clear every workgroup returns at once.
template <class T>
__global__ __launch_bounds__(256) void dgrad_border_kernel(const DirectParams P, const void *dy,
                                                           const void *w, void *dx,
                                                           const int32_t *flags, int32_t nflags,
                                                           int32_t bt, int32_t bb, int32_t bl,
                                                           int32_t br) {
    int any = 0;
    for (int i = threadIdx.x; i < nflags; i += 256) any |= flags[i];
    if (!__syncthreads_or(any)) return;
    const int64_t mid = P.h - bt - bb;
    const int64_t per_img = (int64_t)(bt + bb) * P.w + mid * (bl + br);
    const int64_t total = (int64_t)P.n * per_img * P.c;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * 256) {
        const int c = (int)(e % P.c);
        int64_t f = e / P.c;
        const int64_t pix = f % per_img;
        const int n = (int)(f / per_img);
        int i, j;
        if (pix < (int64_t)bt * P.w) {
            i = (int)(pix / P.w);
            j = (int)(pix % P.w);
        } else if (pix < (int64_t)(bt + bb) * P.w) {
            const int64_t q = pix - (int64_t)bt * P.w;
            i = P.h - bb + (int)(q / P.w);
            j = (int)(q % P.w);
        } else {
            const int64_t q = pix - (int64_t)(bt + bb) * P.w;
            i = bt + (int)(q / (bl + br));
            const int u = (int)(q % (bl + br));
            j = u < bl ? u : P.w - br + (u - bl);
        }
        const int g = c / P.cg;
        const int cc = c - g * P.cg;
        float acc = 0.f;
        for (int kk = 0; kk < P.kg; ++kk) {
            const int k = g * P.kg + kk;
            for (int r = 0; r < P.r; ++r) {
                const int nump = i + P.ph - r * P.dh;
                if (nump < 0 || nump % P.sh) continue;
                const int p = nump / P.sh;
                if (p >= P.p) continue;
                for (int s = 0; s < P.s; ++s) {
                    const int numq = j + P.pw - s * P.dw;
                    if (numq < 0 || numq % P.sw) continue;
                    const int q = numq / P.sw;
                    if (q >= P.q) continue;
                    const float dv =
                        ld16<T>(dy, n * P.ys[0] + k * P.ys[1] + p * P.ys[2] + q * P.ys[3]);
                    const float fv =
                        ld16<T>(w, k * P.wsd[0] + cc * P.wsd[1] + r * P.wsd[2] + s * P.wsd[3]);
                    acc += dv * fv;
                }
            }
        }
        ((uint16_t *)dx)[n * P.xs[0] + c * P.xs[1] + i * P.xs[2] + j * P.xs[3]] =
            (uint16_t)to16<T>(acc * P.alpha);
    }
}

hipError_t launch_dgrad_border(int dtype, const DirectParams &p, const void *dy, const void *w,
                               void *dx, const int32_t *flags, int32_t nflags, int32_t bt,
                               int32_t bb, int32_t bl, int32_t br, hipStream_t st) {
    if (bt + bb == 0 && bl + br == 0) return hipSuccess;
    if (bt < 0 || bb < 0 || bl < 0 || br < 0 || bt + bb > p.h || bl + br > p.w)
        return hipErrorInvalidValue;
    const dim3 grid(256), block(256);
    if (dtype == Half::id)
        hipLaunchKernelGGL(dgrad_border_kernel<Half>, grid, block, 0, st, p, dy, w, dx, flags,
                           nflags, bt, bb, bl, br);
    else
        hipLaunchKernelGGL(dgrad_border_kernel<BFloat>, grid, block, 0, st, p, dy, w, dx, flags,
                           nflags, bt, bb, bl, br);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void pad_channels16_kernel(const uint16_t *__restrict__ src,
                                                             uint16_t *__restrict__ dst,
                                                             int64_t total, int32_t c,
                                                             int32_t c_pad) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int64_t row = i / c_pad;
    const int ch = (int)(i - row * c_pad);
    dst[i] = ch < c ? src[row * c + ch] : (uint16_t)0;
}

// c_pad a multiple of 8 and dst 16-byte aligned: one thread builds one
// 8-channel (16-byte) chunk of the output and stores it whole.
__global__ __launch_bounds__(256) void pad_channels16_vec_kernel(const uint16_t *__restrict__ src,
                                                                 u32x4 *__restrict__ dst,
                                                                 int64_t chunks, int32_t c,
                                                                 int32_t chunks_per_row) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= chunks) return;
    const int64_t row = i / chunks_per_row;
    const int ch0 = (int)(i - row * chunks_per_row) * 8;
    const uint16_t *s = src + row * c;
    uint32_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int a = ch0 + 2 * u, b = a + 1;
        const uint32_t lo = a < c ? s[a] : 0u;
        const uint32_t hi = b < c ? s[b] : 0u;
        v[u] = lo | (hi << 16);
    }
    dst[i] = u32x4{v[0], v[1], v[2], v[3]};
}

// c_pad == 4 and dst 16-byte aligned: one thread builds two 4-channel
// pixels (16 bytes; the last thread of an odd row count one, 8 bytes).
__global__ __launch_bounds__(256) void pad_channels4_vec_kernel(const uint16_t *__restrict__ src,
                                                                u32x4 *__restrict__ dst,
                                                                int64_t rows, int32_t c) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t r0 = 2 * i;
    if (r0 >= rows) return;
    uint32_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int64_t row = r0 + (u >> 1);
        const int a = 2 * (u & 1), b = a + 1;
        const uint16_t *sp = src + row * c;
        const uint32_t lo = row < rows && a < c ? sp[a] : 0u;
        const uint32_t hi = row < rows && b < c ? sp[b] : 0u;
        v[u] = lo | (hi << 16);
    }
    if (r0 + 1 < rows)
        dst[i] = u32x4{v[0], v[1], v[2], v[3]};
    else
        *(u32x2 *)&dst[i] = u32x2{v[0], v[1]};
}

hipError_t launch_pad_channels16(const void *src, void *dst, int64_t rows, int32_t c,
                                 int32_t c_pad, hipStream_t st) {
    const int64_t total = rows * c_pad;
    if (total <= 0) return hipSuccess;
    if (c_pad == 4 && ((uintptr_t)dst % 16) == 0) {
        const int64_t pairs = (rows + 1) / 2;
        hipLaunchKernelGGL(pad_channels4_vec_kernel, dim3((uint32_t)((pairs + 255) / 256)), dim3(256),
                           0, st, (const uint16_t *)src, (u32x4 *)dst, rows, c);
        return hipGetLastError();
    }
    if (c_pad % 8 == 0 && ((uintptr_t)dst % 16) == 0) {
        const int64_t chunks = total / 8;
        hipLaunchKernelGGL(pad_channels16_vec_kernel, dim3((uint32_t)((chunks + 255) / 256)),
                           dim3(256), 0, st, (const uint16_t *)src, (u32x4 *)dst, chunks, c,
                           c_pad / 8);
    } else {
        hipLaunchKernelGGL(pad_channels16_kernel, dim3((uint32_t)((total + 255) / 256)), dim3(256),
                           0, st, (const uint16_t *)src, (uint16_t *)dst, total, c, c_pad);
    }
    return hipGetLastError();
}

}  // namespace nnconv
