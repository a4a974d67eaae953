// depthwise.hip -- depthwise convolution (groups = C = K: one input and one
// output channel per group) in the three training passes, channel-last,
// fp16/bf16 operands with fp32 accumulation.
//
// The work per output is one filter's taps (R*S multiply-adds), far below
// what the matrix cores need to pay off, and the pass is bound by HBM.  The
// kernels therefore run on the vector ALUs and are organised around memory:
//   - a thread owns 8 consecutive channels (one 16-byte vector) of a pixel;
//     consecutive threads take consecutive channel vectors, then pixels, so a
//     wave reads and writes whole contiguous runs of pixel rows;
//   - forward: a thread computes a strip of TP output rows of one output
//     column; every input row the strip touches is loaded once (the next
//     row's loads in flight while the current one is added in) and added
//     into each strip row it feeds (4.5 loads per output for a 3x3 stride-1
//     filter instead of 9), the rest of the reuse comes from L1/L2;
//   - backward-data: workgroups take pixels of one stride phase, which are
//     all reached by the same taps (about 1/s^2 of them for stride s), and
//     gather only those;
//   - backward-weight: workgroups own a pixel range and one filter row;
//     threads accumulate over pixels in a fixed order, the workgroup sums its
//     threads in a fixed order and writes one fp32 partial per split, which
//     the shared split reduction (loss-scale step, overflow flag) finishes.
// Forward and backward-data workgroups cover 64 channels; they stage those
// channels' weights (contiguous in memory) in LDS as [R*S][64], so a tap's 8
// channels are one 16-byte read and every call is a single launch.
#include "launch.hpp"

namespace nnconv {

namespace dwc {

// 8 16-bit values of one 16-byte vector -> fp32
template <class T>
__device__ __forceinline__ void unpack8(u32x4 v, float (&f)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = from16<T>(v[i] & 0xFFFFu);
        f[2 * i + 1] = from16<T>(v[i] >> 16);
    }
}

template <class T>
__device__ __forceinline__ u32x4 pack8(const float (&f)[8], float alpha) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        v[i] = to16<T>(f[2 * i] * alpha) | (to16<T>(f[2 * i + 1] * alpha) << 16);
    return v;
}

__device__ __forceinline__ u32x4 ld16(const uint16_t *p) { return *(const u32x4 *)p; }

constexpr int DW_PIX_BLOCKS = 8;  // backward-data: 32-pixel blocks per workgroup

}  // namespace dwc

// Stage the weights of the workgroup's 64 channels as [R*S][64] in LDS:
// in memory they are [C][R*S] (KRSC = KCRS when each group has one channel),
// so the block is one contiguous run of 64*R*S elements.
template <int R, int S>
__device__ __forceinline__ void stage_weights(const uint16_t *__restrict__ w, int c0, int c,
                                              uint16_t (*wl)[64]) {
    for (int e = threadIdx.x; e < 64 * R * S; e += 256) {
        const int cl = e / (R * S), t = e - cl * (R * S);
        wl[t][cl] = c0 + cl < c ? w[(int64_t)(c0 + cl) * (R * S) + t] : (uint16_t)0;
    }
    __syncthreads();
}

// y[n, p, q, c] = alpha * sum_{r,s} x[n, p*sh - ph + r*dh, q*sw - pw + s*dw, c] * w[c, r, s]
// Workgroup: 64 channels (8 vectors) x 32 output columns (flattened n, q)
// x TP output rows; thread (column tid / 8, channel vector tid % 8).
template <class T, int R, int S, int TP>
__global__ __launch_bounds__(256) void dw_fwd_kernel(const DWParams P, const uint16_t *__restrict__ x,
                                                     const uint16_t *__restrict__ w,
                                                     uint16_t *__restrict__ y) {
    using namespace dwc;
    __shared__ uint16_t wl[R * S][64];
    const int cbk = (int)(blockIdx.x % P.cblocks);
    const int64_t nq = (int64_t)(blockIdx.x / P.cblocks) * 32 + (threadIdx.x >> 3);
    const int c8 = cbk * 8 + (int)(threadIdx.x & 7);
    stage_weights<R, S>(w, cbk * 64, P.c, wl);
    if (nq >= (int64_t)P.n * P.q || c8 >= P.c8) return;  // no barrier below
    const int q = (int)(nq % P.q);
    const int n = (int)(nq / P.q);
    const int p0 = (int)blockIdx.y * TP;
    const int pe = min(P.p, p0 + TP);
    const int c = c8 * 8;
    const int cl = (int)(threadIdx.x & 7) * 8;
    (void)x;

    float acc[TP][8];
#pragma unroll
    for (int i = 0; i < TP; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[i][k] = 0.f;

    // byte offsets of the S taps' input columns within a row (out-of-range
    // columns read zeros through the buffer range check)
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, P.x_bytes);
    uint32_t coff[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const int wc = q * P.sw - P.pw + s * P.dw;
        coff[s] = (unsigned)wc < (unsigned)P.w ? (uint32_t)(wc * P.c + c) * 2u : OOB_OFFSET;
    }
    const uint32_t img = (uint32_t)n * (uint32_t)P.h;  // first row of image n
    auto load_row = [&](int h, u32x4 (&v)[S]) {
        const bool ok = (unsigned)h < (unsigned)P.h;
        const uint32_t roff = ((img + (uint32_t)h) * (uint32_t)P.w) * (uint32_t)P.c * 2u;
#pragma unroll
        for (int s = 0; s < S; ++s)
            v[s] = load16(rx, ok && coff[s] != OOB_OFFSET ? roff + coff[s] : OOB_OFFSET);
    };
    // input rows touched by the strip: h = p*sh - ph + r*dh, p in [p0, pe);
    // the next row's loads are in flight while the current row is added in
    const int h_lo = p0 * P.sh - P.ph;
    const int h_hi = (pe - 1) * P.sh - P.ph + (R - 1) * P.dh;
    u32x4 cur[S], nxt[S];
    load_row(h_lo, cur);
    for (int h = h_lo; h <= h_hi; ++h) {
        if (h < h_hi) load_row(h + 1, nxt);
        float v[S][8];
#pragma unroll
        for (int s = 0; s < S; ++s) unpack8<T>(cur[s], v[s]);
        // strip rows fed by this input row: h = p*sh - ph + r*dh
#pragma unroll
        for (int i = 0; i < TP; ++i) {
            const int p = p0 + i;
            if (p >= pe) continue;
            const int d = h - (p * P.sh - P.ph);
            if (d < 0 || d % P.dh != 0) continue;
            const int r = d / P.dh;
            if (r >= R) continue;
#pragma unroll
            for (int rr = 0; rr < R; ++rr) {
                if (rr != r) continue;
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    // weights are read from LDS at use: holding all taps in
                    // registers would cost occupancy
                    float wf[8];
                    unpack8<T>(*(const u32x4 *)&wl[rr * S + s][cl], wf);
#pragma unroll
                    for (int k = 0; k < 8; ++k) acc[i][k] += v[s][k] * wf[k];
                }
            }
        }
#pragma unroll
        for (int s = 0; s < S; ++s) cur[s] = nxt[s];
    }
    uint16_t *yn = y + (int64_t)n * P.p * P.q * P.c + c;
#pragma unroll
    for (int i = 0; i < TP; ++i) {
        const int p = p0 + i;
        if (p < pe) *(u32x4 *)(yn + ((int64_t)p * P.q + q) * P.c) = pack8<T>(acc[i], P.alpha);
    }
}

// dx[n, i, j, c] = alpha * sum over taps (r, s) with i = p*sh - ph + r*dh and
// j = q*sw - pw + s*dw of dy[n, p, q, c] * w[c, r, s]
// A stride phase (i mod sh, j mod sw) is reached by a fixed set of taps, so
// the pixels are ordered phase by phase: a workgroup covers 64 channels x
// DW_PIX_BLOCKS blocks of 32 pixels of one phase (blockIdx.y) and loops over
// that phase's taps only (the taps of a phase are an arithmetic progression
// along each axis).
template <class T, int R, int S>
__global__ __launch_bounds__(256) void dw_dgrad_kernel(const DWParams P,
                                                       const uint16_t *__restrict__ dy,
                                                       const uint16_t *__restrict__ w,
                                                       uint16_t *__restrict__ dx) {
    using namespace dwc;
    __shared__ uint16_t wl[R * S][64];
    const int phi = (int)blockIdx.y / P.sw, phj = (int)blockIdx.y % P.sw;
    const int mi = (P.h - phi + P.sh - 1) / P.sh;  // rows of this phase
    const int mj = (P.w - phj + P.sw - 1) / P.sw;
    const int cbk = (int)(blockIdx.x % P.cblocks);
    const int c8 = cbk * 8 + (int)(threadIdx.x & 7);
    stage_weights<R, S>(w, cbk * 64, P.c, wl);
    const int64_t npix = (int64_t)P.n * mi * mj;
    if (mi <= 0 || mj <= 0 || c8 >= P.c8) return;  // no barrier below
    const int c = c8 * 8;
    const int cl = (int)(threadIdx.x & 7) * 8;
    // taps of this phase: r = r0, r0 + dr, ... with (i + ph - r*dh) % sh == 0
    int r0 = 0, s0 = 0;
    while (r0 < R && ((phi + P.ph - r0 * P.dh) % P.sh + P.sh) % P.sh != 0) ++r0;
    while (s0 < S && ((phj + P.pw - s0 * P.dw) % P.sw + P.sw) % P.sw != 0) ++s0;
    int dr = 1, ds = 1;
    while (dr < R && (dr * P.dh) % P.sh != 0) ++dr;
    while (ds < S && (ds * P.dw) % P.sw != 0) ++ds;
    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(dy, P.dy_bytes);
    // the workgroup's DW_PIX_BLOCKS blocks of 32 pixels share the staged
    // weights
    const int64_t loc0 = (int64_t)(blockIdx.x / P.cblocks) * (32 * DW_PIX_BLOCKS) + (threadIdx.x >> 3);
    for (int blk = 0; blk < DW_PIX_BLOCKS; ++blk) {
        const int64_t loc = loc0 + blk * 32;
        if (loc >= npix) break;
        const int jj = (int)(loc % mj);
        const int64_t nq = loc / mj;
        const int ii = (int)(nq % mi);
        const int n = (int)(nq / mi);
        const int i = ii * P.sh + phi, j = jj * P.sw + phj;
        // every tap of the phase in flight at once (rows past the phase's
        // taps are skipped by uniform branches); out-of-range taps read zeros
        u32x4 v[R][S];
#pragma unroll
        for (int kr = 0; kr < R; ++kr) {
            const int r = r0 + kr * dr;
            if (r >= R) break;
            const int p = (i + P.ph - r * P.dh) / P.sh;  // exact for this phase
            const bool rok = i + P.ph - r * P.dh >= 0 && p < P.p;
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const int ss = s0 + s * ds;
                const int nw = j + P.pw - ss * P.dw;
                const int q = nw / P.sw;
                const bool ok = ss < S && rok && nw >= 0 && q < P.q;
                const uint32_t off =
                    (uint32_t)((((uint32_t)n * P.p + p) * P.q + q) * P.c + c) * 2u;
                v[kr][s] = load16(rdy, ok ? off : OOB_OFFSET);
            }
        }
        float acc[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] = 0.f;
#pragma unroll
        for (int kr = 0; kr < R; ++kr) {
            const int r = r0 + kr * dr;
            if (r >= R) break;
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const int ss = s0 + s * ds;
                if (ss >= S) break;
                float g[8], wv[8];
                unpack8<T>(v[kr][s], g);
                unpack8<T>(*(const u32x4 *)&wl[r * S + ss][cl], wv);
#pragma unroll
                for (int k = 0; k < 8; ++k) acc[k] += g[k] * wv[k];
            }
        }
        *(u32x4 *)(dx + ((((int64_t)n * P.h + i) * P.w) + j) * P.c + c) = pack8<T>(acc, P.alpha);
    }
}

// Partial sums of dw[c, r, s] = sum_pix dy[pix, c] * x[pix shifted by tap
// (r, s), c] over the pixels of one split, for the filter row r = blockIdx.z
// and the 64 channels of blockIdx.x: ws[split][c][r*S + s].
// Thread (lane group pl = tid / 8, channel vector cb = tid % 8): pixels
// split_begin + pl, + 32, ... in order; then the 32 lane groups are summed
// in a fixed tree order through LDS.
template <class T, int R, int S>
__global__ __launch_bounds__(256) void dw_wgrad_kernel(const DWParams P,
                                                       const uint16_t *__restrict__ x,
                                                       const uint16_t *__restrict__ dy,
                                                       float *__restrict__ ws) {
    using namespace dwc;
    __shared__ float red[32][8][S * 8 + 1];
    const int tid = threadIdx.x;
    const int pl = tid >> 3, cb = tid & 7;
    const int c8 = (int)blockIdx.x * 8 + cb;
    const int split = (int)blockIdx.y;
    const int r = (int)blockIdx.z;
    const bool cok = c8 < P.c8;
    const int c = c8 * 8;
    const int64_t npq = (int64_t)P.n * P.p * P.q;
    const int64_t b0 = (int64_t)split * P.pix_per_split;
    const int64_t b1 = min(npq, b0 + P.pix_per_split);

    float acc[S][8];
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[s][k] = 0.f;

    if (cok) {
        const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, P.x_bytes);
        const __amdgpu_buffer_rsrc_t rdy = make_rsrc(dy, P.dy_bytes);
        // operands of one pixel: dy and the S input vectors of filter row r
        // (zeros outside the image through the range check)
        auto load_pix = [&](int64_t pix, u32x4 &g, u32x4 (&v)[S]) {
            const bool in = pix < b1;
            const int64_t pc = in ? pix : b0;
            const int q = (int)(pc % P.q);
            const int64_t np = pc / P.q;
            const int p = (int)(np % P.p);
            const int n = (int)(np / P.p);
            const int h = p * P.sh - P.ph + r * P.dh;
            const bool hok = in && (unsigned)h < (unsigned)P.h;
            g = load16(rdy, in ? (uint32_t)(pc * P.c + c) * 2u : OOB_OFFSET);
            const uint32_t roff = (uint32_t)(((int64_t)n * P.h + h) * P.w) * (uint32_t)P.c * 2u;
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const int w = q * P.sw - P.pw + s * P.dw;
                const bool ok = hok && (unsigned)w < (unsigned)P.w;
                v[s] = load16(rx, ok ? roff + (uint32_t)(w * P.c + c) * 2u : OOB_OFFSET);
            }
        };
        auto add_pix = [&](u32x4 gv, const u32x4 (&v)[S]) {
            float g[8];
            unpack8<T>(gv, g);
#pragma unroll
            for (int s = 0; s < S; ++s) {
                float xv[8];
                unpack8<T>(v[s], xv);
#pragma unroll
                for (int k = 0; k < 8; ++k) acc[s][k] += g[k] * xv[k];
            }
        };
        // pixels b0 + pl, + 32, ...: two in flight, added in pixel order
        for (int64_t pix = b0 + pl; pix < b1; pix += 64) {
            u32x4 g0, g1, v0[S], v1[S];
            load_pix(pix, g0, v0);
            load_pix(pix + 32, g1, v1);
            add_pix(g0, v0);
            add_pix(g1, v1);  // zeros past the range
        }
    }
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
        for (int k = 0; k < 8; ++k) red[pl][cb][s * 8 + k] = acc[s][k];
    __syncthreads();
    // fixed-order tree over the 32 lane groups
    for (int half = 16; half >= 1; half >>= 1) {
        if (pl < half) {
#pragma unroll
            for (int e = 0; e < S * 8; ++e) red[pl][cb][e] += red[pl + half][cb][e];
        }
        __syncthreads();
    }
    if (pl == 0 && cok) {
        float *o = ws + (int64_t)split * P.c * (R * S);
#pragma unroll
        for (int k = 0; k < 8; ++k)
#pragma unroll
            for (int s = 0; s < S; ++s) o[(int64_t)(c + k) * (R * S) + r * S + s] = red[0][cb][s * 8 + k];
    }
}

template <class T, int R, int S>
static hipError_t launch_dw_rs(int pass, const DWParams &p, const void *a, const void *b, void *out,
                               hipStream_t st) {
    if (pass == 0) {
        constexpr int TP = R <= 5 ? 4 : 2;  // output rows per thread
        const int64_t nb = ((int64_t)p.n * p.q + 31) / 32 * p.cblocks;
        const int64_t ny = (p.p + TP - 1) / TP;
        if (nb > 0x7FFFFFFF || ny > 65535) return hipErrorInvalidValue;
        hipLaunchKernelGGL((dw_fwd_kernel<T, R, S, TP>), dim3((uint32_t)nb, (uint32_t)ny),
                           dim3(256), 0, st, p, (const uint16_t *)a, (const uint16_t *)b,
                           (uint16_t *)out);
    } else if (pass == 1) {
        // pixels per phase at most ceil(h / sh) * ceil(w / sw)
        const int64_t mi = (p.h + p.sh - 1) / p.sh, mj = (p.w + p.sw - 1) / p.sw;
        const int64_t per = 32 * dwc::DW_PIX_BLOCKS;
        const int64_t nb = ((int64_t)p.n * mi * mj + per - 1) / per * p.cblocks;
        const int64_t nph = (int64_t)p.sh * p.sw;
        if (nb > 0x7FFFFFFF || nph > 65535) return hipErrorInvalidValue;
        hipLaunchKernelGGL((dw_dgrad_kernel<T, R, S>), dim3((uint32_t)nb, (uint32_t)nph), dim3(256),
                           0, st, p,
                           (const uint16_t *)a, (const uint16_t *)b, (uint16_t *)out);
    } else {
        const int64_t nbx = p.cblocks;
        if (p.splits > 65535 || nbx > 0x7FFFFFFF) return hipErrorInvalidValue;
        hipLaunchKernelGGL((dw_wgrad_kernel<T, R, S>), dim3((uint32_t)nbx, (uint32_t)p.splits, R),
                           dim3(256), 0, st, p, (const uint16_t *)a, (const uint16_t *)b,
                           (float *)out);
    }
    return hipGetLastError();
}

bool dw_supported(int r, int s) { return r == s && (r == 3 || r == 5 || r == 7); }

template <class T>
static hipError_t launch_dw_t(int pass, const DWParams &p, const void *a, const void *b, void *out,
                              hipStream_t st) {
    switch (p.r) {
        case 3: return launch_dw_rs<T, 3, 3>(pass, p, a, b, out, st);
        case 5: return launch_dw_rs<T, 5, 5>(pass, p, a, b, out, st);
        case 7: return launch_dw_rs<T, 7, 7>(pass, p, a, b, out, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_depthwise(int dtype, int pass, const DWParams &p, const void *a, const void *b,
                            void *out, hipStream_t st) {
    if (dw_tiled(p, pass)) return launch_depthwise_tiled(dtype, pass, p, a, b, out, st);
    if (dtype == Half::id) return launch_dw_t<Half>(pass, p, a, b, out, st);
    return launch_dw_t<BFloat>(pass, p, a, b, out, st);
}

}  // namespace nnconv
