// depthwise_tiled.hip -- LDS-tiled depthwise convolution for the common
// shapes: equal strides of 1 or 2, no dilation, channel-last, fp16/bf16
// operands with fp32 accumulation.
//
// The gather kernels in depthwise.hip keep one input row per thread in
// flight and so wait on memory latency once per row.  Here a workgroup first
// stages a whole input tile (with its halo) in LDS, every load of the tile
// in flight at once, and then computes from LDS:
//   - forward, and backward-data at stride 1 (the forward correlation of dy
//     with the filter rotated by 180 degrees and padding R-1-pad): a
//     workgroup owns TH x TW output pixels of CBV 8-channel vectors; thread
//     (vector, column, row group) computes TP output rows of one column and
//     reads each input row of its strip once; the weights of its 8 channels
//     stay in registers (LDS for 7x7);
//   - backward-data at stride 2: a workgroup owns a tile of dx and the dy
//     pixels it reaches; each output adds only the taps of its row and
//     column parity;
//   - backward-weight: a workgroup owns one channel block and a run of
//     spatial tiles of dy; thread (vector, filter row r, dy row) adds the S
//     taps of filter row r over its dy row with a sliding window of input
//     vectors; the next tile's loads are in flight while the current one is
//     added in; the workgroup then sums its threads in a fixed order and
//     writes one fp32 partial per split for the shared split reduction.
// At stride 2 the tile's input columns are stored even columns first, then
// odd ones, so the lanes of a wave read consecutive LDS addresses.
#include <cstring>

#include "launch.hpp"

namespace nnconv {

namespace dwt {

// acc[k] += x[k] * w[k] for the 8 channels of two 16-byte vectors (two
// channels per 32-bit word).  fp16: v_fma_mix_f32 takes both 16-bit operands
// straight from the packed words, so nothing is converted or kept as fp32
// (its single rounding of the exact product is that of fmaf on the widened
// values).  bf16: widening is a shift or a mask; with CONV_AT_USE the w
// operand is widened at every use instead of being kept widened across uses,
// which would hold R*S*8 fp32 weights in registers.
template <class T, bool CONV_AT_USE>
__device__ __forceinline__ void fma8(float (&acc)[8], u32x4 x, u32x4 w) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if constexpr (T::id == Half::id) {
            asm("v_fma_mix_f32 %0, %1, %2, %0 op_sel_hi:[1,1,0]"
                : "+v"(acc[2 * i])
                : "v"(x[i]), "v"(w[i]));
            asm("v_fma_mix_f32 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,1,0]"
                : "+v"(acc[2 * i + 1])
                : "v"(x[i]), "v"(w[i]));
        } else {
            const float xlo = __builtin_bit_cast(float, x[i] << 16);
            const float xhi = __builtin_bit_cast(float, x[i] & 0xFFFF0000u);
            if constexpr (CONV_AT_USE) {
                // widen and multiply-add in one block: the widened value
                // lives in a scratch register of the block only
                float t;
                asm("v_lshlrev_b32 %1, 16, %3\n\tv_fmac_f32 %0, %2, %1"
                    : "+v"(acc[2 * i]), "=&v"(t)
                    : "v"(xlo), "v"(w[i]));
                asm("v_and_b32 %1, 0xffff0000, %3\n\tv_fmac_f32 %0, %2, %1"
                    : "+v"(acc[2 * i + 1]), "=&v"(t)
                    : "v"(xhi), "v"(w[i]));
            } else {
                acc[2 * i] = __builtin_fmaf(xlo, __builtin_bit_cast(float, w[i] << 16), acc[2 * i]);
                acc[2 * i + 1] =
                    __builtin_fmaf(xhi, __builtin_bit_cast(float, w[i] & 0xFFFF0000u), acc[2 * i + 1]);
            }
        }
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

// LDS column of tile input column c (stride 2: even columns, then odd ones)
template <int SH, int HALF>
__device__ __forceinline__ int colmap(int c) {
    return SH == 1 ? c : (c & 1) * HALF + (c >> 1);
}
// LDS column of input column col*SH + s, with s known at compile time
template <int SH, int HALF>
__device__ __forceinline__ int tapcol(int col, int s) {
    return SH == 1 ? col + s : (s & 1) * HALF + col + (s >> 1);
}

// Forward tile: 256 threads = CBV vectors x TW columns x RG row groups of TP
// rows.  Input tile IH x IW pixels.  The narrow tile (stride 1) has half the
// columns and half the rows per thread, for images narrower than the wide
// tile (7x7).
template <int R, int SH, int CBV, bool NARROW>
struct FwdTile {
    static constexpr int TPW = (SH == 1 && R <= 5) ? 4 : 2;
    static constexpr int TWW = SH == 1 ? (CBV == 2 ? 32 : 16) : 64 / CBV;
    static constexpr int TP = NARROW ? (TPW > 1 ? TPW / 2 : 1) : TPW;
    static constexpr int TW = NARROW ? TWW / 2 : TWW;
    static constexpr int RG = 256 / (CBV * TW);
    static constexpr int TH = RG * TP;
    static constexpr int IH = (TH - 1) * SH + R;
    static constexpr int IW = (TW - 1) * SH + R;
    static constexpr int HALF = (IW + 1) / 2;
    static constexpr int CHUNKS = IH * IW * CBV;  // 16-byte vectors
    static constexpr int NL = (CHUNKS + 255) / 256;
    static constexpr bool WREG = R <= 5;
};

// Stride-2 backward-data tile: TH x TW dx pixels, laid out over the threads
// like the stride-1 forward tile; dy tile DH x DW pixels.  Each output takes
// the taps of its row and column parity: ceil(R/2) or floor(R/2) filter rows
// and columns.
template <int R, int CBV, bool NARROW>
struct Dg2Tile {
    static constexpr int TP = (R <= 5 && !NARROW) ? 4 : 2;  // even: a strip starts on an even row
    static constexpr int TW = (CBV == 2 ? 32 : 16) / (NARROW ? 2 : 1);
    static constexpr int RG = 256 / (CBV * TW);
    static constexpr int TH = RG * TP;
    static constexpr int DH = (TH + R + 1) / 2;
    static constexpr int DW = (TW + R + 1) / 2;
    static constexpr int CHUNKS = DH * DW * CBV;
    static constexpr int NL = (CHUNKS + 255) / 256;
    static constexpr int KS = (R + 1) / 2;  // column taps of one parity (the last may be absent)
};

// Backward-weight tile: dy rows (at most GMAX, one per thread row group) x
// TW dy columns; input tile ((rows-1)*SH + R) x XW pixels, its rows XWP
// vectors apart (XWP = 1 mod 16/CBV, so the R filter rows read by one
// 16-lane LDS pass fall in different banks).
template <int R, int SH, int CBV>
struct WgTile {
    static constexpr int GMAX = 256 / (CBV * R);
    static constexpr int TW = SH == 1 ? 8 : 4;
    static constexpr int XW = (TW - 1) * SH + R;
    static constexpr int M = 16 / CBV;
    static constexpr int XWP = XW + ((1 - XW) % M + M) % M;
    static constexpr int XHMAX = (GMAX - 1) * SH + R;
    static constexpr int XCH = XHMAX * XW * CBV;
    static constexpr int DCH = GMAX * TW * CBV;
    static constexpr int NLX = (XCH + 255) / 256;
    static constexpr int NLD = (DCH + 255) / 256;
};

}  // namespace dwt

// out[n, o, u, c] = alpha * sum_{r,s} in[n, o*SH - ph + r, u*SH - pw + s, c] * w'[c, r, s]
// with w' = w, or w rotated by 180 degrees (FLIP).
template <class T, int R, int SH, int CBV, bool NARROW, bool FLIP>
__global__ __launch_bounds__(256) void dwt_fwd_kernel(const DWTParams P,
                                                      const uint16_t *__restrict__ in,
                                                      const uint16_t *__restrict__ w,
                                                      uint16_t *__restrict__ out) {
    using namespace dwt;
    using F = FwdTile<R, SH, CBV, NARROW>;
    constexpr int S = R, RS = R * S, CW = CBV * 8;
    __shared__ u32x4 tile[F::CHUNKS];
    __shared__ __attribute__((aligned(16))) uint16_t wl[RS][CW];
    const int tid = threadIdx.x;

    // block -> (channel block, tile column, tile row, image); consecutive
    // tiles, which share halo pixels, run on one XCD
    uint32_t b = xcd_remap(blockIdx.x, gridDim.x);
    const int cb = (int)(b % (uint32_t)P.cblocks);
    b /= (uint32_t)P.cblocks;
    const int tw = (int)(b % (uint32_t)P.tiles_w);
    b /= (uint32_t)P.tiles_w;
    const int th = (int)(b % (uint32_t)P.tiles_h);
    const int n = (int)(b / (uint32_t)P.tiles_h);
    const int oh0 = th * F::TH, ow0 = tw * F::TW;
    const int ih0 = oh0 * SH - P.ph, iw0 = ow0 * SH - P.pw;

    // the whole input tile in flight; outside the image (or past the last
    // channel vector) the range check returns zeros
    const __amdgpu_buffer_rsrc_t rin = make_rsrc(in, P.in_bytes);
    const uint32_t img = (uint32_t)n * (uint32_t)P.ih;
    u32x4 ld[F::NL];
#pragma unroll
    for (int k = 0; k < F::NL; ++k) {
        const int e = k * 256 + tid;
        const int row = e / (F::IW * CBV);
        const int rem = e - row * (F::IW * CBV);
        const int col = rem / CBV, cvl = rem - col * CBV;
        const int h = ih0 + row, wc = iw0 + col, cvec = cb * CBV + cvl;
        const bool ok = e < F::CHUNKS && (unsigned)h < (unsigned)P.ih &&
                        (unsigned)wc < (unsigned)P.iw && cvec < P.c8;
        const uint32_t off = ((img + (uint32_t)h) * (uint32_t)P.iw + (uint32_t)wc) * (uint32_t)P.c * 2u +
                             (uint32_t)cvec * 16u;
        ld[k] = load16(rin, ok ? off : OOB_OFFSET);
    }
    // weights of the block's channels as [tap][channel]; in memory they are
    // [C][R*S], so the block is one contiguous run
    for (int e = tid; e < RS * CW; e += 256) {
        const int cl = e / RS, t = e - cl * RS;
        const int ch = cb * CW + cl;
        wl[t][cl] = ch < P.c ? w[(int64_t)ch * RS + (FLIP ? RS - 1 - t : t)] : (uint16_t)0;
    }
#pragma unroll
    for (int k = 0; k < F::NL; ++k) {
        const int e = k * 256 + tid;
        if (F::NL * 256 == F::CHUNKS || e < F::CHUNKS) {
            const int row = e / (F::IW * CBV);
            const int rem = e - row * (F::IW * CBV);
            const int col = rem / CBV, cvl = rem - col * CBV;
            tile[(row * F::IW + colmap<SH, F::HALF>(col)) * CBV + cvl] = ld[k];
        }
    }
    __syncthreads();

    // thread: vector cv of column col, output rows rg*TP .. rg*TP + TP-1
    const int cv = tid % CBV;
    const int col = (tid / CBV) % F::TW;
    const int rg = tid / (CBV * F::TW);
    u32x4 wr[F::WREG ? RS : 1];
    if constexpr (F::WREG) {
#pragma unroll
        for (int t = 0; t < RS; ++t) wr[t] = *(const u32x4 *)&wl[t][cv * 8];
    }
    float acc[F::TP][8];
#pragma unroll
    for (int i = 0; i < F::TP; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[i][k] = 0.f;

    // input rows of the strip: tile row rg*TP*SH + hh feeds output row i
    // through filter row hh - i*SH
    const u32x4 *trow = tile + rg * F::TP * SH * F::IW * CBV + cv;
#pragma unroll
    for (int hh = 0; hh < (F::TP - 1) * SH + R; ++hh) {
        u32x4 xv[S];
#pragma unroll
        for (int s = 0; s < S; ++s) xv[s] = trow[(hh * F::IW + tapcol<SH, F::HALF>(col, s)) * CBV];
#pragma unroll
        for (int i = 0; i < F::TP; ++i) {
            const int r = hh - i * SH;
            if (r < 0 || r >= R) continue;
#pragma unroll
            for (int s = 0; s < S; ++s) {
                u32x4 wv;
                if constexpr (F::WREG)
                    wv = wr[r * S + s];
                else
                    wv = *(const u32x4 *)&wl[r * S + s][cv * 8];
                fma8<T, true>(acc[i], xv[s], wv);
            }
        }
    }

    const int cvec = cb * CBV + cv;
    const int ow = ow0 + col;
    if (cvec < P.c8 && ow < P.ow) {
        uint16_t *o = out + ((int64_t)n * P.oh * P.ow + ow) * P.c + cvec * 8;
#pragma unroll
        for (int i = 0; i < F::TP; ++i) {
            const int oh = oh0 + rg * F::TP + i;
            if (oh < P.oh) *(u32x4 *)(o + (int64_t)oh * P.ow * P.c) = pack8<T>(acc[i], P.alpha);
        }
    }
}

// Stride 2: dx[n, i, j, c] = alpha * sum over the taps (r, s) with i + ph - r
// and j + pw - s even of dy[n, (i+ph-r)/2, (j+pw-s)/2, c] * w[c, r, s].
// PHP = ph % 2 fixes, for each strip row, which filter rows reach it; the
// column parity varies by lane and selects the lane's weight columns once.
template <class T, int R, int CBV, bool NARROW, int PHP>
__global__ __launch_bounds__(256) void dwt_dgrad2_kernel(const DWTParams P,
                                                         const uint16_t *__restrict__ dy,
                                                         const uint16_t *__restrict__ w,
                                                         uint16_t *__restrict__ dx) {
    using namespace dwt;
    using G = Dg2Tile<R, CBV, NARROW>;
    constexpr int S = R, RS = R * S, CW = CBV * 8, KS = G::KS;
    __shared__ u32x4 tile[G::CHUNKS];
    __shared__ __attribute__((aligned(16))) uint16_t wl[R * (S + 1)][CW];  // column S: zeros
    const int tid = threadIdx.x;

    uint32_t b = xcd_remap(blockIdx.x, gridDim.x);
    const int cb = (int)(b % (uint32_t)P.cblocks);
    b /= (uint32_t)P.cblocks;
    const int tw = (int)(b % (uint32_t)P.tiles_w);
    b /= (uint32_t)P.tiles_w;
    const int th = (int)(b % (uint32_t)P.tiles_h);
    const int n = (int)(b / (uint32_t)P.tiles_h);
    const int i0 = th * G::TH, j0 = tw * G::TW;  // both even
    // first dy row / column any output of the tile reaches (floor division)
    const int p0 = (i0 + P.ph - (R - 1)) >> 1;
    const int q0 = (j0 + P.pw - (S - 1)) >> 1;

    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(dy, P.in_bytes);
    const uint32_t img = (uint32_t)n * (uint32_t)P.ih;
    u32x4 ld[G::NL];
#pragma unroll
    for (int k = 0; k < G::NL; ++k) {
        const int e = k * 256 + tid;
        const int row = e / (G::DW * CBV);
        const int rem = e - row * (G::DW * CBV);
        const int col = rem / CBV, cvl = rem - col * CBV;
        const int p = p0 + row, q = q0 + col, cvec = cb * CBV + cvl;
        const bool ok = e < G::CHUNKS && (unsigned)p < (unsigned)P.ih && (unsigned)q < (unsigned)P.iw &&
                        cvec < P.c8;
        const uint32_t off = ((img + (uint32_t)p) * (uint32_t)P.iw + (uint32_t)q) * (uint32_t)P.c * 2u +
                             (uint32_t)cvec * 16u;
        ld[k] = load16(rdy, ok ? off : OOB_OFFSET);
    }
    for (int e = tid; e < R * (S + 1) * CW; e += 256) {
        const int cl = e / (R * (S + 1)), t = e - cl * (R * (S + 1));
        const int r = t / (S + 1), sc = t - r * (S + 1);
        const int ch = cb * CW + cl;
        wl[t][cl] = (sc < S && ch < P.c) ? w[(int64_t)ch * RS + r * S + sc] : (uint16_t)0;
    }
#pragma unroll
    for (int k = 0; k < G::NL; ++k) {
        const int e = k * 256 + tid;
        if (G::NL * 256 == G::CHUNKS || e < G::CHUNKS) tile[e] = ld[k];
    }
    __syncthreads();

    const int cv = tid % CBV;
    const int col = (tid / CBV) % G::TW;
    const int rg = tid / (CBV * G::TW);
    // columns s = s0, s0 + 2, ... reach this lane's output column
    const int s0 = (col + P.pw) & 1;
    u32x4 wr[R][KS];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int k = 0; k < KS; ++k) wr[r][k] = *(const u32x4 *)&wl[r * (S + 1) + s0 + 2 * k][cv * 8];
    // dy tile column of tap s0 + 2k: qb - k
    const int qb = ((P.pw & 1) + col + S - 1 - s0) >> 1;
    float acc[G::TP][8];
#pragma unroll
    for (int t = 0; t < G::TP; ++t)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[t][k] = 0.f;
#pragma unroll
    for (int t = 0; t < G::TP; ++t) {
#pragma unroll
        for (int r = (t + PHP) & 1; r < R; r += 2) {
            // dy tile row of output row i0 + rg*TP + t through filter row r
            const int prow = rg * (G::TP / 2) + (PHP + t + R - 1 - r) / 2;
            const u32x4 *trow = tile + (prow * G::DW + qb) * CBV + cv;
#pragma unroll
            for (int k = 0; k < KS; ++k) {
                if (S % 2 == 1 && k == KS - 1 && s0 == 1) continue;  // tap s0 + 2k == S
                fma8<T, true>(acc[t], trow[-k * CBV], wr[r][k]);
            }
        }
    }

    const int cvec = cb * CBV + cv;
    const int j = j0 + col;
    if (cvec < P.c8 && j < P.ow) {
        uint16_t *o = dx + ((int64_t)n * P.oh * P.ow + j) * P.c + cvec * 8;
#pragma unroll
        for (int t = 0; t < G::TP; ++t) {
            const int i = i0 + rg * G::TP + t;
            if (i < P.oh) *(u32x4 *)(o + (int64_t)i * P.ow * P.c) = pack8<T>(acc[t], P.alpha);
        }
    }
}

// Partials of dw[c, r, s] = sum_pix dy[n, p, q, c] * x[n, p*SH - ph + r, q*SH - pw + s, c]
// over the tiles of one split: ws[split][c][r*S + s].
template <class T, int R, int SH, int CBV>
__global__ __launch_bounds__(256) void dwt_wgrad_kernel(const DWTParams P,
                                                        const uint16_t *__restrict__ x,
                                                        const uint16_t *__restrict__ dy,
                                                        float *__restrict__ ws) {
    using namespace dwt;
    using W = WgTile<R, SH, CBV>;
    constexpr int S = R;
    __shared__ u32x4 xt[W::XHMAX * W::XWP * CBV];
    __shared__ u32x4 dt[W::DCH];
    __shared__ float red[256 * 8];
    const int tid = threadIdx.x;
    // the channel blocks of one split run back to back on one XCD: a block
    // of fewer than 8 vectors uses only part of each 128-byte line, and the
    // other blocks' workgroups then find the rest in the same L2
    const uint32_t b = xcd_remap(blockIdx.x, gridDim.x);
    const int cb = (int)(b % (uint32_t)P.cblocks);
    const int split = (int)(b / (uint32_t)P.cblocks);
    const int ntiles = P.n * P.tiles_h * P.tiles_w;
    const int t_begin = split * P.tiles_per_split;
    const int t_end = min(ntiles, t_begin + P.tiles_per_split);
    const int TH = P.th;
    const int xch = ((TH - 1) * SH + R) * W::XW * CBV;  // input vectors of a tile
    const int dch = TH * W::TW * CBV;                   // dy vectors of a tile

    // role: vector cv, filter row r, dy row g of the tile
    const int cv = tid % CBV;
    const int r = (tid / CBV) % R;
    const int g = tid / (CBV * R);
    const bool active = g < TH;

    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, P.in_bytes);
    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(dy, P.dy_bytes);
    u32x4 lx[W::NLX], ldy[W::NLD];
    auto issue = [&](int t) {
        const int tw = t % P.tiles_w;
        const int t2 = t / P.tiles_w;
        const int th = t2 % P.tiles_h;
        const int n = t2 / P.tiles_h;
        const int p0 = th * TH, q0 = tw * W::TW;
        const int h0 = p0 * SH - P.ph, w0 = q0 * SH - P.pw;
#pragma unroll
        for (int k = 0; k < W::NLX; ++k) {
            const int e = k * 256 + tid;
            const int row = e / (W::XW * CBV);
            const int rem = e - row * (W::XW * CBV);
            const int col = rem / CBV, cvl = rem - col * CBV;
            const int h = h0 + row, wc = w0 + col, cvec = cb * CBV + cvl;
            const bool ok = e < xch && (unsigned)h < (unsigned)P.ih && (unsigned)wc < (unsigned)P.iw &&
                            cvec < P.c8;
            const uint32_t off =
                (((uint32_t)n * (uint32_t)P.ih + (uint32_t)h) * (uint32_t)P.iw + (uint32_t)wc) *
                    (uint32_t)P.c * 2u +
                (uint32_t)cvec * 16u;
            lx[k] = load16(rx, ok ? off : OOB_OFFSET);
        }
#pragma unroll
        for (int k = 0; k < W::NLD; ++k) {
            const int e = k * 256 + tid;
            const int row = e / (W::TW * CBV);
            const int rem = e - row * (W::TW * CBV);
            const int col = rem / CBV, cvl = rem - col * CBV;
            const int p = p0 + row, q = q0 + col, cvec = cb * CBV + cvl;
            const bool ok = e < dch && p < P.oh && q < P.ow && cvec < P.c8;
            const uint32_t off =
                (((uint32_t)n * (uint32_t)P.oh + (uint32_t)p) * (uint32_t)P.ow + (uint32_t)q) *
                    (uint32_t)P.c * 2u +
                (uint32_t)cvec * 16u;
            ldy[k] = load16(rdy, ok ? off : OOB_OFFSET);
        }
    };
    auto commit = [&]() {
#pragma unroll
        for (int k = 0; k < W::NLX; ++k) {
            const int e = k * 256 + tid;
            if (e < xch) {
                const int row = e / (W::XW * CBV);
                const int rem = e - row * (W::XW * CBV);
                const int col = rem / CBV, cvl = rem - col * CBV;
                xt[(row * W::XWP + col) * CBV + cvl] = lx[k];
            }
        }
#pragma unroll
        for (int k = 0; k < W::NLD; ++k) {
            const int e = k * 256 + tid;
            if (e < dch) dt[e] = ldy[k];
        }
    };

    float acc[S][8];
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[s][k] = 0.f;

    if (t_begin < t_end) issue(t_begin);
    for (int t = t_begin; t < t_end; ++t) {
        __syncthreads();  // the previous tile has been read
        commit();
        __syncthreads();
        if (t + 1 < t_end) issue(t + 1);  // in flight while this tile is added in
        if (active) {
            const u32x4 *xr = xt + (g * SH + r) * W::XWP * CBV + cv;
            const u32x4 *dr = dt + g * W::TW * CBV + cv;
            // input columns j*SH .. j*SH + S-1 for dy column j; each column
            // is read from LDS once
            u32x4 xc[W::XW];
#pragma unroll
            for (int j = 0; j < W::TW; ++j) {
                const int lo = j == 0 ? 0 : (j - 1) * SH + S;
#pragma unroll
                for (int ci = lo; ci < j * SH + S; ++ci) xc[ci] = xr[ci * CBV];
                const u32x4 gv = dr[j * CBV];
#pragma unroll
                for (int s = 0; s < S; ++s) fma8<T, false>(acc[s], xc[j * SH + s], gv);
            }
        }
    }

    // sum the dy-row groups in order, one filter column at a time; thread
    // tid = (g*R + r)*CBV + cv holds acc[s][k] for channel vector cv
    for (int s = 0; s < S; ++s) {
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 8; ++k) red[tid * 8 + k] = acc[s][k];
        __syncthreads();
        for (int e = tid; e < CBV * R * 8; e += 256) {
            const int k = e % 8, cr = e / 8;
            float sum = 0.f;
            for (int gg = 0; gg < TH; ++gg) sum += red[(gg * CBV * R + cr) * 8 + k];
            const int ch = (cb * CBV + cr % CBV) * 8 + k;
            if (ch < P.c) ws[((int64_t)split * P.c + ch) * (R * S) + (cr / CBV) * S + s] = sum;
        }
    }
}

namespace {

constexpr int CBV_CHOICES[3] = {8, 4, 2};

// tile sizes (rows, columns, rows per thread) without instantiating the
// kernels: kind 0 = forward / stride-1 backward-data, 1 = stride-2
// backward-data
void tile_dims(int kind, int r, int sh, int cbv, bool narrow, int *th, int *tw, int *tp) {
    if (kind == 0) {
        const int tpw = (sh == 1 && r <= 5) ? 4 : 2;
        const int tww = sh == 1 ? (cbv == 2 ? 32 : 16) : 64 / cbv;
        *tp = narrow ? (tpw > 1 ? tpw / 2 : 1) : tpw;
        *tw = narrow ? tww / 2 : tww;
    } else {
        *tp = (r <= 5 && !narrow) ? 4 : 2;
        *tw = (cbv == 2 ? 32 : 16) / (narrow ? 2 : 1);
    }
    *th = 256 / (cbv * *tw) * *tp;
}

// The (CBV, narrow) pair with the least work: workgroups x rows per thread
// (every thread of a workgroup computes its rows, inside the image or not);
// ties go to the wide tile and the wider block.  Narrow tiles only at
// stride 1 (kind 0) or for backward-data.
struct TilePick {
    int cbv;
    bool narrow;
};
TilePick pick_tile(const DWTParams &q, int kind, int r, int sh) {
    TilePick best = {8, false};
    int64_t best_cost = -1;
    for (int nw = 0; nw < 2; ++nw) {
        if (nw && kind == 0 && sh != 1) continue;
        for (int cbv : CBV_CHOICES) {
            int th, tw, tp;
            tile_dims(kind, r, sh, cbv, nw != 0, &th, &tw, &tp);
            const int64_t cost = (int64_t)((q.c8 + cbv - 1) / cbv) * ((q.oh + th - 1) / th) *
                                 ((q.ow + tw - 1) / tw) * tp;
            if (best_cost < 0 || cost < best_cost) {
                best = {cbv, nw != 0};
                best_cost = cost;
            }
        }
    }
    return best;
}

template <class T, int R, int SH, int CBV, bool NARROW, bool FLIP>
hipError_t launch_fwd_cfg(DWTParams q, const void *in, const void *w, void *out, hipStream_t st) {
    using F = dwt::FwdTile<R, SH, CBV, NARROW>;
    q.cblocks = (q.c8 + CBV - 1) / CBV;
    q.tiles_h = (q.oh + F::TH - 1) / F::TH;
    q.tiles_w = (q.ow + F::TW - 1) / F::TW;
    const int64_t nb = (int64_t)q.n * q.tiles_h * q.tiles_w * q.cblocks;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((dwt_fwd_kernel<T, R, SH, CBV, NARROW, FLIP>), dim3((uint32_t)nb), dim3(256), 0,
                       st, q, (const uint16_t *)in, (const uint16_t *)w, (uint16_t *)out);
    return hipGetLastError();
}

template <class T, int R, int SH, bool FLIP>
hipError_t launch_fwd_rs(const DWTParams &q, const void *in, const void *w, void *out, hipStream_t st) {
    const TilePick t = pick_tile(q, 0, R, SH);
    if constexpr (SH == 1) {
        if (t.narrow) {
            switch (t.cbv) {
                case 2: return launch_fwd_cfg<T, R, SH, 2, true, FLIP>(q, in, w, out, st);
                case 4: return launch_fwd_cfg<T, R, SH, 4, true, FLIP>(q, in, w, out, st);
                default: return launch_fwd_cfg<T, R, SH, 8, true, FLIP>(q, in, w, out, st);
            }
        }
    }
    switch (t.cbv) {
        case 2: return launch_fwd_cfg<T, R, SH, 2, false, FLIP>(q, in, w, out, st);
        case 4: return launch_fwd_cfg<T, R, SH, 4, false, FLIP>(q, in, w, out, st);
        default: return launch_fwd_cfg<T, R, SH, 8, false, FLIP>(q, in, w, out, st);
    }
}

template <class T, bool FLIP>
hipError_t launch_fwd_t(const DWTParams &q, int r, int sh, const void *in, const void *w, void *out,
                        hipStream_t st) {
    if (sh == 1) {
        switch (r) {
            case 3: return launch_fwd_rs<T, 3, 1, FLIP>(q, in, w, out, st);
            case 5: return launch_fwd_rs<T, 5, 1, FLIP>(q, in, w, out, st);
            case 7: return launch_fwd_rs<T, 7, 1, FLIP>(q, in, w, out, st);
        }
    } else if constexpr (!FLIP) {
        switch (r) {
            case 3: return launch_fwd_rs<T, 3, 2, FLIP>(q, in, w, out, st);
            case 5: return launch_fwd_rs<T, 5, 2, FLIP>(q, in, w, out, st);
            case 7: return launch_fwd_rs<T, 7, 2, FLIP>(q, in, w, out, st);
        }
    }
    return hipErrorInvalidValue;
}

template <class T, int R, int CBV, bool NARROW, int PHP>
hipError_t launch_dgrad2_cfg(DWTParams q, const void *dy, const void *w, void *dx, hipStream_t st) {
    using G = dwt::Dg2Tile<R, CBV, NARROW>;
    q.cblocks = (q.c8 + CBV - 1) / CBV;
    q.tiles_h = (q.oh + G::TH - 1) / G::TH;
    q.tiles_w = (q.ow + G::TW - 1) / G::TW;
    const int64_t nb = (int64_t)q.n * q.tiles_h * q.tiles_w * q.cblocks;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((dwt_dgrad2_kernel<T, R, CBV, NARROW, PHP>), dim3((uint32_t)nb), dim3(256), 0, st,
                       q, (const uint16_t *)dy, (const uint16_t *)w, (uint16_t *)dx);
    return hipGetLastError();
}

template <class T, int R, int PHP>
hipError_t launch_dgrad2_rs(const DWTParams &q, const void *dy, const void *w, void *dx, hipStream_t st) {
    const TilePick t = pick_tile(q, 1, R, 2);
    if (t.narrow) {
        switch (t.cbv) {
            case 2: return launch_dgrad2_cfg<T, R, 2, true, PHP>(q, dy, w, dx, st);
            case 4: return launch_dgrad2_cfg<T, R, 4, true, PHP>(q, dy, w, dx, st);
            default: return launch_dgrad2_cfg<T, R, 8, true, PHP>(q, dy, w, dx, st);
        }
    }
    switch (t.cbv) {
        case 2: return launch_dgrad2_cfg<T, R, 2, false, PHP>(q, dy, w, dx, st);
        case 4: return launch_dgrad2_cfg<T, R, 4, false, PHP>(q, dy, w, dx, st);
        default: return launch_dgrad2_cfg<T, R, 8, false, PHP>(q, dy, w, dx, st);
    }
}

template <class T, int PHP>
hipError_t launch_dgrad2_t(const DWTParams &q, int r, const void *dy, const void *w, void *dx,
                           hipStream_t st) {
    switch (r) {
        case 3: return launch_dgrad2_rs<T, 3, PHP>(q, dy, w, dx, st);
        case 5: return launch_dgrad2_rs<T, 5, PHP>(q, dy, w, dx, st);
        case 7: return launch_dgrad2_rs<T, 7, PHP>(q, dy, w, dx, st);
    }
    return hipErrorInvalidValue;
}

int wg_gmax(int r, int cbv) { return 256 / (cbv * r); }

// Backward-weight tiling: per CBV, dy rows per tile balanced over the image
// height (at most GMAX); the CBV with the fewest (channel block, tile) pairs.
// Splits: about 1024 workgroups (four per compute unit); more splits cost more
// than the extra parallelism gives, since each workgroup then walks too few tiles
// to hide its prefetch.
DWWgPlan plan_wgrad(const DWParams &p) {
    DWWgPlan pl;
    const int tw = p.sh == 1 ? 8 : 4;
    int64_t best_cost = -1;
    for (int cbv : CBV_CHOICES) {
        const int gmax = wg_gmax(p.r, cbv);
        const int nth = (p.p + gmax - 1) / gmax;
        const int th = nth > 0 ? (p.p + nth - 1) / nth : 1;
        const int tiles_h = th > 0 ? (p.p + th - 1) / th : 0;
        const int tiles_w = (p.q + tw - 1) / tw;
        const int cblocks = (p.c8 + cbv - 1) / cbv;
        const int64_t cost = (int64_t)cblocks * p.n * tiles_h * tiles_w;
        if (best_cost < 0 || cost < best_cost) {
            best_cost = cost;
            pl.cbv = cbv;
            pl.th = th < 1 ? 1 : th;
            pl.tiles_h = tiles_h;
            pl.tiles_w = tiles_w;
            pl.cblocks = cblocks;
        }
    }
    const int64_t ntiles = (int64_t)p.n * pl.tiles_h * pl.tiles_w;
    if (ntiles <= 0) {
        pl.splits = 1;
        pl.tiles_per_split = 0;
        return pl;
    }
    int64_t splits = 1024 / pl.cblocks;
    if (splits < 1) splits = 1;
    if (splits > ntiles) splits = ntiles;
    if (splits > 65535) splits = 65535;
    const int64_t per = (ntiles + splits - 1) / splits;
    pl.tiles_per_split = (int32_t)per;
    pl.splits = (int32_t)((ntiles + per - 1) / per);
    return pl;
}

template <class T, int R, int SH, int CBV>
hipError_t launch_wgrad_cfg(const DWParams &p, const DWWgPlan &pl, const void *x, const void *dy,
                            float *ws, hipStream_t st) {
    DWTParams q;
    memset(&q, 0, sizeof(q));
    q.n = p.n; q.c = p.c; q.c8 = p.c8; q.cblocks = pl.cblocks;
    q.ih = p.h; q.iw = p.w; q.oh = p.p; q.ow = p.q;
    q.ph = p.ph; q.pw = p.pw;
    q.tiles_h = pl.tiles_h; q.tiles_w = pl.tiles_w;
    q.th = pl.th;
    q.tiles_per_split = pl.tiles_per_split;
    q.splits = pl.splits;
    q.in_bytes = p.x_bytes; q.dy_bytes = p.dy_bytes;
    q.alpha = 1.f;
    if (pl.th > dwt::WgTile<R, SH, CBV>::GMAX || pl.splits != p.splits) return hipErrorInvalidValue;
    const int64_t nb = (int64_t)pl.cblocks * pl.splits;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((dwt_wgrad_kernel<T, R, SH, CBV>), dim3((uint32_t)nb), dim3(256), 0, st, q,
                       (const uint16_t *)x, (const uint16_t *)dy, ws);
    return hipGetLastError();
}

template <class T, int R, int SH>
hipError_t launch_wgrad_rs(const DWParams &p, const DWWgPlan &pl, const void *x, const void *dy,
                           float *ws, hipStream_t st) {
    switch (pl.cbv) {
        case 2: return launch_wgrad_cfg<T, R, SH, 2>(p, pl, x, dy, ws, st);
        case 4: return launch_wgrad_cfg<T, R, SH, 4>(p, pl, x, dy, ws, st);
        default: return launch_wgrad_cfg<T, R, SH, 8>(p, pl, x, dy, ws, st);
    }
}

template <class T>
hipError_t launch_wgrad_t(const DWParams &p, const void *x, const void *dy, float *ws, hipStream_t st) {
    const DWWgPlan pl = plan_wgrad(p);
    if (p.sh == 1) {
        switch (p.r) {
            case 3: return launch_wgrad_rs<T, 3, 1>(p, pl, x, dy, ws, st);
            case 5: return launch_wgrad_rs<T, 5, 1>(p, pl, x, dy, ws, st);
            case 7: return launch_wgrad_rs<T, 7, 1>(p, pl, x, dy, ws, st);
        }
    } else {
        switch (p.r) {
            case 3: return launch_wgrad_rs<T, 3, 2>(p, pl, x, dy, ws, st);
            case 5: return launch_wgrad_rs<T, 5, 2>(p, pl, x, dy, ws, st);
            case 7: return launch_wgrad_rs<T, 7, 2>(p, pl, x, dy, ws, st);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool dw_tiled(const DWParams &p, int pass) {
    const bool plain = p.r == p.s && p.sh == p.sw && p.dh == 1 && p.dw == 1 &&
                       (p.r == 3 || p.r == 5 || p.r == 7);
    if (!plain) return false;
    return p.sh == 1 || p.sh == 2;
}

int32_t dw_tiled_wgrad_splits(const DWParams &p) { return plan_wgrad(p).splits; }

hipError_t launch_depthwise_tiled(int dtype, int pass, const DWParams &p, const void *a, const void *b,
                                  void *out, hipStream_t st) {
    if (!dw_tiled(p, pass)) return hipErrorInvalidValue;
    if (pass == 2) {
        if (dtype == Half::id) return launch_wgrad_t<Half>(p, a, b, (float *)out, st);
        return launch_wgrad_t<BFloat>(p, a, b, (float *)out, st);
    }
    DWTParams q;
    memset(&q, 0, sizeof(q));
    q.n = p.n; q.c = p.c; q.c8 = p.c8;
    q.alpha = p.alpha;
    if (pass == 0) {  // x -> y
        q.ih = p.h; q.iw = p.w; q.oh = p.p; q.ow = p.q;
        q.ph = p.ph; q.pw = p.pw;
        q.in_bytes = p.x_bytes;
        if (dtype == Half::id) return launch_fwd_t<Half, false>(q, p.r, p.sh, a, b, out, st);
        return launch_fwd_t<BFloat, false>(q, p.r, p.sh, a, b, out, st);
    }
    q.ih = p.p; q.iw = p.q; q.oh = p.h; q.ow = p.w;
    q.in_bytes = p.dy_bytes;
    if (p.sh == 2) {  // dy -> dx, taps by output parity
        q.ph = p.ph; q.pw = p.pw;
        if (dtype == Half::id)
            return (p.ph & 1) ? launch_dgrad2_t<Half, 1>(q, p.r, a, b, out, st)
                              : launch_dgrad2_t<Half, 0>(q, p.r, a, b, out, st);
        return (p.ph & 1) ? launch_dgrad2_t<BFloat, 1>(q, p.r, a, b, out, st)
                          : launch_dgrad2_t<BFloat, 0>(q, p.r, a, b, out, st);
    }
    // stride 1: dy -> dx with the rotated filter
    q.ph = p.r - 1 - p.ph; q.pw = p.s - 1 - p.pw;
    if (dtype == Half::id) return launch_fwd_t<Half, true>(q, p.r, 1, a, b, out, st);
    return launch_fwd_t<BFloat, true>(q, p.r, 1, a, b, out, st);
}

}  // namespace nnconv
