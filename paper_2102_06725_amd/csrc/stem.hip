// stem.hip -- forward and backward-weight convolution for 8-channel (16-byte)
// or 4-channel (8-byte) pixels and 64 output channels with a fixed filter
// size and stride (the ResNet stem after padding its 3 input channels to 8 or
// 4): a persistent implicit GEMM that stages an input patch and the whole
// filter in LDS instead of gathering an im2col row per (pixel, tap) from L2.
// The 8-channel form is described here; the 4-channel kernels further down.
//
// Output tiles are 16 x 16 pixels of one image.  The input patch of a tile
// ((16-1)*SH + R rows by (16-1)*SW + S columns of 16-byte pixels) arrives in
// LDS with buffer_load ... lds, columns split by phase (column mod SW), so
// the 16 consecutive output pixels of a fragment read 16 consecutive 16-byte
// entries for any tap.  The filter, [64][taps][8] with the tap count padded to
// an even number (the pad tap is zero) and the row stride made odd in 16-byte
// units, stays in LDS for the workgroup's lifetime.  While one tile is
// computed, the next tile's patch is already being loaded into the other
// patch buffer.
//
// GEMM view per tile: rows = 256 output pixels, columns = 64 output channels,
// reduction = taps x 8 channels; one v_mfma_f32_32x32x16 k-step covers two
// taps, so an operand fragment is one 16-byte LDS read per lane.
#include "launch.hpp"

namespace nnconv {

namespace stem {

constexpr int TH = 16, TW = 16;  // output tile
constexpr int K = 64;            // output channels
// Waves per workgroup (one workgroup per CU): two per SIMD, so one wave's
// LDS fragment reads overlap the other's matrix-core work (one wave per SIMD
// left both kernels waiting on LDS latency: 8 waves are 12 % faster for the
// forward and 30 % for the backward-weight kernel; 16 spill registers).
constexpr int FWD_WAVES = 8;
constexpr int WG_WAVES = 8;
static_assert(8 % FWD_WAVES == 0, "forward: whole 32-pixel fragments per wave");
static_assert((TH * TW * 8) % (64 * FWD_WAVES) == 0, "forward: whole store rounds");
static_assert((TH * TW * K / 8) % (64 * WG_WAVES) == 0, "backward-weight: whole dy loads");

template <int R, int S, int SH, int SW>
struct Geo {
    static constexpr int TAPS = R * S;
    static constexpr int TAPS2 = (TAPS + 1) & ~1;           // even, >= TAPS
    static constexpr int WROW = TAPS2 | 1;                  // odd row stride (16-byte units)
    static constexpr int W_ENT = K * WROW;                  // filter entries
    static constexpr int PR = (TH - 1) * SH + R;            // patch rows
    static constexpr int PC = (TW - 1) * SW + S;            // patch columns
    static constexpr int PHC = (PC + SW - 1) / SW;          // columns per phase
    static constexpr int PROW = SW * PHC;                   // entries per patch row
    static constexpr int P_ENT = ((PR * PROW + 63) / 64) * 64;  // whole 1-KB loads
    static constexpr int C_ENT = TH * TW * K / 8;           // output tile, 16-byte chunks
    static constexpr int LDS_ENT = W_ENT + 2 * P_ENT + C_ENT;
};

}  // namespace stem

template <class T, int R, int S, int SH, int SW>
__global__ __launch_bounds__(stem::FWD_WAVES * 64, 1) void stem_fwd_kernel(const StemParams P) {
    constexpr int FR = 8 / stem::FWD_WAVES;  // 32-pixel output fragments per wave
    using namespace stem;
    using G = Geo<R, S, SH, SW>;
    static_assert(G::LDS_ENT * 16 <= 160 * 1024, "LDS budget");
    __shared__ u32x4 lds[G::LDS_ENT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];
    const uint32_t wbase = lds0;
    const uint32_t pbase0 = lds0 + G::W_ENT * 16;

    const i32x4 dx = desc_of(P.x, P.x_bytes);
    const i32x4 dw = desc_of(P.wt, P.wt_bytes);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(P.y, P.y_bytes);

    const int tiles_q = (P.q + TW - 1) / TW, tiles_p = (P.p + TH - 1) / TH;
    const int per_img = tiles_p * tiles_q;
    const int total = P.n * per_img;

    // filter: entry e = k * WROW + t holds w[k][t][0..7]; taps >= R*S are 0
    for (int e0 = wave * 64; e0 < G::W_ENT; e0 += FWD_WAVES * 64) {
        const int e = e0 + lane;
        const int k = e / G::WROW, t = e - k * G::WROW;
        const uint32_t off = (e < G::W_ENT && t < G::TAPS) ? (uint32_t)(k * G::TAPS + t) * 16u
                                                             : OOB_OFFSET;
        dma16(wbase + (uint32_t)e0 * 16u, off, dw);
    }

    // patch of tile `tile` into buffer b
    auto load_patch = [&](int tile, int b) {
        const int n = tile / per_img;
        const int rem = tile - n * per_img;
        const int tp = rem / tiles_q, tq = rem - tp * tiles_q;
        const int ih0 = tp * TH * SH - P.ph, iw0 = tq * TW * SW - P.pw;
        const uint32_t pb = pbase0 + (uint32_t)(b * G::P_ENT) * 16u;
#pragma unroll
        for (int j = 0; j < (G::P_ENT / 64 + FWD_WAVES - 1) / FWD_WAVES; ++j) {
            const int e0 = (j * FWD_WAVES + wave) * 64;
            if (e0 < G::P_ENT) {
                const int e = e0 + lane;
                const int pr = e / G::PROW;
                const int rem2 = e - pr * G::PROW;
                const int ph = rem2 / G::PHC;
                const int pc = (rem2 - ph * G::PHC) * SW + ph;
                const int ih = ih0 + pr, iw = iw0 + pc;
                const bool ok = pr < G::PR && pc < G::PC && (unsigned)ih < (unsigned)P.h &&
                                (unsigned)iw < (unsigned)P.w;
                const uint32_t off = ok ? (uint32_t)((n * P.h + ih) * P.w + iw) * 16u : OOB_OFFSET;
                dma16(pb + (uint32_t)e0 * 16u, off, dx);
            }
        }
    };

    // wave w owns tile pixels 32*FR*w .. (rows 2*FR*w ..); fragment i covers
    // rows 2*FR*w + 2i, + 2i+1; lane l: row + (l&31)/16, column l&15
    const int l32 = lane & 31, khalf = lane >> 5;
    int a_row[FR];
#pragma unroll
    for (int i = 0; i < FR; ++i) a_row[i] = 2 * FR * wave + 2 * i + (l32 >> 4);
    const int a_col = l32 & 15;
    // entry of (output pixel, tap t) within a patch buffer
    auto a_entry = [&](int i, int t) -> int {
        const int r = t / S, s = t - (t / S) * S;
        return (a_row[i] * SH + r) * G::PROW + (s % SW) * G::PHC + a_col + s / SW;
    };

    int tile = blockIdx.x;
    if (tile < total) load_patch(tile, 0);
    wait_vmcnt<0>();
    barrier_lds();

    int buf = 0;
    for (; tile < total; tile += gridDim.x) {
        const int next = tile + gridDim.x;
        if (next < total) load_patch(next, buf ^ 1);

        f32x16 acc[FR][2];
#pragma unroll
        for (int i = 0; i < FR; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
        const u32x4 *pt = &lds[G::W_ENT + buf * G::P_ENT];
        const u32x4 *wt = &lds[0];
#pragma unroll
        for (int ks = 0; ks < G::TAPS2 / 2; ++ks) {
            const int t = 2 * ks + khalf;
            u32x4 fa[FR], fb[2];
#pragma unroll
            for (int i = 0; i < FR; ++i)
                fa[i] = t < G::TAPS ? pt[a_entry(i, t < G::TAPS ? t : 0)] : wt[G::TAPS];
#pragma unroll
            for (int j = 0; j < 2; ++j) fb[j] = wt[(j * 32 + l32) * G::WROW + t];
#pragma unroll
            for (int i = 0; i < FR; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32<T>(fb[j], fa[i], acc[i][j]);
        }

        // epilogue: C tile [256 px][8 chunks of 8 channels] in LDS (chunk
        // swizzled by pixel), then one 16-byte store per lane
        {
            char *cl = (char *)&lds[G::W_ENT + 2 * G::P_ENT];
#pragma unroll
            for (int i = 0; i < FR; ++i) {
                const int px = 32 * FR * wave + 32 * i + l32;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        // lane holds channels 32j + 8e + 4*khalf + {0..3} of pixel px
                        const int c = 4 * j + e;
                        u32x2 pk;
                        pk[0] = to16<T>(acc[i][j][4 * e + 0] * P.alpha) |
                                (to16<T>(acc[i][j][4 * e + 1] * P.alpha) << 16);
                        pk[1] = to16<T>(acc[i][j][4 * e + 2] * P.alpha) |
                                (to16<T>(acc[i][j][4 * e + 3] * P.alpha) << 16);
                        *(u32x2 *)(cl + (px * 8 + (c ^ (px & 7))) * 16 + khalf * 8) = pk;
                    }
                }
            }
        }
        barrier_lds();  // C tile complete; every wave is done with patch `buf`
        {
            const int n = tile / (tiles_p * tiles_q);
            const int rem = tile - n * tiles_p * tiles_q;
            const int tp = rem / tiles_q, tq = rem - tp * tiles_q;
            // always the same number of store instructions per thread (pixels
            // outside the output are discarded by the range check), so the
            // vmcnt wait below counts exactly these stores
#pragma unroll
            for (int it = 0; it < TH * TW * 8 / (64 * FWD_WAVES); ++it) {
                const int idx = it * (64 * FWD_WAVES) + tid;
                const int px = idx >> 3, c = idx & 7;
                const int oh = tp * TH + (px >> 4), ow = tq * TW + (px & 15);
                const uint32_t o = (oh < P.p && ow < P.q)
                                       ? (uint32_t)(((n * P.p + oh) * P.q + ow) * K + c * 8) * 2u
                                       : OOB_OFFSET;
                const u32x4 v = lds[G::W_ENT + 2 * G::P_ENT + px * 8 + (c ^ (px & 7))];
                // non-temporal (cache policy nt): 411 MB of output at batch
                // 256 need not displace the operands of the kernels that
                // follow (measured 1-7% faster for the stem's forward and
                // backward-weight in the ResNet-50 step, depending on the
                // machine)
                __builtin_amdgcn_raw_buffer_store_b128(v, ry, o, 0, 2);
            }
        }
        // the next patch has landed (its loads precede this tile's stores)
        wait_vmcnt<TH * TW * 8 / (64 * FWD_WAVES)>();
        barrier_lds();  // next patch visible; C tile free for reuse
        buf ^= 1;
    }
    wait_vmcnt<0>();
}

// Backward-weight for the same shapes: each persistent workgroup sums
//   part[k][t*8 + c] = sum over its pixels of dy[pix][k] * patch(pix, t)[c]
// over the output tiles blockIdx.x, blockIdx.x + gridDim.x, ... into fp32
// registers and writes one split-K partial (reduced in a fixed order by the
// split reduction).  Per tile the 16x16 dy block ([pixel][64 channels],
// 128-byte rows, 64-byte segments swizzled) and the input patch come in by
// buffer_load ... lds, double-buffered.  The matrix-core operands need 8
// consecutive pixels per lane; the transposing LDS read supplies them: for dy
// a 4-pixel x 16-channel block per 16 lanes, for the patch 4 pixels x
// (2 taps x 8 channels), since consecutive output pixels of a tile row are
// consecutive patch entries.  Patch entries outside the receptive field of
// the tile's in-range output pixels are loaded as zeros, so pixels past the
// output edge (whose dy rows are zero) add exact zeros.
namespace stem {
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// byte offset of (pixel row p, 16-bit channel co) in a 128-byte-row dy tile:
// 64-byte segment s of row p lives at segment s ^ ((p >> 1) & 1)
__device__ __forceinline__ uint32_t dy_off(int p, int co) {
    const int byte = co * 2;
    return (uint32_t)(p * 128 + ((((byte >> 6) ^ ((p >> 1) & 1))) << 6) + (byte & 63));
}

__device__ __forceinline__ u32x4 pack_tr(s16x4 v0, s16x4 v1) {
    u32x4 r;
    r[0] = (uint32_t)(uint16_t)v0[0] | ((uint32_t)(uint16_t)v0[1] << 16);
    r[1] = (uint32_t)(uint16_t)v0[2] | ((uint32_t)(uint16_t)v0[3] << 16);
    r[2] = (uint32_t)(uint16_t)v1[0] | ((uint32_t)(uint16_t)v1[1] << 16);
    r[3] = (uint32_t)(uint16_t)v1[2] | ((uint32_t)(uint16_t)v1[3] << 16);
    return r;
}
}  // namespace stem

template <class T, int R, int S, int SH, int SW>
__global__ __launch_bounds__(stem::WG_WAVES * 64, 1) void stem_wgrad_kernel(const StemParams P, float *part) {
    using namespace stem;
    using G = Geo<R, S, SH, SW>;
    constexpr int CB = (G::TAPS + 3) / 4;            // 32-column blocks (4 taps each)
    constexpr int DY_ENT = TH * TW * K / 8;          // dy tile, 16-byte entries
    constexpr int BUF_ENT = G::P_ENT + DY_ENT;
    constexpr int LDS_ENT = 2 * BUF_ENT + 1;          // + one zero entry
    static_assert(LDS_ENT * 16 <= 160 * 1024, "LDS budget");
    __shared__ u32x4 lds[LDS_ENT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];
    const i32x4 dx = desc_of(P.x, P.x_bytes);
    const i32x4 ddy = desc_of(P.y, P.y_bytes);

    const int tiles_q = (P.q + TW - 1) / TW, tiles_p = (P.p + TH - 1) / TH;
    const int per_img = tiles_p * tiles_q;
    const int total = P.n * per_img;

    if (tid == 0) lds[2 * BUF_ENT] = u32x4{};

    auto load_tile = [&](int tile, int b) {
        const int n = tile / per_img;
        const int rem = tile - n * per_img;
        const int tp = rem / tiles_q, tq = rem - tp * tiles_q;
        const int vh = min(TH, P.p - tp * TH), vw = min(TW, P.q - tq * TW);
        const int prv = (vh - 1) * SH + R, pcv = (vw - 1) * SW + S;  // receptive field
        const int ih0 = tp * TH * SH - P.ph, iw0 = tq * TW * SW - P.pw;
        const uint32_t pb = lds0 + (uint32_t)(b * BUF_ENT) * 16u;
#pragma unroll
        for (int j = 0; j < (G::P_ENT / 64 + WG_WAVES - 1) / WG_WAVES; ++j) {
            const int e0 = (j * WG_WAVES + wave) * 64;
            if (e0 < G::P_ENT) {
                const int e = e0 + lane;
                const int pr = e / G::PROW;
                const int rem2 = e - pr * G::PROW;
                const int ph = rem2 / G::PHC;
                const int pc = (rem2 - ph * G::PHC) * SW + ph;
                const int ih = ih0 + pr, iw = iw0 + pc;
                const bool ok = pr < prv && pc < pcv && (unsigned)ih < (unsigned)P.h &&
                                (unsigned)iw < (unsigned)P.w;
                const uint32_t off = ok ? (uint32_t)((n * P.h + ih) * P.w + iw) * 16u : OOB_OFFSET;
                dma16(pb + (uint32_t)e0 * 16u, off, dx);
            }
        }
        // dy: entry e = physical chunk of pixel row p = e / 8; physical 64-byte
        // segment (e & 7) >> 2 holds logical segment ^ ((p >> 1) & 1)
        const uint32_t db = pb + (uint32_t)G::P_ENT * 16u;
#pragma unroll
        for (int j = 0; j < DY_ENT / (64 * WG_WAVES); ++j) {
            const int e = (j * WG_WAVES + wave) * 64 + lane;
            const int p = e >> 3, q8 = e & 7;
            const int lchunk = (((q8 >> 2) ^ ((p >> 1) & 1)) << 2) | (q8 & 3);
            const int oh = tp * TH + (p >> 4), ow = tq * TW + (p & 15);
            const uint32_t off = (oh < P.p && ow < P.q)
                                     ? (uint32_t)(((n * P.p + oh) * P.q + ow) * K + lchunk * 8) * 2u
                                     : OOB_OFFSET;
            dma16(db + (uint32_t)((j * WG_WAVES + wave) * 64) * 16u, off, ddy);
        }
    };

    // wave w: column blocks w, w + WG_WAVES, ... (both 32-row halves of K)
    constexpr int MAXC = (CB + WG_WAVES - 1) / WG_WAVES;
    f32x16 acc[MAXC][2];
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[c][i] = f32x16{};

    const int li = lane & 15, g = lane >> 4;
    const int pix_half = 8 * (g >> 1);   // pixel offset of this lane's 8 k-slots
    // dy fragment source (transposing read): pixel row pix_half + 4*rd + li/4,
    // channels 16*(g&1) + 4*(li&3) + 32*rowblock
    // patch fragment source: pixel pix_half + 4*rd + li/4, tap offset
    // ((li&3) >> 1), 8-byte half (li&1)
    const int src_px = pix_half + (li >> 2);
    const int a_ch = 16 * (g & 1) + 4 * (li & 3);
    const int b_tap = 2 * (g & 1) + ((li & 3) >> 1);
    const int b_half = li & 1;
    const uint32_t zero_addr = lds0 + (uint32_t)(2 * BUF_ENT) * 16u;

    int tile = blockIdx.x;
    if (tile < total) load_tile(tile, 0);
    wait_vmcnt<0>();
    barrier_lds();

    int buf = 0;
    for (; tile < total; tile += gridDim.x) {
        const int next = tile + gridDim.x;
        if (next < total) load_tile(next, buf ^ 1);
        const uint32_t pb = lds0 + (uint32_t)(buf * BUF_ENT) * 16u;
        const uint32_t db = pb + (uint32_t)G::P_ENT * 16u;
#pragma unroll
        for (int row = 0; row < TH; ++row) {   // one k16 step = one tile row of 16 pixels
            u32x4 fa[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int p0 = row * TW + src_px;
                const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4 *)(uintptr_t)(db + dy_off(p0, 32 * i + a_ch)));
                const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4 *)(uintptr_t)(db + dy_off(p0 + 4, 32 * i + a_ch)));
                fa[i] = pack_tr(v0, v1);
            }
#pragma unroll
            for (int c = 0; c < MAXC; ++c) {
                const int cb = wave + WG_WAVES * c;
                if (cb < CB) {
                    const int t = cb * 4 + b_tap;
                    uint32_t a0 = zero_addr, a1 = zero_addr;
                    if (t < G::TAPS) {
                        const int r = t / S, s = t - (t / S) * S;
                        const int e = (row * SH + r) * G::PROW + (s % SW) * G::PHC + src_px + s / SW;
                        a0 = pb + (uint32_t)e * 16u + b_half * 8;
                        a1 = a0 + 4 * 16;
                    }
                    const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)a0);
                    const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)a1);
                    const u32x4 fb = pack_tr(v0, v1);
#pragma unroll
                    for (int i = 0; i < 2; ++i) acc[c][i] = mfma32<T>(fa[i], fb, acc[c][i]);
                }
            }
        }
        wait_vmcnt<0>();
        barrier_lds();
        buf ^= 1;
    }

    // partial [64][TAPS*8]: lane holds column l&31 of each block, rows
    // 8*(v/4) + 4*(l/32) + v%4 of each 32-row half
    const int ncol = G::TAPS * 8;
    float *dst = part + (int64_t)blockIdx.x * K * ncol;
    const int l32 = lane & 31, kh = lane >> 5;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int cb = wave + WG_WAVES * c;
        const int col = cb * 32 + l32;
        if (cb < CB && col < ncol) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[(32 * i + 8 * (v >> 2) + 4 * kh + (v & 3)) * ncol + col] = acc[c][i][v];
        }
    }
}

// ---------------------------------------------------------------------------
// The same two passes for 4-channel (8-byte) pixels (the stem's 3 input
// channels padded to 4), 7x7 filter, stride 2, padding 3 on each side, even
// image width.  Half the input bytes of the 8-channel form and 14 k-steps per
// tile instead of 25.
//
// A k-step of 16 reduction elements is four filter columns of one filter row
// times 4 channels.  The columns of filter row r run over 8 slots u = s + 1
// (u = 0 stands for s = -1 and has zero weight), so slots 2p, 2p + 1 are two
// adjacent image columns: with the patch origin on an even image column
// (one column left of the first tap) an operand half of 8 channels is one
// aligned 16-byte LDS entry holding two consecutive pixels, and the image
// edges never split an entry (even width).  The patch is stored in image
// order, 19 entries (38 columns) per row.
namespace stem {
constexpr int P4_ROWB = 38 * 8;                         // bytes per patch row
constexpr int P4_RE = P4_ROWB / 16;                     // 16-byte entries per patch row
constexpr int P4_PR = (TH - 1) * 2 + 7;                 // patch rows
constexpr int P4_ENT = ((P4_PR * P4_RE + 63) / 64) * 64;
constexpr int W4_ROW = 7 * 4 + 1;                       // entries per output channel (odd)
constexpr int W4_ENT = K * W4_ROW;
constexpr int KS4 = 14;                                 // k-steps per tile
constexpr int WG4_WAVES = 8;
}  // namespace stem

template <class T>
__global__ __launch_bounds__(stem::FWD_WAVES * 64, 1) void stem_fwd4_kernel(const StemParams P) {
    using namespace stem;
    constexpr int C_ENT = TH * TW * K / 8;
    constexpr int LDS_ENT = W4_ENT + 2 * P4_ENT + C_ENT;
    static_assert(LDS_ENT * 16 <= 160 * 1024 && FWD_WAVES == 8, "LDS budget, one fragment per wave");
    __shared__ u32x4 lds[LDS_ENT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];
    const uint32_t pbase0 = lds0 + W4_ENT * 16;
    const i32x4 dx = desc_of(P.x, P.x_bytes);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(P.wt, P.wt_bytes);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(P.y, P.y_bytes);

    const int tiles_q = (P.q + TW - 1) / TW, tiles_p = (P.p + TH - 1) / TH;
    const int per_img = tiles_p * tiles_q;
    const int total = P.n * per_img;

    // filter: entry k * W4_ROW + r * 4 + p holds slots 2p, 2p + 1 of filter
    // row r (w[k][r][s][0..3] at s = u - 1; u = 0 is zero)
    for (int i = tid; i < K * 7 * 8; i += FWD_WAVES * 64) {
        const int k = i / 56, rem = i - k * 56, r = rem >> 3, u = rem & 7;
        u32x2 v = u32x2{0u, 0u};
        if (u > 0) {
            const u32x4 w4 = load16(rw, (uint32_t)((k * 49 + r * 7 + u - 1) * 8) & ~15u);
            // the 8 bytes sit in the low or high half of the aligned 16
            const bool hi = (((k * 49 + r * 7 + u - 1) * 8) & 15) != 0;
            v = hi ? u32x2{w4[2], w4[3]} : u32x2{w4[0], w4[1]};
        }
        *(u32x2 *)((char *)&lds[0] + (k * W4_ROW + r * 4 + (u >> 1)) * 16 + (u & 1) * 8) = v;
    }

    // patch of tile `tile` into buffer b: entry e = row e / 19, image
    // columns col0 + 2 (e % 19) and + 1, col0 = the tile's first tap column - 1
    auto load_patch = [&](int tile, int b) {
        const int n = tile / per_img;
        const int rem = tile - n * per_img;
        const int tp = rem / tiles_q, tq = rem - tp * tiles_q;
        const int ih0 = tp * TH * 2 - P.ph, col0 = tq * TW * 2 - P.pw - 1;
        const uint32_t pb = pbase0 + (uint32_t)(b * P4_ENT) * 16u;
#pragma unroll
        for (int j = 0; j < (P4_ENT / 64 + FWD_WAVES - 1) / FWD_WAVES; ++j) {
            const int e0 = (j * FWD_WAVES + wave) * 64;
            if (e0 < P4_ENT) {
                const int e = e0 + lane;
                const int pr = e / P4_RE, jc = e - pr * P4_RE;
                const int ih = ih0 + pr, iw = col0 + 2 * jc;
                const bool ok = pr < P4_PR && (unsigned)ih < (unsigned)P.h &&
                                (unsigned)iw < (unsigned)P.w;
                const uint32_t off = ok ? (uint32_t)((n * P.h + ih) * P.w + iw) * 8u : OOB_OFFSET;
                dma16(pb + (uint32_t)e0 * 16u, off, dx);
            }
        }
    };

    // wave w: tile rows 2w, 2w + 1 (one 32-pixel fragment); lane l: row
    // 2w + (l & 31) / 16, column l & 15
    const int l32 = lane & 31, khalf = lane >> 5;
    const int a_row = 2 * wave + (l32 >> 4), a_col = l32 & 15;

    int tile = blockIdx.x;
    if (tile < total) load_patch(tile, 0);
    wait_vmcnt<0>();
    barrier_lds();

    int buf = 0;
    for (; tile < total; tile += gridDim.x) {
        const int next = tile + gridDim.x;
        if (next < total) load_patch(next, buf ^ 1);

        f32x16 acc[2];
        acc[0] = f32x16{};
        acc[1] = f32x16{};
        const u32x4 *pt = &lds[W4_ENT + buf * P4_ENT];
#pragma unroll
        for (int ks = 0; ks < KS4; ++ks) {
            const int r = ks >> 1, pp = 2 * (ks & 1) + khalf;  // filter row, slot pair
            u32x4 fa = pt[(a_row * 2 + r) * P4_RE + a_col + pp];
            // slot 0 (s = -1) has no tap: its pixel must not meet the zero weight
            if ((ks & 1) == 0 && khalf == 0) {
                fa[0] = 0u;
                fa[1] = 0u;
            }
            u32x4 fb[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) fb[j] = lds[(j * 32 + l32) * W4_ROW + r * 4 + pp];
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[j] = mfma32<T>(fb[j], fa, acc[j]);
        }

        // epilogue as for 8-channel pixels: C tile [256 px][8 chunks] in LDS
        {
            char *cl = (char *)&lds[W4_ENT + 2 * P4_ENT];
            const int px = 32 * wave + l32;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int c = 4 * j + e;
                    u32x2 pk;
                    pk[0] = to16<T>(acc[j][4 * e + 0] * P.alpha) |
                            (to16<T>(acc[j][4 * e + 1] * P.alpha) << 16);
                    pk[1] = to16<T>(acc[j][4 * e + 2] * P.alpha) |
                            (to16<T>(acc[j][4 * e + 3] * P.alpha) << 16);
                    *(u32x2 *)(cl + (px * 8 + (c ^ (px & 7))) * 16 + khalf * 8) = pk;
                }
            }
        }
        barrier_lds();  // C tile complete; every wave is done with patch `buf`
        {
            const int n = tile / per_img;
            const int rem = tile - n * per_img;
            const int tp = rem / tiles_q, tq = rem - tp * tiles_q;
#pragma unroll
            for (int it = 0; it < TH * TW * 8 / (64 * FWD_WAVES); ++it) {
                const int idx = it * (64 * FWD_WAVES) + tid;
                const int px = idx >> 3, c = idx & 7;
                const int oh = tp * TH + (px >> 4), ow = tq * TW + (px & 15);
                const uint32_t o = (oh < P.p && ow < P.q)
                                       ? (uint32_t)(((n * P.p + oh) * P.q + ow) * K + c * 8) * 2u
                                       : OOB_OFFSET;
                const u32x4 v = lds[W4_ENT + 2 * P4_ENT + px * 8 + (c ^ (px & 7))];
                __builtin_amdgcn_raw_buffer_store_b128(v, ry, o, 0, 2);
            }
        }
        wait_vmcnt<TH * TW * 8 / (64 * FWD_WAVES)>();
        barrier_lds();
        buf ^= 1;
    }
    wait_vmcnt<0>();
}

// Backward-weight for 4-channel pixels.  Column block r (32 columns) is
// filter row r: slots u = 0..7 times 4 channels, so the 16 columns a
// transposing read covers are 4 consecutive slots, i.e. 4 consecutive image
// columns (32 bytes of one patch row), and the 4 pixels it reads are 16
// bytes apart.  Slot 0's column (s = -1) is computed and dropped.  The 7
// blocks and both 32-row halves of K go to 4 waves (blocks w and w + 4);
// waves 4-7 do the same for the odd tile rows, so each k-step's dy
// fragments are read by four waves only, and the workgroup writes two
// partials (even and odd rows), part[2 * blockIdx.x + half].
template <class T>
__global__ __launch_bounds__(stem::WG4_WAVES * 64, 1) void stem_wgrad4_kernel(const StemParams P,
                                                                            float *part) {
    using namespace stem;
    constexpr int DY_ENT = TH * TW * K / 8;
    constexpr int BUF_ENT = P4_ENT + DY_ENT;
    constexpr int LDS_ENT = 2 * BUF_ENT;
    static_assert(LDS_ENT * 16 <= 160 * 1024, "LDS budget");
    __shared__ u32x4 lds[LDS_ENT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];
    const i32x4 dx = desc_of(P.x, P.x_bytes);
    const i32x4 ddy = desc_of(P.y, P.y_bytes);

    const int tiles_q = (P.q + TW - 1) / TW, tiles_p = (P.p + TH - 1) / TH;
    const int per_img = tiles_p * tiles_q;
    const int total = P.n * per_img;

    auto load_tile = [&](int tile, int b) {
        const int n = tile / per_img;
        const int rem = tile - n * per_img;
        const int tp = rem / tiles_q, tq = rem - tp * tiles_q;
        const int vh = min(TH, P.p - tp * TH), vw = min(TW, P.q - tq * TW);
        // patch entries of the receptive field of the in-range outputs (the
        // others load as zeros: their dy rows are zero, and an inf or NaN
        // input there must not reach the sums)
        const int prv = (vh - 1) * 2 + 7, jcv = vw + 3;
        const int ih0 = tp * TH * 2 - P.ph, col0 = tq * TW * 2 - P.pw - 1;
        const uint32_t pb = lds0 + (uint32_t)(b * BUF_ENT) * 16u;
#pragma unroll
        for (int j = 0; j < (P4_ENT / 64 + WG4_WAVES - 1) / WG4_WAVES; ++j) {
            const int e0 = (j * WG4_WAVES + wave) * 64;
            if (e0 < P4_ENT) {
                const int e = e0 + lane;
                const int pr = e / P4_RE, jc = e - pr * P4_RE;
                const int ih = ih0 + pr, iw = col0 + 2 * jc;
                const bool ok = pr < prv && jc < jcv && (unsigned)ih < (unsigned)P.h &&
                                (unsigned)iw < (unsigned)P.w;
                const uint32_t off = ok ? (uint32_t)((n * P.h + ih) * P.w + iw) * 8u : OOB_OFFSET;
                dma16(pb + (uint32_t)e0 * 16u, off, dx);
            }
        }
        const uint32_t db = pb + (uint32_t)P4_ENT * 16u;
#pragma unroll
        for (int j = 0; j < DY_ENT / (64 * WG4_WAVES); ++j) {
            const int e = (j * WG4_WAVES + wave) * 64 + lane;
            const int p = e >> 3, q8 = e & 7;
            const int lchunk = (((q8 >> 2) ^ ((p >> 1) & 1)) << 2) | (q8 & 3);
            const int oh = tp * TH + (p >> 4), ow = tq * TW + (p & 15);
            const uint32_t off = (oh < P.p && ow < P.q)
                                     ? (uint32_t)(((n * P.p + oh) * P.q + ow) * K + lchunk * 8) * 2u
                                     : OOB_OFFSET;
            dma16(db + (uint32_t)((j * WG4_WAVES + wave) * 64) * 16u, off, ddy);
        }
    };

    const int half = wave >> 2;       // tile rows of this wave: half, half + 2, ...
    const int cb0 = wave & 3;         // column blocks cb0 and cb0 + 4 (< 7)
    const bool two = cb0 + 4 < 7;
    f32x16 acc[2][2];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[c][i] = f32x16{};

    const int li = lane & 15, g = lane >> 4;
    // this lane's pixel within a 16-pixel k-step (tile row): 8 * (g / 2) +
    // li / 4, and + 4 for the second read
    const int src_px = 8 * (g >> 1) + (li >> 2);
    const int a_ch = 16 * (g & 1) + 4 * (li & 3);
    const int b_slot = 4 * (g & 1) + (li & 3);

    int tile = blockIdx.x;
    if (tile < total) load_tile(tile, 0);
    wait_vmcnt<0>();
    barrier_lds();

    int buf = 0;
    for (; tile < total; tile += gridDim.x) {
        const int next = tile + gridDim.x;
        if (next < total) load_tile(next, buf ^ 1);
        const uint32_t pb = lds0 + (uint32_t)(buf * BUF_ENT) * 16u;
        const uint32_t db = pb + (uint32_t)P4_ENT * 16u;
#pragma unroll
        for (int rr = 0; rr < TH / 2; ++rr) {   // one k16 step = one tile row of 16 pixels
            const int row = 2 * rr + half;
            u32x4 fa[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int p0 = row * TW + src_px;
                const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4 *)(uintptr_t)(db + dy_off(p0, 32 * i + a_ch)));
                const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4 *)(uintptr_t)(db + dy_off(p0 + 4, 32 * i + a_ch)));
                fa[i] = pack_tr(v0, v1);
            }
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                if (c == 0 || two) {
                    const int r = cb0 + 4 * c;
                    // patch row 2 * row + r, image column 2 * ow + slot
                    const uint32_t a0 = pb + (uint32_t)((2 * row + r) * P4_ROWB + (2 * src_px + b_slot) * 8);
                    const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)a0);
                    const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)(a0 + 64));
                    const u32x4 fb = pack_tr(v0, v1);
#pragma unroll
                    for (int i = 0; i < 2; ++i) acc[c][i] = mfma32<T>(fa[i], fb, acc[c][i]);
                }
            }
        }
        wait_vmcnt<0>();
        barrier_lds();
        buf ^= 1;
    }

    // partial [64][49 * 4]: lane holds column l & 31 of its block (slot
    // (l & 31) / 4, channel l % 4) and rows 8 * (v / 4) + 4 * (l / 32) + v % 4
    // of each 32-row half; slot 0 is dropped
    constexpr int NCOL = 49 * 4;
    float *dst = part + (int64_t)(2 * blockIdx.x + half) * K * NCOL;
    const int l32 = lane & 31, kh = lane >> 5;
    const int slot = l32 >> 2, ch = l32 & 3;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        if ((c == 0 || two) && slot > 0) {
            const int col = ((cb0 + 4 * c) * 7 + slot - 1) * 4 + ch;
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[(32 * i + 8 * (v >> 2) + 4 * kh + (v & 3)) * NCOL + col] = acc[c][i][v];
        }
    }
}

template <class T, int R, int S, int SH, int SW>
static hipError_t launch_stem_t(const StemParams &p, int cus, hipStream_t st) {
    const int64_t tiles =
        (int64_t)p.n * ((p.p + stem::TH - 1) / stem::TH) * ((p.q + stem::TW - 1) / stem::TW);
    if (tiles <= 0) return hipSuccess;
    const int grid = (int)(tiles < cus ? tiles : cus);
    hipLaunchKernelGGL((stem_fwd_kernel<T, R, S, SH, SW>), dim3(grid), dim3(stem::FWD_WAVES * 64), 0, st, p);
    return hipGetLastError();
}

bool stem_fwd_supported(int r, int s, int sh, int sw) { return r == 7 && s == 7 && sh == 2 && sw == 2; }

bool stem4_supported(const StemParams &p) {
    return stem_fwd_supported(p.r, p.s, p.sh, p.sw) && p.pw % 2 == 1 && p.w % 2 == 0;
}

hipError_t launch_stem_wgrad(int dtype, const StemParams &p, float *part, int splits,
                             hipStream_t st) {
    if (p.c == 4) {
        if (!stem4_supported(p) || splits < 2 || splits % 2 != 0) return hipErrorInvalidValue;
        if (dtype == Half::id)
            hipLaunchKernelGGL(stem_wgrad4_kernel<Half>, dim3(splits / 2), dim3(stem::WG4_WAVES * 64), 0,
                               st, p, part);
        else
            hipLaunchKernelGGL(stem_wgrad4_kernel<BFloat>, dim3(splits / 2), dim3(stem::WG4_WAVES * 64),
                               0, st, p, part);
        return hipGetLastError();
    }
    if (!stem_fwd_supported(p.r, p.s, p.sh, p.sw) || splits < 1) return hipErrorInvalidValue;
    if (dtype == Half::id)
        hipLaunchKernelGGL((stem_wgrad_kernel<Half, 7, 7, 2, 2>), dim3(splits), dim3(stem::WG_WAVES * 64), 0, st, p,
                           part);
    else
        hipLaunchKernelGGL((stem_wgrad_kernel<BFloat, 7, 7, 2, 2>), dim3(splits), dim3(stem::WG_WAVES * 64), 0, st,
                           p, part);
    return hipGetLastError();
}

hipError_t launch_stem_fwd(int dtype, const StemParams &p, int cus, hipStream_t st) {
    if (p.c == 4) {
        if (!stem4_supported(p)) return hipErrorInvalidValue;
        const int64_t tiles =
            (int64_t)p.n * ((p.p + stem::TH - 1) / stem::TH) * ((p.q + stem::TW - 1) / stem::TW);
        if (tiles <= 0) return hipSuccess;
        const int grid = (int)(tiles < cus ? tiles : cus);
        if (dtype == Half::id)
            hipLaunchKernelGGL(stem_fwd4_kernel<Half>, dim3(grid), dim3(stem::FWD_WAVES * 64), 0, st, p);
        else
            hipLaunchKernelGGL(stem_fwd4_kernel<BFloat>, dim3(grid), dim3(stem::FWD_WAVES * 64), 0, st, p);
        return hipGetLastError();
    }
    if (!stem_fwd_supported(p.r, p.s, p.sh, p.sw)) return hipErrorInvalidValue;
    if (dtype == Half::id) return launch_stem_t<Half, 7, 7, 2, 2>(p, cus, st);
    return launch_stem_t<BFloat, 7, 7, 2, 2>(p, cus, st);
}

}  // namespace nnconv
