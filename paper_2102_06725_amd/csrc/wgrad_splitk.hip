// wgrad_splitk.hip -- backward-weight split-K implicit GEMM with direct-to-LDS
// staging and gfx950 transposing LDS reads.
//
// GEMM view:  dW[k, j] = sum_pix dy[pix, k] * xcol[pix, j],  j = (r, s, c).
// The reduction runs over batch pixels, which is the strided dimension of
// both channel-last operands.  Tiles are staged exactly as they lie in
// memory -- a k-slice is BKP pixel rows of BM dy channels and of BN im2col
// columns -- with buffer_load ... lds, STAGES deep.  The matrix-core
// operands need 8 consecutive pixels per lane; ds_read_b64_tr_b16 delivers
// them: when the 16 lanes of a group address a 4-row x 16-column block of
// 16-bit elements (4 lanes per row, 4 columns each), lane i receives column i
// of the 4 rows.  Two such reads give one lane its 8 pixels.
//
// LDS rows are swizzled in 64-byte segments so the 4 rows of a transposing
// read fall in 4 different 64-byte bank segments.
// Pixels are split into `splits` ranges; each range writes an fp32 partial
// tile to the workspace (summed later in a fixed order).
#include "launch.hpp"

namespace nnconv {

namespace wgs {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Row p of a tile with ROWB-byte rows: logical 64-byte segment s lives at
// physical segment s ^ swz(p).  A transposing read touches rows p0..p0+3
// (p0 a multiple of 4) at one logical segment; this spreads them over four
// 64-byte segments of the 256-byte bank window.
template <int ROWB>
__device__ __forceinline__ int seg_swz(int p) {
    return ROWB >= 256 ? (p & 3) : ((p >> 1) & 1);
}

// byte offset of (row p, 16-bit column co) in a swizzled tile
template <int ROWB>
__device__ __forceinline__ uint32_t tile_off(int p, int co) {
    const int byte = co * 2;
    return (uint32_t)(p * ROWB + (((byte >> 6) ^ seg_swz<ROWB>(p)) << 6) + (byte & 63));
}

}  // namespace wgs

// DIAG: block-diagonal super-group gradients (groups of at most 32 channels
// run as 64-channel super-groups): only the 32x32 blocks whose filter rows
// and input channels lie in the same half of a 64-channel group are kept by
// the reduction, so each wave computes and writes only the column block that
// matches its 32 rows.
template <class T, int BM, int BN, int WM, int WN, int BKP, int STAGES, bool DIAG>
__global__ __launch_bounds__(WM * WN * 64, (STAGES * BKP * (BM + BN) * 2 > 80 * 1024) ? 1
                                           : (STAGES * BKP * (BM + BN) * 2 > 40 * 1024) ? 2
                                                                                       : 4)
void wgrad_splitk_kernel(const WGParams P) {
    using namespace wgs;
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int AROWB = BM * 2, BROWB = BN * 2;      // bytes per pixel row
    constexpr int ACH = AROWB / 16, BCH = BROWB / 16;  // 16-byte chunks per row
    constexpr int A_BYTES = BKP * AROWB, B_BYTES = BKP * BROWB;
    constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    constexpr int A_LD = A_BYTES / (1024 * NW), B_LD = B_BYTES / (1024 * NW);
    constexpr int LOADS = A_LD + B_LD;
    static_assert(A_LD >= 1 && B_LD >= 1 && FM >= 1 && FN >= 1, "tile shape");
    static_assert(AROWB >= 128 && BROWB >= 128, "rows of at least two 64-byte segments");
    static_assert(BKP % 16 == 0, "pixel slice");
    static_assert(!DIAG || (FM == 1 && WTM == 32 && FN == 2 && WTN == 64 && BM % 64 == 0 &&
                            BN % 64 == 0),
                  "block-diagonal: 32-row waves over 64-column pairs");
    constexpr int FNA = DIAG ? 1 : FN;  // accumulated 32-column blocks per wave

    __shared__ u32x4 lds[STAGES * STAGE_BYTES / 16];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;

    // tile: groups x splits x m-tiles x n-tiles, n fastest
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int per_split = P.tiles_m * P.tiles_n;
    const int per_g = per_split * P.splits;
    const int g = (int)lid / per_g;
    int rem = (int)lid - g * per_g;
    const int split = rem / per_split;
    rem -= split * per_split;
    const int tm = rem / P.tiles_n;
    const int tn = rem - tm * P.tiles_n;
    const int k0 = tm * BM, j0 = tn * BN;

    const int pix_begin = split * P.pix_per_split;
    const int pix_end = min(P.npq, pix_begin + P.pix_per_split);
    const int k_iters = pix_end > pix_begin ? (pix_end - pix_begin + BKP - 1) / BKP : 0;

    const i32x4 ddy = desc_of(P.dy, P.dy_bytes);
    const i32x4 dx = desc_of(P.x, P.x_bytes);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];

    // ---- staging roles: load j of a wave covers 1 KB = 1024/ROWB pixel rows
    // dy: lane -> (row lane / ACH, physical chunk lane % ACH)
    int a_row[A_LD];
    uint32_t a_col[A_LD];  // byte offset of the lane's channels within a dy pixel row
    bool a_ok[A_LD];
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
        const int q = lane % ACH;
        const int p = ((wave * A_LD + j) * 64 + lane) / ACH;
        const int lseg = (q >> 2) ^ seg_swz<AROWB>(p);
        const int lchunk = lseg * 4 + (q & 3);
        const int ch = k0 + lchunk * 8;
        a_row[j] = p;
        a_ok[j] = ch < P.kg;
        a_col[j] = (uint32_t)(g * P.kg + ch) * 2u;
    }
    // x: lane -> (row, chunk) likewise; the chunk's column j = (tap, c) is fixed
    int b_row[B_LD], b_dh[B_LD], b_dw[B_LD];
    uint32_t b_col[B_LD];
    bool b_ok[B_LD];
#pragma unroll
    for (int j = 0; j < B_LD; ++j) {
        const int q = lane % BCH;
        const int p = ((wave * B_LD + j) * 64 + lane) / BCH;
        const int lseg = (q >> 2) ^ seg_swz<BROWB>(p);
        const int lchunk = lseg * 4 + (q & 3);
        const int col = j0 + lchunk * 8;
        b_row[j] = p;
        b_ok[j] = col < P.rscg;
        const int cc = b_ok[j] ? col : 0;
        const int tap = (int)fdiv((uint32_t)cc, P.div_cg);
        const int c = cc - tap * P.cg;
        const int r = (int)fdiv((uint32_t)tap, P.div_s);
        const int s = tap - r * (int)P.div_s.d;
        b_dh[j] = r * P.dh - P.ph;
        b_dw[j] = s * P.dw - P.pw;
        b_col[j] = (uint32_t)(g * P.cg + c) * 2u;
    }

    auto issue = [&](int kt, int buf) {
        const int base = pix_begin + kt * BKP;
        const uint32_t sb = lds0 + (uint32_t)(buf * STAGE_BYTES);
#pragma unroll
        for (int j = 0; j < A_LD; ++j) {
            const int pix = base + a_row[j];
            const bool ok = a_ok[j] && pix < pix_end;
            const uint32_t off = (uint32_t)pix * (uint32_t)P.k * 2u + a_col[j];
            dma16(sb + (uint32_t)((wave * A_LD + j) * 1024), ok ? off : OOB_OFFSET, ddy);
        }
#pragma unroll
        for (int j = 0; j < B_LD; ++j) {
            const int pix = base + b_row[j];
            bool ok = b_ok[j] && pix < pix_end;
            const int pc = ok ? pix : 0;
            const int n = (int)fdiv((uint32_t)pc, P.div_pq);
            const int rm = pc - n * (P.p * P.q);
            const int pp = (int)fdiv((uint32_t)rm, P.div_q);
            const int qq = rm - pp * P.q;
            const int h = pp * P.sh + b_dh[j];
            const int w = qq * P.sw + b_dw[j];
            ok = ok && (unsigned)h < (unsigned)P.h && (unsigned)w < (unsigned)P.w;
            const uint32_t off = (uint32_t)((n * P.h + h) * P.w + w) * (uint32_t)P.c * 2u + b_col[j];
            dma16(sb + (uint32_t)(A_BYTES + (wave * B_LD + j) * 1024), ok ? off : OOB_OFFSET, dx);
        }
    };

    f32x16 acc[FM][FNA];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FNA; ++j) acc[i][j] = f32x16{};
    // DIAG: the wave's rows are half wm % 2 of a 64-row group; its column
    // block is the one with the same half of each 64-channel tap block
    const int dcol = DIAG ? wn * WTN + (wm & 1) * 32 : 0;

    // fragment reads: lane group gq = lane/16 covers channels 16*(gq%2) of a
    // 32-wide block and pixels 8*(gq/2) of the 16-pixel k-step
    const int li = lane & 15, gq = lane >> 4;
    const int fr_row = 8 * (gq >> 1) + (li >> 2);      // + 16*ks (+4 for the second read)
    const int fr_col = 16 * (gq & 1) + (li & 3) * 4;   // + 32-wide block base
    auto frag = [&](const char *tile, int rowb_is_a, int ks, int cbase) -> u32x4 {
        const int p = ks * 16 + fr_row;
        uint32_t o0, o1;
        if (rowb_is_a) {
            o0 = tile_off<AROWB>(p, cbase + fr_col);
            o1 = tile_off<AROWB>(p + 4, cbase + fr_col);
        } else {
            o0 = tile_off<BROWB>(p, cbase + fr_col);
            o1 = tile_off<BROWB>(p + 4, cbase + fr_col);
        }
        const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(tile + o0));
        const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(tile + o1));
        u32x4 r;
        r[0] = (uint32_t)(uint16_t)v0[0] | ((uint32_t)(uint16_t)v0[1] << 16);
        r[1] = (uint32_t)(uint16_t)v0[2] | ((uint32_t)(uint16_t)v0[3] << 16);
        r[2] = (uint32_t)(uint16_t)v1[0] | ((uint32_t)(uint16_t)v1[1] << 16);
        r[3] = (uint32_t)(uint16_t)v1[2] | ((uint32_t)(uint16_t)v1[3] << 16);
        return r;
    };

    auto compute = [&](int buf) {
        const char *st = (const char *)&lds[0] + buf * STAGE_BYTES;
#pragma unroll
        for (int ks = 0; ks < BKP / 16; ++ks) {
            u32x4 fa[FM], fb[FNA];
#pragma unroll
            for (int i = 0; i < FM; ++i) fa[i] = frag(st, 1, ks, wm * WTM + i * 32);
#pragma unroll
            for (int j = 0; j < FNA; ++j)
                fb[j] = frag(st + A_BYTES, 0, ks, DIAG ? dcol : wn * WTN + j * 32);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FNA; ++j) acc[i][j] = mfma32<T>(fa[i], fb[j], acc[i][j]);
        }
    };
    if constexpr (STAGES == 1) {
        // one stage: several resident workgroups per CU cover each other's
        // load latency
        for (int kt = 0; kt < k_iters; ++kt) {
            if (kt > 0) barrier_lds();  // previous slice fully read
            issue(kt, 0);
            wait_vmcnt<0>();
            barrier_lds();
            compute(0);
        }
    } else if (k_iters > 0) {
        const int pro = k_iters < STAGES - 1 ? k_iters : STAGES - 1;
        for (int s = 0; s < pro; ++s) issue(s, s);
        for (int kt = 0; kt < k_iters; ++kt) {
            if (kt + STAGES - 2 < k_iters)
                wait_vmcnt<(STAGES - 2) * LOADS>();
            else
                wait_vmcnt<0>();
            barrier_lds();
            if (kt + STAGES - 1 < k_iters) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
            compute(kt % STAGES);
        }
    }

    // lane holds column l32 of each 32-column block and rows 8*e + 4*khalf + {0..3}
    const int l32 = lane & 31, khalf = lane >> 5;
    const int K = P.kg * P.groups;
    float *ws = P.ws + (int64_t)split * K * P.rscg;
#pragma unroll
    for (int j = 0; j < FNA; ++j) {
        const int col = DIAG ? j0 + dcol + l32 : j0 + wn * WTN + j * 32 + l32;
        if (col >= P.rscg) continue;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = k0 + wm * WTM + i * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
                if (row < P.kg) ws[(int64_t)(g * P.kg + row) * P.rscg + col] = acc[i][j][v];
            }
        }
    }
}

template <class T, int BM, int BN, int WM, int WN, int BKP, int STAGES, bool DIAG = false>
static hipError_t launch_wgs(WGParams &p, hipStream_t st) {
    p.tiles_m = (p.kg + BM - 1) / BM;
    p.tiles_n = (p.rscg + BN - 1) / BN;
    const int64_t nb = (int64_t)p.tiles_m * p.tiles_n * p.splits * p.groups;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((wgrad_splitk_kernel<T, BM, BN, WM, WN, BKP, STAGES, DIAG>), dim3((uint32_t)nb),
                       dim3(WM * WN * 64), 0, st, p);
    return hipGetLastError();
}

// Configurations (LDS per workgroup):
//    64x128: 4 waves of 32x64, 64-pixel slices, single stage (24 KB); also
//            block-diagonal (each wave one 32x32 block)
//   128x128: 8 waves of 64x32, 64-pixel slices, 2 stages (64 KB; two
//            workgroups per CU)
//   128x128 single stage: 4 waves of 64x64, 64-pixel slices (32 KB; four
//            workgroups per CU)
//   256x256: 16 waves of 64x64, 32-pixel slices, 2 stages (64 KB)
// The 8- and 16-wave tiles keep more waves per SIMD to hide the LDS
// fragment-read latency; on the ResNet-50 3x3 layers with 128 filters this
// cut the backward-weight time by a fifth against 4 waves of 64x64.
template <class T>
static hipError_t launch_wgs_t(WGConfig cfg, WGParams &p, hipStream_t st) {
    switch (cfg) {
        case WG_64x128: return launch_wgs<T, 64, 128, 2, 2, 64, 1>(p, st);
        case WG_64x128D: return launch_wgs<T, 64, 128, 2, 2, 64, 1, true>(p, st);
        case WG_256x256: return launch_wgs<T, 256, 256, 4, 4, 32, 2>(p, st);
        case WG_128x128S: return launch_wgs<T, 128, 128, 2, 2, 64, 1>(p, st);
        case WG_128x128:
        default: return launch_wgs<T, 128, 128, 2, 4, 64, 2>(p, st);
    }
}

hipError_t launch_wgrad_splitk(int dtype, WGConfig cfg, WGParams &p, hipStream_t st) {
    if (dtype == Half::id) return launch_wgs_t<Half>(cfg, p, st);
    return launch_wgs_t<BFloat>(cfg, p, st);
}

}  // namespace nnconv
