// igemm_c8.hip -- implicit-GEMM convolution (forward pass and each stride
// phase of the backward-data pass) for any per-tap channel count that is a
// multiple of 8 (the stem after padding 3 -> 8 channels, small-C layers),
// with a multi-stage global -> LDS pipeline built on gfx950's direct-to-LDS
// buffer loads.
//
// GEMM view: rows = output pixels gathered through the tap table, columns =
// output channels, reduction = (tap, channel) with channels fastest:
//   - each k-slice is 32 reduction elements (4 x 16-byte chunks per row),
//     which may span several taps;
//   - operand tiles go straight from HBM/L2 into LDS (no register staging),
//     STAGES slices deep, so STAGES-1 slices of loads are in flight while
//     the matrix cores work on the current one;
//   - one barrier per k-slice.
// A buffer_load ... lds instruction writes its 64 lanes' 16-byte chunks to
// 64 consecutive 16-byte LDS slots; which global chunk each lane fetches is
// chosen so that slot order is the swizzled tile layout the fragment reads
// expect.  Padding, ragged edges and the tail slices read zeros through the
// buffer range check.
#include "launch.hpp"

namespace nnconv {

// 64 LDS banks serve 16 lanes of a 16-byte read per cycle: the 16 rows of a
// fragment read must land in 16 distinct 16-byte bank groups of 256 bytes.
// 128-byte rows (BKC 8): parity of r picks the half, (r>>1)&7 the chunk;
// 64-byte rows (BKC 4): r&3 picks the quarter, (r>>2)&3 the chunk.
template <int BKC>
__device__ __forceinline__ int swz_of(int r) {
    return BKC == 8 ? ((r >> 1) & 7) : ((r >> 2) & 3);
}

// Tile layout in LDS: BKC 16-byte chunks per row; row r, logical chunk c at
// slot r*BKC + (c ^ swz(r)).  Eight consecutive rows read at one logical
// chunk hit eight different 16-byte bank groups.
template <int BKC>
__device__ __forceinline__ int slot_of(int r, int c) {
    return r * BKC + (c ^ swz_of<BKC>(r));
}

template <class T, int BM, int BN, int BKC, int STAGES, bool ALIGNED>
__global__ __launch_bounds__(256, 2) void igemm_c8_kernel(const TNParams P) {
    constexpr int WM = 2, WN = 2;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int BK = BKC * 8;                            // reduction elements per slice
    constexpr int A_SLOTS = BM * BKC, B_SLOTS = BN * BKC;  // 16-byte slots per stage
    constexpr int A_LD = A_SLOTS / 256, B_LD = B_SLOTS / 256;  // loads per thread per stage
    constexpr int STAGE_SLOTS = A_SLOTS + B_SLOTS;
    constexpr int LOADS = A_LD + B_LD;
    static_assert(A_LD >= 1 && B_LD >= 1, "tile too small");

    __shared__ u32x4 lds[STAGES * STAGE_SLOTS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;

    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int per_g = P.tiles_m * P.tiles_n;
    const int g = (int)lid / per_g;
    const int rem = (int)lid - g * per_g;
    const int tm = rem / P.tiles_n;
    const int tn = rem - tm * P.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;

    const i32x4 ra = desc_of(P.a, P.a_bytes);
    const i32x4 rb = desc_of(P.b, P.b_bytes);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];

    // Load instruction j of this wave fills slots [(wave*LD + j)*64, +64); lane
    // `lane` fills slot base+lane: row = slot/BKC, physical chunk = lane%BKC.
    const int pch = lane & (BKC - 1);
    int a_pix[A_LD], a_h[A_LD], a_w[A_LD], a_lc[A_LD];
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
        const int slot = (wave * A_LD + j) * 64 + lane;
        const int r = slot / BKC;
        a_lc[j] = pch ^ swz_of<BKC>(r);
        const int m = m0 + r;
        if (m < P.M) {
            const int q1 = (int)fdiv((uint32_t)m, P.div_mj);
            const int jj = m - q1 * P.mj;
            const int n = (int)fdiv((uint32_t)q1, P.div_mi);
            const int ii = q1 - n * P.mi;
            const int bh = ii * P.ai_mul + P.ai_add;
            const int bw = jj * P.aj_mul + P.aj_add;
            a_h[j] = bh;
            a_w[j] = bw;
            a_pix[j] = (n * P.a_h + bh) * P.a_w + bw;
        } else {
            a_h[j] = -(1 << 24);
            a_w[j] = 0;
            a_pix[j] = 0;
        }
    }
    int b_off[B_LD], b_lc[B_LD];
    bool b_ok[B_LD];
#pragma unroll
    for (int j = 0; j < B_LD; ++j) {
        const int slot = (wave * B_LD + j) * 64 + lane;
        const int r = slot / BKC;
        b_lc[j] = pch ^ swz_of<BKC>(r);
        const int col = n0 + r;
        b_ok[j] = col < P.ncols;
        b_off[j] = g * P.b_g_ofs + col * P.b_ld;
    }
    const int a_ch0 = g * P.a_cg_ofs;
    const int crv = P.cr >> 3;

    int next_t = 0, next_c = 0;  // ALIGNED: tap / channel base of the next slice

    // Queue the loads of k-slice `kt` into stage buffer `buf` (always
    // LOADS instructions per thread, so vmcnt bookkeeping is uniform; slices
    // past the end read zeros into a buffer nobody reads).
    auto issue = [&](int kt, int buf) {
        int t_u = 0, c_u = 0;
        if constexpr (ALIGNED) {
            t_u = next_t;
            c_u = next_c;
            next_c += BK;
            if (next_c == P.cr) {
                next_c = 0;
                ++next_t;
            }
        }
        const uint32_t sbase = lds0 + (uint32_t)(buf * STAGE_SLOTS) * 16u;
#pragma unroll
        for (int j = 0; j < A_LD; ++j) {
            int t, c;
            if constexpr (ALIGNED) {
                t = t_u;
                c = c_u + a_lc[j] * 8;
            } else {
                const int gv = kt * BKC + a_lc[j];
                t = (int)fdiv((uint32_t)gv, P.div_crv);
                c = (gv - t * crv) * 8;
            }
            const bool tv = t < P.taps.n && kt < P.k_iters;
            const int tt = tv ? t : 0;
            const int dh = P.taps.dh[tt], dw = P.taps.dw[tt];
            const int h = a_h[j] + dh, w = a_w[j] + dw;
            const bool ok = tv && (unsigned)h < (unsigned)P.a_h && (unsigned)w < (unsigned)P.a_w;
            const int off = ((a_pix[j] + dh * P.a_w + dw) * P.a_c + a_ch0 + c) * 2;
            dma16(sbase + (uint32_t)((wave * A_LD + j) * 64) * 16u, ok ? (uint32_t)off : OOB_OFFSET,
                  ra);
        }
#pragma unroll
        for (int j = 0; j < B_LD; ++j) {
            int t, c;
            if constexpr (ALIGNED) {
                t = t_u;
                c = c_u + b_lc[j] * 8;
            } else {
                const int gv = kt * BKC + b_lc[j];
                t = (int)fdiv((uint32_t)gv, P.div_crv);
                c = (gv - t * crv) * 8;
            }
            const bool tv = t < P.taps.n && kt < P.k_iters;
            const int tt = tv ? t : 0;
            const bool ok = tv && b_ok[j];
            const int off = (b_off[j] + P.taps.boff[tt] + c) * 2;
            dma16(sbase + (uint32_t)(A_SLOTS + (wave * B_LD + j) * 64) * 16u,
                  ok ? (uint32_t)off : OOB_OFFSET, rb);
        }
    };

    f32x16 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x16{};

    const int l32 = lane & 31;
    const int khalf = lane >> 5;

    if (P.k_iters > 0) {
#pragma unroll
        for (int s = 0; s < STAGES - 1; ++s) issue(s, s);
        for (int kt = 0; kt < P.k_iters; ++kt) {
            // slice kt has landed once at most (STAGES-2) slices of loads remain
            wait_vmcnt<(STAGES - 2) * LOADS>();
            barrier_lds();
            issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
            const u32x4 *st = &lds[(kt % STAGES) * STAGE_SLOTS];
#pragma unroll
            for (int ks = 0; ks < BKC / 2; ++ks) {
                const int kc = 2 * ks + khalf;
                u32x4 fp[FM], fw[FN];
#pragma unroll
                for (int i = 0; i < FM; ++i) fp[i] = st[slot_of<BKC>(wm * WTM + i * 32 + l32, kc)];
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    fw[j] = st[A_SLOTS + slot_of<BKC>(wn * WTN + j * 32 + l32, kc)];
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int i = 0; i < FM; ++i) acc[j][i] = mfma32<T>(fw[j], fp[i], acc[j][i]);
            }
        }
        wait_vmcnt<0>();
    }

    // Epilogue: lane holds pixel column l32 of each 32-pixel block and, for
    // each 32-channel block, channels 8*e + 4*khalf + {0..3} (e = 0..3).
    uint16_t *out = (uint16_t *)P.out;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = m0 + wm * WTM + i * 32 + l32;
        if (m >= P.M) continue;
        const int q1 = (int)fdiv((uint32_t)m, P.div_mj);
        const int jj = m - q1 * P.mj;
        const int n = (int)fdiv((uint32_t)q1, P.div_mi);
        const int ii = q1 - n * P.mi;
        const int oh = ii * P.oi_mul + P.oi_add;
        const int ow = jj * P.oj_mul + P.oj_add;
        const int64_t obase =
            ((int64_t)(n * P.o_h + oh) * P.o_w + ow) * P.o_c + (int64_t)g * P.o_cg_ofs;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int ch = n0 + wn * WTN + j * 32 + 8 * e + 4 * khalf;
                if (ch >= P.ncols) continue;
                u32x2 pk;
                pk[0] = to16<T>(acc[j][i][4 * e + 0] * P.alpha) |
                        (to16<T>(acc[j][i][4 * e + 1] * P.alpha) << 16);
                pk[1] = to16<T>(acc[j][i][4 * e + 2] * P.alpha) |
                        (to16<T>(acc[j][i][4 * e + 3] * P.alpha) << 16);
                *(u32x2 *)(out + obase + ch) = pk;
            }
        }
    }
}

template <class T, int BM, int BN, int BKC, int STAGES>
static hipError_t launch_c8_cfg(TNParams &p, hipStream_t st) {
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.ncols + BN - 1) / BN;
    const int64_t nb = (int64_t)p.tiles_m * p.tiles_n * p.groups;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    // k_iters counts BKC*8-element slices here
    p.k_iters = (int32_t)(((int64_t)p.taps.n * p.cr + BKC * 8 - 1) / (BKC * 8));
    if (p.cr % (BKC * 8) == 0)
        hipLaunchKernelGGL((igemm_c8_kernel<T, BM, BN, BKC, STAGES, true>), dim3((uint32_t)nb),
                           dim3(256), 0, st, p);
    else
        hipLaunchKernelGGL((igemm_c8_kernel<T, BM, BN, BKC, STAGES, false>), dim3((uint32_t)nb),
                           dim3(256), 0, st, p);
    return hipGetLastError();
}

template <class T>
static hipError_t launch_c8_t(C8Config cfg, TNParams &p, hipStream_t st) {
    switch (cfg) {
        case C8_256x64: return launch_c8_cfg<T, 256, 64, 4, 4>(p, st);
        case C8_256x128: return launch_c8_cfg<T, 256, 128, 4, 3>(p, st);
        case C8_128x128:
        default: return launch_c8_cfg<T, 128, 128, 4, 4>(p, st);
    }
}

hipError_t launch_igemm_c8(int dtype, C8Config cfg, TNParams &p, hipStream_t st) {
    if (dtype == Half::id) return launch_c8_t<Half>(cfg, p, st);
    return launch_c8_t<BFloat>(cfg, p, st);
}

}  // namespace nnconv
