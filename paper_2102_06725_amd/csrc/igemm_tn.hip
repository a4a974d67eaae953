// igemm_tn.hip -- implicit-GEMM convolution on the gfx950 matrix cores for
// the forward pass and for each stride phase of the backward-data pass.
//
// GEMM view (channel-last operands, both reduction-contiguous):
//   rows    = output pixels (M), read from the A image through the tap table
//   columns = output channels (per group)
//   reduction = (tap, channel), 64 elements per k-iteration
// A workgroup of 4 waves computes a BM x BN tile; each wave a (BM/WM) x
// (BN/WN) sub-tile of 32x32 MFMA blocks.  Global -> register -> LDS staging
// is double buffered (one barrier per k-iteration); padding and ragged edges
// come from buffer-load range checks (masked lanes read zeros).
#include "launch.hpp"

namespace nnconv {

template <class T, int BM, int BN, int WM, int WN, bool ALIGNED>
__global__ __launch_bounds__(256, 2) void igemm_tn_kernel(const TNParams P) {
    constexpr int CH = 8;            // 16-byte chunks in a 64-element row slice
    constexpr int PLD = BM / 32;     // pixel-row chunks each thread stages
    constexpr int WLD = BN / 32;     // weight-row chunks each thread stages
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    static_assert(WM * WN == 4, "4 waves per workgroup");
    static_assert(FM >= 1 && FN >= 1, "wave tile at least 32x32");

    __shared__ u32x4 lds[2][(BM + BN) * CH];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;

    // tile of this workgroup: groups x m-tiles x n-tiles, n fastest
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int per_g = P.tiles_m * P.tiles_n;
    const int g = (int)lid / per_g;
    const int rem = (int)lid - g * per_g;
    const int tm = rem / P.tiles_n;
    const int tn = rem - tm * P.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(P.a, P.a_bytes);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(P.b, P.b_bytes);

    const int cv = tid & 7;     // chunk (8 channels) of the 64-wide slice this thread stages
    const int rsub = tid >> 3;  // first staged row; rows rsub + 32*i

    int pr_pix[PLD], pr_h[PLD], pr_w[PLD];
#pragma unroll
    for (int i = 0; i < PLD; ++i) {
        const int m = m0 + rsub + 32 * i;
        if (m < P.M) {
            const int q1 = (int)fdiv((uint32_t)m, P.div_mj);
            const int jj = m - q1 * P.mj;
            const int n = (int)fdiv((uint32_t)q1, P.div_mi);
            const int ii = q1 - n * P.mi;
            const int bh = ii * P.ai_mul + P.ai_add;
            const int bw = jj * P.aj_mul + P.aj_add;
            pr_h[i] = bh;
            pr_w[i] = bw;
            pr_pix[i] = (n * P.a_h + bh) * P.a_w + bw;
        } else {
            pr_h[i] = -(1 << 24);  // never inside the image
            pr_w[i] = 0;
            pr_pix[i] = 0;
        }
    }
    int wr_off[WLD];
    bool wr_ok[WLD];
#pragma unroll
    for (int i = 0; i < WLD; ++i) {
        const int col = n0 + rsub + 32 * i;
        wr_ok[i] = col < P.ncols;
        wr_off[i] = g * P.b_g_ofs + col * P.b_ld;
    }
    const int a_ch0 = g * P.a_cg_ofs;
    const int crv = P.cr >> 3;

    u32x4 sa[PLD], sw[WLD];
    int next_t = 0, next_c = 0;  // ALIGNED: tap / channel base of the next slice

    auto gload = [&](int kt) {
        int t, c;
        if constexpr (ALIGNED) {
            t = next_t;
            c = next_c + cv * 8;
            next_c += 64;
            if (next_c == P.cr) {
                next_c = 0;
                ++next_t;
            }
        } else {
            const int gv = kt * CH + cv;
            t = (int)fdiv((uint32_t)gv, P.div_crv);
            c = (gv - t * crv) * 8;
        }
        const bool tv = t < P.taps.n;
        const int tt = tv ? t : 0;
        const int dh = P.taps.dh[tt], dw = P.taps.dw[tt], bo = P.taps.boff[tt];
#pragma unroll
        for (int i = 0; i < PLD; ++i) {
            const int h = pr_h[i] + dh, w = pr_w[i] + dw;
            const bool ok = tv && (unsigned)h < (unsigned)P.a_h && (unsigned)w < (unsigned)P.a_w;
            const int off = ((pr_pix[i] + dh * P.a_w + dw) * P.a_c + a_ch0 + c) * 2;
            sa[i] = load16(ra, ok ? (uint32_t)off : OOB_OFFSET);
        }
#pragma unroll
        for (int i = 0; i < WLD; ++i) {
            const bool ok = tv && wr_ok[i];
            const int off = (wr_off[i] + bo + c) * 2;
            sw[i] = load16(rb, ok ? (uint32_t)off : OOB_OFFSET);
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < PLD; ++i) {
            const int r = rsub + 32 * i;
            lds[buf][r * CH + (cv ^ swz(r))] = sa[i];
        }
#pragma unroll
        for (int i = 0; i < WLD; ++i) {
            const int r = rsub + 32 * i;
            lds[buf][(BM + r) * CH + (cv ^ swz(r))] = sw[i];
        }
    };

    f32x16 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x16{};

    if (P.k_iters > 0) {
        gload(0);
        lstore(0);
    }
    __syncthreads();

    const int l32 = lane & 31;
    const int khalf = lane >> 5;
    for (int kt = 0; kt < P.k_iters; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < P.k_iters;
        if (more) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int kc = 2 * ks + khalf;
            u32x4 fp[FM], fw[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int r = wm * WTM + i * 32 + l32;
                fp[i] = lds[buf][r * CH + (kc ^ swz(r))];
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int r = wn * WTN + j * 32 + l32;
                fw[j] = lds[buf][(BM + r) * CH + (kc ^ swz(r))];
            }
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[j][i] = mfma32<T>(fw[j], fp[i], acc[j][i]);
        }
        if (more) lstore(buf ^ 1);
        __syncthreads();
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
                const float v0 = acc[j][i][4 * e + 0] * P.alpha;
                const float v1 = acc[j][i][4 * e + 1] * P.alpha;
                const float v2 = acc[j][i][4 * e + 2] * P.alpha;
                const float v3 = acc[j][i][4 * e + 3] * P.alpha;
                u32x2 pk;
                pk[0] = to16<T>(v0) | (to16<T>(v1) << 16);
                pk[1] = to16<T>(v2) | (to16<T>(v3) << 16);
                *(u32x2 *)(out + obase + ch) = pk;
            }
        }
    }
}

template <class T, int BM, int BN, int WM, int WN>
static hipError_t launch_cfg(TNParams &p, hipStream_t st) {
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.ncols + BN - 1) / BN;
    const int64_t nb = (int64_t)p.tiles_m * p.tiles_n * p.groups;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    const bool aligned = (p.cr % 64) == 0;
    if (aligned)
        hipLaunchKernelGGL((igemm_tn_kernel<T, BM, BN, WM, WN, true>), dim3((uint32_t)nb),
                           dim3(256), 0, st, p);
    else
        hipLaunchKernelGGL((igemm_tn_kernel<T, BM, BN, WM, WN, false>), dim3((uint32_t)nb),
                           dim3(256), 0, st, p);
    return hipGetLastError();
}

template <class T>
static hipError_t launch_t(TNConfig cfg, TNParams &p, hipStream_t st) {
    switch (cfg) {
        case TN_256x64: return launch_cfg<T, 256, 64, 4, 1>(p, st);
        case TN_256x128: return launch_cfg<T, 256, 128, 2, 2>(p, st);
        case TN_128x128:
        default: return launch_cfg<T, 128, 128, 2, 2>(p, st);
    }
}

hipError_t launch_igemm_tn(int dtype, TNConfig cfg, TNParams &p, hipStream_t st) {
    if (dtype == Half::id) return launch_t<Half>(cfg, p, st);
    return launch_t<BFloat>(cfg, p, st);
}

}  // namespace nnconv
