// wgrad_halo.hip -- backward-weight pass of 3x3 stride-1 "same" convolutions
// with 64 input and 64 output channels per group (the 56x56 3x3 layers of
// ResNet-50's first stage, and the 64-channel super-groups of grouped
// layers), without an im2col.
//
//   part[split][k][t * 64 + c] = sum over the split's pixels p of
//                                dy[p][k] * x[p + shift(t)][c]   (zero outside the image)
//
// A block is RB whole image rows of one image (RB * W a multiple of 16
// pixels, at most 128).  Per block, dy (RB * W pixels) and the input rows
// h0 - 1 .. h0 + RB, padded with one zero column on each side, come into LDS
// with buffer_load ... lds; rows and columns outside the image load as
// zeros, so tap (dh, dw) of every pixel is the staged input at the constant
// offset dh * (W + 2) + dw from the pixel's centre position, with no per-tap
// masks.  Each staged pixel takes 144 bytes (64 channels and a zero 16-byte
// pad): the four pixels of a transposing read then fall in four different
// bank groups for any row offset, so tap offsets need no swizzle.
//
// Eight waves, two per SIMD: wave w multiplies for the 32 input channels
// 32 * (w & 1) .. and the taps {0, 1, 2}, {3, 4}, {5, 6} or {7, 8} (w / 2),
// both 32-row halves of the 64 output channels.  A k-step (16 pixels) reads
// two dy fragments and one input fragment per tap, and issues two
// matrix-core instructions per tap.  The workgroup runs its split's
// blocks in order, the next block's staging in flight during the current
// block's k-steps, and writes one fp32 partial (summed in a fixed order by
// the split reduction).  Blocks cycle through three LDS buffers, so two
// blocks' staging is in flight while one is multiplied: a block is about a
// microsecond of matrix-core work, less than a loaded HBM round trip.
#include <type_traits>

#include "launch.hpp"

namespace nnconv {

namespace wgh {

constexpr int PITCH = 144;                  // LDS bytes per staged pixel
constexpr int CHUNKS = PITCH / 16;          // 16-byte chunks per staged pixel (the last is zero)
constexpr int MAXP = 128;                   // pixels per block
constexpr int MAXKS = MAXP / 16;            // k-steps per block
// A buffer is nslot slots of 16 bytes: dy in slots [0, dys) (npix * 9
// rounded up to whole 64-slot loads), the staged input from dys on.
static_assert(WGH_MAX_SLOTS % 64 == 0, "whole loads");

// s_waitcnt vmcnt(n) for a wave-uniform n < 16 known only at run time
__device__ __forceinline__ void wait_vmcnt_rt(int n) {
    switch (n) {
        case 0: wait_vmcnt<0>(); break;
        case 1: wait_vmcnt<1>(); break;
        case 2: wait_vmcnt<2>(); break;
        case 3: wait_vmcnt<3>(); break;
        case 4: wait_vmcnt<4>(); break;
        case 5: wait_vmcnt<5>(); break;
        case 6: wait_vmcnt<6>(); break;
        case 7: wait_vmcnt<7>(); break;
        case 8: wait_vmcnt<8>(); break;
        case 9: wait_vmcnt<9>(); break;
        case 10: wait_vmcnt<10>(); break;
        case 11: wait_vmcnt<11>(); break;
        case 12: wait_vmcnt<12>(); break;
        case 13: wait_vmcnt<13>(); break;
        case 14: wait_vmcnt<14>(); break;
        default: wait_vmcnt<0>(); break;
    }
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ u32x4 pack_tr(s16x4 v0, s16x4 v1) {
    u32x4 r;
    r[0] = (uint32_t)(uint16_t)v0[0] | ((uint32_t)(uint16_t)v0[1] << 16);
    r[1] = (uint32_t)(uint16_t)v0[2] | ((uint32_t)(uint16_t)v0[3] << 16);
    r[2] = (uint32_t)(uint16_t)v1[0] | ((uint32_t)(uint16_t)v1[1] << 16);
    r[3] = (uint32_t)(uint16_t)v1[2] | ((uint32_t)(uint16_t)v1[3] << 16);
    return r;
}

// Operand fragment of 8 consecutive pixels per lane: two transposing reads
// of four staged pixels each, at LDS byte addresses a0 and a1.
__device__ __forceinline__ u32x4 tr_frag(uint32_t a0, uint32_t a1) {
    const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)a0);
    const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)a1);
    return pack_tr(v0, v1);
}

}  // namespace wgh

// WAVES waves (4: taps 0-4 / 5-8 per wave, 8: {0, 1, 2}, {3, 4}, {5, 6},
// {7, 8}), NBUF block buffers in LDS (NBUF - 1 blocks in flight).  Group
// blockIdx.y of 64 channels.  DIAG: block-diagonal 32x32 gradient blocks
// (super-groups of groups of at most 32 channels): a wave computes only the
// 32-row half of the output channels that matches its 32 input channels.
template <class T, int WAVES, int NBUF, bool DIAG>
__global__ __launch_bounds__(WAVES * 64, 1) void wgrad_halo_kernel(const WGHParams P) {
    using namespace wgh;
    static_assert(WAVES == 4 || WAVES == 8, "tap groups");
    static_assert(NBUF == 2 || NBUF == 3, "buffers");
    constexpr int LD = (WGH_MAX_SLOTS / 64 + WAVES - 1) / WAVES;  // loads per wave and block, at most
    constexpr int LDS_BYTES = NBUF * WGH_MAX_SLOTS * 16;
    static_assert(LDS_BYTES <= 160 * 1024 && LD < 16, "LDS budget, wait counts");
    // taps of tap group g: T0(g) .. T0(g) + NT(g) - 1
    constexpr int NG = WAVES / 2, NTMAX = WAVES == 4 ? 5 : 3;
    __shared__ u32x4 lds[LDS_BYTES / 16];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];
    const i32x4 ddy = desc_of(P.dy, P.dy_bytes);
    const i32x4 dx = desc_of(P.x, P.x_bytes);
    const int grp = (int)blockIdx.y;
    const uint32_t goff = (uint32_t)grp * 128u;  // the group's 64 channels, in bytes

    const int W = P.w, H = P.h, RB = P.rb, W2 = P.w + 2;
    const int npix = RB * W;          // pixels per block, a multiple of 16
    const int nx = (RB + 2) * W2;     // staged input pixels per block
    const int ksteps = npix >> 4;
    const int dys = (npix * CHUNKS + 63) & ~63;            // dy slots
    const int nslot = (dys + nx * CHUNKS + 63) & ~63;      // slots per buffer (<= WGH_MAX_SLOTS)
    const uint32_t buf_bytes = (uint32_t)nslot * 16u;
    const uint32_t xoff = (uint32_t)dys * 16u;              // staged input within a buffer

    // ---- staging roles, the same for every block: load j of this wave
    // fills slots (j * WAVES + wave) * 64 .. + 63 of a buffer, all of dy or
    // all of the staged input (the dy slots are whole loads); lane slot e is
    // pixel e / 9, chunk e % 9 of its region.  What changes per block is the
    // image and its first row.  The wave issues nld of its LD loads (those
    // inside the buffer) per block.
    // packed per load: pixel offset from the block's first pixel (bits
    // 0-15, signed), row in the block + 1 (bits 16-23; the staged input's
    // first row is the one above the block), chunk (24-27), valid (31)
    uint32_t pk[LD];
#pragma unroll
    for (int j = 0; j < LD; ++j) {
        const int e = (j * WAVES + wave) * 64 + lane;
        int rel, row, ch;
        bool ok;
        if (e < dys) {
            const int p = e / CHUNKS;
            ch = e - p * CHUNKS;
            rel = p;        // the block's dy pixels are consecutive in memory
            row = p / W;
            ok = p < npix && ch < 8;
        } else {
            const int q = (e - dys) / CHUNKS;
            ch = (e - dys) - q * CHUNKS;
            const int yr = q / W2, xc = q - yr * W2;
            rel = (yr - 1) * W + (xc - 1);
            row = yr - 1;
            ok = q < nx && ch < 8 && xc >= 1 && xc <= W;
        }
        pk[j] = ((uint32_t)rel & 0xFFFFu) | ((uint32_t)(row + 1) & 0xFFu) << 16 |
                (uint32_t)(ch & 15) << 24 | (ok ? 0x80000000u : 0u);
    }

    int nld = 0;
#pragma unroll
    for (int j = 0; j < LD; ++j) nld += (j * WAVES + wave) * 64 < nslot ? 1 : 0;

    auto stage = [&](int b, int buf) {
        const int n = b / P.blocks_per_img;
        const int h0 = (b - n * P.blocks_per_img) * RB;
        const int pix0 = (n * H + h0) * W;   // first pixel of the block
        const uint32_t base = lds0 + (uint32_t)buf * buf_bytes;
#pragma unroll
        for (int j = 0; j < LD; ++j) {
            const int e0 = (j * WAVES + wave) * 64;
            if (e0 >= nslot) {
                // past the buffer: no load
            } else {
                const int rel = (int)(int16_t)(pk[j] & 0xFFFFu);
                const int ih = h0 + (int)((pk[j] >> 16) & 0xFFu) - 1;
                const uint32_t chb = ((pk[j] >> 24) & 15u) * 16u;
                const bool ok = (pk[j] >> 31) != 0 && (unsigned)ih < (unsigned)H;
                if (e0 < dys) {
                    const uint32_t off =
                        ok ? (uint32_t)(pix0 + rel) * (uint32_t)P.k_stride * 2u + goff + chb
                           : OOB_OFFSET;
                    dma16(base + (uint32_t)e0 * 16u, off, ddy);
                } else {
                    const uint32_t off =
                        ok ? (uint32_t)(pix0 + rel) * (uint32_t)P.c_stride * 2u + goff + chb
                           : OOB_OFFSET;
                    dma16(base + (uint32_t)e0 * 16u, off, dx);
                }
            }
        }
    };

    // ---- fragment roles.  Lane group gq = lane / 16 covers channels
    // 16 * (gq & 1) of a 32-channel block and pixels 8 * (gq >> 1) of the
    // k-step; within the group, lane li addresses pixel li / 4 (+4 for the
    // second read), channels 4 * (li & 3).
    const int li = lane & 15, gq = lane >> 4;
    const int fr_row = 8 * (gq >> 1) + (li >> 2);
    const uint32_t fr_col = (uint32_t)(16 * (gq & 1) + 4 * (li & 3)) * 2u;
    const int cb = wave & 1;          // input-channel block of this wave
    const int tg = wave >> 1;         // tap group
    // output-channel halves of this wave: both, or (DIAG) the one of its
    // input-channel block
    constexpr int NI = DIAG ? 1 : 2;
    auto half = [&](int i) { return DIAG ? cb : i; };
    // staged input position of pixel p's centre, in bytes: (p / W + 1) rows
    // of W + 2 pixels, column p % W + 1
    uint32_t xpos[MAXKS][2];
#pragma unroll
    for (int ks = 0; ks < MAXKS; ++ks)
#pragma unroll
        for (int rd = 0; rd < 2; ++rd) {
            const int p = ks * 16 + fr_row + 4 * rd;
            const int hr = p / W, w = p - hr * W;
            xpos[ks][rd] = xoff + (uint32_t)(((hr + 1) * W2 + w + 1) * PITCH) + (uint32_t)cb * 64u +
                           fr_col;
        }
    // tap t = (dh + 1) * 3 + (dw + 1): byte offset of its input pixel
    auto tap_off = [&](int t) -> int { return ((t / 3 - 1) * W2 + (t % 3 - 1)) * PITCH; };

    f32x16 acc[NI][NTMAX];
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int t = 0; t < NTMAX; ++t) acc[i][t] = f32x16{};
    // wave-uniform tap offsets, kept in scalar registers
    int toff[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) toff[t] = __builtin_amdgcn_readfirstlane(tap_off(t));

    // the k-steps of one staged block, taps T0 .. T0 + NT - 1
    auto block = [&](const uint32_t base, auto t0c, auto ntc) {
        constexpr int T0 = decltype(t0c)::value, NT = decltype(ntc)::value;
        // the fragments of k-step ks: NI of dy (the wave's 32-row halves of
        // the output channels), one of the staged input per tap
        auto read = [&](int ks, u32x4 (&fa)[NI], u32x4 (&fb)[NT]) {
            const uint32_t a = base + (uint32_t)((ks * 16 + fr_row) * PITCH) + fr_col;
#pragma unroll
            for (int i = 0; i < NI; ++i)
                fa[i] = tr_frag(a + half(i) * 64, a + half(i) * 64 + 4 * PITCH);
            // the pixel positions of this k-step, opaque to the compiler:
            // otherwise it keeps every (k-step, tap) address in registers
            uint32_t x0 = base + xpos[ks][0], x1 = base + xpos[ks][1];
            asm volatile("" : "+v"(x0), "+v"(x1));
#pragma unroll
            for (int t = 0; t < NT; ++t) fb[t] = tr_frag(x0 + toff[T0 + t], x1 + toff[T0 + t]);
        };
        // each k-step's fragments are read before the previous k-step's
        // matrix-core instructions issue (the fences keep that order and
        // keep the compiler from reading further ahead)
        u32x4 fa[2][NI], fb[2][NT];
        read(0, fa[0], fb[0]);
#pragma unroll
        for (int ks = 0; ks < MAXKS; ++ks) {
            if (ks < ksteps) {
                const int cur = ks & 1;
                if (ks + 1 < MAXKS && ks + 1 < ksteps) read(ks + 1, fa[cur ^ 1], fb[cur ^ 1]);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < NT; ++t)
#pragma unroll
                    for (int i = 0; i < NI; ++i) acc[i][t] = mfma32<T>(fa[cur][i], fb[cur][t], acc[i][t]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    const int b_begin = (int)blockIdx.x * P.blocks_per_split;
    const int b_end = min(P.nblocks, b_begin + P.blocks_per_split);
    // prologue: the split's first NBUF - 1 blocks in flight, wait for the first
    constexpr int AHEAD = NBUF - 1;
#pragma unroll
    for (int i = 0; i < AHEAD; ++i)
        if (b_begin + i < b_end) stage(b_begin + i, i);
    wait_vmcnt_rt(b_begin + AHEAD - 1 < b_end ? (AHEAD - 1) * nld : 0);
    barrier_lds();
    int buf = 0;
    for (int b = b_begin; b < b_end; ++b) {
        // block b + AHEAD into the buffer block b - 1 used: every wave has
        // left it (the barrier that ended block b - 1)
        const bool ahead = b + AHEAD < b_end;
        if (ahead) stage(b + AHEAD, buf == 0 ? NBUF - 1 : buf - 1);
        const uint32_t base = lds0 + (uint32_t)buf * buf_bytes;
        if constexpr (NG == 2) {
            if (tg == 0)
                block(base, std::integral_constant<int, 0>{}, std::integral_constant<int, 5>{});
            else
                block(base, std::integral_constant<int, 5>{}, std::integral_constant<int, 4>{});
        } else {
            if (tg == 0)
                block(base, std::integral_constant<int, 0>{}, std::integral_constant<int, 3>{});
            else if (tg == 1)
                block(base, std::integral_constant<int, 3>{}, std::integral_constant<int, 2>{});
            else if (tg == 2)
                block(base, std::integral_constant<int, 5>{}, std::integral_constant<int, 2>{});
            else
                block(base, std::integral_constant<int, 7>{}, std::integral_constant<int, 2>{});
        }
        // block b + 1 has landed (later ones may still be in flight), and no
        // wave reads block b any more
        wait_vmcnt_rt(ahead ? (AHEAD - 1) * nld : 0);
        barrier_lds();
        buf = buf == NBUF - 1 ? 0 : buf + 1;
    }

    // partial rows grp * 64 .. + 63 of [groups * 64 k][9 * 64]: lane holds
    // column l32 of its 32-channel block and rows 8 * (v / 4) + 4 * (lane /
    // 32) + v % 4 of each of its 32-row halves
    const int l32 = lane & 31, kh = lane >> 5;
    constexpr int NCOL = 9 * 64;
    float *dst = P.ws + ((int64_t)blockIdx.x * P.groups + grp) * 64 * NCOL;
    const int t0 = NG == 2 ? 5 * tg : (tg == 0 ? 0 : 2 * tg + 1);
    const int nt = NG == 2 ? (tg == 0 ? 5 : 4) : (tg == 0 ? 3 : 2);
#pragma unroll
    for (int t = 0; t < NTMAX; ++t) {
        if (t < nt) {
            const int col = (t0 + t) * 64 + cb * 32 + l32;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[(32 * half(i) + 8 * (v >> 2) + 4 * kh + (v & 3)) * NCOL + col] = acc[i][t][v];
        }
    }
}

int wgh_slots(int rb, int w) {
    const int dys = (rb * w * wgh::CHUNKS + 63) & ~63;
    return (dys + (rb + 2) * (w + 2) * wgh::CHUNKS + 63) & ~63;
}

hipError_t launch_wgrad_halo(int dtype, const WGHParams &p, hipStream_t st) {
    if (p.rb < 1 || p.w < 1 || p.rb * p.w > wgh::MAXP || (p.rb * p.w) % 16 != 0 ||
        wgh_slots(p.rb, p.w) > WGH_MAX_SLOTS || p.blocks_per_split < 1 || p.splits < 1 ||
        p.groups < 1 || p.groups > 65535 || p.c_stride < 64 * p.groups ||
        p.k_stride < 64 * p.groups)
        return hipErrorInvalidValue;
    // 8 waves and 3 buffers: on the 56x56 layer at batch 256, 86 us against
    // 87 with 2 buffers and 117-120 with 4 waves (one per SIMD does not hide
    // the transposing reads' latency)
    constexpr int WV = 8, NB = 3;
    const dim3 grid((uint32_t)p.splits, (uint32_t)p.groups);
    if (dtype == Half::id) {
        if (p.diag32)
            hipLaunchKernelGGL((wgrad_halo_kernel<Half, WV, NB, true>), grid, dim3(WV * 64), 0, st, p);
        else
            hipLaunchKernelGGL((wgrad_halo_kernel<Half, WV, NB, false>), grid, dim3(WV * 64), 0, st, p);
    } else {
        if (p.diag32)
            hipLaunchKernelGGL((wgrad_halo_kernel<BFloat, WV, NB, true>), grid, dim3(WV * 64), 0, st, p);
        else
            hipLaunchKernelGGL((wgrad_halo_kernel<BFloat, WV, NB, false>), grid, dim3(WV * 64), 0, st, p);
    }
    return hipGetLastError();
}

}  // namespace nnconv
