// igemm_c64.hip -- large-tile implicit-GEMM convolution for the forward pass
// and each stride phase of the backward-data pass, for reductions whose
// per-tap channel count is a multiple of 64 (every ResNet-50 layer but the
// stem).
//
// Design (gfx950):
//   - block tile BM x BN, NW = WM x WN waves, wave tiles built from
//     v_mfma_f32_32x32x16 blocks (up to 128 x 64 per wave): few LDS fragment
//     reads and few global loads per matrix-core instruction;
//   - k-slices of BKC x 8 reduction elements staged straight from memory
//     into LDS with buffer_load ... lds, STAGES deep, one barrier per slice;
//     configurations are sized so two workgroups share a CU, so one
//     workgroup's barrier wait is covered by the other's MFMAs;
//   - per-lane load offsets are fixed for the whole kernel; the part that
//     changes from slice to slice (tap and channel base) is uniform and is
//     folded into the buffer descriptor's base address with scalar
//     instructions, so a slice costs almost no vector ALU work;
//   - zero padding: rows outside the GEMM get an out-of-range offset once;
//     for padded convolutions each staged row carries a bitmask of the taps
//     that land inside the image, tested per load.
#include "igemm_store.hpp"

namespace nnconv {

namespace c64 {

// LDS tile: BKC 16-byte chunks per row; row r, logical chunk c at slot
// r*BKC + (c ^ swz(r)).  The 64 LDS banks serve a 16-byte read for 16 lanes
// per cycle, and a fragment read has 16 consecutive rows at one logical
// chunk: the swizzle spreads them over 16 distinct 16-byte bank groups
// (128-byte rows: parity picks the half, (r>>1)&7 the chunk; 64-byte rows:
// r&3 picks the quarter, (r>>2)&3 the chunk).
template <int BKC>
__device__ __forceinline__ int swz(int r) {
    return BKC == 8 ? ((r >> 1) & 7) : ((r >> 2) & 3);
}
template <int BKC>
__device__ __forceinline__ int slot(int r, int c) {
    return r * BKC + (c ^ swz<BKC>(r));
}

}  // namespace c64

// DIAG: the per-tap 64x64 weight blocks of every 64-column group are
// block-diagonal in 32x32 blocks (grouped convolution run as 64-channel
// super-groups, groups of at most 32 channels), so a wave's 32 output
// columns meet only the matching 32 reduction channels of each 64-channel
// slice: two of its four k-steps.
//
// RING: the k-slices cycle through an LDS ring of STAGES buffers (STAGES - 1
// slices in flight while one is multiplied), and each wave reads the
// fragments of the next k-step -- across the slice boundary too -- before it
// issues the matrix-core instructions of the current one, so LDS latency
// overlaps MFMA work inside the wave instead of relying on other waves.
// OCC: resident workgroups per CU the register budget is sized for.
template <class T, int BM, int BN, int WM, int WN, int BKC, int STAGES, bool PAD, bool DIAG,
          bool RING, int OCC>
__global__ __launch_bounds__(WM * WN * 64, OCC)
void igemm_c64_kernel(const TNParams P) {
    using namespace c64;
    constexpr int NW = WM * WN;             // waves per workgroup
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int BK = BKC * 8;             // reduction elements per slice
    constexpr int RPI = 64 / BKC;           // rows covered by one 64-lane load
    constexpr int A_LD = BM / (RPI * NW);   // loads per thread per slice (A)
    constexpr int B_LD = BN / (RPI * NW);   // loads per thread per slice (B)
    constexpr int A_SLOTS = BM * BKC, B_SLOTS = BN * BKC;
    constexpr int STAGE_SLOTS = A_SLOTS + B_SLOTS;
    constexpr int LOADS = A_LD + B_LD;
    static_assert(FM >= 1 && FN >= 1 && A_LD >= 1 && B_LD >= 1, "tile shape");
    static_assert(!DIAG || (FN == 1 && WTN == 32 && BKC == 8), "block-diagonal: 32-column waves");

    constexpr int LDS_SLOTS = STAGES * STAGE_SLOTS > BM * BN / 8 ? STAGES * STAGE_SLOTS : BM * BN / 8;
    __shared__ u32x4 lds[LDS_SLOTS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM, wn = wave / WM;

    // phase of this workgroup: phases own consecutive ranges of hardware
    // block ids, which the dispatcher deals round-robin to the XCDs, so every
    // XCD gets a share of every phase; within a phase, consecutive tiles are
    // then renumbered onto the same XCD
    int phi = 0;
    for (int i = 1; i < P.nphase; ++i)
        if ((int)blockIdx.x >= P.ph[i].block_start) phi = i;
    const TNPhase &F = P.ph[phi];
    const int phase_blocks =
        (phi + 1 < P.nphase ? P.ph[phi + 1].block_start : (int)gridDim.x) - F.block_start;
    const int local = (int)xcd_remap(blockIdx.x - F.block_start, phase_blocks);
    const int per_g = F.tiles_m * P.tiles_n;
    const int g = local / per_g;
    const int rem = local - g * per_g;
    const int tm = rem / P.tiles_n;
    const int tn = rem - tm * P.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;
    const int tap0 = F.tap_start, ntaps = F.tap_count;

    // Staging role: load j of this wave fills rows (wave*LD + j)*RPI + lane/BKC,
    // physical chunk lane%BKC, i.e. logical chunk (lane%BKC) ^ swz(row).
    const int lrow = lane / BKC;
    const int pch = lane & (BKC - 1);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];

    uint32_t a_voff[A_LD];
    uint64_t a_mask[A_LD];
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
        const int r = (wave * A_LD + j) * RPI + lrow;
        const int lchunk = pch ^ swz<BKC>(r);
        const int m = m0 + r;
        a_mask[j] = 0;
        if (m < F.M) {
            const int q1 = (int)fdiv((uint32_t)m, F.div_mj);
            const int jj = m - q1 * F.mj;
            const int n = (int)fdiv((uint32_t)q1, F.div_mi);
            const int ii = q1 - n * F.mi;
            const int bh = ii * P.ai_mul + P.ai_add;
            const int bw = jj * P.aj_mul + P.aj_add;
            // byte offset of this row's base pixel and chunk (may wrap below 0
            // for padded rows: only used together with a valid tap shift)
            a_voff[j] = (uint32_t)(((n * P.a_h + bh) * P.a_w + bw) * P.a_c + g * P.a_cg_ofs) * 2u +
                        (uint32_t)lchunk * 16u;
            if constexpr (PAD) {
                for (int t = 0; t < ntaps; ++t) {
                    const int h = bh + P.taps.dh[tap0 + t], w = bw + P.taps.dw[tap0 + t];
                    if ((unsigned)h < (unsigned)P.a_h && (unsigned)w < (unsigned)P.a_w)
                        a_mask[j] |= (uint64_t)1 << t;
                }
            }
        } else {
            a_voff[j] = OOB_OFFSET;
        }
    }
    uint32_t b_voff[B_LD];
#pragma unroll
    for (int j = 0; j < B_LD; ++j) {
        const int r = (wave * B_LD + j) * RPI + lrow;
        const int lchunk = pch ^ swz<BKC>(r);
        const int col = n0 + r;
        b_voff[j] = col < P.ncols
                        ? (uint32_t)(g * P.b_g_ofs + col * P.b_ld) * 2u + (uint32_t)lchunk * 16u
                        : OOB_OFFSET;
    }

    int ld_t = 0, ld_c = 0;  // tap and channel base of the next slice to load

    // Per-tap byte shifts, tap t held by lane t: the loop reads them back
    // with v_readlane instead of loading the tap table from memory each slice.
    const int tl = tap0 + (lane < ntaps ? lane : 0);
    const uint32_t tap_ashift =
        (uint32_t)(P.taps.dh[tl] * P.a_w + P.taps.dw[tl]) * (uint32_t)P.a_c * 2u;
    const uint32_t tap_boff = (uint32_t)P.taps.boff[tl] * 2u;

    // One slice's staging, split so that its loads can be spread between
    // matrix-core instructions: prepare() sets the slice's descriptors and
    // shifts (wave-uniform) and advances to the next slice, load(j) issues load
    // j (the A loads, then the B loads).  A slice past the end of the
    // reduction (live = false) gets empty descriptors: its loads deliver
    // zeros without touching memory.
    uint32_t sl_ashift = 0, sl_sb = 0;
    int sl_t = 0;
    i32x4 sl_da = {}, sl_db = {};
    auto prepare = [&](int buf, bool live) {
        // A: x / dy rows; the tap's pixel shift can be negative, so it is
        // added to the lane offsets; the channel base moves the descriptor
        sl_ashift = (uint32_t)__builtin_amdgcn_readlane((int)tap_ashift, ld_t);
        const uint32_t bshift = (uint32_t)__builtin_amdgcn_readlane((int)tap_boff, ld_t);
        sl_da = desc_at(P.a, live ? P.a_bytes : 0u, (uint32_t)ld_c * 2u);
        sl_db = desc_at(P.b, live ? P.b_bytes : 0u, bshift + (uint32_t)ld_c * 2u);
        sl_sb = lds0 + (uint32_t)(buf * STAGE_SLOTS) * 16u;
        sl_t = ld_t;
        // taps inner, channel slices outer: the taps of one channel slice
        // re-read overlapping pixels back to back, while they are still in L2
        if (++ld_t == ntaps) {
            ld_t = 0;
            ld_c += BK;
        }
    };
    auto load = [&](int j) {
        if (j < A_LD) {
            uint32_t off = a_voff[j] + sl_ashift;
            if constexpr (PAD) {
                if (!((a_mask[j] >> sl_t) & 1)) off = OOB_OFFSET;
            } else {
                if (a_voff[j] == OOB_OFFSET) off = OOB_OFFSET;
            }
            dma16(sl_sb + (uint32_t)((wave * A_LD + j) * 64) * 16u, off, sl_da);
        } else {
            const int jb = j - A_LD;
            dma16(sl_sb + (uint32_t)(A_SLOTS + (wave * B_LD + jb) * 64) * 16u, b_voff[jb], sl_db);
        }
    };
    auto issue = [&](int buf) {
        prepare(buf, true);
#pragma unroll
        for (int j = 0; j < LOADS; ++j) load(j);
    };

    f32x16 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x16{};

    const int l32 = lane & 31;
    const int khalf = lane >> 5;
    const int k_iters = ntaps * (P.cr / BK);

    auto compute = [&](const u32x4 *st) {
        if constexpr (DIAG) {
            // k-steps 2h, 2h+1 carry the reduction channels 32h .. 32h+31 of
            // the slice, h = the half of the 64-column group the wave's
            // columns lie in
            const int h = (wn * WTN / 32) & 1;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const int kc = 2 * (2 * h + kk) + khalf;
                u32x4 fp[FM];
#pragma unroll
                for (int i = 0; i < FM; ++i) fp[i] = st[slot<BKC>(wm * WTM + i * 32 + l32, kc)];
                const u32x4 fw = st[A_SLOTS + slot<BKC>(wn * WTN + l32, kc)];
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[0][i] = mfma32<T>(fw, fp[i], acc[0][i]);
            }
            return;
        }
#pragma unroll
        for (int ks = 0; ks < BKC / 2; ++ks) {
            const int kc = 2 * ks + khalf;
            u32x4 fp[FM], fw[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) fp[i] = st[slot<BKC>(wm * WTM + i * 32 + l32, kc)];
#pragma unroll
            for (int j = 0; j < FN; ++j)
                fw[j] = st[A_SLOTS + slot<BKC>(wn * WTN + j * 32 + l32, kc)];
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[j][i] = mfma32<T>(fw[j], fp[i], acc[j][i]);
        }
    };

    if constexpr (STAGES == 1) {
        // short reductions: no pipeline; several resident workgroups per CU
        // overlap each other's loads, MFMAs and stores instead
        for (int kt = 0; kt < k_iters; ++kt) {
            if (kt > 0) barrier_lds();  // previous slice fully read
            issue(0);
            wait_vmcnt<0>();
            barrier_lds();
            compute(&lds[0]);
        }
    } else if constexpr (RING) {
        static_assert(!DIAG && STAGES >= 2 && BKC % 4 == 0, "ring: dense, 2+ stages, even k-steps");
        constexpr int KS = BKC / 2;  // 16-deep k-steps per slice (even)
        u32x4 fa[2][FM], fb[2][FN];
        auto read_frags = [&](const u32x4 *st, int ks, u32x4 (&a)[FM], u32x4 (&b)[FN]) {
            const int kc = 2 * ks + khalf;
#pragma unroll
            for (int i = 0; i < FM; ++i) a[i] = st[slot<BKC>(wm * WTM + i * 32 + l32, kc)];
#pragma unroll
            for (int j = 0; j < FN; ++j) b[j] = st[A_SLOTS + slot<BKC>(wn * WTN + j * 32 + l32, kc)];
        };
        auto mma = [&](const u32x4 (&a)[FM], const u32x4 (&b)[FN]) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[j][i] = mfma32<T>(b[j], a[i], acc[j][i]);
        };
        // the same k-step with the loads of a prepared slice placed between
        // its matrix-core instructions (the scheduling fences keep them
        // there), so issuing them costs no matrix-core time
        auto mma_loads = [&](const u32x4 (&a)[FM], const u32x4 (&b)[FN]) {
            constexpr int NM = FM * FN;
            constexpr int STRIDE = NM >= 2 * LOADS ? NM / LOADS : 1;
#pragma unroll
            for (int j = 0; j < FN; ++j) {
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    const int m = j * FM + i;
                    acc[j][i] = mfma32<T>(b[j], a[i], acc[j][i]);
                    if (m % STRIDE == 0 && m / STRIDE < LOADS) {
                        __builtin_amdgcn_sched_barrier(0);
                        load(m / STRIDE);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            }
#pragma unroll
            for (int l = (NM + STRIDE - 1) / STRIDE; l < LOADS; ++l) load(l);
        };
        // the k-steps of one slice but its last: each reads the next k-step's
        // fragments, then multiplies
        auto slice_body = [&](const u32x4 *st) {
#pragma unroll
            for (int ks = 0; ks + 1 < KS; ++ks) {
                read_frags(st, ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
                mma(fa[ks & 1], fb[ks & 1]);
            }
        };
        if (k_iters > 0) {
            // prologue: every buffer of the ring gets a slice (slices past
            // the end load nothing, but keep the wait counts uniform)
            for (int s = 0; s < STAGES; ++s) {
                prepare(s, s < k_iters);
#pragma unroll
                for (int j = 0; j < LOADS; ++j) load(j);
            }
            wait_vmcnt<(STAGES - 1) * LOADS>();  // slice 0 landed
            barrier_lds();
            read_frags(&lds[0], 0, fa[0], fb[0]);
            for (int kt = 0; kt + 1 < k_iters; ++kt) {
                slice_body(&lds[(kt % STAGES) * STAGE_SLOTS]);
                // slice kt + 1 has landed once at most STAGES - 2 later
                // slices are pending; after the barrier no wave reads slice
                // kt any more (its last fragments are in registers), so its
                // buffer takes slice kt + STAGES.  The fence keeps the
                // k-steps above ahead of the wait.
                __builtin_amdgcn_sched_barrier(0);
                wait_vmcnt<(STAGES - 2) * LOADS>();
                barrier_lds();
                read_frags(&lds[((kt + 1) % STAGES) * STAGE_SLOTS], 0, fa[0], fb[0]);
                prepare(kt % STAGES, kt + STAGES < k_iters);
                mma_loads(fa[1], fb[1]);
            }
            slice_body(&lds[((k_iters - 1) % STAGES) * STAGE_SLOTS]);
            mma(fa[1], fb[1]);
            // slices past the end may still be landing (as zeros) in the
            // buffers the epilogue reuses
            wait_vmcnt<0>();
        }
    } else if (k_iters > 0) {
        const int pro = k_iters < STAGES - 1 ? k_iters : STAGES - 1;
        for (int s = 0; s < pro; ++s) issue(s);
        for (int kt = 0; kt < k_iters; ++kt) {
            // slice kt has landed once at most (STAGES-2) later slices are pending
            if (kt + STAGES - 2 < k_iters)
                wait_vmcnt<(STAGES - 2) * LOADS>();
            else
                wait_vmcnt<0>();
            barrier_lds();
            if (kt + STAGES - 1 < k_iters) issue((kt + STAGES - 1) % STAGES);
            compute(&lds[(kt % STAGES) * STAGE_SLOTS]);
        }
    }

    static_assert(BM * BN / 8 <= LDS_SLOTS, "C tile must fit in LDS");
    store_tile<T, BM, BN, WM, WN, FM, FN>(acc, &lds[0], P, F, m0, n0, g);
}

template <class T, int BM, int BN, int WM, int WN, int BKC, int STAGES, bool DIAG = false,
          bool RING = false,
          int OCC = (WM * WN == 4) ? ((BM * BN <= 128 * 128) ? 4 : 2) : 1>
static hipError_t launch_c64_cfg(TNParams &p, bool pad, hipStream_t st) {
    p.tiles_n = (p.ncols + BN - 1) / BN;
    int64_t nb = 0;
    for (int i = 0; i < p.nphase; ++i) {
        p.ph[i].tiles_m = (p.ph[i].M + BM - 1) / BM;
        p.ph[i].block_start = (int32_t)nb;
        nb += (int64_t)p.ph[i].tiles_m * p.tiles_n * p.groups;
    }
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (pad)
        hipLaunchKernelGGL((igemm_c64_kernel<T, BM, BN, WM, WN, BKC, STAGES, true, DIAG, RING, OCC>),
                           dim3((uint32_t)nb), dim3(WM * WN * 64), 0, st, p);
    else
        hipLaunchKernelGGL((igemm_c64_kernel<T, BM, BN, WM, WN, BKC, STAGES, false, DIAG, RING, OCC>),
                           dim3((uint32_t)nb), dim3(WM * WN * 64), 0, st, p);
    return hipGetLastError();
}

// Configurations (LDS per workgroup in parentheses):
//   256x256: 8 waves of 128x64, 64-element slices, 2 stages (128 KB)
//   256x256 wide: 16 waves of 64x64, same LDS; four waves per SIMD hide
//            the fragment-read latency better on some mid-size layers
//   128x128: 4 waves of 64x64, 64-element slices, 2 stages (64 KB; two
//            workgroups per CU)
// Single-stage tiles, whose small LDS footprint lets 3-5 workgroups share a
// CU and cover each other's load latency:
//   128x128: 4 waves of 64x64 (32 KB);  128x64: 4 waves of 64x32 (24 KB),
//   also with block-diagonal 32x32 weight blocks (half the k-steps)
template <class T>
static hipError_t launch_c64_t(C64Config cfg, TNParams &p, bool pad, hipStream_t st) {
    switch (cfg) {
        case C64_256x256: return launch_c64_cfg<T, 256, 256, 2, 4, 8, 2>(p, pad, st);
        case C64W_256x256: return launch_c64_cfg<T, 256, 256, 4, 4, 8, 2>(p, pad, st);
        case C64_128x128: return launch_c64_cfg<T, 128, 128, 2, 2, 8, 2>(p, pad, st);
        case C64S_128x64: return launch_c64_cfg<T, 128, 64, 2, 2, 8, 1>(p, pad, st);
        case C64D_128x64: return launch_c64_cfg<T, 128, 64, 2, 2, 8, 1, true>(p, pad, st);
        case C64R_256x256: return launch_c64_cfg<T, 256, 256, 2, 2, 4, 4, false, true, 1>(p, pad, st);
        case C64R_256x128: return launch_c64_cfg<T, 256, 128, 2, 2, 4, 3, false, true, 2>(p, pad, st);
        case C64R_256x64: return launch_c64_cfg<T, 256, 64, 4, 1, 4, 4, false, true, 2>(p, pad, st);
        case C64S_128x128:
        default: return launch_c64_cfg<T, 128, 128, 2, 2, 8, 1>(p, pad, st);
    }
}

hipError_t launch_igemm_c64(int dtype, C64Config cfg, TNParams &p, bool pad, hipStream_t st) {
    if (dtype == Half::id) return launch_c64_t<Half>(cfg, p, pad, st);
    return launch_c64_t<BFloat>(cfg, p, pad, st);
}

}  // namespace nnconv
