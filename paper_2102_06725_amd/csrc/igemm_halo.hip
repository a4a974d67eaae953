// igemm_halo.hip -- implicit-GEMM convolution with halo staging, for the
// stride-1 "same" geometries: the 3x3, padding-1 convolutions of the
// ResNet-50 bottlenecks, in the forward pass and in the backward-data pass
// (whose single stride phase is again a stride-1 correlation, Sec. 3.2).
//
// The 64-channel-slice kernel (igemm_c64.hip) stages an A tile per
// (tap, channel slice): a 3x3 filter stages every input pixel nine times.
// Here a tile is 256 consecutive output pixels in raster order (image,
// row, column).  At stride 1 with an A image of the output's size, tap t
// reads pixel m + shift(t) for output pixel m, shift(t) = dh*W + dw, so the
// pixels every tap of the tile needs form one run [m0 + lo, m0 + 256 + hi)
// of 256 + 2W + 2 pixels for a 3x3 filter.  That run -- the halo -- is staged
// once per channel slice; each tap reads its A fragments from it at the
// tap's shift, and a per-(pixel, tap) mask turns the fragments of taps that
// fall outside the image (the zero padding, and the neighbouring rows or
// images the run wraps into) into zeros.  B (the weights) is still staged
// per tap.  For a 3x3 layer with 64 output channels the staged bytes per
// tile drop from 9 x (256 + 64) rows to (256 + 2W + 2) + 9 x 64 rows.
//
// Loop: channel slices outer, taps inner.  B tiles are double-buffered (the
// next tap's tile loads while the current one is multiplied); the halo has
// one buffer, loaded at each slice boundary, which keeps a workgroup's LDS
// small enough for two to share a CU and cover each other's waits.
//
// Measured on MI355X (ResNet-50, batch 256): against the 64-channel-slice
// tiles this wins on the 7x7 stage (each input pixel is otherwise staged
// once per tap and per 64-column tile) and ties or loses on the wider
// images, where the per-tap B staging and the slice-boundary wait dominate.
// A double-buffered halo and a persistent one-workgroup-per-CU form were
// slower still: with one wave per SIMD the LDS and barrier latencies of
// short (16-MFMA) steps are exposed.
#include "igemm_store.hpp"

namespace nnconv {

namespace halo {

constexpr int BKC = 8;    // 16-byte chunks per 64-channel row
constexpr int RPI = 8;    // rows per 64-lane load (64 lanes x 16 bytes)

// LDS row swizzle (rows of 8 chunks): logical chunk c of row r at physical
// chunk c ^ ((r >> 1) & 7).  Any 16 consecutive rows read at one logical
// chunk occupy 16 distinct 16-byte bank groups (row parity picks the half of
// the 64 banks, (r >> 1) & 7 the chunk), whatever row they start at -- the
// taps read the halo at arbitrary row offsets.
__device__ __forceinline__ int slot(int r, int c) { return r * BKC + (c ^ ((r >> 1) & 7)); }

}  // namespace halo

// TPS: taps per step (B tiles staged together between two barriers).
template <class T, int BM, int BN, int WM, int WN, int HRMAX, int TPS, int OCC>
__global__ __launch_bounds__(WM * WN * 64, OCC)
void igemm_halo_kernel(const TNParams P) {
    using namespace halo;
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int H_LD = HRMAX / (RPI * NW);   // halo loads per thread per slice
    constexpr int B_LD = BN / (RPI * NW);      // B loads per thread per tap
    constexpr int H_SLOTS = HRMAX * BKC, B_SLOTS = BN * BKC;
    static_assert(FM >= 1 && FN >= 1 && H_LD >= 1 && B_LD >= 1 &&
                      HRMAX % (RPI * NW) == 0 && BN % (RPI * NW) == 0,
                  "tile shape");
    constexpr int MAIN_SLOTS = H_SLOTS + 2 * TPS * B_SLOTS;
    constexpr int LDS_SLOTS = MAIN_SLOTS > BM * BN / 8 ? MAIN_SLOTS : BM * BN / 8;
    __shared__ u32x4 lds[LDS_SLOTS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int l32 = lane & 31, khalf = lane >> 5;

    const TNPhase &F = P.ph[0];
    const int local = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int tm = local / P.tiles_n;
    const int tn = local - tm * P.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;
    const int ntaps = F.tap_count;

    // Tap t reads A pixel (i + eh, j + ew) for output pixel (i, j): the
    // raster shift eh * a_w + ew.  lo / hi: the smallest / largest shift.
    int lo = 0x7FFFFFFF, hi = -0x7FFFFFFF;
    for (int t = 0; t < ntaps; ++t) {
        const int s = (P.ai_add + P.taps.dh[t]) * P.a_w + P.aj_add + P.taps.dw[t];
        lo = s < lo ? s : lo;
        hi = s > hi ? s : hi;
    }
    const int hrows = BM + hi - lo;  // staged halo rows (the host checks <= HRMAX)

    // per-tap values, tap t held by lane t (read back with v_readlane):
    // halo row offset and B element offset
    const int tl = lane < ntaps ? lane : 0;
    const int tap_eh = P.ai_add + P.taps.dh[tl];
    const int tap_ew = P.aj_add + P.taps.dw[tl];
    const int tap_hoff = tap_eh * P.a_w + tap_ew - lo;
    const uint32_t tap_boff = (uint32_t)P.taps.boff[tl] * 2u;

    // Which taps land inside the image, for the pixel of each of this lane's
    // fragment rows (bit t of amask[i]); pixels past the end get none.
    uint32_t amask[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        amask[i] = 0;
        const int m = m0 + wm * WTM + i * 32 + l32;
        if (m < F.M) {
            const int q1 = (int)fdiv((uint32_t)m, F.div_mj);
            const int jj = m - q1 * F.mj;
            const int ii = q1 - (int)fdiv((uint32_t)q1, F.div_mi) * F.mi;
            for (int t = 0; t < ntaps; ++t) {
                const int h = ii + P.ai_add + P.taps.dh[t];
                const int w = jj + P.aj_add + P.taps.dw[t];
                if ((unsigned)h < (unsigned)P.a_h && (unsigned)w < (unsigned)P.a_w)
                    amask[i] |= 1u << t;
            }
        }
    }

    // Staging roles.  Halo load j of this wave fills halo rows
    // (j*NW + wave)*8 + lane/8, B load j rows (wave*B_LD + j)*8 + lane/8;
    // lane % 8 is the physical chunk, holding logical chunk (lane%8) ^ swz.
    const int lrow = lane >> 3;
    const int pch = lane & 7;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)&lds[0];
    uint32_t h_voff[H_LD];
#pragma unroll
    for (int j = 0; j < H_LD; ++j) {
        const int r = (j * NW + wave) * RPI + lrow;
        const int p = m0 + lo + r;  // A pixel (raster index) of halo row r
        h_voff[j] = (r < hrows && p >= 0 && p < F.M)
                        ? (uint32_t)p * (uint32_t)P.a_c * 2u +
                              (uint32_t)(pch ^ ((r >> 1) & 7)) * 16u
                        : OOB_OFFSET;
    }
    uint32_t b_voff[B_LD];
#pragma unroll
    for (int j = 0; j < B_LD; ++j) {
        const int r = (wave * B_LD + j) * RPI + lrow;
        const int col = n0 + r;
        b_voff[j] = col < P.ncols ? (uint32_t)col * (uint32_t)P.b_ld * 2u +
                                        (uint32_t)(pch ^ ((r >> 1) & 7)) * 16u
                                  : OOB_OFFSET;
    }

    auto halo_load = [&](int j, const i32x4 &d, uint32_t base) {
        dma16(base + (uint32_t)((j * NW + wave) * 64) * 16u, h_voff[j], d);
    };
    // the halo of channel slice c
    auto issue_halo = [&](int c) {
        const i32x4 d = desc_at(P.a, P.a_bytes, (uint32_t)c * 128u);
#pragma unroll
        for (int j = 0; j < H_LD; ++j) halo_load(j, d, lds0);
    };
    // the B tiles of step u (taps u*TPS .. u*TPS + TPS - 1 that exist) of
    // channel slice c into B buffer bb
    auto issue_b = [&](int u, int c, int bb) {
#pragma unroll
        for (int e = 0; e < TPS; ++e) {
            const int t = u * TPS + e;
            if (t < ntaps) {
                const uint32_t bshift = (uint32_t)__builtin_amdgcn_readlane((int)tap_boff, t);
                const i32x4 d = desc_at(P.b, P.b_bytes, bshift + (uint32_t)c * 128u);
                const uint32_t base = lds0 + (uint32_t)(H_SLOTS + (bb * TPS + e) * B_SLOTS) * 16u;
#pragma unroll
                for (int j = 0; j < B_LD; ++j)
                    dma16(base + (uint32_t)((wave * B_LD + j) * 64) * 16u, b_voff[j], d);
            }
        }
    };

    f32x16 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x16{};

    // One tap of one channel slice: A fragments from the halo at the tap's
    // row offset, zeroed for pixels where the tap falls outside the image;
    // B fragments from the tap's tile.  With few fragments per k-step all
    // four k-steps' reads are issued first (one wait instead of one per
    // k-step); larger wave tiles would run out of registers doing so.
    auto compute = [&](int bb, int e, int t) {
        constexpr int KS = BKC / 2;
        constexpr bool BATCH = FM + FN <= 4;
        const u32x4 *hs = &lds[0];
        const u32x4 *bs = &lds[H_SLOTS + (bb * TPS + e) * B_SLOTS];
        const int hoff = __builtin_amdgcn_readlane(tap_hoff, t);
        u32x4 fa[BATCH ? KS : 1][FM], fb[BATCH ? KS : 1][FN];
        auto read = [&](int ks, int e) {
            const int kc = 2 * ks + khalf;
#pragma unroll
            for (int i = 0; i < FM; ++i) fa[e][i] = hs[slot(wm * WTM + i * 32 + l32 + hoff, kc)];
#pragma unroll
            for (int j = 0; j < FN; ++j) fb[e][j] = bs[slot(wn * WTN + j * 32 + l32, kc)];
        };
        auto mma = [&](int e) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
                if (!((amask[i] >> t) & 1u)) fa[e][i] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[j][i] = mfma32<T>(fb[e][j], fa[e][i], acc[j][i]);
        };
        if constexpr (BATCH) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) read(ks, ks);
            // keep the reads ahead of the matrix-core instructions (the
            // scheduler would otherwise pair each k-step's reads with a wait)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) mma(ks);
        } else {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                read(ks, 0);
                mma(0);
            }
        }
    };

    const int nslices = P.cr / 64;
    const int nsteps = (ntaps + TPS - 1) / TPS;  // steps per slice
    const int k_iters = nsteps * nslices;
    if (k_iters > 0) {
        issue_halo(0);
        issue_b(0, 0, 0);
        int u = 0, c = 0;
        for (int kt = 0; kt < k_iters; ++kt) {
            if (u == 0 && c > 0) {
                barrier_lds();  // every wave is done with slice c - 1
                issue_halo(c);
            }
            wait_vmcnt<0>();
            barrier_lds();  // halo and B tiles of this step landed; step kt-1 done
            int u1 = u + 1, c1 = c;
            if (u1 == nsteps) {
                u1 = 0;
                ++c1;
            }
            if (kt + 1 < k_iters) issue_b(u1, c1, (kt + 1) & 1);
#pragma unroll
            for (int e = 0; e < TPS; ++e)
                if (u * TPS + e < ntaps) compute(kt & 1, e, u * TPS + e);
            u = u1;
            c = c1;
        }
    }

    store_tile<T, BM, BN, WM, WN, FM, FN>(acc, &lds[0], P, F, m0, n0, 0);
}

namespace {

template <class T, int BM, int BN, int WM, int WN, int TPS, int OCC>
hipError_t launch_halo_cfg(TNParams &p, hipStream_t st) {
    if (!halo_supported(p)) return hipErrorInvalidValue;
    p.tiles_n = (p.ncols + BN - 1) / BN;
    const int64_t tiles_m = (p.ph[0].M + BM - 1) / BM;
    p.ph[0].tiles_m = (int32_t)tiles_m;
    p.ph[0].block_start = 0;
    const int64_t nb = tiles_m * p.tiles_n;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    // halo buffer: BM + HALO_SPAN rows
    hipLaunchKernelGGL((igemm_halo_kernel<T, BM, BN, WM, WN, BM + HALO_SPAN, TPS, OCC>), dim3((uint32_t)nb),
                       dim3(WM * WN * 64), 0, st, p);
    return hipGetLastError();
}

// Configurations (LDS per workgroup):
//   256x64:  4 waves of 64x64 (64 KB; two workgroups per CU)
//   256x128: 4 waves of 128x64 (80 KB; two per CU)
template <class T>
hipError_t launch_halo_t(HaloConfig cfg, TNParams &p, hipStream_t st) {
    switch (cfg) {
        case HALO_256x128: return launch_halo_cfg<T, 256, 128, 2, 2, 1, 2>(p, st);
        case HALO_256x64_2T: return launch_halo_cfg<T, 256, 64, 4, 1, 2, 2>(p, st);
        case HALO_256x64:
        default: return launch_halo_cfg<T, 256, 64, 4, 1, 1, 2>(p, st);
    }
}

}  // namespace

int halo_tap_span(const TNParams &p) {
    const TNPhase &F = p.ph[0];
    int64_t lo = INT64_MAX, hi = INT64_MIN;
    for (int t = 0; t < F.tap_count; ++t) {
        const int64_t s = (int64_t)(p.ai_add + p.taps.dh[t]) * p.a_w + p.aj_add + p.taps.dw[t];
        lo = s < lo ? s : lo;
        hi = s > hi ? s : hi;
    }
    const int64_t span = hi - lo;
    return span > 0x7FFFFFFF ? 0x7FFFFFFF : (int)span;
}

bool halo_supported(const TNParams &p, bool grouped) {
    if (p.nphase != 1 || p.groups < 1 || p.cr <= 0 || p.cr % 64 != 0) return false;
    if (p.groups == 1 ? p.a_c != p.cr
                      : !grouped || (int64_t)p.a_c != (int64_t)p.groups * p.cr ||
                            p.a_cg_ofs != p.cr || (int64_t)p.o_c != (int64_t)p.groups * p.ncols ||
                            p.o_cg_ofs != p.ncols)
        return false;
    const TNPhase &F = p.ph[0];
    if (p.ai_mul != 1 || p.aj_mul != 1 || p.oi_mul != 1 || p.oj_mul != 1 || F.oi_add != 0 ||
        F.oj_add != 0 || F.mi != p.a_h || F.mj != p.a_w || F.tap_start != 0 ||
        F.tap_count < 1 || F.tap_count > 32)
        return false;
    return halo_tap_span(p) <= HALO_SPAN;
}

int halo_cfg_span(HaloConfig cfg) {
    return cfg == HALO_R256x128 ? 64 : cfg == HALO_R224x256 ? 32 : HALO_SPAN;
}

bool halo_cfg_supported(const TNParams &p, HaloConfig cfg) {
    // the single-slice tile takes groups of 64 reduction channels into 64
    // output columns; every other configuration one group
    if (cfg == HALO_R256x64S)
        return hring_supported(p, halo_cfg_span(cfg), true) && p.cr == 64 &&
               (p.groups == 1 || p.ncols == 64);
    if (hring_config(cfg)) return hring_supported(p, halo_cfg_span(cfg));
    return halo_supported(p);
}

hipError_t launch_igemm_halo(int dtype, HaloConfig cfg, TNParams &p, void *pack, bool diag32,
                             hipStream_t st) {
    if (hring_config(cfg)) return launch_igemm_hring(dtype, cfg, p, pack, diag32, st);
    if (dtype == Half::id) return launch_halo_t<Half>(cfg, p, st);
    return launch_halo_t<BFloat>(cfg, p, st);
}

}  // namespace nnconv
