// igemm_hring.hip -- halo-staged implicit-GEMM convolution whose weight
// fragments come straight from L2 into registers, for the stride-1 "same"
// geometries (3x3, padding 1: the forward pass and the single-phase
// backward-data pass of the ResNet-50 bottleneck 3x3 layers).
//
// As in igemm_halo.hip, a tile is BM consecutive output pixels in raster
// order, and a 64-channel slice of the input is staged in LDS once per tile
// as the halo run all taps read from (tap t at raster shift dh*W + dw).  A
// step is one tap of one channel slice.  What differs:
//   - the B operand (weights; for backward-data the re-laid [R][S][Cg][Kg]
//     copy) never goes through LDS.  A pre-pass (pack_hring_b_kernel)
//     writes it in fragment order: for each (channel slice, tap, 32-column
//     block, k-step) the 64 lanes' 16-byte MFMA fragments lie in one
//     contiguous kilobyte, so a wave loads a fragment with one buffer load
//     that reads whole cache lines (a lane-per-column load would touch 32
//     lines for 32 bytes each, and the per-CU load path would bound the
//     kernel).  Each wave loads its fragments D steps ahead into a ring of
//     registers; the packed weights are small and stay in L2.  The LDS then
//     holds only the halo (double-buffered), and the per-step barrier of a
//     shared B tile disappears: waves meet once per channel slice;
//   - the next slice's halo is loaded into registers during the first step
//     of a slice and written to the other LDS buffer in the second, so
//     every load is an ordinary one the compiler counts: its waits cover
//     exactly the loads a use depends on;
//   - fragment addresses: a k-step flips bits 5-6 of a fragment's LDS
//     address (the swizzle is an XOR on the 16-byte chunk), so the row,
//     swizzle and tap mask of each A fragment are worked out once per step;
//     taps outside the image read a zero row of LDS.
// With one wave per SIMD, each wave reads the next k-step's A fragments
// before it issues the current k-step's matrix-core instructions.
#include "igemm_store.hpp"

namespace nnconv {

namespace hring {

constexpr int BKC = 8;  // 16-byte chunks per 64-channel row
constexpr int RPI = 8;  // rows per 64-lane load (64 lanes x 16 bytes)
constexpr int KS = 4;   // 16-deep k-steps per 64-channel slice

}  // namespace hring

// BM x BN output tile, WM x WN waves, HR halo rows per LDS buffer, NT filter
// taps, D steps of weight fragments in flight (D divides NT: a channel slice
// is unrolled over its taps, so every ring index and every load is fixed at
// compile time and the compiler's wait counts are exact).  NB halo buffers:
// 2 (double-buffered slices, one workgroup per CU), or 1 for a reduction of
// a single 64-channel slice (the host checks cr == 64), where a tile stages
// its halo once and OCC workgroups share a CU, one's staging and output
// stage covered by the others' matrix-core work.  The single-slice tile also
// runs P.groups > 1 groups of 64 channels (super-groups of a grouped
// convolution), each its own GEMM; DIAG: their 64x64 weight blocks are
// block-diagonal in 32x32 blocks, so a 32-column block of a wave meets only
// the matching 32 channels (two of the four k-steps) and the others are
// neither loaded nor multiplied.
template <class T, int BM, int BN, int WM, int WN, int HR, int NT, int D, int NB, int OCC,
          bool DIAG = false>
__global__ __launch_bounds__(WM * WN * 64, OCC)
void igemm_hring_kernel(const TNParams P) {
    using namespace hring;
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int H_LD = HR / (RPI * NW);  // halo loads per lane per slice
    constexpr int H_SLOTS = HR * BKC;
    constexpr int ZERO = NB * H_SLOTS;     // one row of zeros
    static_assert(NB == 1 || NB == 2, "halo buffers");
    static_assert(!DIAG || (NB == 1 && BN == 64), "block-diagonal: single-slice 64-column tile");
    // the output stage reuses the LDS for the BM x BN tile, which can be
    // larger than the two halo buffers
    constexpr int LDS_SLOTS = ZERO + BKC > BM * BN / 8 ? ZERO + BKC : BM * BN / 8;
    static_assert(FM >= 1 && FN >= 1 && HR % (RPI * NW) == 0, "tile shape");
    static_assert(NT >= 1 && NT <= 32 && NT % D == 0, "taps");
    static_assert(BM * BN / 8 <= LDS_SLOTS, "C tile must fit in LDS");
    static_assert(LDS_SLOTS * 16 <= 160 * 1024, "LDS");
    __shared__ u32x4 lds[LDS_SLOTS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int l32 = lane & 31, khalf = lane >> 5;

    const TNPhase &F = P.ph[0];
    // group, then column tile outer: the workgroups of one XCD (consecutive
    // local ids) share the column tile's packed weights in that XCD's L2
    const int local = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int per_g = F.tiles_m * P.tiles_n;
    const int g = local / per_g;
    const int rem = local - g * per_g;
    const int tn = rem / F.tiles_m;
    const int tm = rem - tn * F.tiles_m;
    const int m0 = tm * BM, n0 = tn * BN;
    constexpr int ntaps = NT;  // the host checks F.tap_count == NT
    const int nslices = P.cr / 64;
    const int K = ntaps * nslices;  // steps

    // raster shift of tap t: (ai_add + dh[t]) * W + aj_add + dw[t]; lo / hi
    // the smallest / largest (the host checks hi - lo <= HR - BM)
    int lo = 0x7FFFFFFF, hi = -0x7FFFFFFF;
    for (int t = 0; t < ntaps; ++t) {
        const int s = (P.ai_add + P.taps.dh[t]) * P.a_w + P.aj_add + P.taps.dw[t];
        lo = s < lo ? s : lo;
        hi = s > hi ? s : hi;
    }
    const int hrows = BM + hi - lo;

    // per-tap halo row offset, tap t held by lane t
    const int tl = lane < ntaps ? lane : 0;
    const int tap_hoff =
        (P.ai_add + P.taps.dh[tl]) * P.a_w + P.aj_add + P.taps.dw[tl] - lo;

    // bit t: tap t lands inside the image for the pixel of fragment row i
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

    // Halo load j of this lane: halo row (wave * H_LD + j) * 8 + lane / 8,
    // logical chunk lane % 8; it goes to LDS slot row * 8 + (chunk ^ swizzle).
    const int lrow = lane >> 3;
    const int lch = lane & 7;
    uint32_t h_goff[H_LD], h_loff[H_LD];
#pragma unroll
    for (int j = 0; j < H_LD; ++j) {
        const int r = (wave * H_LD + j) * RPI + lrow;
        const int p = m0 + lo + r;  // A pixel (raster index) of halo row r
        h_goff[j] = (r < hrows && p >= 0 && p < F.M)
                        ? ((uint32_t)p * (uint32_t)P.a_c + (uint32_t)(g * P.a_cg_ofs)) * 2u +
                              (uint32_t)lch * 16u
                        : OOB_OFFSET;
        h_loff[j] = (uint32_t)(r * 128 + ((lch ^ ((r >> 1) & 7)) << 4));
    }
    // Packed weights: fragment (group, slice c, tap t, column block cb,
    // k-step ks) is the kilobyte at ((((group * nslices + c) * NT + t) * ncb +
    // cb) * KS + ks) * 1024, lane l's 16 bytes at l * 16.  B fragment j of
    // this wave is column block (n0 + wn * WTN) / 32 + j.
    const int ncb = (P.ncols + 31) / 32;
    const uint32_t b_gshift = (uint32_t)(g * nslices * NT * ncb) * (uint32_t)(KS * 1024);
    // DIAG: whether k-step ks meets column block j of this wave
    auto live_block = [&](int ks, int j) {
        return !DIAG || (ks >> 1) == (((wn * WTN) >> 5) + j) % 2;
    };
    uint32_t b_goff[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j)
        b_goff[j] = (uint32_t)(((n0 + wn * WTN) / 32 + j) * KS * 1024 + lane * 16);

    const char *lbase = (const char *)&lds[0];
    char *lbase_w = (char *)&lds[0];

    // Buffer resource over [p, p + bytes): the words are made wave-uniform
    // explicitly, or the compiler may treat the address as divergent and
    // wrap every load in a loop over lanes.
    auto rsrc = [&](const char *p, uint32_t bytes) {
        const uint64_t a = (uint64_t)p;
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
        const char *q = (const char *)(((uint64_t)hi << 32) | lo);
        return make_rsrc(q, (uint32_t)__builtin_amdgcn_readfirstlane((int)bytes));
    };

    // Kernel arguments the loop needs, kept in scalar registers: the
    // compiler would otherwise reload them from the argument segment inside
    // the loop, and a scalar load shares its wait counter with the LDS reads
    // (waiting for it waits for every read in flight).
    const char *a_ptr = (const char *)P.a, *b_ptr = (const char *)P.b;
    uint32_t a_bytes = P.a_bytes, b_bytes = P.b_bytes;
    asm volatile("" : "+s"(a_ptr), "+s"(b_ptr), "+s"(a_bytes), "+s"(b_bytes));

    // ---- loads
    u32x4 hreg[H_LD];
    // slice c of the halo into registers (past the last slice: zeros)
    auto load_halo = [&](int c) {
        const uint32_t shift = (uint32_t)c * 128u;
        const __amdgpu_buffer_rsrc_t r =
            rsrc(a_ptr + shift, (c < nslices && a_bytes > shift) ? a_bytes - shift : 0u);
#pragma unroll
        for (int j = 0; j < H_LD; ++j) hreg[j] = load16(r, h_goff[j]);
    };
    auto store_halo = [&](int hb) {  // ... and from the registers into buffer hb
#pragma unroll
        for (int j = 0; j < H_LD; ++j)
            *(u32x4 *)(lbase_w + hb * H_SLOTS * 16 + h_loff[j]) = hreg[j];
    };
    u32x4 fbr[D][KS][FN];
    // the weight fragments of step (tap t, slice c) into ring entry e; past
    // the last step (live = false) nothing is read (zeros)
    auto load_b = [&](int t, int c, bool live, u32x4 (&e)[KS][FN]) {
        const uint32_t shift =
            b_gshift + (uint32_t)((c * NT + t) * ncb) * (uint32_t)(KS * 1024);
        const __amdgpu_buffer_rsrc_t r =
            rsrc(b_ptr + shift, (live && b_bytes > shift) ? b_bytes - shift : 0u);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                if (live_block(ks, j)) e[ks][j] = load16(r, b_goff[j] + (uint32_t)ks * 1024u);
    };

    f32x16 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x16{};

    // k-step 0 A fragment addresses of step (tap t, halo buffer hb)
    auto step_addrs = [&](int t, int hb, uint32_t (&aa)[FM]) {
        const int hoff = __builtin_amdgcn_readlane(tap_hoff, t);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int r = wm * WTM + i * 32 + l32 + hoff;
            const uint32_t in_img =
                (uint32_t)(hb * H_SLOTS * 16 + r * 128 + ((khalf ^ ((r >> 1) & 7)) << 4));
            const uint32_t zero_row = (uint32_t)(ZERO * 16 + (khalf << 4));
            // branch-free select (a branch per fragment costs more issue slots)
            const uint32_t sel = 0u - ((amask[i] >> t) & 1u);
            aa[i] = (in_img & sel) | (zero_row & ~sel);
        }
    };
    auto read_a = [&](const uint32_t (&aa)[FM], int ks, u32x4 (&fa)[FM]) {
        const uint32_t kx = (uint32_t)ks << 5;
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[i] = *(const u32x4 *)(lbase + (aa[i] ^ kx));
    };
    auto mma = [&](const u32x4 (&fa)[FM], const u32x4 (&fb)[FN], int ks) {
#pragma unroll
        for (int j = 0; j < FN; ++j)
            if (live_block(ks, j))
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[j][i] = mfma32<T>(fb[j], fa[i], acc[j][i]);
    };

    // ---- prologue: zero row, halo of slice 0, weights of steps 0 .. D-1
    if (tid < BKC) lds[ZERO + tid] = u32x4{0u, 0u, 0u, 0u};
    load_halo(0);
#pragma unroll
    for (int e = 0; e < D; ++e) load_b(e % NT, e / NT, e < K, fbr[e]);
    store_halo(0);
    barrier_lds();

    u32x4 fa[2][FM];
    uint32_t aa[FM];
    step_addrs(0, 0, aa);
    read_a(aa, 0, fa[0]);
    for (int c = 0; c < nslices; ++c) {
        const int hb = NB == 2 ? (c & 1) : 0;
        // the next slice's halo: into registers at the first step, into the
        // other LDS buffer (free since the barrier that opened this slice)
        // at the last, then the barrier that opens the next slice
        if constexpr (NB == 2) load_halo(c + 1);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int k = c * NT + t;
            uint32_t aa1[FM];
            step_addrs(t + 1 < NT ? t + 1 : 0, t + 1 < NT ? hb : (hb ^ (NB - 1)), aa1);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int cur = ks & 1, nxt = cur ^ 1;
                // the next k-step's A fragments (after a slice's last step
                // they are read again after the barrier: the read here is
                // harmless and keeps the code straight-line)
                if (ks + 1 < KS)
                    read_a(aa, ks + 1, fa[nxt]);
                else
                    read_a(aa1, 0, fa[nxt]);
                __builtin_amdgcn_sched_barrier(0);
                mma(fa[cur], fbr[t % D][ks], ks);
                __builtin_amdgcn_sched_barrier(0);
            }
            // ring entry t % D is free: the weights of step k + D
            load_b((t + D) % NT, c + (t + D) / NT, k + D < K, fbr[t % D]);
#pragma unroll
            for (int i = 0; i < FM; ++i) aa[i] = aa1[i];
        }
        if constexpr (NB == 2) {
            store_halo(hb ^ 1);
            // every wave has stored its share of the next slice's halo and
            // is done with this slice's
            barrier_lds();
            read_a(aa, 0, fa[0]);
        }
    }

    store_tile<T, BM, BN, WM, WN, FM, FN>(acc, &lds[0], P, F, m0, n0, g);
}

// Packs the B operand of a single-phase implicit GEMM (group gr, row `col`,
// tap t, reduction channel ch at element gr * b_g_ofs + col * b_ld + boff[t]
// + ch of p.b) into the fragment order igemm_hring_kernel reads: 16 bytes per
// thread, dst[((((gr * nslices + c) * ntaps + t) * ncb + cb) * 4 + ks) * 64 +
// l] = the 8 channels c * 64 + ks * 16 + (l / 32) * 8 .. +7 of column
// cb * 32 + l % 32 (zeros past ncols).
__global__ __launch_bounds__(256)
void pack_hring_b_kernel(const TNParams P, u32x4 *dst, int32_t total) {
    const int e = (int)(blockIdx.x * 256 + threadIdx.x);
    if (e >= total) return;
    const int ntaps = P.ph[0].tap_count;
    const int ncb = (P.ncols + 31) / 32;
    const int nslices = P.cr / 64;
    const int l = e & 63;
    int f = e >> 6;
    const int ks = f & 3;
    f >>= 2;
    const int cb = f % ncb;
    f /= ncb;
    const int t = f % ntaps;
    f /= ntaps;
    const int c = f % nslices;
    const int gr = f / nslices;
    const int col = cb * 32 + (l & 31);
    const int ch = c * 64 + ks * 16 + (l >> 5) * 8;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (col < P.ncols) {
        const __amdgpu_buffer_rsrc_t r = make_rsrc(P.b, P.b_bytes);
        v = load16(r, (uint32_t)(gr * P.b_g_ofs + col * P.b_ld + P.taps.boff[t] + ch) * 2u);
    }
    dst[e] = v;
}

size_t hring_pack_bytes(int64_t ncols, int64_t cr, int64_t groups) {
    return (size_t)groups * (size_t)HRING_TAPS * (size_t)(cr / 64) *
           (size_t)((ncols + 31) / 32) * 4096u;
}

hipError_t launch_hring_pack(const TNParams &p, void *dst, hipStream_t st) {
    const int64_t total = (int64_t)hring_pack_bytes(p.ncols, p.cr, p.groups) / 16;
    if (total <= 0) return hipSuccess;
    if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(pack_hring_b_kernel, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0, st,
                       p, (u32x4 *)dst, (int32_t)total);
    return hipGetLastError();
}

namespace {

template <class T, int BM, int BN, int WM, int WN, int HR, int NB = 2, int OCC = 1, int D = 3>
hipError_t launch_hring_cfg(TNParams &p, bool diag32, hipStream_t st) {
    // groups (of 64 channels into 64 columns) and block-diagonal weights on
    // the single-slice tile only
    constexpr bool SINGLE = NB == 1 && BN == 64;
    if (!hring_supported(p, HR - BM, SINGLE) || (NB == 1 && p.cr != 64) ||
        (p.groups > 1 && p.ncols != 64))
        return hipErrorInvalidValue;
    p.tiles_n = (p.ncols + BN - 1) / BN;
    const int64_t tiles_m = (p.ph[0].M + BM - 1) / BM;
    p.ph[0].tiles_m = (int32_t)tiles_m;
    p.ph[0].block_start = 0;
    const int64_t nb = tiles_m * p.tiles_n * p.groups;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    // 3x3 filters (the host admits no other tap count)
    if constexpr (SINGLE) {
        if (diag32) {
            // half the weight fragments: three steps of them fit in flight
            hipLaunchKernelGGL((igemm_hring_kernel<T, BM, BN, WM, WN, HR, HRING_TAPS, 3, NB, OCC, true>),
                               dim3((uint32_t)nb), dim3(WM * WN * 64), 0, st, p);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((igemm_hring_kernel<T, BM, BN, WM, WN, HR, HRING_TAPS, D, NB, OCC>), dim3((uint32_t)nb),
                       dim3(WM * WN * 64), 0, st, p);
    return hipGetLastError();
}

// Configurations (4 waves; one workgroup per CU but the single-slice one):
//   256x128: 4 waves of 128x64, halo of 320 rows (taps within 64 raster
//            positions: 3x3 on images up to 31 wide), 80 KB of LDS
//   128x256: 4 waves of 128x64 side by side, halo of 256 rows (within 128:
//            up to 63 wide), 64 KB
//   224x256: 4 waves of 224x64 side by side, halo of 256 rows (within 32:
//            up to 15 wide), 64 KB; 224 tiles for the 14x14 3x3 layers at
//            batch 256: one round on 256 CUs
//   256x64 single slice: 4 waves of 64x64, one halo buffer of 384 rows
//            (within 128), 48 KB, three workgroups per CU (the weight
//            fragments loaded one step ahead, 134 registers: three steps
//            ahead need 207, two workgroups; s2b0b forward / backward-data
//            in the sweep 88 / 93 -> 85 / 90 us): 64-channel
//            reductions with at most 64 output columns per tile
template <class T>
hipError_t launch_hring_t(HaloConfig cfg, TNParams &p, bool diag32, hipStream_t st) {
    switch (cfg) {
        case HALO_R256x128: return launch_hring_cfg<T, 256, 128, 2, 2, 320>(p, false, st);
        case HALO_R224x256: return launch_hring_cfg<T, 224, 256, 1, 4, 256>(p, false, st);
        case HALO_R256x64S: return launch_hring_cfg<T, 256, 64, 4, 1, 384, 1, 3, 1>(p, diag32, st);
        case HALO_R128x256:
        default: return launch_hring_cfg<T, 128, 256, 1, 4, 256>(p, false, st);
    }
}

}  // namespace

bool hring_supported(const TNParams &p, int span, bool grouped) {
    return halo_supported(p, grouped) && p.ph[0].tap_count == HRING_TAPS &&
           halo_tap_span(p) <= span;
}

hipError_t launch_igemm_hring(int dtype, HaloConfig cfg, TNParams &p, void *pack, bool diag32,
                              hipStream_t st) {
    if (!halo_cfg_supported(p, cfg) || !pack) return hipErrorInvalidValue;
    const size_t pb = hring_pack_bytes(p.ncols, p.cr, p.groups);
    if (pb > 0xFFFFFFFFu) return hipErrorInvalidValue;
    hipError_t e = launch_hring_pack(p, pack, st);
    if (e != hipSuccess) return e;
    TNParams q = p;
    q.b = pack;
    q.b_bytes = (uint32_t)pb;
    if (dtype == Half::id) return launch_hring_t<Half>(cfg, q, diag32, st);
    return launch_hring_t<BFloat>(cfg, q, diag32, st);
}

}  // namespace nnconv
