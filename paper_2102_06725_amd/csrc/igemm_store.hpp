// igemm_store.hpp -- the output stage shared by the matrix-core implicit-GEMM
// kernels (igemm_c64.hip, igemm_halo.hip).
#pragma once

#include "launch.hpp"

namespace nnconv {

// Writes a BM x BN accumulator tile held by WM x WN waves (wave tiles of
// FM x FN 32x32 MFMA blocks) to the channel-last output, scaled by alpha and
// rounded to the 16-bit type.  The tile goes through LDS as [BM pixel rows]
// [BN channels] (16-byte chunks swizzled by row) and is read back one 16-byte
// chunk per lane, consecutive lanes along a row, so every global store
// writes whole cache lines of one output pixel.  Lane (MFMA layout) holds
// pixel l32 of each 32-pixel block and, of each 32-channel block, channels
// 8*e + 4*khalf + {0..3} (e = 0..3).  `lds` must hold BM * BN / 8 chunks and
// no other wave may still read it (the first barrier waits for that).
template <class T, int BM, int BN, int WM, int WN, int FM, int FN>
__device__ __forceinline__ void store_tile(const f32x16 (&acc)[FN][FM], u32x4 *lds,
                                           const TNParams &P, const TNPhase &F, int m0, int n0,
                                           int g) {
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int CPR = BN / 8;                    // 16-byte chunks per tile row
    constexpr int CSW = CPR < 16 ? CPR - 1 : 15;   // chunk swizzle mask
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int l32 = lane & 31, khalf = lane >> 5;
    barrier_lds();  // every wave is done reading the last k-slice
    {
        char *cl = (char *)lds;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
#pragma unroll
            for (int j = 0; j < FN; ++j) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int c = (wn * WTN + j * 32) / 8 + e;
                    u32x2 pk;
                    pk[0] = to16<T>(acc[j][i][4 * e + 0] * P.alpha) |
                            (to16<T>(acc[j][i][4 * e + 1] * P.alpha) << 16);
                    pk[1] = to16<T>(acc[j][i][4 * e + 2] * P.alpha) |
                            (to16<T>(acc[j][i][4 * e + 3] * P.alpha) << 16);
                    *(u32x2 *)(cl + (r * CPR + (c ^ (r & CSW))) * 16 + khalf * 8) = pk;
                }
            }
        }
    }
    barrier_lds();
    uint16_t *out = (uint16_t *)P.out;
    constexpr int ROWS_PER_PASS = NW * 64 / CPR;
#pragma unroll 4
    for (int r = tid / CPR; r < BM; r += ROWS_PER_PASS) {
        const int c = tid % CPR;
        const int m = m0 + r;
        const int ch = n0 + c * 8;
        if (m >= F.M || ch >= P.ncols) continue;
        const int q1 = (int)fdiv((uint32_t)m, F.div_mj);
        const int jj = m - q1 * F.mj;
        const int n = (int)fdiv((uint32_t)q1, F.div_mi);
        const int ii = q1 - n * F.mi;
        const int oh = ii * P.oi_mul + F.oi_add;
        const int ow = jj * P.oj_mul + F.oj_add;
        const int64_t obase =
            ((int64_t)(n * P.o_h + oh) * P.o_w + ow) * P.o_c + (int64_t)g * P.o_cg_ofs;
        // streaming store: the output is not read again by this pass, so it
        // should not displace operand lines in L2
        __builtin_nontemporal_store(lds[r * CPR + (c ^ (r & CSW))], (u32x4 *)(out + obase + ch));
    }
}

}  // namespace nnconv
