// wgrad.hip -- backward-weight pass: split-K implicit GEMM on the gfx950
// matrix cores, then a fixed-order reduction with the loss-scale epilogue.
//
// GEMM view:  dW[k, j] = sum_pix dy[pix, k] * xcol[pix, j],  j = (r, s, c)
// The reduction runs over batch pixels, which is the strided dimension of
// both channel-last operands.  Each thread loads PPT consecutive pixels x 8
// consecutive channels (16-byte, coalesced along channels), transposes the
// block in registers and writes it to LDS as rows of pixels, so the MFMA
// fragment reads are the same 16-byte row reads as in the forward kernel.
// Pixels are split into `splits` ranges; each range writes an fp32 partial
// tile to the workspace.
#include <type_traits>

#include "launch.hpp"

namespace nnconv {

// Write a PPT-pixel x 8-channel register block transposed into LDS rows
// row0..row0+7 (one row per channel) at pixel offset pix0 of a 64-pixel row.
template <int PPT>
__device__ __forceinline__ void store_transposed(uint32_t *lds, int row0, int pix0,
                                                 const u32x4 (&v)[PPT]) {
    static_assert(PPT == 2 || PPT == 4, "2 or 4 pixels per thread");
#pragma unroll
    for (int e8 = 0; e8 < 8; ++e8) {
        uint32_t wds[PPT / 2];
#pragma unroll
        for (int a = 0; a < PPT / 2; ++a) {
            const uint32_t lo = v[2 * a][e8 >> 1];
            const uint32_t hi = v[2 * a + 1][e8 >> 1];
            wds[a] = (e8 & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
        }
        const int r = row0 + e8;
        const int pc = (pix0 >> 3) ^ swz(r);
        const int addr = (r * 8 + pc) * 4 + ((pix0 & 7) >> 1);
        if constexpr (PPT == 4) {
            u32x2 w2;
            w2[0] = wds[0];
            w2[1] = wds[1];
            *(u32x2 *)(lds + addr) = w2;
        } else {
            lds[addr] = wds[0];
        }
    }
}

template <class T, int BMK, int BNJ, int WM, int WN>
__global__ __launch_bounds__(256, 2) void wgrad_splitk_kernel(const WGParams P) {
    constexpr int CH = 8;                   // 16-byte chunks per 64-pixel LDS row
    constexpr int KCH = BMK / 8;            // channel chunks of the dy tile
    constexpr int JCH = BNJ / 8;            // column chunks of the x tile
    constexpr int PPTK = 64 * KCH / 256;    // pixels per thread, dy tile
    constexpr int PPTJ = 64 * JCH / 256;    // pixels per thread, x tile
    constexpr int WTM = BMK / WM, WTN = BNJ / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    static_assert(WM * WN == 4, "4 waves per workgroup");

    __shared__ u32x4 lds[2][(BMK + BNJ) * CH];

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
    const int k0 = tm * BMK, j0 = tn * BNJ;

    const int pix_begin = split * P.pix_per_split;
    const int pix_end = min(P.npq, pix_begin + P.pix_per_split);
    const int k_iters = pix_end > pix_begin ? (pix_end - pix_begin + 63) / 64 : 0;

    const __amdgpu_buffer_rsrc_t rx = make_rsrc(P.x, P.x_bytes);
    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(P.dy, P.dy_bytes);

    // dy staging role: channel chunk kc, pixel group pgk
    const int kc = tid % KCH, pgk = tid / KCH;
    const bool k_ok = k0 + kc * 8 < P.kg;
    const int dy_ch = g * P.kg + k0 + kc * 8;
    // x staging role: column chunk jc (fixed tap and channel), pixel group pgj
    const int jc = tid % JCH, pgj = tid / JCH;
    const int jcol = j0 + jc * 8;
    const bool j_ok = jcol < P.rscg;
    int tap_dh = 0, tap_dw = 0, x_ch = 0;
    if (j_ok) {
        const int tap = (int)fdiv((uint32_t)jcol, P.div_cg);
        const int c0 = jcol - tap * P.cg;
        const int r = (int)fdiv((uint32_t)tap, P.div_s);
        const int ss = tap - r * (int)P.div_s.d;
        tap_dh = r * P.dh - P.ph;
        tap_dw = ss * P.dw - P.pw;
        x_ch = g * P.cg + c0;
    }

    u32x4 sk[PPTK], sj[PPTJ];
    auto gload = [&](int kt) {
        const int base = pix_begin + kt * 64;
#pragma unroll
        for (int e = 0; e < PPTK; ++e) {
            const int pix = base + pgk * PPTK + e;
            const bool ok = k_ok && pix < pix_end;
            const uint32_t off = (uint32_t)(pix * P.k + dy_ch) * 2u;
            sk[e] = load16(rdy, ok ? off : OOB_OFFSET);
        }
#pragma unroll
        for (int e = 0; e < PPTJ; ++e) {
            const int pix = base + pgj * PPTJ + e;
            bool ok = j_ok && pix < pix_end;
            const int pc = ok ? pix : 0;
            const int n = (int)fdiv((uint32_t)pc, P.div_pq);
            const int rm = pc - n * (P.p * P.q);
            const int pp = (int)fdiv((uint32_t)rm, P.div_q);
            const int qq = rm - pp * P.q;
            const int h = pp * P.sh + tap_dh;
            const int w = qq * P.sw + tap_dw;
            ok = ok && (unsigned)h < (unsigned)P.h && (unsigned)w < (unsigned)P.w;
            const int off = (((n * P.h + h) * P.w + w) * P.c + x_ch) * 2;
            sj[e] = load16(rx, ok ? (uint32_t)off : OOB_OFFSET);
        }
    };
    auto lstore = [&](int buf) {
        uint32_t *base = (uint32_t *)&lds[buf][0];
        store_transposed<PPTK>(base, kc * 8, pgk * PPTK, sk);
        store_transposed<PPTJ>(base + BMK * CH * 4, jc * 8, pgj * PPTJ, sj);
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};

    if (k_iters > 0) {
        gload(0);
        lstore(0);
    }
    __syncthreads();

    const int l32 = lane & 31;
    const int khalf = lane >> 5;
    for (int kt = 0; kt < k_iters; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < k_iters;
        if (more) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int kq = 2 * ks + khalf;
            u32x4 fa[FM], fb[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int r = wm * WTM + i * 32 + l32;
                fa[i] = lds[buf][r * CH + (kq ^ swz(r))];
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int r = wn * WTN + j * 32 + l32;
                fb[j] = lds[buf][(BMK + r) * CH + (kq ^ swz(r))];
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<T>(fa[i], fb[j], acc[i][j]);
        }
        if (more) lstore(buf ^ 1);
        __syncthreads();
    }

    // lane holds column l32 of each 32-column block and rows 8*e + 4*khalf + {0..3}
    const int K = P.kg * P.groups;
    float *ws = P.ws + (int64_t)split * K * P.rscg;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int col = j0 + wn * WTN + j * 32 + l32;
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

template <class T, int BMK, int BNJ, int WM, int WN>
static hipError_t launch_wg(WGParams &p, hipStream_t st) {
    p.tiles_m = (p.kg + BMK - 1) / BMK;
    p.tiles_n = (p.rscg + BNJ - 1) / BNJ;
    const int64_t nb = (int64_t)p.tiles_m * p.tiles_n * p.splits * p.groups;
    if (nb <= 0) return hipSuccess;
    if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((wgrad_splitk_kernel<T, BMK, BNJ, WM, WN>), dim3((uint32_t)nb), dim3(256),
                       0, st, p);
    return hipGetLastError();
}

template <class T>
static hipError_t launch_wg_t(WGConfig cfg, WGParams &p, hipStream_t st) {
    if (cfg == WG_64x128) return launch_wg<T, 64, 128, 2, 2>(p, st);
    return launch_wg<T, 128, 128, 2, 2>(p, st);
}

hipError_t launch_wgrad_splitk(int dtype, WGConfig cfg, WGParams &p, hipStream_t st) {
    if (dtype == Half::id) return launch_wg_t<Half>(cfg, p, st);
    return launch_wg_t<BFloat>(cfg, p, st);
}

// ---------------------------------------------------------------------------
// reduction over splits + loss-scale epilogue
// ---------------------------------------------------------------------------

template <int OUT>  // 0 = f16, 1 = bf16, 2 = f32
__device__ __forceinline__ bool reduce_store(float sum, int64_t e, void *dw, float inv_scale,
                                             int accumulate, int kcrs, int32_t cg, int32_t rs) {
    int64_t oe = e;
    if (kcrs) {  // [K][R][S][Cg] index -> [K][Cg][R][S] index
        const int64_t rscg = (int64_t)rs * cg;
        const int64_t k = e / rscg;
        const int64_t j = e - k * rscg;
        const int64_t tap = j / cg;
        const int64_t c = j - tap * cg;
        oe = (k * cg + c) * rs + tap;
    }
    float v = sum * inv_scale;
    if constexpr (OUT == 2) {
        float *o = (float *)dw;
        if (accumulate) v = o[oe] + v;
        o[oe] = v;
        return !__builtin_isfinite(v);
    } else {
        using T = typename std::conditional<OUT == 0, Half, BFloat>::type;
        uint16_t *o = (uint16_t *)dw;
        if (accumulate) v = from16<T>(o[oe]) + v;
        const uint32_t bits = to16<T>(v);
        o[oe] = (uint16_t)bits;
        return !__builtin_isfinite(from16<T>(bits));
    }
}

// Final value of four consecutive [K][R][S][Cg] elements stored as one
// vector (channel-last weight layout).
template <int OUT>
__device__ __forceinline__ bool reduce_store4(f32x4 sum, int64_t e, void *dw, float inv_scale,
                                              int accumulate) {
    f32x4 v = sum * inv_scale;
    bool bad = false;
    if constexpr (OUT == 2) {
        f32x4 *o = (f32x4 *)((float *)dw + e);
        if (accumulate) v = *o + v;
        *o = v;
#pragma unroll
        for (int u = 0; u < 4; ++u) bad |= !__builtin_isfinite(v[u]);
    } else {
        using T = typename std::conditional<OUT == 0, Half, BFloat>::type;
        u32x2 *o = (u32x2 *)((uint16_t *)dw + e);
        u32x2 old = accumulate ? *o : u32x2{};
        uint32_t bits[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float x = v[u];
            if (accumulate) x = from16<T>((uint16_t)(old[u >> 1] >> (16 * (u & 1)))) + x;
            bits[u] = to16<T>(x) & 0xFFFFu;
            bad |= !__builtin_isfinite(from16<T>(bits[u]));
        }
        *o = u32x2{bits[0] | (bits[1] << 16), bits[2] | (bits[3] << 16)};
    }
    return bad;
}

// Sums the split partials in a fixed order (results are bitwise
// reproducible for a given shape), then applies the loss-scale step.
//
// VEC (count a multiple of 4): a workgroup's 256 threads are 256/L float4
// columns x L split lanes.  Split lane l adds splits l, l+L, l+2L, ... in
// increasing order; lane 0 then adds the L lane sums in increasing lane
// order.  L grows with the split count when there are few output elements,
// so enough independent loads stay in flight.
template <int OUT, int L>
__global__ __launch_bounds__(256) void wgrad_reduce_vec_kernel(const float *__restrict__ ws,
                                                               int32_t splits, int64_t count,
                                                               void *dw, float inv_scale,
                                                               int accumulate, int32_t *flag,
                                                               int kcrs, int32_t cg, int32_t rs,
                                                               int vec_out) {
    constexpr int COLS = 256 / L;
    const int col = threadIdx.x % COLS, sl = threadIdx.x / COLS;
    const int64_t e4 = ((int64_t)blockIdx.x * COLS + col) * 4;
    f32x4 sum = f32x4{};
    if (e4 < count) {
        const float *src = ws + (int64_t)sl * count + e4;
        const int64_t step = (int64_t)L * count;
        int sp = sl;
        for (; sp + 3 * L < splits; sp += 4 * L, src += 4 * step) {
            const f32x4 a = *(const f32x4 *)src;
            const f32x4 b = *(const f32x4 *)(src + step);
            const f32x4 c = *(const f32x4 *)(src + 2 * step);
            const f32x4 d = *(const f32x4 *)(src + 3 * step);
            sum += a;
            sum += b;
            sum += c;
            sum += d;
        }
        for (; sp < splits; sp += L, src += step) sum += *(const f32x4 *)src;
    }
    if constexpr (L > 1) {
        __shared__ f32x4 part[L][COLS];
        part[sl][col] = sum;
        __syncthreads();
        if (sl != 0) return;
        sum = part[0][col];
#pragma unroll
        for (int l = 1; l < L; ++l) sum += part[l][col];
    }
    if (e4 >= count) return;
    bool bad = false;
    if (!vec_out) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            bad |= reduce_store<OUT>(sum[u], e4 + u, dw, inv_scale, accumulate, kcrs, cg, rs);
    } else {
        bad = reduce_store4<OUT>(sum, e4, dw, inv_scale, accumulate);
    }
    if (bad && flag) *flag = 1;
}

// Scalar fallback (count not a multiple of 4): one element per thread.
template <int OUT>
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float *__restrict__ ws,
                                                           int32_t splits, int64_t count,
                                                           void *dw, float inv_scale,
                                                           int accumulate, int32_t *flag,
                                                           int kcrs, int32_t cg, int32_t rs) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= count) return;
    float sum = 0.f;
    for (int sp = 0; sp < splits; ++sp) sum += ws[(int64_t)sp * count + t];
    if (reduce_store<OUT>(sum, t, dw, inv_scale, accumulate, kcrs, cg, rs) && flag) *flag = 1;
}

template <int OUT, int L>
static void launch_reduce_vec(const float *ws, int32_t splits, int64_t count, void *dw,
                              float inv_scale, int accumulate, int32_t *flag, int kcrs,
                              int32_t cg, int32_t rs, hipStream_t st) {
    constexpr int COLS = 256 / L;
    const int64_t nb = (count / 4 + COLS - 1) / COLS;
    // one vector store per float4 column when dw is aligned for it
    const int vec_out = !kcrs && ((uintptr_t)dw % (OUT == 2 ? 16 : 8)) == 0;
    hipLaunchKernelGGL((wgrad_reduce_vec_kernel<OUT, L>), dim3((uint32_t)nb), dim3(256), 0, st, ws,
                       splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, vec_out);
}

// Split lanes per float4 column: enough threads to cover the chip with
// loads (about 2^19 threads), at most 16 and at most one per split.
int reduce_split_lanes(int32_t splits, int64_t count) {
    int l = 1;
    while (l < 16 && 2 * l <= splits && (count / 4) * l < (1 << 19)) l *= 2;
    return l;
}

template <int OUT>
static void launch_reduce_out(const float *ws, int32_t splits, int64_t count, void *dw,
                              float inv_scale, int accumulate, int32_t *flag, int kcrs, int32_t cg,
                              int32_t rs, hipStream_t st) {
    if (count % 4 == 0) {
        switch (reduce_split_lanes(splits, count)) {
            case 1: launch_reduce_vec<OUT, 1>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st); break;
            case 2: launch_reduce_vec<OUT, 2>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st); break;
            case 4: launch_reduce_vec<OUT, 4>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st); break;
            case 8: launch_reduce_vec<OUT, 8>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st); break;
            default: launch_reduce_vec<OUT, 16>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st); break;
        }
    } else {
        const int64_t nb = (count + 255) / 256;
        hipLaunchKernelGGL((wgrad_reduce_kernel<OUT>), dim3((uint32_t)nb), dim3(256), 0, st, ws,
                           splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs);
    }
}

hipError_t launch_wgrad_reduce(const float *ws, int32_t splits, int64_t count, void *dw,
                               int out_dtype, float inv_scale, int accumulate, int32_t *flag,
                               int kcrs, int32_t cg, int32_t rs, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    if (out_dtype == 2)
        launch_reduce_out<2>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st);
    else if (out_dtype == 0)
        launch_reduce_out<0>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st);
    else
        launch_reduce_out<1>(ws, splits, count, dw, inv_scale, accumulate, flag, kcrs, cg, rs, st);
    return hipGetLastError();
}

}  // namespace nnconv
