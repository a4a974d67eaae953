// wgrad_reduce.hip -- second half of the backward-weight pass: the sum of
// the split-K fp32 partials in a fixed order, the loss-scale step
// (multiply by the inverse loss scale, optional accumulation into the old
// gradient), conversion to the output type and the non-finite check.
#include <type_traits>

#include "launch.hpp"

namespace nnconv {

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

// Grouped convolution run as super-groups of SG channels with block-diagonal
// weights: the partials hold the whole [K][R*S][SG] super-group gradient;
// this keeps only each output channel's own group (m channels starting at
// ((k % SG) / m) * m) and finishes it like the other reductions.  One final
// element (in [K][R][S][m] order) per thread, splits in increasing order.
template <int OUT>
__global__ __launch_bounds__(256) void wgrad_reduce_diag_kernel(
    const float *__restrict__ ws, int32_t splits, int64_t count, int64_t pcount, int32_t rs,
    int32_t m, int32_t sg, void *dw, float inv_scale, int accumulate, int32_t *flag, int kcrs) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= count) return;
    const int64_t per_k = (int64_t)rs * m;
    const int64_t k = e / per_k;
    const int64_t rem = e - k * per_k;
    const int64_t tap = rem / m;
    const int64_t c = rem - tap * m;
    const int64_t pe = k * rs * sg + tap * sg + ((k % sg) / m) * m + c;
    float sum = 0.f;
    for (int sp = 0; sp < splits; ++sp) sum += ws[(int64_t)sp * pcount + pe];
    if (reduce_store<OUT>(sum, e, dw, inv_scale, accumulate, kcrs, m, rs) && flag) *flag = 1;
}

hipError_t launch_wgrad_reduce_diag(const float *ws, int32_t splits, int64_t k, int32_t rs,
                                    int32_t m, int32_t sg, void *dw, int out_dtype,
                                    float inv_scale, int accumulate, int32_t *flag, int kcrs,
                                    hipStream_t st) {
    const int64_t count = k * rs * m, pcount = k * rs * sg;
    if (count <= 0) return hipSuccess;
    const int64_t nb = (count + 255) / 256;
    if (out_dtype == 2)
        hipLaunchKernelGGL((wgrad_reduce_diag_kernel<2>), dim3((uint32_t)nb), dim3(256), 0, st, ws,
                           splits, count, pcount, rs, m, sg, dw, inv_scale, accumulate, flag, kcrs);
    else if (out_dtype == 0)
        hipLaunchKernelGGL((wgrad_reduce_diag_kernel<0>), dim3((uint32_t)nb), dim3(256), 0, st, ws,
                           splits, count, pcount, rs, m, sg, dw, inv_scale, accumulate, flag, kcrs);
    else
        hipLaunchKernelGGL((wgrad_reduce_diag_kernel<1>), dim3((uint32_t)nb), dim3(256), 0, st, ws,
                           splits, count, pcount, rs, m, sg, dw, inv_scale, accumulate, flag, kcrs);
    return hipGetLastError();
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
