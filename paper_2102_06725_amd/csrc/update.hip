// update.hip -- the training-step pieces after the backward passes, kept on
// the device so a step needs no host synchronisation:
//   - dynamic loss scaling (Sec. 3.3, Listing 6) as a one-thread state
//     machine over a device-resident state and the overflow flag that the
//     backward-weight reduction sets;
//   - the fp32 master-weight update (momentum SGD with L2 weight decay),
//     which divides the loss-scaled gradient by the current scale, skips
//     itself when the flag reports an inf or NaN, and refreshes the 16-bit
//     working copy of the weights.
#include "launch.hpp"

static_assert(sizeof(nnconv_loss_scaler) == 24, "scaler state is part of the C ABI");

namespace nnconv {

__global__ __launch_bounds__(64) void loss_scaler_init_kernel(nnconv_loss_scaler *s, float scale,
                                                              float factor, int32_t interval) {
    if (threadIdx.x != 0) return;
    s->scale = scale;
    s->factor = factor;
    s->interval = interval;
    s->counter = 0;
    s->skipped = 0;
    s->reserved = 0;
}

// One step: overflow -> scale /= factor, counter = 0 (update skipped);
// otherwise grow the scale once the counter has passed the interval, then
// count the step.  The flag is cleared for the next step.
__global__ __launch_bounds__(64) void loss_scaler_update_kernel(nnconv_loss_scaler *s,
                                                                int32_t *flag) {
    if (threadIdx.x != 0) return;
    if (*flag != 0) {
        s->scale = s->scale / s->factor;
        s->counter = 0;
        s->skipped = s->skipped + 1;
    } else {
        if (s->counter > s->interval) {
            s->scale = s->scale * s->factor;
            s->counter = 0;
        }
        s->counter = s->counter + 1;
    }
    *flag = 0;
}

// g = grad / scale + wd * w;  v = mu * v + g;  w -= lr * v
__device__ __forceinline__ void sgd_one(float &w, float &v, float g, float inv_scale, float lr,
                                        float mu, float wd) {
    const float gg = g * inv_scale + wd * w;
    v = mu * v + gg;
    w = w - lr * v;
    // The 16-bit copy must be the rounding of the stored fp32 master; keep
    // the compiler from fusing the last multiply-add into the conversion
    // (a mixed-precision fma that rounds once, straight to 16 bits).
    asm volatile("" : "+v"(w));
}

// OUT: 0 writes an f16 copy of the new master, 1 a bf16 copy, -1 none.
// VEC: four elements per thread with 16-byte loads and stores.
template <int OUT, bool VEC>
__global__ __launch_bounds__(256) void sgd_update_kernel(int64_t count, float *__restrict__ master,
                                                         float *__restrict__ mom,
                                                         uint16_t *__restrict__ w16,
                                                         const float *__restrict__ grad,
                                                         const nnconv_loss_scaler *state,
                                                         const int32_t *flag, float lr, float mu,
                                                         float wd) {
    if (flag && *flag != 0) return;  // inf/NaN in this step's gradients: skip
    const float inv_scale = state ? 1.0f / state->scale : 1.0f;
    using T = typename std::conditional<OUT == 1, BFloat, Half>::type;
    if constexpr (VEC) {
        const int64_t i4 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
        if (i4 >= count) return;
        f32x4 w = *(const f32x4 *)(master + i4);
        f32x4 v = *(const f32x4 *)(mom + i4);
        const f32x4 g = *(const f32x4 *)(grad + i4);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float wu = w[u], vu = v[u];
            sgd_one(wu, vu, g[u], inv_scale, lr, mu, wd);
            w[u] = wu;
            v[u] = vu;
        }
        *(f32x4 *)(master + i4) = w;
        *(f32x4 *)(mom + i4) = v;
        if constexpr (OUT >= 0) {
            const uint32_t b0 = to16<T>(w[0]) & 0xFFFFu, b1 = to16<T>(w[1]) & 0xFFFFu;
            const uint32_t b2 = to16<T>(w[2]) & 0xFFFFu, b3 = to16<T>(w[3]) & 0xFFFFu;
            *(u32x2 *)(w16 + i4) = u32x2{b0 | (b1 << 16), b2 | (b3 << 16)};
        }
    } else {
        const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
        if (i >= count) return;
        float w = master[i], v = mom[i];
        sgd_one(w, v, grad[i], inv_scale, lr, mu, wd);
        master[i] = w;
        mom[i] = v;
        if constexpr (OUT >= 0) w16[i] = (uint16_t)to16<T>(w);
    }
}

hipError_t launch_loss_scaler_init(nnconv_loss_scaler *s, float scale, float factor,
                                   int32_t interval, hipStream_t st) {
    hipLaunchKernelGGL(loss_scaler_init_kernel, dim3(1), dim3(64), 0, st, s, scale, factor,
                       interval);
    return hipGetLastError();
}

hipError_t launch_loss_scaler_update(nnconv_loss_scaler *s, int32_t *flag, hipStream_t st) {
    hipLaunchKernelGGL(loss_scaler_update_kernel, dim3(1), dim3(64), 0, st, s, flag);
    return hipGetLastError();
}

template <int OUT>
static void launch_sgd_out(int64_t count, float *master, float *mom, uint16_t *w16,
                           const float *grad, const nnconv_loss_scaler *state, const int32_t *flag,
                           float lr, float mu, float wd, hipStream_t st) {
    const bool vec = count % 4 == 0 && (uintptr_t)master % 16 == 0 && (uintptr_t)mom % 16 == 0 &&
                     (uintptr_t)grad % 16 == 0 && (OUT < 0 || (uintptr_t)w16 % 8 == 0);
    if (vec) {
        const int64_t nb = (count / 4 + 255) / 256;
        hipLaunchKernelGGL((sgd_update_kernel<OUT, true>), dim3((uint32_t)nb), dim3(256), 0, st,
                           count, master, mom, w16, grad, state, flag, lr, mu, wd);
    } else {
        const int64_t nb = (count + 255) / 256;
        hipLaunchKernelGGL((sgd_update_kernel<OUT, false>), dim3((uint32_t)nb), dim3(256), 0, st,
                           count, master, mom, w16, grad, state, flag, lr, mu, wd);
    }
}

hipError_t launch_sgd_update(int64_t count, float *master, float *mom, void *w16, int w16_dtype,
                             const float *grad, const nnconv_loss_scaler *state, const int32_t *flag,
                             float lr, float mu, float wd, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    if ((count + 255) / 256 > 0x7FFFFFFF) return hipErrorInvalidValue;
    uint16_t *o = (uint16_t *)w16;
    if (!o)
        launch_sgd_out<-1>(count, master, mom, o, grad, state, flag, lr, mu, wd, st);
    else if (w16_dtype == BFloat::id)
        launch_sgd_out<1>(count, master, mom, o, grad, state, flag, lr, mu, wd, st);
    else
        launch_sgd_out<0>(count, master, mom, o, grad, state, flag, lr, mu, wd, st);
    return hipGetLastError();
}

}  // namespace nnconv
