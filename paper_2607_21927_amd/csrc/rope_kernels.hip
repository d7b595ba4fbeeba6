// RoPE with long-context scaling, in place on [heads, N, D].
//
// One thread owns one (token, pair i) and walks every head, so the float64
// angle and sincos (needed: a float32 angle at position 65,535 is off by up to
// ~4e-3 rad) are paid once per (token, pair) and amortised over the heads.
// Consecutive threads take consecutive pairs of one token: each wave touches
// contiguous half-rows, x[i] and x[i + D/2].  Elementwise and HBM-bound.
#include "ris_device.h"
#include "ris_internal.h"

namespace ris {
namespace {

constexpr int kThreads = 256;

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_rope(void* xv, int heads, int64_t N, int D,
                                                   int64_t pos0, RopeTable tab) {
    const int half = D >> 1;
    const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t t = gid / half;
    const int i = (int)(gid - t * half);
    if (t >= N) return;
    const double ang = (double)(pos0 + t) * tab.inv_freq[i];
    double sd, cd;
    sincos(ang, &sd, &cd);
    const float c = (float)(cd * tab.mscale);
    const float s = (float)(sd * tab.mscale);
    for (int h = 0; h < heads; ++h) {
        const int64_t row = ((int64_t)h * N + t) * D;
        if constexpr (BF16) {
            uint16_t* x = static_cast<uint16_t*>(xv) + row;
            const float x0 = bf16_to_f32(x[i]), x1 = bf16_to_f32(x[i + half]);
            x[i] = f32_to_bf16(x0 * c - x1 * s);
            x[i + half] = f32_to_bf16(x1 * c + x0 * s);
        } else {
            float* x = static_cast<float*>(xv) + row;
            const float x0 = x[i], x1 = x[i + half];
            x[i] = x0 * c - x1 * s;
            x[i + half] = x1 * c + x0 * s;
        }
    }
}

}  // namespace

hipError_t launch_rope(void* x, int dtype_bf16, int heads, int64_t N, int D, int64_t pos0,
                       const RopeTable& tab, hipStream_t st) {
    const int64_t work = N * (D / 2);
    const unsigned blocks = (unsigned)((work + kThreads - 1) / kThreads);
    if (dtype_bf16)
        hipLaunchKernelGGL(k_rope<true>, dim3(blocks), dim3(kThreads), 0, st, x, heads, N, D, pos0, tab);
    else
        hipLaunchKernelGGL(k_rope<false>, dim3(blocks), dim3(kThreads), 0, st, x, heads, N, D, pos0, tab);
    return hipGetLastError();
}

}  // namespace ris
