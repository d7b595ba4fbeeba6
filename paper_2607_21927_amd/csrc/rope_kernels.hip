// RoPE with long-context scaling: [heads, N, D] rotated into a contiguous
// destination, from a source with any head and token strides (the same
// buffer for an in-place rotation, or e.g. a head's columns of a token-major
// projection output, which fuses the head-major copy with the rotation).
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
__global__ __launch_bounds__(kThreads) void k_rope(const void* src, int64_t hs, int64_t ts, void* dst,
                                                   int heads, int64_t N, int D, int64_t pos0, RopeTable tab) {
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
        const int64_t in = (int64_t)h * hs + t * ts;      // source row (h, t)
        const int64_t row = ((int64_t)h * N + t) * D;     // destination row
        if constexpr (BF16) {
            const uint16_t* x = static_cast<const uint16_t*>(src) + in;
            uint16_t* y = static_cast<uint16_t*>(dst) + row;
            const float x0 = bf16_to_f32(x[i]), x1 = bf16_to_f32(x[i + half]);
            y[i] = f32_to_bf16(x0 * c - x1 * s);
            y[i + half] = f32_to_bf16(x1 * c + x0 * s);
        } else {
            const float* x = static_cast<const float*>(src) + in;
            float* y = static_cast<float*>(dst) + row;
            const float x0 = x[i], x1 = x[i + half];
            y[i] = x0 * c - x1 * s;
            y[i + half] = x1 * c + x0 * s;
        }
    }
}

}  // namespace

hipError_t launch_rope(const void* src, int64_t head_stride, int64_t token_stride, void* dst, int dtype_bf16,
                       int heads, int64_t N, int D, int64_t pos0, const RopeTable& tab, hipStream_t st) {
    const int64_t work = N * (D / 2);
    const unsigned blocks = (unsigned)((work + kThreads - 1) / kThreads);
    if (dtype_bf16)
        hipLaunchKernelGGL(k_rope<true>, dim3(blocks), dim3(kThreads), 0, st, src, head_stride, token_stride, dst,
                           heads, N, D, pos0, tab);
    else
        hipLaunchKernelGGL(k_rope<false>, dim3(blocks), dim3(kThreads), 0, st, src, head_stride, token_stride, dst,
                           heads, N, D, pos0, tab);
    return hipGetLastError();
}

}  // namespace ris
