// Elementwise layers of the host models around the sparse attention: the
// residual add fused with RMSNorm, and the SwiGLU activation of the MLP.
// Both are HBM-bound; one pass over the data each, float32 arithmetic.
#include "ris_device.h"
#include "ris_internal.h"

namespace ris {
namespace {

constexpr int kNormThreads = 256;

__device__ __forceinline__ float load_elt(const void* p, int64_t i, bool bf16) {
    return bf16 ? bf16_to_f32(static_cast<const uint16_t*>(p)[i]) : static_cast<const float*>(p)[i];
}
__device__ __forceinline__ void store_elt(void* p, int64_t i, float v, bool bf16) {
    if (bf16)
        static_cast<uint16_t*>(p)[i] = f32_to_bf16(v);
    else
        static_cast<float*>(p)[i] = v;
}

// One workgroup per row.  r = x (+ residual); residual <- r when given (the
// stored value, rounded to the element type, is what the norm reads back, so
// the residual stream and the norm see the same numbers); out = r * rsqrt(mean
// (r^2) + eps) * w.
__global__ __launch_bounds__(kNormThreads) void k_rmsnorm(const void* x, void* residual, const void* w,
                                                          void* out, int64_t cols, float eps, int bf16) {
    __shared__ float red[kNormThreads / 64];
    const int64_t row = blockIdx.x;
    const int64_t base = row * cols;
    float ss = 0.f;
    for (int64_t c = threadIdx.x; c < cols; c += kNormThreads) {
        float r = load_elt(x, base + c, bf16);
        if (residual) {
            r += load_elt(residual, base + c, bf16);
            store_elt(residual, base + c, r, bf16);
            r = load_elt(residual, base + c, bf16);
        }
        ss += r * r;
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kNormThreads / 64; ++i) tot += red[i];
    const float inv = rsqrtf(tot / (float)cols + eps);
    for (int64_t c = threadIdx.x; c < cols; c += kNormThreads) {
        const float r = residual ? load_elt(residual, base + c, bf16) : load_elt(x, base + c, bf16);
        store_elt(out, base + c, r * inv * load_elt(w, c, bf16), bf16);
    }
}

// out[r, c] = silu(gu[r, c]) * gu[r, I + c], silu(g) = g / (1 + exp(-g)).
__global__ void k_swiglu(const void* gu, void* out, int64_t rows, int64_t inter, int bf16) {
    const int64_t n = rows * inter;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / inter, c = i - r * inter;
        const float g = load_elt(gu, r * 2 * inter + c, bf16);
        const float u = load_elt(gu, r * 2 * inter + inter + c, bf16);
        store_elt(out, i, g / (1.0f + expf(-g)) * u, bf16);
    }
}

}  // namespace

hipError_t launch_rmsnorm(const void* x, void* residual, const void* w, void* out, int64_t rows,
                          int64_t cols, float eps, int bf16, hipStream_t st) {
    hipLaunchKernelGGL(k_rmsnorm, dim3((unsigned)rows), dim3(kNormThreads), 0, st, x, residual, w, out, cols,
                       eps, bf16);
    return hipGetLastError();
}

hipError_t launch_swiglu(const void* gu, void* out, int64_t rows, int64_t inter, int bf16, hipStream_t st) {
    const int64_t n = rows * inter;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_swiglu, dim3((unsigned)blocks), dim3(256), 0, st, gu, out, rows, inter, bf16);
    return hipGetLastError();
}

}  // namespace ris
