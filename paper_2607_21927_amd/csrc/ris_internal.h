// Internal launch interfaces between the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ris {

// Resolved geometry parameters (block already fixed for Structural mode).
struct MaskParams {
    uint64_t seed;
    int64_t N;
    int32_t mode;
    int32_t ppm;
    int32_t n_seeds;
    int32_t layer;
    int32_t heads;
    int32_t causal;
    int32_t block;
};

hipError_t launch_mask_count(const MaskParams& p, int64_t* row_ptr, hipStream_t st);
hipError_t launch_mask_fused(const MaskParams& p, int64_t* row_ptr, int32_t* col_idx,
                             int64_t capacity, hipStream_t st);
hipError_t launch_mask_fill(const MaskParams& p, const int64_t* row_ptr, int32_t* col_idx,
                            int64_t capacity, hipStream_t st);

constexpr int kMaxRopeHalf = 256;
struct RopeTable {
    double inv_freq[kMaxRopeHalf];
    double mscale;
};
hipError_t launch_rope(void* x, int dtype_bf16, int heads, int64_t N, int D, int64_t pos0,
                       const RopeTable& tab, hipStream_t st);

struct AttnParams {
    const void* Q;
    const void* K;
    const void* V;
    const int64_t* row_ptr;
    const int32_t* col_idx;
    void* out;
    int64_t N;
    int32_t Hq, Hkv, G, D;
    int32_t in_bf16, out_bf16;
    int32_t mode, block, causal;
    float scale;
};
hipError_t launch_attn_gather(const AttnParams& a, hipStream_t st);
hipError_t launch_attn_tile(const AttnParams& a, hipStream_t st);

}  // namespace ris
