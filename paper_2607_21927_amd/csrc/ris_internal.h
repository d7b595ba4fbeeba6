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
    int32_t window;   // local window L (0 = none)
    int32_t anchor;   // initial-token anchor A (0 = none)
    int64_t q0;       // rows [q0, q0 + nq) of each head are built;
    int64_t nq;       // row r = h * nq + (q - q0)
    uint32_t spin_limit;   // one-pass build: look-back polls before a row gives up
    int64_t poison_row;    // one-pass build test hook: this row publishes poison (-1 = none)
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
hipError_t launch_rope(const void* src, int64_t head_stride, int64_t token_stride, void* dst, int dtype_bf16,
                       int heads, int64_t N, int D, int64_t pos0, const RopeTable& tab, hipStream_t st);

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
    // Per 32-row tile, the tiled kernel takes tiles whose union density
    // (tile nnz / (rows x key range walked)) is >= tau and the gather kernel
    // the rest.
    float tau;
};

// Rows per tile of the tiled kernel; also the unit of the dispatch decision.
constexpr int kTileRows = 32;

// Density decision for the tile of rows [q0, q0 + kTileRows) of KV head g,
// taken by a whole wave (every lane active, uniform arguments; the result is
// the same in every lane and in every wave that asks).  The tiled kernel's
// cost follows the key range it walks, the gather kernel's the entries, so a
// tile is dense when its entries fill at least a fraction tau of rows x keys
// over the range from its rows' smallest first key to their largest last
// key, capped at the key span [0, q1) (causal) or [0, N).  Tiles dense over
// the whole span are settled by two reads of row_ptr; the others read every
// row's first and last key.
__device__ __forceinline__ bool tile_is_dense(const AttnParams& a, int g, int64_t q0) {
    const int64_t q1 = q0 + kTileRows < a.N ? q0 + kTileRows : a.N;
    const int64_t* rp = a.row_ptr + (int64_t)g * a.N;
    const int64_t nnz = rp[q1] - rp[q0];
    const double rows = (double)(q1 - q0);
    const int64_t span = a.causal ? q1 : a.N;
    if ((double)nnz >= (double)a.tau * rows * (double)span) return true;
    const int lane = threadIdx.x & 63;
    int lo = 0x7FFFFFFF, hi = -1;
    if (lane < q1 - q0) {
        const int64_t s = rp[q0 + lane], e = rp[q0 + lane + 1];
        if (s >= 0 && e > s) {
            int f = a.col_idx[s], l = a.col_idx[e - 1];
            if (f < 0) f = 0;
            if ((int64_t)l > a.N - 1) l = (int)(a.N - 1);
            if (f <= l) { lo = f; hi = l; }
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        lo = min(lo, __shfl_xor(lo, off));
        hi = max(hi, __shfl_xor(hi, off));
    }
    int64_t range = hi >= lo ? (int64_t)hi - lo + 1 : 1;
    if (range > span) range = span;
    return (double)nnz >= (double)a.tau * rows * (double)range;
}
hipError_t launch_attn_gather(const AttnParams& a, hipStream_t st);
hipError_t launch_attn_tile(const AttnParams& a, hipStream_t st);

// Decode step (Hybrid Anchor).  Each row's virtual key list is cut into
// kDecodeTileKeys-key tiles dealt round-robin to the row's `parts` waves
// (kDecodeWaves per workgroup); every wave writes one partial (its max, sum
// and unnormalised output per head).
constexpr int kDecodeWaves = 4;
constexpr int kDecodeTileKeys = 32;
constexpr int kDecodeMaxParts = 1024;
constexpr int kDecodeTargetWaves = 2048;   // 256 CUs x 8 resident waves
struct DecodeParams {
    const void* Q;                // [B, Hq, D] bf16
    const void* K;                // [B, Hkv, max_len, D] bf16
    const void* V;
    const int64_t* pos;           // [B]
    const int64_t* anchor_ptr;    // [B, Hkv + 1]
    const int32_t* anchor_idx;    // [B, anchor_stride]
    void* out;                    // [B, Hq, D]
    float* part_o;                // [B * Hkv, parts, G, D]
    float* part_ml;               // [B * Hkv, parts, G, 2]
    int64_t max_len, anchor_stride;
    int32_t B, Hq, Hkv, G, D;
    int32_t out_bf16;
    int32_t window, sink;
    int32_t parts;                // partials per row (a multiple of kDecodeWaves)
    float scale;
};
hipError_t launch_decode(const DecodeParams& p, hipStream_t st);

// Host-model layers around the attention (model-level prefill).
hipError_t launch_rmsnorm(const void* x, void* residual, const void* w, void* out, int64_t rows,
                          int64_t cols, float eps, int bf16, hipStream_t st);
hipError_t launch_swiglu(const void* gu, void* out, int64_t rows, int64_t inter, int bf16, hipStream_t st);

}  // namespace ris
