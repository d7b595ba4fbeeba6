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

// Density decision for the tile of rows [q0, q0 + kTileRows) of KV head g.
// The tiled kernel's cost follows the key range it walks, the gather
// kernel's the entries, so a tile is dense when its entries fill at least a
// fraction tau of rows x keys over the causal span [0, q1) (or [0, N)) or,
// failing that, over the range from the tile's first CSR entry (the first
// key of its first non-empty row) to its last (the last key of its last
// non-empty row), capped at the span.  Two reads of row_ptr, and two of
// col_idx for tiles sparse over the span; every thread that asks gets the
// same answer.
__device__ __forceinline__ bool tile_is_dense(const AttnParams& a, int g, int64_t q0) {
    const int64_t q1 = q0 + kTileRows < a.N ? q0 + kTileRows : a.N;
    const int64_t* rp = a.row_ptr + (int64_t)g * a.N;
    const int64_t s0 = rp[q0], s1 = rp[q1];
    const int64_t nnz = s1 - s0;
    const double rows = (double)(q1 - q0);
    const int64_t span = a.causal ? q1 : a.N;
    if ((double)nnz >= (double)a.tau * rows * (double)span) return true;
    if (s0 < 0 || nnz <= 0) return false;
    int64_t f = a.col_idx[s0], l = a.col_idx[s1 - 1];
    if (f < 0) f = 0;
    if (l > a.N - 1) l = a.N - 1;
    int64_t range = l >= f ? l - f + 1 : 1;
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
