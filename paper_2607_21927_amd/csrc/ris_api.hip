// C ABI of the RIS library: argument validation, parameter resolution and
// kernel dispatch.  Nothing here allocates device memory or keeps state.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <atomic>

#include "ris.h"
#include "ris_device.h"
#include "ris_internal.h"

namespace {

using ris::MaskParams;

int validate_mask(const ris_mask_desc* d) {
    if (!d) return RIS_E_ARG;
    if (d->mode != RIS_STOCHASTIC && d->mode != RIS_STRUCTURAL) return RIS_E_ARG;
    if (d->density_ppm < 1 || d->density_ppm > 1000000) return RIS_E_ARG;
    if (d->n_seeds < 1 || d->n_seeds > RIS_MAX_SEEDS) return RIS_E_ARG;
    if (d->layer < 0) return RIS_E_ARG;
    if (d->N < 1 || d->N > RIS_MAX_N) return RIS_E_ARG;
    if (d->heads < 1 || d->heads > 8192) return RIS_E_ARG;
    if (d->causal != 0 && d->causal != 1) return RIS_E_ARG;
    if (d->block < 0) return RIS_E_ARG;
    if (d->window < 0 || d->anchor < 0) return RIS_E_ARG;
    if (d->mode == RIS_STRUCTURAL && !d->causal) return RIS_E_UNSUPPORTED;
    if ((d->window > 0 || d->anchor > 0) && !d->causal) return RIS_E_UNSUPPORTED;
    return RIS_OK;
}

// Rows [q_begin, q_begin + q_count) of every head; one workgroup per row.
int validate_rows(const ris_mask_desc* d, int64_t q_begin, int64_t q_count) {
    const int st = validate_mask(d);
    if (st != RIS_OK) return st;
    if (q_begin < 0 || q_count < 1 || q_begin > d->N - q_count) return RIS_E_ARG;
    if ((int64_t)d->heads * q_count > 0x7FFFFFFFll) return RIS_E_UNSUPPORTED;
    return RIS_OK;
}

// Structural block size: explicit, or min(floor(N / 10), B_max) with B_max the
// count rule evaluated on n = N (at least 1).
int32_t resolve_block(const ris_mask_desc* d) {
    if (d->mode != RIS_STRUCTURAL) return 1;
    if (d->block > 0) return d->block;
    int64_t b = ris::row_count(d->density_ppm, d->N);
    if (d->N / 10 < b) b = d->N / 10;
    return b < 1 ? 1 : (int32_t)b;
}

// Polls of a predecessor's status before a row of the one-pass build gives
// up (about 0.7 s of waiting; every wait ends long before in a healthy run).
// RIS_DEBUG_LOOKBACK_SPINS overrides it: a test hook that makes the give-up
// path run (0 = give up at the first wait).
uint32_t lookback_spin_limit() {
    const char* s = getenv("RIS_DEBUG_LOOKBACK_SPINS");
    if (s && *s) {
        char* end = nullptr;
        const unsigned long v = strtoul(s, &end, 10);
        if (end && *end == '\0') return v > 0xFFFFFFFFul ? 0xFFFFFFFFu : (uint32_t)v;
    }
    return 1u << 24;
}

// RIS_DEBUG_POISON_ROW=<r>: a second test hook.  Row r of the one-pass
// build publishes poison in place of its look-back, as if its wait had given
// up, so that the poison path runs whatever the timing (-1 = none).
int64_t lookback_poison_row() {
    const char* s = getenv("RIS_DEBUG_POISON_ROW");
    if (s && *s) {
        char* end = nullptr;
        const long long v = strtoll(s, &end, 10);
        if (end && *end == '\0' && v >= 0) return (int64_t)v;
    }
    return -1;
}

MaskParams make_params(const ris_mask_desc* d, int64_t q0, int64_t nq) {
    MaskParams p;
    p.spin_limit = lookback_spin_limit();
    p.poison_row = lookback_poison_row();
    p.q0 = q0;
    p.nq = nq;
    p.seed = d->seed;
    p.N = d->N;
    p.mode = d->mode;
    p.ppm = d->density_ppm;
    p.n_seeds = d->n_seeds;
    p.layer = d->layer;
    p.heads = d->heads;
    p.causal = d->causal;
    p.block = resolve_block(d);
    p.window = d->window;
    p.anchor = d->anchor;
    return p;
}

int64_t nnz_bound(const MaskParams& p) {
    int64_t total = 0;
    for (int64_t q = p.q0; q < p.q0 + p.nq; ++q) {
        int64_t row;
        if (p.mode == RIS_STOCHASTIC) {
            const int64_t n = p.causal ? q + 1 : p.N;
            const int64_t k = ris::row_count(p.ppm, n) * p.n_seeds;
            row = k < n ? k : n;
        } else {
            const int64_t start = (q / p.block) * (int64_t)p.block;
            const int64_t clique = q - start + 1;
            int64_t kg = ris::row_count(p.ppm, q + 1) - clique;
            if (kg < 0) kg = 0;
            if (kg > start) kg = start;
            const int64_t g = kg * p.n_seeds;
            row = clique + (g < start ? g : start);
        }
        if (p.window > 0 || p.anchor > 0) {
            row += (p.window < q + 1 ? p.window : q + 1) + (p.anchor < q + 1 ? p.anchor : q + 1);
            if (row > q + 1) row = q + 1;
        }
        total += row;
    }
    return total * p.heads;
}

int hip_status(hipError_t e) { return e == hipSuccess ? RIS_OK : RIS_E_HIP; }

// Union density of a 32-row tile (entries over rows x the key range the
// tiled kernel walks) from which the tiled kernel takes it.  Measured on
// MI355X for layers whose tiles are all alike (Qwen2 shape, Stochastic 1%,
// 4-6 seeds, N = 32k and 64k), the two kernels cross near 5.7%; the gather
// kernel left with only a minority of a layer's tiles runs below its
// full-load rate, which moves the best split for mixed layers lower (32k
// Structural with B = 64: 4.5 ms at 6.8%, 3.8 ms at 5%), so the threshold
// sits at 5%, still above the 4.9% union of five seeds, which the gather
// kernel serves 15% faster.
constexpr float kAutoDensity = 0.05f;

}  // namespace

extern "C" {

int ris_version(void) { return (2 << 16) | 4; }

const char* ris_status_string(int status) {
    switch (status) {
        case RIS_OK: return "RIS_OK";
        case RIS_E_ARG: return "RIS_E_ARG: null pointer or out-of-range argument";
        case RIS_E_SHAPE: return "RIS_E_SHAPE: inconsistent sizes";
        case RIS_E_DTYPE: return "RIS_E_DTYPE: unknown element type";
        case RIS_E_CAPACITY: return "RIS_E_CAPACITY: col_idx capacity below nnz";
        case RIS_E_UNSUPPORTED: return "RIS_E_UNSUPPORTED: valid request outside what is implemented";
        case RIS_E_HIP: return "RIS_E_HIP: HIP runtime error";
        case RIS_E_INCOMPLETE: return "RIS_E_INCOMPLETE: one-pass geometry build gave up (row_ptr total < 0)";
        default: return "unknown ris_status";
    }
}

int64_t ris_mask_rows_nnz_bound(const ris_mask_desc* desc, int64_t q_begin, int64_t q_count) {
    const int st = validate_rows(desc, q_begin, q_count);
    if (st != RIS_OK) return st;
    return nnz_bound(make_params(desc, q_begin, q_count));
}

int64_t ris_mask_nnz_bound(const ris_mask_desc* desc) {
    if (!desc) return RIS_E_ARG;
    return ris_mask_rows_nnz_bound(desc, 0, desc->N);
}

int ris_mask_build_rows(const ris_mask_desc* desc, int64_t q_begin, int64_t q_count,
                        int64_t* row_ptr, int32_t* col_idx, int64_t col_capacity, void* stream) {
    const int st = validate_rows(desc, q_begin, q_count);
    if (st != RIS_OK) return st;
    if (!row_ptr) return RIS_E_ARG;
    const MaskParams p = make_params(desc, q_begin, q_count);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!col_idx) return hip_status(ris::launch_mask_count(p, row_ptr, s));
    if (col_capacity < 0) return RIS_E_ARG;
    // Capacity covers every possible row: one fused pass computes row_ptr too.
    if (col_capacity >= nnz_bound(p))
        return hip_status(ris::launch_mask_fused(p, row_ptr, col_idx, col_capacity, s));
    {
        int64_t nnz = 0;
        const int64_t rows = (int64_t)p.heads * p.nq;
        if (hipMemcpyAsync(&nnz, row_ptr + rows, sizeof(nnz), hipMemcpyDeviceToHost, s) != hipSuccess)
            return RIS_E_HIP;
        if (hipStreamSynchronize(s) != hipSuccess) return RIS_E_HIP;
        if (nnz > col_capacity || nnz < 0) return RIS_E_CAPACITY;
    }
    return hip_status(ris::launch_mask_fill(p, row_ptr, col_idx, col_capacity, s));
}

int ris_mask_build(const ris_mask_desc* desc, int64_t* row_ptr, int32_t* col_idx,
                   int64_t col_capacity, void* stream) {
    if (!desc) return RIS_E_ARG;
    return ris_mask_build_rows(desc, 0, desc->N, row_ptr, col_idx, col_capacity, stream);
}

int ris_rope(void* x, int32_t dtype, int32_t heads, int64_t N, int32_t D, int64_t pos0,
             const ris_rope_desc* desc, void* stream) {
    return ris_rope_from(x, N * D, D, x, dtype, heads, N, D, pos0, desc, stream);
}

int ris_rope_from(const void* src, int64_t head_stride, int64_t token_stride, void* x, int32_t dtype,
                  int32_t heads, int64_t N, int32_t D, int64_t pos0, const ris_rope_desc* desc, void* stream) {
    if (!src || !x || !desc) return RIS_E_ARG;
    if (head_stride < 0 || token_stride < 0) return RIS_E_ARG;
    if (dtype != RIS_F32 && dtype != RIS_BF16) return RIS_E_DTYPE;
    if (heads < 1 || N < 1 || pos0 < 0) return RIS_E_ARG;
    if (D < 2 || (D & 1) || D / 2 > ris::kMaxRopeHalf) return RIS_E_SHAPE;
    if (desc->kind < RIS_ROPE_PLAIN || desc->kind > RIS_ROPE_YARN) return RIS_E_ARG;
    if (!(desc->base > 1.0) || !isfinite(desc->base)) return RIS_E_ARG;
    if (!(desc->factor >= 0.0) || !isfinite(desc->factor)) return RIS_E_ARG;
    if (!(desc->beta_slow >= 0.0) || !(desc->beta_fast >= 0.0)) return RIS_E_ARG;
    if (desc->kind != RIS_ROPE_PLAIN && desc->orig_max_pos < 1) return RIS_E_ARG;
    if (N > (1ll << 32) || pos0 > (1ll << 52)) return RIS_E_ARG;

    // Factor: requested window / native limit (at least 1) unless given.
    double s = desc->factor;
    if (desc->kind != RIS_ROPE_PLAIN && !(s > 0.0)) {
        s = (double)(pos0 + N) / (double)desc->orig_max_pos;
        if (s < 1.0) s = 1.0;
    }
    ris::RopeTable tab;
    const int half = D / 2;
    const double base = desc->base;
    for (int i = 0; i < half; ++i) {
        const double plain = 1.0 / pow(base, 2.0 * i / D);
        double f = plain;
        if (desc->kind == RIS_ROPE_LINEAR) {
            f = plain / s;
        } else if (desc->kind == RIS_ROPE_YARN) {
            const double b_slow = desc->beta_slow > 0.0 ? desc->beta_slow : 1.0;
            const double b_fast = desc->beta_fast > 0.0 ? desc->beta_fast : 32.0;
            const double L0 = (double)desc->orig_max_pos;
            const double c_fast = D * log(L0 / (b_fast * 2.0 * M_PI)) / (2.0 * log(base));
            const double c_slow = D * log(L0 / (b_slow * 2.0 * M_PI)) / (2.0 * log(base));
            double lo = floor(c_fast), hi = ceil(c_slow);
            if (lo < 0.0) lo = 0.0;
            if (hi > D - 1) hi = D - 1;
            if (lo == hi) hi += 0.001;
            double t = (i - lo) / (hi - lo);
            t = t < 0.0 ? 0.0 : (t > 1.0 ? 1.0 : t);
            f = t * (plain / s) + (1.0 - t) * plain;
        }
        tab.inv_freq[i] = f;
    }
    tab.mscale = (desc->kind == RIS_ROPE_YARN && s > 1.0) ? 0.1 * log(s) + 1.0 : 1.0;
    return hip_status(ris::launch_rope(src, head_stride, token_stride, x, dtype == RIS_BF16, heads, N, D, pos0,
                                       tab, static_cast<hipStream_t>(stream)));
}

int ris_sparse_attn(const void* Q, const void* K, const void* V, const int64_t* row_ptr,
                    const int32_t* col_idx, void* out, const ris_attn_desc* desc, void* stream) {
    if (!Q || !K || !V || !row_ptr || !col_idx || !out || !desc) return RIS_E_ARG;
    const ris_attn_desc& d = *desc;
    if ((d.dtype_in != RIS_F32 && d.dtype_in != RIS_BF16) ||
        (d.dtype_out != RIS_F32 && d.dtype_out != RIS_BF16))
        return RIS_E_DTYPE;
    if (d.Hq < 1 || d.Hkv < 1 || d.N < 1 || d.N > RIS_MAX_N) return RIS_E_ARG;
    if (d.Hq % d.Hkv != 0) return RIS_E_SHAPE;
    if (d.Hq / d.Hkv > 8) return RIS_E_UNSUPPORTED;
    if (d.D != 64 && d.D != 128) return RIS_E_UNSUPPORTED;
    if (!(d.scale >= 0.0f) || !isfinite(d.scale)) return RIS_E_ARG;
    if (d.mode != RIS_STOCHASTIC && d.mode != RIS_STRUCTURAL) return RIS_E_ARG;
    if (d.algo < RIS_ATTN_AUTO || d.algo > RIS_ATTN_TILE) return RIS_E_ARG;
    if ((int64_t)d.Hkv * d.N > 0x7FFFFFFFll) return RIS_E_UNSUPPORTED;

    ris::AttnParams a;
    a.Q = Q; a.K = K; a.V = V;
    a.row_ptr = row_ptr; a.col_idx = col_idx; a.out = out;
    a.N = d.N; a.Hq = d.Hq; a.Hkv = d.Hkv; a.G = d.Hq / d.Hkv; a.D = d.D;
    a.in_bf16 = d.dtype_in == RIS_BF16; a.out_bf16 = d.dtype_out == RIS_BF16;
    a.mode = d.mode; a.block = d.block; a.causal = d.causal;
    a.scale = d.scale > 0.0f ? d.scale : 1.0f / sqrtf((float)d.D);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // The tiled MFMA kernel needs bf16 operands; float32 inputs take the gather kernel.
    if (d.algo == RIS_ATTN_TILE && !a.in_bf16) return RIS_E_UNSUPPORTED;
    if (d.algo == RIS_ATTN_GATHER || !a.in_bf16) {
        a.tau = INFINITY;                       // every tile to the gather kernel
        return hip_status(ris::launch_attn_gather(a, s));
    }
    if (d.algo == RIS_ATTN_TILE) {
        a.tau = -1.0f;                          // every tile to the tiled kernel
        return hip_status(ris::launch_attn_tile(a, s));
    }
    // AUTO: per 32-row tile by union density.  The tiled kernel's cost grows
    // with the key range its rows touch, the gather kernel's with the entries
    // (kAutoDensity).
    a.tau = kAutoDensity;
    const int st = hip_status(ris::launch_attn_tile(a, s));
    if (st != RIS_OK) return st;
    return hip_status(ris::launch_attn_gather(a, s));
}

}  // extern "C"

// ---- decode step

namespace {

// Partials (waves) per row.  Any value covers every key (the tiles are dealt
// round-robin); this one aims at ~2048 resident waves over the batch without
// giving a wave less than one tile of a typical row (the anchor slice shared
// evenly by the kv heads, plus window and initial tokens).
int64_t decode_parts(const ris_decode_desc& d) {
    const int64_t win = d.window < d.max_len ? d.window : d.max_len;
    const int64_t snk = d.sink < d.max_len ? d.sink : d.max_len;
    const int64_t keys = (d.anchor_stride + d.Hkv - 1) / d.Hkv + win + snk;
    const int64_t tiles = (keys + ris::kDecodeTileKeys - 1) / ris::kDecodeTileKeys;
    const int64_t rows = (int64_t)d.batch * d.Hkv;
    int64_t parts = (ris::kDecodeTargetWaves + rows - 1) / rows;
    if (parts > tiles) parts = tiles;
    parts = (parts + ris::kDecodeWaves - 1) / ris::kDecodeWaves * ris::kDecodeWaves;
    if (parts < ris::kDecodeWaves) parts = ris::kDecodeWaves;
    if (parts > ris::kDecodeMaxParts) parts = ris::kDecodeMaxParts;
    return parts;
}

int validate_decode(const ris_decode_desc* d) {
    if (!d) return RIS_E_ARG;
    if (d->dtype_in != RIS_F32 && d->dtype_in != RIS_BF16) return RIS_E_DTYPE;
    if (d->dtype_out != RIS_F32 && d->dtype_out != RIS_BF16) return RIS_E_DTYPE;
    if (d->dtype_in != RIS_BF16) return RIS_E_UNSUPPORTED;
    if (d->batch < 1 || d->Hq < 1 || d->Hkv < 1) return RIS_E_ARG;
    if (d->Hq % d->Hkv != 0) return RIS_E_SHAPE;
    if (d->Hq / d->Hkv > 8) return RIS_E_UNSUPPORTED;
    if (d->D != 64 && d->D != 128) return RIS_E_UNSUPPORTED;
    if (d->max_len < 1 || d->max_len > (1ll << 31)) return RIS_E_ARG;
    if (d->anchor_stride < 0 || d->anchor_stride > (1ll << 40)) return RIS_E_ARG;
    if (d->window < 0 || d->sink < 0) return RIS_E_ARG;
    if (!(d->scale >= 0.0f) || !isfinite(d->scale)) return RIS_E_ARG;
    if ((int64_t)d->batch * d->Hkv > 65535) return RIS_E_UNSUPPORTED;
    if ((int64_t)d->batch * d->Hq > 0x7FFFFFFFll) return RIS_E_UNSUPPORTED;
    return RIS_OK;
}

int64_t decode_workspace(const ris_decode_desc& d) {
    const int64_t per = (int64_t)d.batch * d.Hkv * decode_parts(d) * (d.Hq / d.Hkv);
    return per * (d.D + 2) * (int64_t)sizeof(float);
}

}  // namespace

extern "C" {

int ris_rmsnorm(const void* x, void* residual, const void* weight, void* out, int64_t rows,
                int64_t cols, float eps, int32_t dtype, void* stream) {
    if (!x || !weight || !out) return RIS_E_ARG;
    if (dtype != RIS_F32 && dtype != RIS_BF16) return RIS_E_DTYPE;
    if (rows < 1 || rows > 0x7FFFFFFFll || cols < 1 || cols > (1 << 20)) return RIS_E_ARG;
    if (!(eps > 0.0f) || !isfinite(eps)) return RIS_E_ARG;
    return hip_status(ris::launch_rmsnorm(x, residual, weight, out, rows, cols, eps, dtype == RIS_BF16,
                                          static_cast<hipStream_t>(stream)));
}

int ris_swiglu(const void* gate_up, void* out, int64_t rows, int64_t inter, int32_t dtype, void* stream) {
    if (!gate_up || !out) return RIS_E_ARG;
    if (dtype != RIS_F32 && dtype != RIS_BF16) return RIS_E_DTYPE;
    if (rows < 1 || inter < 1 || rows > (1ll << 40) / inter) return RIS_E_ARG;
    return hip_status(ris::launch_swiglu(gate_up, out, rows, inter, dtype == RIS_BF16,
                                         static_cast<hipStream_t>(stream)));
}

int64_t ris_decode_workspace_bytes(const ris_decode_desc* desc) {
    const int st = validate_decode(desc);
    if (st != RIS_OK) return st;
    return decode_workspace(*desc);
}

}  // extern "C"

// ---- decode step without a caller workspace

namespace {

// The partials of ris_decode_attn_static: a file-scope device array, one copy
// per GPU, alive until the process ends.  Host code never passes the array's
// name to a kernel (on the host it is only a stand-in); it passes the device
// address hipGetSymbolAddress gives on the current device.
constexpr int64_t kDecodeStaticBytes = RIS_DECODE_STATIC_BYTES;
__device__ __align__(256) unsigned char scratch[kDecodeStaticBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of the current device's copy of `scratch`, looked up once
// per device (a lookup, no allocation); nullptr on failure.
void* device_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    void* ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (ptr) return ptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev].store(ptr, std::memory_order_release);
    return ptr;
}

}  // namespace

extern "C" {

int ris_decode_attn_static(const void* Q, const void* K, const void* V, const int64_t* pos,
                           const int64_t* anchor_ptr, const int32_t* anchor_idx, void* out,
                           const ris_decode_desc* desc, void* stream) {
    const int st = validate_decode(desc);
    if (st != RIS_OK) return st;
    if (decode_workspace(*desc) > kDecodeStaticBytes) return RIS_E_CAPACITY;
    void* ws = device_scratch();
    if (!ws) return RIS_E_HIP;
    return ris_decode_attn(Q, K, V, pos, anchor_ptr, anchor_idx, out, ws, kDecodeStaticBytes, desc, stream);
}

int ris_decode_attn(const void* Q, const void* K, const void* V, const int64_t* pos,
                    const int64_t* anchor_ptr, const int32_t* anchor_idx, void* out,
                    void* workspace, int64_t workspace_bytes, const ris_decode_desc* desc,
                    void* stream) {
    const int st = validate_decode(desc);
    if (st != RIS_OK) return st;
    if (!Q || !K || !V || !pos || !anchor_ptr || !out || !workspace) return RIS_E_ARG;
    if (!anchor_idx && desc->anchor_stride > 0) return RIS_E_ARG;
    if (workspace_bytes < decode_workspace(*desc)) return RIS_E_CAPACITY;
    const ris_decode_desc& d = *desc;
    ris::DecodeParams p;
    p.Q = Q; p.K = K; p.V = V;
    p.pos = pos; p.anchor_ptr = anchor_ptr; p.anchor_idx = anchor_idx;
    p.out = out;
    p.max_len = d.max_len; p.anchor_stride = d.anchor_stride;
    p.B = d.batch; p.Hq = d.Hq; p.Hkv = d.Hkv; p.G = d.Hq / d.Hkv; p.D = d.D;
    p.out_bf16 = d.dtype_out == RIS_BF16;
    p.window = d.window; p.sink = d.sink;
    p.parts = (int32_t)decode_parts(d);
    p.scale = d.scale > 0.0f ? d.scale : 1.0f / sqrtf((float)d.D);
    const int64_t n_o = (int64_t)d.batch * d.Hkv * p.parts * p.G * d.D;
    p.part_o = static_cast<float*>(workspace);
    p.part_ml = p.part_o + n_o;
    return hip_status(ris::launch_decode(p, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
