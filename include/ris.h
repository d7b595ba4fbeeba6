/*
 * ris.h -- C ABI of the RIS sparse-attention library for AMD Instinct MI355X
 * (gfx950).  Plain C types only: device pointers, sizes and small descriptor
 * structs.  Every call is asynchronous on the given HIP stream (a
 * hipStream_t passed as void*, NULL = the default stream) unless its comment
 * says otherwise.
 *
 * Errors: every call returns RIS_OK (0) or a negative ris_status.  Arguments
 * are validated on the host before anything is launched; a call that fails
 * validation launches nothing and writes nothing.  A HIP runtime failure maps
 * to RIS_E_HIP.  Nothing aborts and no exception crosses the ABI.
 *
 * Ownership: the caller allocates every buffer; the library keeps no global
 * mutable state and no allocation alive between calls.
 *
 * The operations follow the paper "RIS-Kernel: A Model-Agnostic Architecture
 * for Long-Context LLM Inference via Sparse Attention": geometry generation
 * (Methods, "Memory-Bounded Geometry Generation" and "Sampling Modes"),
 * RoPE scaling (Methods, "Dynamic RoPE Scaling") and one softmax over the
 * unified index set (Methods, "Hybrid Anchor and Pre-Fusion Unified
 * Softmax").
 */
#ifndef RIS_H
#define RIS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RIS_OK = 0,
    RIS_E_ARG = -1,          /* null pointer or out-of-range scalar          */
    RIS_E_SHAPE = -2,        /* inconsistent sizes (e.g. Hq % Hkv != 0)      */
    RIS_E_DTYPE = -3,        /* unknown element type                         */
    RIS_E_CAPACITY = -4,     /* col_idx capacity below the number of entries */
    RIS_E_UNSUPPORTED = -5,  /* valid request outside what is implemented    */
    RIS_E_HIP = -6,          /* HIP runtime error                            */
    RIS_E_INCOMPLETE = -7    /* a one-pass geometry build reported an        */
                             /* incomplete CSR (row_ptr[heads*N] < 0); the   */
                             /* library's calls never return it, the caller  */
                             /* that reads row_ptr does                      */
} ris_status;

typedef enum { RIS_STOCHASTIC = 0, RIS_STRUCTURAL = 1 } ris_mode;
typedef enum { RIS_F32 = 0, RIS_BF16 = 1 } ris_dtype;
typedef enum { RIS_ROPE_PLAIN = 0, RIS_ROPE_LINEAR = 1, RIS_ROPE_YARN = 2 } ris_rope_kind;
typedef enum { RIS_ATTN_AUTO = 0, RIS_ATTN_GATHER = 1, RIS_ATTN_TILE = 2 } ris_attn_algo;

/* Largest sequence length the geometry kernels accept (one row's pool is a
 * bitmap in on-chip LDS). */
#define RIS_MAX_N 262144
/* Largest ensemble size per call. */
#define RIS_MAX_SEEDS 4096

/* ------------------------------------------------------------------------ */
/* Geometry: per-query key sets as CSR                                       */
/* ------------------------------------------------------------------------ */

/*
 * What one layer's geometry depends on.
 *
 * Row r = kv_head * N + q holds I(kv_head, q), the union over the seeds
 * seed, seed+1, ..., seed+n_seeds-1 of each seed's set, ascending and without
 * duplicates (the seeds merge into one master set; Methods, "Memory-Bounded
 * Geometry Generation"; ensemble union, Results, "Ensemble Coverage
 * Analysis").
 *
 * Per seed, with pool size n_q = q+1 (causal) or N, the row draws exactly
 *   k(q) = clamp(floor((density_ppm * n_q + 500000) / 1000000), 1, n_q)
 * distinct keys, uniformly (Methods, "Sampling Modes", Stochastic).  In
 * Structural mode the row holds its block clique [bB, q] (b = floor(q/B)) plus
 * k_g = min(bB, max(0, k(q) - (q - bB + 1))) keys drawn uniformly from
 * [0, bB): the clique's cost is deducted from the global budget (Methods,
 * "Sampling Modes", Structural).  The draw of seed s for row (layer, kv_head,
 * q) is {P(0), ..., P(k-1)} for P a keyed Feistel permutation of the pool
 * (m-bit words, m = bitlen(n-1) with small-pool adjustments, cycle walking;
 * 16-bit multiply-xorshift rounds, 6 from 8 bits on and 12 below) whose round
 * keys are the 32-bit words of Philox4x64-10(counter = (q, kv_head, layer, 0),
 * key = (s, 0)); a keyed permutation yields distinct keys with no dedupe.
 *
 * The full geometry adds two contiguous ranges to the same union (Methods,
 * "Ensemble Stochastic Projection and Retrieval Coverage": dense local window
 * plus a global anchor over the initial tokens): the local window
 * [max(0, q - window + 1), q] and the anchor [0, min(anchor, q + 1)).  They
 * leave the per-seed draw counts unchanged.  0 disables either; both require
 * causal = 1.
 */
typedef struct {
    int32_t  mode;          /* ris_mode                                        */
    int32_t  density_ppm;   /* density d in parts per million, 1..1000000      */
    uint64_t seed;          /* first ensemble seed                             */
    int32_t  n_seeds;       /* S, 1..RIS_MAX_SEEDS                             */
    int32_t  layer;         /* layer index (>= 0), enters the hash             */
    int64_t  N;             /* sequence length, 1..RIS_MAX_N                   */
    int32_t  heads;         /* KV heads (>= 1); query heads of a group share   */
    int32_t  causal;        /* 1 = pool [0, q]; 0 = pool [0, N) (Stochastic)   */
    int32_t  block;         /* Structural block B; 0 = min(N/10, B_max) with   */
                            /* B_max = k evaluated on n = N                    */
    int32_t  window;        /* local window L (>= 0; 0 = none)                 */
    int32_t  anchor;        /* initial-token anchor A (>= 0; 0 = none)         */
} ris_mask_desc;

/*
 * Build the CSR of one layer's geometry: in one pass into a col_idx sized
 * from ris_mask_nnz_bound(), or in two phases for an exactly sized col_idx.
 *
 * row_ptr: device int64[heads*N + 1].  col_idx: device int32[col_capacity].
 *
 * Count phase (col_idx == NULL): writes row_ptr, the exclusive prefix sum of
 *   the row sizes (row_ptr[0] = 0, row_ptr[heads*N] = nnz).  The caller then
 *   reads row_ptr[heads*N] (8 bytes) to size col_idx, or sizes it with
 *   ris_mask_nnz_bound() and skips that read.
 * One-pass build (col_idx != NULL, col_capacity >= ris_mask_nnz_bound(desc)):
 *   row_ptr need not hold anything; the call writes both row_ptr and col_idx,
 *   generating every row once, fully asynchronously.  This is the fast path.
 *   Each row finds its offset by waiting on its predecessors' sizes; that wait
 *   is bounded (about 0.7 s, far beyond any healthy run).  A row that gives
 *   up, or whose predecessors' offsets are unknown because one gave up, writes
 *   no keys and -1 as its row_ptr entry, and row_ptr[heads*N] is then -1:
 *   the CSR is incomplete and must not be used (rebuild it, e.g. in two
 *   phases).  The call itself still returns RIS_OK, since it does not wait
 *   for the device; check row_ptr[heads*N] >= 0 where it is read back.  The
 *   environment variable RIS_DEBUG_LOOKBACK_SPINS=<polls> lowers the bound
 *   (a test hook: 0 gives up at the first wait), and RIS_DEBUG_POISON_ROW=<r>
 *   makes row r (of the rows built, head-major) give up without waiting (a
 *   test hook: row r, any row whose look-back reaches its status, and the
 *   total are then reported as -1).
 * Fill phase (col_idx != NULL, smaller capacity): row_ptr must hold the
 *   count phase's output for the same descriptor; the call first reads
 *   row_ptr[heads*N] (synchronising the stream), returns RIS_E_CAPACITY,
 *   writing nothing, when col_capacity < nnz, and otherwise writes
 *   col_idx[row_ptr[r] .. row_ptr[r+1]) for every row.
 * Writes never leave col_idx[0 .. col_capacity).
 * Requires Structural mode to be causal.
 */
int ris_mask_build(const ris_mask_desc* desc, int64_t* row_ptr, int32_t* col_idx,
                   int64_t col_capacity, void* stream);

/*
 * The same geometry for the rows [q_begin, q_begin + q_count) of every KV head
 * only: row r = kv_head * q_count + (q - q_begin), so row_ptr holds
 * heads*q_count + 1 entries.  Phases, capacity rule and errors as in
 * ris_mask_build (which is this call with q_begin = 0, q_count = N); the
 * bound is ris_mask_rows_nnz_bound.  Requires 0 <= q_begin and
 * q_begin + q_count <= N.  Serves chunked prefill and the decode anchor: the
 * stochastic anchor of a sequence whose first generated token sits at
 * position t0 is row t0 (q_begin = t0, q_count = 1) of a descriptor with
 * window = anchor = 0 (Methods, "Hybrid Anchor and Pre-Fusion Unified
 * Softmax").
 */
int ris_mask_build_rows(const ris_mask_desc* desc, int64_t q_begin, int64_t q_count,
                        int64_t* row_ptr, int32_t* col_idx, int64_t col_capacity, void* stream);

/* ris_mask_nnz_bound restricted to the rows [q_begin, q_begin + q_count). */
int64_t ris_mask_rows_nnz_bound(const ris_mask_desc* desc, int64_t q_begin, int64_t q_count);

/*
 * Host-only closed-form upper bound on nnz for the descriptor:
 * sum over rows of min(pool, n_seeds * draws) (+ clique), times heads; with a
 * window or anchor, each row adds min(window, q+1) + min(anchor, q+1) and is
 * capped at q + 1.  Exact when n_seeds == 1 and there is no window or anchor.
 * Returns a negative ris_status on a bad descriptor.
 */
int64_t ris_mask_nnz_bound(const ris_mask_desc* desc);

/* ------------------------------------------------------------------------ */
/* RoPE with the paper's long-context scaling                               */
/* ------------------------------------------------------------------------ */

/*
 * Scaling of the rotary frequencies (Methods, "Dynamic RoPE Scaling"; Results,
 * "Linear Interpolation" and "YaRN").  The factor is requested window /
 * native limit; the frequencies are those of the Hugging Face configuration
 * pathway the paper hooks:
 *   plain:  f_i = base^(-2i/D)
 *   linear: f_i / s
 *   YaRN:   ramp t_i = clamp((i - lo) / (hi - lo), 0, 1) with
 *           lo = max(floor(c(beta_fast)), 0), hi = min(ceil(c(beta_slow)), D-1),
 *           c(r) = D ln(orig_max_pos / (2 pi r)) / (2 ln base);
 *           f'_i = t_i f_i / s + (1 - t_i) f_i;  cos, sin scaled by
 *           0.1 ln s + 1 when s > 1.
 */
typedef struct {
    int32_t kind;            /* ris_rope_kind                                  */
    double  base;            /* rotary base (theta), > 1                       */
    int64_t orig_max_pos;    /* native positional limit (linear/YaRN), > 0     */
    double  factor;          /* s; 0 = max(1, (pos0 + N) / orig_max_pos)       */
    double  beta_slow;       /* YaRN; 0 = 1                                    */
    double  beta_fast;       /* YaRN; 0 = 32                                   */
} ris_rope_desc;

/*
 * Rotate x in place: x is device [heads, N, D] contiguous, element type dtype
 * (ris_dtype).  Token t has position pos0 + t.  Dimension i pairs with
 * i + D/2: y_i = x_i c - x_{i+D/2} s, y_{i+D/2} = x_{i+D/2} c + x_i s, with the
 * angle (pos0 + t) f'_i evaluated in float64, c and s (times the YaRN factor)
 * rounded to float32, the rotation in float32, and bf16 results rounded to
 * nearest even.  D must be even, 2..512.
 */
int ris_rope(void* x, int32_t dtype, int32_t heads, int64_t N, int32_t D, int64_t pos0,
             const ris_rope_desc* desc, void* stream);

/*
 * The same rotation read from a strided source and written to x, device
 * [heads, N, D] contiguous: element (h, t, d) of the source is at src +
 * h * head_stride + t * token_stride + d (strides in elements, >= 0, of the
 * same dtype).  src is only read.  x may be src itself with head_stride =
 * N * D and token_stride = D (that is ris_rope); any other overlap of the two
 * ranges is undefined.  Serves out-of-place rotation and, with head_stride =
 * D and token_stride = the row length of a token-major projection output,
 * the head-major layout and the rotation in one pass.
 */
int ris_rope_from(const void* src, int64_t head_stride, int64_t token_stride, void* x, int32_t dtype,
                  int32_t heads, int64_t N, int32_t D, int64_t pos0, const ris_rope_desc* desc,
                  void* stream);

/* ------------------------------------------------------------------------ */
/* Sparse attention over the unified index sets                             */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t dtype_in;        /* ris_dtype of Q, K, V                            */
    int32_t dtype_out;       /* ris_dtype of out                                */
    int32_t Hq;              /* query heads                                     */
    int32_t Hkv;             /* KV heads; Hq % Hkv == 0, G = Hq / Hkv <= 8       */
    int64_t N;               /* sequence length                                 */
    int32_t D;               /* head dimension: 64 or 128                       */
    float   scale;           /* score scale; 0 = 1 / sqrt(D)                    */
    int32_t mode;            /* ris_mode the CSR was built with                 */
    int32_t block;           /* its Structural block (as in ris_mask_desc)      */
    int32_t causal;          /* as in ris_mask_desc                             */
    int32_t algo;            /* ris_attn_algo: GATHER = per-row gather kernel;  */
                             /* TILE = 32-row tiles on MFMA (bf16 only); AUTO  */
                             /* = per 32-row tile, TILE when the tile's entries */
                             /* fill >= 5% of rows x keys over the causal span */
                             /* or over the range from its first CSR entry to  */
                             /* its last, GATHER otherwise                     */
} ris_attn_desc;

/*
 * out[h, q, :] = sum_{j in I(g, q)} softmax_j(scale <Q[h,q], K[g,j]>) V[g, j]
 * with g = floor(h / G): one normalisation over the whole unified set of the
 * row, every index once (Pre-Fusion Unified Softmax; Methods, "Hybrid Anchor
 * and Pre-Fusion Unified Softmax").  Q, out: device [Hq, N, D]; K, V: device
 * [Hkv, N, D]; contiguous.  row_ptr / col_idx: the CSR from ris_mask_build
 * with heads = Hkv and the same N (ascending rows, entries in [0, N)).
 * Accumulation is float32.  An empty row yields zeros, and so does a row
 * whose offsets are negative (a one-pass build that reported itself
 * incomplete; such a CSR is not a valid input, this only keeps every read
 * inside the buffers).
 */
int ris_sparse_attn(const void* Q, const void* K, const void* V, const int64_t* row_ptr,
                    const int32_t* col_idx, void* out, const ris_attn_desc* desc, void* stream);

/* ------------------------------------------------------------------------ */
/* Decode step with the Hybrid Anchor                                       */
/* ------------------------------------------------------------------------ */

/*
 * One generated token per sequence of a batch (Methods, "Hybrid Anchor and
 * Pre-Fusion Unified Softmax"): the stochastic anchor, computed once at the
 * first generated position and cached, merges with the local window of the
 * current position and the initial tokens, every index once, and each query
 * head takes one softmax over the merged set.
 */
typedef struct {
    int32_t dtype_in;        /* ris_dtype of Q and the K/V caches: RIS_BF16    */
    int32_t dtype_out;       /* ris_dtype of out                               */
    int32_t batch;           /* B sequences (B * Hkv <= 65535)                  */
    int32_t Hq;              /* query heads                                    */
    int32_t Hkv;             /* KV heads; G = Hq / Hkv <= 8                     */
    int32_t D;               /* head dimension: 64 or 128                      */
    int64_t max_len;         /* cache capacity per (sequence, kv head)         */
    int64_t anchor_stride;   /* anchor entries reserved per sequence           */
    int32_t window;          /* local window L (>= 0; 0 = none)                */
    int32_t sink;            /* initial tokens A (>= 0; 0 = none)               */
    float   scale;           /* score scale; 0 = 1 / sqrt(D)                    */
} ris_decode_desc;

/* Bytes of device workspace ris_decode_attn needs for the descriptor (host
 * only; negative ris_status on a bad descriptor). */
int64_t ris_decode_workspace_bytes(const ris_decode_desc* desc);

/*
 * out[b, h, :] = sum_{j in I_b,g} softmax_j(scale <Q[b,h], K[b,g,j]>) V[b,g,j],
 * g = floor(h / G), t = pos[b],
 * I_b,g = unique({j in anchor row (b, g) : j <= t} U [max(0, t - L + 1), t]
 *                U [0, min(A, t + 1))).
 *
 * Q, out: device [B, Hq, D].  K, V: device [B, Hkv, max_len, D] caches that
 * already hold the token at position pos[b].  pos: device int64[B].
 * anchor_ptr: device int64[B * (Hkv + 1)]; sequence b's anchor is a CSR of
 * Hkv rows with offsets anchor_ptr[b*(Hkv+1) .. b*(Hkv+1)+Hkv] into its slice
 * anchor_idx[b*anchor_stride .. (b+1)*anchor_stride) -- exactly what
 * ris_mask_build_rows(desc, t0, 1, ...) writes into those two slices.
 * workspace: device memory of at least ris_decode_workspace_bytes(desc)
 * bytes (RIS_E_CAPACITY otherwise); its contents need no initialisation.
 * Reads stay inside the buffers as described whatever the device data hold:
 * offsets are clipped to [0, anchor_stride], anchor entries outside
 * [0, t] are ignored, and a sequence whose pos lies outside [0, max_len)
 * gets zeros, as does an empty set.  Accumulation is float32; the softmax
 * weights enter the PV product rounded to bf16.
 */
int ris_decode_attn(const void* Q, const void* K, const void* V, const int64_t* pos,
                    const int64_t* anchor_ptr, const int32_t* anchor_idx, void* out,
                    void* workspace, int64_t workspace_bytes, const ris_decode_desc* desc,
                    void* stream);

/*
 * ris_decode_attn for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same step, with no workspace argument.  The partials live in a
 * library-owned device array of RIS_DECODE_STATIC_BYTES per GPU, created
 * with the library's code on that GPU and held until the process ends; the
 * call itself allocates nothing.  Returns RIS_E_CAPACITY, launching nothing,
 * when ris_decode_workspace_bytes(desc) exceeds RIS_DECODE_STATIC_BYTES.
 * Every call on one GPU uses that GPU's one array: calls that may overlap in
 * time on the same GPU (unordered streams, several host threads) race on it
 * and must not be made; calls ordered on one stream are safe.  Its contents
 * need no initialisation (every partial is written before it is read).
 * Arguments and results otherwise as ris_decode_attn.
 */
#define RIS_DECODE_STATIC_BYTES (32ll << 20)
int ris_decode_attn_static(const void* Q, const void* K, const void* V, const int64_t* pos,
                           const int64_t* anchor_ptr, const int32_t* anchor_idx, void* out,
                           const ris_decode_desc* desc, void* stream);

/* ------------------------------------------------------------------------ */
/* Host-model layers for a model-level prefill                               */
/* ------------------------------------------------------------------------ */

/*
 * The host models' normalisation, not part of the method (the paper replaces
 * only the attention kernel and leaves weights and every other component
 * untouched; Methods, opening of "The RIS Implementation").  Row-major [rows, cols] tensors of element type dtype
 * (ris_dtype); weight has cols entries.  With residual != NULL:
 * r = x + residual, residual <- r (rounded to dtype), out = rmsnorm(r);
 * otherwise out = rmsnorm(x).  rmsnorm(r) = r / sqrt(mean(r^2) + eps) * weight,
 * in float32 with one rounding at the store.  out may alias x.
 */
int ris_rmsnorm(const void* x, void* residual, const void* weight, void* out, int64_t rows,
                int64_t cols, float eps, int32_t dtype, void* stream);

/*
 * The SwiGLU activation of the host models' MLP: gate_up is [rows, 2*inter]
 * (gate in the first inter columns, up in the rest), out is [rows, inter] with
 * out = silu(gate) * up, silu(g) = g / (1 + exp(-g)), in float32.
 */
int ris_swiglu(const void* gate_up, void* out, int64_t rows, int64_t inter, int32_t dtype, void* stream);

/* Human-readable name of a ris_status (static string, never NULL). */
const char* ris_status_string(int status);

/* Library ABI version: (major << 16) | minor.  2.0 added window and anchor to
 * ris_mask_desc; 2.1 added the row-range build and the decode step; 2.2 the
 * host-model layers (RMSNorm, SwiGLU); 2.3 the strided rotation
 * ris_rope_from; 2.4 changed the draws' round function (the same descriptor
 * now yields different, equally distributed sets). */
int ris_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RIS_H */
