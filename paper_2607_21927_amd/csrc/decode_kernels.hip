// Hybrid-Anchor decode step: the newest token of each sequence attends to the
// unique merge of its frozen stochastic anchor (the seed-ensemble union of the
// first generated position), its local window and the initial tokens, with
// one softmax per query head (Methods, "Hybrid Anchor and Pre-Fusion Unified
// Softmax").
//
// The key list of a (sequence, kv head) row is virtual and disjoint by
// construction: the anchor entries that fall neither in the window nor in the
// initial-token range, then the window [w_lo, t], then the initial tokens
// below the window.  Reading the three segments in turn is the unique()
// merge without sorting, and no index is visited twice.
//
// Split-K: the list is cut into 32-key tiles dealt round-robin to the P
// waves of the row (4 waves per workgroup), so any row length is covered
// whatever P the host picks.  A wave runs a flash-style pass over its tiles:
//   * S^T = K Q^T on MFMA 16x16x32 bf16, K rows gathered straight from HBM
//     into the A-operand layout (lane: key l%16, 8 dims at 8(l/16)), the G
//     query heads of the group as the 16-wide MFMA dimension;
//   * the online softmax per head (lane l owns head l%16; two cross-lane
//     exchanges per tile for the max);
//   * O += P V on MFMA with P packed to bf16 in registers and V staged
//     row-major in wave-private LDS and read transposed (ds_read_b64_tr_b16).
// The next tile's K/V loads issue before the current tile is computed.  Each
// wave writes its partial (max, sum, unnormalised output); a second kernel
// merges the partials of each (sequence, query head).
#include "ris_device.h"
#include "ris_internal.h"

namespace ris {
namespace {

constexpr int kTileKeys = kDecodeTileKeys;
constexpr float kNegBig = -1e30f;   // finite start of the running max

struct RowSegs {
    int64_t na, nw, ns;   // anchor entries, window keys, initial keys below the window
    int64_t w_lo;         // window [w_lo, t]; initial tokens [0, ns)
    const int32_t* aidx;  // this row's anchor entries
};

// Key of virtual position v of the row, or -1 (an anchor entry already
// covered by the window or the initial range, or v past the end).
__device__ __forceinline__ int64_t key_of(const RowSegs& r, int64_t v) {
    if (v < r.na) {
        const int64_t j = r.aidx[v];
        return (j >= r.ns && j < r.w_lo) ? j : -1;
    }
    v -= r.na;
    if (v < r.nw) return r.w_lo + v;
    v -= r.nw;
    return v < r.ns ? v : -1;
}

template <int D>
struct KVTile {
    u32x4_t k[2][D / 32];
    u32x4_t v[2][D / 32];
    uint32_t valid;       // bit 16 kb + i: key slot 16 kb + i is a real key
};

template <int D>
__device__ __forceinline__ void load_tile(const RowSegs& r, const uint16_t* Kr, const uint16_t* Vr,
                                          int64_t v0, int li, int lg, KVTile<D>& T) {
    uint32_t vm = 0;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int64_t j = key_of(r, v0 + 16 * kb + li);
        vm |= (uint32_t)(__ballot(j >= 0) & 0xFFFFull) << (16 * kb);
        const int64_t jj = j >= 0 ? j : 0;              // row 0 always exists
        const uint16_t* kp = Kr + jj * D + 8 * lg;
        const uint16_t* vp = Vr + jj * D + 8 * lg;
#pragma unroll
        for (int s = 0; s < D / 32; ++s) {
            T.k[kb][s] = *reinterpret_cast<const u32x4_t*>(kp + 32 * s);
            T.v[kb][s] = *reinterpret_cast<const u32x4_t*>(vp + 32 * s);
        }
    }
    T.valid = vm;
}

template <int D>
__global__ __launch_bounds__(64 * kDecodeWaves, 2) void k_decode_partial(DecodeParams p, float c) {
    constexpr int SL = D / 32;         // k-slices of the score product
    constexpr int DB = D / 16;         // 16-dim blocks of the output
    constexpr int VS = D + 16;         // V row stride in LDS (bf16 elements)
    __shared__ __align__(16) uint16_t vlds[kDecodeWaves * kTileKeys * VS];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int row = blockIdx.y;                       // b * Hkv + g
    const int b = row / p.Hkv, g = row - b * p.Hkv;
    const int G = p.G;
    const int64_t part = (int64_t)blockIdx.x * kDecodeWaves + wave;
    uint16_t* vw = vlds + wave * kTileKeys * VS;

    // ---- the row's three segments
    const int64_t t = p.pos[b];
    RowSegs r{0, 0, 0, 0, p.anchor_idx};
    if (t >= 0 && t < p.max_len) {
        const int64_t* ap = p.anchor_ptr + (int64_t)b * (p.Hkv + 1) + g;
        int64_t lo = ap[0], hi = ap[1];
        lo = lo < 0 ? 0 : (lo > p.anchor_stride ? p.anchor_stride : lo);
        hi = hi < lo ? lo : (hi > p.anchor_stride ? p.anchor_stride : hi);
        r.na = hi - lo;
        r.aidx = p.anchor_idx + (int64_t)b * p.anchor_stride + lo;
        r.w_lo = p.window > 0 ? (t - p.window + 1 > 0 ? t - p.window + 1 : 0) : t + 1;
        r.nw = t + 1 - r.w_lo;
        r.ns = p.sink < r.w_lo ? p.sink : r.w_lo;
    }
    const int64_t total = r.na + r.nw + r.ns;
    const int64_t stride = (int64_t)p.parts * kTileKeys;   // this wave's tiles: part, part + P, ...
    const uint16_t* Kr = static_cast<const uint16_t*>(p.K) + (int64_t)row * p.max_len * D;
    const uint16_t* Vr = static_cast<const uint16_t*>(p.V) + (int64_t)row * p.max_len * D;

    // ---- Q^T as the B operand: lane l holds head l%16, dims 32 s + 8 (l/16) ..
    u32x4_t qf[SL];
    {
        const bool hv = li < G;
        const uint16_t* qp = static_cast<const uint16_t*>(p.Q) +
                             ((int64_t)b * p.Hq + (int64_t)g * G + (hv ? li : 0)) * D + 8 * lg;
        const u32x4_t zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const u32x4_t v = *reinterpret_cast<const u32x4_t*>(qp + 32 * s);
            qf[s] = hv ? v : zero;
        }
    }

    f32x4_t o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = kNegBig, l_run = 0.f;

    const int64_t v_first = part * kTileKeys;
    if (v_first < total) {
        KVTile<D> cur;
        load_tile<D>(r, Kr, Vr, v_first, li, lg, cur);
        for (int64_t v0 = v_first; v0 < total; v0 += stride) {
            KVTile<D> nxt;
            const bool more = v0 + stride < total;
            if (more) load_tile<D>(r, Kr, Vr, v0 + stride, li, lg, nxt);

            // V rows into this wave's LDS, row-major (key slot 16 kb + l%16).
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int s = 0; s < SL; ++s)
                    *reinterpret_cast<u32x4_t*>(vw + (16 * kb + li) * VS + 32 * s + 8 * lg) = cur.v[kb][s];

            // S^T = K Q^T: lane l holds head l%16 at key slots 16 kb + 4 (l/16) + i.
            f32x4_t st[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                st[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < SL; ++s)
                    st[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.k[kb][s]),
                                                                      as_bf16x8(qf[s]), st[kb], 0, 0, 0);
            }

            // Online softmax over the tile (scores in the log2 domain).
            float sc[2][4];
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const bool ok = (cur.valid >> (16 * kb + 4 * lg + i)) & 1u;
                    sc[kb][i] = ok ? st[kb][i] * c : -INFINITY;
                    mx = fmaxf(mx, sc[kb][i]);
                }
            mx = quad_max16(mx);
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            float pv[2][4];
            float ps = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[kb][i] = __builtin_amdgcn_exp2f(sc[kb][i] - m_new);
                    ps += pv[kb][i];
                }
            l_run = l_run * alpha + ps;
            m_run = m_new;

            // Rescale the output rows: lane l holds heads 4 (l/16) + i.
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float a = __shfl(alpha, 4 * lg + i);
#pragma unroll
                for (int db = 0; db < DB; ++db) o[db][i] *= a;
            }

            // P as the A operand: head l%16, k slots 8 (l/16) + e hold keys
            // 4 (l/16) + e (e < 4) and 16 + 4 (l/16) + e - 4 (e >= 4).
            const u32x4_t pk = {pack_bf16x2(pv[0][0], pv[0][1]), pack_bf16x2(pv[0][2], pv[0][3]),
                                pack_bf16x2(pv[1][0], pv[1][1]), pack_bf16x2(pv[1][2], pv[1][3])};
            // V as the B operand with the same key order: lane l addresses key
            // row l/4 (then 16 + l/4) at dims 16 db + 4 (l%4).
            const uint16_t* v_lo = vw + (lane >> 2) * VS + 4 * (lane & 3);
            const uint16_t* v_hi = v_lo + 16 * VS;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const uint2 a = lds_read_tr16(v_lo + 16 * db);
                const uint2 e = lds_read_tr16(v_hi + 16 * db);
                const u32x4_t vb = {a.x, a.y, e.x, e.y};
                o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(pk), as_bf16x8(vb), o[db], 0, 0, 0);
            }
            if (more) cur = nxt;
        }
    }

    // ---- this wave's partial
    l_run = quad_sum16(l_run);
    const int64_t slot = (int64_t)row * p.parts + part;
    float* pml = p.part_ml + slot * G * 2;
    if (lane < G) {
        pml[2 * lane] = m_run;
        pml[2 * lane + 1] = l_run;
    }
    float* po = p.part_o + slot * G * D;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = 4 * lg + i;
        if (h < G) {
#pragma unroll
            for (int db = 0; db < DB; ++db) po[h * D + 16 * db + li] = o[db][i];
        }
    }
}

// Merge the partials of one (sequence, query head), one thread per dim: the
// threads first find the common max and each partial's weight together (in
// LDS), then every thread sums its dim over the partials.
template <int D>
__global__ __launch_bounds__(D) void k_decode_combine(DecodeParams p) {
    __shared__ float wgt[kDecodeMaxParts];
    __shared__ float red[D / 64][2];
    const int d = threadIdx.x, lane = d & 63, wv = d >> 6;
    const int64_t bh = blockIdx.x;
    const int b = (int)(bh / p.Hq), h = (int)(bh % p.Hq);
    const int g = h / p.G, hh = h - g * p.G;
    const int64_t row = (int64_t)b * p.Hkv + g;
    const int64_t step_ml = (int64_t)p.G * 2, step_o = (int64_t)p.G * D;
    const float* ml = p.part_ml + row * p.parts * step_ml + 2 * hh;
    const float* po = p.part_o + row * p.parts * step_o + (int64_t)hh * D + d;
    float M = kNegBig;
    for (int i = d; i < p.parts; i += D) M = fmaxf(M, ml[i * step_ml]);
    M = wave_max(M);
    if (lane == 0) red[wv][0] = M;
    __syncthreads();
    M = red[0][0];
#pragma unroll
    for (int w = 1; w < D / 64; ++w) M = fmaxf(M, red[w][0]);
    float L = 0.f;
    for (int i = d; i < p.parts; i += D) {
        const float w = __builtin_amdgcn_exp2f(ml[i * step_ml] - M);
        wgt[i] = w;
        L += w * ml[i * step_ml + 1];
    }
    L = wave_sum(L);
    if (lane == 0) red[wv][1] = L;
    __syncthreads();
    L = red[0][1];
#pragma unroll
    for (int w = 1; w < D / 64; ++w) L += red[w][1];
    float O = 0.f;
#pragma unroll 8
    for (int i = 0; i < p.parts; ++i) O += wgt[i] * po[i * step_o];
    const float y = L > 0.f ? O / L : 0.f;
    const int64_t at = bh * D + d;
    if (p.out_bf16)
        static_cast<uint16_t*>(p.out)[at] = f32_to_bf16(y);
    else
        static_cast<float*>(p.out)[at] = y;
}

template <int D>
hipError_t launch_d(const DecodeParams& p, float c, hipStream_t st) {
    const dim3 grid((unsigned)(p.parts / kDecodeWaves), (unsigned)(p.B * p.Hkv));
    if (p.parts % kDecodeWaves != 0 || p.parts > kDecodeMaxParts) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_decode_partial<D>, grid, dim3(64 * kDecodeWaves), 0, st, p, c);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_decode_combine<D>, dim3((unsigned)((int64_t)p.B * p.Hq)), dim3(D), 0, st, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, hipStream_t st) {
    const float c = p.scale * 1.4426950408889634f;   // scores in the log2 domain
    return p.D == 128 ? launch_d<128>(p, c, st) : launch_d<64>(p, c, st);
}

}  // namespace ris
