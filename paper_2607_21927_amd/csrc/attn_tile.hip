// Sparse attention, tiled form: one workgroup per (kv_head g, 32 consecutive
// query rows), two wavefronts per query head of the GQA group (one per half
// of the 32 rows).
//
// When a row's unified set covers a sizeable share of its keys (a 70-seed
// ensemble at 1% reaches ~50%), the sets of 32 neighbouring rows together
// touch nearly every key block, so the work is a dense contraction under a
// mask.  For every key block (kKeys keys: 96 at D = 128, 128 at D = 64, the
// most that double-buffered K/V and a triple-buffered bias fit in LDS) the
// workgroup
//   1. stages K[g, block] and V[g, block] in LDS, row-major, once for all
//      32 rows x G heads (double-buffered: block kb+1 is staged while block
//      kb is computed, one workgroup barrier per block);
//   2. turns each row's CSR entries that fall in the block into a score
//      bias in LDS, 0 at the row's keys and -inf elsewhere (windows of 64
//      entries from the row's cursor, enough to cover kKeys entries, the
//      rows being ascending and unique);
//   3. per wave (head h, 16 rows): S^T = bias + K_blk Q^T on MFMA (16x16x32
//      bf16; the bias is the initial accumulator, so masking costs no
//      vector instructions), one online-softmax update per query over the
//      block, and O^T += V_blk^T P^T on MFMA with P kept in registers and V^T
//      read from the row-major block with the LDS transpose read
//      (ds_read_b64_tr_b16); the row sums of P come from the same product
//      with an all-ones A operand, so numerator and denominator use the
//      same bf16 weights.
// In both products lane l holds query l % 16 (keys or dims 4 (l/16) + i of
// each 16-wide tile), so the rescale needs no exchange and a query's running
// max lives in four lanes (permlane swaps combine them).  The reference max
// moves only when a block's max exceeds it by more than kSlack (log2 units),
// so rescales of O are rare.  Every index of a row's set enters one
// normalisation (Pre-Fusion Unified Softmax; Methods, "Hybrid Anchor and
// Pre-Fusion Unified Softmax").  In Structural mode the block clique is the
// diagonal key block: the dense local tile runs on MFMA in the same softmax
// state as the sampled global keys.
//
// 2G waves of at most ~150 VGPRs sit three or four to a SIMD: the MFMA work
// of one wave overlaps the softmax of another.
#include "ris_device.h"
#include "ris_internal.h"

namespace ris {
namespace {

constexpr float kSlack = 8.0f;

template <int D, int G, int kKeys>
__global__ __launch_bounds__(128 * G) void k_attn_tile16(AttnParams a, float c) {
    static_assert(kKeys % 32 == 0 && kKeys <= 128, "key blocks of 32-key steps, at most two CSR windows");
    constexpr int KT = kKeys / 16;                   // 16-key tiles of a block
    constexpr int KU = kKeys / 32;                   // 32-key steps of the PV product
    constexpr int WN = (kKeys + 63) / 64;            // 64-entry CSR windows per row
    constexpr int NW = 2 * G;                        // waves: (head, row half)
    constexpr int NT = 64 * NW;
    constexpr int KS = D + 16;          // K row stride in LDS (bf16 elements)
    constexpr int VS = D + 16;         // V row stride: the 4 rows a 16-lane transpose read
                                       // touches start 8 banks apart
    constexpr int BS = kKeys + 4;      // bias row stride (floats)
    constexpr int RPW = (kTileRows + NW - 1) / NW;       // bias rows per wave
    constexpr int KSL = D / 32;                      // k-steps of the score product
    constexpr int DT = D / 16;                       // 16-dim tiles of the output
    constexpr int PIECES = kKeys * (D / 8);          // 16-byte pieces of a K (or V) block
    constexpr int PPT = (PIECES + NT - 1) / NT;      // per thread
    // Double-buffered: block kb+1 is staged while block kb is computed.
    __shared__ __align__(16) uint16_t Ks_[2][kKeys * KS];
    __shared__ __align__(16) uint16_t Vs_[2][kKeys * VS];
    // Score bias per (row, key) of a block: 0 for the row's entries, -inf
    // elsewhere; it is the initial accumulator of the score product.  Three
    // buffers: block kb+1's is written while block kb's is read, and block
    // kb+2's is reset to -inf (its last reader was block kb-1, before the
    // previous barrier).
    __shared__ __align__(16) float bias_[3][kTileRows * BS];
    __shared__ int64_t rstart_s[kTileRows];
    __shared__ int32_t rlen_s[kTileRows];
    __shared__ int32_t kb_range[2];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int hh = w >> 1, rh = w & 1;               // head of the group, row half
    const int64_t N = a.N;
    const int64_t tiles = (N + kTileRows - 1) / kTileRows;
    const int64_t bid = blockIdx.x;
    const int64_t tile = tiles - 1 - bid / a.Hkv;     // late (heavy) tiles first
    const int g = (int)(bid % a.Hkv);
    const int64_t q0 = tile * kTileRows;
    const int h = g * G + hh;
    const int qr = 16 * rh + li;                     // this lane's query row in the tile
    const uint16_t* Kg = static_cast<const uint16_t*>(a.K) + (int64_t)g * N * D;
    const uint16_t* Vg = static_cast<const uint16_t*>(a.V) + (int64_t)g * N * D;
    if (!tile_is_dense(a, g, q0)) return;   // a sparse tile belongs to the gather kernel

    // ---- per-row CSR extents, bias buffers at -inf
    for (int i = tid; i < 3 * kTileRows * BS; i += NT) (&bias_[0][0])[i] = -INFINITY;
    if (tid < kTileRows) {
        const int64_t q = q0 + tid;
        int64_t s = 0, L = 0;
        if (q < N) {
            s = a.row_ptr[g * N + q];
            L = a.row_ptr[g * N + q + 1] - s;
            if (s < 0 || L < 0) { s = 0; L = 0; }   // an incomplete build's rows: empty
        }
        rstart_s[tid] = s;
        rlen_s[tid] = (int)L;
    }
    __syncthreads();
    // Key-block range touched by any row: first and last entries of each row.
    if (w == 0) {
        int lo = 0x7FFFFFFF, hi = -1;
        if (lane < kTileRows && rlen_s[lane] > 0) {
            const int64_t nb = (N - 1) / kKeys;
            int64_t f = a.col_idx[rstart_s[lane]] / kKeys;
            int64_t l = a.col_idx[rstart_s[lane] + rlen_s[lane] - 1] / kKeys;
            f = f < 0 ? 0 : (f > nb ? nb : f);
            l = l < 0 ? 0 : (l > nb ? nb : l);
            lo = (int)f;
            hi = (int)l;
        }
        for (int off = 32; off > 0; off >>= 1) {
            lo = min(lo, __shfl_xor(lo, off));
            hi = max(hi, __shfl_xor(hi, off));
        }
        if (lane == 0) { kb_range[0] = lo; kb_range[1] = hi; }
    }

    // ---- this lane's query row of Q_h as the B operand: dims 32 ks + 8 (l/16) ..
    u32x4_t qf[KSL];
    {
        const int64_t q = q0 + qr;
        const uint16_t* Qrow = static_cast<const uint16_t*>(a.Q) + ((int64_t)h * N + (q < N ? q : 0)) * D;
        const u32x4_t zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int ks = 0; ks < KSL; ++ks) {
            const u32x4_t v = *reinterpret_cast<const u32x4_t*>(Qrow + 32 * ks + 8 * lg);
            qf[ks] = q < N ? v : zero;
        }
    }
    float m_run = -INFINITY;   // reference max of this lane's query, log2 domain (scores x c)
    f32x4_t o[DT];
    // Row sums of P on the matrix unit: an all-ones A operand makes every
    // output row of lsum the sum over keys of this lane's query.
    f32x4_t lsum = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const u32x4_t ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    __syncthreads();

    // Rows whose bias this wave writes: r = w + NW*i.
    int64_t rst[RPW];
    int rln[RPW], cur[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        // the wave's rows: uniform values, kept in scalar registers so that
        // the window addresses are scalar arithmetic
        const int r = w + NW * i;
        const int64_t st = r < kTileRows ? rstart_s[r] : 0;
        rst[i] = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(st >> 32)) << 32) |
                           (uint32_t)__builtin_amdgcn_readfirstlane((int)st));
        rln[i] = __builtin_amdgcn_readfirstlane(r < kTileRows ? rlen_s[r] : 0);
        cur[i] = 0;
    }
    const int kb_lo = kb_range[0], kb_hi = kb_range[1];

    // ---- register staging of one block (K and V pieces, CSR windows)
    u32x4_t kreg[PPT], vreg[PPT];
    int wreg[RPW];
    auto load_kv = [&](int kb) {
        const int k0 = kb * kKeys;
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * NT;
            const int key = e / (D / 8), ch = e % (D / 8);
            const int64_t j = min(k0 + key, (int)N - 1);   // rows past N are masked out
            if (PIECES % NT == 0 || e < PIECES) {
                kreg[u] = *reinterpret_cast<const u32x4_t*>(Kg + j * D + ch * 8);
                vreg[u] = *reinterpret_cast<const u32x4_t*>(Vg + j * D + ch * 8);
            }
        }
    };
    // The first 64-entry window from each row's cursor is prefetched a block
    // ahead; a block with more entries than that (only when the row's set
    // is denser than 64 per kKeys keys) reads the rest when it is staged.
    auto load_windows = [&]() {
#pragma unroll
        for (int i = 0; i < RPW; ++i)
            wreg[i] = lane < rln[i] - cur[i] ? (a.col_idx + (rst[i] + cur[i]))[lane] : -1;
    };

    // Stage block kb (its K/V pieces are in kreg/vreg, its CSR windows in
    // wreg) into LDS buffer p, with its bias.
    auto stage = [&](int kb, int p, float* bias) {
        const int64_t k0 = (int64_t)kb * kKeys;
        uint16_t* Ks = Ks_[p];
        uint16_t* Vs = Vs_[p];
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * NT;
            if (PIECES % NT == 0 || e < PIECES) {
                const int key = e / (D / 8), ch = e % (D / 8);
                *reinterpret_cast<u32x4_t*>(&Ks[key * KS + ch * 8]) = kreg[u];   // rows past N: masked
                u32x4_t v = vreg[u];
                if (k0 + kKeys > N && k0 + key >= N) v = u32x4_t{0u, 0u, 0u, 0u};   // V rows past N read as zeros
                *reinterpret_cast<u32x4_t*>(&Vs[key * VS + ch * 8]) = v;
            }
        }
        const int k0i = kb * kKeys;
        const uint32_t lim = (uint32_t)min(kKeys, (int)N - k0i);   // keys of the block inside [0, N)
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int r = w + NW * i;
            if (r < kTileRows) {
                // the window starts at the row's first unconsumed entry, so every
                // valid entry is >= k0i; empty lanes hold -1
                int taken = 0;
                int wv = wreg[i];
#pragma unroll
                for (int x = 0; x < WN; ++x) {
                    const uint32_t d = (uint32_t)(wv - k0i);
                    const bool inb = d < lim;
                    const uint64_t bal = __ballot(inb);
                    if (inb) bias[r * BS + d] = 0.f;
                    taken += __popcll(bal);
                    // the rows are ascending: unless the whole window lay in
                    // the block, the block's entries end inside it
                    if (x + 1 == WN || bal != ~0ull) break;
                    const int pos = cur[i] + taken + lane;
                    wv = pos < rln[i] ? a.col_idx[rst[i] + pos] : -1;
                }
                cur[i] += taken;
            }
        }
    };

    if (kb_lo <= kb_hi) {
        load_kv(kb_lo);
        load_windows();
        stage(kb_lo, kb_lo & 1, bias_[kb_lo % 3]);
        if (kb_lo < kb_hi) {
            load_kv(kb_lo + 1);
            load_windows();
        }
    }
    __syncthreads();
    // One barrier per block: at iteration kb the workgroup stages block kb+1
    // into the other buffer (last read during iteration kb-1, before the
    // previous barrier) and computes block kb (staged before it).
    int b3 = kb_lo % 3;                  // bias buffer of block kb
    for (int kb = kb_lo; kb <= kb_hi; ++kb) {
        const int p = kb & 1;
        const int b3n = b3 == 2 ? 0 : b3 + 1, b3c = b3n == 2 ? 0 : b3n + 1;
        {
            // reset block kb+2's bias buffer
            float* bc = bias_[b3c];
            for (int e = tid; e < kTileRows * (kKeys / 4); e += NT) {
                const int r = e / (kKeys / 4), c4 = e % (kKeys / 4);
                *reinterpret_cast<f32x4_t*>(&bc[r * BS + 4 * c4]) = f32x4_t{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
            }
        }
        if (kb < kb_hi) {
            stage(kb + 1, p ^ 1, bias_[b3n]);
            if (kb + 1 < kb_hi) {
                load_kv(kb + 2);
                load_windows();
            }
        }
        const uint16_t* Ks = Ks_[p];
        const uint16_t* Vs = Vs_[p];
        const float* bias = bias_[b3];
        b3 = b3n;
        {
            // Every block of the range is computed: at the union densities the
            // tiled kernel takes, a key block with no entry in any of the
            // 32 rows is rare, and a fully masked block adds exact zeros.
            // ---- S^T[key, query] = K_blk Q_h^T; st[kt][i] is key 16 kt + 4 (l/16) + i
            f32x4_t st[KT];
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
                st[kt] = *reinterpret_cast<const f32x4_t*>(&bias[qr * BS + 16 * kt + 4 * lg]);
#pragma unroll
                for (int ks = 0; ks < KSL; ++ks) {
                    const u32x4_t av = *reinterpret_cast<const u32x4_t*>(&Ks[(16 * kt + li) * KS + 32 * ks + 8 * lg]);
                    st[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av), as_bf16x8(qf[ks]), st[kt],
                                                                      0, 0, 0);
                }
            }
            // ---- mask, one online-softmax step for this lane's query
            float mx = -INFINITY;
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, st[kt][i]);
            // The reference max moves only when the block's max exceeds it by
            // more than kSlack (log2 units): weights stay below 2^kSlack, and
            // numerator and denominator share every rescale, so the result is
            // the same up to rounding while rescales become rare.
            const float mxc = quad_max16(mx) * c;
            const bool move = mxc > m_run + kSlack;
            const float m_new = move ? mxc : m_run;
            const float mc = m_new == -INFINITY ? 0.f : m_new;
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) st[kt][i] = __builtin_amdgcn_exp2f(fmaf(st[kt][i], c, -mc));
            if (__ballot(move) != 0ull) {
                const float corr = __builtin_amdgcn_exp2f(m_run - mc);   // 0 on a query's first entries
                lsum *= corr;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) o[dt] *= corr;
            }
            m_run = m_new;
            // ---- P^T as the B operand: 32-key step u holds keys 32u + 4 (l/16) + i
            // (slots 0..3) and 32u + 16 + 4 (l/16) + i (slots 4..7)
            u32x4_t pb[KU];
#pragma unroll
            for (int u = 0; u < KU; ++u)
                pb[u] = u32x4_t{pack_bf16x2(st[2 * u][0], st[2 * u][1]), pack_bf16x2(st[2 * u][2], st[2 * u][3]),
                                pack_bf16x2(st[2 * u + 1][0], st[2 * u + 1][1]),
                                pack_bf16x2(st[2 * u + 1][2], st[2 * u + 1][3])};
            // ---- O^T[d, query] += V_blk^T P^T: lane l addresses key row l/4
            // (then 16 + l/4) of the step at dims 16 dt + 4 (l%4)
#pragma unroll
            for (int u = 0; u < KU; ++u) {
                const uint16_t* v_lo = &Vs[(32 * u + (lane >> 2)) * VS + 4 * (lane & 3)];
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const uint2 lo = lds_read_tr16(v_lo + 16 * dt);
                    const uint2 hi = lds_read_tr16(v_lo + 16 * VS + 16 * dt);
                    const u32x4_t av = {lo.x, lo.y, hi.x, hi.y};
                    o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av), as_bf16x8(pb[u]), o[dt], 0, 0, 0);
                }
                lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ones), as_bf16x8(pb[u]), lsum, 0, 0, 0);
            }
        }
        __syncthreads();
    }

    // ---- normalise and store: o[dt][i] is dim 16 dt + 4 (l/16) + i of the query
    const float l_run = lsum[0];
    const int64_t q = q0 + qr;
    if (q < N) {
        const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
        const int64_t base = ((int64_t)h * N + q) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = 16 * dt + 4 * lg;
            const float v0 = o[dt][0] * inv, v1 = o[dt][1] * inv;
            const float v2 = o[dt][2] * inv, v3 = o[dt][3] * inv;
            if (a.out_bf16) {
                *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + base + d) =
                    make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
            } else {
                *reinterpret_cast<float4*>(static_cast<float*>(a.out) + base + d) =
                    make_float4(v0, v1, v2, v3);
            }
        }
    }
}

template <int D, int G>
hipError_t launch_d_g(const AttnParams& a, float c, hipStream_t st) {
    const int64_t tiles = (a.N + kTileRows - 1) / kTileRows;
    const dim3 grid((unsigned)(tiles * a.Hkv));
    // Larger blocks amortise the per-block work (barrier, max exchange, bias
    // reset, loop overhead) over more keys: 128 keys at D = 64, and 96 at
    // D = 128, where 128 would not fit LDS.
    constexpr int kKeys = D == 64 ? 128 : 96;
    hipLaunchKernelGGL((k_attn_tile16<D, G, kKeys>), grid, dim3(128 * G), 0, st, a, c);
    return hipGetLastError();
}

template <int D>
hipError_t launch_d(const AttnParams& a, float c, hipStream_t st) {
    switch (a.G) {
        case 1: return launch_d_g<D, 1>(a, c, st);
        case 2: return launch_d_g<D, 2>(a, c, st);
        case 3: return launch_d_g<D, 3>(a, c, st);
        case 4: return launch_d_g<D, 4>(a, c, st);
        case 5: return launch_d_g<D, 5>(a, c, st);
        case 6: return launch_d_g<D, 6>(a, c, st);
        case 7: return launch_d_g<D, 7>(a, c, st);
        default: return launch_d_g<D, 8>(a, c, st);
    }
}

}  // namespace

hipError_t launch_attn_tile(const AttnParams& a, hipStream_t st) {
    const float c = a.scale * 1.4426950408889634f;   // scores to the log2 domain
    return a.D == 128 ? launch_d<128>(a, c, st) : launch_d<64>(a, c, st);
}

}  // namespace ris
