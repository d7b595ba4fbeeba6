// Geometry kernels: per-row key sets of the seed ensemble, emitted as CSR.
//
// Each row (kv_head, q) is built by one workgroup.  The row's pool is a
// bitmap in LDS; every (seed, draw) pair of the ensemble is spread over the
// 256 lanes, each lane evaluates the keyed permutation and ORs its key into
// the bitmap.
// The bitmap *is* the union over seeds (the paper merges every seed into one
// master set and discards the seed; Methods, "Memory-Bounded Geometry
// Generation"), and reading it in word order yields the row ascending and
// without duplicates (the unique() merge; Methods, "Hybrid Anchor and
// Pre-Fusion Unified Softmax").
//
// Two-pass build: the count pass writes each row's size (popcount) to
// row_ptr[r + 1], a single-workgroup scan turns sizes into offsets, and the
// fill pass regenerates the bitmap and places every key by a block-wide prefix
// over word popcounts; rows are launched in descending q (their cost grows
// with q) so the heavy rows start first.  One-pass build (col_idx sized from
// the closed-form bound): a persistent grid builds every bitmap once and
// finds each row's offset by a decoupled look-back (see k_mask_fused).
#include "ris_device.h"
#include "ris_internal.h"
#include "lookback.h"

namespace ris {
namespace {

constexpr int kThreads = 256;
constexpr int kSeedBatch = 256;  // row words of this many seeds live in LDS at once
// A lane's slice of a batch, ceil(seeds * draws / kThreads) draws, is then at
// most one seed's draws long: it spans at most one seed boundary.
static_assert(kSeedBatch <= kThreads, "a lane's slice of a batch must not exceed one seed's draws");

// LDS words of the seed batch's row words: a batch never holds more than
// min(n_seeds, kSeedBatch) seeds.
__host__ __device__ __forceinline__ int64_t rks_words(const MaskParams& p) {
    return (int64_t)(p.n_seeds < kSeedBatch ? p.n_seeds : kSeedBatch) * kRowWords;
}

// Bitmap words of the largest pool of the built rows: q0 + nq keys (causal)
// or N.
__host__ __device__ __forceinline__ int64_t bitmap_words(const MaskParams& p) {
    const int64_t span = p.causal ? p.q0 + p.nq : p.N;
    return (span + 31) / 32;
}

struct RowGeom {
    uint32_t pool;          // draw pool [0, pool)
    uint32_t draws;         // keys per seed
    uint32_t clique_start;  // Structural clique [clique_start, q]
    uint32_t clique_len;
};

__device__ __forceinline__ RowGeom row_geometry(const MaskParams& p, int64_t q) {
    RowGeom g;
    if (p.mode == 0) {
        const int64_t n = p.causal ? q + 1 : p.N;
        g.pool = (uint32_t)n;
        g.draws = (uint32_t)row_count(p.ppm, n);
        g.clique_start = 0;
        g.clique_len = 0;
    } else {
        const int64_t start = (q / p.block) * (int64_t)p.block;
        const int64_t clique = q - start + 1;
        const int64_t k = row_count(p.ppm, q + 1);
        int64_t kg = k - clique;
        if (kg < 0) kg = 0;
        if (kg > start) kg = start;
        g.pool = (uint32_t)start;
        g.draws = (uint32_t)kg;
        g.clique_start = (uint32_t)start;
        g.clique_len = (uint32_t)clique;
    }
    return g;
}

// Seed index s and draw index j of flat index idx = s * draws + j (idx < 2^24,
// so the float quotient is off by at most one and is corrected).
__device__ __forceinline__ void split_draw(uint32_t idx, uint32_t draws, float inv_draws, int& s, int& j) {
    s = (int)((float)idx * inv_draws);
    j = (int)idx - s * (int)draws;
    if (j < 0) { --s; j += (int)draws; }
    if (j >= (int)draws) { ++s; j -= (int)draws; }
}


// One lane's share of the batch's (seed, draw) pairs, OR-ed into the bitmap.
// Lane t takes the contiguous flat indices [t per, (t+1) per) (flat index =
// seed * draws + draw) and works through them with two walkers held in the
// low and high 16-bit halves of the same registers, so that one packed round
// advances both: walker A takes the lane's draws from the front, walker B
// from the back, until they meet; the lane ends when its last draw is done
// rather than when the slower of two fixed halves is.  A walker's seed -- and
// the round keys it holds -- changes at most a few times per batch.  Each
// walker moves one permutation step per iteration: a walker whose value lands
// in the pool emits it and starts its next draw at once, so cycle walks of
// different lengths do not hold the wave at the slowest lane.  Every walk
// returns to the pool within the domain size (the cycle through j < n returns
// to j), and every iteration advances an unfinished draw, so (slice length)
// * size iterations bound the loop; the bound, from the longest slice, is
// the same in every lane, so the counter lives in scalar registers.
template <int ROUNDS>
__device__ __forceinline__ void walk_draws(const FeistelDomain& dom, const uint32_t* rks,
                                           uint32_t* bits, uint32_t total, uint32_t draws,
                                           float inv_draws) {
    const uint32_t per = (total + kThreads - 1) / kThreads;
    const uint32_t lo = threadIdx.x * per;
    const uint32_t hi = min(lo + per, total);
    if (lo >= hi) return;
    // Walker A takes the lane's draws from the front, walker B from the back;
    // iA and iB are the flat indices they hold (iB = hi when B never starts),
    // and a walker is done when its next index is the other's.
    bool actA = true, actB = hi - lo >= 2;
    uint32_t iA = lo, iB = actB ? hi - 1u : hi;
    int sA = 0, jA = 0, sB = 0, jB = 0;
    split_draw(lo, draws, inv_draws, sA, jA);
    if (actB) split_draw(hi - 1, draws, inv_draws, sB, jB);
    uint32_t KM[ROUNDS], KX[ROUNDS];
    auto key = [&](int s, int r) -> uint32_t {
        return r < kRowWords ? rks[s * kRowWords + r] : (rks[s * kRowWords + r - kRowWords] ^ kKeyTweak);
    };
    auto load_A = [&]() {
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) {
            const uint32_t k = key(sA, r);
            KM[r] = (KM[r] & 0xFFFF0000u) | (k >> 16) | 1u;
            KX[r] = (KX[r] & 0xFFFF0000u) | (k & 0xFFFFu);
        }
    };
    auto load_B = [&]() {
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) {
            const uint32_t k = key(sB, r);
            KM[r] = (KM[r] & 0xFFFFu) | (k & 0xFFFF0000u) | 0x10000u;
            KX[r] = (KX[r] & 0xFFFFu) | (k << 16);
        }
    };
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) { KM[r] = 0x00010001u; KX[r] = 0u; }
    load_A();
    if (actB) load_B();
    const uint32_t b = dom.b, mb = (1u << b) - 1u, n = dom.n;
    const u16x2_t sh_a = {(unsigned short)(16u - dom.a), (unsigned short)(16u - dom.a)};
    const u16x2_t sh_b = {(unsigned short)(16u - b), (unsigned short)(16u - b)};
    uint32_t xA = (uint32_t)jA, xB = (uint32_t)jB;
    // per >= hi - lo, and per and the domain size are the same in every lane.
    const uint64_t max_it = (uint64_t)per * dom.size;
    for (uint64_t it = 0; it < max_it; ++it) {
        uint32_t L = (xA >> b) | ((xB >> b) << 16);
        uint32_t R = (xA & mb) | ((xB & mb) << 16);
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) feistel_round_x2(L, R, KM[r], KX[r], (r & 1) ? sh_b : sh_a);
        xA = ((L & 0xFFFFu) << b) | (R & 0xFFFFu);
        xB = ((L >> 16) << b) | (R >> 16);
        if (actA && xA < n) {
            atomicOr(&bits[xA >> 5], 1u << (xA & 31u));
            if (iA + 1u == iB) {
                actA = false;
            } else {
                ++iA;
                if (++jA == (int)draws) {
                    jA = 0;
                    ++sA;
                    load_A();
                }
                xA = (uint32_t)jA;
            }
        }
        if (actB && xB < n) {
            atomicOr(&bits[xB >> 5], 1u << (xB & 31u));
            if (iB - 1u == iA) {
                actB = false;
            } else {
                --iB;
                if (jB == 0) {
                    jB = (int)draws;
                    --sB;
                    load_B();
                }
                --jB;
                xB = (uint32_t)jB;
            }
        }
        if (!actA && !actB) break;
    }
}

// The same walk for domains of at most 16 bits (pools of at most 65536 keys,
// fewer than 65536 draws per seed): both walkers' values share one register
// X, A in the low and B in the high 16 bits, so the split into halves and the
// recombination after the rounds are one or two packed instructions each.  J
// holds the two walkers' draw indices within their seeds the same way.  rem
// counts the lane's draws that neither walker has started: a walker that
// finishes a draw takes the next one from its end if rem was positive, and
// stops otherwise (rem may go below zero once both have stopped).  A lane's
// slice spans at most one seed boundary (kSeedBatch <= kThreads): a walker
// that crosses it moves into the other walker's seed and copies that walker's
// round keys from the other half of KM and KX.  The set of draws and each
// draw's walk are those of walk_draws, so the bitmap is identical.
// One step of the lane's count of draws not yet started (never negative):
// true when none was left, else the count drops by one.  A single clamped
// subtract does both: its borrow is the branch's lane mask, and the clamp
// keeps an exhausted count at 0, so the other walker stops at its next draw
// too.
__device__ __forceinline__ bool take_last(int& rem) {
    uint64_t borrow;
    asm volatile("v_sub_co_u32 %0, %1, %2, 1 clamp" : "=v"(rem), "=s"(borrow) : "v"(rem));
    return __builtin_amdgcn_inverse_ballot_w64(borrow);
}

// Walker B's step to the previous draw: the high half of J (B's draw
// index) drops by one; true when it was 0, which the subtract's borrow
// reports as the branch's lane mask (the half then reads 0xFFFF).
__device__ __forceinline__ bool step_down_wraps(uint32_t& J) {
    uint64_t borrow;
    asm volatile("v_sub_co_u32 %0, %1, %2, %3" : "=v"(J), "=s"(borrow) : "v"(J), "s"(0x10000u));
    return __builtin_amdgcn_inverse_ballot_w64(borrow);
}

template <int ROUNDS>
__device__ __forceinline__ void walk_draws16(const FeistelDomain& dom, const uint32_t* rks,
                                             uint32_t* bits, uint32_t total, uint32_t draws,
                                             float inv_draws) {
    const uint32_t per = (total + kThreads - 1) / kThreads;
    const uint32_t lo = threadIdx.x * per;
    const uint32_t hi = min(lo + per, total);
    if (lo >= hi) return;
    bool actA = true, actB = hi - lo >= 2;
    int rem = (int)(hi - lo) - (actB ? 2 : 1);
    int sA = 0, jA = 0, sB = 0, jB = 0;
    split_draw(lo, draws, inv_draws, sA, jA);
    if (actB) split_draw(hi - 1, draws, inv_draws, sB, jB);
    else { sB = sA; jB = jA; }
    uint32_t KM[ROUNDS], KX[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
        const uint32_t ka = r < kRowWords ? rks[sA * kRowWords + r] : (rks[sA * kRowWords + r - kRowWords] ^ kKeyTweak);
        const uint32_t kb = r < kRowWords ? rks[sB * kRowWords + r] : (rks[sB * kRowWords + r - kRowWords] ^ kKeyTweak);
        KM[r] = (kb & 0xFFFF0000u) | (ka >> 16) | 0x00010001u;
        KX[r] = (kb << 16) | (ka & 0xFFFFu);
    }
    const uint32_t b = dom.b, mb = (1u << b) - 1u, n = dom.n;
    const uint32_t mb2 = mb | (mb << 16);
    const u16x2_t shx = {(unsigned short)b, (unsigned short)b};
    const u16x2_t sh_a = {(unsigned short)(16u - dom.a), (unsigned short)(16u - dom.a)};
    const u16x2_t sh_b = {(unsigned short)(16u - b), (unsigned short)(16u - b)};
    uint32_t J = (uint32_t)jA | ((uint32_t)jB << 16);
    uint32_t X = J;
    const uint64_t max_it = (uint64_t)per * dom.size;
    for (uint64_t it = 0; it < max_it; ++it) {
        uint32_t L = as_u32(as_u16x2(X) >> shx);
        uint32_t R = X & mb2;
        asm("" : "+v"(L), "+v"(R));
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) feistel_round_x2(L, R, KM[r], KX[r], (r & 1) ? sh_b : sh_a);
        X = as_u32(as_u16x2(L) << shx) | R;
        if (actA && (X & 0xFFFFu) < n) {
            uint32_t w = __builtin_amdgcn_ubfe(X, 5, 11);
            asm("" : "+v"(w));
            atomicOr(&bits[w], 1u << (X & 31u));
            if (take_last(rem)) {
                actA = false;
            } else {
                ++J;
                if ((J & 0xFFFFu) == draws) {
                    J &= 0xFFFF0000u;
#pragma unroll
                    for (int r = 0; r < ROUNDS; ++r) {
                        KM[r] = __builtin_amdgcn_perm(KM[r], KM[r], 0x03020302u);
                        KX[r] = __builtin_amdgcn_perm(KX[r], KX[r], 0x03020302u);
                    }
                }
                X = __builtin_amdgcn_perm(X, J, 0x07060100u);
            }
        }
        if (actB && (X >> 16) < n) {
            uint32_t w = X >> 21;
            asm("" : "+v"(w));
            atomicOr(&bits[w], 1u << ((X >> 16) & 31u));
            if (take_last(rem)) {
                actB = false;
            } else {
                if (step_down_wraps(J)) {
                    // B's draw index was 0 and its half now reads 0xFFFF:
                    // it continues at draws - 1 of the previous seed
                    J -= (0x10000u - draws) << 16;
#pragma unroll
                    for (int r = 0; r < ROUNDS; ++r) {
                        KM[r] = __builtin_amdgcn_perm(KM[r], KM[r], 0x01000100u);
                        KX[r] = __builtin_amdgcn_perm(KX[r], KX[r], 0x01000100u);
                    }
                }
                X = __builtin_amdgcn_perm(J, X, 0x07060100u);
            }
        }
        if (!actA && !actB) break;
    }
}

// Bits [lo, hi) that fall in word w.
__device__ __forceinline__ uint32_t range_bits(uint32_t w, uint32_t lo, uint32_t hi) {
    const uint32_t b0 = w * 32u, b1 = b0 + 32u;
    const uint32_t a = lo > b0 ? lo : b0, e = hi < b1 ? hi : b1;
    if (a >= e) return 0u;
    const uint32_t n = e - a;
    return (n == 32u ? ~0u : ((1u << n) - 1u)) << (a - b0);
}

// Fill `bits` (W words, already visible to the whole block) with the union of
// every seed's draws for row (h, q), on top of the local window and the
// initial-token anchor clipped to the pool (above the pool they lie inside the
// Structural clique, which is emitted as a range of its own).  Ends with a
// block barrier.
__device__ void build_row_bitmap(const MaskParams& p, int64_t q, int h, const RowGeom& g,
                                 uint32_t* rks, uint32_t* bits) {
    const int tid = threadIdx.x;
    const uint32_t W = (g.pool + 31u) >> 5;
    const uint32_t qe = (uint32_t)q + 1u;
    const uint32_t a_hi = min((uint32_t)p.anchor, min(qe, g.pool));
    const uint32_t w_lo = p.window > 0 && (uint32_t)p.window < qe ? qe - (uint32_t)p.window : 0u;
    const uint32_t w_hi = p.window > 0 ? min(qe, g.pool) : 0u;
    for (uint32_t w = tid; w < W; w += kThreads)
        bits[w] = range_bits(w, 0u, a_hi) | range_bits(w, w_lo, w_hi);
    if (g.draws == 0) {
        __syncthreads();
        return;
    }
    const FeistelDomain dom = make_domain(g.pool);
    const float inv_draws = 1.0f / (float)g.draws;
    // Batches keep the flat (seed, draw) index below 2^24 for the float split.
    const int batch = (int)min((uint32_t)kSeedBatch, (1u << 24) / g.draws);
    for (int s0 = 0; s0 < p.n_seeds; s0 += batch) {
        const int sb = min(batch, p.n_seeds - s0);
        __syncthreads();   // bitmap cleared / previous batch's keys no longer read
        // Row words of the batch's seeds, one Philox evaluation per lane.
        for (int t = tid; t < sb; t += kThreads) {
            uint32_t w[kRowWords];
            row_round_keys(p.seed + (uint64_t)(s0 + t), (uint64_t)q, (uint64_t)h, (uint64_t)p.layer, w);
            *reinterpret_cast<u32x4_t*>(&rks[t * kRowWords]) = u32x4_t{w[0], w[1], w[2], w[3]};
            *reinterpret_cast<u32x4_t*>(&rks[t * kRowWords + 4]) = u32x4_t{w[4], w[5], w[6], w[7]};
        }
        __syncthreads();
        const uint32_t total = (uint32_t)sb * g.draws;
        if (dom.size <= 65536u && g.draws < 65536u) {
            if (dom.rounds == 6)
                walk_draws16<6>(dom, rks, bits, total, g.draws, inv_draws);
            else
                walk_draws16<12>(dom, rks, bits, total, g.draws, inv_draws);
        } else {
            walk_draws<6>(dom, rks, bits, total, g.draws, inv_draws);
        }
    }
    __syncthreads();
}

__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* red) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v = wave_sum_u32(v);
    if (lane == 0) red[wid] = v;
    __syncthreads();
    const uint32_t t = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    return t;
}

// Exclusive prefix of v over the block; *total receives the block sum.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* red, uint32_t* total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const uint32_t inc = wave_inclusive_scan(v);
    if (lane == 63) red[wid] = inc;
    __syncthreads();
    uint32_t before = 0;
    for (int w = 0; w < wid; ++w) before += red[w];
    *total = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    return before + inc - v;
}

// Write the row: the set bits of bits[0, W) as keys 32 w + b, ascending, at
// out[0, ..), then the Structural clique; nothing at out[limit] or beyond.
// A lane's keys of one word are contiguous in out, so it writes them four at
// a time with 16-byte stores (global stores need only 4-byte alignment) and
// the last one to three with an 8- and a 4-byte store: the store
// instructions, whose address processing limits this loop, are about a
// quarter of one key per store.
__device__ void emit_row(const uint32_t* bits, uint32_t W, int32_t* out, int64_t limit, const RowGeom& g,
                         uint32_t* red, int64_t count) {
    // The whole row fits below limit in every valid build; the guarded path
    // is for a truncated or inconsistent row_ptr.
    const bool whole = limit >= count;
    uint32_t done = 0;
    for (uint32_t w0 = 0; w0 < W; w0 += kThreads) {
        const uint32_t w = w0 + threadIdx.x;
        uint32_t word = w < W ? bits[w] : 0u;
        uint32_t total;
        const uint32_t pos0 = done + block_exclusive_scan(__popc(word), red, &total);
        const int32_t k0 = (int32_t)(w * 32u);
        auto next_key = [&]() {
            const uint32_t b = (uint32_t)__builtin_ctz(word);   // v_ffbl_b32 (word != 0 here)
            word &= word - 1u;
            return k0 + (int32_t)b;
        };
        // Groups of four keys as 16-byte stores at any 4-byte-aligned position,
        // then the last one to three keys.
        if (whole) {
            int32_t* o = out + pos0;
            for (uint32_t n = __popc(word); n >= 4u; n -= 4u) {
                const int32_t a = next_key(), b = next_key(), c = next_key(), d = next_key();
                *reinterpret_cast<int4*>(o) = make_int4(a, b, c, d);
                o += 4;
            }
            if (__popc(word) >= 2) {
                const int32_t a = next_key(), b = next_key();
                *reinterpret_cast<int2*>(o) = make_int2(a, b);
                o += 2;
            }
            if (word) *o = next_key();
        } else {
            int64_t pos = pos0;
            while (__popc(word) >= 4) {
                const int32_t a = next_key(), b = next_key(), c = next_key(), d = next_key();
                if (pos + 4 <= limit) {
                    *reinterpret_cast<int4*>(out + pos) = make_int4(a, b, c, d);
                } else {
                    if (pos < limit) out[pos] = a;
                    if (pos + 1 < limit) out[pos + 1] = b;
                    if (pos + 2 < limit) out[pos + 2] = c;
                }
                pos += 4;
            }
            if (__popc(word) >= 2) {
                const int32_t a = next_key(), b = next_key();
                if (pos + 2 <= limit) {
                    *reinterpret_cast<int2*>(out + pos) = make_int2(a, b);
                } else if (pos < limit) {
                    out[pos] = a;
                }
                pos += 2;
            }
            if (word) {
                const int32_t k = next_key();
                if (pos < limit) out[pos] = k;
                ++pos;
            }
        }
        done += total;
    }
    for (uint32_t t = threadIdx.x; t < g.clique_len; t += kThreads) {
        const int64_t pos = (int64_t)done + t;
        if (pos < limit) out[pos] = (int32_t)(g.clique_start + t);
    }
}

// Workgroup -> (row r, query q, head h), heavy (late) rows first.
__device__ __forceinline__ void row_of_block(const MaskParams& p, int64_t& r, int64_t& q, int& h) {
    const int64_t i = blockIdx.x;
    const int64_t local = p.nq - 1 - i / p.heads;
    h = (int)(i % p.heads);
    q = p.q0 + local;
    r = (int64_t)h * p.nq + local;
}

__global__ __launch_bounds__(kThreads) void k_mask_count(MaskParams p, int64_t* row_ptr) {
    extern __shared__ __align__(16) uint32_t smem[];
    __shared__ uint32_t red[4];
    uint32_t* rks = smem;
    uint32_t* bits = smem + rks_words(p);
    int64_t r, q; int h;
    row_of_block(p, r, q, h);
    const RowGeom g = row_geometry(p, q);
    build_row_bitmap(p, q, h, g, rks, bits);
    const uint32_t W = (g.pool + 31u) >> 5;
    uint32_t c = 0;
    for (uint32_t w = threadIdx.x; w < W; w += kThreads) c += __popc(bits[w]);
    const uint32_t total = block_sum(c, red);
    if (threadIdx.x == 0) row_ptr[r + 1] = (int64_t)total + g.clique_len;
}

__global__ __launch_bounds__(kThreads) void k_mask_fill(MaskParams p, const int64_t* row_ptr,
                                                        int32_t* col_idx, int64_t capacity) {
    extern __shared__ __align__(16) uint32_t smem[];
    __shared__ uint32_t red[4];
    uint32_t* rks = smem;
    uint32_t* bits = smem + rks_words(p);
    int64_t r, q; int h;
    row_of_block(p, r, q, h);
    const int64_t base = row_ptr[r];
    int64_t limit = row_ptr[r + 1] - base;
    // Never write outside col_idx[0, capacity), whatever row_ptr holds.
    if (base < 0 || limit < 0 || base > capacity) return;
    if (limit > capacity - base) limit = capacity - base;
    const RowGeom g = row_geometry(p, q);
    build_row_bitmap(p, q, h, g, rks, bits);
    const uint32_t W = (g.pool + 31u) >> 5;
    uint32_t c = 0;
    for (uint32_t w = threadIdx.x; w < W; w += kThreads) c += __popc(bits[w]);
    const int64_t count = (int64_t)block_sum(c, red) + g.clique_len;
    emit_row(bits, W, col_idx + base, limit, g, red, count);
}

// ---------------------------------------------------------------------------
// A block-uniform 64-bit value held in scalar registers.
__device__ __forceinline__ int64_t uniform_i64(int64_t v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// One-pass build (count, scan and fill fused), used when col_idx is sized from
// the closed-form bound.  A persistent grid of workgroups takes tickets --
// one or two consecutive rows each, in row order -- and builds each row's
// bitmap once.  A row's offset is
// found by a decoupled look-back over its predecessors' status words, which
// live in row_ptr itself (the protocol and its flags are in lookback.h).  A
// workgroup publishes a row's size as soon as its bitmap is built and keeps
// the bitmap in LDS while it builds the next rows; it looks back for the row's
// offset (64 predecessors per step, one per lane) and writes its keys only
// after up to two more rows, when the predecessors, whose rows were taken
// earlier, have almost always published their sizes.  Every wait ends: a
// row is held only by a running workgroup, and a workgroup waits only for
// rows below the one it resolves, each of which its holder builds and
// publishes after waits for still smaller rows (induction over the rows).
// The wait is bounded anyway (p.spin_limit
// polls): past the bound the row publishes poison and writes nothing, any row
// whose look-back reaches a poisoned prefix does the same, and k_strip_status
// makes the total row_ptr[R] negative, so that an incomplete CSR is reported
// rather than used.  Status words are read and written with relaxed
// agent-scope atomics: they carry the only data exchanged.
__device__ __forceinline__ int64_t status_load(const int64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void status_store(int64_t* p, int64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A row of the one-pass build whose size is published but whose keys are not
// yet written: its bitmap waits in LDS until its offset is known.
struct PendingRow {
    int64_t row;
    int64_t count;
    RowGeom g;
    uint32_t* bits;
};

// Find the offset of row x.row by the decoupled look-back, publish its
// inclusive prefix and write its keys.  Block-wide; starts and ends with every
// thread of the block present.
__device__ void resolve_and_emit(const MaskParams& p, int64_t* row_ptr, int32_t* col_idx, int64_t capacity,
                                 const PendingRow& x, uint32_t* red, int64_t* s_base) {
    namespace lb = lookback;
    if (threadIdx.x < 64) {
        // Wave-wide look-back: lane i reads the status of row j-1-i, so each
        // step covers 64 predecessors.  The step ends at the nearest row whose
        // inclusive prefix is known, once every row before it is ready.
        const int lane = threadIdx.x;
        int64_t prefix = 0;
        bool poisoned = x.row == p.poison_row;   // test hook: as if the wait had given up
        uint32_t spins = 0;
        for (int64_t j = poisoned ? 0 : x.row; j > 0;) {
            const int64_t idx = j - lane;                       // row idx-1's status
            const int64_t v = idx > 0 ? status_load(&row_ptr[idx]) : lb::inclusive(0, false);
            const int first = lb::step_end(__ballot(lb::is_inclusive(v)), __ballot(lb::is_ready(v)));
            if (first < 0) {
                if (spins++ >= p.spin_limit) { poisoned = true; break; }
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            // Lanes before `first` hold single row counts (below 2^32); lane
            // `first` holds an inclusive prefix, or poison.
            int64_t part = (int64_t)wave_sum_u32(lane < first ? (uint32_t)lb::value(v) : 0u);
            if (first < 64) {
                const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, first);
                const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), first);
                const int64_t vf = (int64_t)(((uint64_t)hi << 32) | lo);
                if (lb::is_poisoned(vf)) { poisoned = true; break; }
                part += lb::value(vf);
            }
            prefix += part;
            if (first < 64) break;
            j -= 64;
        }
        if (lane == 0) {
            status_store(&row_ptr[x.row + 1], lb::inclusive(prefix + x.count, poisoned));
            *s_base = poisoned ? -1 : prefix;
        }
    }
    __syncthreads();
    const int64_t base = uniform_i64(*s_base);
    if (base >= 0 && base <= capacity) {
        int64_t limit = x.count;
        if (limit > capacity - base) limit = capacity - base;
        emit_row(x.bits, (x.g.pool + 31u) >> 5, col_idx + base, limit, x.g, red, x.count);
    }
}

// Persistent one-pass build.  Every workgroup takes rows (tickets of
// kRowsPerTicket consecutive rows, in row order) until none is left.  It
// publishes a row's size as soon as the row's
// bitmap is built, but looks back for the row's offset only after building
// kDepth more rows: by then its predecessors have almost always published
// their sizes, so the look-back rarely waits (kDepth = 0: at once).
// kDepth + 1 bitmaps per workgroup rotate through the rows.
template <int kDepth, int kRowsPerTicket>
__global__ __launch_bounds__(kThreads, kDepth == 2 ? 6 : 8) void k_mask_fused(MaskParams p, int64_t* row_ptr,
                                                                             int32_t* col_idx, int64_t capacity) {
    static_assert(kDepth >= 0 && kDepth <= 2, "at most two rows wait for their offsets");
    extern __shared__ __align__(16) uint32_t smem[];
    __shared__ uint32_t red[4];
    __shared__ int64_t s_ticket, s_base;
    namespace lb = lookback;
    uint32_t* rks = smem;
    uint32_t* bitmaps = smem + rks_words(p);
    const int64_t bw = bitmap_words(p);
    const int64_t R = (int64_t)p.heads * p.nq;
    PendingRow q0 = {}, q1 = {};
    int n = 0;
    // Tickets that carry rows; every workgroup takes tickets until one is
    // past them, so T + gridDim.x tickets are taken in all, and the last one
    // restores row_ptr[0] to 0.
    const int64_t T = (R + kRowsPerTicket - 1) / kRowsPerTicket;
    // With two rows per ticket, s_next holds the pair's second row until its
    // turn (R when there is none); thread 0 alone uses it, and it lives in LDS
    // so that no register holds it through the walk.
    __shared__ int64_t s_next;
    if (kRowsPerTicket > 1 && threadIdx.x == 0) s_next = R;
    for (int it = 0;; ++it) {
        if (threadIdx.x == 0) {
            if constexpr (kRowsPerTicket == 1) {
                const int64_t t = (int64_t)atomicAdd(reinterpret_cast<unsigned long long*>(row_ptr), 1ull);
                s_ticket = t;
                if (t == T + (int64_t)gridDim.x - 1) status_store(row_ptr, 0);
            } else if (s_next >= R) {
                const int64_t t = (int64_t)atomicAdd(reinterpret_cast<unsigned long long*>(row_ptr), 1ull);
                if (t == T + (int64_t)gridDim.x - 1) status_store(row_ptr, 0);
                const int64_t first = t < T ? t * kRowsPerTicket : R;
                s_ticket = first;
                s_next = first + 1 < R ? first + 1 : R;
            } else {
                s_ticket = s_next;
                s_next = R;
            }
        }
        __syncthreads();   // also: the bitmap emitted last iteration is no longer read
        const int64_t r = uniform_i64(s_ticket);
        if (r >= R) {
            if (kDepth > 0 && n > 0) resolve_and_emit(p, row_ptr, col_idx, capacity, q0, red, &s_base);
            if (kDepth > 1 && n > 1) resolve_and_emit(p, row_ptr, col_idx, capacity, q1, red, &s_base);
            break;
        }
        PendingRow fresh;
        fresh.row = r;
        fresh.bits = bitmaps + (int64_t)(it % (kDepth + 1)) * bw;
        {
            const int h = (int)(r / p.nq);
            const int64_t q = p.q0 + (r - (int64_t)h * p.nq);
            fresh.g = row_geometry(p, q);
            build_row_bitmap(p, q, h, fresh.g, rks, fresh.bits);
            const uint32_t W = (fresh.g.pool + 31u) >> 5;
            uint32_t c = 0;
            for (uint32_t w = threadIdx.x; w < W; w += kThreads) c += __popc(fresh.bits[w]);
            fresh.count = (int64_t)__builtin_amdgcn_readfirstlane((int)block_sum(c, red)) + fresh.g.clique_len;
            if (threadIdx.x == 0) status_store(&row_ptr[r + 1], lb::aggregate(fresh.count));
        }
        if (kDepth == 0) {
            resolve_and_emit(p, row_ptr, col_idx, capacity, fresh, red, &s_base);
            continue;
        }
        if (n == kDepth) {
            resolve_and_emit(p, row_ptr, col_idx, capacity, q0, red, &s_base);
            if (kDepth > 1) q0 = q1;
            --n;
        }
        if (n == 0) q0 = fresh;
        else q1 = fresh;
        ++n;
    }
}

__global__ void k_fill_i64(int64_t* x, int64_t n, int64_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) x[i] = v;
}

// After the one-pass build: strip the status flags of row_ptr[1 .. R].  A
// poisoned row's entry becomes -1; if any row is poisoned, row_ptr[R] becomes
// -1 as well.  row_ptr[0] is 0 when this runs (the fused kernel's last ticket
// restores it); here it counts finished workgroups (low 32 bits) and poisoned
// ones (high bits), and the last workgroup to finish resets it to 0.
__global__ __launch_bounds__(256) void k_strip_status(int64_t* row_ptr, int64_t R) {
    const int64_t i = 1 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool poison = false;
    if (i <= R) {
        const int64_t v = row_ptr[i];
        poison = lookback::is_poisoned(v);
        row_ptr[i] = lookback::stripped(v);
    }
    const int any = __syncthreads_or(poison);
    if (threadIdx.x == 0) {
        const uint64_t add = 1ull | (any ? (1ull << 32) : 0ull);
        const uint64_t old = __hip_atomic_fetch_add(reinterpret_cast<uint64_t*>(row_ptr), add,
                                                    __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        if ((old & 0xFFFFFFFFull) == (uint64_t)gridDim.x - 1) {
            // every other workgroup has stripped its entries
            if (((old + add) >> 32) != 0) status_store(&row_ptr[R], -1);
            status_store(row_ptr, 0);
        }
    }
}

// In-place inclusive scan of row_ptr[1 .. R] (row sizes -> end offsets);
// row_ptr[0] = 0.  One workgroup walks the array in coalesced chunks.
constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;

__global__ __launch_bounds__(kScanThreads) void k_scan_rows(int64_t* row_ptr, int64_t R) {
    __shared__ int64_t wave_tot[kScanThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    int64_t carry = 0;
    if (tid == 0) row_ptr[0] = 0;
    for (int64_t base = 1; base <= R; base += (int64_t)kScanThreads * kScanItems) {
        int64_t v[kScanItems];
        int64_t run = 0;
#pragma unroll
        for (int e = 0; e < kScanItems; ++e) {
            const int64_t idx = base + (int64_t)tid * kScanItems + e;
            run += idx <= R ? row_ptr[idx] : 0;
            v[e] = run;
        }
        int64_t inc = run;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int64_t t = __shfl_up(inc, off);
            if (lane >= off) inc += t;
        }
        if (lane == 63) wave_tot[wid] = inc;
        __syncthreads();
        int64_t before = carry;
        int64_t chunk = 0;
        for (int w = 0; w < kScanThreads / 64; ++w) {
            if (w < wid) before += wave_tot[w];
            chunk += wave_tot[w];
        }
        before += inc - run;
#pragma unroll
        for (int e = 0; e < kScanItems; ++e) {
            const int64_t idx = base + (int64_t)tid * kScanItems + e;
            if (idx <= R) row_ptr[idx] = before + v[e];
        }
        carry += chunk;
        __syncthreads();
    }
}

size_t mask_smem_bytes(const MaskParams& p, int bitmaps = 1) {
    return (size_t)(rks_words(p) + bitmaps * bitmap_words(p)) * sizeof(uint32_t);
}

// Workgroups per CU below which a deeper one-pass pipeline costs more
// occupancy than its shorter waits gain.
constexpr int kMinResidentRows = 6;
// Expected draws per row below which the one-pass build takes two rows per
// ticket (measured crossover on MI355X between 4,900 and 6,600).
constexpr int64_t kTicketPairDraws = 5000;

template <int kDepth>
hipError_t fused_occupancy(const MaskParams& p, int* blocks) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, k_mask_fused<kDepth, 1>, kThreads,
                                                        mask_smem_bytes(p, kDepth + 1));
}

}  // namespace

hipError_t launch_mask_count(const MaskParams& p, int64_t* row_ptr, hipStream_t st) {
    const int64_t rows = (int64_t)p.heads * p.nq;
    hipLaunchKernelGGL(k_mask_count, dim3((unsigned)rows), dim3(kThreads), mask_smem_bytes(p), st, p,
                       row_ptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan_rows, dim3(1), dim3(kScanThreads), 0, st, row_ptr, rows);
    return hipGetLastError();
}

hipError_t launch_mask_fused(const MaskParams& p, int64_t* row_ptr, int32_t* col_idx,
                             int64_t capacity, hipStream_t st) {
    const int64_t rows = (int64_t)p.heads * p.nq;
    const unsigned eb = (unsigned)((rows + 1 + 255) / 256);
    hipLaunchKernelGGL(k_fill_i64, dim3(eb), dim3(256), 0, st, row_ptr, rows + 1, (int64_t)0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // Persistent: as many workgroups as fit on the device at once, each
    // taking rows until none is left.
    // Pipeline depth: the deepest (at most 2) that keeps at least 6 workgroups
    // resident per CU; else 0 (each row looks back right after its bitmap).
    int dev = 0, cus = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    int depth = 0, per_cu = 0;
    for (int d = 2; d >= 0; --d) {
        int b = 0;
        e = d == 2 ? fused_occupancy<2>(p, &b) : d == 1 ? fused_occupancy<1>(p, &b) : fused_occupancy<0>(p, &b);
        if (e != hipSuccess) return e;
        if (b >= kMinResidentRows || d == 0) {
            depth = d;
            per_cu = b;
            break;
        }
    }
    // Rows per ticket.  One same-address atomic per row caps the build at a
    // row per ~12.5 ns on MI355X whatever the row's work; light rows (expected
    // draws per row, seeds x k at the middle row, below kTicketPairDraws)
    // take two consecutive rows per ticket, which halves that floor.  Heavier
    // rows keep one: a pair's second row publishes its size an iteration
    // later, and the look-backs behind it wait (measured: 32k layer with 10
    // seeds 0.84 -> 0.63 ms with pairs, 64k with 70 seeds 4.93 -> 5.47 ms).
    const int64_t mid = p.q0 + p.nq / 2;
    const int64_t work = (int64_t)p.n_seeds * row_count(p.ppm, p.causal ? mid + 1 : p.N);
    const bool pairs = work < kTicketPairDraws;
    const int64_t tickets = pairs ? (rows + 1) / 2 : rows;
    int64_t grid = (int64_t)(per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1);
    if (grid > tickets) grid = tickets;
    const size_t smem = mask_smem_bytes(p, depth + 1);
    const dim3 g3((unsigned)grid), b3(kThreads);
    if (depth == 2) {
        if (pairs) hipLaunchKernelGGL((k_mask_fused<2, 2>), g3, b3, smem, st, p, row_ptr, col_idx, capacity);
        else hipLaunchKernelGGL((k_mask_fused<2, 1>), g3, b3, smem, st, p, row_ptr, col_idx, capacity);
    } else if (depth == 1) {
        if (pairs) hipLaunchKernelGGL((k_mask_fused<1, 2>), g3, b3, smem, st, p, row_ptr, col_idx, capacity);
        else hipLaunchKernelGGL((k_mask_fused<1, 1>), g3, b3, smem, st, p, row_ptr, col_idx, capacity);
    } else {
        if (pairs) hipLaunchKernelGGL((k_mask_fused<0, 2>), g3, b3, smem, st, p, row_ptr, col_idx, capacity);
        else hipLaunchKernelGGL((k_mask_fused<0, 1>), g3, b3, smem, st, p, row_ptr, col_idx, capacity);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned sb = (unsigned)((rows + 255) / 256);
    hipLaunchKernelGGL(k_strip_status, dim3(sb), dim3(256), 0, st, row_ptr, rows);
    return hipGetLastError();
}

hipError_t launch_mask_fill(const MaskParams& p, const int64_t* row_ptr, int32_t* col_idx,
                            int64_t capacity, hipStream_t st) {
    const int64_t rows = (int64_t)p.heads * p.nq;
    hipLaunchKernelGGL(k_mask_fill, dim3((unsigned)rows), dim3(kThreads), mask_smem_bytes(p), st, p,
                       row_ptr, col_idx, capacity);
    return hipGetLastError();
}

}  // namespace ris
