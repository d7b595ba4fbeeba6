// Device helpers shared by the RIS kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ris {

// ---------------------------------------------------------------------------
// Counter-based hashing of (seed, layer, kv_head, query) rows.
// ---------------------------------------------------------------------------

// Philox4x64-10 (Salmon et al., SC'11): two 64x64->128 multiplies per round,
// Weyl-sequence key schedule between rounds.
struct Philox4x64Out { uint64_t v[4]; };

__device__ __forceinline__ Philox4x64Out philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                                       uint64_t c3, uint64_t k0, uint64_t k1) {
    constexpr uint64_t kMul0 = 0xD2E7470EE14C6C93ull, kMul1 = 0xCA5A826395121157ull;
    constexpr uint64_t kWeyl0 = 0x9E3779B97F4A7C15ull, kWeyl1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) { k0 += kWeyl0; k1 += kWeyl1; }
        const uint64_t lo0 = kMul0 * c0, hi0 = __umul64hi(kMul0, c0);
        const uint64_t lo1 = kMul1 * c2, hi1 = __umul64hi(kMul1, c2);
        const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    }
    Philox4x64Out o; o.v[0] = c0; o.v[1] = c1; o.v[2] = c2; o.v[3] = c3;
    return o;
}

// The eight 32-bit words of one row (round-key material): the four Philox
// outputs, low word first; key = (seed, 0), counter = (q, kv_head, layer, 0).
constexpr int kRowWords = 8;
__device__ __forceinline__ void row_round_keys(uint64_t seed, uint64_t q, uint64_t kv_head,
                                               uint64_t layer, uint32_t w[kRowWords]) {
    const Philox4x64Out o = philox4x64_10(q, kv_head, layer, 0ull, seed, 0ull);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        w[2 * i] = (uint32_t)o.v[i];
        w[2 * i + 1] = (uint32_t)(o.v[i] >> 32);
    }
}

// ---------------------------------------------------------------------------
// Vector types and register / LDS helpers of the attention kernels.
// ---------------------------------------------------------------------------

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));

// LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane i receives element i mod 4 of what lanes 4e + i/4 (e = 0..3) address;
// so if lane j addresses 4 consecutive dims of key row j/4 at dim offset
// 4 (j mod 4), lane i gets dim i of four consecutive keys.
__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {
    typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;
    const s16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
    return __builtin_bit_cast(uint2, v);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) { return __builtin_bit_cast(bf16x8_t, v); }

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Keyed permutation of [0, n) used for exact-k draws: a Feistel network on
// m-bit words, restricted to [0, n) by cycle walking.  m = max(2,
// bitlen(n - 1)), rounded up to even below 6 bits; left half a = m/2 bits
// (high), right half b = m - a (low); each round replaces the left half, so
// the widths alternate (a, b), (b, a), ...; 6 rounds from 8 bits on, 12
// below.  Round r, key word k (word r, or word r - 8 xor 0x9E3779B9), all on
// 16-bit words: t = R * ((k >> 16) | 1) + (k & 0xFFFF); t ^= t >> 8;
// t *= 0x9E37; the round value is the top |L| bits of t.  Halves never exceed
// 16 bits (m <= 32), so two draws share a register, one per 16-bit half, and
// one packed 16-bit instruction advances both.
struct FeistelDomain {
    uint32_t n;       // pool size (>= 1)
    uint32_t a, b;    // left / right half widths
    uint32_t rounds;  // 6 or 12
    uint32_t size;    // 2^m
};

__host__ __device__ __forceinline__ FeistelDomain make_domain(uint32_t n) {
    uint32_t bits = 0;
    for (uint32_t v = n > 0 ? n - 1 : 0; v; v >>= 1) ++bits;
    if (bits < 2) bits = 2;
    if (bits < 6) bits += bits & 1u;
    FeistelDomain d;
    d.n = n; d.a = bits / 2; d.b = bits - d.a;
    d.rounds = bits >= 8 ? 6u : 12u;
    d.size = 1u << bits;
    return d;
}

constexpr uint32_t kKeyTweak = 0x9E3779B9u;
constexpr unsigned short kMixMul = 0x9E37;

typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u16x2_t as_u16x2(uint32_t v) { return __builtin_bit_cast(u16x2_t, v); }
__device__ __forceinline__ uint32_t as_u32(u16x2_t v) { return __builtin_bit_cast(uint32_t, v); }

// One round on two draws at once.  L and R hold the two draws' half words in
// their low and high 16 bits; km and kx pack the two draws' round multipliers
// ((k >> 16) | 1) and offsets (k & 0xFFFF); shift = 16 - width of L.
__device__ __forceinline__ void feistel_round_x2(uint32_t& L, uint32_t& R, uint32_t km, uint32_t kx,
                                                 u16x2_t shift) {
    u16x2_t t = as_u16x2(R) * as_u16x2(km) + as_u16x2(kx);
    t ^= t >> (u16x2_t){8, 8};
    t *= (u16x2_t){kMixMul, kMixMul};
    t = t >> shift;
    const uint32_t nr = L ^ as_u32(t);
    L = R;
    R = nr;
}

// Count rule: clamp(round_half_up(ppm * n / 1e6), 1, n).
__host__ __device__ __forceinline__ int64_t row_count(int64_t ppm, int64_t n) {
    int64_t k = (ppm * n + 500000) / 1000000;
    if (k < 1) k = 1;
    if (k > n) k = n;
    return k;
}

// ---------------------------------------------------------------------------
// Numeric helpers.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// ---------------------------------------------------------------------------
// Exchanges between the lanes l, l^16, l^32, l^48 (gfx950 permlane swaps).
// ---------------------------------------------------------------------------

// max / sum of x over this lane and the lane 32 away (v_permlane32_swap:
// with both operands x, the two results hold x at lanes l and l^32).
__device__ __forceinline__ float pair_max32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// max / sum of x over the four lanes l, l^16, l^32, l^48 (v_permlane16_swap
// and v_permlane32_swap: with both operands x, lanes l and l^16 -- or l^32 --
// receive the pair {x[l], x[l^16]}).
__device__ __forceinline__ float quad_max16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return pair_max32(fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1])));
}
__device__ __forceinline__ float quad_sum16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return pair_sum32(__uint_as_float(r[0]) + __uint_as_float(r[1]));
}

// ---------------------------------------------------------------------------
// Wavefront (64-lane) reductions via DPP; every lane receives the result.
// ---------------------------------------------------------------------------

// Lanes whose row is disabled by ROW_MASK (or whose source is out of range)
// receive `identity`, so op(v, result) leaves them unchanged.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp(float v, float identity) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(identity), __float_as_int(v),
                                                      CTRL, ROW_MASK, 0xF, false));
}

__device__ __forceinline__ float wave_max(float v) {
    const float id = -INFINITY;
    v = fmaxf(v, dpp<0xB1>(v, id));          // quad_perm [1,0,3,2]
    v = fmaxf(v, dpp<0x4E>(v, id));          // quad_perm [2,3,0,1]
    v = fmaxf(v, dpp<0x141>(v, id));         // row_half_mirror
    v = fmaxf(v, dpp<0x140>(v, id));         // row_mirror: each lane holds its row of 16
    v = fmaxf(v, dpp<0x142, 0xA>(v, id));    // row_bcast:15 into rows 1 and 3
    v = fmaxf(v, dpp<0x143, 0xC>(v, id));    // row_bcast:31 into rows 2 and 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_sum(float v) {
    v += dpp<0xB1>(v, 0.0f);
    v += dpp<0x4E>(v, 0.0f);
    v += dpp<0x141>(v, 0.0f);
    v += dpp<0x140>(v, 0.0f);
    v += dpp<0x142, 0xA>(v, 0.0f);
    v += dpp<0x143, 0xC>(v, 0.0f);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Inclusive prefix sum across the 64 lanes of a wave: Hillis-Steele steps
// within each row of 16 (row_shr, out-of-row sources read 0), then the row
// totals carried by row_bcast:15 (into rows 1 and 3) and row_bcast:31 (into
// rows 2 and 3).
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, true);   // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, true);   // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, true);   // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, true);   // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return v;
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_inclusive_scan(v), 63);
}

}  // namespace ris
