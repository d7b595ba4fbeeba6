// Sparse attention, gather form: one wavefront per (kv_head g, query row q),
// for the 32-row tiles whose union density leaves the tiled kernel idle.
//
// bf16 inputs (k_attn_gather16): the matrix unit does both products.  The
// row's unified index set I(g, q) (CSR) is walked in 32-key tiles; each key
// row of K and V is gathered once for all G query heads of the group (the
// heads are the 16-wide MFMA dimension), one online softmax per head runs
// over the whole set, and the next tile's rows are loaded while the current
// one is computed.  Every index of the set enters the single normalisation
// once (Pre-Fusion Unified Softmax; Methods, "Hybrid Anchor and Pre-Fusion
// Unified Softmax").
//
// float32 inputs (k_attn_gather): vector-unit form.  Chunks of 64 keys:
//   1. scores  -- lane l owns key j_l of the chunk, reads K[g, j_l] once and
//      forms <Q[h, q], K[g, j_l]> for every query head h of the GQA group
//      (the G query rows sit in LDS and are read as broadcasts);
//   2. softmax -- one running (max, sum) per head over the whole set:
//      wavefront max and sum by DPP, rescale of the accumulators when the
//      max grows;
//   3. PV      -- lanes switch to owning D/64 consecutive dimensions; for each
//      key of the chunk the wave reads the value row as one contiguous
//      segment and accumulates p_h * V for all G heads.
// Scores are kept in the log2 domain (scale * log2(e) folded in) so the
// exponentials are exp2.  Rows are launched in descending q: the heavy rows
// start first.
#include "ris_device.h"
#include "ris_internal.h"

namespace ris {
namespace {

constexpr int kGMax = 8;

template <bool BF16>
__device__ __forceinline__ float load_elem(const void* base, int64_t idx) {
    if constexpr (BF16) return bf16_to_f32(static_cast<const uint16_t*>(base)[idx]);
    else return static_cast<const float*>(base)[idx];
}

// Unpack one 16-byte vector of inputs into floats.
template <bool BF16>
__device__ __forceinline__ void unpack16(const uint4& u, float* f) {
    if constexpr (BF16) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            f[2 * e] = __uint_as_float(w[e] << 16);
            f[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
        }
    } else {
        f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
        f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
    }
}

// DPL consecutive elements of a row starting at element `off`.
template <bool BF16, int DPL>
__device__ __forceinline__ void load_dims(const void* base, int64_t off, float* v) {
    if constexpr (BF16) {
        const uint16_t* p = static_cast<const uint16_t*>(base) + off;
        if constexpr (DPL == 2) {
            const uint32_t w = *reinterpret_cast<const uint32_t*>(p);
            v[0] = __uint_as_float(w << 16);
            v[1] = __uint_as_float(w & 0xFFFF0000u);
        } else {
            v[0] = bf16_to_f32(p[0]);
        }
    } else {
        const float* p = static_cast<const float*>(base) + off;
        if constexpr (DPL == 2) {
            const float2 w = *reinterpret_cast<const float2*>(p);
            v[0] = w.x; v[1] = w.y;
        } else {
            v[0] = p[0];
        }
    }
}

template <int D>
__global__ __launch_bounds__(64) void k_attn_gather(AttnParams a, float qscale) {
    constexpr bool BF16 = false;                      // float32 inputs (bf16 runs on k_attn_gather16)
    constexpr int DPL = D / 64;                       // dims per lane in PV
    constexpr int VEC = BF16 ? 8 : 4;                 // elements per 16-byte load
    constexpr int NV = D / VEC;
    __shared__ __align__(16) float qs[kGMax][D];
    __shared__ __align__(16) float ps[64][kGMax];

    const int lane = threadIdx.x;
    const int G = a.G;
    const int64_t N = a.N;
    const int64_t i = blockIdx.x;
    const int64_t q = N - 1 - i / a.Hkv;
    const int g = (int)(i % a.Hkv);
    if (tile_is_dense(a, g, q - q % kTileRows)) return;   // that tile runs on the tiled kernel
    const int64_t r = (int64_t)g * N + q;
    int64_t start = a.row_ptr[r];
    int64_t L = a.row_ptr[r + 1] - start;
    if (start < 0 || L < 0) { start = 0; L = 0; }   // an incomplete build's rows: empty

    for (int e = lane; e < G * D; e += 64) {
        const int hh = e / D, d = e - hh * D;
        qs[hh][d] = load_elem<BF16>(a.Q, ((int64_t)(g * G + hh) * N + q) * D + d) * qscale;
    }
    __syncthreads();

    float m[kGMax], l[kGMax], acc[kGMax][DPL];
#pragma unroll
    for (int hh = 0; hh < kGMax; ++hh) {
        m[hh] = -INFINITY; l[hh] = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[hh][e] = 0.f;
    }

    const char* Kbase = static_cast<const char*>(a.K) + (int64_t)g * N * D * (BF16 ? 2 : 4);
    const char* Vbase = static_cast<const char*>(a.V) + (int64_t)g * N * D * (BF16 ? 2 : 4);

    for (int64_t c0 = 0; c0 < L; c0 += 64) {
        const int cnt = (int)(L - c0 < 64 ? L - c0 : 64);
        int j = lane < cnt ? a.col_idx[start + c0 + lane] : 0;
        // An index outside [0, N) is ignored (masked) rather than dereferenced.
        const bool valid = lane < cnt && (uint32_t)j < (uint32_t)N;
        if (!valid) j = 0;

        // ---- scores for all G heads from one read of K[g, j]
        const uint4* krow = reinterpret_cast<const uint4*>(Kbase + (int64_t)j * D * (BF16 ? 2 : 4));
        uint4 kraw[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) kraw[v] = krow[v];
        float s[kGMax];
#pragma unroll
        for (int hh = 0; hh < kGMax; ++hh) s[hh] = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            float kf[VEC];
            unpack16<BF16>(kraw[v], kf);
#pragma unroll
            for (int hh = 0; hh < kGMax; ++hh) {
                if (hh < G) {
                    const float4* qv = reinterpret_cast<const float4*>(&qs[hh][v * VEC]);
#pragma unroll
                    for (int e4 = 0; e4 < VEC / 4; ++e4) {
                        const float4 qq = qv[e4];
                        s[hh] = fmaf(qq.x, kf[4 * e4 + 0], s[hh]);
                        s[hh] = fmaf(qq.y, kf[4 * e4 + 1], s[hh]);
                        s[hh] = fmaf(qq.z, kf[4 * e4 + 2], s[hh]);
                        s[hh] = fmaf(qq.w, kf[4 * e4 + 3], s[hh]);
                    }
                }
            }
        }

        // ---- one online softmax per head over the unified set
#pragma unroll
        for (int hh = 0; hh < kGMax; ++hh) {
            if (hh < G) {
                const float sv = valid ? s[hh] : -INFINITY;
                const float mn = fmaxf(m[hh], wave_max(sv));
                // No valid entry yet (every index so far outside [0, N)): the
                // reference stays -inf, and a finite stand-in keeps corr and p
                // at 0 instead of exp2(-inf - -inf) = NaN.
                const float mc = mn == -INFINITY ? 0.f : mn;
                const float corr = exp2f(m[hh] - mc);
                const float p = exp2f(sv - mc);
                l[hh] = l[hh] * corr + wave_sum(p);
#pragma unroll
                for (int e = 0; e < DPL; ++e) acc[hh][e] *= corr;
                m[hh] = mn;
                ps[lane][hh] = p;
            }
        }
        __syncthreads();

        // ---- PV: lane owns dims [lane*DPL, lane*DPL + DPL)
        const int64_t doff = (int64_t)lane * DPL;
        int c = 0;
        for (; c + 4 <= cnt; c += 4) {
            float vv[4][DPL];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int jc = __builtin_amdgcn_readlane(j, c + u);
                load_dims<BF16, DPL>(Vbase, (int64_t)jc * D + doff, vv[u]);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float4 p0 = *reinterpret_cast<const float4*>(&ps[c + u][0]);
                const float4 p1 = *reinterpret_cast<const float4*>(&ps[c + u][4]);
                const float pp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
                for (int hh = 0; hh < kGMax; ++hh) {
                    if (hh < G) {
#pragma unroll
                        for (int e = 0; e < DPL; ++e) acc[hh][e] = fmaf(pp[hh], vv[u][e], acc[hh][e]);
                    }
                }
            }
        }
        for (; c < cnt; ++c) {
            float vv[DPL];
            const int jc = __builtin_amdgcn_readlane(j, c);
            load_dims<BF16, DPL>(Vbase, (int64_t)jc * D + doff, vv);
            const float4 p0 = *reinterpret_cast<const float4*>(&ps[c][0]);
            const float4 p1 = *reinterpret_cast<const float4*>(&ps[c][4]);
            const float pp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
            for (int hh = 0; hh < kGMax; ++hh) {
                if (hh < G) {
#pragma unroll
                    for (int e = 0; e < DPL; ++e) acc[hh][e] = fmaf(pp[hh], vv[e], acc[hh][e]);
                }
            }
        }
        __syncthreads();
    }

    // ---- normalise and store
#pragma unroll
    for (int hh = 0; hh < kGMax; ++hh) {
        if (hh < G) {
            const float inv = l[hh] > 0.f ? 1.0f / l[hh] : 0.f;
            const int64_t o = ((int64_t)(g * G + hh) * N + q) * D + (int64_t)lane * DPL;
#pragma unroll
            for (int e = 0; e < DPL; ++e) {
                const float val = acc[hh][e] * inv;
                if (a.out_bf16) static_cast<uint16_t*>(a.out)[o + e] = f32_to_bf16(val);
                else static_cast<float*>(a.out)[o + e] = val;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// bf16 gather on the matrix unit: one wavefront per (kv_head g, query row q),
// four rows per workgroup, no workgroup barriers (each wave owns a private
// LDS slice).  The row's set is walked in 32-key tiles; the next tile's K and
// V rows are loaded into registers before the current one is computed:
//   * S^T = K Q^T on MFMA 16x16x32 bf16 with the G query heads of the group
//     as the 16-wide dimension (K rows gathered straight from HBM into the
//     A-operand layout: lane l loads key l%16 of a 16-key half, dims
//     8 (l/16) + 32 s .. ), so one gather of a key row serves all G heads;
//   * one online softmax per head (lane l owns head l%16; a head's running
//     max and sum live in four lanes, combined with permlane swaps);
//   * O += P V on MFMA with P packed to bf16 in registers and V staged
//     row-major in the wave's LDS slice and read transposed.
// ---------------------------------------------------------------------------
constexpr int kGWaves = 4;            // rows (waves) per workgroup
constexpr int kGTile = 32;            // keys per tile
constexpr float kGNegBig = -1e30f;    // finite start of the running max


template <int D>
struct GTile {
    u32x4_t k[2][D / 32];
    u32x4_t v[2][D / 32];
    uint32_t valid;       // bit 16 kb + i: key slot 16 kb + i is a real key
};

// Keys [v0, v0 + 32) of the row's CSR list (slot 16 kb + l%16 per lane).
template <int D>
__device__ __forceinline__ void gather_tile(const int32_t* idx, int64_t L, int64_t N, const uint16_t* Kg,
                                            const uint16_t* Vg, int64_t v0, int li, int lg, GTile<D>& T) {
    uint32_t vm = 0;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int64_t v = v0 + 16 * kb + li;
        int64_t j = v < L ? (int64_t)idx[v] : -1;
        if (j >= N) j = -1;                            // an index outside [0, N) is ignored
        vm |= (uint32_t)(__ballot(j >= 0) & 0xFFFFull) << (16 * kb);
        const int64_t jj = j >= 0 ? j : 0;             // row 0 always exists
        const uint16_t* kp = Kg + jj * D + 8 * lg;
        const uint16_t* vp = Vg + jj * D + 8 * lg;
#pragma unroll
        for (int s = 0; s < D / 32; ++s) {
            T.k[kb][s] = *reinterpret_cast<const u32x4_t*>(kp + 32 * s);
            T.v[kb][s] = *reinterpret_cast<const u32x4_t*>(vp + 32 * s);
        }
    }
    T.valid = vm;
}

template <int D>
__global__ __launch_bounds__(64 * kGWaves, 2) void k_attn_gather16(AttnParams a, float c) {
    constexpr int SL = D / 32;         // k-slices of the score product
    constexpr int DB = D / 16;         // 16-dim blocks of the output
    constexpr int VS = D + 16;         // V row stride in LDS (bf16 elements)
    __shared__ __align__(16) uint16_t vlds[kGWaves * kGTile * VS];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int64_t N = a.N;
    const int64_t f = (int64_t)blockIdx.x * kGWaves + wave;   // heavy rows first
    if (f >= (int64_t)a.Hkv * N) return;
    const int64_t q = N - 1 - f / a.Hkv;
    const int g = (int)(f % a.Hkv);
    if (tile_is_dense(a, g, q - q % kTileRows)) return;   // that tile runs on the tiled kernel
    const int G = a.G;
    uint16_t* vw = vlds + wave * kGTile * VS;
    int64_t start = a.row_ptr[(int64_t)g * N + q];
    int64_t L = a.row_ptr[(int64_t)g * N + q + 1] - start;
    if (start < 0 || L < 0) { start = 0; L = 0; }   // an incomplete build's rows: empty
    const int32_t* idx = a.col_idx + start;
    const uint16_t* Kg = static_cast<const uint16_t*>(a.K) + (int64_t)g * N * D;
    const uint16_t* Vg = static_cast<const uint16_t*>(a.V) + (int64_t)g * N * D;

    // ---- Q^T as the B operand: lane l holds head l%16, dims 32 s + 8 (l/16) ..
    u32x4_t qf[SL];
    {
        const bool hv = li < G;
        const uint16_t* qp = static_cast<const uint16_t*>(a.Q) + ((int64_t)(g * G + (hv ? li : 0)) * N + q) * D + 8 * lg;
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
    float m_run = kGNegBig, l_run = 0.f;

    if (L > 0) {
        GTile<D> cur;
        gather_tile<D>(idx, L, N, Kg, Vg, 0, li, lg, cur);
        for (int64_t v0 = 0; v0 < L; v0 += kGTile) {
            GTile<D> nxt;
            const bool more = v0 + kGTile < L;
            if (more) gather_tile<D>(idx, L, N, Kg, Vg, v0 + kGTile, li, lg, nxt);

            // V rows into this wave's LDS slice, row-major (key slot 16 kb + l%16)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int s = 0; s < SL; ++s)
                    *reinterpret_cast<u32x4_t*>(vw + (16 * kb + li) * VS + 32 * s + 8 * lg) = cur.v[kb][s];

            // S^T = K Q^T: lane l holds head l%16 at key slots 16 kb + 4 (l/16) + i
            f32x4_t st[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                st[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < SL; ++s)
                    st[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.k[kb][s]), as_bf16x8(qf[s]),
                                                                      st[kb], 0, 0, 0);
            }
            // online softmax over the tile (scores in the log2 domain)
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
            // rescale the output rows: lane l holds heads 4 (l/16) + i
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float al = __shfl(alpha, 4 * lg + i);
#pragma unroll
                for (int db = 0; db < DB; ++db) o[db][i] *= al;
            }
            // P as the A operand (head l%16; k slots 8 (l/16) + e hold keys
            // 4 (l/16) + e and 16 + 4 (l/16) + e - 4); V as the B operand in
            // the same key order via the transpose read
            const u32x4_t pk = {pack_bf16x2(pv[0][0], pv[0][1]), pack_bf16x2(pv[0][2], pv[0][3]),
                                pack_bf16x2(pv[1][0], pv[1][1]), pack_bf16x2(pv[1][2], pv[1][3])};
            const uint16_t* v_lo = vw + (lane >> 2) * VS + 4 * (lane & 3);
            const uint16_t* v_hi = v_lo + 16 * VS;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const uint2 x = lds_read_tr16(v_lo + 16 * db);
                const uint2 y = lds_read_tr16(v_hi + 16 * db);
                const u32x4_t vb = {x.x, x.y, y.x, y.y};
                o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(pk), as_bf16x8(vb), o[db], 0, 0, 0);
            }
            if (more) cur = nxt;
        }
    }

    // ---- normalise and store: o[db][i] is dim 16 db + l%16 of head 4 (l/16) + i
    l_run = quad_sum16(l_run);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = 4 * lg + i;
        const float lh = __shfl(l_run, h);
        if (h < G) {
            const float inv = lh > 0.f ? 1.0f / lh : 0.f;
            const int64_t base = ((int64_t)(g * G + h) * N + q) * D + li;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const float val = o[db][i] * inv;
                if (a.out_bf16) static_cast<uint16_t*>(a.out)[base + 16 * db] = f32_to_bf16(val);
                else static_cast<float*>(a.out)[base + 16 * db] = val;
            }
        }
    }
}

}  // namespace

hipError_t launch_attn_gather(const AttnParams& a, hipStream_t st) {
    const float qscale = a.scale * 1.4426950408889634f;   // log2(e): scores in log2 domain
    if (a.in_bf16) {
        const int64_t rows = (int64_t)a.Hkv * a.N;
        const dim3 grid((unsigned)((rows + kGWaves - 1) / kGWaves)), block(64 * kGWaves);
        if (a.D == 128) hipLaunchKernelGGL((k_attn_gather16<128>), grid, block, 0, st, a, qscale);
        else hipLaunchKernelGGL((k_attn_gather16<64>), grid, block, 0, st, a, qscale);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((int64_t)a.Hkv * a.N)), block(64);
    if (a.D == 128) hipLaunchKernelGGL((k_attn_gather<128>), grid, block, 0, st, a, qscale);
    else hipLaunchKernelGGL((k_attn_gather<64>), grid, block, 0, st, a, qscale);
    return hipGetLastError();
}

}  // namespace ris
