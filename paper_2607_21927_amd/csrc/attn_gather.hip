// Sparse attention, gather form: one wavefront per (kv_head g, query row q).
//
// The row's unified index set I(g, q) (CSR) is walked in chunks of 64 keys:
//   1. scores  -- lane l owns key j_l of the chunk, reads K[g, j_l] once and
//      forms <Q[h, q], K[g, j_l]> for every query head h of the GQA group
//      (the G query rows sit in LDS and are read as broadcasts), so one
//      gather of the key row serves all G heads;
//   2. softmax -- one running (max, sum) per head over the whole set:
//      wavefront max and sum by DPP, rescale of the accumulators when the
//      max grows.  Every index of the set enters this single normalisation
//      once (Pre-Fusion Unified Softmax; Methods, "Hybrid Anchor and
//      Pre-Fusion Unified Softmax");
//   3. PV      -- lanes switch to owning D/64 consecutive dimensions; for each
//      key of the chunk the wave reads the value row as one contiguous
//      segment and accumulates p_h * V for all G heads.
// Scores are kept in the log2 domain (scale * log2(e) folded into Q) so the
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

template <int D, bool BF16>
__global__ __launch_bounds__(64) void k_attn_gather(AttnParams a, float qscale) {
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
    const int64_t start = a.row_ptr[r];
    const int64_t L = a.row_ptr[r + 1] - start;

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
                const float corr = exp2f(m[hh] - mn);
                const float p = exp2f(sv - mn);
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

}  // namespace

hipError_t launch_attn_gather(const AttnParams& a, hipStream_t st) {
    const float qscale = a.scale * 1.4426950408889634f;   // log2(e): scores in log2 domain
    const dim3 grid((unsigned)((int64_t)a.Hkv * a.N)), block(64);
    if (a.D == 128) {
        if (a.in_bf16) hipLaunchKernelGGL((k_attn_gather<128, true>), grid, block, 0, st, a, qscale);
        else hipLaunchKernelGGL((k_attn_gather<128, false>), grid, block, 0, st, a, qscale);
    } else {
        if (a.in_bf16) hipLaunchKernelGGL((k_attn_gather<64, true>), grid, block, 0, st, a, qscale);
        else hipLaunchKernelGGL((k_attn_gather<64, false>), grid, block, 0, st, a, qscale);
    }
    return hipGetLastError();
}

}  // namespace ris
