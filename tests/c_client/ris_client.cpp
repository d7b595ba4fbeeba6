// A plain C++ caller of the RIS C ABI (no Python, no torch): reads bf16 Q, K, V
// from files, builds the geometry and runs the sparse attention with device
// buffers it allocates itself, and writes the CSR and the output back.
//
//   int ris_client_run(in_dir, out_dir, N, Hq, Hkv, D, density_ppm, n_seeds)
//
// in_dir holds q.bin [Hq,N,D], k.bin and v.bin [Hkv,N,D] (bf16, raw); out_dir
// receives row_ptr.bin (int64), col_idx.bin (int32, nnz entries) and out.bin
// (float32 [Hq,N,D]).  Every library status is checked; the result is 0 only
// when every call succeeded.  Built as a shared object so that a test can
// call it in its own process.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string>
#include <vector>

#include "ris.h"

static bool read_file(const std::string& path, void* dst, size_t bytes) {
    FILE* f = fopen(path.c_str(), "rb");
    if (!f) return false;
    const size_t got = fread(dst, 1, bytes, f);
    fclose(f);
    return got == bytes;
}

static bool write_file(const std::string& path, const void* src, size_t bytes) {
    FILE* f = fopen(path.c_str(), "wb");
    if (!f) return false;
    const size_t put = fwrite(src, 1, bytes, f);
    fclose(f);
    return put == bytes;
}

#define HIP_OK(call)                                                              \
    do {                                                                          \
        hipError_t e_ = (call);                                                   \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));            \
            return 2;                                                             \
        }                                                                         \
    } while (0)

#define RIS_OK(call)                                                              \
    do {                                                                          \
        int s_ = (call);                                                          \
        if (s_ != RIS_OK) {                                                       \
            fprintf(stderr, "%s: %s\n", #call, ris_status_string(s_));            \
            return 3;                                                             \
        }                                                                         \
    } while (0)

extern "C" int ris_client_run(const char* in_dir, const char* out_dir, int64_t N, int32_t Hq, int32_t Hkv,
                              int32_t D, int32_t ppm, int32_t S) {
    if (!in_dir || !out_dir || N <= 0 || Hq <= 0 || Hkv <= 0 || D <= 0) return 1;
    const std::string in = in_dir, out = out_dir;
    const size_t nq = (size_t)Hq * N * D, nk = (size_t)Hkv * N * D;

    std::vector<uint16_t> hq(nq), hk(nk), hv(nk);
    if (!read_file(in + "/q.bin", hq.data(), nq * 2) || !read_file(in + "/k.bin", hk.data(), nk * 2) ||
        !read_file(in + "/v.bin", hv.data(), nk * 2)) {
        fprintf(stderr, "cannot read the inputs in %s\n", in.c_str());
        return 1;
    }

    ris_mask_desc md = {};
    md.mode = RIS_STOCHASTIC;
    md.density_ppm = ppm;
    md.seed = 0;
    md.n_seeds = S;
    md.layer = 0;
    md.N = N;
    md.heads = Hkv;
    md.causal = 1;
    const int64_t cap = ris_mask_nnz_bound(&md);
    if (cap < 0) {
        fprintf(stderr, "ris_mask_nnz_bound: %s\n", ris_status_string((int)cap));
        return 3;
    }

    void *dq, *dk, *dv, *dout;
    int64_t* drp;
    int32_t* dci;
    HIP_OK(hipMalloc(&dq, nq * 2));
    HIP_OK(hipMalloc(&dk, nk * 2));
    HIP_OK(hipMalloc(&dv, nk * 2));
    HIP_OK(hipMalloc(&dout, nq * 4));
    HIP_OK(hipMalloc(&drp, ((size_t)Hkv * N + 1) * sizeof(int64_t)));
    HIP_OK(hipMalloc(&dci, (size_t)(cap > 0 ? cap : 1) * sizeof(int32_t)));
    HIP_OK(hipMemcpy(dq, hq.data(), nq * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dk, hk.data(), nk * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dv, hv.data(), nk * 2, hipMemcpyHostToDevice));
    hipStream_t st;
    HIP_OK(hipStreamCreate(&st));

    // One pass into the bound-sized index buffer, then attention on the same stream.
    RIS_OK(ris_mask_build(&md, drp, dci, cap, st));
    ris_attn_desc ad = {};
    ad.dtype_in = RIS_BF16;
    ad.dtype_out = RIS_F32;
    ad.Hq = Hq;
    ad.Hkv = Hkv;
    ad.N = N;
    ad.D = D;
    ad.scale = 0.0f;
    ad.mode = RIS_STOCHASTIC;
    ad.block = 0;
    ad.causal = 1;
    ad.algo = RIS_ATTN_AUTO;
    RIS_OK(ris_sparse_attn(dq, dk, dv, drp, dci, dout, &ad, st));
    HIP_OK(hipStreamSynchronize(st));

    std::vector<int64_t> rp((size_t)Hkv * N + 1);
    HIP_OK(hipMemcpy(rp.data(), drp, rp.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
    const int64_t nnz = rp.back();
    std::vector<int32_t> ci((size_t)nnz);
    if (nnz > 0) HIP_OK(hipMemcpy(ci.data(), dci, (size_t)nnz * sizeof(int32_t), hipMemcpyDeviceToHost));
    std::vector<float> ho(nq);
    HIP_OK(hipMemcpy(ho.data(), dout, nq * 4, hipMemcpyDeviceToHost));
    if (!write_file(out + "/row_ptr.bin", rp.data(), rp.size() * sizeof(int64_t)) ||
        !write_file(out + "/col_idx.bin", ci.data(), ci.size() * sizeof(int32_t)) ||
        !write_file(out + "/out.bin", ho.data(), nq * 4)) {
        fprintf(stderr, "cannot write the outputs in %s\n", out.c_str());
        return 1;
    }
    HIP_OK(hipStreamDestroy(st));
    HIP_OK(hipFree(dq));
    HIP_OK(hipFree(dk));
    HIP_OK(hipFree(dv));
    HIP_OK(hipFree(dout));
    HIP_OK(hipFree(drp));
    HIP_OK(hipFree(dci));
    return 0;
}
