// Micro-benchmark of the projection GEMM kernels (built as dash_gemm_bench next to
// libdash.so): for the decoder shapes of the workloads and a range of decode batch
// sizes, times the tiling launch_gemm / launch_gemm_qkv_rope choose against the other
// kernels of gemm.hip, and checks that every alternative gives the same bits.  Weights
// rotate through enough copies (>= 1 GiB in total) that every launch reads them from HBM,
// as in a decode step where each layer's weights were evicted by the other layers.
//
//   dash_gemm_bench [reps]
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <random>
#include <string>
#include <vector>

#include "gemm.hip"

#define CK(x)                                                                                          \
    do {                                                                                               \
        hipError_t e_ = (x);                                                                           \
        if (e_ != hipSuccess) {                                                                        \
            fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_));          \
            exit(1);                                                                                   \
        }                                                                                              \
    } while (0)

using namespace dash;

namespace {

struct ModelShape {
    const char* name;
    int d, n_heads, n_kv, hd;
};

uint16_t to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFF + ((u >> 16) & 1);
    return (uint16_t)(u >> 16);
}

struct Dev {
    void* p = nullptr;
    size_t n = 0;
    explicit Dev(size_t bytes) : n(bytes) { CK(hipMalloc(&p, bytes)); }
    ~Dev() { (void)hipFree(p); }
};

std::vector<uint16_t> randn_bf16(size_t n, float scale, std::mt19937& rng) {
    std::normal_distribution<float> nd(0.f, 1.f);
    std::vector<uint16_t> v(n);
    for (auto& x : v) x = to_bf16(nd(rng) * scale);
    return v;
}

using Launch = std::function<hipError_t(const void* w)>;

double time_us(const Launch& f, int n_w, size_t w_bytes, const void* w0, int reps, hipStream_t st) {
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    for (int i = 0; i < 3; ++i) CK(f((const char*)w0 + (i % n_w) * w_bytes));
    CK(hipEventRecord(e0, st));
    for (int i = 0; i < reps; ++i) CK(f((const char*)w0 + (i % n_w) * w_bytes));
    CK(hipEventRecord(e1, st));
    CK(hipEventSynchronize(e1));
    float ms;
    CK(hipEventElapsedTime(&ms, e0, e1));
    CK(hipEventDestroy(e0));
    CK(hipEventDestroy(e1));
    return ms * 1e3 / reps;
}

}  // namespace

int main(int argc, char** argv) {
    const int reps = argc > 1 ? atoi(argv[1]) : 20;
    const ModelShape shapes[] = {{"0.5b", 896, 14, 2, 64}, {"1.5b", 1536, 12, 2, 128}, {"3b", 2048, 16, 2, 128}};
    const int batches[] = {256, 512, 768, 1024, 2048};
    hipStream_t st;
    CK(hipStreamCreate(&st));
    std::mt19937 rng(7);
    printf("kernel timings in us (weights cold); alternatives marked = give the production bits\n");
    for (const ModelShape& sh : shapes) {
        const int d = sh.d, hq = sh.n_heads * sh.hd, qr = (sh.n_heads + 2 * sh.n_kv) * sh.hd;
        for (int M : batches) {
            // ---- output projection: C[M, d] = o[M, hq] . W_o[d, hq]^T (fp32, unsplit)
            {
                const int N = d, K = hq;
                const size_t w_bytes = (size_t)N * K * 2;
                const int n_w = (int)std::min<size_t>(16, (1ull << 30) / w_bytes + 1);
                Dev a((size_t)M * K * 2), w(w_bytes * n_w), c0((size_t)M * N * 4), c1((size_t)M * N * 4);
                auto ha = randn_bf16((size_t)M * K, 1.f, rng), hw = randn_bf16((size_t)N * K, 0.02f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                for (int i = 0; i < n_w; ++i)
                    CK(hipMemcpy((char*)w.p + i * w_bytes, hw.data(), w_bytes, hipMemcpyHostToDevice));
                auto prod = [&](const void* wp, void* c) { return launch_gemm(1, EPI_STORE_F32, a.p, wp, c, M, N, K, N, 1, 0, st); };
                CK(prod(w.p, c0.p));
                CK(hipStreamSynchronize(st));
                std::vector<char> r0((size_t)M * N * 4), r1(r0.size());
                CK(hipMemcpy(r0.data(), c0.p, r0.size(), hipMemcpyDeviceToHost));
                const double tp = time_us([&](const void* wp) { return prod(wp, c1.p); }, n_w, w_bytes, w.p, reps, st);
                printf("%-5s o    M=%4d N=%4d K=%4d  production %7.1f", sh.name, M, N, K, tp);
                struct Alt {
                    const char* name;
                    std::function<hipError_t(const void*, void*)> f;
                };
                const Alt alts[] = {
                    {"lds128x64", [&](const void* wp, void* c) { return run_lds<128, 64, 2, 2, 4, EPI_STORE_F32>(a.p, wp, c, M, N, K, N, 1, 0, st); }},
                    {"lds64x64", [&](const void* wp, void* c) { return run_lds<64, 64, 2, 2, 4, EPI_STORE_F32>(a.p, wp, c, M, N, K, N, 1, 0, st); }},
                    {"lds64x128", [&](const void* wp, void* c) { return run_lds<64, 128, 2, 2, 4, EPI_STORE_F32>(a.p, wp, c, M, N, K, N, 1, 0, st); }},
                    {"lds128x128", [&](const void* wp, void* c) { return run_lds<128, 128, 2, 2, 4, EPI_STORE_F32>(a.p, wp, c, M, N, K, N, 1, 0, st); }},
                };
                for (const Alt& alt : alts) {
                    CK(hipMemset(c1.p, 0xFF, r1.size()));
                    CK(alt.f(w.p, c1.p));
                    CK(hipStreamSynchronize(st));
                    CK(hipMemcpy(r1.data(), c1.p, r1.size(), hipMemcpyDeviceToHost));
                    const bool same = memcmp(r0.data(), r1.data(), r0.size()) == 0;
                    const double t = time_us([&](const void* wp) { return alt.f(wp, c1.p); }, n_w, w_bytes, w.p, reps, st);
                    printf("  %s %6.1f%s", alt.name, t, same ? "=" : " MISMATCH");
                }
                printf("\n");
                fflush(stdout);
            }
            // ---- QKV projection with bias, RoPE and the KV append (fused epilogue)
            if (gemm_qkv_fusable(1, sh.n_heads, sh.n_kv, sh.hd)) {
                const int N = qr, K = d, hd = sh.hd, ps = 32;
                const size_t w_bytes = (size_t)N * K * 2;
                const int n_w = (int)std::min<size_t>(16, (1ull << 30) / w_bytes + 1);
                Dev a((size_t)M * K * 2), w(w_bytes * n_w), bias((size_t)N * 2), cs((size_t)M * hd * 4);
                Dev pos((size_t)M * 4), slot((size_t)M * 4), table((size_t)M * 4), status(256);
                const size_t pool_elems = (size_t)M * sh.n_kv * 2 * ps * hd;  // one page per row, one layer
                Dev pool0(pool_elems * 2), pool1(pool_elems * 2), q0((size_t)M * hq * 2), q1((size_t)M * hq * 2);
                auto ha = randn_bf16((size_t)M * K, 1.f, rng), hw = randn_bf16((size_t)N * K, 0.02f, rng);
                auto hb = randn_bf16(N, 0.02f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                for (int i = 0; i < n_w; ++i)
                    CK(hipMemcpy((char*)w.p + i * w_bytes, hw.data(), w_bytes, hipMemcpyHostToDevice));
                CK(hipMemcpy(bias.p, hb.data(), hb.size() * 2, hipMemcpyHostToDevice));
                std::vector<int32_t> hp(M), hs(M), ht(M);
                std::vector<float> hcs((size_t)M * hd);
                for (int m = 0; m < M; ++m) {
                    hp[m] = 5 + m % 27;
                    hs[m] = m;
                    ht[m] = m;
                    for (int i = 0; i < hd / 2; ++i) {
                        const double ang = hp[m] * std::pow(1e6, -2.0 * i / hd);
                        hcs[((size_t)m * (hd / 2) + i) * 2] = (float)std::cos(ang);
                        hcs[((size_t)m * (hd / 2) + i) * 2 + 1] = (float)std::sin(ang);
                    }
                }
                CK(hipMemcpy(pos.p, hp.data(), M * 4, hipMemcpyHostToDevice));
                CK(hipMemcpy(slot.p, hs.data(), M * 4, hipMemcpyHostToDevice));
                CK(hipMemcpy(table.p, ht.data(), M * 4, hipMemcpyHostToDevice));
                CK(hipMemcpy(cs.p, hcs.data(), hcs.size() * 4, hipMemcpyHostToDevice));
                CK(hipMemset(status.p, 0, 4));
                KVGeom g{1, M, sh.n_kv, hd, ps, 1, M, 2048, 0};
                auto args = [&](void* pool, void* q) {
                    return QkvRopeArgs{(const bf16_t*)bias.p, (const float*)cs.p, (const int32_t*)pos.p,
                                       (const int32_t*)slot.p, (const int32_t*)table.p, (bf16_t*)pool, g, 0,
                                       (bf16_t*)q, sh.n_heads, (uint32_t*)status.p};
                };
                CK(hipMemset(pool0.p, 0, pool0.n));
                CK(hipMemset(pool1.p, 0, pool1.n));
                // the production path (fused above its size threshold, else the unfused GEMM + RoPE kernel)
                auto prod = [&](const void* wp, void* pool, void* q) -> hipError_t {
                    const QkvRopeArgs qa = args(pool, q);
                    if (gemm_qkv_fuse_pays(M, N)) return launch_gemm_qkv_rope(a.p, wp, M, N, K, qa, st);
                    return run_bf16<64, 128, 2, 4, 2, EPI_QKV_ROPE>(a.p, wp, nullptr, M, N, K, 0, 1, 0, st, qa);
                };
                CK(prod(w.p, pool0.p, q0.p));
                CK(hipStreamSynchronize(st));
                std::vector<char> rq0(q0.n), rp0(pool0.n), rq1(q0.n), rp1(pool0.n);
                CK(hipMemcpy(rq0.data(), q0.p, q0.n, hipMemcpyDeviceToHost));
                CK(hipMemcpy(rp0.data(), pool0.p, pool0.n, hipMemcpyDeviceToHost));
                const double tp = time_us([&](const void* wp) { return prod(wp, pool1.p, q1.p); }, n_w, w_bytes, w.p,
                                          reps, st);
                printf("%-5s qkv  M=%4d N=%4d K=%4d  fused     %7.1f", sh.name, M, N, K, tp);
                struct Alt {
                    const char* name;
                    std::function<hipError_t(const void*, void*, void*)> f;
                };
                const Alt alts[] = {
                    {"lds64x128", [&](const void* wp, void* pool, void* q) { return run_lds<64, 128, 2, 2, 4, EPI_QKV_ROPE>(a.p, wp, nullptr, M, N, K, 0, 1, 0, st, args(pool, q)); }},
                    {"lds64x128s3", [&](const void* wp, void* pool, void* q) { return run_lds<64, 128, 2, 2, 3, EPI_QKV_ROPE>(a.p, wp, nullptr, M, N, K, 0, 1, 0, st, args(pool, q)); }},
                };
                for (const Alt& alt : alts) {
                    CK(hipMemset(pool1.p, 0, pool1.n));
                    CK(hipMemset(q1.p, 0xFF, q1.n));
                    CK(alt.f(w.p, pool1.p, q1.p));
                    CK(hipStreamSynchronize(st));
                    CK(hipMemcpy(rq1.data(), q1.p, q1.n, hipMemcpyDeviceToHost));
                    CK(hipMemcpy(rp1.data(), pool1.p, pool1.n, hipMemcpyDeviceToHost));
                    const bool same = rq0 == rq1 && rp0 == rp1;
                    const double t = time_us([&](const void* wp) { return alt.f(wp, pool1.p, q1.p); }, n_w, w_bytes,
                                             w.p, reps, st);
                    printf("  %s %6.1f%s", alt.name, t, same ? "=" : " MISMATCH");
                }
                uint32_t hst = 0;
                CK(hipMemcpy(&hst, status.p, 4, hipMemcpyDeviceToHost));
                printf("%s\n", hst ? "  (status set!)" : "");
                fflush(stdout);
            }
        }
    }
    return 0;
}
