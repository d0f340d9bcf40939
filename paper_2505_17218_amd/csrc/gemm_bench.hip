// Micro-benchmark of the projection GEMM kernels (built as dash_gemm_bench next to
// libdash.so): for the decoder shapes of the workloads and a range of decode batch
// sizes, times the tiling launch_gemm / launch_gemm_qkv_rope choose ("production")
// against the other kernels of gemm.hip, and checks that every alternative gives the
// same bits (output, QKV, gate/up, down projections and the 1.5B LM head).  Weights rotate through
// enough copies (>= 1 GiB in total) that every launch reads them from HBM, as in a
// decode step where each layer's weights were evicted by the other layers.  The
// variants of a case are timed in interleaved rounds after a common warm-up of about
// 20 ms, and each reports its median round: timing one variant after another instead
// made whichever ran first up to 10% slower (clock ramp after the host-side set-up).
//
//   dash_gemm_bench [reps per round] [small]
//
// With "small", the decode batches of one 64-row block (16, 32 and 64 rows) instead:
// the tiles that stream the weights, with two to eight k-steps in flight per thread,
// and the fused QKV kernel against the projection followed by the RoPE / KV-append
// kernel of elementwise.hip (the path the decode step takes at these batches).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <random>
#include <string>
#include <vector>

#include "elementwise.hip"
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
    int d, n_heads, n_kv, hd, ff;
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

int weight_copies(int N, int K) { return (int)std::min<size_t>(16, (1ull << 30) / ((size_t)N * K * 2) + 1); }

// Weight copies of one projection, each read cold by the launch that uses it.
struct Weights {
    size_t bytes;
    int copies;
    Dev w;
    Weights(int N, int K, std::mt19937& rng)
        : bytes((size_t)N * K * 2), copies(weight_copies(N, K)), w((size_t)N * K * 2 * weight_copies(N, K)) {
        const auto h = randn_bf16((size_t)N * K, 0.02f, rng);
        for (int i = 0; i < copies; ++i) CK(hipMemcpy((char*)w.p + i * bytes, h.data(), bytes, hipMemcpyHostToDevice));
    }
    const void* copy(int i) const { return (const char*)w.p + (size_t)(i % copies) * bytes; }
};

// A variant launches into the reference outputs (ref = true) or the scratch ones.
struct Variant {
    std::string name;
    std::function<hipError_t(const void* w, bool ref)> f;
};

// Runs variant 0 (production) into the reference outputs, every other variant into the
// scratch outputs and compares (same_as_ref), then times all of them interleaved; prints
// one line with the median microseconds per launch of each.
void bench_case(const char* label, const std::vector<Variant>& vs, const Weights& w, int reps, hipStream_t st,
                const std::function<void()>& clear_scratch, const std::function<bool()>& same_as_ref) {
    std::vector<bool> same(vs.size(), true);
    CK(vs[0].f(w.copy(0), true));
    CK(hipStreamSynchronize(st));
    for (size_t v = 1; v < vs.size(); ++v) {
        clear_scratch();
        CK(vs[v].f(w.copy(0), false));
        CK(hipStreamSynchronize(st));
        same[v] = same_as_ref();
    }
    // common warm-up: every variant over every weight copy, repeated until ~20 ms have passed
    const auto t0 = std::chrono::steady_clock::now();
    do {
        for (const Variant& v : vs)
            for (int i = 0; i < w.copies; ++i) CK(v.f(w.copy(i), false));
        CK(hipStreamSynchronize(st));
    } while (std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count() < 0.02);
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    constexpr int kRounds = 5;
    std::vector<std::vector<double>> t(vs.size());
    for (int r = 0; r < kRounds; ++r)
        for (size_t v = 0; v < vs.size(); ++v) {
            CK(hipEventRecord(e0, st));
            for (int i = 0; i < reps; ++i) CK(vs[v].f(w.copy(i), false));
            CK(hipEventRecord(e1, st));
            CK(hipEventSynchronize(e1));
            float ms;
            CK(hipEventElapsedTime(&ms, e0, e1));
            t[v].push_back(ms * 1e3 / reps);
        }
    CK(hipEventDestroy(e0));
    CK(hipEventDestroy(e1));
    printf("%s", label);
    for (size_t v = 0; v < vs.size(); ++v) {
        std::sort(t[v].begin(), t[v].end());
        printf("  %s %6.1f%s", vs[v].name.c_str(), t[v][kRounds / 2], v == 0 ? "" : (same[v] ? "=" : " MISMATCH"));
    }
    printf("\n");
    fflush(stdout);
}

// Compare two device buffers of n bytes.
bool same_bytes(const Dev& x, const Dev& y) {
    std::vector<char> a(x.n), b(y.n);
    CK(hipMemcpy(a.data(), x.p, x.n, hipMemcpyDeviceToHost));
    CK(hipMemcpy(b.data(), y.p, y.n, hipMemcpyDeviceToHost));
    return a == b;
}

// The QKV projection with the fused bias / RoPE / KV-append epilogue on M rows: one
// page per row in a one-layer pool (two copies, reference and scratch), positions 5..31.
struct QkvCase {
    const ModelShape& sh;
    int M, N, K, hd;
    Weights w;
    Dev a, bias, cs, pos, slot, table, status, pool0, pool1, q0, q1;
    KVGeom g;
    QkvCase(const ModelShape& s, int m, std::mt19937& rng)
        : sh(s), M(m), N((s.n_heads + 2 * s.n_kv) * s.hd), K(s.d), hd(s.hd), w(N, K, rng), a((size_t)M * K * 2),
          bias((size_t)N * 2), cs((size_t)M * hd * 4), pos((size_t)M * 4), slot((size_t)M * 4), table((size_t)M * 4),
          status(256), pool0(pool_bytes()), pool1(pool_bytes()), q0((size_t)M * s.n_heads * hd * 2),
          q1((size_t)M * s.n_heads * hd * 2), g{1, M, s.n_kv, hd, 32, 1, M, 2048, 0} {
        const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
        const auto hb = randn_bf16(N, 0.02f, rng);
        CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
        CK(hipMemcpy(bias.p, hb.data(), hb.size() * 2, hipMemcpyHostToDevice));
        std::vector<int32_t> hp(M), hs(M), ht(M);
        std::vector<float> hcs((size_t)M * hd);
        for (int r = 0; r < M; ++r) {
            hp[r] = 5 + r % 27;
            hs[r] = r;
            ht[r] = r;
            for (int i = 0; i < hd / 2; ++i) {
                const double ang = hp[r] * std::pow(1e6, -2.0 * i / hd);
                hcs[((size_t)r * (hd / 2) + i) * 2] = (float)std::cos(ang);
                hcs[((size_t)r * (hd / 2) + i) * 2 + 1] = (float)std::sin(ang);
            }
        }
        CK(hipMemcpy(pos.p, hp.data(), M * 4, hipMemcpyHostToDevice));
        CK(hipMemcpy(slot.p, hs.data(), M * 4, hipMemcpyHostToDevice));
        CK(hipMemcpy(table.p, ht.data(), M * 4, hipMemcpyHostToDevice));
        CK(hipMemcpy(cs.p, hcs.data(), hcs.size() * 4, hipMemcpyHostToDevice));
        CK(hipMemset(status.p, 0, 4));
        CK(hipMemset(pool0.p, 0, pool0.n));
        CK(hipMemset(pool1.p, 0, pool1.n));
    }
    size_t pool_bytes() const { return (size_t)M * sh.n_kv * 2 * 32 * sh.hd * 2; }  // one page per row, one layer
    QkvRopeArgs args(bool ref) const {
        return QkvRopeArgs{(const bf16_t*)bias.p, (const float*)cs.p, (const int32_t*)pos.p, (const int32_t*)slot.p,
                           (const int32_t*)table.p, (bf16_t*)(ref ? pool0.p : pool1.p), g, 0,
                           (bf16_t*)(ref ? q0.p : q1.p), sh.n_heads, (uint32_t*)status.p};
    }
    // times the variants (0 = reference) and checks q and the appended K/V against it
    void run(const char* label, const std::vector<Variant>& vs, int reps, hipStream_t st) {
        bench_case(label, vs, w, reps, st,
                   [&] {
                       CK(hipMemset(pool1.p, 0, pool1.n));
                       CK(hipMemset(q1.p, 0xFF, q1.n));
                   },
                   [&] { return same_bytes(q0, q1) && same_bytes(pool0, pool1); });
        uint32_t hst = 0;
        CK(hipMemcpy(&hst, status.p, 4, hipMemcpyDeviceToHost));
        if (hst) printf("  (status set!)\n");
    }
};

// Batches of one 64-row block: the projections stream their weights (every weight byte
// read by one work-group) and each work-group's k-loop is a chain of dependent loads,
// so the variants differ in how many k-steps each thread keeps in flight.
void bench_small(const ModelShape* shapes, int n_shapes, int reps, hipStream_t st, std::mt19937& rng) {
    constexpr int W = kWeightStream;
    char label[128];
    for (int si = 0; si < n_shapes; ++si) {
        const ModelShape& sh = shapes[si];
        const int d = sh.d, hq = sh.n_heads * sh.hd, qr = (sh.n_heads + 2 * sh.n_kv) * sh.hd;
        for (int M : {16, 32, 64}) {
            // QKV (unfused at this batch), output and down projections: fp32 stores
            struct Proj {
                const char* name;
                int N, K;
            };
            const Proj projs[] = {{"qkv ", qr, d}, {"o   ", d, hq}, {"down", d, sh.ff}};
            for (const Proj& pj : projs) {
                const int N = pj.N, K = pj.K;
                const int ns = gemm_pick_splits(1, EPI_STORE_F32, N, K);
                Weights w(N, K, rng);
                const size_t cn = (size_t)ns * M * N, ss = (size_t)M * N;
                Dev a((size_t)M * K * 2), c0(cn * 4), c1(cn * 4);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                const std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_STORE_F32, a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"pd2", [&](const void* wp, bool r) { return run_bf16<64, 32, 2, 1, 2, EPI_STORE_F32, W>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"pd6", [&](const void* wp, bool r) { return run_bf16<64, 32, 2, 1, 6, EPI_STORE_F32, W>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"pd8", [&](const void* wp, bool r) { return run_bf16<64, 32, 2, 1, 8, EPI_STORE_F32, W>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"pd4cached", [&](const void* wp, bool r) { return run_bf16<64, 32, 2, 1, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                };
                snprintf(label, sizeof label, "%-5s %s M=%4d N=%5d K=%5d s%d  ", sh.name, pj.name, M, N, K, ns);
                bench_case(label, vs, w, reps, st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            }
            // gate/up projection with the SwiGLU epilogue
            {
                const int ff = sh.ff, N = 2 * ff, K = d;
                Weights w(N, K, rng);
                Dev a((size_t)M * K * 2), c0((size_t)M * ff * 2), c1((size_t)M * ff * 2);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                const std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_SWIGLU, a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"64x128pd2", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 2, 2, EPI_SWIGLU, W>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"64x128pd4", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 2, 4, EPI_SWIGLU, W>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"64x128pd6", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 2, 6, EPI_SWIGLU, W>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"64x64pd2", [&](const void* wp, bool r) { return run_bf16<64, 64, 2, 1, 2, EPI_SWIGLU, W>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"64x64pd4", [&](const void* wp, bool r) { return run_bf16<64, 64, 2, 1, 4, EPI_SWIGLU, W>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                };
                snprintf(label, sizeof label, "%-5s gu   M=%4d N=%5d K=%5d     ", sh.name, M, N, K);
                bench_case(label, vs, w, reps, st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            }
            // the QKV projection with its fused epilogue (at these batches the decode step runs
            // the unfused projection and a separate RoPE / append kernel instead)
            if (gemm_qkv_fusable(1, sh.n_heads, sh.n_kv, sh.hd)) {
                QkvCase c(sh, M, rng);
                const void* A = c.a.p;
                const int N = c.N, K = c.K;
                Dev qkv32((size_t)M * N * 4);
                const std::vector<Variant> vs = {
                    // the decode step's path at these batches: projection to fp32, then the RoPE / append kernel
                    {"unfused", [&](const void* wp, bool r) -> hipError_t {
                         const QkvRopeArgs qa = c.args(r);
                         const hipError_t e = launch_gemm(1, EPI_STORE_F32, A, wp, qkv32.p, M, N, K, N, 1, 0, st);
                         if (e != hipSuccess) return e;
                         return launch_qkv_rope_append(1, (const float*)qkv32.p, 1, 0, qa.bias, qa.cs, qa.pos, qa.slot,
                                                       qa.page_table, qa.pool, qa.g, 0, qa.q_out, M, qa.n_heads, qa.status, st);
                     }},
                    {"fused64x128", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 4, 2, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, c.args(r)); }},
                    {"stream", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 4, 2, EPI_QKV_ROPE, W>(A, wp, nullptr, M, N, K, 0, 1, 0, st, c.args(r)); }},
                    {"stream_pd4", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 4, 4, EPI_QKV_ROPE, W>(A, wp, nullptr, M, N, K, 0, 1, 0, st, c.args(r)); }},
                    {"stream_w4pd4", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 2, 4, EPI_QKV_ROPE, W>(A, wp, nullptr, M, N, K, 0, 1, 0, st, c.args(r)); }},
                };
                snprintf(label, sizeof label, "%-5s qkvf M=%4d N=%5d K=%5d     ", sh.name, M, N, K);
                c.run(label, vs, reps, st);
            }
        }
    }
}

// Gate/up at 512-2048 rows, cut by columns: the 256x256 tiles of the whole rounds (256 of
// them per round) timed on their own, and the remaining columns on smaller tiles, each on a
// projection of that width.  The sum estimates a two-launch split against the production
// tiling of the whole width.
void bench_gu_split(const ModelShape* shapes, int n_shapes, int reps, hipStream_t st, std::mt19937& rng) {
    char label[160];
    for (int si = 0; si < n_shapes; ++si) {
        const ModelShape& sh = shapes[si];
        for (int M : {1024, 2048}) {
            const int K = sh.d, mb = (M + 255) / 256;
            const int round_cols = 256 / mb * 128;  // h columns of one round of 256x256 tiles
            const int full = sh.ff / round_cols * round_cols, rest = sh.ff - full;
            auto one = [&](int ff, const char* what, bool split_variants) {
                const int N = 2 * ff;
                Weights w(N, K, rng);
                Dev a((size_t)M * K * 2), c0((size_t)M * ff * 2), c1((size_t)M * ff * 2);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_SWIGLU, a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"256x256", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 4, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                };
                if (split_variants) {
                    vs.push_back({"128x128", [&](const void* wp, bool r) { return run_bf16<128, 128, 4, 2, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }});
                    vs.push_back({"64x128", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 2, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }});
                    vs.push_back({"64x64", [&](const void* wp, bool r) { return run_bf16<64, 64, 2, 1, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }});
                    vs.push_back({"128x256", [&](const void* wp, bool r) { return run_bf16<128, 256, 4, 4, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }});
                }
                snprintf(label, sizeof label, "%-5s gu %-9s M=%4d ff=%5d     ", sh.name, what, M, ff);
                bench_case(label, vs, w, reps, st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            };
            one(sh.ff, "whole", false);
            if (full > 0 && rest > 0) {
                one(full, "rounds", false);
                one(rest, "rest", true);
            }
        }
    }
    // the 1.5B LM head (151,936 columns, fp32 logits) the same way
    for (int M : {1024, 2048}) {
        const int K = 1536, V = 151936, mb = (M + 255) / 256;
        const int full = (int)((long)mb * ((V + 255) / 256) / 256 * 256 / mb) * 256, rest = V - full;
        auto one = [&](int N, const char* what, bool split_variants) {
            Weights w(N, K, rng);
            Dev a((size_t)M * K * 2), c0((size_t)M * N * 4), c1((size_t)M * N * 4);
            const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
            CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
            auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
            std::vector<Variant> vs = {
                {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_STORE_F32, a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                {"256x256", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
            };
            if (split_variants) {
                vs.push_back({"128x256", [&](const void* wp, bool r) { return run_bf16<128, 256, 4, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }});
                vs.push_back({"128x128", [&](const void* wp, bool r) { return run_bf16<128, 128, 4, 2, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }});
                vs.push_back({"256x128", [&](const void* wp, bool r) { return run_bf16<256, 128, 4, 2, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }});
                vs.push_back({"64x128", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }});
            }
            snprintf(label, sizeof label, "1.5b  lm %-9s M=%4d N=%6d     ", what, M, N);
            bench_case(label, vs, w, std::max(2, reps / 8), st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                       [&] { return same_bytes(c0, c1); });
        };
        one(V, "whole", false);
        if (full > 0 && rest > 0) {
            one(full, "rounds", false);
            one(rest, "rest", true);
        }
    }
}

}  // namespace

int main(int argc, char** argv) {
    const int reps = argc > 1 ? atoi(argv[1]) : 20;
    const ModelShape shapes[] = {{"0.5b", 896, 14, 2, 64, 4864}, {"1.5b", 1536, 12, 2, 128, 8960},
                                 {"3b", 2048, 16, 2, 128, 11008}};
    if (argc > 2 && strcmp(argv[2], "small") == 0) {
        hipStream_t st;
        CK(hipStreamCreate(&st));
        std::mt19937 rng(7);
        printf("kernel timings in us at 16-64 rows (weights cold, median of interleaved rounds); alternatives "
               "marked = give the production bits\n");
        bench_small(shapes, 3, reps, st, rng);
        return 0;
    }
    if (argc > 2 && strcmp(argv[2], "split") == 0) {
        hipStream_t st;
        CK(hipStreamCreate(&st));
        std::mt19937 rng(7);
        printf("gate/up kernel timings in us by column range (weights cold, median of interleaved rounds)\n");
        bench_gu_split(shapes, 3, reps, st, rng);
        return 0;
    }
    const int batches[] = {256, 512, 768, 1024, 2048};
    hipStream_t st;
    CK(hipStreamCreate(&st));
    std::mt19937 rng(7);
    printf("kernel timings in us (weights cold, median of interleaved rounds); alternatives marked = give the "
           "production bits\n");
    char label[128];
    for (const ModelShape& sh : shapes) {
        const int d = sh.d, hq = sh.n_heads * sh.hd, qr = (sh.n_heads + 2 * sh.n_kv) * sh.hd;
        for (int M : batches) {
            // ---- output projection: C[M, d] = o[M, hq] . W_o[d, hq]^T (fp32, unsplit)
            {
                const int N = d, K = hq;
                Weights w(N, K, rng);
                Dev a((size_t)M * K * 2), c0((size_t)M * N * 4), c1((size_t)M * N * 4);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                const std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_STORE_F32, a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"lds128x64", [&](const void* wp, bool r) { return run_lds<128, 64, 2, 2, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"lds64x64", [&](const void* wp, bool r) { return run_lds<64, 64, 2, 2, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"lds64x128", [&](const void* wp, bool r) { return run_lds<64, 128, 2, 2, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"lds128x128", [&](const void* wp, bool r) { return run_lds<128, 128, 2, 2, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                };
                snprintf(label, sizeof label, "%-5s o    M=%4d N=%5d K=%5d     ", sh.name, M, N, K);
                bench_case(label, vs, w, reps, st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            }
            // ---- gate/up projection with the SwiGLU epilogue: h[M, ff] (bf16), unsplit
            if (M >= 512) {
                const int ff = sh.ff, N = 2 * ff, K = d;
                Weights w(N, K, rng);
                Dev a((size_t)M * K * 2), c0((size_t)M * ff * 2), c1((size_t)M * ff * 2);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                const std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_SWIGLU, a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"128x128w8", [&](const void* wp, bool r) { return run_bf16<128, 128, 4, 2, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"128x128w4", [&](const void* wp, bool r) { return run_bf16<128, 128, 2, 2, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"256x128w8", [&](const void* wp, bool r) { return run_bf16<256, 128, 4, 2, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"128x256w16", [&](const void* wp, bool r) { return run_bf16<128, 256, 4, 4, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"256x256w16", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 4, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                    {"256x256w8", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 2, 2, EPI_SWIGLU>(a.p, wp, out(r), M, N, K, ff, 1, 0, st); }},
                };
                snprintf(label, sizeof label, "%-5s gu   M=%4d N=%5d K=%5d     ", sh.name, M, N, K);
                bench_case(label, vs, w, reps, st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            }
            // ---- down projection: fp32 split-K partials [splits][M, d]
            if (M >= 512) {
                const int N = d, K = sh.ff;
                const int ns = gemm_pick_splits(1, EPI_STORE_F32, N, K);
                Weights w(N, K, rng);
                const size_t cn = (size_t)ns * M * N, ss = (size_t)M * N;
                Dev a((size_t)M * K * 2), c0(cn * 4), c1(cn * 4);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                const std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_STORE_F32, a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"128x256w16", [&](const void* wp, bool r) { return run_bf16<128, 256, 4, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"256x128w8", [&](const void* wp, bool r) { return run_bf16<256, 128, 4, 2, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"256x256w16", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"256x256w8", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 2, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"256x256w8t", [&](const void* wp, bool r) { return run_bf16<256, 256, 2, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                    {"lds128x128", [&](const void* wp, bool r) { return run_lds<128, 128, 2, 2, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, ns, ss, st); }},
                };
                snprintf(label, sizeof label, "%-5s down M=%4d N=%5d K=%5d s%d  ", sh.name, M, N, K, ns);
                bench_case(label, vs, w, reps, st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            }
            // ---- LM head (tied embedding, fp32 logits over the whole vocabulary), on the 1.5B shape
            if (M >= 512 && sh.d == 1536) {
                const int N = 151936, K = d;
                Weights w(N, K, rng);
                Dev a((size_t)M * K * 2), c0((size_t)M * N * 4), c1((size_t)M * N * 4);
                const auto ha = randn_bf16((size_t)M * K, 1.f, rng);
                CK(hipMemcpy(a.p, ha.data(), ha.size() * 2, hipMemcpyHostToDevice));
                auto out = [&](bool ref) { return ref ? c0.p : c1.p; };
                const std::vector<Variant> vs = {
                    {"production", [&](const void* wp, bool r) { return launch_gemm(1, EPI_STORE_F32, a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"256x256w16", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"256x256w8", [&](const void* wp, bool r) { return run_bf16<256, 256, 4, 2, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"256x256w8t", [&](const void* wp, bool r) { return run_bf16<256, 256, 2, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"128x256w16", [&](const void* wp, bool r) { return run_bf16<128, 256, 4, 4, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"256x128w8", [&](const void* wp, bool r) { return run_bf16<256, 128, 4, 2, 2, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                    {"lds128x128", [&](const void* wp, bool r) { return run_lds<128, 128, 2, 2, 4, EPI_STORE_F32>(a.p, wp, out(r), M, N, K, N, 1, 0, st); }},
                };
                snprintf(label, sizeof label, "%-5s lm   M=%4d N=%6d K=%4d    ", sh.name, M, N, K);
                bench_case(label, vs, w, std::max(2, reps / 8), st, [&] { CK(hipMemset(c1.p, 0xFF, c1.n)); },
                           [&] { return same_bytes(c0, c1); });
            }
            // ---- QKV projection with bias, RoPE and the KV append (fused epilogue)
            if (gemm_qkv_fusable(1, sh.n_heads, sh.n_kv, sh.hd)) {
                QkvCase c(sh, M, rng);
                const int N = qr, K = d;
                auto args = [&](bool ref) { return c.args(ref); };
                const void* A = c.a.p;
                const std::vector<Variant> vs = {
                    // the production path: fused above its size threshold, else the unfused GEMM + RoPE kernel
                    {"production", [&](const void* wp, bool r) -> hipError_t {
                         if (gemm_qkv_fuse_pays(M, N)) return launch_gemm_qkv_rope(A, wp, M, N, K, args(r), st);
                         return run_bf16<64, 128, 2, 4, 2, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, args(r));
                     }},
                    {"lds64x128", [&](const void* wp, bool r) { return run_lds<64, 128, 2, 2, 4, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, args(r)); }},
                    {"lds64x128s3", [&](const void* wp, bool r) { return run_lds<64, 128, 2, 2, 3, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, args(r)); }},
                    {"64x128pd3", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 4, 3, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, args(r)); }},
                    {"64x128pd4", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 4, 4, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, args(r)); }},
                    {"64x128w4pd3", [&](const void* wp, bool r) { return run_bf16<64, 128, 2, 2, 3, EPI_QKV_ROPE>(A, wp, nullptr, M, N, K, 0, 1, 0, st, args(r)); }},
                };
                snprintf(label, sizeof label, "%-5s qkv  M=%4d N=%5d K=%5d     ", sh.name, M, N, K);
                c.run(label, vs, reps, st);
            }
        }
    }
    return 0;
}
