// Native rollout benchmark over the C ABI alone (no Python, no torch): synthetic
// bfloat16 weights of a Qwen2.5-shaped decoder, prompts duplicated into groups,
// one warm-up and one timed dash_rollout, then the advantage filter of synthetic
// rewards.  Besides timing, it is the program hardware-counter runs of the rollout
// kernels profile (a plain device copy of known size runs first, as the reference
// for byte counters), and a usage example of include/dash.h.
// --attn 1 then compares decode attention per row (dash_decode_step) with the
// prefix-shared form (dash_decode_step_grouped, each prompt's G samples one group)
// on the same batch at three context lengths: the attention kernels' time per layer
// from the library's kernel-class timing, and the whole step's time.
//
//   dash_native_bench [--layers 28] [--d 1536] [--heads 12] [--kv 2] [--hd 128] [--ff 8960]
//                     [--vocab 151936] [--prompts 128] [--group 8] [--prompt 256] [--gen 1024]
//                     [--graph 1] [--copy-mib 1024] [--rollouts 2] [--attn 0]
#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "dash.h"

namespace {

#define CHECK_HIP(x)                                                                           \
    do {                                                                                       \
        hipError_t e_ = (x);                                                                   \
        if (e_ != hipSuccess) {                                                                \
            std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));                \
            std::exit(2);                                                                      \
        }                                                                                      \
    } while (0)
#define CHECK_DASH(x)                                                                          \
    do {                                                                                       \
        int s_ = (x);                                                                          \
        if (s_ != DASH_OK) {                                                                   \
            std::fprintf(stderr, "%s: %s (%s)\n", #x, dash_status_str(s_), dash_last_error()); \
            std::exit(3);                                                                      \
        }                                                                                      \
    } while (0)

__device__ uint32_t mix(uint32_t x) {  // integer hash (xorshift-multiply rounds)
    x ^= x >> 16;
    x *= 0x7feb352dU;
    x ^= x >> 15;
    x *= 0x846ca68bU;
    x ^= x >> 16;
    return x;
}

// Uniform values in [-a, a] (a = 0.02 * sqrt(3): standard deviation 0.02), rounded to bf16.
__global__ void fill_bf16(uint16_t* p, size_t n, uint32_t seed, float a) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        const float u = (float)(mix((uint32_t)i ^ mix(seed + (uint32_t)(i >> 32))) >> 8) * (1.0f / 16777216.0f);
        uint32_t b;
        const float f = (2.0f * u - 1.0f) * a;
        std::memcpy(&b, &f, 4);
        b += 0x7FFFu + ((b >> 16) & 1u);
        p[i] = (uint16_t)(b >> 16);
    }
}

__global__ void fill_u16(uint16_t* p, size_t n, uint16_t v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

__global__ void fill_tokens(int32_t* p, size_t n, int vocab, uint32_t seed) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = (int32_t)(mix((uint32_t)i ^ seed) % (uint32_t)vocab);
}

__global__ void fill_rewards(float* p, size_t n, uint32_t seed) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = (float)(mix((uint32_t)i ^ seed) & 1u);
}

int arg(int argc, char** argv, const char* name, int def) {
    for (int i = 1; i + 1 < argc; ++i)
        if (!std::strcmp(argv[i], name)) return std::atoi(argv[i + 1]);
    return def;
}

void* dev_alloc(size_t bytes) {
    void* p = nullptr;
    CHECK_HIP(hipMalloc(&p, bytes ? bytes : 256));
    return p;
}

}  // namespace

int main(int argc, char** argv) {
    dash_model_desc d{};
    d.n_layers = arg(argc, argv, "--layers", 28);
    d.d_model = arg(argc, argv, "--d", 1536);
    d.n_heads = arg(argc, argv, "--heads", 12);
    d.n_kv_heads = arg(argc, argv, "--kv", 2);
    d.head_dim = arg(argc, argv, "--hd", 128);
    d.d_ff = arg(argc, argv, "--ff", 8960);
    d.vocab = arg(argc, argv, "--vocab", 151936);
    d.dtype = DASH_BF16;
    d.rope_theta = 1e6f;
    d.rms_eps = 1e-6f;
    const int n_prompts = arg(argc, argv, "--prompts", 128), G = arg(argc, argv, "--group", 8);
    const int P = arg(argc, argv, "--prompt", 256), T = arg(argc, argv, "--gen", 1024);
    const int use_graph = arg(argc, argv, "--graph", 1), copy_mib = arg(argc, argv, "--copy-mib", 1024);
    const int rollouts = arg(argc, argv, "--rollouts", 2), attn_cmp = arg(argc, argv, "--attn", 0);
    const int N = n_prompts * G, ps = 32;

    hipStream_t st;
    CHECK_HIP(hipStreamCreate(&st));
    if (copy_mib > 0) {  // reference for byte counters: a plain device-to-device copy of known size
        const size_t bytes = (size_t)copy_mib << 20;
        void* a = dev_alloc(bytes);
        void* b = dev_alloc(bytes);
        CHECK_HIP(hipMemcpyAsync(b, a, bytes, hipMemcpyDeviceToDevice, st));
        CHECK_HIP(hipStreamSynchronize(st));
        CHECK_HIP(hipFree(a));
        CHECK_HIP(hipFree(b));
        std::printf("copy calibration: %d MiB device-to-device\n", copy_mib);
    }

    // weights
    const int nw = dash_weight_count(&d);
    const size_t qr = (size_t)(d.n_heads + 2 * d.n_kv_heads) * d.head_dim;
    std::vector<size_t> elems(nw, 0);
    std::vector<int> is_norm(nw, 0);
    elems[0] = (size_t)d.vocab * d.d_model;
    elems[1] = d.d_model;
    is_norm[1] = 1;
    for (int l = 0; l < d.n_layers; ++l) {
        const int b = 3 + 7 * l;
        elems[b + 0] = d.d_model;
        is_norm[b + 0] = 1;
        elems[b + 1] = qr * d.d_model;
        elems[b + 2] = qr;
        elems[b + 3] = (size_t)d.d_model * d.n_heads * d.head_dim;
        elems[b + 4] = d.d_model;
        is_norm[b + 4] = 1;
        elems[b + 5] = (size_t)2 * d.d_ff * d.d_model;
        elems[b + 6] = (size_t)d.d_model * d.d_ff;
    }
    std::vector<void*> w(nw, nullptr);
    for (int i = 0; i < nw; ++i) {
        if (!elems[i]) continue;  // the tied LM head stays NULL
        w[i] = dev_alloc(elems[i] * 2);
        if (is_norm[i])
            fill_u16<<<256, 256, 0, st>>>((uint16_t*)w[i], elems[i], 0x3F80);  // 1.0
        else
            fill_bf16<<<1024, 256, 0, st>>>((uint16_t*)w[i], elems[i], 977u * i + 1u, 0.0346410f);
        CHECK_HIP(hipGetLastError());
    }
    dash_model* model = nullptr;
    CHECK_DASH(dash_model_create(&d, (const void* const*)w.data(), nw, &model));

    // KV cache: shared prompt pages once per prompt, private pages for the rest
    const int max_ctx = P + T;
    const size_t pages = (size_t)n_prompts * (P / ps) + (size_t)N * ((max_ctx + ps - 1) / ps - P / ps) + 8;
    const size_t page_bytes = dash_kv_page_bytes(model, ps);
    void* pool = dev_alloc(pages * page_bytes);
    CHECK_HIP(hipMemsetAsync(pool, 0, pages * page_bytes, st));
    void* table = dev_alloc(dash_kv_table_bytes(N, max_ctx, ps));
    dash_kv* kv = nullptr;
    CHECK_DASH(dash_kv_create(model, pool, pages * page_bytes, ps, N, max_ctx, table, st, &kv));

    const size_t ws_bytes = dash_rollout_workspace_bytes(model, n_prompts, P, G, max_ctx);
    void* ws = dev_alloc(ws_bytes);
    int32_t* prompts = (int32_t*)dev_alloc((size_t)n_prompts * P * 4);
    fill_tokens<<<256, 256, 0, st>>>(prompts, (size_t)n_prompts * P, d.vocab, 12345u);
    int32_t* toks = (int32_t*)dev_alloc((size_t)N * T * 4);
    float* lps = (float*)dev_alloc((size_t)N * T * 4);
    float* rewards = (float*)dev_alloc((size_t)N * 4);
    fill_rewards<<<64, 256, 0, st>>>(rewards, N, 777u);
    float* adv = (float*)dev_alloc((size_t)N * 4);
    int32_t* kept = (int32_t*)dev_alloc((size_t)N * 4);
    int32_t* kept_n = (int32_t*)dev_alloc(4);
    CHECK_HIP(hipStreamSynchronize(st));
    std::printf("model %d layers, d %d, vocab %d; %d sequences (%d prompts x %d), prompt %d, gen %d; pool %.1f GiB\n",
                d.n_layers, d.d_model, d.vocab, N, n_prompts, G, P, T, pages * page_bytes / 1073741824.0);

    for (int r = 0; r < rollouts; ++r) {
        const auto t0 = std::chrono::steady_clock::now();
        CHECK_DASH(dash_rollout(model, kv, prompts, n_prompts, P, G, T, nullptr, 1.0f, 7u, toks, lps, use_graph, ws,
                                ws_bytes, st));
        CHECK_DASH(dash_group_advantage_filter(rewards, n_prompts, G, DASH_ADV_STD_SAMPLE, 1e-6f, 0.1f, adv, kept,
                                               kept_n, st));
        CHECK_HIP(hipStreamSynchronize(st));
        const double s = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        std::printf("rollout %d: %.3f s, %.1f generated tokens/s\n", r, s, (double)N * T / s);
    }

    if (attn_cmp) {
        // one prefill of the whole batch, then decode steps at fixed contexts (each step
        // rewrites the K/V of its position, so the context stays the same)
        std::vector<int32_t> slots(N);
        for (int i = 0; i < N; ++i) slots[i] = i;
        float* logits = (float*)dev_alloc((size_t)N * d.vocab * 4);
        int32_t* d_slot = (int32_t*)dev_alloc((size_t)N * 4);
        int32_t* d_pos = (int32_t*)dev_alloc((size_t)N * 4);
        int32_t* d_tok = (int32_t*)dev_alloc((size_t)N * 4);
        int32_t* d_off = (int32_t*)dev_alloc((size_t)(n_prompts + 1) * 4);
        std::vector<int32_t> off(n_prompts + 1);
        for (int i = 0; i <= n_prompts; ++i) off[i] = i * G;
        CHECK_HIP(hipMemcpy(d_slot, slots.data(), (size_t)N * 4, hipMemcpyHostToDevice));
        CHECK_HIP(hipMemcpy(d_off, off.data(), off.size() * 4, hipMemcpyHostToDevice));
        fill_tokens<<<64, 256, 0, st>>>(d_tok, N, d.vocab, 99u);
        CHECK_DASH(dash_prefill(model, kv, prompts, n_prompts, P, G, slots.data(), logits, ws, ws_bytes, st));
        const int shared = P / ps * ps;
        const int reps = 5;
        for (const int c : {P + 1, (P + max_ctx) / 2, max_ctx}) {
            CHECK_DASH(dash_kv_reserve(kv, slots.data(), N, c, st));
            std::vector<int32_t> pos(N, c - 1);
            CHECK_HIP(hipMemcpy(d_pos, pos.data(), (size_t)N * 4, hipMemcpyHostToDevice));
            double attn_us[2], step_ms[2];
            for (int v = 0; v < 2; ++v) {
                auto step = [&]() {
                    if (v == 0) CHECK_DASH(dash_decode_step(model, kv, d_tok, d_slot, d_pos, N, logits, ws, ws_bytes, st));
                    else
                        CHECK_DASH(dash_decode_step_grouped(model, kv, d_tok, d_slot, d_pos, N, d_off, n_prompts, G,
                                                            shared, logits, ws, ws_bytes, st));
                };
                step();
                step();
                CHECK_HIP(hipStreamSynchronize(st));
                const auto t0 = std::chrono::steady_clock::now();
                for (int r = 0; r < reps; ++r) step();
                CHECK_HIP(hipStreamSynchronize(st));
                step_ms[v] = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count() / reps;
                double ms[DASH_K_COUNT];
                int64_t n[DASH_K_COUNT];
                CHECK_DASH(dash_profile_read(ms, n, 1));
                CHECK_DASH(dash_profile_enable(1u << DASH_K_ATTN));
                for (int r = 0; r < reps; ++r) step();
                CHECK_DASH(dash_profile_read(ms, n, 1));
                CHECK_DASH(dash_profile_enable(0));
                attn_us[v] = ms[DASH_K_ATTN] * 1e3 / (double)(n[DASH_K_ATTN] ? n[DASH_K_ATTN] : 1);
            }
            std::printf("context %d: decode attention per layer %.1f us per row, %.1f us prefix-shared; "
                        "step %.2f ms vs %.2f ms\n", c, attn_us[0], attn_us[1], step_ms[0], step_ms[1]);
        }
        for (void* p : {(void*)logits, (void*)d_slot, (void*)d_pos, (void*)d_tok, (void*)d_off}) CHECK_HIP(hipFree(p));
    }

    dash_kv_destroy(kv);
    dash_model_destroy(model);
    for (void* p : w)
        if (p) CHECK_HIP(hipFree(p));
    for (void* p : {pool, table, ws, (void*)prompts, (void*)toks, (void*)lps, (void*)rewards, (void*)adv,
                    (void*)kept, (void*)kept_n})
        CHECK_HIP(hipFree(p));
    CHECK_HIP(hipStreamDestroy(st));
    return 0;
}
