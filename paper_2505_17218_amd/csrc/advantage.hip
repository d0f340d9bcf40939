// GRPO group advantage with the gradient-filter compaction, and the live-row
// compaction of ragged decoding.  Both are tiny (N <= a few thousand): one
// workgroup of 1024 threads walks the input in chunks, and a ballot / mbcnt
// prefix inside each wave plus an LDS scan across the 16 waves gives every
// kept element its output slot, so kept indices come out in ascending order
// with no atomics (deterministic).
//
// Group statistics (groups of G <= 64): samples are spread over "virtual
// lanes", P2 = next power of two >= G lanes per group with the tail zero, so a
// group sits in an aligned run of P2 lanes of one wave and an xor butterfly
// (offsets 1, 2, 4, ...) forms the pairwise sum, adjacent pairs first.  Groups
// with 64 < G <= 1024 use the same tree in LDS, one group at a time; larger
// groups (up to 65536, e.g. the single-path baseline over a whole batch) give
// each thread a power-of-two run of the group, summed pairwise with a binary
// counter, then the LDS tree over the threads: the same tree, level by level.
// Modes: mean-centred (Eq. (4)), / (std + eps) with ddof 0 or 1, and the
// leave-one-out baseline r - (S - r) / (G - 1).
// Built with -ffp-contract=off: see sampler_math.h.
#include "common.h"
#include "kernels.h"
#include "sampler_math.h"

namespace dash {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

// Exclusive prefix of `flag` over the workgroup, in thread order; returns the
// prefix and writes the total to *total.  `scan` is LDS of kWaves ints.
DASH_DEV int block_excl_scan(bool flag, int* scan, int* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t bal = __ballot(flag);
    const int in_wave = __popcll(bal & ((1ull << lane) - 1ull));
    __syncthreads();
    if (lane == 0) scan[w] = __popcll(bal);
    __syncthreads();
    int before = 0, tot = 0;
    for (int i = 0; i < kWaves; ++i) {
        const int c = scan[i];
        before += i < w ? c : 0;
        tot += c;
    }
    *total = tot;
    return before + in_wave;
}

constexpr int kModeLoo = 3;

// Leave-one-out advantage from the reward x and its group's sum S.
DASH_DEV float adv_loo(float x, float S, int G) { return x - div_rn(S - x, (float)(G - 1)); }

DASH_DEV float adv_of(float d, float ss, int G, int mode, float eps) {
    if (mode == 0) return d;
    const int ddof = mode == 2 ? 1 : 0;
    float sd = 0.f;
    if (G - ddof > 0) sd = sqrt_rn(div_rn(ss, (float)(G - ddof)));
    return div_rn(d, sd + eps);
}

__global__ void __launch_bounds__(kThreads) adv_filter_wave_k(const float* __restrict__ r, int n_groups, int G, int P2,
                                                              int mode, float eps, float tau, float* __restrict__ adv,
                                                              int32_t* __restrict__ kept, int32_t* __restrict__ count) {
    __shared__ int scan[kWaves];
    const int total_v = n_groups * P2;
    int base = 0;
    for (int c0 = 0; c0 < total_v; c0 += kThreads) {
        const int v = c0 + threadIdx.x;
        const int grp = v / P2, j = v % P2;
        const bool valid = v < total_v && j < G;
        const int n = grp * G + j;
        const float x = valid ? r[n] : 0.f;
        float s = x;
        for (int o = 1; o < P2; o <<= 1) s = s + __shfl_xor(s, o, 64);
        const float mu = div_rn(s, (float)G);
        const float d = x - mu;
        float q = valid ? d * d : 0.f;
        if (mode != 0 && mode != kModeLoo)
            for (int o = 1; o < P2; o <<= 1) q = q + __shfl_xor(q, o, 64);
        const float a = mode == kModeLoo ? adv_loo(x, s, G) : adv_of(d, q, G, mode, eps);
        const bool keep = valid && fabsf(a) >= tau;
        if (valid) adv[n] = a;
        int tot;
        const int at = block_excl_scan(keep, scan, &tot);
        if (keep) kept[base + at] = n;
        base += tot;
    }
    if (threadIdx.x == 0) *count = base;
}

__global__ void __launch_bounds__(kThreads) adv_filter_lds_k(const float* __restrict__ r, int n_groups, int G, int P2,
                                                             int mode, float eps, float tau, float* __restrict__ adv,
                                                             int32_t* __restrict__ kept, int32_t* __restrict__ count) {
    __shared__ float buf[kThreads];
    __shared__ int scan[kWaves];
    const int j = threadIdx.x;
    int base = 0;
    for (int grp = 0; grp < n_groups; ++grp) {
        const bool valid = j < G;
        const int n = grp * G + j;
        const float x = valid ? r[n] : 0.f;
        if (j < P2) buf[j] = x;
        __syncthreads();
        for (int half = P2 >> 1; half >= 1; half >>= 1) {  // a[i] = a[2i] + a[2i+1]
            float t = 0.f;
            if (j < half) t = buf[2 * j] + buf[2 * j + 1];
            __syncthreads();
            if (j < half) buf[j] = t;
            __syncthreads();
        }
        const float S = buf[0];
        const float mu = div_rn(S, (float)G);
        const float d = x - mu;
        __syncthreads();
        if (j < P2) buf[j] = valid ? d * d : 0.f;
        __syncthreads();
        for (int half = P2 >> 1; half >= 1; half >>= 1) {
            float t = 0.f;
            if (j < half) t = buf[2 * j] + buf[2 * j + 1];
            __syncthreads();
            if (j < half) buf[j] = t;
            __syncthreads();
        }
        const float a = mode == kModeLoo ? adv_loo(x, S, G) : adv_of(d, buf[0], G, mode, eps);
        __syncthreads();
        const bool keep = valid && fabsf(a) >= tau;
        if (valid) adv[n] = a;
        int tot;
        const int at = block_excl_scan(keep, scan, &tot);
        if (keep) kept[base + at] = n;
        base += tot;
    }
    if (threadIdx.x == 0) *count = base;
}

constexpr int kMaxRunLog = 6;  // runs of up to 64 samples per thread: groups up to 65536

// Pairwise sum of val(0 .. kThreads * c - 1) (c a power of two <= 2^kMaxRunLog):
// thread t sums its run [t c, (t + 1) c) with a binary counter (a finished pair
// of 2^k-sums merges left + right, as one level of the tree), then LDS adds
// adjacent thread results level by level.  Returns the total in every thread.
template <typename F>
DASH_DEV float block_pairwise_sum(F val, int c, float* buf) {
    const int t = threadIdx.x;
    float st[kMaxRunLog];
    float run = 0.f;
    for (int i = 0; i < c; ++i) {
        float v = val(t * c + i);
        bool placed = false;
#pragma unroll
        for (int k = 0; k < kMaxRunLog; ++k) {
            if (!placed) {
                if ((i >> k) & 1) {
                    v = st[k] + v;
                } else {
                    st[k] = v;
                    placed = true;
                }
            }
        }
        run = v;  // after the last element every level has merged: the run's total
    }
    __syncthreads();
    buf[t] = run;
    __syncthreads();
    for (int half = kThreads >> 1; half >= 1; half >>= 1) {
        float x = 0.f;
        if (t < half) x = buf[2 * t] + buf[2 * t + 1];
        __syncthreads();
        if (t < half) buf[t] = x;
        __syncthreads();
    }
    const float total = buf[0];
    __syncthreads();
    return total;
}

__global__ void __launch_bounds__(kThreads) adv_filter_big_k(const float* __restrict__ r, int n_groups, int G, int P2,
                                                             int mode, float eps, float tau, float* __restrict__ adv,
                                                             int32_t* __restrict__ kept, int32_t* __restrict__ count) {
    __shared__ float buf[kThreads];
    __shared__ int scan[kWaves];
    const int c = P2 / kThreads;
    int base = 0;
    for (int grp = 0; grp < n_groups; ++grp) {
        const float* rg = r + (size_t)grp * G;
        const float S = block_pairwise_sum([&](int j) { return j < G ? rg[j] : 0.f; }, c, buf);
        const float mu = div_rn(S, (float)G);
        float ss = 0.f;
        if (mode != 0 && mode != kModeLoo)
            ss = block_pairwise_sum(
                [&](int j) {
                    if (j >= G) return 0.f;
                    const float d = rg[j] - mu;
                    return d * d;
                },
                c, buf);
        for (int c0 = 0; c0 < G; c0 += kThreads) {
            const int j = c0 + threadIdx.x;
            const bool valid = j < G;
            const float x = valid ? rg[j] : 0.f;
            const float a = mode == kModeLoo ? adv_loo(x, S, G) : adv_of(x - mu, ss, G, mode, eps);
            const bool keep = valid && fabsf(a) >= tau;
            if (valid) adv[(size_t)grp * G + j] = a;
            int tot;
            const int at = block_excl_scan(keep, scan, &tot);
            if (keep) kept[base + at] = grp * G + j;
            base += tot;
        }
    }
    if (threadIdx.x == 0) *count = base;
}

__global__ void __launch_bounds__(kThreads)
live_compact_k(const int32_t* __restrict__ tok, const int32_t* __restrict__ slot, const int32_t* __restrict__ pos,
               const int32_t* __restrict__ step, const int32_t* __restrict__ uid, const int32_t* __restrict__ budget,
               int eos_id, int n, int32_t* __restrict__ tok_o, int32_t* __restrict__ slot_o,
               int32_t* __restrict__ pos_o, int32_t* __restrict__ step_o, int32_t* __restrict__ uid_o,
               int32_t* __restrict__ count) {
    __shared__ int scan[kWaves];
    int base = 0;
    for (int c0 = 0; c0 < n; c0 += kThreads) {
        const int i = c0 + threadIdx.x;
        bool live = false;
        if (i < n) live = (step[i] + 1 < budget[uid[i]]) && !(eos_id >= 0 && tok[i] == eos_id);
        int tot;
        const int at = block_excl_scan(live, scan, &tot);
        if (live) {
            const int o = base + at;
            tok_o[o] = tok[i];
            slot_o[o] = slot[i];
            pos_o[o] = pos[i] + 1;
            step_o[o] = step[i] + 1;
            uid_o[o] = uid[i];
        }
        base += tot;
    }
    if (threadIdx.x == 0) *count = base;
}

// Loss over the kept samples, float64, reproducible bit for bit.  Each thread takes
// kept samples k, k + 256, ... and sums a sample's per-token values in token order;
// the 256 partials are then added as a pairwise tree.  Surrogate: A S (PG, no old log-probs) or PPO's
// min(rho A, clip(rho, 1 - eps, 1 + eps) A) with rho = exp(S - S_old); the KL sums
// (if given) enter with weight beta.  stats[4 n ..] = (S, S_old, KL, dloss/dS).
__global__ void __launch_bounds__(kThreads)
policy_loss_k(const float* __restrict__ lp, const float* __restrict__ lp_old, const float* __restrict__ kl, int64_t ld,
              int T, const int32_t* __restrict__ len, const float* __restrict__ adv,
              const int32_t* __restrict__ kept, const int32_t* __restrict__ kept_count, int n_total, double clip_eps,
              double beta, double* __restrict__ loss, double* __restrict__ seq_lp, double* __restrict__ stats) {
    __shared__ double buf[kThreads], kbuf[kThreads];
    const int K = *kept_count;
    const double N = (double)n_total;
    double acc = 0.0, kacc = 0.0;
    for (int k = threadIdx.x; k < K; k += kThreads) {
        const int n = kept[k];
        const int L = len ? min(max(len[n], 0), T) : T;
        const float* row = lp + (int64_t)n * ld;
        double S = 0.0;
        for (int t = 0; t < L; ++t) S += (double)row[t];
        double S_old = S, Kn = 0.0;
        if (lp_old) {
            const float* ro = lp_old + (int64_t)n * ld;
            S_old = 0.0;
            for (int t = 0; t < L; ++t) S_old += (double)ro[t];
        }
        if (kl) {
            const float* rk = kl + (int64_t)n * ld;
            for (int t = 0; t < L; ++t) Kn += (double)rk[t];
        }
        const double A = (double)adv[n];
        double sur, w;
        if (!lp_old) {
            sur = A * S;
            w = -A / N;
        } else {
            const double rho = exp(S - S_old);
            const double un = rho * A;
            const double cl = fmin(fmax(rho, 1.0 - clip_eps), 1.0 + clip_eps) * A;
            sur = fmin(un, cl);
            w = un <= cl ? -A * rho / N : 0.0;
        }
        if (seq_lp) seq_lp[n] = S;
        if (stats) {
            stats[4 * (int64_t)n + 0] = S;
            stats[4 * (int64_t)n + 1] = S_old;
            stats[4 * (int64_t)n + 2] = Kn;
            stats[4 * (int64_t)n + 3] = w;
        }
        acc += sur;
        kacc += Kn;
    }
    buf[threadIdx.x] = acc;
    kbuf[threadIdx.x] = kacc;
    __syncthreads();
    const int tid = threadIdx.x;
    for (int half = kThreads >> 1; half >= 1; half >>= 1) {
        double x = 0.0, y = 0.0;
        if (tid < half) {
            x = buf[2 * tid] + buf[2 * tid + 1];
            y = kbuf[2 * tid] + kbuf[2 * tid + 1];
        }
        __syncthreads();
        if (tid < half) {
            buf[tid] = x;
            kbuf[tid] = y;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        double l = -buf[0] / N;
        if (kl) l += beta * kbuf[0] / N;
        *loss = l;
    }
}

}  // namespace

hipError_t launch_policy_loss(const float* lp, const float* lp_old, const float* kl, int64_t ld, int T,
                              const int32_t* len, const float* adv, const int32_t* kept, const int32_t* kept_count,
                              int n_total, double clip_eps, double beta, double* loss, double* seq_lp, double* stats,
                              hipStream_t st) {
    policy_loss_k<<<1, kThreads, 0, st>>>(lp, lp_old, kl, ld, T, len, adv, kept, kept_count, n_total, clip_eps, beta,
                                          loss, seq_lp, stats);
    return hipGetLastError();
}

hipError_t launch_pg_loss(const float* lp, int64_t ld, int T, const int32_t* len, const float* adv,
                          const int32_t* kept, const int32_t* kept_count, int n_total, double* loss, double* seq_lp,
                          hipStream_t st) {
    return launch_policy_loss(lp, nullptr, nullptr, ld, T, len, adv, kept, kept_count, n_total, 0.0, 0.0, loss, seq_lp,
                              nullptr, st);
}

hipError_t launch_group_advantage_filter(const float* r, int n_groups, int group, int mode, float eps, float tau,
                                         float* adv, int32_t* kept, int32_t* count, hipStream_t st) {
    int P2 = 1;
    while (P2 < group) P2 <<= 1;
    if (P2 > (kThreads << kMaxRunLog)) return hipErrorInvalidValue;
    if (P2 <= 64)
        adv_filter_wave_k<<<1, kThreads, 0, st>>>(r, n_groups, group, P2, mode, eps, tau, adv, kept, count);
    else if (P2 <= kThreads)
        adv_filter_lds_k<<<1, kThreads, 0, st>>>(r, n_groups, group, P2, mode, eps, tau, adv, kept, count);
    else
        adv_filter_big_k<<<1, kThreads, 0, st>>>(r, n_groups, group, P2, mode, eps, tau, adv, kept, count);
    return hipGetLastError();
}

hipError_t launch_live_compact(const int32_t* tok, const int32_t* slot, const int32_t* pos, const int32_t* step,
                               const int32_t* uid, const int32_t* budget, int eos_id, int n, int32_t* tok_o,
                               int32_t* slot_o, int32_t* pos_o, int32_t* step_o, int32_t* uid_o, int32_t* count,
                               hipStream_t st) {
    live_compact_k<<<1, kThreads, 0, st>>>(tok, slot, pos, step, uid, budget, eos_id, n, tok_o, slot_o, pos_o, step_o,
                                           uid_o, count);
    return hipGetLastError();
}

}  // namespace dash
