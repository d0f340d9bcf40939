// Vocab-wide temperature sampling: Gumbel-max with counter-based Philox noise.
//
// One workgroup of kThreads (1024) threads per row.  Thread t walks vocab entries
// in groups of four (one Philox call yields the noise of four consecutive
// entries) with a stride of kThreads groups, so a wave reads 1 KB of logits per
// step, coalesced.  Each thread keeps its best (score, index) and an online (max,
// sum of exp) for the log-normaliser; waves merge with xor shuffles, then LDS
// merges the sixteen waves in order.  Ties in the score go to the smaller vocab index.  Built with
// -ffp-contract=off: see sampler_math.h.
//
// Screening.  The exact noise -ln(-ln u) (two correctly rounded divisions) is
// the expensive part, so every entry is first scored with a cheap noise from the
// hardware logarithm, whose distance to the exact noise is below kScreenTol for
// every value u can take (checked exhaustively by dash_sampler_check).  With the
// fp32 rounding of the sums added, each entry's exact score lies within a margin
// of its cheap score.  The wave keeps a shared lower bound on the best exact
// score seen so far (exact scores of evaluated entries, cheap score minus margin
// of the rest); an entry whose cheap score plus margin falls below it cannot be
// the argmax and is skipped, every other entry gets its exact score.  The winner
// is therefore always evaluated exactly: tokens are bit-identical to scoring
// every entry exactly.  Before the cheap noise, an upper bound on the exact noise
// read off the random word's leading ones (noise_bound) already rules out almost
// every entry once the bound has risen, without any logarithm.
#include <cstring>

#include "common.h"
#include "kernels.h"
#include "sampler_math.h"

namespace dash {

namespace {

// Threads per row of the sampler and of the log-prob gather (the two must sum a row's
// log-normaliser in the same order).  1024 rather than 256: the sampler is VALU-bound,
// and 256 threads per row left most SIMDs idle at small batches (measured sampling time
// -59% at 64 rows, -19% at 1024 rows).
constexpr int kThreads = 1024;
constexpr int kKlThreads = 256;  // row KL (its fp64 sums need the registers of 4 waves per SIMD)
// bound on |cheap noise - exact noise|: 8x the exhaustive maximum (1.9e-6) on gfx950
constexpr float kScreenTol = 1.6e-5f;

DASH_DEV bool better(float s, int i, float bs, int bi) { return s > bs || (s == bs && i < bi); }

// One entry x into an online (max mx, sum z of e^(v - mx)): a new maximum rescales the
// sum (z e^(mx - x) + 1), any other entry adds e^(x - mx).  Both cases are one
// exponential of -|x - mx| (x - mx and mx - x are exact negations), chosen without a
// branch; the sampler and the log-prob gather share it, so they sum in the same way.
DASH_DEV void lse_push(float& mx, float& z, float x) {
    const float d = x - mx;  // +inf while mx is -inf
    const float e = __expf(-fabsf(d));
    const bool up = d > 0.f;
    z = up ? z * e + 1.0f : z + e;
    mx = up ? x : mx;
}

// Non-temporal (streaming) vector load, for logits read once.
DASH_DEV float4 load_stream4(const float* p) {
    const f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p));
    return make_float4(v[0], v[1], v[2], v[3]);
}

// -ln(-ln u) with the hardware logarithm; u = ((x >> 8) | 1) 2^-24 as in gumbel_from_bits
DASH_DEV float cheap_gumbel(uint32_t x) {
    const float u = (float)((x >> 8) | 1u) * (1.0f / 16777216.0f);
    return -__logf(-__logf(u));
}

// Interval half-width around a cheap score sa that contains the exact score.
DASH_DEV float screen_margin(float sa) { return kScreenTol + fabsf(sa) * (1.0f / 1048576.0f); }

// Upper bound on the exact noise of the random word x, from its leading ones alone:
// k leading ones leave u < 1 - 2^-(k+1), and -ln(1 - e) >= e gives
// g = -ln(-ln u) < -ln(2^-(k+1)) = (k+1) ln 2 (0.6931472f is above ln 2; at most 25
// terms, so the product's rounding stays far inside the margin added by the caller).
DASH_DEV float noise_bound(uint32_t x) { return (float)(min(__clz(~x), 24) + 1) * 0.6931472f; }

// Maximum over the wave's 64 lanes, returned wave-uniform: data-parallel-primitive moves
// within each row of 16 lanes (quad swaps, then the half-row and row mirrors), row
// broadcasts up to lane 63, then that lane read into a scalar register.  Every step is a
// register move inside the vector unit; exchanges through LDS (one per xor distance)
// each waited for the LDS round trip.
DASH_DEV float wave_max_f(float v) {
    int x = __float_as_int(v);
    x = __float_as_int(fmaxf(__int_as_float(x), __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false))));
    x = __float_as_int(fmaxf(__int_as_float(x), __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false))));
    x = __float_as_int(fmaxf(__int_as_float(x), __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false))));
    x = __float_as_int(fmaxf(__int_as_float(x), __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false))));
    // row_bcast15 into rows 1 and 3, row_bcast31 into rows 2 and 3 (rows not in the mask keep x)
    x = __float_as_int(fmaxf(__int_as_float(x), __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false))));
    x = __float_as_int(fmaxf(__int_as_float(x), __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x143, 0xC, 0xF, false))));
    return __int_as_float(__builtin_amdgcn_readlane(x, 63));
}

// Raw words of entries 4g .. 4g+3 of a row through a buffer resource over the row:
// the same load instructions for every lane and every g, no branch (entries past the
// resource read as zeros without a memory access), so the compiler's wait before a
// group is used covers only the loads issued before it, not the ones still ahead.
// VEC4 rows (16-byte aligned, vocab % 4 == 0) are read in 16-byte groups, other rows
// word by word.  The caller masks entries >= vocab (vocab_mask).
DASH_DEV __amdgpu_buffer_rsrc_t row_rsrc(const float* row, int vocab) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(row), 0, vocab * 4, kBufferDword3);
}
template <bool VEC4>
DASH_DEV void fetch_raw4(__amdgpu_buffer_rsrc_t rs, int g, float (&l)[4]) {
    const uint32_t off = (uint32_t)g * 16u;
    if constexpr (VEC4) {
        const f32x4_t v = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
        l[0] = v[0]; l[1] = v[1]; l[2] = v[2]; l[3] = v[3];
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            l[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off + 4u * j, 0, 0));
    }
}
// A register copy the compiler must keep.  The loop below copies a group out of its
// load registers before the next load into them; with a plain copy the compiler kept
// the group in the load registers, sent the next load elsewhere and moved the sets
// back at the end of the iteration, which needs every load to have landed.
DASH_DEV float copy_out(float v) {
    float r;
    asm volatile("v_mov_b32 %0, %1" : "=v"(r) : "v"(v));
    return r;
}

// Entries at or past vocab become NaN (skipped like any non-finite logit).
DASH_DEV void vocab_mask(float (&l)[4], int g, int vocab) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (4 * g + j >= vocab) l[j] = NAN;
}

// Entries 4g .. 4g+3 of a row (NaN past the vocabulary or for g >= n4): one 16-byte
// load when the row allows it.
DASH_DEV void fetch4(const float* row, int g, int n4, int vocab, int vec4, float (&l)[4]) {
    if (g < n4 && vec4 && 4 * g + 3 < vocab) {
        const float4 v = *reinterpret_cast<const float4*>(row + 4 * g);
        l[0] = v.x; l[1] = v.y; l[2] = v.z; l[3] = v.w;
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) l[j] = (g < n4 && 4 * g + j < vocab) ? row[4 * g + j] : NAN;
    }
}

// UNIT_T: temperature 1, no division (a runtime select would still evaluate the
// exact division for every entry).  The entries of the next two iterations are in
// flight while the current ones are scored, so their latency overlaps the arithmetic
// (with the earlier per-lane branches around the loads the compiler waited for every
// outstanding load before scoring, and only the noise generation hid the latency).
// TRAJ: the launch writes the trajectory outputs (traj, traj_lp) instead of the per-row
// ones (lp_out, row_ml).  The output pointers stay in scalar registers through the
// vocabulary loop: with all six of them live the kernel took 82 scalar registers and
// ran 30% slower (250 vs 190 us at 1024 x 151,936 on gfx950) than with 70-76, the
// same instructions otherwise.  Scalar registers are allocated in blocks of 16, so 82
// occupies 96 of them per wave where 76 occupies 80.
template <bool UNIT_T, bool TRAJ, bool VEC4>
__global__ void __launch_bounds__(kThreads)
sample_k(const float* __restrict__ logits, int64_t ld, int vocab, const int32_t* __restrict__ row_of,
         const int32_t* __restrict__ uid, const int32_t* __restrict__ step, float temperature, uint32_t k0,
         uint32_t k1, int32_t* __restrict__ tok_out, float* __restrict__ lp_out, float* __restrict__ row_ml,
         uint32_t* __restrict__ status, int32_t* __restrict__ traj, float* __restrict__ traj_lp, int traj_ld) {
    __shared__ float red_s[kThreads / 64];
    __shared__ int red_i[kThreads / 64];
    __shared__ float red_m[kThreads / 64];
    __shared__ float red_z[kThreads / 64];
    const int b = blockIdx.x;
    const int r = row_of ? row_of[b] : b;
    const float* row = logits + (int64_t)r * ld;
    const uint32_t u_id = (uint32_t)uid[b], st = (uint32_t)step[b];

    float best_s = -INFINITY;
    int best_i = 0x7FFFFFFF;
    float mx = -INFINITY, z = 0.f;
    float floor_w = -INFINITY;  // wave-shared lower bound on the best exact score seen
    const int n4 = (vocab + 3) >> 2;
    // every lane of the wave runs the same number of iterations (the shared bound needs all
    // lanes); the loop counter lives in a scalar register, so its branches are uniform
    const int lane0 = __builtin_amdgcn_readfirstlane(threadIdx.x & ~63);
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(row, vocab);
    // Scores one group of four entries of this lane (g = its group) and refreshes the
    // wave's shared bound.
    auto score4 = [&](float (&l)[4], int g) {
        vocab_mask(l, g, vocab);
        float floor_t = floor_w;
        if (g < n4) {
            // the round keys are derived here rather than kept: precomputed they held 20
            // scalar registers through the loop
            uint32_t kk0 = k0, kk1 = k1;
            asm volatile("" : "+s"(kk0), "+s"(kk1));
            const U4 x = philox4x32_10(U4{(uint32_t)g, st, u_id, 0u}, kk0, kk1);
            const uint32_t xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (!isfinite(l[j])) continue;
                const float sc = UNIT_T ? l[j] : div_rn(l[j], temperature);
                // even the largest noise this word allows cannot reach the bound: skip the logs
                const float hi = sc + noise_bound(xs[j]);
                if (hi + screen_margin(hi) < floor_t) {
                    lse_push(mx, z, sc);
                    continue;
                }
                const float sa = sc + cheap_gumbel(xs[j]);
                const float mg = screen_margin(sa);
                if (sa + mg >= floor_t) {
                    const float s = sc + gumbel_from_bits(xs[j]);  // exact
                    if (s > best_s) {  // indices grow within a thread: strict > keeps the smallest on ties
                        best_s = s;
                        best_i = 4 * g + j;
                    }
                    floor_t = fmaxf(floor_t, s);
                } else {
                    floor_t = fmaxf(floor_t, sa - mg);
                }
                lse_push(mx, z, sc);
            }
        }
        floor_w = wave_max_f(floor_t);
    };
    // Two groups in flight per lane, in two register sets that take turns: a set is
    // copied out right after the other set's load has been issued (so the wait before the
    // copy leaves that newer load in flight) and then refilled two groups ahead (copying a
    // set that is still loading would make the compiler wait for it).
    if (lane0 < n4) {  // one block for the set-up loads and the first copy (their order matters)
        float set_a[4], set_b[4], l[4];
        // (the scheduling barriers keep set_a's load first and its copy after set_b's load)
        fetch_raw4<VEC4>(rs, threadIdx.x, set_a);
        __builtin_amdgcn_sched_barrier(0);
        fetch_raw4<VEC4>(rs, threadIdx.x + kThreads, set_b);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) l[j] = copy_out(set_a[j]);
        fetch_raw4<VEC4>(rs, threadIdx.x + 2 * kThreads, set_a);
        for (int g0 = lane0; g0 < n4; g0 += 2 * kThreads) {
            const int g = g0 + (threadIdx.x & 63);
            score4(l, g);
            if (g0 + kThreads >= n4) break;  // wave-uniform
#pragma unroll
            for (int j = 0; j < 4; ++j) l[j] = copy_out(set_b[j]);
            fetch_raw4<VEC4>(rs, g + 3 * kThreads, set_b);
            score4(l, g + kThreads);
#pragma unroll
            for (int j = 0; j < 4; ++j) l[j] = copy_out(set_a[j]);
            fetch_raw4<VEC4>(rs, g + 4 * kThreads, set_a);
        }
    }
    // wave merge
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float os = __shfl_xor(best_s, o, 64);
        const int oi = __shfl_xor(best_i, o, 64);
        if (better(os, oi, best_s, best_i)) {
            best_s = os;
            best_i = oi;
        }
        const float om = __shfl_xor(mx, o, 64), oz = __shfl_xor(z, o, 64);
        const float nm = fmaxf(mx, om);
        z = (mx == -INFINITY ? 0.f : z * __expf(mx - nm)) + (om == -INFINITY ? 0.f : oz * __expf(om - nm));
        mx = nm;
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red_s[w] = best_s;
        red_i[w] = best_i;
        red_m[w] = mx;
        red_z[w] = z;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    for (int i = 1; i < kThreads / 64; ++i) {
        if (better(red_s[i], red_i[i], best_s, best_i)) {
            best_s = red_s[i];
            best_i = red_i[i];
        }
        const float nm = fmaxf(mx, red_m[i]);
        z = (mx == -INFINITY ? 0.f : z * __expf(mx - nm)) + (red_m[i] == -INFINITY ? 0.f : red_z[i] * __expf(red_m[i] - nm));
        mx = nm;
    }
    int tok = -1;
    float lp = NAN, lse = NAN;
    if (best_i != 0x7FFFFFFF) {
        tok = best_i;
        const float lt = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)tok * 4u, 0, 0));
        const float sc = UNIT_T ? lt : div_rn(lt, temperature);
        const float lz = logf(z);
        lp = sc - mx - lz;
        lse = mx + lz;
    } else if (status) {
        atomicOr(status, 2u);  // no finite logit: nothing can be drawn
    }
    tok_out[b] = tok;
    if constexpr (TRAJ) {
        traj[(size_t)u_id * traj_ld + st] = tok;
        if (traj_lp) traj_lp[(size_t)u_id * traj_ld + st] = lp;
    } else {
        if (lp_out) lp_out[b] = lp;
        if (row_ml) {
            row_ml[2 * (size_t)b] = tok >= 0 ? mx : NAN;
            row_ml[2 * (size_t)b + 1] = lse;
        }
    }
}

// Largest |cheap noise - exact noise| over every value u can take: (x >> 8) | 1
// is odd, so x = (2k + 1) << 8 for k < 2^23 covers them all.  The maximum (float
// bits, max-reduced) lands in a device variable of this file, so the check needs
// no allocation.
__device__ unsigned g_screen_max_err;

__global__ void screen_check_k(unsigned* max_err_bits) {
    const uint32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= (1u << 23)) return;
    const uint32_t x = (2u * k + 1u) << 8;
    const float e = fabsf(cheap_gumbel(x) - gumbel_from_bits(x));
    atomicMax(max_err_bits, __float_as_uint(isfinite(e) ? e : INFINITY));
}

// Log-probability of a given token under softmax(logits) (temperature 1), one
// workgroup per row, with sample_k's log-normaliser computed in sample_k's order
// (entries in groups of four with a stride of kThreads groups, wave xor tree, the
// waves in order): on the same logits it returns sample_k's log-prob bit for bit.
__global__ void __launch_bounds__(kThreads)
logprob_gather_k(const float* __restrict__ logits, int64_t ld, int vocab, const int32_t* __restrict__ tokens,
                 int per, int stride, int off, float* __restrict__ lp_out, int vec4) {
    __shared__ float red_m[kThreads / 64];
    __shared__ float red_z[kThreads / 64];
    const int b = blockIdx.x;
    const float* row = logits + (int64_t)b * ld;
    float mx = -INFINITY, z = 0.f;
    const int n4 = (vocab + 3) >> 2;
    float nxt[4];
    fetch4(row, threadIdx.x, n4, vocab, vec4, nxt);
    for (int g = threadIdx.x; g < n4; g += kThreads) {
        float l[4] = {nxt[0], nxt[1], nxt[2], nxt[3]};
        fetch4(row, g + kThreads, n4, vocab, vec4, nxt);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (!isfinite(l[j])) continue;
            lse_push(mx, z, l[j]);
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float om = __shfl_xor(mx, o, 64), oz = __shfl_xor(z, o, 64);
        const float nm = fmaxf(mx, om);
        z = (mx == -INFINITY ? 0.f : z * __expf(mx - nm)) + (om == -INFINITY ? 0.f : oz * __expf(om - nm));
        mx = nm;
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red_m[w] = mx;
        red_z[w] = z;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    for (int i = 1; i < kThreads / 64; ++i) {
        const float nm = fmaxf(mx, red_m[i]);
        z = (mx == -INFINITY ? 0.f : z * __expf(mx - nm)) + (red_m[i] == -INFINITY ? 0.f : red_z[i] * __expf(red_m[i] - nm));
        mx = nm;
    }
    const int t = tokens[(int64_t)(b / per) * stride + off + b % per];
    const float l = (t >= 0 && t < vocab) ? row[t] : NAN;
    lp_out[b] = l - mx - logf(z);
}

// KL divergence between the next-token distributions of two models, one
// workgroup of kKlThreads per row pair, walking entries in groups of four with a
// stride of kKlThreads groups.  Each side keeps, over its entries of nonzero probability (logit
// not -inf), a running maximum m, z = sum e^(x - m) and w = sum e^(x - m) (x - y)
// with y the other side's logit: exponentials by the hardware, sums in fp64.  Then
//   D_KL(p_x || p_y) = w_x / z_x - (m_x - m_y) - (ln z_x - ln z_y),
// and identical rows give exactly 0 (both sides run the same operations).  An
// entry with mass on one side and none on the other makes that direction +inf.
struct KlAcc {
    float m;
    double z, w;
    int inf;
};

DASH_DEV void kl_push(KlAcc& s, float x, float y) {
    if (x == -INFINITY) return;
    const bool none = y == -INFINITY;
    const double d = none ? 0.0 : (double)x - (double)y;
    s.inf |= none;
    if (x > s.m) {
        const double c = s.m == -INFINITY ? 0.0 : (double)__expf(s.m - x);
        s.z = s.z * c + 1.0;
        s.w = s.w * c + d;
        s.m = x;
    } else {  // also NaN, which then reaches z and the result
        const double e = (double)__expf(x - s.m);
        s.z += e;
        s.w += e * d;
    }
}

DASH_DEV void kl_merge(KlAcc& s, float om, double oz, double ow, int oinf) {
    s.inf |= oinf;
    const float m = fmaxf(s.m, om);
    const double a = s.m == -INFINITY ? 0.0 : (double)__expf(s.m - m);
    const double b = om == -INFINITY ? 0.0 : (double)__expf(om - m);
    s.z = s.z * a + oz * b;
    s.w = s.w * a + ow * b;
    s.m = m;
}

DASH_DEV double kl_final(const KlAcc& x, const KlAcc& y) {
    if (x.inf) return INFINITY;
    return x.w / x.z - ((double)x.m - (double)y.m) - (log(x.z) - log(y.z));
}

__global__ void __launch_bounds__(kKlThreads)
kl_rows_k(const float* __restrict__ theta, const float* __restrict__ base, int64_t ld, int vocab,
          float* __restrict__ kl, float* __restrict__ kl_rev, int vec4) {
    __shared__ float red_m[2][kKlThreads / 64];
    __shared__ double red_z[2][kKlThreads / 64], red_w[2][kKlThreads / 64];
    __shared__ int red_inf[2][kKlThreads / 64];
    const int r = blockIdx.x;
    const float* ra = theta + (int64_t)r * ld;
    const float* rb = base + (int64_t)r * ld;
    KlAcc sa{-INFINITY, 0.0, 0.0, 0}, sb{-INFINITY, 0.0, 0.0, 0};
    const int n4 = (vocab + 3) >> 2;
    for (int g = threadIdx.x; g < n4; g += kKlThreads) {
        float a[4], b[4];
        if (vec4 && 4 * g + 3 < vocab) {
            const float4 va = load_stream4(ra + 4 * g);
            const float4 vb = load_stream4(rb + 4 * g);
            a[0] = va.x; a[1] = va.y; a[2] = va.z; a[3] = va.w;
            b[0] = vb.x; b[1] = vb.y; b[2] = vb.z; b[3] = vb.w;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {  // entries past the vocabulary have no mass on either side
                a[j] = 4 * g + j < vocab ? ra[4 * g + j] : -INFINITY;
                b[j] = 4 * g + j < vocab ? rb[4 * g + j] : -INFINITY;
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            kl_push(sa, a[j], b[j]);
            kl_push(sb, b[j], a[j]);
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        kl_merge(sa, __shfl_xor(sa.m, o, 64), __shfl_xor(sa.z, o, 64), __shfl_xor(sa.w, o, 64), __shfl_xor(sa.inf, o, 64));
        kl_merge(sb, __shfl_xor(sb.m, o, 64), __shfl_xor(sb.z, o, 64), __shfl_xor(sb.w, o, 64), __shfl_xor(sb.inf, o, 64));
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red_m[0][w] = sa.m; red_z[0][w] = sa.z; red_w[0][w] = sa.w; red_inf[0][w] = sa.inf;
        red_m[1][w] = sb.m; red_z[1][w] = sb.z; red_w[1][w] = sb.w; red_inf[1][w] = sb.inf;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    for (int i = 1; i < kKlThreads / 64; ++i) {
        kl_merge(sa, red_m[0][i], red_z[0][i], red_w[0][i], red_inf[0][i]);
        kl_merge(sb, red_m[1][i], red_z[1][i], red_w[1][i], red_inf[1][i]);
    }
    kl[r] = (float)kl_final(sb, sa);  // D_KL(p_base || p_theta)
    if (kl_rev) kl_rev[r] = (float)kl_final(sa, sb);
}

}  // namespace

hipError_t launch_logprob_gather(const float* logits, int64_t ld, int rows, int vocab, const int32_t* tokens, int per,
                                 int stride, int off, float* lp_out, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (per < 1) return hipErrorInvalidValue;
    const int vec4 = ((ld & 3) == 0 && ((uintptr_t)logits & 15) == 0) ? 1 : 0;
    logprob_gather_k<<<rows, kThreads, 0, st>>>(logits, ld, vocab, tokens, per, stride, off, lp_out, vec4);
    return hipGetLastError();
}

hipError_t launch_logits_kl(const float* theta, const float* base, int64_t ld, int rows, int vocab, float* kl,
                            float* kl_rev, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (vocab < 1 || ld < vocab) return hipErrorInvalidValue;
    const int vec4 =
        ((ld & 3) == 0 && ((uintptr_t)theta & 15) == 0 && ((uintptr_t)base & 15) == 0) ? 1 : 0;
    kl_rows_k<<<rows, kKlThreads, 0, st>>>(theta, base, ld, vocab, kl, kl_rev, vec4);
    return hipGetLastError();
}

float sampler_screen_tol() { return kScreenTol; }

hipError_t sampler_screen_check(float* max_err) {
    unsigned* d = nullptr;
    hipError_t e = hipGetSymbolAddress((void**)&d, HIP_SYMBOL(g_screen_max_err));
    if (e != hipSuccess) return e;
    const unsigned zero = 0;
    if ((e = hipMemcpy(d, &zero, 4, hipMemcpyHostToDevice)) != hipSuccess) return e;
    screen_check_k<<<(1 << 23) / 256, 256, 0, nullptr>>>(d);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    unsigned bits = 0;
    if ((e = hipMemcpy(&bits, d, 4, hipMemcpyDeviceToHost)) != hipSuccess) return e;
    std::memcpy(max_err, &bits, 4);
    return hipSuccess;
}

hipError_t launch_sample(const float* logits, int64_t ld, int rows, int vocab, const int32_t* row_of,
                         const int32_t* uid, const int32_t* step, float temperature, uint64_t seed,
                         int32_t* tok_out, float* lp_out, float* row_ml, uint32_t* status, int32_t* traj,
                         float* traj_lp, int traj_ld, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (traj ? (lp_out || row_ml) : traj_lp != nullptr) return hipErrorInvalidValue;  // one output set per launch
    if (vocab <= 0 || vocab > (1 << 28)) return hipErrorInvalidValue;  // byte offsets of a row stay below 2^30
    const bool vec4 = (ld & 3) == 0 && (vocab & 3) == 0 && ((uintptr_t)logits & 15) == 0;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#define DASH_SAMPLE_LAUNCH(U, TR, V4)                                                                          \
    sample_k<U, TR, V4><<<rows, kThreads, 0, st>>>(logits, ld, vocab, row_of, uid, step, temperature, k0, k1,     \
                                                   tok_out, lp_out, row_ml, status, traj, traj_lp, traj_ld)
#define DASH_SAMPLE_LAUNCH_V(U, TR)     \
    do {                                \
        if (vec4)                       \
            DASH_SAMPLE_LAUNCH(U, TR, true); \
        else                            \
            DASH_SAMPLE_LAUNCH(U, TR, false); \
    } while (0)
    if (temperature == 1.0f) {
        if (traj) DASH_SAMPLE_LAUNCH_V(true, true);
        else DASH_SAMPLE_LAUNCH_V(true, false);
    } else {
        if (traj) DASH_SAMPLE_LAUNCH_V(false, true);
        else DASH_SAMPLE_LAUNCH_V(false, false);
    }
#undef DASH_SAMPLE_LAUNCH_V
#undef DASH_SAMPLE_LAUNCH
    return hipGetLastError();
}

}  // namespace dash
