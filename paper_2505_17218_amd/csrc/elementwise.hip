// Row-wise kernels around the projection GEMMs: embedding gather, residual add
// + RMSNorm, the RoPE table, q/k RoPE with KV-page append, page copies, and the
// rollout row-state helpers.  All are HBM/latency bound: one workgroup per
// token row, coalesced along the feature dimension.
#include "common.h"
#include "kernels.h"

namespace dash {

namespace {

constexpr int kRowThreads = 256;

// Row kernels (embedding + norm, residual add + norm): one workgroup of 256
// threads per row, so even a small decode batch spreads over many CUs; a thread
// holds up to kMaxV float4 of the row (d <= 256 * 4 * kMaxV), the row is read
// once, and the sum of squares is reduced with shuffles and one LDS step.
constexpr int kMaxV = 4;
constexpr int kMaxSplits = 8;  // split-K partials summed by add_rmsnorm_k

template <typename T>
DASH_DEV void store4(T* p, float4 v);
template <>
DASH_DEV void store4<float>(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
template <>
DASH_DEV void store4<bf16_t>(bf16_t* p, float4 v) {
    const uint32_t lo = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
    const uint32_t hi = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
    *reinterpret_cast<uint2*>(p) = make_uint2(lo, hi);
}
template <typename T>
DASH_DEV float4 load4(const T* p);
template <>
DASH_DEV float4 load4<float>(const float* p) { return *reinterpret_cast<const float4*>(p); }
template <>
DASH_DEV float4 load4<bf16_t>(const bf16_t* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xFFFF0000u));
}

DASH_DEV float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
DASH_DEV float dot4(float4 a) { return a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w; }

// x[r] = E[tok[r]]; y[r] = RMSNorm(x[r]) * w.  A token outside [0, vocab) is never
// used as an index: the row becomes NaN (so everything computed from it shows it)
// and bit 2 of the status word is set.
template <typename T>
__global__ void __launch_bounds__(kRowThreads) embed_rmsnorm_k(const int32_t* __restrict__ tok,
                                                               const T* __restrict__ E,
                                                               const T* __restrict__ w, float* __restrict__ x,
                                                               T* __restrict__ y, int d, int vocab, float eps,
                                                               uint32_t* __restrict__ status) {
    __shared__ float red[kRowThreads / 64];
    const int r = blockIdx.x;
    const int t = tok[r];
    const int d4 = d >> 2;
    if (t < 0 || t >= vocab) {  // the same for the whole workgroup
        const float4 nan4 = make_float4(NAN, NAN, NAN, NAN);
        for (int i = threadIdx.x; i < d4; i += kRowThreads) {
            *reinterpret_cast<float4*>(x + (size_t)r * d + 4 * i) = nan4;
            store4(y + (size_t)r * d + 4 * i, nan4);
        }
        if (status && threadIdx.x == 0) atomicOr(status, 4u);
        return;
    }
    float4 v[kMaxV];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxV; ++j) {
        const int i = threadIdx.x + kRowThreads * j;
        if (i < d4) {
            v[j] = load4(E + (size_t)t * d + 4 * i);
            ss += dot4(v[j]);
        }
    }
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int j = 0; j < kMaxV; ++j) {
        const int i = threadIdx.x + kRowThreads * j;
        if (i < d4) {
            *reinterpret_cast<float4*>(x + (size_t)r * d + 4 * i) = v[j];
            const float4 g = load4(w + 4 * i);
            store4(y + (size_t)r * d + 4 * i, make_float4(v[j].x * inv * g.x, v[j].y * inv * g.y, v[j].z * inv * g.z,
                                                          v[j].w * inv * g.w));
        }
    }
}

// Row i_out (input row r = row_map ? row_map[i_out] : i_out):
// x[r] += sum of the nsplit partials delta[s][r] (in split order); y[i_out] =
// RMSNorm(x[r]) * w; x is written back if write_x.
template <typename T, int NT = kRowThreads, int MV = kMaxV>
__global__ void __launch_bounds__(NT) add_rmsnorm_k(float* __restrict__ x, const float* __restrict__ delta,
                                                             int nsplit, size_t split_stride,
                                                             const T* __restrict__ w, T* __restrict__ y,
                                                             const int32_t* __restrict__ row_map, int d,
                                                             float eps, int write_x) {
    __shared__ float red[NT / 64];
    const int i_out = blockIdx.x;
    const int r = row_map ? row_map[i_out] : i_out;
    const int d4 = d >> 2;
    float4 v[MV], wt[MV];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < MV; ++j) {
        const int i = threadIdx.x + NT * j;
        if (i < d4) {
            wt[j] = load4(w + 4 * i);  // the norm weights too, so no load waits after the reduction
            // all loads of this float4 are issued before the first add
            float4 p[kMaxSplits];
#pragma unroll
            for (int s = 0; s < kMaxSplits; ++s)
                if (delta && s < nsplit)
                    p[s] = *reinterpret_cast<const float4*>(delta + s * split_stride + (size_t)r * d + 4 * i);
            float4 a = *reinterpret_cast<const float4*>(x + (size_t)r * d + 4 * i);
            float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int s = 0; s < kMaxSplits; ++s)
                if (delta && s < nsplit) sum = s ? add4(sum, p[s]) : p[s];
            if (delta && nsplit > 0) a = add4(a, sum);
            v[j] = a;
            ss += dot4(a);
        }
    }
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int j = 0; j < MV; ++j) {
        const int i = threadIdx.x + NT * j;
        if (i < d4) {
            if (write_x) *reinterpret_cast<float4*>(x + (size_t)r * d + 4 * i) = v[j];
            const float4 g = wt[j];
            store4(y + (size_t)i_out * d + 4 * i, make_float4(v[j].x * inv * g.x, v[j].y * inv * g.y,
                                                              v[j].z * inv * g.z, v[j].w * inv * g.w));
        }
    }
}

__global__ void rope_table_k(const int32_t* __restrict__ pos, float* __restrict__ cs, int rows, int half,
                             int head_dim, double theta) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= rows * half) return;
    const int r = idx / half, i = idx - r * half;
    const double freq = pow(theta, -2.0 * (double)i / (double)head_dim);
    const double a = (double)pos[r] * freq;
    cs[2 * (size_t)idx] = (float)cos(a);
    cs[2 * (size_t)idx + 1] = (float)sin(a);
}

// grid (rows, ceil(items / 256)): one RoPE pair of q or k, or one v element, per thread.
// KV-cache appends: non-temporal stores, as in the QKV GEMM's fused epilogue (a decode step
// writes a few bytes into lines that later steps read from memory anyway).
template <typename T> DASH_DEV void st_kv(T* p, float v);
template <> DASH_DEV void st_kv<float>(float* p, float v) { __builtin_nontemporal_store(v, p); }
template <> DASH_DEV void st_kv<bf16_t>(bf16_t* p, float v) { __builtin_nontemporal_store(f2bf(v), p); }

template <typename T>
__global__ void __launch_bounds__(kRowThreads)
qkv_rope_append_k(const float* __restrict__ qkv, int nsplit, size_t split_stride, const T* __restrict__ bias,
                  const float* __restrict__ cs, const int32_t* __restrict__ pos, const int32_t* __restrict__ slot,
                  const int32_t* __restrict__ page_table, T* __restrict__ pool, KVGeom g, int layer,
                  T* __restrict__ q_out, int n_heads, uint32_t* status) {
    const int r = blockIdx.x;
    const int hd = g.head_dim, half = hd >> 1, n_kv = g.n_kv;
    const int qkv_rows = (n_heads + 2 * n_kv) * hd;
    const float* row = qkv + (size_t)r * qkv_rows;
    auto val = [&](int j) {
        float v = row[j];
        for (int s = 1; s < nsplit; ++s) v += row[s * split_stride + j];
        return v + ld_elem(bias + j);
    };
    const int n_rope = (n_heads + n_kv) * half;
    const int it = blockIdx.y * blockDim.x + threadIdx.x;
    // The operands are read before the cache page is looked up (position and slot,
    // then the page table), so the two chains of loads overlap.
    const bool is_rope = it < n_rope, is_v = !is_rope && it < n_rope + n_kv * hd;
    const int h = is_rope ? it / half : (it - n_rope) / hd;
    const int i = is_rope ? it - h * half : (it - n_rope) - h * hd;  // pair index / v dim
    float a = 0.f, b = 0.f, c = 1.f, sn = 0.f;
    if (is_rope) {
        const int j = h * hd + i;
        a = val(j);
        b = val(j + half);
        const float* c_s = cs + ((size_t)r * half + i) * 2;
        c = c_s[0];
        sn = c_s[1];
    } else if (is_v) {
        a = val((n_heads + n_kv) * hd + (it - n_rope));
    }
    const int p = pos[r];
    const int page = kv_page_of(g, page_table, slot[r], p);
    if (page < 0 && blockIdx.y == 0 && threadIdx.x == 0 && status) atomicOr(status, 1u);
    const int key = p % g.page_size;
    if (is_rope) {
        float lo, hi;
        rope_pair(a, b, c, sn, lo, hi);
        if (h < n_heads) {
            T* q = q_out + ((size_t)r * n_heads + h) * hd;
            st_elem(q + i, lo);
            st_elem(q + i + half, hi);
        } else if (page >= 0) {
            T* kb = pool + kv_block(g, layer, page, h - n_heads, 0);
            st_kv(kb + k_index<T>(g, key, i), lo);
            st_kv(kb + k_index<T>(g, key, i + half), hi);
        }
    } else if (is_v && page >= 0) {
        T* vb = pool + kv_block(g, layer, page, h, 1);
        st_kv(vb + v_index<T>(g, key, i), a);
    }
}

// Copy all layers of page pairs[2i] to page pairs[2i+1]; grid (n, n_layers).
__global__ void copy_pages_k(uint4* __restrict__ pool, KVGeom g, size_t page_layer_vec, const int32_t* pairs) {
    const int i = blockIdx.x, layer = blockIdx.y;
    const int src = pairs[2 * i], dst = pairs[2 * i + 1];
    const uint4* s = pool + ((size_t)layer * g.n_pages + src) * page_layer_vec;
    uint4* t = pool + ((size_t)layer * g.n_pages + dst) * page_layer_vec;
    for (size_t k = threadIdx.x; k < page_layer_vec; k += blockDim.x) t[k] = s[k];
}

__global__ void rows_init_k(int32_t* slot, int32_t* uid, int32_t* pos, int32_t* step, int n, int pos0, int step0) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    slot[i] = i;
    uid[i] = i;
    pos[i] = pos0;
    step[i] = step0;
}

__global__ void rows_advance_k(int32_t* pos, int32_t* step, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    pos[i] += 1;
    step[i] += 1;
}

__global__ void fill_i32_k(int32_t* p, int32_t v, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void iota_div_k(int32_t* p, int n, int div) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = i / div;
}

inline unsigned cdiv(size_t a, size_t b) { return (unsigned)((a + b - 1) / b); }

}  // namespace

hipError_t launch_embed_rmsnorm(int dtype, const int32_t* tok, const void* E, const void* w, float* x, void* y,
                                int rows, int d, int vocab, float eps, uint32_t* status, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (d % 4 || d > kRowThreads * 4 * kMaxV) return hipErrorInvalidValue;
    const unsigned blocks = (unsigned)rows;
    if (dtype == 1)
        embed_rmsnorm_k<bf16_t><<<blocks, kRowThreads, 0, st>>>(tok, (const bf16_t*)E, (const bf16_t*)w, x,
                                                                (bf16_t*)y, d, vocab, eps, status);
    else
        embed_rmsnorm_k<float><<<blocks, kRowThreads, 0, st>>>(tok, (const float*)E, (const float*)w, x, (float*)y,
                                                               d, vocab, eps, status);
    return hipGetLastError();
}

// Inputs u * 256 + j (j < 256) per thread over all 2^32 float32 patterns: the count of
// those whose f2bf result differs from bf16_rne_bits, reduced into a device variable of
// this file (no allocation).
namespace {

__device__ unsigned long long g_bf16_mismatch;

__global__ void bf16_round_check_k(unsigned long long* cnt) {
    const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;  // < 2^24
    unsigned n = 0;
    for (uint32_t j = 0; j < 256; ++j) {
        const float f = __uint_as_float(t * 256u + j);
        n += f2bf(f) != bf16_rne_bits(f);
    }
    if (n) atomicAdd(cnt, (unsigned long long)n);
}

}  // namespace

hipError_t bf16_round_check(unsigned long long* mismatches) {
    unsigned long long* d = nullptr;
    hipError_t e = hipGetSymbolAddress((void**)&d, HIP_SYMBOL(g_bf16_mismatch));
    if (e != hipSuccess) return e;
    const unsigned long long zero = 0;
    if ((e = hipMemcpy(d, &zero, 8, hipMemcpyHostToDevice)) != hipSuccess) return e;
    bf16_round_check_k<<<(1u << 24) / 256, 256, 0, nullptr>>>(d);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hipMemcpy(mismatches, d, 8, hipMemcpyDeviceToHost);
}

hipError_t launch_add_rmsnorm(int dtype, float* x, const float* delta, int nsplit, size_t split_stride,
                              const void* w, void* y, const int32_t* row_map, int rows, int d, float eps,
                              int write_x, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (d % 4 || d > kRowThreads * 4 * kMaxV || nsplit > kMaxSplits) return hipErrorInvalidValue;
    const unsigned blocks = (unsigned)rows;
    // one float4 per thread where the row has 257-512 of them (d_model 1028-2048): every
    // thread carries one chain of loads instead of some two (measured 2% less norm time
    // at d = 1536 and 2048)
    const int d4 = d / 4;
    if (dtype == 1 && d4 > 256 && d4 <= 384)
        add_rmsnorm_k<bf16_t, 384, 1><<<blocks, 384, 0, st>>>(x, delta, nsplit, split_stride, (const bf16_t*)w,
                                                              (bf16_t*)y, row_map, d, eps, write_x);
    else if (dtype == 1 && d4 > 384 && d4 <= 512)
        add_rmsnorm_k<bf16_t, 512, 1><<<blocks, 512, 0, st>>>(x, delta, nsplit, split_stride, (const bf16_t*)w,
                                                              (bf16_t*)y, row_map, d, eps, write_x);
    else if (dtype == 1)
        add_rmsnorm_k<bf16_t><<<blocks, kRowThreads, 0, st>>>(x, delta, nsplit, split_stride, (const bf16_t*)w,
                                                              (bf16_t*)y, row_map, d, eps, write_x);
    else
        add_rmsnorm_k<float><<<blocks, kRowThreads, 0, st>>>(x, delta, nsplit, split_stride, (const float*)w,
                                                             (float*)y, row_map, d, eps, write_x);
    return hipGetLastError();
}

hipError_t launch_rope_table(const int32_t* pos, float* cs, int rows, int head_dim, float theta, hipStream_t st) {
    const int half = head_dim / 2;
    if (rows <= 0) return hipSuccess;
    rope_table_k<<<cdiv((size_t)rows * half, 256), 256, 0, st>>>(pos, cs, rows, half, head_dim, (double)theta);
    return hipGetLastError();
}

hipError_t launch_qkv_rope_append(int dtype, const float* qkv, int nsplit, size_t split_stride, const void* bias,
                                  const float* cs, const int32_t* pos, const int32_t* slot,
                                  const int32_t* page_table, void* pool, const KVGeom& g, int layer,
                                  void* q_out, int rows, int n_heads, uint32_t* status, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    const int items = (n_heads + g.n_kv) * (g.head_dim / 2) + g.n_kv * g.head_dim;
    dim3 grid(rows, cdiv(items, kRowThreads));
    if (dtype == 1)
        qkv_rope_append_k<bf16_t><<<grid, kRowThreads, 0, st>>>(qkv, nsplit, split_stride, (const bf16_t*)bias, cs,
                                                                pos, slot, page_table, (bf16_t*)pool, g, layer,
                                                                (bf16_t*)q_out, n_heads, status);
    else
        qkv_rope_append_k<float><<<grid, kRowThreads, 0, st>>>(qkv, nsplit, split_stride, (const float*)bias, cs,
                                                               pos, slot, page_table, (float*)pool, g, layer,
                                                               (float*)q_out, n_heads, status);
    return hipGetLastError();
}

hipError_t launch_copy_pages(int dtype, void* pool, const KVGeom& g, const int32_t* pairs, int n, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const size_t esz = dtype == 1 ? 2 : 4;
    const size_t page_layer_bytes = (size_t)g.n_kv * 2 * g.page_size * g.head_dim * esz;
    dim3 grid(n, g.n_layers);
    copy_pages_k<<<grid, 256, 0, st>>>((uint4*)pool, g, page_layer_bytes / 16, pairs);
    return hipGetLastError();
}

hipError_t launch_rows_init(int32_t* slot, int32_t* uid, int32_t* pos, int32_t* step, int n, int pos0, int step0,
                            hipStream_t st) {
    if (n <= 0) return hipSuccess;
    rows_init_k<<<cdiv(n, 256), 256, 0, st>>>(slot, uid, pos, step, n, pos0, step0);
    return hipGetLastError();
}

hipError_t launch_rows_advance(int32_t* pos, int32_t* step, int n, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    rows_advance_k<<<cdiv(n, 256), 256, 0, st>>>(pos, step, n);
    return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t st) {
    if (n == 0) return hipSuccess;
    const unsigned blocks = n / 256 + 1 < 4096 ? (unsigned)(n / 256 + 1) : 4096u;
    fill_i32_k<<<blocks, 256, 0, st>>>(p, v, n);
    return hipGetLastError();
}

hipError_t launch_iota_div(int32_t* p, int n, int div, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    iota_div_k<<<cdiv(n, 256), 256, 0, st>>>(p, n, div);
    return hipGetLastError();
}

}  // namespace dash
