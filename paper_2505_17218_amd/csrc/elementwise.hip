// Row-wise kernels around the projection GEMMs: embedding gather, residual add
// + RMSNorm, the RoPE table, q/k RoPE with KV-page append, page copies, and the
// rollout row-state helpers.  All are HBM/latency bound: one workgroup per
// token row, coalesced along the feature dimension.
#include "common.h"
#include "kernels.h"

namespace dash {

namespace {

constexpr int kRowThreads = 256;

// x[r] = E[tok[r]]; y[r] = RMSNorm(x[r]) * w.
template <typename T>
__global__ void __launch_bounds__(kRowThreads) embed_rmsnorm_k(const int32_t* __restrict__ tok,
                                                               const T* __restrict__ E,
                                                               const T* __restrict__ w, float* __restrict__ x,
                                                               T* __restrict__ y, int d, int vocab, float eps) {
    __shared__ float red[16];
    const int r = blockIdx.x;
    int t = tok[r];
    t = t < 0 ? 0 : (t >= vocab ? vocab - 1 : t);  // never index outside the table
    const T* e = E + (size_t)t * d;
    float* xr = x + (size_t)r * d;
    float ss = 0.f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
        const float v = ld_elem(e + i);
        xr[i] = v;
        ss += v * v;
    }
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    T* yr = y + (size_t)r * d;
    for (int i = threadIdx.x; i < d; i += blockDim.x) st_elem(yr + i, xr[i] * inv * ld_elem(w + i));
}

template <typename T>
__global__ void __launch_bounds__(kRowThreads) add_rmsnorm_k(float* __restrict__ x, const float* __restrict__ delta,
                                                             int nsplit, size_t split_stride,
                                                             const T* __restrict__ w, T* __restrict__ y,
                                                             const int32_t* __restrict__ row_map, int d, float eps,
                                                             int write_x) {
    __shared__ float red[16];
    const int i_out = blockIdx.x;
    const int r = row_map ? row_map[i_out] : i_out;
    float* xr = x + (size_t)r * d;
    T* yr = y + (size_t)i_out * d;
    // keep up to 8 values per thread in registers (d <= 2048); beyond that, re-read x
    constexpr int kReg = 8;
    float v_reg[kReg];
    float ss = 0.f;
    int j = 0;
    for (int i = threadIdx.x; i < d; i += blockDim.x, ++j) {
        float v = xr[i];
        if (delta)
            for (int s = 0; s < nsplit; ++s) v += delta[s * split_stride + (size_t)r * d + i];
        if (write_x) xr[i] = v;
        if (j < kReg) v_reg[j] = v;
        ss += v * v;
    }
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    j = 0;
    for (int i = threadIdx.x; i < d; i += blockDim.x, ++j) {
        float v;
        if (j < kReg) {
            v = v_reg[j];
        } else {
            v = xr[i];
            if (!write_x && delta)
                for (int s = 0; s < nsplit; ++s) v += delta[s * split_stride + (size_t)r * d + i];
        }
        st_elem(yr + i, v * inv * ld_elem(w + i));
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
    const float* c_s = cs + (size_t)r * half * 2;
    const int p = pos[r];
    const int page = kv_page_of(g, page_table, slot[r], p);
    if (page < 0 && threadIdx.x == 0 && status) atomicOr(status, 1u);
    const int key = p % g.page_size;
    auto val = [&](int j) {
        float v = row[j];
        for (int s = 1; s < nsplit; ++s) v += row[s * split_stride + j];
        return v + ld_elem(bias + j);
    };
    const int n_rope = (n_heads + n_kv) * half;
    const int n_items = n_rope + n_kv * hd;
    for (int it = threadIdx.x; it < n_items; it += blockDim.x) {
        if (it < n_rope) {
            const int h = it / half, i = it - h * half;
            const int j = h * hd + i;
            const float a = val(j), b = val(j + half);
            const float c = c_s[2 * i], s = c_s[2 * i + 1];
            const float lo = a * c - b * s, hi = b * c + a * s;
            if (h < n_heads) {
                T* q = q_out + ((size_t)r * n_heads + h) * hd;
                st_elem(q + i, lo);
                st_elem(q + i + half, hi);
            } else if (page >= 0) {
                T* kb = pool + kv_block(g, layer, page, h - n_heads, 0);
                st_elem(kb + k_index<T>(g, key, i), lo);
                st_elem(kb + k_index<T>(g, key, i + half), hi);
            }
        } else if (page >= 0) {
            const int jj = it - n_rope;
            const int h = jj / hd, dd = jj - h * hd;
            const float v = val((n_heads + n_kv) * hd + jj);
            T* vb = pool + kv_block(g, layer, page, h, 1);
            st_elem(vb + v_index<T>(g, key, dd), v);
        }
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
                                  int rows, int d, int vocab, float eps, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (dtype == 1)
        embed_rmsnorm_k<bf16_t><<<rows, kRowThreads, 0, st>>>(tok, (const bf16_t*)E, (const bf16_t*)w, x,
                                                              (bf16_t*)y, d, vocab, eps);
    else
        embed_rmsnorm_k<float><<<rows, kRowThreads, 0, st>>>(tok, (const float*)E, (const float*)w, x, (float*)y,
                                                             d, vocab, eps);
    return hipGetLastError();
}

hipError_t launch_add_rmsnorm(int dtype, float* x, const float* delta, int nsplit, size_t split_stride,
                              const void* w, void* y, const int32_t* row_map, int rows, int d, float eps,
                              int write_x, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (dtype == 1)
        add_rmsnorm_k<bf16_t><<<rows, kRowThreads, 0, st>>>(x, delta, nsplit, split_stride, (const bf16_t*)w,
                                                            (bf16_t*)y, row_map, d, eps, write_x);
    else
        add_rmsnorm_k<float><<<rows, kRowThreads, 0, st>>>(x, delta, nsplit, split_stride, (const float*)w,
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
    if (dtype == 1)
        qkv_rope_append_k<bf16_t><<<rows, kRowThreads, 0, st>>>(qkv, nsplit, split_stride, (const bf16_t*)bias, cs,
                                                                pos, slot, page_table, (bf16_t*)pool, g, layer,
                                                                (bf16_t*)q_out, n_heads, status);
    else
        qkv_rope_append_k<float><<<rows, kRowThreads, 0, st>>>(qkv, nsplit, split_stride, (const float*)bias, cs,
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
