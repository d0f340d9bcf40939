// Device-side helpers shared by the HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define DASH_DEV __device__ __forceinline__

namespace dash {

typedef uint16_t bf16_t;  // bfloat16 bit pattern

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Fourth dword of a raw buffer resource on gfx9-family GPUs (stride 0, 32-bit data
// format): loads past num_records return zeros without touching memory.
constexpr int kBufferDword3 = 0x00020000;

DASH_DEV float bf2f(bf16_t u) { return __uint_as_float(static_cast<uint32_t>(u) << 16); }

// float -> bfloat16, round to nearest even (NaN stays NaN, with its quiet bit set): the
// conversion instruction of gfx950 (v_cvt_pk_bf16_f32, two values per instruction).  It
// gives the bits of integer rounding of the pattern (bf16_rne_bits) for every one of the
// 2^32 inputs, NaNs included; dash_bf16_round_check verifies that on the device in use.
DASH_DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f)); }

// The same rounding on the integer bit pattern: add 0x7FFF plus the lowest kept bit and
// truncate; a NaN keeps its top half with the quiet bit set.
DASH_DEV bf16_t bf16_rne_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<bf16_t>(u >> 16);
}

// Work-item index for block `bid` of `nb`: the GPU deals consecutive block ids
// round-robin to its 8 XCDs (each with its own L2), so this gives each XCD one
// contiguous run of work items instead; neighbouring items (the same weight
// tile, the rows of one prompt group) then share an L2.
constexpr int kXcds = 8;
DASH_DEV int xcd_remap(int bid, int nb) {
    const int x = bid % kXcds, j = bid / kXcds;
    const int q = nb / kXcds, r = nb % kXcds;
    return x * q + (x < r ? x : r) + j;
}

// Rotate-half RoPE of the pair (a, b) = (z_i, z_{i + hd/2}) by the angle with
// cosine c and sine s: lo = a c - b s, hi = b c + a s.  Written as one fused
// multiply-add over a separately rounded product, so every kernel that rotates
// (the QKV GEMM epilogue and the standalone kernel) produces the same bits
// whatever the compiler's contraction setting.
DASH_DEV void rope_pair(float a, float b, float c, float s, float& lo, float& hi) {
    lo = __builtin_fmaf(a, c, -(b * s));
    hi = __builtin_fmaf(b, c, a * s);
}

// Element access for the two storage types (float or bfloat16 bits).
template <typename T> DASH_DEV float ld_elem(const T* p);
template <> DASH_DEV float ld_elem<float>(const float* p) { return *p; }
template <> DASH_DEV float ld_elem<bf16_t>(const bf16_t* p) { return bf2f(*p); }
template <typename T> DASH_DEV void st_elem(T* p, float v);
template <> DASH_DEV void st_elem<float>(float* p, float v) { *p = v; }
template <> DASH_DEV void st_elem<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

DASH_DEV float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

DASH_DEV float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// Sum over a workgroup of blockDim.x threads (multiple of 64, <= 1024).
// `red` is LDS scratch of at least 16 floats.  All threads get the result.
DASH_DEV float block_sum(float v, float* red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float s = 0.f;
    for (int i = 0; i < nw; ++i) s += red[i];
    return s;
}

// Layout of one KV page block (one layer, one page, one kv head, K or V).
// Pool offset of the block, in elements:
//   ((((layer * n_pages + page) * n_kv + kvh) * 2 + kind) * page_size * head_dim
// kind 0 = K, 1 = V.
//   float32 cache: K and V blocks are [page_size][head_dim].
//   bfloat16 cache: K block is [head_dim/32][page_size][32] (32-dim chunks, so a
//     wave reads 16 keys x 64 B of one chunk as one contiguous 1 KB); V block is
//     [head_dim][page_size] (transposed), and inside every 32-key run the keys
//     are permuted: key k sits at 8*((k%16)/4) + 4*(k/16) + k%4, which is the
//     order in which the decode-attention MFMA holds probabilities per lane.
struct KVGeom {
    int n_layers, n_pages, n_kv, head_dim, page_size;
    int max_pages;  // page-table row length (pages per slot)
    int max_seqs;   // page-table rows (slots)
    int split_keys; // decode attention context split (multiple of 32, fixed per cache)
    int shared_keys; // positions below this are shared by several rows (a prompt group's full
                     // pages): decode attention keeps them cached, the rest it streams
};

// Page backing position `pos` of `slot`, or -1 if the slot, position or table entry is out of range.
DASH_DEV int kv_page_of(const KVGeom& g, const int32_t* page_table, int slot, int pos) {
    if (slot < 0 || slot >= g.max_seqs || pos < 0) return -1;
    const int pi = pos / g.page_size;
    if (pi >= g.max_pages) return -1;
    const int page = page_table[(size_t)slot * g.max_pages + pi];
    return (page >= 0 && page < g.n_pages) ? page : -1;
}

DASH_DEV size_t kv_block(const KVGeom& g, int layer, int page, int kvh, int kind) {
    return ((((size_t)layer * g.n_pages + page) * g.n_kv + kvh) * 2 + kind) * (size_t)g.page_size * g.head_dim;
}


// Element index inside a block.
DASH_DEV size_t k_index_f32(const KVGeom& g, int key, int d) { return (size_t)key * g.head_dim + d; }
DASH_DEV size_t k_index_bf16(const KVGeom& g, int key, int d) {
    return ((size_t)(d >> 5) * g.page_size + key) * 32 + (d & 31);
}
// bf16 V block: [ps / 32][4][hd][8].  Each run of 32 keys is split into four
// groups of 8 (group j: keys 4j .. 4j+3 and 16+4j .. 16+4j+3, the keys whose scores
// one lane of the score MFMA holds), stored dim-major with the group's 8 keys
// contiguous: a lane's P.V operand is one 16-byte read, and appending one key
// writes 16-byte-strided values (32 lines of 64 bytes per kv head at hd = 128).
DASH_DEV size_t v_index_bf16(const KVGeom& g, int key, int d) {
    const int kk = key & 31, grp = (kk & 15) >> 2, p = (kk & 3) + ((kk >> 4) << 2);
    return ((size_t)((key >> 5) * 4 + grp) * g.head_dim + d) * 8 + p;
}

template <typename T> DASH_DEV size_t k_index(const KVGeom& g, int key, int d);
template <> DASH_DEV size_t k_index<float>(const KVGeom& g, int key, int d) { return k_index_f32(g, key, d); }
template <> DASH_DEV size_t k_index<bf16_t>(const KVGeom& g, int key, int d) { return k_index_bf16(g, key, d); }
template <typename T> DASH_DEV size_t v_index(const KVGeom& g, int key, int d);
template <> DASH_DEV size_t v_index<float>(const KVGeom& g, int key, int d) { return k_index_f32(g, key, d); }
template <> DASH_DEV size_t v_index<bf16_t>(const KVGeom& g, int key, int d) { return v_index_bf16(g, key, d); }

}  // namespace dash
