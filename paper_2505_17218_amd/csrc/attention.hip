// Attention over the paged KV cache.
//
// Decode (bf16): one wave per (row, kv head, context split).  All query heads
// that share the kv head (GQA group, <= 16) ride in the N dimension of
// v_mfma_f32_16x16x32_bf16:
//   S^T[key, head] = K[key, :] . Q[head, :]      (A = K tile, B = Q^T)
//   O^T[dim, head] += V^T[dim, key] . P^T[key, head]   (A = V^T tile, B = P^T)
// The K page layout ([chunk of 32 dims][key][32]) and the transposed V page
// layout (dim-major groups of 8 keys, see v_index_bf16) make every A-operand load
// a 16-byte read per lane (K: a contiguous 1 KB per wave; V: four 256-byte runs),
// straight from HBM into VGPRs: nothing is shared between waves, so there is no
// LDS round trip.  The S^T accumulator
// gives each lane 4 consecutive keys of one head per 16-key half; those 8
// probabilities are exactly the lane's P^T operand, so no shuffles are needed
// between the two MFMAs.  Online softmax in fp32 (base 2), with per-lane partial
// denominators reduced once at the end.  Long contexts are split across
// workgroups and merged by a second kernel in a fixed order (deterministic).
//
// Prefill (bf16): the same MFMA block step with the 16 columns being 16
// consecutive query positions of one head, masked causally per column.
//
// Generic (fp32 caches): one wave per (row, query head), scores with lanes over
// keys and the value sum with lanes over dims.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace dash {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
// Cache policies of the K/V block loads.  Decode streams (non-temporal) the blocks
// that only one row reads: measured on gfx950 with the last-level cache cold, the
// plain policy streams the cache at ~4.4 TB/s and the non-temporal one at ~6.0 TB/s.
// Blocks below KVGeom::shared_keys (a prompt group's shared pages, read by all the
// group's rows at about the same time) keep the default policy.
// Prefill keeps the default: each key block is read again by every 16-query column
// block of its sequence and should stay cached (streaming it measured 1.75x slower).
constexpr int kKvStream = 2, kKvReuse = 0;

// s_waitcnt vmcnt(n), the other counters left alone (gfx9 encoding, n < 64)
template <int n>
DASH_DEV void vm_wait() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (n & 15) | ((n >> 4) << 14));
}

// ---- shared MFMA block step ---------------------------------------------
// A wave attends 16 "columns" (decode: the query heads of one GQA group;
// prefill: 16 consecutive query positions of one head) to one block of 32 keys.

template <int HD>
struct KVRegs {
    uint4 k[2][HD / 32];  // A operand of S^T = K Q^T: keys h*16 + (lane & 15), dims c*32 + (lane >> 4)*8 ..
    uint4 v[HD / 16];     // A operand of O^T = V^T P^T: dims d*16 + (lane & 15), 8 permuted keys of lane group
};

// Load the block of 32 keys starting at key `kin` of a page (kin % 32 == 0).
// Buffer loads over the page's K and V blocks: an unbacked page gets an empty
// range and reads as zeros, so the loads carry no branch and the next block can
// be in flight while the current one is multiplied.  Keys from `nvalid` on (past
// the row's context in its last block) are not read: their K loads, and the V
// loads of a lane group whose eight keys all lie there, take an offset past the
// range and return zeros without touching memory.  Their scores are masked and
// their V zeroed by the block step anyway, so the results are the same.
template <int HD, int POLICY>
DASH_DEV void load_kv(KVRegs<HD>& r, const bf16_t* kb, const bf16_t* vb, int ps, int kin, bool ok, int col, int grp,
                      int nvalid = 32) {
    const int bytes = ok ? ps * HD * 2 : 0;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(kb), 0, bytes, kBufferDword3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(vb), 0, bytes, kBufferDword3);
    constexpr uint32_t kOut = 0x80000000u;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const bool kin_ctx = h * 16 + col < nvalid;
#pragma unroll
        for (int c = 0; c < HD / 32; ++c) {
            const uint32_t off = (uint32_t)(((c * ps + kin + h * 16 + col) * 32 + grp * 8) * 2);
            r.k[h][c] = __builtin_bit_cast(
                uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, kin_ctx ? off : kOut, 0, POLICY));
        }
    }
    const bool vin_ctx = grp * 4 < nvalid;  // keys grp*4 .. +3 and 16 + grp*4 .. +3
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
        const uint32_t off = (uint32_t)(((((kin >> 5) * 4 + grp) * HD + d * 16 + col) * 8) * 2);
        r.v[d] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, vin_ctx ? off : kOut, 0, POLICY));
    }
}

template <int HD>
struct AttnState {
    f32x4_t acc[HD / 16];  // acc[d][i] = O^T[dim d*16 + grp*4 + i][column]
    float m, l;            // running max (log2 domain) and this lane's partial denominator
};

template <int HD>
DASH_DEV void attn_init(AttnState<HD>& st) {
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) st.acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m = -INFINITY;
    st.l = 0.f;
}

// Maximum over the four lanes of a column (lanes col, col+16, col+32, col+48), in every
// one of them: the gfx950 lane-swap moves exchange 16-lane rows within each half, then the
// halves, so both steps stay in the vector unit (an LDS permute each would put two LDS
// round trips on every block's chain).  A swap of a value with itself hands each lane its
// partner's value in one of the two results, and max is symmetric: the same bits as
// max(x, x of lane ^ 16) then ^ 32.
DASH_DEV float wave_max_cols(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// One block: keys key0 .. key0+31; this lane's column sees keys < lim; keys >= vlim
// (wave-uniform) may hold stale data and have their V zeroed.
template <int HD>
DASH_DEV void attn_block(AttnState<HD>& st, KVRegs<HD>& r, const bf16x8_t (&qf)[HD / 32], int key0, int lim, int vlim,
                         float scale_log2, int grp) {
    f32x4_t s[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        s[h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < HD / 32; ++c)
            s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, r.k[h][c]), qf[c], s[h], 0, 0, 0);
    }
    // lane holds keys key0 + h*16 + grp*4 + i of its column
    float t[8];
    float mx = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int key = key0 + h * 16 + grp * 4 + i;
            const float v = key < lim ? s[h][i] * scale_log2 : -INFINITY;
            t[h * 4 + i] = v;
            mx = fmaxf(mx, v);
        }
    mx = wave_max_cols(mx);
    const float m_new = fmaxf(st.m, mx);
    // a column with no visible key yet keeps m = -inf: use 0 as the reference so no NaN appears
    const float ref = m_new == -INFINITY ? 0.f : m_new;
    // the hardware exp2 (v_exp_f32): the library exp2f adds a rescaling step for results
    // below 2^-126, which it would otherwise flush to zero; a probability that small
    // changes none of the fp32 sums it enters (the largest entry contributes 1)
    const float alpha = __builtin_amdgcn_exp2f(st.m - ref);
    st.m = m_new;
    // The probabilities enter the P.V MFMA as two bf16 operands, p = hi + lo with
    // hi = bf16(p) and lo = bf16(p - hi) (the difference is exact in fp32): the product
    // then carries p to ~2^-17 relative instead of bf16's 2^-9, in step with the fp32
    // denominator.  Rounding p to bf16 alone moved the 1.5B-shape logits by up to 0.06
    // through 28 layers; the second MFMA is nearly free in this memory-bound kernel.
    float psum = 0.f;
    uint32_t pk[4], pl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float p0 = __builtin_amdgcn_exp2f(t[2 * i] - ref), p1 = __builtin_amdgcn_exp2f(t[2 * i + 1] - ref);
        psum += p0 + p1;
        const bf16_t h0 = f2bf(p0), h1 = f2bf(p1);
        pk[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        pl[i] = (uint32_t)f2bf(p0 - bf2f(h0)) | ((uint32_t)f2bf(p1 - bf2f(h1)) << 16);
    }
    st.l = st.l * alpha + psum;
    const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, make_uint4(pk[0], pk[1], pk[2], pk[3]));
    const bf16x8_t pf_lo = __builtin_bit_cast(bf16x8_t, make_uint4(pl[0], pl[1], pl[2], pl[3]));
    if (key0 + 32 > vlim) {  // zero V of keys past the written context (0 * non-finite stale data = NaN)
#pragma unroll
        for (int d = 0; d < HD / 16; ++d) {
            uint32_t w[4] = {r.v[d].x, r.v[d].y, r.v[d].z, r.v[d].w};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int kk = j < 4 ? grp * 4 + j : 16 + grp * 4 + (j - 4);
                if (key0 + kk >= vlim) w[j >> 1] &= (j & 1) ? 0x0000FFFFu : 0xFFFF0000u;
            }
            r.v[d] = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
        st.acc[d] *= alpha;
        st.acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, r.v[d]), pf_lo, st.acc[d], 0, 0, 0);
        st.acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, r.v[d]), pf, st.acc[d], 0, 0, 0);
    }
}

// Sum the per-lane partial denominators of each column (lanes col, col+16, col+32, col+48).
template <int HD>
DASH_DEV float attn_denominator(const AttnState<HD>& st) {
    float l = st.l;
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    return l;
}

// Store the normalised column (4 consecutive dims per 16-dim block) as bf16.
template <int HD>
DASH_DEV void attn_store(const AttnState<HD>& st, float l, bf16_t* orow, int grp) {
    const float inv = l > 0.f ? 1.0f / l : 0.f;
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
        const uint32_t lo = (uint32_t)f2bf(st.acc[d][0] * inv) | ((uint32_t)f2bf(st.acc[d][1] * inv) << 16);
        const uint32_t hi = (uint32_t)f2bf(st.acc[d][2] * inv) | ((uint32_t)f2bf(st.acc[d][3] * inv) << 16);
        *reinterpret_cast<uint2*>(orow + d * 16 + grp * 4) = make_uint2(lo, hi);
    }
}

// The online-softmax state of one column in memory (kPrefixStateStride<HD> floats per
// row and query head): the accumulators in the partial layout (dims d*16 + grp*4 ..
// +4), then each lane group's partial denominator, then the running max.  Storing and
// reloading it moves the exact register values, so a chain continued from it gives
// the same bits as one run through.
template <int HD>
constexpr int kPrefixStateStride = HD + 8;

template <int HD>
DASH_DEV void attn_state_store(const AttnState<HD>& st, float* sp, int grp) {
#pragma unroll
    for (int d = 0; d < HD / 16; ++d)
        *reinterpret_cast<float4*>(sp + d * 16 + grp * 4) = make_float4(st.acc[d][0], st.acc[d][1], st.acc[d][2], st.acc[d][3]);
    sp[HD + grp] = st.l;
    if (grp == 0) sp[HD + 4] = st.m;
}

template <int HD>
DASH_DEV void attn_state_load(AttnState<HD>& st, const float* sp, int grp) {
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
        const float4 v = *reinterpret_cast<const float4*>(sp + d * 16 + grp * 4);
        st.acc[d] = f32x4_t{v.x, v.y, v.z, v.w};
    }
    st.l = sp[HD + grp];
    st.m = sp[HD + 4];
}

// ---- decode ----------------------------------------------------------------

// Head dim 64 asks the compiler for four waves per SIMD (122 registers instead of 150:
// 9-10% less attention time at 257-768 keys for the 0.5B shape); head dim 128 keeps its
// two (the same target there gave it 211 registers and was 2% slower at 1280 keys).
template <int HD, bool PRE = false>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(HD == 64 ? 4 : 1)))
decode_attn_bf16_k(const bf16_t* __restrict__ q, const int32_t* __restrict__ pos,
                                                         const int32_t* __restrict__ slot,
                                                         const int32_t* __restrict__ page_table,
                                                         const bf16_t* __restrict__ pool, KVGeom g, int layer,
                                                         int n_heads, bf16_t* __restrict__ o, int max_splits,
                                                         float* __restrict__ part, float scale_log2,
                                                         const float* __restrict__ pre_state, int pre_blocks) {
    constexpr int NC = HD / 32;
    constexpr int ND = HD / 16;
    const int lane = threadIdx.x;
    const int n_kv = g.n_kv;
    // work items: split fastest, then kv head, then row, dealt to XCDs in contiguous
    // runs.  Every XCD gets whole rows with all their splits (the splits past a short
    // context, which exit at once, are spread evenly instead of filling the last XCDs),
    // and the rows of one prompt group read their shared prompt pages through one L2.
    const int wi = xcd_remap(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
    const int rk = wi / gridDim.y, split = wi % gridDim.y;
    const int row = rk / n_kv, kvh = rk % n_kv;
    const int rep = n_heads / n_kv;
    const int head = lane & 15, grp = lane >> 4;
    const int ctx = pos[row] + 1;
    const int sl = slot[row];
    const int nblk = (ctx + 31) >> 5;
    const int per = g.split_keys >> 5;  // key blocks per split
    const int nsplit = min((nblk + per - 1) / per, max_splits);  // rows past max_ctx are not valid input
    if (split >= nsplit) return;
    int b_begin = split * per;
    const int b_end = min(nblk, b_begin + per);

    // Q^T operand per 32-dim chunk: lane holds q[head][c*32 + grp*8 .. +8] (zero for padding heads).
    bf16x8_t qf[NC];
    {
        const bf16_t* qrow = q + ((size_t)row * n_heads + kvh * rep + (head < rep ? head : 0)) * HD;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            uint4 v = head < rep ? *reinterpret_cast<const uint4*>(qrow + c * 32 + grp * 8) : make_uint4(0, 0, 0, 0);
            qf[c] = __builtin_bit_cast(bf16x8_t, v);
        }
    }
    AttnState<HD> st;
    attn_init(st);
    if (PRE && split == 0 && pre_blocks > 0) {
        // the row's first pre_blocks blocks (its group's shared prompt pages) were run by
        // decode_attn_prefix_k: continue the chain from the state it left
        if (head < rep) attn_state_load<HD>(st, pre_state + ((size_t)row * n_heads + kvh * rep + head) * kPrefixStateStride<HD>, grp);
        b_begin = pre_blocks;
    }
    // two register sets: block b + 1 is fetched while block b is multiplied
    KVRegs<HD> r[2];
    auto fetch = [&](KVRegs<HD>& dst, int b) {
        const int key0 = b << 5;
        int page = kv_page_of(g, page_table, sl, key0);
        const bool ok = page >= 0;
        page = ok ? page : 0;
        const bf16_t* kb = pool + kv_block(g, layer, page, kvh, 0);
        const bf16_t* vb = pool + kv_block(g, layer, page, kvh, 1);
        if (key0 < g.shared_keys)  // wave-uniform: a prompt page the other rows of the group read too
            load_kv<HD, kKvReuse>(dst, kb, vb, g.page_size, key0 % g.page_size, ok, head, grp, ctx - key0);
        else
            load_kv<HD, kKvStream>(dst, kb, vb, g.page_size, key0 % g.page_size, ok, head, grp, ctx - key0);
    };
    if (!PRE || b_begin < b_end) {  // only a continued chain can be empty
        fetch(r[0], b_begin);
        for (int b = b_begin; b < b_end; b += 2) {
            fetch(r[1], min(b + 1, b_end - 1));
            attn_block<HD>(st, r[0], qf, b << 5, ctx, ctx, scale_log2, grp);
            if (b + 1 >= b_end) break;
            fetch(r[0], min(b + 2, b_end - 1));
            attn_block<HD>(st, r[1], qf, (b + 1) << 5, ctx, ctx, scale_log2, grp);
        }
    }
    const float l = attn_denominator(st);
    if (head >= rep) return;
    const int qh = kvh * rep + head;
    if (nsplit == 1) {  // the only split: normalise and store
        attn_store<HD>(st, l, o + ((size_t)row * n_heads + qh) * HD, grp);
    } else {
        const size_t base = ((size_t)row * n_heads + qh) * max_splits + split;
        float* op = part + base * HD;
#pragma unroll
        for (int d = 0; d < ND; ++d)
            *reinterpret_cast<float4*>(op + d * 16 + grp * 4) =
                make_float4(st.acc[d][0], st.acc[d][1], st.acc[d][2], st.acc[d][3]);
        if (grp == 0) {
            float* ml = part + (size_t)(gridDim.x / n_kv) * n_heads * max_splits * HD + base * 2;
            ml[0] = st.m;
            ml[1] = l;
        }
    }
}

// ---- decode, prefix-shared groups --------------------------------------------
// The G samples of a prompt share the prompt's full pages (the group fork), and for
// every query column the per-row chain above starts with those shared blocks.  This
// kernel runs that first part of the chain once per (group, kv head) for all the
// group's query columns, G x rep of them in tiles of 16, one wave per tile, with the
// group's shared pages fetched once into LDS (whole pages, copied verbatim by
// direct-to-LDS loads, so a lane's fragment sits at the same offset as in memory);
// it leaves each column's state for decode_attn_bf16_k, which continues every row over
// its own blocks.  Per column the blocks, the arithmetic and its order are those of
// the per-row chain, so the results are bit-identical to decode_attn_bf16_k alone.
// Column c of group [r0, r1) is row r0 + c / rep, query head kvh * rep + c % rep.
// Pages go through LDS in chunks of kPrefixLdsBytes (all of a 256-key prompt's pages
// at head dim 128 and page size 32).
constexpr int kPrefixLdsBytes = 128 * 1024;

template <int HD>
__global__ void __launch_bounds__(512) decode_attn_prefix_k(const bf16_t* __restrict__ q, const int32_t* __restrict__ pos,
                                                            const int32_t* __restrict__ slot,
                                                            const int32_t* __restrict__ page_table,
                                                            const bf16_t* __restrict__ pool, KVGeom g, int layer,
                                                            int n_heads, const int32_t* __restrict__ group_off,
                                                            int pre_blocks, float* __restrict__ state, float scale_log2) {
    constexpr int NC = HD / 32, ND = HD / 16;
    __shared__ __attribute__((aligned(1024))) char lds[kPrefixLdsBytes];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nw = blockDim.x >> 6;
    const int n_kv = g.n_kv;
    const int gi = blockIdx.x / n_kv, kvh = blockIdx.x % n_kv;
    const int r0 = group_off[gi], r1 = group_off[gi + 1];
    if (r1 <= r0) return;  // uniform over the workgroup
    const int rep = n_heads / n_kv;
    const int head = lane & 15, grp = lane >> 4;
    const int c = w * 16 + head;  // this lane's column
    const bool valid = c < (r1 - r0) * rep;
    const int row = valid ? r0 + c / rep : r0;
    const int qh = kvh * rep + (valid ? c % rep : 0);
    const int ctx = pos[row] + 1;

    bf16x8_t qf[NC];
    {
        const bf16_t* qrow = q + ((size_t)row * n_heads + qh) * HD;
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            uint4 v = valid ? *reinterpret_cast<const uint4*>(qrow + i * 32 + grp * 8) : make_uint4(0, 0, 0, 0);
            qf[i] = __builtin_bit_cast(bf16x8_t, v);
        }
    }
    AttnState<HD> st;
    attn_init(st);

    const int ps = g.page_size;
    const int blk_bytes = ps * HD * 2;        // a page's K (or V) block
    const int units = blk_bytes >> 10;        // 1 KB copies per block
    const int ppc = kPrefixLdsBytes / (2 * blk_bytes);  // pages per LDS chunk (>= 1, checked by the launcher)
    const int bpp = ps >> 5;                  // 32-key blocks per page
    const int n_pages = pre_blocks / bpp;
    const int sl0 = slot[r0];
    for (int p0 = 0; p0 < n_pages; p0 += ppc) {
        const int np = min(ppc, n_pages - p0);
        // copy: unit u = (page j, kind, 1 KB piece) lands at LDS (2 j + kind) * blk_bytes + piece * 1 KB
        int issued = 0;
        for (int u = w; u < np * 2 * units; u += nw) {
            const int j = u / (2 * units), kind = (u / units) & 1, piece = u % units;
            int page = kv_page_of(g, page_table, sl0, (p0 + j) * ps);
            const bool ok = page >= 0;
            page = ok ? page : 0;
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<bf16_t*>(pool + kv_block(g, layer, page, kvh, kind)), 0, ok ? blk_bytes : 0, kBufferDword3);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void*)(lds + (2 * j + kind) * blk_bytes + piece * 1024), 16,
                piece * 1024 + lane * 16, 0, 0, 0);
            if ((++issued & 15) == 0) vm_wait<32>();  // at most 48 copies in flight per wave
        }
        vm_wait<0>();     // this wave's copies have landed
        __syncthreads();                     // and every other wave's
        for (int b = p0 * bpp; b < (p0 + np) * bpp; ++b) {
            const int j = b / bpp - p0, kin = (b % bpp) << 5;
            const char* kb = lds + (2 * j) * blk_bytes;
            const char* vb = kb + blk_bytes;
            KVRegs<HD> r;
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int i = 0; i < NC; ++i)
                    r.k[h][i] = *reinterpret_cast<const uint4*>(kb + ((i * ps + kin + h * 16 + head) * 32 + grp * 8) * 2);
#pragma unroll
            for (int d = 0; d < ND; ++d)
                r.v[d] = *reinterpret_cast<const uint4*>(vb + ((((kin >> 5) * 4 + grp) * HD + d * 16 + head) * 8) * 2);
            attn_block<HD>(st, r, qf, b << 5, ctx, ctx, scale_log2, grp);
        }
        __syncthreads();  // the chunk's LDS is refilled next
    }
    if (valid) attn_state_store<HD>(st, state + ((size_t)row * n_heads + qh) * kPrefixStateStride<HD>, grp);
}

// ---- prefill ---------------------------------------------------------------
// One wave per (prompt, query head, 16 consecutive query positions), causal.
// Rows of a prompt are contiguous: row = prompt * P + position.

template <int HD>
__global__ void __launch_bounds__(64) prefill_attn_bf16_k(const bf16_t* __restrict__ q, const int32_t* __restrict__ slot,
                                                          const int32_t* __restrict__ page_table,
                                                          const bf16_t* __restrict__ pool, KVGeom g, int layer,
                                                          int n_heads, int P, bf16_t* __restrict__ o, float scale_log2) {
    constexpr int NC = HD / 32;
    const int lane = threadIdx.x, col = lane & 15, grp = lane >> 4;
    const int qblocks = (P + 15) >> 4;
    const int prompt = blockIdx.x / qblocks, q0 = (blockIdx.x % qblocks) * 16;
    const int h = blockIdx.y, kvh = h / (n_heads / g.n_kv);
    const int qp = q0 + col;                 // this column's query position
    const bool valid = qp < P;
    const int row = prompt * P + (valid ? qp : q0);
    const int sl = slot[(size_t)prompt * P];
    const int last = min(P, q0 + 16);        // keys < last are written
    bf16x8_t qf[NC];
    {
        const bf16_t* qrow = q + ((size_t)row * n_heads + h) * HD;
#pragma unroll
        for (int c = 0; c < NC; ++c) qf[c] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + c * 32 + grp * 8));
    }
    AttnState<HD> st;
    attn_init(st);
    const int lim = valid ? qp + 1 : 1;
    const int nblk = (last + 31) >> 5;
    KVRegs<HD> r[2];
    auto fetch = [&](KVRegs<HD>& dst, int b) {
        const int key0 = b << 5;
        int page = kv_page_of(g, page_table, sl, key0);
        const bool ok = page >= 0;
        page = ok ? page : 0;
        load_kv<HD, kKvReuse>(dst, pool + kv_block(g, layer, page, kvh, 0), pool + kv_block(g, layer, page, kvh, 1),
                              g.page_size, key0 % g.page_size, ok, col, grp);
    };
    fetch(r[0], 0);
    for (int b = 0; b < nblk; b += 2) {
        fetch(r[1], min(b + 1, nblk - 1));
        attn_block<HD>(st, r[0], qf, b << 5, lim, last, scale_log2, grp);
        if (b + 1 >= nblk) break;
        fetch(r[0], min(b + 2, nblk - 1));
        attn_block<HD>(st, r[1], qf, (b + 1) << 5, lim, last, scale_log2, grp);
    }
    const float l = attn_denominator(st);
    if (valid) attn_store<HD>(st, l, o + ((size_t)row * n_heads + h) * HD, grp);
}

// Merge the context splits of rows that have more than one, in split order:
// o = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.  One wave per (row, head), a
// lane per output dim (two for hd = 128).  Up to MS splits every load is issued
// before any arithmetic (the row's split count only masks which values enter), so a
// merge costs one memory round trip instead of three dependent ones; loads of
// splits past the row's count stay inside the partial buffer and are never used.
template <typename T, int MS>
__global__ void __launch_bounds__(64) combine_k(const float* __restrict__ part, const int32_t* __restrict__ pos,
                                                int rows, int n_heads, int max_splits, int split_keys, int hd,
                                                T* __restrict__ o) {
    const int rh = blockIdx.x;  // row * n_heads + head
    const int row = rh / n_heads;
    const int d0 = threadIdx.x, d1 = threadIdx.x + 64;
    const bool two = d1 < hd;
    const float* ml = part + (size_t)rows * n_heads * max_splits * hd + (size_t)rh * max_splits * 2;
    const float* pr = part + (size_t)rh * max_splits * hd;
    const int p = pos[row];
    float mv[MS], lv[MS], x0[MS], x1[MS];
#pragma unroll
    for (int s = 0; s < MS; ++s) {
        mv[s] = lv[s] = x0[s] = x1[s] = 0.f;
        if (s < max_splits) {
            mv[s] = ml[2 * s];
            lv[s] = ml[2 * s + 1];
            x0[s] = pr[(size_t)s * hd + d0];
            x1[s] = two ? pr[(size_t)s * hd + d1] : 0.f;
        }
    }
    const int ns = min((p + split_keys) / split_keys, max_splits);  // ceil((pos + 1) / split keys)
    if (ns <= 1) return;  // written directly by the attention kernel
    float M = -INFINITY;
#pragma unroll
    for (int s = 0; s < MS; ++s)
        if (s < ns) M = fmaxf(M, mv[s]);
    float den = 0.f, n0 = 0.f, n1 = 0.f;
#pragma unroll
    for (int s = 0; s < MS; ++s) {
        if (s < ns) {
            const float w = exp2f(mv[s] - M);
            den += w * lv[s];
            n0 += w * x0[s];
            n1 += w * x1[s];
        }
    }
    const float inv = den > 0.f ? 1.0f / den : 0.f;
    st_elem(o + (size_t)rh * hd + d0, n0 * inv);
    if (two) st_elem(o + (size_t)rh * hd + d1, n1 * inv);
}

// The same merge for rows with more splits than combine_k unrolls (loads per split).
template <typename T>
__global__ void __launch_bounds__(64) combine_many_k(const float* __restrict__ part, const int32_t* __restrict__ pos,
                                                     int rows, int n_heads, int max_splits, int split_keys, int hd,
                                                     T* __restrict__ o) {
    const int rh = blockIdx.x;
    const int row = rh / n_heads;
    const int ns = min((pos[row] + split_keys) / split_keys, max_splits);
    if (ns <= 1) return;
    const float* ml = part + (size_t)rows * n_heads * max_splits * hd + (size_t)rh * max_splits * 2;
    const float* pr = part + (size_t)rh * max_splits * hd;
    float M = -INFINITY;
    for (int s = 0; s < ns; ++s) M = fmaxf(M, ml[2 * s]);
    for (int d = threadIdx.x; d < hd; d += 64) {
        float den = 0.f, num = 0.f;
        for (int s = 0; s < ns; ++s) {
            const float w = exp2f(ml[2 * s] - M);
            den += w * ml[2 * s + 1];
            num += w * pr[(size_t)s * hd + d];
        }
        st_elem(o + (size_t)rh * hd + d, num * (den > 0.f ? 1.0f / den : 0.f));
    }
}

// Generic paged attention: grid (rows, n_heads), one wave.  Row r attends to
// positions 0..pos[r] of slot[r].
template <typename T>
__global__ void __launch_bounds__(64) attn_generic_k(const T* __restrict__ q, const int32_t* __restrict__ pos,
                                                     const int32_t* __restrict__ slot,
                                                     const int32_t* __restrict__ page_table,
                                                     const T* __restrict__ pool, KVGeom g, int layer, int n_heads,
                                                     T* __restrict__ o, float scale) {
    __shared__ float qs[128];
    __shared__ float ps[64];
    __shared__ int pg[64];
    const int row = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    const int hd = g.head_dim, rep = n_heads / g.n_kv, kvh = h / rep;
    const int ctx = pos[row] + 1, sl = slot[row];
    const T* qrow = q + ((size_t)row * n_heads + h) * hd;
    for (int d = lane; d < hd; d += 64) qs[d] = ld_elem(qrow + d);
    __syncthreads();
    float m_run = -INFINITY, l_run = 0.f, acc0 = 0.f, acc1 = 0.f;
    for (int base = 0; base < ctx; base += 64) {
        const int key = base + lane;
        float s = -INFINITY;
        int page = -1;
        if (key < ctx) {
            page = kv_page_of(g, page_table, sl, key);
            if (page >= 0) {
                const T* kb = pool + kv_block(g, layer, page, kvh, 0);
                const int kin = key % g.page_size;
                float dot = 0.f;
                for (int d = 0; d < hd; ++d) dot += qs[d] * ld_elem(kb + k_index<T>(g, kin, d));
                s = dot * scale;
            }
        }
        const float cmax = wave_max(s);
        const float m_new = fmaxf(m_run, cmax);
        const float alpha = m_new == -INFINITY ? 1.f : __expf(m_run - m_new);
        const float p = s == -INFINITY ? 0.f : __expf(s - m_new);
        l_run = l_run * alpha + wave_sum(p);
        acc0 *= alpha;
        acc1 *= alpha;
        m_run = m_new;
        ps[lane] = p;
        pg[lane] = page;
        __syncthreads();
        const int n = min(64, ctx - base);
        for (int j = 0; j < n; ++j) {
            const float pj = ps[j];
            const int pgj = pg[j];
            if (pj == 0.f || pgj < 0) continue;
            const T* vb = pool + kv_block(g, layer, pgj, kvh, 1);
            const int kin = (base + j) % g.page_size;
            if (lane < hd) acc0 += pj * ld_elem(vb + v_index<T>(g, kin, lane));
            if (lane + 64 < hd) acc1 += pj * ld_elem(vb + v_index<T>(g, kin, lane + 64));
        }
        __syncthreads();
    }
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
    T* orow = o + ((size_t)row * n_heads + h) * hd;
    if (lane < hd) st_elem(orow + lane, acc0 * inv);
    if (lane + 64 < hd) st_elem(orow + lane + 64, acc1 * inv);
}

}  // namespace

int attention_split_keys(int max_seqs, int n_kv, int max_ctx, int head_dim) {
    const auto waves = [&](long s) { return (long)max_seqs * n_kv * ((max_ctx + s - 1) / s); };
    // about as many waves as fit the GPU at once: the hd-128 kernel's registers allow two
    // per SIMD; for hd 64 (four per SIMD) three per SIMD measured best (at 512 sequences of
    // the 0.5B shape: split 512, 18% less attention time than split 1024, and the whole
    // rollout 2% faster than split 256)
    const long target = head_dim == 64 ? 3L * kAttnTargetWaves / 2 : kAttnTargetWaves;
    int s = kAttnMinSplitKeys;
    while (s < max_ctx && s < (1 << 20) && waves(2L * s) >= target) s *= 2;
    return s;
}

size_t attention_partial_floats(int rows, int n_heads, int head_dim, int max_ctx) {
    const int ms = (max_ctx + kAttnMinSplitKeys - 1) / kAttnMinSplitKeys;
    if (ms <= 1) return 0;
    return (size_t)rows * n_heads * ms * (head_dim + 2);
}

hipError_t launch_decode_attention(int dtype, const void* q, const int32_t* pos, const int32_t* slot,
                                   const int32_t* page_table, const void* pool, const KVGeom& g, int layer,
                                   int n_heads, void* o, int rows, int max_ctx, float* ws_part, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    const float scale = 1.0f / sqrtf((float)g.head_dim);
    if (dtype == 1) {
        const int ms = std::max(1, (max_ctx + g.split_keys - 1) / g.split_keys);
        dim3 grid(rows * g.n_kv, ms);
        const float sl2 = scale * kLog2e;
        if (g.head_dim == 128)
            decode_attn_bf16_k<128><<<grid, 64, 0, st>>>((const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool,
                                                          g, layer, n_heads, (bf16_t*)o, ms, ws_part, sl2, nullptr, 0);
        else if (g.head_dim == 64)
            decode_attn_bf16_k<64><<<grid, 64, 0, st>>>((const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool,
                                                         g, layer, n_heads, (bf16_t*)o, ms, ws_part, sl2, nullptr, 0);
        else
            return hipErrorInvalidValue;
        return hipGetLastError();
    }
    dim3 grid(rows, n_heads);
    attn_generic_k<float><<<grid, 64, 0, st>>>((const float*)q, pos, slot, page_table, (const float*)pool, g, layer,
                                               n_heads, (float*)o, scale);
    return hipGetLastError();
}

bool decode_attention_prefix_ok(const KVGeom& g, int n_heads, int group_size, int shared_len) {
    const int blk_bytes = g.page_size * g.head_dim * 2;
    return (g.head_dim == 64 || g.head_dim == 128) && g.page_size % 32 == 0 && blk_bytes % 1024 == 0 &&
           2 * blk_bytes <= kPrefixLdsBytes && shared_len >= g.page_size && g.split_keys >= g.page_size &&
           group_size >= 1 && ((long)group_size * (n_heads / g.n_kv) + 15) / 16 <= 8;
}

size_t decode_attention_prefix_state_bytes(int rows, int n_heads, int head_dim) {
    return (size_t)rows * n_heads * (head_dim + 8) * 4;
}

hipError_t launch_decode_attention_grouped(const void* q, const int32_t* pos, const int32_t* slot,
                                           const int32_t* page_table, const void* pool, const KVGeom& g, int layer,
                                           int n_heads, const int32_t* group_off, int n_groups, int group_size,
                                           int shared_len, void* o, int rows, int max_ctx, float* ws_part,
                                           float* ws_state, hipStream_t st) {
    if (rows <= 0 || n_groups <= 0) return hipSuccess;
    if (!ws_state || !decode_attention_prefix_ok(g, n_heads, group_size, shared_len)) return hipErrorInvalidValue;
    const float sl2 = kLog2e / sqrtf((float)g.head_dim);
    // the prefix covers the shared pages inside the first context split (whole pages)
    const int pre_keys = std::min(shared_len, g.split_keys / g.page_size * g.page_size);
    const int pre_blocks = pre_keys >> 5;
    const int nw = (group_size * (n_heads / g.n_kv) + 15) / 16;
    const int ms = std::max(1, (max_ctx + g.split_keys - 1) / g.split_keys);
    dim3 grid(rows * g.n_kv, ms);
    if (g.head_dim == 128) {
        decode_attn_prefix_k<128><<<n_groups * g.n_kv, 64 * nw, 0, st>>>(
            (const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool, g, layer, n_heads, group_off, pre_blocks,
            ws_state, sl2);
        decode_attn_bf16_k<128, true><<<grid, 64, 0, st>>>((const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool,
                                                            g, layer, n_heads, (bf16_t*)o, ms, ws_part, sl2, ws_state,
                                                            pre_blocks);
    } else {
        decode_attn_prefix_k<64><<<n_groups * g.n_kv, 64 * nw, 0, st>>>(
            (const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool, g, layer, n_heads, group_off, pre_blocks,
            ws_state, sl2);
        decode_attn_bf16_k<64, true><<<grid, 64, 0, st>>>((const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool,
                                                           g, layer, n_heads, (bf16_t*)o, ms, ws_part, sl2, ws_state,
                                                           pre_blocks);
    }
    return hipGetLastError();
}

hipError_t launch_attention_combine(int dtype, const int32_t* pos, int rows, int n_heads, int head_dim,
                                    int max_ctx, int split_keys, const float* ws_part, void* o, hipStream_t st) {
    const int ms = (max_ctx + split_keys - 1) / split_keys;
    if (dtype != 1 || ms <= 1 || rows <= 0) return hipSuccess;
    if (head_dim != 64 && head_dim != 128) return hipErrorInvalidValue;
    const int grid = rows * n_heads;
    if (ms <= 8)
        combine_k<bf16_t, 8><<<grid, 64, 0, st>>>(ws_part, pos, rows, n_heads, ms, split_keys, head_dim, (bf16_t*)o);
    else if (ms <= 16)
        combine_k<bf16_t, 16><<<grid, 64, 0, st>>>(ws_part, pos, rows, n_heads, ms, split_keys, head_dim, (bf16_t*)o);
    else
        combine_many_k<bf16_t><<<grid, 64, 0, st>>>(ws_part, pos, rows, n_heads, ms, split_keys, head_dim, (bf16_t*)o);
    return hipGetLastError();
}

hipError_t launch_prefill_attention(int dtype, const void* q, const int32_t* pos, const int32_t* slot,
                                    const int32_t* page_table, const void* pool, const KVGeom& g, int layer,
                                    int n_heads, void* o, int rows, int prompt_len, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    const float scale = 1.0f / sqrtf((float)g.head_dim);
    if (dtype == 1 && prompt_len > 0 && rows % prompt_len == 0) {
        dim3 grid((rows / prompt_len) * ((prompt_len + 15) / 16), n_heads);
        const float sl2 = scale * kLog2e;
        if (g.head_dim == 128)
            prefill_attn_bf16_k<128><<<grid, 64, 0, st>>>((const bf16_t*)q, slot, page_table, (const bf16_t*)pool, g,
                                                           layer, n_heads, prompt_len, (bf16_t*)o, sl2);
        else if (g.head_dim == 64)
            prefill_attn_bf16_k<64><<<grid, 64, 0, st>>>((const bf16_t*)q, slot, page_table, (const bf16_t*)pool, g,
                                                          layer, n_heads, prompt_len, (bf16_t*)o, sl2);
        else
            return hipErrorInvalidValue;
        return hipGetLastError();
    }
    dim3 grid(rows, n_heads);
    if (dtype == 1)
        attn_generic_k<bf16_t><<<grid, 64, 0, st>>>((const bf16_t*)q, pos, slot, page_table, (const bf16_t*)pool, g,
                                                    layer, n_heads, (bf16_t*)o, scale);
    else
        attn_generic_k<float><<<grid, 64, 0, st>>>((const float*)q, pos, slot, page_table, (const float*)pool, g,
                                                   layer, n_heads, (float*)o, scale);
    return hipGetLastError();
}

}  // namespace dash
