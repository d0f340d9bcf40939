// Projection GEMMs C = A[M,K] . W[N,K]^T (fp32 accumulation).
//
// bfloat16: v_mfma_f32_32x32x16_bf16 tiles (on gfx950 this MFMA sustains about
// twice the rate of 16x16x32: measured ~2.1 vs ~1.24 PFLOP/s with register-only
// operands).  A workgroup of WGM x WGN waves owns a BM x BN output tile; K
// advances in steps of 64 through a double-buffered LDS tile (row-major, rows
// padded to 72 elements so fragment reads of 16 consecutive rows hit distinct
// banks).  Operands are fetched with raw buffer loads (rows outside the operand
// read as zeros, no branches), PD k-steps ahead of the multiply.  Work items
// (split, m-tile, n-tile) are enumerated m-fastest and dealt to XCDs in
// contiguous runs, so blocks that share a weight tile run on the same XCD and
// reuse it from that XCD's L2.
//
// float32: a plain LDS-tiled VALU kernel (the fp32 shapes are tiny correctness
// configurations).
//
// Epilogues: fp32 store (with split-K partials that the consumer sums in a
// fixed order, so results are deterministic) or SwiGLU, where the B tile pairs
// gate row j with up row j in the same lane and h = silu(gate) * up is stored in
// the model dtype.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace dash {

namespace {

constexpr int kBK = 64;
constexpr int kLdsStride = kBK + 8;  // bf16 elements per LDS row

DASH_DEV float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// ---- direct-to-LDS operand path ----------------------------------------------
// Operand tiles can also go from memory straight into LDS (buffer_load ... lds, 16 bytes
// per lane: one wave instruction fills 1 KB, 8 rows of 64 elements), through a ring of S
// stages: step k + S - 1 is in flight while step k is multiplied, without registers to
// hold it.  LDS rows are unpadded; the 16-byte chunks of a row are XOR-swizzled so that
// 16 consecutive rows read at one logical chunk hit 16 distinct 4-bank groups.
typedef __attribute__((address_space(3))) void lds_void;

template <int BM, int BN>
struct LdsStage {
    bf16_t a[BM * kBK];
    bf16_t b[BN * kBK];
};

DASH_DEV int lds_swizzle(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Fill one stage: AI instructions of 8 A rows, then BI of 8 B rows.  kb is the step's
// byte offset along K; kb >= 2^31 (a step past the end) makes every in-range row read
// out of range, which returns zeros without touching memory, so every step issues the
// same instructions (padding rows, out of range already, may wrap to a harmless read).
template <int AI, int BI, int BM, int BN>
DASH_DEV void lds_dma_stage(LdsStage<BM, BN>& s, const bf16_t* A, int a_bytes, const bf16_t* W, int w_bytes,
                            const uint32_t* a_off, const uint32_t* b_off, uint32_t kb, int wave, int wpol) {
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(A), 0, a_bytes, kBufferDword3);
    const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(W), 0, w_bytes, kBufferDword3);
#pragma unroll
    for (int j = 0; j < AI; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (lds_void*)&s.a[(wave * AI + j) * 8 * kBK], 16, a_off[j] + kb, 0, 0,
                                                 0);
#pragma unroll
    for (int j = 0; j < BI; ++j) {
        if (wpol)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, (lds_void*)&s.b[(wave * BI + j) * 8 * kBK], 16, b_off[j] + kb,
                                                     0, 0, 2);
        else
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, (lds_void*)&s.b[(wave * BI + j) * 8 * kBK], 16, b_off[j] + kb,
                                                     0, 0, 0);
    }
}

// s_waitcnt vmcnt(n) with the other counters left alone (n < 64)
template <int n>
DASH_DEV void wait_vmcnt() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (n & 15) | ((n >> 4) << 14));
}

// s_waitcnt vmcnt(n) lgkmcnt(0): the vector-memory wait, and every LDS read this wave
// has issued has returned its data (n < 64)
template <int n>
DASH_DEV void wait_vmcnt_lds_reads() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0070 | (n & 15) | ((n >> 4) << 14));
}

// ---- epilogues shared by the GEMM kernels ------------------------------------
// acc[i * TN + j][r] of a wave holds row (r / 4) * 8 + (lane / 32) * 4 + r % 4 and column
// lane % 32 of its 32 x 32 block (i, j).

template <int BM, int BN, int WGM, int WGN>
DASH_DEV void store_f32_epilogue(const f32x16_t* acc, float* Cp, int M, int N, int ldc, int m0, int nt, int lane,
                                 int wr, int wc) {
    constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    const int rbase = (lane >> 5) * 4, ccol = lane & 31;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = nt * BN + wc * WN + j * 32 + ccol;
            if (n >= N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wr * WM + i * 32 + (r >> 2) * 8 + rbase + (r & 3);
                if (m < M) Cp[(size_t)m * ldc + n] = acc[i * TN + j][r];
            }
        }
}

// h = silu(gate) * up: a wave's column blocks hold TN/2 gate blocks, then the TN/2 up
// blocks of the same columns
template <int BM, int BN, int WGM, int WGN>
DASH_DEV void swiglu_epilogue(const f32x16_t* acc, bf16_t* H, int M, int N, int ldc, int m0, int nt, int lane, int wr,
                              int wc) {
    constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    const int rbase = (lane >> 5) * 4, ccol = lane & 31;
    const int ff = N >> 1;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN / 2; ++j) {
            const int col = nt * (BN / 2) + wc * (WN / 2) + j * 32 + ccol;
            if (col >= ff) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wr * WM + i * 32 + (r >> 2) * 8 + rbase + (r & 3);
                if (m < M) H[(size_t)m * ldc + col] = f2bf(silu(acc[i * TN + j][r]) * acc[i * TN + j + TN / 2][r]);
            }
        }
}

// The same h through LDS: each wave writes its values of the BM x BN/2 output tile into
// LDS (rows padded by 8 elements), then every thread stores whole 16-byte runs of 8
// columns, so a tile row leaves as full lines instead of 2-byte stores per element.
// Needs ldc and the tile's columns in whole runs of 8 and H 16-byte aligned (the caller
// checks); Hs is dead operand LDS of at least BM * (BN/2 + 8) elements, and every wave
// must be past its last read of it.
template <int BM, int BN, int WGM, int WGN>
DASH_DEV void swiglu_epilogue_lds(const f32x16_t* acc, bf16_t* Hs, bf16_t* H, int M, int N, int ldc, int m0, int nt,
                                  int tid, int wr, int wc) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    constexpr int OW = BN / 2, OS = OW + 8;  // output tile width and LDS row stride (elements)
    constexpr int RUNS = BM * OW / 8;        // 16-byte runs in the tile
    static_assert(RUNS % NT == 0, "runs per thread");
    const int lane = tid & 63;
    const int rbase = (lane >> 5) * 4, ccol = lane & 31;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN / 2; ++j) {
            const int c = wc * (WN / 2) + j * 32 + ccol;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rr = wr * WM + i * 32 + (r >> 2) * 8 + rbase + (r & 3);
                Hs[rr * OS + c] = f2bf(silu(acc[i * TN + j][r]) * acc[i * TN + j + TN / 2][r]);
            }
        }
    __syncthreads();
    const int ff = N >> 1;
#pragma unroll
    for (int u = 0; u < RUNS / NT; ++u) {
        const int run = tid + u * NT, rr = run / (OW / 8), c8 = (run % (OW / 8)) * 8;
        const int m = m0 + rr, col = nt * OW + c8;
        if (m < M && col < ff)
            *reinterpret_cast<uint4*>(H + (size_t)m * ldc + col) = *reinterpret_cast<const uint4*>(Hs + rr * OS + c8);
    }
}

// QKV epilogue inputs (fetched before the main loop so that their latency, for the k / v
// tiles a dependent chain of position and slot, then the page table, hides behind it):
// per tile row its cache page (or -1) and key within the page (row_page / row_key, LDS);
// per thread the bias and the RoPE cosines / sines of its pairs.
template <int BM, int BN, int NT>
struct QkvPre {
    static constexpr int kRows = BM * (BN / 2) / NT;  // RoPE pairs per thread
    static constexpr int kRowsV = BM * BN / NT;       // v elements per thread
    float2 rope_cs[kRows > 0 ? kRows : 1];
    float bias_a = 0.f, bias_b = 0.f;
};

template <int BM, int BN, int NT>
DASH_DEV void qkv_prefetch(const QkvRopeArgs& qa, int M, int N, int m0, int nt, int tid, int* row_page, int* row_key,
                           QkvPre<BM, BN, NT>& pre) {
    static_assert(BN == 128, "the QKV epilogue works on 128-column tiles (whole heads)");
    static_assert(BM * (BN / 2) % NT == 0 && NT % (BN / 2) == 0, "RoPE pair mapping");
    static_assert(BM * BN % NT == 0 && NT % BN == 0, "v mapping");
    const KVGeom& g = qa.g;
    const int hd = g.head_dim, half = hd >> 1;
    const int lg_half = hd == 128 ? 6 : 5;  // head_dim is 64 or 128
    const int n0 = nt * BN;
    const int q_cols = qa.n_heads * hd, k_end_col = q_cols + g.n_kv * hd;
    if (n0 >= q_cols && tid < BM) {
        const int m = m0 + tid;
        int page = -1, key = 0;
        if (m < M) {
            const int p = qa.pos[m];
            page = kv_page_of(g, qa.page_table, qa.slot[m], p);
            key = p % g.page_size;
            if (page < 0 && n0 < k_end_col && qa.status) atomicOr(qa.status, 1u);
        }
        row_page[tid] = page;
        row_key[tid] = key;
    }
    if (n0 < k_end_col) {  // q / k tile: thread t takes pair t % (BN/2) of rows t / (BN/2) + u NT / (BN/2)
        const int pi = tid % (BN / 2), r0 = tid / (BN / 2);
        const int hl = pi >> lg_half, i = pi & (half - 1);
        const int n = n0 + hl * hd + i;
        pre.bias_a = bf2f(qa.bias[n]);
        pre.bias_b = bf2f(qa.bias[n + half]);
#pragma unroll
        for (int u = 0; u < QkvPre<BM, BN, NT>::kRows; ++u) {
            const int m = min(m0 + r0 + u * (NT / (BN / 2)), M - 1);
            pre.rope_cs[u] = *reinterpret_cast<const float2*>(qa.cs + ((size_t)m * half + i) * 2);
        }
    } else {  // v tile: thread t takes column t % BN of rows t / BN + u NT / BN
        const int n = n0 + tid % BN;
        pre.bias_a = n < N ? bf2f(qa.bias[n]) : 0.f;
    }
}

// Stage the fp32 tile in LDS (Cs: BM x (BN + 4) floats of LDS that no wave reads any
// more), then one thread per RoPE pair (q, k tiles) or v element adds the bias, rotates
// and writes q or the cache slot.
template <int BM, int BN, int WGM, int WGN>
DASH_DEV void qkv_epilogue(const f32x16_t* acc, float* Cs, const QkvRopeArgs& qa, int M, int N, int m0, int nt,
                           int tid, int wr, int wc, const int* row_page, const int* row_key,
                           const QkvPre<BM, BN, 64 * WGM * WGN>& pre) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    constexpr int CS = BN + 4;
    constexpr int kRows = QkvPre<BM, BN, NT>::kRows, kRowsV = QkvPre<BM, BN, NT>::kRowsV;
    const int lane = tid & 63;
    const int rbase = (lane >> 5) * 4, ccol = lane & 31;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                Cs[(wr * WM + i * 32 + (r >> 2) * 8 + rbase + (r & 3)) * CS + wc * WN + j * 32 + ccol] = acc[i * TN + j][r];
    __syncthreads();
    const KVGeom& g = qa.g;
    const int hd = g.head_dim, half = hd >> 1;
    const int lg_half = hd == 128 ? 6 : 5, lg_hd = lg_half + 1;  // head indices by shifts, not divisions
    const int n0 = nt * BN;
    const int q_cols = qa.n_heads * hd, k_end = q_cols + g.n_kv * hd;
    if (n0 < k_end) {
        const int pi = tid % (BN / 2), r0 = tid / (BN / 2);
        const int hl = pi >> lg_half, i = pi & (half - 1);
        const int c = hl * hd + i, n = n0 + c;
#pragma unroll
        for (int u = 0; u < kRows; ++u) {
            const int rl = r0 + u * (NT / (BN / 2)), m = m0 + rl;
            if (m >= M) continue;
            const float a = Cs[rl * CS + c] + pre.bias_a;
            const float b = Cs[rl * CS + c + half] + pre.bias_b;
            float lo, hi;
            rope_pair(a, b, pre.rope_cs[u].x, pre.rope_cs[u].y, lo, hi);
            if (n < q_cols) {
                bf16_t* q = qa.q_out + ((size_t)m * qa.n_heads + (n >> lg_hd)) * hd;
                q[i] = f2bf(lo);
                q[i + half] = f2bf(hi);
            } else if (row_page[rl] >= 0) {
                bf16_t* kb = qa.pool + kv_block(g, qa.layer, row_page[rl], (n - q_cols) >> lg_hd, 0);
                // cache appends are non-temporal stores (see the v append below)
                __builtin_nontemporal_store(f2bf(lo), &kb[k_index_bf16(g, row_key[rl], i)]);
                __builtin_nontemporal_store(f2bf(hi), &kb[k_index_bf16(g, row_key[rl], i + half)]);
            }
        }
    } else {
        const int c = tid % BN, r0 = tid / BN;
        const int n = n0 + c, jj = n - k_end;
#pragma unroll
        for (int u = 0; u < kRowsV; ++u) {
            const int rl = r0 + u * (NT / BN), m = m0 + rl;
            if (m >= M || n >= N || row_page[rl] < 0) continue;
            const float v = Cs[rl * CS + c] + pre.bias_a;
            bf16_t* vb = qa.pool + kv_block(g, qa.layer, row_page[rl], jj >> lg_hd, 1);
            // A decode step writes one key per row: 2 bytes into each of the 16-byte groups
            // of 8 keys, lines that later steps read from memory anyway.  Non-temporal
            // stores keep these partial lines out of L2: measured 8% less QKV time and 2%
            // less decode-attention time at 1.5B, 1024 sequences.
            __builtin_nontemporal_store(f2bf(v), &vb[v_index_bf16(g, row_key[rl], jj & (hd - 1))]);
        }
    }
}

// On gfx950 the 32x32x16 bf16 MFMA sustains about twice the rate of 16x16x32
// (measured: ~2.1 vs ~1.24 PFLOP/s with register-only operands), so the main
// kernel uses 32 x 32 output blocks.  Operand layout (per 16-wide k-step): lane l
// holds row (l % 32) and k (l / 32) * 8 .. +8; output register i of lane l is
// row (i / 4) * 8 + (l / 32) * 4 + i % 4, column l % 32.
// LDS tiles are row-major with rows padded to 72 elements (fragment reads of 16
// consecutive rows hit distinct banks); global loads fill full 128-byte rows.
template <int BM, int BN, int WGM, int WGN, int PD, int EPI, int WPOL = 0>
__global__ void __launch_bounds__(64 * WGM * WGN)
gemm_bf16_k(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, void* __restrict__ C, int M, int N, int K,
             int ldc, int m_tiles, int n_tiles, int nt0, int kps, size_t split_stride, QkvRopeArgs qa) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    constexpr int A_CH = BM * 8 / NT, B_CH = BN * 8 / NT;  // 16-byte chunks per thread per k-step
    static_assert(A_CH >= 1 && B_CH >= 1 && BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile / thread mismatch");
    static_assert(TM >= 1 && TN >= 1, "wave tile smaller than one MFMA block");
    static_assert(EPI != EPI_SWIGLU || TN % 2 == 0, "SwiGLU pairs gate/up blocks inside a wave");
    static_assert(EPI != EPI_QKV_ROPE || BN == 128, "the QKV epilogue works on 128-column tiles (whole heads)");
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * kLdsStride];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * kLdsStride];

    const int w = xcd_remap(blockIdx.x, gridDim.x);
    const int mt = w % m_tiles;
    const int rest = w / m_tiles;
    const int nt = nt0 + rest % n_tiles;  // a launch may cover the column tiles from nt0 on
    const int split = rest / n_tiles;
    const int m0 = mt * BM;
    const int k_begin = split * kps;
    const int k_end = min(K, k_begin + kps);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave / WGN, wc = wave % WGN;

    // Operands are read with buffer loads: a row outside the operand gets a byte
    // offset past the buffer's extent, which the hardware returns as zeros, so the
    // loads need no branches and the compiler keeps PD k-steps of them in flight.
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(A), 0, (int)((size_t)M * K * 2), kBufferDword3);
    const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(W), 0, (int)((size_t)N * K * 2), kBufferDword3);
    constexpr uint32_t kOut = 0x80000000u;
    uint32_t a_off[A_CH];
    int a_lds[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
        const int idx = tid + i * NT, row = idx >> 3, kc = idx & 7;
        const int m = m0 + row;
        a_off[i] = m < M ? (uint32_t)(((size_t)m * K + kc * 8) * 2) : kOut;
        a_lds[i] = row * kLdsStride + kc * 8;
    }
    uint32_t b_off[B_CH];
    int b_lds[B_CH];
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
        const int idx = tid + i * NT, row = idx >> 3, kc = idx & 7;
        int n;
        bool ok;
        if (EPI == EPI_SWIGLU) {
            // a wave's N range holds WN/2 gate rows then the WN/2 up rows of the same columns
            const int ff = N >> 1;
            const int wcol = row / WN, rr = row % WN;
            const int j = nt * (BN / 2) + wcol * (WN / 2) + (rr % (WN / 2));
            ok = j < ff;
            n = rr < WN / 2 ? j : ff + j;
        } else {
            n = nt * BN + row;
            ok = n < N;
        }
        b_off[i] = ok ? (uint32_t)(((size_t)n * K + kc * 8) * 2) : kOut;
        b_lds[i] = row * kLdsStride + kc * 8;
    }

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    uint4 ra[PD][A_CH], rb[PD][B_CH];
    auto load = [&](int st, int k0) {
        const uint32_t kb = (uint32_t)k0 * 2;
#pragma unroll
        for (int i = 0; i < A_CH; ++i)
            ra[st][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsA, a_off[i] + kb, 0, 0));
#pragma unroll
        for (int i = 0; i < B_CH; ++i)
            rb[st][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsW, b_off[i] + kb, 0, WPOL));
    };
    auto store = [&](int st, int buf) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) *reinterpret_cast<uint4*>(&As[buf][a_lds[i]]) = ra[st][i];
#pragma unroll
        for (int i = 0; i < B_CH; ++i) *reinterpret_cast<uint4*>(&Bs[buf][b_lds[i]]) = rb[st][i];
    };
    const int frow = lane & 31, fk = (lane >> 5) * 8;
    auto compute = [&](int buf) {
        // let the scheduler interleave LDS reads with the MFMAs (measured: 4-10% faster,
        // same results); the 256x256 tile keeps the variant that does not spill
        if constexpr (BM * BN >= 256 * 256) __builtin_amdgcn_iglp_opt(1);
        else __builtin_amdgcn_iglp_opt(0);
#pragma unroll
        for (int ks = 0; ks < kBK; ks += 16) {
            bf16x8_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const bf16x8_t*>(&As[buf][(wr * WM + i * 32 + frow) * kLdsStride + ks + fk]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(&Bs[buf][(wc * WN + j * 32 + frow) * kLdsStride + ks + fk]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    };

    // QKV epilogue inputs, fetched before the main loop so that their latency hides behind it
    [[maybe_unused]] __shared__ int row_page[EPI == EPI_QKV_ROPE ? BM : 1], row_key[EPI == EPI_QKV_ROPE ? BM : 1];
    [[maybe_unused]] QkvPre<BM, BN, NT> pre;
    if constexpr (EPI == EPI_QKV_ROPE) qkv_prefetch<BM, BN, NT>(qa, M, N, m0, nt, tid, row_page, row_key, pre);

    const int n_k = (k_end - k_begin + kBK - 1) / kBK;
#pragma unroll
    for (int p = 0; p < PD; ++p) load(p, k_begin + p * kBK);
    store(0, 0);
    __syncthreads();
    for (int kt = 0; kt < n_k; kt += PD) {
#pragma unroll
        for (int u = 0; u < PD; ++u) {
            const int k = kt + u;
            // register stage u held step k (already in LDS): refill it with step k + PD
            load(u, k_begin + (k + PD) * kBK);
            if (k < n_k) compute(k & 1);
            if (k + 1 < n_k) store((u + 1) % PD, (k + 1) & 1);
            __syncthreads();
        }
    }

    if constexpr (EPI == EPI_QKV_ROPE) {
        // the fp32 tile is staged in the B operand LDS (dead after the loop's last barrier)
        static_assert(BM * (BN + 4) * 4 <= (int)sizeof(Bs), "C tile must fit the B operand LDS");
        qkv_epilogue<BM, BN, WGM, WGN>(&acc[0][0], reinterpret_cast<float*>(&Bs[0][0]), qa, M, N, m0, nt, tid, wr, wc,
                                       row_page, row_key, pre);
    } else if constexpr (EPI == EPI_STORE_F32) {
        store_f32_epilogue<BM, BN, WGM, WGN>(&acc[0][0], reinterpret_cast<float*>(C) + split * split_stride, M, N, ldc,
                                             m0, nt, lane, wr, wc);
    } else {
        static_assert(EPI == EPI_SWIGLU, "unknown epilogue");
        static_assert(BM * (BN / 2 + 8) <= (int)(sizeof(As) / sizeof(bf16_t)), "h tile must fit the A operand LDS");
        // whole 16-byte runs: ldc, the output width and the base all multiples of 8 elements
        if (((ldc | (N >> 1)) & 7) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0)
            swiglu_epilogue_lds<BM, BN, WGM, WGN>(&acc[0][0], &As[0][0], reinterpret_cast<bf16_t*>(C), M, N, ldc, m0, nt,
                                                  tid, wr, wc);
        else
            swiglu_epilogue<BM, BN, WGM, WGN>(&acc[0][0], reinterpret_cast<bf16_t*>(C), M, N, ldc, m0, nt, lane, wr, wc);
    }
}

// The same product with the direct-to-LDS operand path: S LDS stages, one barrier per
// k-step.  At step k a wave waits until its own part of step k has landed and its own
// reads of step k - 1's stage have returned; the barrier then guarantees every wave's
// part and that no wave still reads step k - 1's stage, which is refilled with step
// k + S - 1, and step k is multiplied.  The wait for the reads matters: a copy into LDS
// is written whenever its data comes back from memory, in no order with LDS reads other
// waves have issued but not completed, so without it a slow read could see the next
// step's data.  (That happened with two decode steps running at once on two streams:
// 32-row blocks of some rows' outputs changed from run to run.)  Each
// stage is its own LDS variable, so the compiler lets the loads of the other stages stay
// in flight while a stage is read.  Same fragments, same MFMA order as gemm_bf16_k:
// identical results.  Measured on the 1.5B decode shapes at 1024 rows (weights cold):
// the output projection 14.7 -> 10.6 us, the QKV projection 15.5 -> 11.5 us with
// 128 x 64 tiles; gate/up, down and the LM head gain nothing (their per-CU rate stays
// at ~30% of the MFMA peak either way), so they keep gemm_bf16_k.
template <int BM, int BN, int WGM, int WGN, int S, int EPI, int WPOL = 0>
__global__ void __launch_bounds__(64 * WGM * WGN)
gemm_lds_k(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, void* __restrict__ C, int M, int N, int K,
           int ldc, int m_tiles, int n_tiles, int kps, size_t split_stride, QkvRopeArgs qa) {
    constexpr int NT = 64 * WGM * WGN, NW = WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    constexpr int AI = BM / 8 / NW, BI = BN / 8 / NW;  // 1 KB load instructions per wave per k-step
    constexpr int DPS = AI + BI;
    static_assert(AI >= 1 && BI >= 1 && BM / 8 % NW == 0 && BN / 8 % NW == 0, "load split");
    static_assert(S >= 3 && S <= 4, "stages");
    static_assert(TM >= 1 && TN >= 1, "wave tile smaller than one MFMA block");
    static_assert(EPI == EPI_STORE_F32 || EPI == EPI_QKV_ROPE, "epilogue");
    __shared__ __attribute__((aligned(1024))) LdsStage<BM, BN> st0;
    __shared__ __attribute__((aligned(1024))) LdsStage<BM, BN> st1;
    __shared__ __attribute__((aligned(1024))) LdsStage<BM, BN> st2;
    __shared__ __attribute__((aligned(1024))) LdsStage<(S > 3 ? BM : 8), (S > 3 ? BN : 8)> st3;

    const int w = xcd_remap(blockIdx.x, gridDim.x);
    const int mt = w % m_tiles;
    const int rest = w / m_tiles;
    const int nt = rest % n_tiles;
    const int split = rest / n_tiles;
    const int m0 = mt * BM;
    const int k_begin = split * kps;
    const int k_end = min(K, k_begin + kps);
    const int n_k = (k_end - k_begin) / kBK;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave / WGN, wc = wave % WGN;
    const int a_bytes = (int)((size_t)M * K * 2), w_bytes = (int)((size_t)N * K * 2);

    // lane l of load instruction j fills LDS chunk l % 8 of row l / 8 of its 8-row group:
    // it loads the logical chunk that the swizzle puts there
    constexpr uint32_t kOut = 0x80000000u;
    uint32_t a_off[AI], b_off[BI];
#pragma unroll
    for (int j = 0; j < AI; ++j) {
        const int row = (wave * AI + j) * 8 + (lane >> 3);
        const int m = m0 + row;
        a_off[j] = m < M ? (uint32_t)(((size_t)m * K + k_begin + lds_swizzle(row, lane & 7) * 8) * 2) : kOut;
    }
#pragma unroll
    for (int j = 0; j < BI; ++j) {
        const int row = (wave * BI + j) * 8 + (lane >> 3);
        const int n = nt * BN + row;
        b_off[j] = n < N ? (uint32_t)(((size_t)n * K + k_begin + lds_swizzle(row, lane & 7) * 8) * 2) : kOut;
    }

    [[maybe_unused]] __shared__ int row_page[EPI == EPI_QKV_ROPE ? BM : 1], row_key[EPI == EPI_QKV_ROPE ? BM : 1];
    [[maybe_unused]] QkvPre<BM, BN, NT> pre;
    if constexpr (EPI == EPI_QKV_ROPE) qkv_prefetch<BM, BN, NT>(qa, M, N, m0, nt, tid, row_page, row_key, pre);

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int frow = lane & 31, fhalf = lane >> 5;
    auto compute = [&](const LdsStage<BM, BN>& sg) {
#pragma unroll
        for (int ks = 0; ks < kBK / 16; ++ks) {
            bf16x8_t af[TM], bfr[TN];
            const int c = ks * 2 + fhalf;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wr * WM + i * 32 + frow;
                af[i] = *reinterpret_cast<const bf16x8_t*>(&sg.a[row * kBK + (lds_swizzle(row, c) << 3)]);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int row = wc * WN + j * 32 + frow;
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(&sg.b[row * kBK + (lds_swizzle(row, c) << 3)]);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    };
    auto stage = [&](int i) -> LdsStage<BM, BN>& {
        if (i == 0) return st0;
        if (i == 1) return st1;
        if constexpr (S > 3) {
            if (i == 3) return st3;
        }
        return st2;
    };
    auto step_bytes = [&](int k) { return k < n_k ? (uint32_t)k * kBK * 2 : 0x80000000u; };
#pragma unroll
    for (int p = 0; p < S - 1; ++p)
        lds_dma_stage<AI, BI>(stage(p), A, a_bytes, W, w_bytes, a_off, b_off, step_bytes(p), wave, WPOL);
    // one k-step from stage ST (the stage index is a constant in every expansion)
#define DASH_LDS_STEP(ST, KK)                                                                               \
    do {                                                                                                   \
        const int k_ = (KK);                                                                               \
        wait_vmcnt_lds_reads<(S - 2) * DPS>();                                                             \
        __builtin_amdgcn_s_barrier();                                                                      \
        lds_dma_stage<AI, BI>(stage(((ST) + S - 1) % S), A, a_bytes, W, w_bytes, a_off, b_off,              \
                              step_bytes(k_ + S - 1), wave, WPOL);                                         \
        compute(stage(ST));                                                                                \
    } while (0)
    int k = 0;
    for (; k + S <= n_k; k += S) {
        DASH_LDS_STEP(0, k);
        DASH_LDS_STEP(1, k + 1);
        DASH_LDS_STEP(2, k + 2);
        if constexpr (S > 3) DASH_LDS_STEP(3, k + 3);
    }
    if (k < n_k) DASH_LDS_STEP(0, k++);
    if (k < n_k) DASH_LDS_STEP(1, k++);
    if constexpr (S > 3) {
        if (k < n_k) DASH_LDS_STEP(2, k++);
    }
#undef DASH_LDS_STEP

    if constexpr (EPI == EPI_QKV_ROPE) {
        // the fp32 tile is staged in LDS of its own (a stage is too small for it)
        __shared__ __attribute__((aligned(16))) float cstage[BM * (BN + 4)];
        wait_vmcnt<0>();  // the out-of-range loads of the steps past the end still write their stage
        qkv_epilogue<BM, BN, WGM, WGN>(&acc[0][0], cstage, qa, M, N, m0, nt, tid, wr, wc, row_page, row_key, pre);
    } else {
        store_f32_epilogue<BM, BN, WGM, WGN>(&acc[0][0], reinterpret_cast<float*>(C) + split * split_stride, M, N, ldc,
                                             m0, nt, lane, wr, wc);
        wait_vmcnt<0>();  // the out-of-range loads of the steps past the end still write their stage
    }
}

template <int BM, int BN, int WGM, int WGN, int S, int EPI, int WPOL = 0>
hipError_t run_lds(const void* A, const void* W, void* C, int M, int N, int K, int ldc, int nsplit,
                   size_t split_stride, hipStream_t st, const QkvRopeArgs& qa = QkvRopeArgs{}) {
    const int m_tiles = (M + BM - 1) / BM;
    const int n_tiles = (N + BN - 1) / BN;
    int kps = K;
    if (nsplit > 1) {
        kps = (K + nsplit - 1) / nsplit;
        kps = (kps + kBK - 1) / kBK * kBK;
    }
    if ((K + kps - 1) / kps != nsplit) return hipErrorInvalidValue;
    if (K % kBK || (size_t)M * K * 2 >= (1u << 31) || (size_t)N * K * 2 >= (1u << 31)) return hipErrorInvalidValue;
    gemm_lds_k<BM, BN, WGM, WGN, S, EPI, WPOL><<<m_tiles * n_tiles * nsplit, 64 * WGM * WGN, 0, st>>>(
        (const bf16_t*)A, (const bf16_t*)W, C, M, N, K, ldc, m_tiles, n_tiles, kps, split_stride, qa);
    return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int PD, int EPI, int WPOL = 0>
hipError_t run_bf16(const void* A, const void* W, void* C, int M, int N, int K, int ldc, int nsplit,
                     size_t split_stride, hipStream_t st, const QkvRopeArgs& qa = QkvRopeArgs{}) {
    const int m_tiles = (M + BM - 1) / BM;
    const int cols = EPI == EPI_SWIGLU ? N / 2 : N;
    const int tn = EPI == EPI_SWIGLU ? BN / 2 : BN;
    const int n_tiles = (cols + tn - 1) / tn;
    int kps = K;
    if (nsplit > 1) {
        kps = (K + nsplit - 1) / nsplit;
        kps = (kps + kBK - 1) / kBK * kBK;
    }
    if ((K + kps - 1) / kps != nsplit) return hipErrorInvalidValue;
    // k-steps of 64 never straddle the end of K or of a split; byte offsets fit 31 bits
    if (K % kBK || (size_t)M * K * 2 >= (1u << 31) || (size_t)N * K * 2 >= (1u << 31)) return hipErrorInvalidValue;
    const int blocks = m_tiles * n_tiles * nsplit;
    gemm_bf16_k<BM, BN, WGM, WGN, PD, EPI, WPOL><<<blocks, 64 * WGM * WGN, 0, st>>>(
        (const bf16_t*)A, (const bf16_t*)W, C, M, N, K, ldc, m_tiles, n_tiles, 0, kps, split_stride, qa);
    return hipGetLastError();
}

// Gate/up with the SwiGLU epilogue over output columns [col0, col1) of h only (col0 a
// multiple of the tile's BN / 2 output columns): the same tiles, hence the same bits, as
// the launch over every column.
template <int BM, int BN, int WGM, int WGN, int PD>
hipError_t run_bf16_swiglu_cols(const void* A, const void* W, void* C, int M, int N, int K, int ldc, int col0,
                                int col1, hipStream_t st) {
    constexpr int tn = BN / 2;
    if (col0 % tn || col0 < 0 || col1 <= col0 || col1 > N / 2) return hipErrorInvalidValue;
    if (K % kBK || (size_t)M * K * 2 >= (1u << 31) || (size_t)N * K * 2 >= (1u << 31)) return hipErrorInvalidValue;
    const int m_tiles = (M + BM - 1) / BM;
    const int n_tiles = (col1 - col0 + tn - 1) / tn;
    gemm_bf16_k<BM, BN, WGM, WGN, PD, EPI_SWIGLU><<<m_tiles * n_tiles, 64 * WGM * WGN, 0, st>>>(
        (const bf16_t*)A, (const bf16_t*)W, C, M, N, K, ldc, m_tiles, n_tiles, col0 / tn, K, 0, QkvRopeArgs{});
    return hipGetLastError();
}

// fp32: 64 x 64 output tile per 256 threads (16 x 16, 4 x 4 each), BK = 16.
template <int EPI>
__global__ void __launch_bounds__(256) gemm_f32_k(const float* __restrict__ A, const float* __restrict__ W,
                                                  void* __restrict__ C, int M, int N, int K, int ldc) {
    __shared__ float As[16][65];
    __shared__ float Bs[16][65];
    __shared__ float Cs[EPI == EPI_SWIGLU ? 64 : 1][65];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int m0 = blockIdx.y * 64;
    const int ff = N >> 1;
    // B tile rows: STORE: n0 + r;  SWIGLU: r < 32 gate j0 + r, r >= 32 up ff + j0 + r - 32.
    auto wrow = [&](int r, bool& ok) {
        if (EPI == EPI_SWIGLU) {
            const int j = blockIdx.x * 32 + (r & 31);
            ok = j < ff;
            return r < 32 ? j : ff + j;
        }
        const int n = blockIdx.x * 64 + r;
        ok = n < N;
        return n;
    };
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
        for (int e = threadIdx.x; e < 64 * 16; e += 256) {
            const int r = e >> 4, k = e & 15;
            const int m = m0 + r;
            As[k][r] = (m < M && k0 + k < K) ? A[(size_t)m * K + k0 + k] : 0.f;
            bool ok;
            const int n = wrow(r, ok);
            Bs[k][r] = (ok && k0 + k < K) ? W[(size_t)n * K + k0 + k] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] += As[k][ty * 4 + i] * Bs[k][tx * 4 + j];
        __syncthreads();
    }
    if (EPI == EPI_STORE_F32) {
        float* Cp = reinterpret_cast<float*>(C);
        for (int i = 0; i < 4; ++i)
            for (int j = 0; j < 4; ++j) {
                const int m = m0 + ty * 4 + i, n = blockIdx.x * 64 + tx * 4 + j;
                if (m < M && n < N) Cp[(size_t)m * ldc + n] = acc[i][j];
            }
    } else {
        for (int i = 0; i < 4; ++i)
            for (int j = 0; j < 4; ++j) Cs[ty * 4 + i][tx * 4 + j] = acc[i][j];
        __syncthreads();
        float* H = reinterpret_cast<float*>(C);
        for (int e = threadIdx.x; e < 64 * 32; e += 256) {
            const int r = e >> 5, c = e & 31;
            const int m = m0 + r, col = blockIdx.x * 32 + c;
            if (m < M && col < ff) H[(size_t)m * ldc + col] = silu(Cs[r][c]) * Cs[r][c + 32];
        }
    }
}

}  // namespace

// Split-K count as a function of the weight shape only (never of M), so that a
// row's result does not depend on how many other rows share the launch: the
// whole path is batch-invariant, bit for bit.  Only long reductions are split
// (the down projection, K = d_ff): with 128 x 256 tiles, one workgroup per CU,
// a decode batch of ~1k rows then gives close to one tile per CU (1.5B:
// 8 x 6 tiles x 5 splits = 240 of 256 CUs).  Short reductions (QKV, O, K = d)
// run unsplit on small tiles instead, which was measured faster than split-K
// plus the partial sums it leaves for the consumer to read.
int gemm_pick_splits(int dtype, int epi, int N, int K) {
    if (dtype != 1 || epi != EPI_STORE_F32 || K < 4096) return 1;
    const int nt = (N + 255) / 256;
    int s = std::max(1, (32 + nt / 2) / nt);  // ~32 tile-splits per 128-row block of the batch
    s = std::min(s, std::min(8, K / 512));
    int kps = (K + s - 1) / s;
    kps = (kps + kBK - 1) / kBK * kBK;
    return (K + kps - 1) / kps;
}

bool gemm_qkv_fusable(int dtype, int n_heads, int n_kv, int head_dim) {
    return dtype == 1 && (head_dim == 64 || head_dim == 128) && (n_heads * head_dim) % 128 == 0 &&
           (n_kv * head_dim) % 128 == 0;
}

bool gemm_qkv_fuse_pays(int M, int N) { return (long)((M + 63) / 64) * (N / 128) >= 128; }

hipError_t launch_gemm_qkv_rope(const void* A, const void* W, int M, int N, int K, const QkvRopeArgs& qa,
                                hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (!gemm_qkv_fusable(1, qa.n_heads, qa.g.n_kv, qa.g.head_dim) ||
        N != (qa.n_heads + 2 * qa.g.n_kv) * qa.g.head_dim)
        return hipErrorInvalidValue;
    return run_bf16<64, 128, 2, 4, 2, EPI_QKV_ROPE>(A, W, nullptr, M, N, K, 0, 1, 0, st, qa);
}

// Cache policy of the weight loads where the batch fits one 64-row block: every
// weight byte is then read by exactly one work-group, so the loads stream past the
// caches (the same non-temporal policy as the decode attention's private K/V loads).
constexpr int kWeightStream = 2;

hipError_t launch_gemm(int dtype, int epi, const void* A, const void* W, void* C, int M, int N, int K, int ldc,
                       int nsplit, size_t split_stride, hipStream_t st) {
    if (M <= 0 || N <= 0) return hipSuccess;
    if (dtype == 1) {
        // Tile choice may depend on M: every configuration accumulates each output
        // element with the same chain of 32x32x16 MFMAs over k, so results do not.
        // Small batches stream the weights: narrow tiles give enough workgroups
        // (>= 256) to pull them from HBM at full rate.
        if (epi == EPI_SWIGLU) {
            if (nsplit != 1) return hipErrorInvalidValue;
            if (M > 384) {
                const int ff = N / 2;
                const long mb = (M + 255) / 256;
                const long t256_all = mb * ((ff + 127) / 128);
                const long split_tiles = t256_all / 256 * 256 / mb;  // column tiles of the whole rounds
                if (t256_all > 256 && t256_all < 4 * 256 && t256_all % 256 && t256_all % 256 < 128 &&
                    split_tiles >= 1) {
                    // Whole rounds of 256x256 tiles leave a last round under half full: those
                    // rounds run as one launch over the columns they cover, the remaining
                    // columns as a second launch on the largest of 128x256, 128x128 and 64x128
                    // tiles that still gives it 128 or more work-groups (else 64x128).  Measured
                    // with dash_gemm_bench at 1024 and 2048 rows: 1.5B 70.9 -> 63.0 us and
                    // 132.1 -> 114.5 us, 3B at 1024 rows 108.7 -> 96.9 us, 0.5B at 2048 rows
                    // 44.9 -> 43.0 us (a last round at least half full runs whole, as below).
                    const int c_split = (int)split_tiles * 128;
                    hipError_t e = run_bf16_swiglu_cols<256, 256, 4, 4, 2>(A, W, C, M, N, K, ldc, 0, c_split, st);
                    if (e != hipSuccess) return e;
                    const long rc = ff - c_split, m128 = (M + 127) / 128;
                    if (m128 * ((rc + 127) / 128) >= 128)
                        return run_bf16_swiglu_cols<128, 256, 4, 4, 2>(A, W, C, M, N, K, ldc, c_split, ff, st);
                    if (m128 * ((rc + 63) / 64) >= 128)
                        return run_bf16_swiglu_cols<128, 128, 4, 2, 2>(A, W, C, M, N, K, ldc, c_split, ff, st);
                    return run_bf16_swiglu_cols<64, 128, 2, 2, 2>(A, W, C, M, N, K, ldc, c_split, ff, st);
                }
                // Past 384 rows the tile is chosen by how its work-groups fill the 256 CUs
                // (one 256x256 or 128x256 work-group per CU, two 128x128 ones): 256x256 where
                // they fill one round (128-256 tiles), or leave a last round at least half
                // full, or run four rounds or more; else 128x256 under the same test; else
                // 128x128.  Measured with dash_gemm_bench on the 0.5B, 1.5B and 3B shapes at
                // 512-2048 rows (weights cold, interleaved rounds): each choice the fastest
                // tiling or within 2% of it (256x256: 1.5B 7% / 19% faster than 128x128 at
                // 512 / 768 rows, 3B 13% at 2048; 128x128: 0.5B 20% faster than 256x256 at
                // 2048 rows); 256x256 also measured 15-19% faster at 4096-16384 rows.
                const long cols = (N / 2 + 127) / 128;
                const long t256 = (M + 255) / 256 * cols, t128 = (M + 127) / 128 * cols;
                if ((t256 >= 128 && t256 <= 256) || t256 % 256 >= 128 || t256 >= 4 * 256)
                    return run_bf16<256, 256, 4, 4, 2, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
                if (t128 <= 256 || t128 % 256 >= 128)
                    return run_bf16<128, 256, 4, 4, 2, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
                return run_bf16<128, 128, 4, 2, 2, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
            }
            if (M > 256) return run_bf16<128, 128, 4, 2, 2, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
            // Small batches: 64 column pairs per tile read the batch rows half as often as
            // 32; worth it where that still leaves >= 128 work-groups per 64-row block
            // (d_ff >= 8192).  Measured on the 1.5B and 3B shapes: 9-11% faster up to 64
            // rows (three k-steps in flight), 5-16% at 129-256 rows, 3-5% slower at 65-128.
            if ((N / 2 + 63) / 64 >= 128) {
                if (M <= 64)
                    return run_bf16<64, 128, 2, 2, 3, EPI_SWIGLU, kWeightStream>(A, W, C, M, N, K, ldc, 1, 0, st);
                if (M > 128) return run_bf16<64, 128, 2, 2, 2, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
            }
            if (M <= 64) return run_bf16<64, 64, 2, 1, 2, EPI_SWIGLU, kWeightStream>(A, W, C, M, N, K, ldc, 1, 0, st);
            return run_bf16<64, 64, 2, 1, 2, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
        }
        if (N >= 8192) {  // LM head: many tiles, the largest tile that the batch fills wins
            if (M <= 64)
                return run_bf16<64, 256, 1, 4, 2, EPI_STORE_F32, kWeightStream>(A, W, C, M, N, K, ldc, nsplit,
                                                                               split_stride, st);
            if (M <= 128)  // measured 10-18% faster than 256x256 at 96-128 rows
                return run_bf16<128, 256, 4, 4, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            return run_bf16<256, 256, 4, 4, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        }
        if (K < 4096 && M >= 256 && M <= 4096) {
            // Unsplit short reductions (the output projection; QKV where it is not fused):
            // the direct-to-LDS kernel, on the largest tile that still gives the launch
            // about 160 or more work-groups.  Measured on the 0.5B, 1.5B and 3B shapes at
            // 256-2048 rows (dash_gemm_bench, weights cold): 7-36% faster than the
            // register-staged tiles (1.5B at 1024 rows: 14.8 -> 10.5 us).
            // 64x64 tiles while they fit one round (<= 256 work-groups): 15-17% faster than
            // 128x64 for the 0.5B shape at 768-1024 rows
            if ((long)((M + 63) / 64) * ((N + 63) / 64) <= 256)
                return run_lds<64, 64, 2, 2, 4, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            if (M <= 1024 || (long)(M / 128) * ((N + 127) / 128) < 160)
                return run_lds<128, 64, 2, 2, 4, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            return run_lds<128, 128, 2, 2, 4, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        }
        if (M <= 256 && (K < 4096 || M <= 64)) {
            // Few work-groups stream the weights here; four k-steps in flight per thread
            // instead of two pull them faster while the launch is small (unsplit K, or one
            // 64-row block): measured 22-28% faster on the 1.5B and 3B QKV / O shapes up to
            // 256 rows and on the split down projection up to 64 rows.
            if (M <= 64)
                return run_bf16<64, 32, 2, 1, 4, EPI_STORE_F32, kWeightStream>(A, W, C, M, N, K, ldc, nsplit,
                                                                              split_stride, st);
            return run_bf16<64, 32, 2, 1, 4, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        }
        // Larger batches: the largest tile that still gives the launch enough work-groups.
        // Measured crossovers on the 0.5B, 1.5B and 3B shapes: the split down projection
        // 64x64 three k-steps ahead up to 128 rows and two up to 384 (12-19% faster than
        // 64x32 there), the direct-to-LDS 128x128 tiles up to 640, 128x256 up to 1024,
        // 256x256 past that (12-18% faster from 1536 rows); QKV / O 64x64 three k-steps ahead up to 512 rows (10-15% faster than two),
        // 64x64 up to 1024, 128x128 up to 4096 (4-30% faster from 1536), 256x256 past that
        // (15-26% faster at 8192-16384).
        if (K >= 4096) {
            if (M <= 128)
                return run_bf16<64, 64, 2, 2, 3, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            if (M <= 384)
                return run_bf16<64, 64, 2, 2, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            if (M <= 640)  // direct-to-LDS 128x128: 23-35% faster at 512 rows on all three shapes
                return run_lds<128, 128, 2, 2, 4, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            if (M <= 1024)
                return run_bf16<128, 256, 4, 4, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
            return run_bf16<256, 256, 4, 4, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        }
        if (M <= 512)
            return run_bf16<64, 64, 2, 2, 3, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        if (M <= 1024)  // decode QKV / O: unsplit, small tiles fill the GPU
            return run_bf16<64, 64, 2, 2, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        if (M <= 4096)
            return run_bf16<128, 128, 4, 2, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
        return run_bf16<256, 256, 4, 4, 2, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
    }
    if (nsplit != 1) return hipErrorInvalidValue;
    if (epi == EPI_SWIGLU) {
        dim3 grid((N / 2 + 31) / 32, (M + 63) / 64);
        gemm_f32_k<EPI_SWIGLU><<<grid, 256, 0, st>>>((const float*)A, (const float*)W, C, M, N, K, ldc);
    } else {
        dim3 grid((N + 63) / 64, (M + 63) / 64);
        gemm_f32_k<EPI_STORE_F32><<<grid, 256, 0, st>>>((const float*)A, (const float*)W, C, M, N, K, ldc);
    }
    return hipGetLastError();
}

}  // namespace dash
