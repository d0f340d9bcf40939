// Projection GEMMs C = A[M,K] . W[N,K]^T (fp32 accumulation).
//
// bfloat16: MFMA v_mfma_f32_16x16x32_bf16 tiles.  A workgroup of 4 waves owns a
// BM x BN output tile (2 x 2 waves, each (BM/2) x (BN/2)); K advances in steps
// of 64 through a double-buffered LDS tile (rows padded to 72 elements so the
// 16-byte fragment reads of 16 consecutive rows hit distinct banks).  While
// one k-step is multiplied, the next one is already in flight from HBM into
// registers.  Work items (split, m-tile, n-tile) are enumerated m-fastest and
// dealt to XCDs in contiguous runs, so the blocks that share a weight tile run
// on the same XCD and reuse it from that XCD's L2.
//
// float32: a plain LDS-tiled VALU kernel (the fp32 shapes are tiny correctness
// configurations; there is no fp32 MFMA rate worth chasing there).
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
constexpr int kThreads = 256;
constexpr int kXcds = 8;

DASH_DEV float silu(float g) { return g / (1.0f + __expf(-g)); }

// Block id -> work index so that each XCD (block ids congruent mod 8) gets one
// contiguous run of work items.
DASH_DEV int xcd_remap(int bid, int nb) {
    const int x = bid % kXcds, j = bid / kXcds;
    const int q = nb / kXcds, r = nb % kXcds;
    return x * q + (x < r ? x : r) + j;
}

template <int BM, int BN, int EPI>
__global__ void __launch_bounds__(kThreads) gemm_bf16_k(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W,
                                                        void* __restrict__ C, int M, int N, int K, int ldc,
                                                        int m_tiles, int n_tiles, int kps, size_t split_stride) {
    constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
    constexpr int A_CH = BM * 8 / kThreads, B_CH = BN * 8 / kThreads;  // 16-byte chunks per thread
    static_assert(A_CH >= 1 && B_CH >= 1, "tile too small");
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * kLdsStride];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * kLdsStride];

    const int w = xcd_remap(blockIdx.x, gridDim.x);
    const int mt = w % m_tiles;
    const int rest = w / m_tiles;
    const int nt = rest % n_tiles;
    const int split = rest / n_tiles;
    const int m0 = mt * BM;
    const int k_begin = split * kps;
    const int k_end = min(K, k_begin + kps);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;

    // Global row pointers of this thread's chunks.
    const bf16_t* a_ptr[A_CH];
    int a_lds[A_CH], a_kc[A_CH];
    bool a_ok[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
        const int idx = tid + i * kThreads, row = idx >> 3, kc = idx & 7;
        const int m = m0 + row;
        a_ok[i] = m < M;
        a_ptr[i] = A + (size_t)(a_ok[i] ? m : 0) * K + kc * 8;
        a_lds[i] = row * kLdsStride + kc * 8;
        a_kc[i] = kc * 8;
    }
    const bf16_t* b_ptr[B_CH];
    int b_lds[B_CH], b_kc[B_CH];
    bool b_ok[B_CH];
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
        const int idx = tid + i * kThreads, row = idx >> 3, kc = idx & 7;
        int n;
        bool ok;
        if (EPI == EPI_SWIGLU) {
            // tile row -> (wave column, gate/up half, offset); ff = N / 2 gate rows then ff up rows
            const int ff = N >> 1;
            const int wcol = row / (BN / 2), rr = row % (BN / 2);
            const int j = nt * (BN / 2) + wcol * (BN / 4) + (rr % (BN / 4));
            ok = j < ff;
            n = (rr < BN / 4) ? j : ff + j;
        } else {
            n = nt * BN + row;
            ok = n < N;
        }
        b_ok[i] = ok;
        b_ptr[i] = W + (size_t)(ok ? n : 0) * K + kc * 8;
        b_lds[i] = row * kLdsStride + kc * 8;
        b_kc[i] = kc * 8;
    }

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    uint4 ra[A_CH], rb[B_CH];
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            const bool ok = a_ok[i] && (k0 + a_kc[i] < k_end);
            ra[i] = ok ? *reinterpret_cast<const uint4*>(a_ptr[i] + k0) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) {
            const bool ok = b_ok[i] && (k0 + b_kc[i] < k_end);
            rb[i] = ok ? *reinterpret_cast<const uint4*>(b_ptr[i] + k0) : make_uint4(0, 0, 0, 0);
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) *reinterpret_cast<uint4*>(&As[buf][a_lds[i]]) = ra[i];
#pragma unroll
        for (int i = 0; i < B_CH; ++i) *reinterpret_cast<uint4*>(&Bs[buf][b_lds[i]]) = rb[i];
    };

    const int n_k = (k_end - k_begin + kBK - 1) / kBK;
    if (n_k > 0) {
        load(k_begin);
        store(0);
    }
    __syncthreads();
    const int frag_row = lane & 15, frag_k = (lane >> 4) * 8;
    for (int kt = 0; kt < n_k; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < n_k) load(k_begin + (kt + 1) * kBK);
#pragma unroll
        for (int ks = 0; ks < kBK; ks += 32) {
            bf16x8_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const bf16x8_t*>(
                    &As[buf][(wr * WM + i * 16 + frag_row) * kLdsStride + ks + frag_k]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(
                    &Bs[buf][(wc * WN + j * 16 + frag_row) * kLdsStride + ks + frag_k]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < n_k) store(buf ^ 1);
        __syncthreads();
    }

    // Output fragment: acc[i][j][r] = C[row (lane>>4)*4 + r][col lane&15] of the 16x16 block (i, j).
    const int out_r = (lane >> 4) * 4, out_c = lane & 15;
    if (EPI == EPI_STORE_F32) {
        float* Cp = reinterpret_cast<float*>(C) + split * split_stride;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = nt * BN + wc * WN + j * 16 + out_c;
                if (n >= N) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = m0 + wr * WM + i * 16 + out_r + r;
                    if (m < M) Cp[(size_t)m * ldc + n] = acc[i][j][r];
                }
            }
    } else {
        bf16_t* H = reinterpret_cast<bf16_t*>(C);
        const int ff = N >> 1;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN / 2; ++j) {
                const int col = nt * (BN / 2) + wc * (BN / 4) + j * 16 + out_c;
                if (col >= ff) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = m0 + wr * WM + i * 16 + out_r + r;
                    if (m < M) H[(size_t)m * ldc + col] = f2bf(silu(acc[i][j][r]) * acc[i][j + TN / 2][r]);
                }
            }
    }
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

template <int BM, int BN, int EPI>
hipError_t run_bf16(const void* A, const void* W, void* C, int M, int N, int K, int ldc, int nsplit,
                    size_t split_stride, hipStream_t st) {
    const int m_tiles = (M + BM - 1) / BM;
    const int n_cols = EPI == EPI_SWIGLU ? N / 2 : N;
    const int n_tiles = (n_cols + (EPI == EPI_SWIGLU ? BN / 2 : BN) - 1) / (EPI == EPI_SWIGLU ? BN / 2 : BN);
    int kps = K;
    if (nsplit > 1) {
        kps = (K + nsplit - 1) / nsplit;
        kps = (kps + kBK - 1) / kBK * kBK;
    }
    const int splits = (K + kps - 1) / kps;
    if (splits != nsplit) return hipErrorInvalidValue;
    const int blocks = m_tiles * n_tiles * splits;
    gemm_bf16_k<BM, BN, EPI><<<blocks, kThreads, 0, st>>>((const bf16_t*)A, (const bf16_t*)W, C, M, N, K, ldc,
                                                          m_tiles, n_tiles, kps, split_stride);
    return hipGetLastError();
}

}  // namespace

// Split-K count as a function of the weight shape only (never of M), so that a
// row's result does not depend on how many other rows share the launch: the
// whole path is batch-invariant, bit for bit.  Narrow outputs (few 128-column
// tiles) are split so that a decode batch of ~1k rows still gives ~400 work items.
int gemm_pick_splits(int dtype, int epi, int N, int K) {
    if (dtype != 1 || epi != EPI_STORE_F32) return 1;
    const int n_tiles = (N + 127) / 128;
    if (n_tiles >= 48 || K < 512) return 1;
    int s = (48 + n_tiles - 1) / n_tiles;
    s = std::min(s, std::min(8, K / 256));
    int kps = (K + s - 1) / s;
    kps = (kps + kBK - 1) / kBK * kBK;
    return (K + kps - 1) / kps;
}

hipError_t launch_gemm(int dtype, int epi, const void* A, const void* W, void* C, int M, int N, int K, int ldc,
                       int nsplit, size_t split_stride, hipStream_t st) {
    if (M <= 0 || N <= 0) return hipSuccess;
    if (dtype == 1) {
        if (epi == EPI_SWIGLU) {
            if (nsplit != 1) return hipErrorInvalidValue;
            return M <= 64 ? run_bf16<64, 128, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st)
                           : run_bf16<128, 128, EPI_SWIGLU>(A, W, C, M, N, K, ldc, 1, 0, st);
        }
        return M <= 64 ? run_bf16<64, 128, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st)
                       : run_bf16<128, 128, EPI_STORE_F32>(A, W, C, M, N, K, ldc, nsplit, split_stride, st);
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
