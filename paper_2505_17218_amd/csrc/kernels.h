// Host-side launchers of the HIP kernels.  All launch on `st` and return the
// hipError_t of the launch.  Shapes are validated by the caller (runtime.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace dash {

// ---- elementwise (elementwise.hip) ----
// x[r] = E[tok[r]] (fp32); y[r] = RMSNorm(x[r]) * w in the model dtype.  A token id
// outside [0, vocab) is never used as an index: its rows of x and y become NaN and
// bit 2 of *status (nullable) is set.
hipError_t launch_embed_rmsnorm(int dtype, const int32_t* tok, const void* E, const void* w, float* x, void* y,
                                int rows, int d, int vocab, float eps, uint32_t* status, hipStream_t st);
// For output row i, r = row_map ? row_map[i] : i: v = x[r] + sum_s delta[s*split_stride + r*d];
// if write_x, x[r] = v; y[i] = RMSNorm(v) * w.
hipError_t launch_add_rmsnorm(int dtype, float* x, const float* delta, int nsplit, size_t split_stride,
                              const void* w, void* y, const int32_t* row_map, int rows, int d, float eps,
                              int write_x, hipStream_t st);
// cos/sin table [rows][head_dim/2][2] of pos[r] * theta^(-2i/head_dim), evaluated in float64.
hipError_t launch_rope_table(const int32_t* pos, float* cs, int rows, int head_dim, float theta, hipStream_t st);
// qkv (sum of nsplit fp32 partials) + bias; RoPE on q and k; q -> q_out (model dtype,
// [rows][Hq][hd]); k, v -> KV pages of (slot[r], pos[r]) at `layer`.
hipError_t launch_qkv_rope_append(int dtype, const float* qkv, int nsplit, size_t split_stride, const void* bias,
                                  const float* cs, const int32_t* pos, const int32_t* slot,
                                  const int32_t* page_table, void* pool, const KVGeom& g, int layer,
                                  void* q_out, int rows, int n_heads, uint32_t* status, hipStream_t st);
// Copy every layer of `src_page` to `dst_pages[i]` (i < n).
hipError_t launch_copy_pages(int dtype, void* pool, const KVGeom& g, const int32_t* pairs, int n,
                             hipStream_t st);
// Rollout row state helpers.
hipError_t launch_rows_init(int32_t* slot, int32_t* uid, int32_t* pos, int32_t* step, int n, int pos0, int step0,
                            hipStream_t st);
hipError_t launch_rows_advance(int32_t* pos, int32_t* step, int n, hipStream_t st);
hipError_t launch_fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t st);
hipError_t launch_iota_div(int32_t* p, int n, int div, hipStream_t st);  // p[i] = i / div

// ---- GEMM (gemm.hip) ----
enum { EPI_STORE_F32 = 0, EPI_SWIGLU = 1, EPI_QKV_ROPE = 2 };
// Arguments of the fused QKV epilogue (bf16 models): q/k/v bias, RoPE of q and k
// (cos/sin table cs [rows][hd/2][2]), q written to q_out [rows][n_heads][hd], k and
// v appended to the cache at pos[row] of slot[row] (status bit 0 for unbacked).
struct QkvRopeArgs {
    const bf16_t* bias;
    const float* cs;
    const int32_t* pos;
    const int32_t* slot;
    const int32_t* page_table;
    bf16_t* pool;
    KVGeom g;
    int layer;
    bf16_t* q_out;
    int n_heads;
    uint32_t* status;
};
// C = A[M,K] . W[N,K]^T with fp32 accumulation.
//   EPI_STORE_F32: C fp32 (row stride ldc) ; split-K into nsplit partials at C + s*split_stride.
//   EPI_SWIGLU:    W rows [0, N/2) are gate, [N/2, N) up; writes h[M, N/2] (model dtype, row stride ldc)
//                  = silu(gate) * up.  nsplit must be 1.
hipError_t launch_gemm(int dtype, int epi, const void* A, const void* W, void* C, int M, int N, int K, int ldc,
                       int nsplit, size_t split_stride, hipStream_t st);
// Split-K count for a weight of N x K (independent of M: results are batch-invariant).
int gemm_pick_splits(int dtype, int epi, int N, int K);
// QKV projection with bias, RoPE and the KV append in the epilogue: the same values
// as launch_gemm(EPI_STORE_F32, nsplit 1) followed by launch_qkv_rope_append, bit for
// bit.  Available for bf16 models whose q and kv column ranges are multiples of 128
// (a 128-column tile then holds whole heads); gemm_qkv_fusable says so.
bool gemm_qkv_fusable(int dtype, int n_heads, int n_kv, int head_dim);
// The fused kernel's 128-column tiles leave few work-groups for small batches; it
// pays when it has at least half a work-group per CU (the unfused GEMM plus RoPE /
// append kernel gives the same bits, so the choice may depend on the row count).
bool gemm_qkv_fuse_pays(int M, int N);
hipError_t launch_gemm_qkv_rope(const void* A, const void* W, int M, int N, int K, const QkvRopeArgs& qa,
                                hipStream_t st);

// ---- attention (attention.hip) ----
// Decode attention over the paged cache for rows with 1 query each.  bf16: MFMA
// kernel; a row's context is cut into splits of g.split_keys keys (depending on
// its own length and the cache only, so results are batch-invariant) merged by a
// second kernel; partials live in ws_part (attention_partial_floats).  fp32:
// generic kernel.  q [rows][Hq][hd]; o [rows][Hq*hd].
// 128 rather than 256: measured 10% less attention time for 64 sequences of the 3B
// shape (contexts 513-1536), the merge cost unchanged.
constexpr int kAttnMinSplitKeys = 128;
constexpr int kAttnTargetWaves = 2048;  // 2 waves per SIMD over 256 CUs (hd 128; 3 per SIMD for hd 64)
// Split length for a cache: the largest power of two >= kAttnMinSplitKeys whose
// split count still gives max_seqs * n_kv * splits >= kAttnTargetWaves at max_ctx
// (and no longer than max_ctx needs).  Long splits mean fewer partials to write and
// merge; short ones give small batches enough waves.
int attention_split_keys(int max_seqs, int n_kv, int max_ctx, int head_dim);
hipError_t launch_decode_attention(int dtype, const void* q, const int32_t* pos, const int32_t* slot,
                                   const int32_t* page_table, const void* pool, const KVGeom& g, int layer,
                                   int n_heads, void* o, int rows, int max_ctx, float* ws_part, hipStream_t st);
// Partial-result floats for any cache of this max_ctx (sized for the shortest split).
size_t attention_partial_floats(int rows, int n_heads, int head_dim, int max_ctx);
// Decode attention for batches made of groups of rows that share a prefix: rows
// [group_off[i], group_off[i+1]) (at most group_size of them) share their first
// shared_len positions (the same pages, read from the group's first row).  A first
// kernel runs the shared pages (those inside the first context split) once per group
// and kv head, leaving each row's online-softmax state in ws_state
// (decode_attention_prefix_state_bytes), and the per-row kernel continues from it.
// Same results as launch_decode_attention, bit for bit; bf16 only.  hipErrorInvalidValue
// unless decode_attention_prefix_ok holds and ws_state is set.
bool decode_attention_prefix_ok(const KVGeom& g, int n_heads, int group_size, int shared_len);
size_t decode_attention_prefix_state_bytes(int rows, int n_heads, int head_dim);
hipError_t launch_decode_attention_grouped(const void* q, const int32_t* pos, const int32_t* slot,
                                           const int32_t* page_table, const void* pool, const KVGeom& g, int layer,
                                           int n_heads, const int32_t* group_off, int n_groups, int group_size,
                                           int shared_len, void* o, int rows, int max_ctx, float* ws_part,
                                           float* ws_state, hipStream_t st);
// Second pass of decode attention: merge the splits of rows longer than one split (bf16 only).
hipError_t launch_attention_combine(int dtype, const int32_t* pos, int rows, int n_heads, int head_dim,
                                    int max_ctx, int split_keys, const float* ws_part, void* o, hipStream_t st);
// Causal attention of prefill rows: rows are whole prompts of prompt_len positions, row
// r = prompt * prompt_len + position, all rows of a prompt in slot[prompt * prompt_len].
// bf16: MFMA kernel; fp32: generic kernel (row r attends to 0..pos[r] of slot[r]).
hipError_t launch_prefill_attention(int dtype, const void* q, const int32_t* pos, const int32_t* slot,
                                    const int32_t* page_table, const void* pool, const KVGeom& g, int layer,
                                    int n_heads, void* o, int rows, int prompt_len, hipStream_t st);

// Exhaustive check of f2bf against integer rounding of the bit pattern (synchronous, on
// the null stream): the number of float32 inputs on which they differ.
hipError_t bf16_round_check(unsigned long long* mismatches);

// ---- sampling / advantage (sampler.hip, advantage.hip) ----
// Screening tolerance of the sampler, and an exhaustive check of it (synchronous, on
// the null stream): the largest |cheap noise - exact noise| over all noise values.
float sampler_screen_tol();
hipError_t sampler_screen_check(float* max_err);
// Row b samples logits row row_of ? row_of[b] : b.  Optional outputs: lp_out [rows]
// (log-prob of the drawn token), row_ml [rows][2] (max of l/T and the log of the
// normaliser), traj / traj_lp (the token and log-prob also stored at
// [uid][step] with row stride traj_ld).  A row without a finite logit draws -1
// and sets bit 1 of *status (nullable).
hipError_t launch_sample(const float* logits, int64_t ld, int rows, int vocab, const int32_t* row_of,
                         const int32_t* uid, const int32_t* step, float temperature, uint64_t seed,
                         int32_t* tok_out, float* lp_out, float* row_ml, uint32_t* status, int32_t* traj,
                         float* traj_lp, int traj_ld, hipStream_t st);
// lp_out[b] = log softmax(logits row b)[y_b] with y_b = tokens[(b / per) * stride + off + b % per]
// (rows grouped per sequence: `per` scored positions of a sequence whose tokens
// start every `stride` entries, the first scored token at `off`); NaN for a token
// outside [0, vocab); non-finite logits are left out of the normaliser.
hipError_t launch_logprob_gather(const float* logits, int64_t ld, int rows, int vocab, const int32_t* tokens, int per,
                                 int stride, int off, float* lp_out, hipStream_t st);
// Per row pair: D_KL(softmax(base) || softmax(theta)) into kl and the reverse
// direction into kl_rev (may be null); -inf logits have probability zero.
hipError_t launch_logits_kl(const float* theta, const float* base, int64_t ld, int rows, int vocab, float* kl,
                            float* kl_rev, hipStream_t st);
// *loss = -(1/n_total) sum over kept samples n of A[n] * sum_{t < len[n]} lp[n][t] (float64);
// seq_lp[n] (nullable) receives each kept sample's sequence log-prob.
hipError_t launch_pg_loss(const float* lp, int64_t ld, int T, const int32_t* len, const float* adv,
                          const int32_t* kept, const int32_t* kept_count, int n_total, double* loss, double* seq_lp,
                          hipStream_t st);
// The general form: surrogate A S, or PPO's clipped min(rho A, clip(rho, 1 +- eps) A)
// with rho = exp(S - S_old) when lp_old is given; plus (beta / n_total) times the
// kept KL sums when kl is given.  lp, lp_old and kl share the row stride ld.
// stats[4 n ..] (nullable) = (S, S_old, KL sum, d loss / d S) of each kept n.
hipError_t launch_policy_loss(const float* lp, const float* lp_old, const float* kl, int64_t ld, int T,
                              const int32_t* len, const float* adv, const int32_t* kept, const int32_t* kept_count,
                              int n_total, double clip_eps, double beta, double* loss, double* seq_lp, double* stats,
                              hipStream_t st);
hipError_t launch_group_advantage_filter(const float* r, int n_groups, int group, int mode, float eps, float tau,
                                         float* adv, int32_t* kept, int32_t* count, hipStream_t st);
hipError_t launch_live_compact(const int32_t* tok, const int32_t* slot, const int32_t* pos, const int32_t* step,
                               const int32_t* uid, const int32_t* budget, int eos_id, int n, int32_t* tok_o,
                               int32_t* slot_o, int32_t* pos_o, int32_t* step_o, int32_t* uid_o, int32_t* count,
                               hipStream_t st);

}  // namespace dash
