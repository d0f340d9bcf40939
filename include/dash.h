/*
 * dash.h — C ABI of the DASH rollout hot path on AMD MI355X (gfx950).
 *
 * DASH (arXiv 2505.17218) is GRPO with preemptive sampling and gradient
 * filtering.  The part of a DASH iteration that dominates its run time is the
 * rollout: one large batch of prompts, each duplicated into a group of G
 * samples (Sec. 3.4 and the preemptive-sampling figure), is decoded
 * autoregressively by the policy LM (Sec. 3, Eq. (1): trajectories are drawn
 * from pi_theta).  The rewards of the finished trajectories then give the GRPO
 * group advantage (Sec. 3.3, Eq. (4)), and samples whose advantage is small
 * are dropped before backpropagation (Sec. 3.5, gradient filtering).
 *
 * This library computes exactly that path on one GPU:
 *   dash_prefill                 prompt forward pass, KV cache write, group fork
 *   dash_decode_step             one autoregressive step over a batch of rows
 *   dash_sample                  temperature sampling (Gumbel-max, Philox noise)
 *   dash_group_advantage_filter  GRPO advantage and |A| >= tau compaction
 * plus the lifecycle, paged-KV bookkeeping and a native rollout driver that
 * chains them.
 *
 * Conventions
 *   - Every function returning int returns a dash_status.  Nothing aborts or
 *     throws across this boundary; dash_last_error() gives the text of the
 *     last failure on the calling thread.
 *   - Pointers named d_* are device memory owned by the caller; h_* are host
 *     memory owned by the caller.  The library never allocates device memory:
 *     weights, KV pool, page table and workspaces are caller buffers.  Its only
 *     device memory of its own is part of the loaded code: the 64 MiB workspace
 *     array of dash_decode_step_noalloc and the small result variables of the
 *     diagnostics dash_sampler_check and dash_bf16_round_check.  Handles
 *     (dash_model, dash_kv) are library-owned host objects; a dash_kv also owns a small
 *     pinned host staging ring for page-table uploads, and kernel timing
 *     (dash_profile_enable) creates HIP events.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     compute calls enqueue work on it and return without synchronising;
 *     device outputs are valid after the stream has been synchronised.
 *   - Argument errors are detected on the host before any launch and return
 *     DASH_EINVAL (bad value), DASH_ECAPACITY (page pool, page table or
 *     workspace too small) or DASH_ENOTSUP (a shape the kernels do not cover).
 *     DASH_EDEVICE reports a failed HIP call.
 *   - Handles are not thread-safe; use one per thread or serialise calls.
 */
#ifndef DASH_H
#define DASH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DASH_ABI_VERSION 2

typedef enum dash_status {
    DASH_OK = 0,
    DASH_EINVAL = 1,
    DASH_ENOMEM = 2,
    DASH_ECAPACITY = 3,
    DASH_EDEVICE = 4,
    DASH_ENOTSUP = 5
} dash_status;

/* Element type of weights, activations and the KV cache. */
enum { DASH_F32 = 0, DASH_BF16 = 1 };

/* Advantage normalisation (Sec. 3.3): Eq. (4) is the group-mean baseline;
 * the std-normalised variants divide by the group std (+ eps), population
 * (ddof 0) or Bessel-corrected (ddof 1). */
enum { DASH_ADV_MEAN_ONLY = 0, DASH_ADV_STD_POP = 1, DASH_ADV_STD_SAMPLE = 2, DASH_ADV_LOO = 3 };

/*
 * Decoder description.  The policy LM is a pre-norm decoder (the paper uses
 * Qwen2.5 base models, Sec. 4.1): x = E[tok]; per layer
 *   x += W_o . Attn(RoPE(W_q y + b_q), RoPE(W_k y + b_k), W_v y + b_v),  y = RMSNorm(x)
 *   x += W_down (silu(W_gate y) * (W_up y)),                           y = RMSNorm(x)
 * logits = RMSNorm(x) . E^T (embedding tied to the LM head).  Grouped-query
 * attention: query head h reads kv head h / (n_heads / n_kv_heads); scale
 * 1/sqrt(head_dim); rotate-half RoPE with frequencies theta^(-2i/head_dim).
 */
typedef struct dash_model_desc {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t d_ff;
    int32_t vocab;
    int32_t dtype;       /* DASH_F32 or DASH_BF16 */
    float rope_theta;
    float rms_eps;
} dash_model_desc;

typedef struct dash_model dash_model;
typedef struct dash_kv dash_kv;

/* ---- library ------------------------------------------------------------ */

/* DASH_ABI_VERSION of the built library. */
int dash_abi_version(void);

/* Static text for a dash_status value (never NULL). */
const char* dash_status_str(int status);

/* Text of the last error on the calling thread ("" if none).  Valid until the
 * next failing call on the same thread. */
const char* dash_last_error(void);

/* ---- model -------------------------------------------------------------- */

/* Number of device pointers dash_model_create expects: 3 + 7 * n_layers. */
int32_t dash_weight_count(const dash_model_desc* desc);

/*
 * Create a model handle over caller-owned device weights (not copied; they
 * must outlive the handle).  d_weights[] lists, in this order, arrays of the
 * model dtype, row-major:
 *   [0] embed      [vocab, d_model]     (also the tied LM head)
 *   [1] final_norm [d_model]
 *   [2] lm_head    must be NULL (embeddings are tied)
 *   then for each layer l, at 3 + 7 l:
 *   +0 attn_norm [d_model]
 *   +1 w_qkv     [(n_heads + 2 n_kv_heads) head_dim, d_model]   rows: q, then k, then v
 *   +2 b_qkv     [(n_heads + 2 n_kv_heads) head_dim]
 *   +3 w_o       [d_model, n_heads head_dim]
 *   +4 mlp_norm  [d_model]
 *   +5 w_gate_up [2 d_ff, d_model]                             rows: gate, then up
 *   +6 w_down    [d_model, d_ff]
 * Every pointer must be 16-byte aligned.  Shapes the kernels cover
 * (d_model <= 4096 and vocab <= 2^28 always):
 *   DASH_BF16: head_dim in {64, 128}, d_model % 64 == 0, d_ff % 64 == 0,
 *              n_heads / n_kv_heads <= 16;
 *   DASH_F32:  head_dim <= 128, d_model, d_ff multiples of 4.
 * Returns DASH_EINVAL for inconsistent shapes, DASH_ENOTSUP outside the above.
 */
int dash_model_create(const dash_model_desc* desc, const void* const* d_weights,
                      int32_t n_weights, dash_model** out);
void dash_model_destroy(dash_model* model);

/* ---- paged KV cache ----------------------------------------------------- */

/*
 * The KV cache is a pool of pages; a page holds page_size consecutive
 * positions of one sequence for every layer, both K and V and all kv heads.
 * A sequence lives in a "slot" (0 <= slot < max_seqs) whose page-table row
 * lists its pages.  Pages are reference counted: the G samples of a prompt
 * share the prompt's full pages (the group fork of Sec. 3.4), and a partial
 * last prompt page is copied for each sample.
 *
 * dash_kv_page_bytes: bytes of one page for this model and page size.
 * dash_kv_table_bytes: bytes of the device page-table buffer (int32
 *   [max_seqs, ceil(max_ctx / page_size)] plus a status word).
 * page_size: DASH_BF16 needs a multiple of 32; DASH_F32 any value in [1, 1024].
 */
size_t dash_kv_page_bytes(const dash_model* model, int32_t page_size);
size_t dash_kv_table_bytes(int32_t max_seqs, int32_t max_ctx, int32_t page_size);

/*
 * Create a KV handle over a caller-owned device pool (pool_bytes /
 * dash_kv_page_bytes pages, 256-byte aligned) and page-table buffer
 * (dash_kv_table_bytes).  Enqueues a clear of the page table on `stream`.
 * max_ctx bounds every slot's length (prompt + generated tokens).
 * Decode attention cuts a slot's context into splits whose length is fixed here
 * from max_seqs, the kv heads, the head dim and max_ctx (long splits for large capacities,
 * short ones so that small batches still fill the GPU); a sequence's results in
 * one cache therefore never depend on which other rows share its batch.
 */
int dash_kv_create(const dash_model* model, void* d_pool, size_t pool_bytes, int32_t page_size,
                   int32_t max_seqs, int32_t max_ctx, void* d_page_table, void* stream,
                   dash_kv** out);
void dash_kv_destroy(dash_kv* kv);

/* Pages currently free in the pool, the current length of one slot, and the
 * decode-attention split length (keys) chosen at creation. */
int dash_kv_free_pages(const dash_kv* kv, int32_t* out);
int dash_kv_slot_len(const dash_kv* kv, int32_t slot, int32_t* out);
int dash_kv_split_keys(const dash_kv* kv, int32_t* out);

/*
 * Grow the listed slots so that positions [0, new_len) are backed by pages
 * (allocating from the free list) and set their length to new_len.  The
 * page-table update is uploaded on `stream`.  Slots already at least that long
 * are left unchanged.  DASH_ECAPACITY (and no change at all) if the pool or
 * max_ctx cannot hold the growth.
 */
int dash_kv_reserve(dash_kv* kv, const int32_t* h_slots, int32_t n, int32_t new_len, void* stream);

/* Drop the listed slots: their pages' reference counts fall and pages that
 * reach zero return to the free list; the slots become empty.  Host-only
 * bookkeeping: pages are reused only by later stream-ordered work. */
int dash_kv_release(dash_kv* kv, const int32_t* h_slots, int32_t n);

/* Device status bits.  Faults found inside kernels are recorded as sticky bits
 * of a status word instead of stopping the stream:
 *   DASH_ST_UNBACKED          a position without a backing page was met (its
 *                             cache write was skipped);
 *   DASH_ST_NO_FINITE_LOGIT   a sampled row had no finite logit (its token is -1);
 *   DASH_ST_BAD_TOKEN         a token fed to the decoder was outside [0, vocab)
 *                             (its hidden-state row, and all that depends on it,
 *                             is NaN; the id is never used as an index). */
enum { DASH_ST_UNBACKED = 1u, DASH_ST_NO_FINITE_LOGIT = 2u, DASH_ST_BAD_TOKEN = 4u };

/* Read (and clear) the device status word of a cache after synchronising
 * `stream`: the bits set by dash_prefill, dash_decode_step, the teacher-forced
 * calls and dash_rollout (which also records its sampler's bits here). */
int dash_kv_device_status(dash_kv* kv, uint32_t* out, void* stream);

/* ---- workspace ---------------------------------------------------------- */

/* Bytes of device workspace dash_prefill / dash_decode_step need for up to
 * max_rows token rows per call (prefill rows = prompts in one chunk x prompt
 * length; prefill splits a batch the workspace cannot hold at once into the
 * fewest chunks of whole prompts, of equal size but for a smaller last one).
 * max_ctx: the max_ctx of the kv handle used with it (sizes the decode
 * attention's per-split partial results; 0 for a prefill-only workspace). */
size_t dash_workspace_bytes(const dash_model* model, int32_t max_rows, int32_t max_ctx);

/* ---- the hot path ------------------------------------------------------- */

/*
 * Prefill (Sec. 3.4: one large batch of prompts, each duplicated into a group).
 * d_prompt_tokens: int32 [n_prompts, prompt_len], ids in [0, vocab).
 * h_slots: int32 [n_prompts * group]; sample j of prompt p uses slot
 *   h_slots[p * group + j].  All these slots must be empty.
 * Runs the decoder over every prompt at positions 0..prompt_len-1, writes the
 * prompt K/V once per prompt into pages shared by the group's slots (a partial
 * last page is copied per slot), sets every slot's length to prompt_len, and
 * writes the next-token logits at position prompt_len-1: float32
 * d_logits [n_prompts, vocab].  The first token of every sample is drawn from
 * its prompt's row (dash_sample with d_row_of[n] = n / group).
 * d_ws: dash_workspace_bytes(model, rows, 0) bytes with rows >= prompt_len.
 * DASH_ECAPACITY (before any launch) if the pool cannot hold the prompts.
 */
int dash_prefill(dash_model* model, dash_kv* kv, const int32_t* d_prompt_tokens, int32_t n_prompts,
                 int32_t prompt_len, int32_t group, const int32_t* h_slots, float* d_logits,
                 void* d_ws, size_t ws_bytes, void* stream);

/*
 * One decode step over n_rows rows: every token of a trajectory is drawn from
 * pi_theta(. | x, y_<t) (Sec. 3 problem statement, Eq. (1)), and preemptive
 * sampling runs the whole large batch of samples through the policy at once
 * (Sec. 3.4); this call computes those next-token distributions, as logits,
 * for one position of every row.  Row b feeds token d_tokens[b] at position
 * d_pos[b] of slot d_slots[b]: its K/V are appended to the cache at that
 * position and float32 d_logits [n_rows, vocab] receives the next-token
 * logits.  A token outside [0, vocab) sets DASH_ST_BAD_TOKEN.  Positions must be backed by pages (dash_kv_reserve with
 * new_len > pos); the kernels skip unbacked writes and set status bit 0.
 * Attention of row b covers positions 0..d_pos[b] of its slot.  Steps over
 * disjoint slots may run at the same time on different streams, each with its
 * own workspace and logits (with kernel timing off the call changes no host
 * state); a row's logits do not depend on the other rows of its call.
 */
int dash_decode_step(dash_model* model, dash_kv* kv, const int32_t* d_tokens, const int32_t* d_slots,
                     const int32_t* d_pos, int32_t n_rows, float* d_logits, void* d_ws, size_t ws_bytes,
                     void* stream);

/*
 * dash_decode_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The step's workspace is a 64 MiB device
 * array inside the library (one per device, created with the loaded code and
 * held until the process ends); nothing is allocated by the call.  The caller
 * passes inputs and outputs as for dash_decode_step and gets the same logits
 * bit for bit.  DASH_ECAPACITY (before any launch) when
 * dash_workspace_bytes(model, n_rows, kv max_ctx) exceeds 64 MiB (up to 496
 * rows for the Qwen2.5-1.5B shape at max_ctx 1280, 752 for 0.5B, 361 for 3B at
 * max_ctx 1536).  Every call on a device shares that
 * device's array: calls that overlap in time on one device (different streams
 * or threads) race and give undefined results; serialise them.
 */
int dash_decode_step_noalloc(dash_model* model, dash_kv* kv, const int32_t* d_tokens, const int32_t* d_slots,
                             const int32_t* d_pos, int32_t n_rows, float* d_logits, void* stream);

/*
 * dash_decode_step for a batch made of prefix-sharing groups (the G samples of a
 * prompt after the group fork, Sec. 3.4): rows d_group_off[i] .. d_group_off[i+1]-1
 * (int32 device array of n_groups + 1 ascending offsets, the first 0 and the last
 * equal to n_rows, each group at most group_size <= 8 rows) share their first
 * shared_len positions, i.e. the same pages (shared_len a multiple of page_size, at
 * most max_ctx and at most the prompt's full pages).  Decode attention then runs
 * those shared pages once per group and kv head, for all the group's query heads
 * at once, and continues every row from the online-softmax state this leaves
 * (kept in the workspace) over its own pages.  Results are bit-identical to
 * dash_decode_step.  DASH_ENOTSUP for group_size > 8; fp32 models, and shapes the
 * prefix kernel does not cover, run the per-row kernel (same results).
 */
int dash_decode_step_grouped(dash_model* model, dash_kv* kv, const int32_t* d_tokens, const int32_t* d_slots,
                             const int32_t* d_pos, int32_t n_rows, const int32_t* d_group_off, int32_t n_groups,
                             int32_t group_size, int32_t shared_len, float* d_logits, void* d_ws, size_t ws_bytes,
                             void* stream);

/*
 * Temperature sampling by Gumbel-max with counter-based noise: the draw
 * y_t ~ pi_theta(. | x, y_<t) of Sec. 3 (problem statement, Eq. (1)) for every
 * sample of the batch, G samples per prompt (Sec. 3.4), at temperature T (pure
 * temperature sampling: the paper names no top-k / top-p filter).
 * Row b reads float32 logits row r = d_row_of ? d_row_of[b] : b at
 * d_logits + r * ld, and draws token argmax_v (l_v / T + g_v) over finite l_v
 * (ties to the smallest v; -1 if no l_v is finite), which is a draw from
 * softmax(l / T).  The noise g_v = -L(-L(u)) with u = ((x >> 8) | 1) 2^-24 and
 * x = Philox4x32-10(counter = (v >> 2, d_step[b], d_seq_uid[b], 0),
 * key = (seed mod 2^32, seed >> 32)) word v & 3; L is the library's own
 * float32 natural log (argument reduction to [sqrt(1/2), sqrt(2)] and the
 * series 2 atanh((m - 1)/(m + 1)), each operation rounded separately), so a
 * draw depends only on (seed, seq_uid, step, logits) and is bit-reproducible.
 * d_tokens_out [n_rows] int32; d_logprob_out [n_rows] float32 (nullable):
 * log softmax(l / T) at the drawn token; d_row_max_lse [n_rows, 2] float32
 * (nullable): per row m = max_v l_v / T and ln sum_v exp(l_v / T), so that
 * log softmax(l / T)_v = l_v / T - that second value for any v (both NaN for a
 * row without a finite logit); d_status (nullable, device uint32): bits OR-ed
 * in, DASH_ST_NO_FINITE_LOGIT when a row has no finite logit.  DASH_EINVAL if
 * temperature <= 0 or not finite, vocab < 1 or > 2^28, or ld < vocab.
 */
int dash_sample(const float* d_logits, int64_t ld, int32_t n_rows, int32_t vocab, const int32_t* d_row_of,
                const int32_t* d_seq_uid, const int32_t* d_step, float temperature, uint64_t seed,
                int32_t* d_tokens_out, float* d_logprob_out, float* d_row_max_lse, uint32_t* d_status,
                void* stream);

/*
 * Self-check of the sampler's screening.  dash_sample first scores every entry
 * with a cheap noise (hardware logarithm) and computes the exact noise only for
 * entries that can still win; this is exact provided the cheap noise is within
 * the tolerance of the exact one for every possible u.  This call measures the
 * largest |cheap - exact| over all 2^23 values u can take, on the current
 * device, and returns it with the tolerance the sampler assumes (h_max_err <
 * h_tol means the screening is exact here).  Synchronous (null stream); the
 * maximum is reduced into a device variable of the library, so the call
 * allocates nothing.
 */
int dash_sampler_check(double* h_max_err, double* h_tol);

/*
 * Self-check of the bfloat16 rounding.  Every bf16 value the kernels store (weights
 * aside: those come in bf16) is the round-to-nearest-even of a float32, which the
 * kernels take from the GPU's conversion instruction; the bf16 storage points of
 * the decoder (Sec. 4.1 runs it in bf16) are defined by that rounding.  This call
 * converts all 2^32 float32 bit patterns on the current device and counts those
 * whose result differs from integer rounding of the pattern (add 0x7FFF plus the
 * lowest kept bit, truncate; NaNs keep their top half with the quiet bit set);
 * 0 means the two agree everywhere.  Synchronous (null stream); the count is
 * reduced into a device variable of the library, so the call allocates nothing.
 */
int dash_bf16_round_check(uint64_t* h_mismatches);

/*
 * GRPO group advantage (Sec. 3.3, Eq. (4)) and gradient filter (Sec. 3.5).
 * d_rewards: float32 [n_groups * group], group k = samples k*group .. k*group+group-1.
 * mean = S(r)/G, d = r - mean, A = d (MEAN_ONLY) or d / (sqrt(S(d*d)/(G - ddof)) + eps)
 * (std = 0 when G - ddof <= 0); DASH_ADV_LOO: the leave-one-out baseline of
 * Sec. 3.3, A = r - (S(r) - r)/(G - 1) (eps unused).  S is a pairwise sum
 * (zero-padded to a power of two, adjacent pairs first) and every float32
 * operation is rounded on its own, so results are bit-reproducible.  One group
 * of all N samples is the single-path estimate, Eq. (3).
 * Outputs: d_adv float32 [N]; d_kept_idx int32 [N] capacity, the ascending
 * indices n with |A_n| >= tau; d_kept_count int32 [1].  (tau = 0 keeps all;
 * the smallest positive float keeps exactly the nonzero advantages.)
 * DASH_EINVAL for group < 1 (< 2 for LOO), n_groups < 1, bad mode, eps < 0,
 * tau < 0 or NaN; DASH_ENOTSUP for group > 65536 or N > 2^24.
 */
int dash_group_advantage_filter(const float* d_rewards, int32_t n_groups, int32_t group, int32_t mode,
                                float eps, float tau, float* d_adv, int32_t* d_kept_idx,
                                int32_t* d_kept_count, void* stream);

/*
 * Stream compaction of live decode rows (ragged rollouts retire rows as they
 * finish, so the decode batch shrinks).  Input row b is (token, slot, pos,
 * step, uid) after its token for `step` was sampled; it stays live iff
 * step + 1 < d_budget[uid] and token != eos_id (eos_id < 0: no EOS).  Live
 * rows are written in order to the output arrays advanced by one position
 * (pos + 1, step + 1), and their count to d_count [1].  In- and output arrays
 * must not overlap.
 */
int dash_live_compact(const int32_t* d_tok, const int32_t* d_slot, const int32_t* d_pos, const int32_t* d_step,
                      const int32_t* d_uid, const int32_t* d_budget, int32_t eos_id, int32_t n_rows,
                      int32_t* d_tok_out, int32_t* d_slot_out, int32_t* d_pos_out, int32_t* d_step_out,
                      int32_t* d_uid_out, int32_t* d_count, void* stream);

/* ---- after the filter: log-probs of the kept samples and the PG loss ------ */

/*
 * Teacher-forced log-probabilities (the forward half of the policy-gradient
 * step that follows the filter: Sec. 3.2's PG estimate needs
 * log pi_theta(y | x) = sum_t log pi_theta(y_t | x, y_<t) for every kept
 * sample).  d_tokens: int32 [n_seqs, seq_len], each row a prompt (first
 * prompt_len tokens) followed by its completion.  d_logprobs: float32
 * [n_seqs, seq_len - prompt_len]; entry (b, t) = log softmax(logits at position
 * prompt_len - 1 + t)[d_tokens[b, prompt_len + t]] at temperature 1.
 * The sequences are run through the prefill path (causal attention over the
 * whole sequence, KV written to pages of slots 0 .. c-1, which must be empty
 * and are released again) in chunks of c sequences, the largest c for which
 * dash_teacher_forced_workspace_bytes(model, c, seq_len, prompt_len) <=
 * ws_bytes and the pool holds c sequences.  The LM head output of a chunk is
 * kept in the workspace (c * (seq_len - prompt_len) * vocab floats).
 * DASH_ECAPACITY if not even one sequence fits.
 */
size_t dash_teacher_forced_workspace_bytes(const dash_model* model, int32_t seqs_per_chunk, int32_t seq_len,
                                           int32_t prompt_len);
int dash_teacher_forced_logprobs(dash_model* model, dash_kv* kv, const int32_t* d_tokens, int32_t n_seqs,
                                 int32_t seq_len, int32_t prompt_len, float* d_logprobs, void* d_ws,
                                 size_t ws_bytes, void* stream);

/*
 * Policy-gradient loss over the kept samples (Sec. 3.2, Eq. (2) with the
 * group advantage of Sec. 3.3 and gradient filtering of Sec. 3.5; no 1/len
 * weight): loss = -(1/n_total) * sum over k < *d_kept_count of
 * A[n] * sum_{t < len[n]} lp[n][t], n = d_kept_idx[k], in float64.
 * d_logprobs float32 [n_total, ld] (ld >= T); d_lengths int32 [n_total]
 * (nullable: every sample has T tokens; values are clamped to [0, T]);
 * d_adv float32 [n_total]; d_kept_idx / d_kept_count as written by
 * dash_group_advantage_filter.  Outputs: d_loss float64 [1];
 * d_seq_logprob float64 [n_total] (nullable): the sequence log-prob of every
 * kept sample.  Deterministic (fixed reduction order).
 */
int dash_pg_loss(const float* d_logprobs, int64_t ld, int32_t T, const int32_t* d_lengths, const float* d_adv,
                 const int32_t* d_kept_idx, const int32_t* d_kept_count, int32_t n_total, double* d_loss,
                 double* d_seq_logprob, void* stream);

/*
 * KL regulariser (Sec. 3.2: the divergence D_KL(pi_base || pi_theta) from the
 * original model, weighted by beta).  Per row pair of float32 logits
 * d_theta / d_base [rows, ld] (ld >= vocab; entries past vocab are ignored):
 * d_kl[r] = D_KL(softmax(base_r) || softmax(theta_r)) and, if d_kl_rev is not
 * NULL, d_kl_rev[r] = D_KL(softmax(theta_r) || softmax(base_r)), float32, at
 * temperature 1.  A -inf logit has probability zero; an entry with mass on one
 * side and -inf on the other makes that direction +inf; NaN logits give NaN.
 * Exponentials in float32, sums in float64: identical rows give exactly 0.
 */
int dash_logits_kl(const float* d_theta, const float* d_base, int64_t ld, int32_t rows, int32_t vocab, float* d_kl,
                   float* d_kl_rev, void* stream);

/*
 * Teacher-forced KL along sampled completions: for every completion position of
 * d_tokens (layout as in dash_teacher_forced_logprobs), the exact KL between the
 * next-token distributions of the base model and the policy after the same
 * prefix, summed later over positions by dash_policy_loss.  base must have the
 * policy's architecture (same dash_model_desc values); kv belongs to model and
 * serves both forwards (the base model's pass runs first, slots 0 .. c-1 must
 * be empty and are released).  Outputs float32 [n_seqs, seq_len - prompt_len]:
 * d_logprobs (nullable; bit-identical to dash_teacher_forced_logprobs), d_kl
 * (D_KL(base || policy)), d_kl_rev (nullable, D_KL(policy || base)).  Chunks of
 * c sequences, the largest c with dash_teacher_forced_kl_workspace_bytes(model,
 * c, seq_len, prompt_len) <= ws_bytes (two logits buffers per chunk).
 */
size_t dash_teacher_forced_kl_workspace_bytes(const dash_model* model, int32_t seqs_per_chunk, int32_t seq_len,
                                              int32_t prompt_len);
int dash_teacher_forced_kl(dash_model* model, dash_model* base, dash_kv* kv, const int32_t* d_tokens, int32_t n_seqs,
                           int32_t seq_len, int32_t prompt_len, float* d_logprobs, float* d_kl, float* d_kl_rev,
                           void* d_ws, size_t ws_bytes, void* stream);

/*
 * Regularised policy loss over the kept samples (Sec. 3.2), float64.  With
 * S_n = sum_{t < len[n]} lp[n][t]:
 *   d_logprobs_old == NULL: surrogate_n = A_n S_n (the PG loss of dash_pg_loss);
 *   otherwise PPO with the whole-trajectory ratio rho_n = exp(S_n - S_old,n)
 *   (the ratio Sec. 3.2 writes) and the clipped surrogate
 *   min(rho_n A_n, clip(rho_n, 1 - clip_eps, 1 + clip_eps) A_n), clip_eps in [0, 1).
 * loss = -(1/n_total) sum_kept surrogate_n + (beta/n_total) sum_kept KL_n, where
 * KL_n sums d_kl[n][t] over t < len[n] (d_kl NULL: no KL term, beta unused).
 * d_logprobs, d_logprobs_old and d_kl are float32 [n_total, ld] (ld >= T);
 * d_lengths, d_adv, d_kept_idx, d_kept_count as for dash_pg_loss.  Outputs:
 * d_loss float64 [1]; d_stats float64 [n_total, 4] (nullable), for each kept n:
 * (S_n, S_old,n (= S_n without old log-probs), KL_n, d loss / d S_n), the last
 * being the weight a backward pass puts on grad S_n: -A_n/n_total (PG),
 * -A_n rho_n/n_total where the unclipped term is the minimum (PPO), else 0.
 * Deterministic; with d_logprobs_old and d_kl NULL the loss equals
 * dash_pg_loss's bit for bit.
 */
int dash_policy_loss(const float* d_logprobs, const float* d_logprobs_old, const float* d_kl, int64_t ld, int32_t T,
                     const int32_t* d_lengths, const float* d_adv, const int32_t* d_kept_idx,
                     const int32_t* d_kept_count, int32_t n_total, double clip_eps, double beta, double* d_loss,
                     double* d_stats, void* stream);

/* ---- native rollout driver ---------------------------------------------- */

/*
 * A whole preemptive-sampling rollout: prefill of n_prompts prompts, G samples
 * each (sample n = prompt * G + j, slot n), then decode steps until every
 * sample has its tokens.  Sample n generates h_budget ? h_budget[n] : gen_len
 * tokens (1 <= budget <= gen_len); rows retire when done and the batch is
 * compacted.  Pages are reserved one page ahead as sequences grow and released
 * as samples finish.
 * Outputs: d_out_tokens int32 [N, gen_len] (entries after a sample's budget
 * are -1) and d_out_logprobs float32 [N, gen_len] (nullable).
 * The kv handle must have max_seqs >= N, max_ctx >= prompt_len + gen_len and
 * be empty.  d_ws: dash_rollout_workspace_bytes(model, n_prompts, prompt_len, group, kv max_ctx).
 * use_graph != 0 captures the fixed-batch decode step (decode + sample +
 * advance) once as a HIP graph and replays it (ragged rollouts, whose batch
 * shrinks, run eagerly).  Kernel-class timing (dash_profile_enable) also works
 * under graphs: the timed launches become event-record nodes of the graph.
 */
size_t dash_rollout_workspace_bytes(const dash_model* model, int32_t n_prompts, int32_t prompt_len,
                                    int32_t group, int32_t max_ctx);
int dash_rollout(dash_model* model, dash_kv* kv, const int32_t* d_prompt_tokens, int32_t n_prompts,
                 int32_t prompt_len, int32_t group, int32_t gen_len, const int32_t* h_budget,
                 float temperature, uint64_t seed, int32_t* d_out_tokens, float* d_out_logprobs,
                 int32_t use_graph, void* d_ws, size_t ws_bytes, void* stream);

/* ---- kernel timing (diagnostics) ---------------------------------------- */

/* Kernel classes of the path. */
enum {
    DASH_K_PREFILL = 0,      /* every kernel of dash_prefill */
    DASH_K_EMBED = 1,        /* embedding gather + first RMSNorm */
    DASH_K_NORM = 2,         /* residual add + RMSNorm */
    DASH_K_ROPE = 3,         /* RoPE table, q/k RoPE + KV append */
    DASH_K_GEMM_QKV = 4,
    DASH_K_ATTN = 5,         /* decode attention (per context split) */
    DASH_K_ATTN_COMBINE = 6, /* merge of context splits */
    DASH_K_GEMM_O = 7,
    DASH_K_GEMM_GATE_UP = 8, /* with the SwiGLU epilogue */
    DASH_K_GEMM_DOWN = 9,
    DASH_K_GEMM_LM_HEAD = 10,
    DASH_K_SAMPLE = 11,
    DASH_K_ADVANTAGE = 12,
    DASH_K_OTHER = 13,       /* row bookkeeping, compaction, page copies */
    DASH_K_COUNT = 14
};

/*
 * While a class's bit is set in `class_mask`, the library brackets each launch
 * of that class with a pair of HIP events on the launch stream and accumulates
 * the elapsed time (GPU clock).  Under stream capture the two records become
 * event-record nodes of the graph, so each replay times its launches (the
 * rollout driver reads a replay's times back before replaying that graph
 * again).  0 turns timing off.  Not thread-safe.
 */
int dash_profile_enable(uint32_t class_mask);

/* Limit the timing of per-layer classes (norm, rope, attention, the layer
 * GEMMs) to the launches of decoder layer `layer`; -1 (the default) times every
 * layer.  Every layer runs the same kernels on the same shapes, so one layer's
 * launches give the average launch time with a fraction of the event records. */
int dash_profile_layer(int32_t layer);

/* Wait for the pending event pairs, then report per class the summed time in
 * milliseconds (ms_out[DASH_K_COUNT]) and the number of timed launches
 * (launches_out[DASH_K_COUNT]); reset != 0 clears the sums afterwards.
 * DASH_EDEVICE (outputs still filled) if an event record or read-back failed
 * since the last call; those launches are missing from the sums. */
int dash_profile_read(double* ms_out, int64_t* launches_out, int32_t reset);

#ifdef __cplusplus
}
#endif

#endif /* DASH_H */
