/*
 * hdl.h -- C ABI of libhdl.so, the MI355X (gfx950) hindsight re-scoring path
 * of Hindsight-Divergence Localization (HDL).
 *
 * The paper re-scores each sampled root twice with teacher forcing, once
 * under the original context and once under the hindsight context (Sec. 3.1,
 * Eq. 1), scores every policy-generated token by the absolute change of its
 * log-likelihood (Sec. 3.2, Eq. 2) and keeps the highest-scoring positions of
 * each root as branch points (Sec. 3.2; two per root in Sec. 4.1).
 *
 * Conventions shared by every entry point
 *  - All array pointers are DEVICE pointers to caller-owned memory.  The
 *    library allocates no device memory and keeps no pointer after a call
 *    returns.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL means
 *    the default stream).  Outputs are valid once the caller synchronises the
 *    stream.  The library never synchronises.
 *  - Kernels launch on the calling thread's current HIP device; `stream` and
 *    every pointer must belong to that device.
 *  - Argument errors are reported synchronously by a negative return value,
 *    before anything is enqueued.  A failed kernel launch returns
 *    HDL_ERR_HIP.  hdl_last_hip_error() describes the most recent failure of
 *    the calling thread (an argument error or a HIP error).  No C++ exception crosses this boundary.
 *  - Row-major layouts throughout; "[a, b]" means a rows of b contiguous
 *    elements.
 */
#ifndef HDL_H_
#define HDL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of `hidden` and `w_vocab`.  Accumulation, the log-sum-exp and
 * all outputs are fp32 for both. */
/* Element type of hidden states and the vocabulary projection (the last
 * enumerator only keeps the type int-sized; it is not a valid dtype). */
typedef enum { HDL_F32 = 0, HDL_BF16 = 1, HDL_DTYPE_INT_ = 0x7fffffff } hdl_dtype;

enum {
  HDL_OK = 0,
  HDL_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, bad alignment */
  HDL_ERR_UNSUPPORTED = -2, /* unknown dtype, d not a multiple of 8, k > 1024 */
  HDL_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required    */
  HDL_ERR_HIP = -4          /* a HIP call or kernel launch failed            */
};

/* Largest k accepted by hdl_select_branch_points. */
#define HDL_MAX_K 1024

/*
 * Bytes of device workspace hdl_token_logprobs needs for these sizes
 * (0 if the sizes are invalid).  The workspace holds the compacted list of
 * scored rows and the per-vocabulary-chunk partial log-sum-exp states.
 */
size_t hdl_token_logprobs_workspace_size(int64_t n_rows, int64_t d, int64_t vocab,
                                         hdl_dtype dtype);

/*
 * Teacher-forced log-likelihood of each row's sampled token (Eq. 1):
 *
 *     logp[n] = z_n[tokens[n]] - log sum_v exp(z_n[v]),   z_n = W_vocab h_n,
 *
 * computed by one fused kernel: the lm-head contraction on bf16 (or fp32)
 * MFMA tiles with fp32 accumulation, an online max / log-sum-exp carried
 * across vocabulary tiles, and capture of the sampled token's logit.  The
 * n_rows x vocab logits are never written to memory.
 *
 *  hidden   [n_rows, d]  dtype; row n is the final hidden state that PREDICTS
 *                        tokens[n] (the caller applies the teacher-forcing
 *                        shift).  For HDL both contexts go in one call, rows
 *                        ordered [context][root][t]; W is shared (Eq. 1 uses
 *                        the same parameters for both contexts).  16-byte
 *                        aligned.
 *  w_vocab  [vocab, d]   dtype, the lm-head weight (nn.Linear layout).
 *                        16-byte aligned.
 *  tokens   [n_rows]     int32 sampled tokens.  Precondition: 0 <= t < vocab;
 *                        a row that violates it gets logp = NaN (never an
 *                        error).  A NaN or infinite hidden-state element
 *                        likewise gives its row logp = NaN and lse = NaN; the
 *                        other rows are unaffected.
 *  mask     [n_rows]     uint8, or NULL for "all rows".  Only rows with
 *                        mask != 0 (policy-generated tokens, Sec. 3.1) are
 *                        computed; the others get logp = 0 and lse = 0 and
 *                        cost no matrix work.
 *  d                     multiple of 8.
 *  logp     [n_rows]     fp32 out.
 *  lse_out  [n_rows]     fp32 out (log-sum-exp of the row), or NULL.
 *  workspace             device memory of at least
 *                        hdl_token_logprobs_workspace_size(...) bytes,
 *                        256-byte aligned; contents on entry are ignored.
 *
 * Deterministic: the same inputs give bitwise-identical outputs, and a row's
 * result does not depend on the other rows of the call.  Calls whose hidden
 * states span more than 4 GiB are processed in several launches internally.
 */
int hdl_token_logprobs(const void* hidden, const void* w_vocab, const int32_t* tokens,
                       const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab,
                       hdl_dtype dtype, float* logp, float* lse_out, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * hdl_token_logprobs plus the next-token entropy of every scored row,
 *
 *     entropy[n] = - sum_v p_n(v) log p_n(v) = ln S_n - E_{p_n}[z - m_n],
 *     S_n = sum_v exp(z_v - m_n),  m_n = max_v z_v,
 *
 * accumulated in the same pass over W (one more online accumulator,
 * sum_v exp(z_v - m) (z_v - m), carried relative to the running max so that
 * both terms are non-negative and nothing cancels for large logits).  The Entropy localization baseline the paper
 * compares against ranks positions by this quantity under the original
 * context (Sec. 4.1, "Rollout protocols"; Table 4).
 *
 *  entropy  [n_rows] fp32 out (required; 0 for masked rows).  All other
 *           arguments, the workspace size and the error behaviour are those
 *           of hdl_token_logprobs.
 */
int hdl_token_logprobs_entropy(const void* hidden, const void* w_vocab, const int32_t* tokens,
                               const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab,
                               hdl_dtype dtype, float* logp, float* lse_out, float* entropy,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * hdl_token_logprobs without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  The library allocates nothing for it
 * either: its workspace is a fixed 32 MiB device array inside the library
 * (one per GPU, held until the process ends; its address is looked up once
 * per device on the first call on that device, with that device current).
 *
 * Arguments, outputs, numerics and error behaviour are those of
 * hdl_token_logprobs (without the entropy).  The caller still provides every
 * input and output buffer.  Where the default vocabulary chunking's partials
 * do not fit the array, the call uses fewer, longer chunks, so results may
 * differ from hdl_token_logprobs by rounding (the same bound holds); where
 * they fit, the results are bit-identical.  A launch (at most 4 GiB of hidden
 * states) needs 16 bytes of the array per row: a call whose launch would
 * cover more than about 2.09 million rows (only possible for d * element
 * size below 2 KiB) returns HDL_ERR_UNSUPPORTED before touching the GPU.
 *
 * Every call on one GPU uses that GPU's array and leaves its contents
 * behind; nothing in it has to start at zero.  Calls that overlap on one GPU
 * (concurrent streams or threads) race on the array: serialise them.
 */
int hdl_token_logprobs_noalloc(const void* hidden, const void* w_vocab, const int32_t* tokens,
                               const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab,
                               hdl_dtype dtype, float* logp, float* lse_out, void* stream);

/*
 * Hindsight-divergence score and per-root branch-point selection (Eq. 2 and
 * the ranking of Sec. 3.2):
 *
 *     s[r, t] = | logp_hind[r, t] - logp_orig[r, t] |     (fp32 subtraction)
 *
 * over eligible positions (mask != 0 and a finite difference; NaN rows never
 * qualify).  For each root the k eligible positions with the largest s are
 * returned ordered by (s descending, t ascending); an exact tie at the k-th
 * place goes to the lower t.
 *
 *  logp_orig, logp_hind [n_roots, T] fp32, as written by hdl_token_logprobs.
 *  mask         [n_roots, T] uint8, or NULL for "all positions".
 *  k            1 .. HDL_MAX_K.
 *  idx          [n_roots, k] int32 out: selected positions, -1 padding.
 *  score        [n_roots, k] fp32 out: their s, 0 padding.
 *  count        [n_roots]    int32 out: min(k, number of eligible positions).
 *  delta_signed [n_roots, T] fp32 out (logp_hind - logp_orig on eligible
 *               positions, 0 elsewhere), or NULL.
 */
int hdl_select_branch_points(const float* logp_orig, const float* logp_hind,
                             const uint8_t* mask, int64_t n_roots, int64_t T, int32_t k,
                             int32_t* idx, float* score, int32_t* count,
                             float* delta_signed, void* stream);

/*
 * Per-root top-k of an arbitrary per-position value (for example the
 * next-token entropy of the Entropy baseline, Sec. 4.1): for each root, the
 * k positions with mask != 0 and a finite value that have the largest value,
 * ordered (value descending, t ascending); -0 ranks as +0.
 *
 *  values [n_roots, T] fp32; mask [n_roots, T] uint8 or NULL; k 1 .. HDL_MAX_K.
 *  idx [n_roots, k] int32 out (-1 padding), score [n_roots, k] fp32 out
 *  (0 padding), count [n_roots] int32 out.
 */
int hdl_select_top_k(const float* values, const uint8_t* mask, int64_t n_roots, int64_t T,
                     int32_t k, int32_t* idx, float* score, int32_t* count, void* stream);

/*
 * Bytes of device workspace hdl_token_logprobs_backward needs for these sizes
 * (0 if the sizes are invalid or unsupported).  Dominated by one chunk's
 * logit gradient, 2 * min(round_up(n_rows, 256), 32768) * round_up(vocab, 64)
 * bytes (10 GB for 32768 rows and a 151,936-token vocabulary), plus the
 * chunk's gathered hidden rows and the partial sums of its dH rows (about
 * 0.4 GB for 32768 rows at d = 2048).
 */
size_t hdl_token_logprobs_backward_workspace_size(int64_t n_rows, int64_t d, int64_t vocab,
                                                  hdl_dtype dtype);

/*
 * Backward pass of hdl_token_logprobs for a loss L = sum_n g_n log p_n(y_n)
 * (the policy loss of Sec. 3.3 is such a sum over the tokens it trains on;
 * g_n is its derivative with respect to each token's log-likelihood):
 *
 *     G[n][v]  = g_n (1[v == y_n] - p_n(v))          (dL/dz, never stored whole)
 *     dL/dh_n  = sum_v G[n][v] W[v]                  -> grad_hidden
 *     dL/dW_v  = sum_n G[n][v] h_n                   -> grad_w
 *
 * The logits are recomputed tile by tile from hidden and w_vocab; G exists
 * only for one chunk of at most 32768 scored rows at a time, as bf16; the two
 * contractions run on bf16 MFMA tiles with fp32 accumulation.
 *
 *  hidden, w_vocab, tokens, mask, n_rows, d, vocab: as for hdl_token_logprobs;
 *               dtype must be HDL_BF16; vocab must not exceed 2^30 and d
 *               2^23 (HDL_ERR_UNSUPPORTED otherwise).  Hidden states over
 *               4 GiB are processed in blocks of rows internally.
 *  lse          [n_rows] fp32: the log-sum-exp hdl_token_logprobs returned
 *               for the same inputs (read for scored rows only).
 *  grad_logp    [n_rows] fp32: g_n (read for scored rows only).
 *  grad_hidden  [n_rows, d] fp32 out; rows with mask == 0 are set to 0.
 *  grad_w       [vocab, d] fp32 out; overwritten, or accumulated into when
 *               accumulate_w != 0.
 *  workspace    hdl_token_logprobs_backward_workspace_size(...) bytes,
 *               256-byte aligned.
 *
 * A token outside [0, vocab) contributes no indicator term (G = -g p).
 * Deterministic: fixed chunking and fixed-order sums, no atomics.
 */
int hdl_token_logprobs_backward(const void* hidden, const void* w_vocab, const int32_t* tokens,
                                const uint8_t* mask, const float* lse, const float* grad_logp,
                                int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype,
                                float* grad_hidden, float* grad_w, int accumulate_w,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Per-root selection under the branch-point constraints that the paper
 * applies to every localization method (Sec. 4.3; an allowed index range
 * and a minimum distance between a root's points, whose values it does not
 * give, Sec. 4.4 and the Reflection prompt's lo/hi fields).
 *
 *  a, b      [n_roots, T] fp32.  b != NULL: rank s = |b - a| (a = logp_orig,
 *            b = logp_hind, as hdl_select_branch_points).  b == NULL: rank
 *            a's values themselves (e.g. next-token entropy).
 *  mask      [n_roots, T] uint8 or NULL.
 *  lo, hi    [n_roots] int32 or NULL: candidates are positions lo[r] <= t <= hi[r].
 *  min_gap   retained points of a root are at least min_gap positions apart
 *            (0 or 1: no spacing constraint).
 *  refill    0: rank the k best candidates and drop, in rank order, any point
 *            closer than min_gap to a better retained one (a root may end with
 *            fewer than k points, as in the paper when two points are too close);
 *            1: walk down the ranking (at most the best HDL_MAX_K candidates)
 *            until k points are retained.
 *  idx, score [n_roots, k], count [n_roots]: retained points in rank order
 *            (score descending, t ascending), -1 / 0 padding.
 */
int hdl_select_constrained(const float* a, const float* b, const uint8_t* mask, int64_t n_roots,
                           int64_t T, int32_t k, const int32_t* lo, const int32_t* hi,
                           int32_t min_gap, int refill, int32_t* idx, float* score,
                           int32_t* count, void* stream);

/*
 * Continuation slots of each root (Sec. 3.3, Sec. 4.1 "Rollout protocols":
 * three and four continuations for a root's two branch points; Sec. 4.4:
 * a root left with one valid point takes all of its continuations there).
 *
 *  idx [n_roots, k], count [n_roots]: a selection's output (device).
 *  alloc        HOST array of k slot counts, in rank order (e.g. {3, 4});
 *               k <= 16, 1 <= sum <= 4096.
 *  fallback_pos branch position used when a root has no point at all.
 *  branch_pos   [n_roots, sum(alloc)] int32 out: the position each
 *               continuation branches at (it reuses the root's prefix y_<pos).
 *               Rank j's alloc[j] slots follow rank j-1's; a missing rank's
 *               slots branch at the root's best point.
 *  branch_rank  [n_roots, sum(alloc)] int32 out (or NULL): the rank each slot
 *               branches at, -1 for the fallback.
 */
int hdl_allocate_continuations(const int32_t* idx, const int32_t* count, int64_t n_roots,
                               int32_t k, const int32_t* alloc, int32_t fallback_pos,
                               int32_t* branch_pos, int32_t* branch_rank, void* stream);

/*
 * Group-relative advantages without standard-deviation normalisation
 * (Sec. 3, A_j = R_j - mean(R); Sec. 4.1 follows Dr. GRPO): rewards and adv
 * are [n_groups, group_size] fp32; one group is a problem's M roots and
 * G - M continuations.  The mean is a fixed-order fp32 sum.
 */
int hdl_group_advantages(const float* rewards, int64_t n_groups, int32_t group_size, float* adv,
                         void* stream);

/*
 * Per-token factor g = dL/d log pi of the clipped policy loss (Sec. 4.1
 * "Training": asymmetric clipping, no KL, token-level aggregation), the
 * grad_logp input of hdl_token_logprobs_backward:
 *
 *     r = exp(logp_new - logp_old),  l = -min(r A, clip(r, 1 - eps_low, 1 + eps_high) A)
 *     g = scale * dl/dlogp_new = -scale * A r  where the unclipped term is the minimum, else 0
 *
 *  adv [n_traj] fp32; traj [n_tokens] int32: each token's trajectory (a
 *  token whose index is out of [0, n_traj) contributes nothing).
 *  pos, start (both or neither): pos [n_tokens] int32 is the token's position
 *  in its trajectory and start [n_traj] int32 the first trained position --
 *  0 for a root, the branch position for a continuation (only the newly
 *  sampled suffix is trained, Sec. 3.3).
 *  loss_mask [n_tokens] uint8 or NULL (policy-generated tokens).
 *  scale  the aggregation factor; scale <= 0 asks for the token-level mean of
 *         Sec. 4.1 ("Training"), scale = 1 / max(1, T) with T the number of
 *         trained tokens (in the mask, of a trajectory in [0, n_traj), at or
 *         after its first trained position), counted on the device.
 *  grad_logp [n_tokens] fp32 out (0 for untrained tokens); loss [n_tokens]
 *  fp32 out (scale * l, 0 for untrained tokens) or NULL.
 *  n_trained  device int64 [1] out or NULL: T; required (and used as the
 *         count's scratch) when scale <= 0.  8-byte aligned.
 *  A NaN scale, or scale <= 0 without n_trained, is HDL_ERR_INVALID_ARG.
 */
int hdl_policy_loss_grad(const float* adv, int64_t n_traj, const int32_t* traj, const int32_t* pos,
                         const int32_t* start, const float* logp_new, const float* logp_old,
                         const uint8_t* loss_mask, int64_t n_tokens, float eps_low, float eps_high,
                         float scale, float* grad_logp, float* loss, int64_t* n_trained, void* stream);

/* Static description of a status code. */
const char* hdl_status_string(int status);

/* Description of the calling thread's most recent failure, an argument
 * error or a HIP error ("" if the last call succeeded); thread-local. */
const char* hdl_last_hip_error(void);

/* ABI version of this library (increments on incompatible changes). */
int hdl_abi_version(void);

/*
 * Kernel timing for measurement tools.  While enabled, every
 * hdl_token_logprobs(_entropy) call brackets its fused lm-head kernel, every
 * hdl_token_logprobs_backward call its gradient-mode and GEMM launches, and
 * every selection call its kernel, with HIP events on the caller's stream.  hdl_profile_read waits for those
 * events, returns the summed time of the fused kernel's launches in
 * milliseconds and their number since the last read, and resets that tally.
 * Disabled by default; enabling adds two event records per timed launch.
 * The tallies are shared by all threads of the process.
 */
int hdl_profile_enable(int on);
int hdl_profile_read(double* total_ms, int64_t* launches);

/* The same tally for one kind of kernel: the fused lm-head kernel (what
 * hdl_profile_read reports), its gradient mode in hdl_token_logprobs_backward,
 * the backward pass's GEMMs, or the per-root selection kernel of
 * hdl_select_branch_points, hdl_select_top_k and hdl_select_constrained. */
enum { HDL_PROFILE_LMHEAD = 0, HDL_PROFILE_GRAD = 1, HDL_PROFILE_GEMM = 2, HDL_PROFILE_SELECT = 3 };
int hdl_profile_read_kind(int kind, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* HDL_H_ */
