/*
 * grpo.h -- C ABI of libgrpo, the MI355X (gfx950) GRPO scoring + loss library.
 *
 * The library computes, for every sampled rollout token, the policy
 * log-probability under an LM head and the GRPO objective of AutoTriton
 * (Sec. 3.3, Eq. 1 with the group advantage of Eq. 2), together with the
 * gradients of the loss with respect to the final hidden states and the
 * LM-head weight, without ever storing the N x V logits.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is caller-owned, contiguous DEVICE memory unless
 *    stated otherwise. The library never allocates or frees device memory:
 *    temporary storage is the caller's workspace, sized by
 *    grpo_workspace_bytes().
 *  - Work is enqueued on `stream` (NULL = the legacy default stream) and is
 *    asynchronous; no call synchronises except grpo_check_error().
 *  - Arguments are validated on the host before anything is launched. On
 *    error nothing is enqueued and a nonzero grpo_status is returned.
 *    No C++ exception crosses this interface.
 *  - Errors that depend on device data (a token id outside [0, V), a
 *    malformed cu_seqlens) cannot be seen on the host. Kernels then record
 *    a flag in the workspace and skip the offending item instead of
 *    trapping; grpo_check_error() reads the flag back. Each call clears the
 *    flags of its workspace when it starts, so the check reports the most
 *    recent call that used that workspace.
 *  - Layouts are row-major: hidden [N, H], weight [V, H] (the nn.Linear
 *    layout, one row per vocabulary entry), grad_hidden [N, H],
 *    grad_weight [V, H].
 *  - A "row" is one token position. Rollout b owns rows
 *    cu_seqlens[b] .. cu_seqlens[b+1]-1; a padded batch of B rollouts of
 *    length T uses cu_seqlens[b] = b*T. A row takes part iff its mask byte
 *    is nonzero (mask == NULL: every row). Outputs of masked rows are 0.
 *  - Calls on distinct streams are thread-safe. Calls that share a
 *    workspace must be ordered by the caller.
 *  - Workspace size. max_valid (0 = N) bounds the number of valid rows a
 *    call will see: the token-indexed scratch is sized for it (a ragged
 *    batch with half its rows masked needs about half). The capacity is
 *    max_valid rounded up to a multiple of 256; a call whose mask has more
 *    valid rows than that records GRPO_ERR_CAPACITY and treats no row as
 *    valid (all outputs as for masked rows). dz_budget (0 = 16 GiB) bounds
 *    the bytes of the logits-gradient chunks of the backward pass; a smaller
 *    budget means narrower vocabulary chunks and more passes over the fp32
 *    dL/dhidden accumulator: the gradients are then summed in another
 *    grouping (equal up to fp32 rounding; the same arguments always give the
 *    same bits). Pass the same values to grpo_workspace_bytes and to the
 *    call, with GRPO_WS_TILED_WEIGHT in the op when the call is given a
 *    tiled weight (grpo_tile_weight): the workspace then holds no copy of W.
 */
#ifndef GRPO_H_
#define GRPO_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t;

typedef enum grpo_status {
  GRPO_OK = 0,
  GRPO_ERR_NULL = 1,        /* a required pointer is NULL */
  GRPO_ERR_SHAPE = 2,       /* a size is out of range or inconsistent */
  GRPO_ERR_DTYPE = 3,       /* unknown or unsupported dtype */
  GRPO_ERR_PARAM = 4,       /* a hyper-parameter is out of range */
  GRPO_ERR_ALIGN = 5,       /* a pointer lacks the required alignment */
  GRPO_ERR_WORKSPACE = 6,   /* workspace NULL, misaligned or too small */
  GRPO_ERR_DEVICE = 7,      /* no usable gfx950 device */
  GRPO_ERR_HIP = 8,         /* a HIP runtime call failed */
  GRPO_ERR_TOKEN_RANGE = 9, /* (device) a token id was outside [0, V) */
  GRPO_ERR_SEQLENS = 10,    /* (device) cu_seqlens not monotone from 0 to N */
  GRPO_ERR_CAPACITY = 11    /* (device) more valid rows than the max_valid capacity */
} grpo_status;

/* GRPO_BF16 is the production path (MFMA contractions). GRPO_F32 is an
 * exact-arithmetic parity path for small problems (e.g. H = 64, V = 1000):
 * plain fp32 FMA loops, no matrix cores, H <= 8192, and dL/dweight re-reads
 * every valid hidden row once per vocabulary row (O(V * N * H) loads), so
 * its cost grows far faster than the bf16 path's. */
typedef enum grpo_dtype {
  GRPO_F32 = 0, /* IEEE binary32 */
  GRPO_BF16 = 1 /* bfloat16; fp32 accumulation, round-to-nearest-even stores */
} grpo_dtype;

/* How the per-token terms of Eq. 1 are averaged into the loss. */
typedef enum grpo_agg {
  /* Eq. 1 as written: mean over the tokens of each rollout (1/|o_i|), then
   * mean over all B = P*G rollouts. Weight of a token of rollout b is
   * 1 / (B * |o_b|); an empty rollout adds 0 but still counts in B. */
  GRPO_AGG_SEQ_MEAN = 0,
  /* One global mean over all valid tokens: weight 1 / sum_b |o_b|. */
  GRPO_AGG_TOKEN_MEAN = 1
} grpo_agg;

/* Operation selector for grpo_workspace_bytes(). */
typedef enum grpo_op {
  GRPO_OP_LOGPROB_FWD = 0,
  GRPO_OP_LOSS_FWD_BWD = 1,
  GRPO_OP_SFT_FWD_BWD = 2
} grpo_op;

/* OR-ed into the op of grpo_workspace_bytes for a bf16 call that will be
 * given weight_tiled: the workspace then holds no tiled copy of the weight. */
#define GRPO_WS_TILED_WEIGHT 0x100

/*
 * group_advantages -- Eq. 2 of AutoTriton Sec. 3.3: the advantage of
 * rollout i of a prompt is (r_i - mean) / (std + std_eps), where mean and
 * std are taken over the G = group_size rollouts of the same prompt (the
 * paper's set {o_i}, i = 1..G, that the rollouts are sampled as). The paper
 * fixes neither the std convention nor an epsilon: unbiased_std != 0 selects
 * the (G-1) estimate, 0 the population one. If all G rewards of a group are
 * equal the advantages are exactly 0.
 *
 *   rewards  [num_prompts * group_size] fp32, prompt-major (the G rollouts
 *            of one prompt contiguous). Device.
 *   adv      [num_prompts * group_size] fp32 output, same order. Device.
 * Requires 1 <= num_prompts <= 4 * (2^24 - 1) (one wave per prompt; the
 * grid stays below 2^32 threads), group_size >= 2, std_eps >= 0 (and finite).
 * Computed in fp32 with a fixed reduction order (bitwise reproducible).
 */
grpo_status group_advantages(const float* rewards, int64_t num_prompts, int32_t group_size,
                             float std_eps, int32_t unbiased_std, float* adv,
                             hipStream_t stream);

/*
 * grpo_pack_valid -- the token counts |o_b| of Eq. 1 and the compacted list
 * of rows that take part (mask set), in increasing row order.
 *
 *   mask        [N] uint8, or NULL (every row valid). Device.
 *   cu_seqlens  [num_seqs + 1] int64 row offsets, cu[0] = 0, cu[B] = N,
 *               non-decreasing. Device.
 *   rows        [N] int32 output: the first *num_valid entries are the valid
 *               rows; the rest are left unspecified. Device.
 *   counts      [num_seqs] int32 output: |o_b|. Device.
 *   num_valid   [1] int32 output. Device.
 *   workspace   at least grpo_workspace_bytes(GRPO_OP_LOGPROB_FWD, ...) for
 *               the same N (only its small header is used). Device.
 * Integer results are exact. Requires 1 <= N < 2^31.
 */
grpo_status grpo_pack_valid(const uint8_t* mask, const int64_t* cu_seqlens, int64_t num_seqs,
                            int64_t N, int32_t* rows, int32_t* counts, int32_t* num_valid,
                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * grpo_pack_valid_static -- grpo_pack_valid for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same outputs, with the scratch (error words,
 * valid count, per-rollout offsets) in a static device array of the library
 * instead of a caller workspace. No allocation of any kind.
 *   mask, cu_seqlens, num_seqs, N, rows, counts, num_valid  as grpo_pack_valid.
 *   error_out  [1] int32 output or NULL: GRPO_ERR_SEQLENS if cu_seqlens was
 *              not monotone from 0 to N (those rollouts count as empty), else
 *              0. Device.
 * Limit: num_seqs <= 2^20 (GRPO_ERR_WORKSPACE above). Every call on one GPU
 * shares that GPU's array: calls that overlap on a GPU (other streams or
 * threads) race and must be ordered by the caller.
 */
grpo_status grpo_pack_valid_static(const uint8_t* mask, const int64_t* cu_seqlens,
                                   int64_t num_seqs, int64_t N, int32_t* rows, int32_t* counts,
                                   int32_t* num_valid, int32_t* error_out, hipStream_t stream);

/*
 * grpo_logprob_fwd -- the policy probability inside the ratio of Eq. 1,
 * pi_theta(o_t | q, o_<t): for each valid row t,
 *   z_{t,v} = <hidden_t, weight_v>              (all v in [0, V))
 *   lse_t   = log sum_v exp z_{t,v}
 *   logp_t  = z_{t, tokens_t} - lse_t
 * The logits are reduced tile by tile (online max / sum-exp) and never
 * stored.
 *
 *   dt        GRPO_BF16 (hidden, weight bf16; MFMA, fp32 accumulation) or
 *             GRPO_F32 (fp32 throughout).
 *   hidden    [N, H] dt. Device.       weight [V, H] dt. Device.
 *   weight_tiled  NULL, or grpo_tile_weight's output for this weight (bf16
 *             only): the call reads it instead of tiling weight into the
 *             workspace (see grpo_tile_weight). Device, 256-byte aligned.
 *   tokens    [N] int64 sampled ids.   mask   [N] uint8 or NULL.
 *   logp, lse [N] fp32 outputs (0 on masked rows). Either may be NULL.
 *   workspace >= grpo_workspace_bytes(GRPO_OP_LOGPROB_FWD, dt, N, H, V, 1,
 *             max_valid, 0) (with GRPO_WS_TILED_WEIGHT in the op when
 *             weight_tiled is given), 256-byte aligned.
 *   max_valid 0 (= N) or the most valid rows the mask will have, <= N.
 * Requires N, H, V >= 1, N < 2^31, V < 2^31, H < 2^20; bf16 also needs
 * H % 8 == 0, (ceil(V/256) + 32) * ceil(N/256) < 2^31 and 16-byte aligned
 * hidden/weight; fp32 needs H <= 8192. fp32 arrays are 4-byte aligned.
 */
grpo_status grpo_logprob_fwd(grpo_dtype dt, const void* hidden, const void* weight,
                             const void* weight_tiled, const int64_t* tokens,
                             const uint8_t* mask, int64_t N, int64_t H, int64_t V, float* logp,
                             float* lse, void* workspace, size_t workspace_bytes,
                             int64_t max_valid, hipStream_t stream);

/*
 * grpo_loss_fwd_bwd -- loss = -J of Eq. 1 (AutoTriton Sec. 3.3) and its
 * gradients. For each valid row t of rollout b, with logp_t as in
 * grpo_logprob_fwd:
 *   rho   = exp(logp_t - old_logp_t)                       (pi_theta / pi_theta_old)
 *   pg    = -min(rho * A_b, clip(rho, 1-clip_eps, 1+clip_eps) * A_b)
 *   kl    = exp(ref_logp_t - logp_t) - (ref_logp_t - logp_t) - 1      (k3 estimator)
 *   ell_t = pg + beta * kl
 *   loss  = sum_b c_b * sum_{valid t in b} ell_t     (c_b from `agg`, see grpo_agg)
 * and the exact gradients dL/dhidden, dL/dweight through the log-softmax.
 * A tie rho*A == clip(rho)*A takes the unclipped branch; the clipped branch
 * has zero slope. With bf16 the logits gradient g_t (1[v = y_t] - p_tv) enters
 * the matrix-core products as -g_t p_tv rounded to bf16, and the sampled id's
 * g_t is applied in fp32 (to dL/dhidden_t as g_t * weight_{y_t}, to
 * dL/dweight_{y_t} as a fixed-order sum of g_t * hidden_t), so the gradients'
 * error is that of the bf16 rounding of the small -g p terms.
 *
 *   dt, hidden, weight, weight_tiled, tokens, mask, N, H, V
 *              as grpo_logprob_fwd (weight is read as well: the sampled
 *              ids' rows).
 *   cu_seqlens [num_seqs + 1] int64. Device.
 *   old_logp   [N] fp32: log pi_theta_old of each row. Device.
 *   ref_logp   [N] fp32: log pi_ref of each row; may be NULL iff beta == 0.
 *   adv        [num_seqs] fp32: A_b (e.g. from group_advantages). Device.
 *   clip_eps   in (0, 1); beta >= 0.
 *   lse_in     [N] fp32 or NULL: the row's log-sum-exp from an earlier
 *              grpo_logprob_fwd on the same hidden/weight; when given, the
 *              forward vocabulary pass is skipped.
 * Outputs (device, any may be NULL except loss):
 *   loss        [1] fp32, reduced in a fixed order (bitwise reproducible).
 *   logp_out, lse_out, token_loss (ell_t), dlogp (dL/dlogp_t)  [N] fp32.
 *   clip_flag   [N] uint8: 1 where the clipped branch was taken.
 *   grad_hidden [N, H] of grad_hidden_dt (GRPO_F32 or GRPO_BF16; bf16 needs
 *               dt == GRPO_BF16). Zero rows where masked.
 *   grad_weight [V, H] fp32: overwritten, or added to when
 *               accumulate_grad_weight != 0.
 * workspace >= grpo_workspace_bytes(GRPO_OP_LOSS_FWD_BWD, dt, N, H, V, num_seqs,
 * max_valid, dz_budget) (see the workspace-size convention above; with
 * GRPO_WS_TILED_WEIGHT in the op when weight_tiled is given).
 * Sizes as grpo_logprob_fwd, and for bf16 N <= 2^22 (4,194,304 rows per call;
 * larger batches are split by the caller, accumulating grad_weight).
 */
grpo_status grpo_loss_fwd_bwd(grpo_dtype dt, const void* hidden, const void* weight,
                              const void* weight_tiled, const int64_t* tokens,
                              const uint8_t* mask, const int64_t* cu_seqlens,
                              int64_t num_seqs, int64_t N, int64_t H, int64_t V,
                              const float* old_logp, const float* ref_logp,
                              const float* adv, float clip_eps, float beta, grpo_agg agg,
                              const float* lse_in, float* loss, float* logp_out, float* lse_out,
                              float* token_loss, float* dlogp, uint8_t* clip_flag,
                              void* grad_hidden, grpo_dtype grad_hidden_dt, float* grad_weight,
                              int32_t accumulate_grad_weight, void* workspace,
                              size_t workspace_bytes, int64_t max_valid, size_t dz_budget,
                              hipStream_t stream);

/*
 * sft_ce_fwd_bwd -- the supervised fine-tuning stage that precedes GRPO
 * (AutoTriton Sec. 3.2; sequences of up to 16,384 tokens, Sec. 4.1): the
 * next-token cross-entropy of the LM head, averaged over the supervised
 * tokens, and its gradients, again without storing the logits:
 *   loss = -(1 / n_valid) * sum_{valid t} logp_t      (0 when n_valid = 0)
 * with logp_t as in grpo_logprob_fwd (tokens_t is the target id of row t;
 * the caller shifts labels). dL/dlogp_t = -1 / n_valid, and dL/dhidden,
 * dL/dweight follow through the log-softmax exactly as in grpo_loss_fwd_bwd.
 *
 *   dt, hidden, weight, weight_tiled, tokens, mask, N, H, V
 *               as grpo_loss_fwd_bwd (mask marks the supervised rows, e.g.
 *               the response tokens).
 *   loss        [1] fp32 output, fixed-order reduction. Device.
 *   logp_out    [N] fp32 or NULL (0 on masked rows). Device.
 *   grad_hidden, grad_hidden_dt, grad_weight, accumulate_grad_weight
 *               as grpo_loss_fwd_bwd (either gradient may be NULL).
 * workspace >= grpo_workspace_bytes(GRPO_OP_SFT_FWD_BWD, dt, N, H, V, 1, max_valid,
 * dz_budget) (GRPO_WS_TILED_WEIGHT in the op when weight_tiled is given).
 * Sizes and errors as grpo_loss_fwd_bwd (a token id outside [0, V) sets the flag that
 * grpo_check_error reports).
 */
grpo_status sft_ce_fwd_bwd(grpo_dtype dt, const void* hidden, const void* weight,
                           const void* weight_tiled, const int64_t* tokens, const uint8_t* mask,
                           int64_t N, int64_t H, int64_t V, float* loss, float* logp_out,
                           void* grad_hidden, grpo_dtype grad_hidden_dt, float* grad_weight,
                           int32_t accumulate_grad_weight, void* workspace,
                           size_t workspace_bytes, int64_t max_valid, size_t dz_budget,
                           hipStream_t stream);

/*
 * adamw_step -- the optimiser step applied to the LM head after its gradient
 * (AutoTriton Sec. 4.1 trains the actor with learning rate 1e-6; the
 * optimiser is not named, AdamW with decoupled weight decay is taken). For
 * every element, with t = step >= 1:
 *   m = beta1*m + (1-beta1)*g
 *   v = beta2*v + (1-beta2)*g^2
 *   w = w*(1 - lr*weight_decay) - (lr/(1-beta1^t)) * m / (sqrt(v)/sqrt(1-beta2^t) + eps)
 * in one HBM pass, in fp32, in place.
 *   weight, exp_avg, exp_avg_sq [n] fp32, device, read and overwritten;
 *   grad [n] fp32, device (e.g. grad_weight of grpo_loss_fwd_bwd);
 *   weight_bf16 [n] bf16 output (round to nearest even of the new weight), or
 *   NULL: the copy the next forward pass reads.
 * Requires n >= 1, step >= 1, 0 <= beta1, beta2 < 1, eps > 0, lr >= 0,
 * weight_decay >= 0 (finite); fp32 arrays 16-byte and the bf16 copy 8-byte
 * aligned. Enqueued on `stream`, no workspace.
 */
grpo_status adamw_step(float* weight, float* exp_avg, float* exp_avg_sq, const float* grad,
                       uint16_t* weight_bf16, int64_t n, float lr, float beta1, float beta2,
                       float eps, float weight_decay, int64_t step, hipStream_t stream);

/*
 * triton_rule_reward -- the reward of the RL stage (AutoTriton Sec. 3.3,
 * Eq. 3): R = 1 if is_Triton(completion) and test_passed, else 0; or, with
 * weighted = 1, R = rule_weight * is_Triton + exec_weight * test_passed (the
 * rule-based reward given alongside the execution reward, Sec. 4), in fp32.
 * is_Triton is the lexical rule Sec. 4 describes -- a function decorated
 * with @triton.jit -- and, with require_launch = 1, that function launched
 * as name[grid](...) somewhere in the completion (Sec. 4's hack of a kernel
 * that is never called). Exact rule: a decorator is "@triton.jit" with only
 * blanks (space, tab, CR) before it on its line and no identifier byte or "."
 * after it, optional balanced "(...)" arguments, then only blanks or a "#"
 * comment to the newline; blank, comment and other decorator lines may
 * follow; then a line "def NAME(" (blanks allowed around NAME). A launch is
 * NAME not preceded by an identifier byte, blanks, "[", a bracket-balanced
 * run, "]", blanks, "(". Strings and comments are not otherwise parsed.
 *   text        the completions' bytes, concatenated; 16-byte aligned.
 *               Device.
 *   text_bytes  bytes readable at text (>= 0); nothing beyond is read.
 *   offsets     [num_completions + 1] int64: completion b is
 *               text[offsets[b], offsets[b+1]); a decreasing pair, or one
 *               with an offset outside [0, text_bytes], counts as an empty
 *               completion. Device.
 *   test_passed [num_completions] u8, nonzero = the execution harness's
 *               tests passed (that harness is outside this library). Device.
 *   is_triton   [num_completions] u8 output (0/1). Device.
 *   reward      [num_completions] fp32 output, the input of
 *               group_advantages. Device.
 * Requires require_launch, weighted in {0, 1}, finite weights, text_bytes
 * >= 0. Enqueued on `stream`, no workspace; num_completions = 0 does nothing
 * (no pointer is read).
 */
grpo_status triton_rule_reward(const uint8_t* text, int64_t text_bytes, const int64_t* offsets,
                               int64_t num_completions, const uint8_t* test_passed,
                               int32_t require_launch, int32_t weighted, float rule_weight,
                               float exec_weight, uint8_t* is_triton, float* reward,
                               hipStream_t stream);

/* Bytes of workspace an operation needs for these sizes (0 if the sizes are
 * invalid). For GRPO_OP_LOGPROB_FWD and GRPO_OP_SFT_FWD_BWD pass
 * num_seqs = 1; max_valid and dz_budget as described under "Workspace size"
 * (dz_budget is ignored for GRPO_OP_LOGPROB_FWD). op may carry
 * GRPO_WS_TILED_WEIGHT (bf16 only). Host only. */
size_t grpo_workspace_bytes(grpo_op op, grpo_dtype dt, int64_t N, int64_t H, int64_t V,
                            int64_t num_seqs, int64_t max_valid, size_t dz_budget);

/*
 * grpo_tile_weight -- the LM head W [V, H] (bf16, row-major) in the tiled
 * layout that the bf16 scoring and gradient products of Eq. 1 read: 256-row
 * by 32-column blocks (16 KiB each), tile-row r's blocks at
 * (r * (ceil(H/32) + 1) + k) * 8192 elements, rows >= V and columns >= H zero.
 * grpo_logprob_fwd, grpo_loss_fwd_bwd and sft_ce_fwd_bwd tile W themselves
 * unless given this copy as weight_tiled, so a caller whose W stays fixed over
 * several calls (a frozen reference model, the policy over the micro-batches
 * of one optimiser step) tiles it once: 2 * V * H bytes read and written
 * (0.55 ms at V = 155136, H = 4096). The copy is only valid while W is
 * unchanged; the library cannot tell when it is stale.
 *   weight   [V, H] bf16, 16-byte aligned. Device.
 *   out      grpo_weight_tiled_bytes(V, H) bytes, 256-byte aligned. Device,
 *            caller-owned.
 * Requires 1 <= V < 2^31 - 256, 1 <= H < 2^20, H % 8 == 0. Errors:
 * GRPO_ERR_NULL, GRPO_ERR_SHAPE (also out_bytes too small), GRPO_ERR_ALIGN.
 * Enqueued on `stream`.
 */
size_t grpo_weight_tiled_bytes(int64_t V, int64_t H);
grpo_status grpo_tile_weight(const void* weight, int64_t V, int64_t H, void* out,
                             size_t out_bytes, hipStream_t stream);

/* Synchronises `stream`, then reads and clears the device error flags kept in
 * the workspace by the most recent call that used it. Returns GRPO_OK,
 * GRPO_ERR_SEQLENS, GRPO_ERR_TOKEN_RANGE or GRPO_ERR_CAPACITY (or
 * GRPO_ERR_HIP if a copy fails). */
grpo_status grpo_check_error(void* workspace, hipStream_t stream);

/* Static description of a status code. Never NULL. */
const char* grpo_status_string(grpo_status status);

/*
 * Kernel timing (for benchmarks). When enabled, every kernel launch is
 * bracketed by a pair of HIP events recorded on the launch stream, and
 * grpo_profile_query() reports, per kernel kind, the launch count and the
 * summed event time. Querying synchronises the recorded events. Disabled by
 * default; enabling costs two event records per launch.
 */
void grpo_profile_enable(int32_t on);
void grpo_profile_reset(void);
int32_t grpo_profile_num_kinds(void);
const char* grpo_profile_kind_name(int32_t kind);
grpo_status grpo_profile_query(int32_t kind, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* GRPO_H_ */
