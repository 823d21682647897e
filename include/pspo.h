/*
 * pspo.h -- C ABI of libpspo: the hot path of a PS-PPO policy update on one
 * AMD Instinct MI355X (gfx950).
 *
 * PS-PPO (prefix-sampling PPO) backpropagates only through a random prefix
 * t <= H of each completion and reweights every kept token by 1/xi_t, where
 * xi_t = Pr(H >= t | x) is a per-prompt survival table, so the truncated
 * update stays an unbiased estimate of the full one (Sec. 3.2, "Unbiased
 * Stochastic Truncation", the truncated estimator G-hat; App. B).  The three
 * calls below are the three steps of the update pass that Algorithm 1 lists
 * after the cutoff design: draw one cutoff per completion, keep the prefixes
 * (with their weights), and compute the reweighted clipped-ratio PPO loss
 * (Sec. 3.1) through the LM head together with its gradient.
 *
 * Conventions shared by every call
 *  - Pointers marked "device" must be device memory on the current HIP
 *    device; "host" pointers are host memory.  Sizes and scalars are by value.
 *  - The caller allocates and owns every buffer; the library never allocates
 *    or frees memory and keeps no mutable global state, so calls on distinct
 *    streams are independent (pspo_design_cutoffs_noalloc's static array is
 *    the one exception; see there).  Outputs must not alias inputs.
 *  - No call synchronises (outside debug mode) or records a memset, so every
 *    call can be captured into a HIP graph and replayed; a replay repeats the
 *    call with the arguments it was captured with (sizes included).  The
 *    first call on a device checks the device's architecture, and the first
 *    pspo_design_cutoffs_noalloc call looks up its array's address: make
 *    those first calls outside a capture.
 *  - Every call is asynchronous on `stream` (0 = the null stream) and returns
 *    a pspo_status.  Errors detectable from the arguments alone are returned
 *    before anything is enqueued (the thread-local pspo_last_error() says
 *    which argument).  Errors only the device can see (a target id outside
 *    [0, V), an invalid xi table, a capacity overflow) are OR-ed into the
 *    optional device word `err_flag` (PSPO_DEVERR_* bits); the call does not
 *    synchronise to report them.  A kernel launch that fails returns
 *    PSPO_ERR_HIP naming the kernel.
 *  - Debug mode: with the environment variable PSPO_DEBUG set (to anything
 *    but "" or "0"; read at every launch) every call synchronises its stream
 *    after each kernel and returns PSPO_ERR_HIP naming the kernel whose
 *    execution failed.  Results are the same bits as without it.
 *  - Tracing: each call opens a roctx range named after it while it enqueues
 *    its work (rocprofv3 --marker-trace shows it next to its kernels).
 *  - bf16 tensors are passed as their raw 16-bit patterns (uint16_t).
 *  - Rollouts are prompt-major: completion k of prompt p is r = p*K + k.
 */
#ifndef PSPO_H_
#define PSPO_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PSPO_OK = 0,
  PSPO_ERR_INVALID_ARG = 1,   /* null / misaligned pointer, negative size, bad scalar */
  PSPO_ERR_BAD_XI = 2,        /* survival table not in (0,1] or not non-increasing (host check) */
  PSPO_ERR_WORKSPACE = 3,     /* workspace smaller than pspo_loss_workspace_bytes() */
  PSPO_ERR_UNSUPPORTED = 4,   /* shape or device the kernels do not handle */
  PSPO_ERR_HIP = 5            /* a HIP runtime call failed */
} pspo_status;

/* Bits OR-ed into the optional device word err_flag. */
#define PSPO_DEVERR_TARGET   1  /* a target id outside [0, V); that token's loss and gradient are 0 */
#define PSPO_DEVERR_BAD_XI   2  /* a xi value outside (0,1] or an increase along t */
#define PSPO_DEVERR_CAPACITY 4  /* sum of cutoffs exceeds `capacity`; nothing past it is written */
#define PSPO_DEVERR_SEQ_ID   8  /* a seq_id outside [0, R); that token's loss and gradient are 0 */
#define PSPO_DEVERR_NONFINITE 16 /* pspo_loss_fwd_bwd: a non-finite lse, ratio, loss term or delta in a token
                                    whose loss term is computed (e.g. a NaN or Inf hidden row, head row, old
                                    log-prob or weight); the loss and gradients are then not finite either */

/* Flags of pspo_loss_fwd_bwd. */
#define PSPO_ACCUMULATE_DW   1u /* d_w_head += gradient instead of d_w_head = gradient */
#define PSPO_KEEP_LOGITS     4u /* opt-in trade of memory for matrix-core work: the forward keeps the
                                    logits of the first vocabulary chunk (Vc x N of them, as fp16 offsets
                                    from each 384-row tile's per-column maximum) and the backward converts
                                    them instead of recomputing that chunk's logit tiles.  The same loss,
                                    log-probs and stats (bitwise), gradients within ~1e-5 relative (the
                                    fp16 rounding of the kept offsets), a workspace larger by Vc x Npad x 2
                                    bytes.  Without it no logit is ever stored.  (Bit 2 is retired.) */

/* Human-readable name of a status code (static storage). */
const char* pspo_status_string(int status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* pspo_last_error(void);

/* Version of this ABI (incremented on any change of its calls). */
int pspo_abi_version(void);

/*
 * Host-side check of survival tables (Sec. 3.2: 1 >= xi_1 >= ... >= xi_T > 0).
 *  xi      host, float64 [xi_off[P]]: xi[xi_off[p] + t - 1] = xi_{p,t}, t = 1..T_p.
 *  xi_off  host, int64 [P+1], non-decreasing, xi_off[0] = 0.
 * Returns PSPO_OK, PSPO_ERR_BAD_XI or PSPO_ERR_INVALID_ARG.  Touches no GPU.
 */
int pspo_validate_xi_host(const double* xi, const int64_t* xi_off, int32_t P);

/*
 * Cutoff sampling: one independent cutoff per completion drawn from the
 * survival function xi of its prompt (Sec. 3.2, Pr(H >= t | x) = xi_t;
 * Algorithm 1, the cutoff-sampling step).
 *
 * The table is realised exactly on 32-bit uniforms: q_{p,0} = 2^32,
 * q_{p,t} = max(1, floor(xi_{p,t} * 2^32)); x_r is word 0 of
 * Philox4x32-10(counter = (r, 0, lo32(offset), hi32(offset)),
 * key = (lo32(seed), hi32(seed))) (Salmon et al., SC'11);
 * H_r = min(T_r, max{t in [0, T_p] : x_r < q_{p,t}}).  Hence
 * Pr(H_r >= t) = q_{p,t} / 2^32 for t <= T_r.
 *
 *  xi        device, float64 [xi_off[P]] survival tables (layout as above);
 *            T_p = xi_off[p+1] - xi_off[p] must be >= every T_r of prompt p.
 *  xi_off    device, int64 [P+1].
 *  lengths   device, int32 [P*K], T_r >= 0.
 *  seed, offset  the Philox key and the high half of the counter.
 *  cutoffs   device, int32 [P*K] out: H_r in [0, T_r].
 *  err_flag  device, int32 [1] or NULL: PSPO_DEVERR_BAD_XI if a table is invalid
 *            (the cutoffs are then still in [0, T_r] but not from the law above).
 * P = 0 or K = 0 is valid and enqueues nothing.
 */
int pspo_sample_cutoffs(const double* xi, const int64_t* xi_off, const int32_t* lengths,
                        int32_t P, int32_t K, uint64_t seed, uint64_t offset,
                        int32_t* cutoffs, int32_t* err_flag, hipStream_t stream);

/*
 * Prefix packing: keep tokens t <= H_r of every completion, concatenated in
 * rollout order (varlen layout), each with its weight 1/xi_t realised as
 * float32(2^32 / (double)q_{p,t}) (Sec. 3.2 / 3.3, the 1/xi_t factor of the
 * truncated estimator; Algorithm 1, the reweighting of token losses).
 *
 *  cutoffs, lengths  device, int32 [R], R = P*K <= 65535; a cutoff is clamped to
 *                    [0, min(T_r, T_p)] (its length and its prompt's table horizon).
 *  xi, xi_off        device, as in pspo_sample_cutoffs.
 *  capacity          host-known bound >= sum_r H_r (e.g. sum_r T_r); sizes the
 *                    per-token outputs.  Excess tokens raise PSPO_DEVERR_CAPACITY.
 *  target_full       device, int32 [sum T_r] or NULL: token ids of all completions.
 *  logp_old_full     device, float32 [sum T_r] or NULL: old-policy log-probs.
 *  hidden_full       device, bf16 bits [sum T_r, d] row-major or NULL (16-byte
 *                    aligned, d % 8 == 0): final hidden states of all tokens.
 *  cu_seqlens        device, int32 [R+1] out: cu[0] = 0, cu[r+1] = cu[r] + H_r.
 *  full_off          device, int32 [R+1] out: offsets of completions in the
 *                    unpacked arrays (exclusive scan of lengths).
 *  src_row, seq_id   device, int32 [capacity] out: packed row i = cu[r] + j
 *                    comes from unpacked row full_off[r] + j of completion r.
 *  weight            device, float32 [capacity] out.
 *  target, logp_old  device [capacity] out, gathered; may be NULL iff the
 *                    corresponding *_full input is NULL.
 *  hidden            device, bf16 bits [capacity, d] out, gathered; NULL iff
 *                    hidden_full is NULL.
 *  n_tokens          device, int32 [1] out: N = cu[R].
 *  err_flag          device, int32 [1] or NULL.
 */
int pspo_pack_prefixes(const int32_t* cutoffs, const int32_t* lengths,
                       const double* xi, const int64_t* xi_off, int32_t P, int32_t K,
                       int32_t capacity,
                       const int32_t* target_full, const float* logp_old_full,
                       const uint16_t* hidden_full, int32_t d,
                       int32_t* cu_seqlens, int32_t* full_off, int32_t* src_row,
                       int32_t* seq_id, float* weight, int32_t* target, float* logp_old,
                       uint16_t* hidden, int32_t* n_tokens, int32_t* err_flag,
                       hipStream_t stream);

/*
 * Bytes of device workspace pspo_loss_fwd_bwd needs for N tokens (host-only,
 * pure function of its arguments).
 */
size_t pspo_loss_workspace_bytes(int32_t N, int32_t d, int32_t V, uint32_t flags);

/*
 * Fused LM-head + prefix-weighted PPO loss, forward and backward.
 *
 * For every packed token i with hidden row h_i, target o_i, old log-prob
 * lold_i, weight c_i and completion r = seq_id[i] with advantage A_r:
 *   z_i   = W h_i                                  (App. D: LM-head logits, no bias)
 *   l_i   = z_{i,o_i} - logsumexp(z_i)             (App. D, first log-sum-exp)
 *   rho_i = exp(l_i - lold_i)                      (Sec. 3.1, importance ratio)
 *   s_i   = min(rho_i A, clip(rho_i, 1-eps_low, 1+eps_high) A)   (Sec. 3.1, PPO objective)
 *   loss  = -loss_scale * sum_i c_i s_i            (Sec. 3.2/3.3 truncated estimator, negated)
 * and the exact gradients of `loss`:
 *   delta_i = -loss_scale c_i mu_i rho_i A, mu_i = 1 iff the unclipped branch is active
 *             (A > 0 and rho <= 1+eps_high, or A < 0 and rho >= 1-eps_low);
 *   G_i     = delta_i (e_{o_i} - softmax(z_i))     (App. D: grad log p(o) = (e_o - p) h^T)
 *   d_hidden[i] = G_i W,   d_w_head = sum_i G_i^T h_i.
 * The [N, V] logits are never written to memory: the forward keeps per-token
 * softmax statistics only, and the backward recomputes the logit tiles one
 * vocabulary chunk at a time.  G is applied in two parts: -delta_i p_i as one
 * chunk of bf16 values at a time (in two layouts) through the matrix cores,
 * and the one-hot part delta_i e_{o_i} in float32 (d_hidden[i] += delta_i W[o_i];
 * d_w_head[v] += sum_{i : o_i = v} delta_i h_i, each row's terms summed in token
 * order), so the largest entry of each row of G is never rounded to bf16.
 * The chunk width is about Vb = 384 * 256 / gcd(ceil(d / 256), 256) rows: the
 * vocabulary (padded to 384) is split evenly into floor(V / Vb) chunks, or one
 * more when the remainder exceeds Vb / 4 (one chunk if V < Vb), each a
 * multiple of 384 rows; three chunks of 50688 rows at d = 3584, V = 152064.  Every
 * result is deterministic (no floating-point atomics).
 *
 *  hidden     device, bf16 bits [N, d] row-major (packed prefix tokens).
 *  w_head     device, bf16 bits [V, d] row-major.
 *  target     device, int32 [N]; logp_old, weight: device float32 [N];
 *  seq_id     device, int32 [N] in [0, R);  advantage: device float32 [R].
 *  N >= 0, R >= 1 if N > 0, V >= 1, d > 0 with d % 8 == 0.  All device
 *  pointers 16-byte aligned.  Size limits (PSPO_ERR_UNSUPPORTED beyond them):
 *  N rounded up to 768, V rounded up to 384, and d each at most 2097120
 *  (65535 x 32: the operand copies put 32-row blocks on the grid's y axis);
 *  device memory binds first (about 240 KB of workspace and buffers per
 *  token at d = 3584, V = 152064).
 *  eps_low, eps_high in [0, 1); loss_scale finite (e.g. 1/(P*K)).
 *  flags      PSPO_ACCUMULATE_DW | PSPO_KEEP_LOGITS or 0.
 *  loss       device, float64 [1] out.
 *  d_hidden   device, float32 [>= N rows, d] out (rows 0 .. N-1 written).
 *  d_w_head   device, float32 [V, d] out (or accumulated, see flags).
 *  logp_new   device, float32 [N] out, or NULL.  When NULL, the forward
 *             computes logits only for the tokens of completions with A != 0:
 *             a zero advantage makes a token's loss term and gradient exactly
 *             zero, and every other output is unchanged (bitwise).
 *  stats      device, float64 [5] out, or NULL: { loss_scale * sum_i |c_i s_i|,
 *             #tokens with A != 0 and mu = 0 (clipped), #tokens with A == 0,
 *             max_i c_i, #tokens with delta_i != 0 }.  Only the last group
 *             of tokens enters the backward products: every other token has
 *             delta_i = 0, hence a zero row of G, a zero d_hidden row and no
 *             d_w_head term, so skipping it is exact.
 *  err_flag   device, int32 [1] or NULL (PSPO_DEVERR_TARGET, PSPO_DEVERR_SEQ_ID,
 *             PSPO_DEVERR_NONFINITE).
 *  workspace  device, >= pspo_loss_workspace_bytes(N, d, V, flags) bytes,
 *             256-byte aligned; its contents on entry are ignored.
 * N = 0 is valid: loss = 0 and d_w_head is zeroed (unless accumulating).
 */
int pspo_loss_fwd_bwd(const uint16_t* hidden, const uint16_t* w_head, const int32_t* target,
                      const float* logp_old, const float* weight, const int32_t* seq_id,
                      const float* advantage, int32_t N, int32_t d, int32_t V, int32_t R,
                      float eps_low, float eps_high, float loss_scale, uint32_t flags,
                      double* loss, float* d_hidden, float* d_w_head, float* logp_new,
                      double* stats, int32_t* err_flag, void* workspace, size_t workspace_bytes,
                      hipStream_t stream);

/*
 * Bytes of device workspace pspo_score_proxy needs (host-only, pure function).
 */
size_t pspo_score_proxy_workspace_bytes(int32_t N, int32_t d, int32_t V);

/*
 * Output-head score proxy of the cutoff design, forward only (Sec. 3.3,
 * Eq. gamma_proxy; App. D, output-head score proxy).  Run under the old policy
 * over every completion token before the cutoff probabilities are designed.
 * For every row i with hidden state h_i, logits z_i = W h_i,
 * p_i = softmax(z_i) and generated token o_i:
 *   gamma_i = ||h_i||^2 ||e_{o_i} - p_i||^2 = ||h_i||^2 (1 - 2 p_i(o_i) + ||p_i||^2),
 * the squared Frobenius norm of grad_W log p_i(o_i) (App. D).  The kernels form
 * ||e_o - p||^2 from per-tile sums of exp(z - m) and exp(2 (z - m)) over the
 * non-target entries (the second reduction of App. D, split so that no term
 * cancels as p(o) -> 1).  The [N, V] logits are never written to memory.
 *
 *  hidden     device, bf16 bits [N, d] row-major; w_head: device, bf16 bits [V, d].
 *  target     device, int32 [N]: the generated token of each row.
 *  N >= 0, V >= 1, d > 0 with d % 8 == 0; device pointers 16-byte aligned.
 *  N rounded up to 256, V rounded up to 384, and d each at most 2097120
 *  (PSPO_ERR_UNSUPPORTED beyond).
 *  gamma      device, float32 [N] out.
 *  logp       device, float32 [N] out, or NULL: log p_i(o_i) (the old-policy
 *             log-probs the update later consumes).
 *  p_sq       device, float32 [N] out, or NULL: ||p_i||^2 = exp(l2 - 2 l1).
 *  err_flag   device, int32 [1] or NULL: PSPO_DEVERR_TARGET if a target lies
 *             outside [0, V); that row's outputs are NaN.
 *  workspace  device, >= pspo_score_proxy_workspace_bytes(N, d, V) bytes,
 *             256-byte aligned; contents on entry ignored.
 * N = 0 is valid and does nothing.
 */
int pspo_score_proxy(const uint16_t* hidden, const uint16_t* w_head, const int32_t* target,
                     int32_t N, int32_t d, int32_t V, float* gamma, float* logp, float* p_sq,
                     int32_t* err_flag, void* workspace, size_t workspace_bytes,
                     hipStream_t stream);

/* Variants of the cutoff design (Sec. 4 ablation: Optimized, Heuristic, Uniform, Time prior). */
enum {
  PSPO_DESIGN_OPTIMIZED = 0,
  PSPO_DESIGN_HEURISTIC = 1,
  PSPO_DESIGN_UNIFORM = 2,
  PSPO_DESIGN_TIME_PRIOR = 3
};

/*
 * Per-step weights of the cutoff design ("Computing xi", Algorithm 1; Sec. 3.3,
 * Eq. wtilde_factorized1; App. E).  For prompt p (completions r = pK+k,
 * k < K, lengths T_r) and step t = 1..T_p (T_p = max_k T_{pK+k}), over the
 * n_t completions with T_r >= t:
 *   gamma_bar_t = (1/n_t) sum_r gamma_r(t),
 *   u_t = 1/2 - 1/(2 n_t) || sum_{r succeeded} pi_r(.|t) - sum_{r failed} pi_r(.|t) ||_1,
 *   w_t = gamma_bar_t u_t,
 * i.e. App. E's 1/2 - 1/2 || p pibar_G - (1-p) pibar_B ||_1 with p, pibar_G and
 * pibar_B estimated from the completions alive at t.  pi_r(.|t) is the
 * old policy's next-token distribution at completion token t, known through its
 * top-k entries; the mass outside them counts as one coordinate shared by all
 * completions.  Float64 throughout.
 *
 *  gamma       device, float32 [S]: the score proxy of every completion token
 *              (pspo_score_proxy), completions laid out one after another.
 *  topk_ids    device, int32 [S, topk]; topk_logp: device, float32 [S, topk]:
 *              the top-k next-token ids and log-probs at each completion token
 *              (as the rollout engine reports them; distinct ids per row).
 *  lengths     device, int32 [P K]; full_off: device, int32 [P K + 1], the
 *              exclusive scan of lengths (as pspo_pack_prefixes writes it).
 *  rewards     device, float32 [P K]; a completion succeeded iff reward > 1/2.
 *  xi_off      device, int64 [P + 1]: the layout of the per-step outputs (the
 *              xi-table layout: xi_off[p+1] - xi_off[p] = T_p); total_T = xi_off[P]
 *              (host value, sizes the launch).
 *  1 <= K <= 64, topk >= 1, K * topk <= 256.
 *  w           device, float64 [total_T] out; gamma_bar, u: device, float64
 *              [total_T] out, or NULL.
 *  err_flag    PSPO_DEVERR_BAD_XI if some step of a table has no alive
 *              completion (the table is longer than the prompt's completions);
 *              w = NaN there.
 */
int pspo_design_weights(const float* gamma, const int32_t* topk_ids, const float* topk_logp,
                        int32_t topk, const int32_t* lengths, const int32_t* full_off,
                        const float* rewards, const int64_t* xi_off, int32_t P, int32_t K,
                        int64_t total_T, double* w, double* gamma_bar, double* u,
                        int32_t* err_flag, hipStream_t stream);

/* Bytes of device workspace pspo_design_cutoffs needs (host-only). */
size_t pspo_design_workspace_bytes(int64_t total_T);

/*
 * Cutoff survival tables from the per-step weights (Sec. 3.3, Eq. design_problem;
 * App. F).  Per prompt: minimise sum_t w_t / xi_t subject to
 * sum_t xi_t = budget (the expected prefix length) and 1 >= xi_1 >= ... >= xi_T > 0.
 * PSPO_DESIGN_OPTIMIZED: Pooling Adjacent Violators gives blocks with scores
 * s_m = sqrt(W_m / L_m) non-increasing (App. F); xi = min(1, kappa s_m) with the
 * saturated prefix at 1 and kappa spending the rest of the budget.
 * PSPO_DESIGN_HEURISTIC: min(1, budget sqrt(w_t) / sum_j sqrt(w_j)) followed by a
 * running minimum.  PSPO_DESIGN_UNIFORM: xi_t = (T - t + 1) / T (H uniform on
 * 1..T).  PSPO_DESIGN_TIME_PRIOR: xi_t = exp(-lambda (t - 1)).  If budget >= T
 * every xi is 1; if every weight is 0, xi = budget / T.  Every xi is floored at
 * 2^-32 (the sampler's resolution).  The result is a valid input of
 * pspo_sample_cutoffs.
 *
 *  w           device, float64 [total_T] (xi_off layout), finite and >= 0
 *              (else PSPO_DEVERR_BAD_XI and that prompt's table is NaN).
 *  xi_off      device, int64 [P + 1]; total_T = xi_off[P] (host value).
 *  budget      > 0.  lambda >= 0 (used by PSPO_DESIGN_TIME_PRIOR only).
 *  xi          device, float64 [total_T] out.
 *  workspace   device, >= pspo_design_workspace_bytes(total_T) bytes, 256-byte aligned.
 */
int pspo_design_cutoffs(const double* w, const int64_t* xi_off, int32_t P, int64_t total_T,
                        double budget, int32_t variant, double lambda, double* xi,
                        void* workspace, size_t workspace_bytes, int32_t* err_flag,
                        hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * survival tables as pspo_design_cutoffs, bitwise, with no workspace argument.
 * The PAV block stack lives in a static device array of 8 MiB that the library
 * holds on each GPU it runs on until the process ends, so total_T <= 2^19
 * (524288 steps); a larger total_T returns PSPO_ERR_UNSUPPORTED before
 * anything is enqueued.  The call allocates and frees nothing.  Every call on
 * one GPU shares that GPU's array: calls that overlap on one GPU (concurrent
 * streams or threads) race and must be ordered by the caller.  The array needs
 * no clearing between calls (the solve writes each entry before reading it).
 * Other arguments, conventions and errors as in pspo_design_cutoffs.
 */
int pspo_design_cutoffs_noalloc(const double* w, const int64_t* xi_off, int32_t P, int64_t total_T,
                                double budget, int32_t variant, double lambda, double* xi,
                                int32_t* err_flag, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Measurement entry points.  Not steps of the method: they exist so that a
 * benchmark can time each matrix-core product of a call with HIP events on
 * the call's own stream, and report the sustained matrix-core rate next to
 * the products' achieved rate.
 * ------------------------------------------------------------------------ */

/* Product kinds of the per-product timing (index of pspo_timing_stop's arrays). */
enum {
  PSPO_TIME_FORWARD = 0,      /* pspo_loss_fwd_bwd: the forward logit product (all its launches)     */
  PSPO_TIME_LOGIT_GRAD = 1,   /* pspo_loss_fwd_bwd: one vocabulary chunk's logit-gradient product
                                 (or, with PSPO_KEEP_LOGITS, the kept chunk's conversion)            */
  PSPO_TIME_DW = 2,           /* pspo_loss_fwd_bwd: one chunk's dW product with its K-split tail      */
  PSPO_TIME_DH = 3,           /* pspo_loss_fwd_bwd: one chunk's dH product with its K-split tail      */
  PSPO_TIME_PROXY = 4,        /* pspo_score_proxy: the score-proxy logit product (all its launches)  */
  PSPO_TIMED_KINDS = 5
};

/*
 * Starts per-product timing on the calling thread: until pspo_timing_stop,
 * each pspo_loss_fwd_bwd and pspo_score_proxy call made on this thread records
 * a pair of HIP events on its stream around each of its matrix-core products
 * (one record per product and chunk, as listed above), for the first
 * `max_records` records; later products are not timed.  The events are
 * created here (2 * max_records hipEventCreate), so start outside any graph
 * capture.  The recording adds two event records per product and no
 * synchronisation.
 *  max_records  1 .. 2^20.
 * Errors: PSPO_ERR_INVALID_ARG if timing is already started on this thread
 * or max_records is out of range; PSPO_ERR_HIP if an event cannot be created.
 */
int pspo_timing_start(int32_t max_records);

/*
 * Stops the timing started on this thread: waits for every recorded event and
 * returns, per product kind, the summed elapsed milliseconds and the number
 * of records, then destroys the events.
 *  ms     host, float64 [PSPO_TIMED_KINDS], written.
 *  count  host, int32 [PSPO_TIMED_KINDS], written.
 * Errors: PSPO_ERR_INVALID_ARG if timing is not started on this thread, or
 * if a pointer is NULL; PSPO_ERR_HIP if an event wait fails.  Once timing was
 * started, the call ends it whatever it returns (the events are destroyed).
 */
int pspo_timing_stop(double* ms, int32_t* count);

/*
 * `blocks` work-groups of 256 threads each run `iters` rounds of 16
 * independent v_mfma_f32_16x16x32_bf16 per wave (the block form and tied
 * accumulators of the loss products, random bf16 operands alternating between
 * consecutive MFMAs), with no memory traffic, so that a caller timing it with
 * stream events gets the sustained bf16 matrix-core rate:
 * blocks * 4 * iters * 16 * 16384 flops.
 *  iters, blocks  >= 1.
 *  out            device, float32 [blocks * 256], written (values meaningless).
 */
int pspo_mfma_loop(int32_t iters, int32_t blocks, float* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PSPO_H_ */
