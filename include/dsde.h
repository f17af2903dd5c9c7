/*
 * dsde.h -- C ABI of the DSDE speculative-verification hot path on MI355X.
 *
 * DSDE (arXiv 2509.01083) verifies, in one batched step, a ragged set of
 * drafted tokens: sequence b proposes SL_b tokens (its own speculation length,
 * Sec. 3.2 "Ragged Q"); the target model scores SL_b + 1 positions and the draft
 * model SL_b.  This library computes, from the two models' logits:
 *   - for every drafted position, the tempered softmaxes p (target) and
 *     q (draft) and the per-token KL(p || q) used by the SL adapter (Sec. 3.1.2);
 *   - the speculative-sampling acceptance scan (accept while u < min(1, p/q)),
 *     the draw from the normalised residual max(0, p - q) at the first
 *     rejection, or the bonus token from the extra target row when every drafted
 *     token is accepted (Secs. 2.1 and 3.2);
 *   - the KLD stability signal: mu_KLD,last, the recency-weighted mean and
 *     variance over a short and a long window, WVIR and SF (Eqs. 3-7);
 *   - the next speculation length per sequence (Eqs. 2 and 8) under the batch
 *     cap SL_cap = mean of the predicted lengths (Sec. 3.3, Eqs. 9-11).
 *
 * Conventions (every function):
 *   - Every array pointer is a caller-owned DEVICE buffer (e.g. a tensor's data
 *     pointer), contiguous, of the stated shape and type.  The library never
 *     allocates, frees or synchronises on these paths; work is enqueued
 *     asynchronously on `stream` (a hipStream_t; NULL means the null stream).
 *   - Scratch space comes from a caller workspace sized by
 *     dsde_verify_workspace_bytes.  Calls with distinct workspaces and outputs
 *     may run concurrently on different streams.
 *   - Host-side argument errors are detected before any HIP call and return
 *     DSDE_INVALID_ARG or DSDE_WORKSPACE_TOO_SMALL; nothing is enqueued then.
 *     DSDE_DEVICE_ERROR reports a failed kernel launch.
 *   - Data errors found on the device are reported per sequence in seq_err[b]
 *     (bits DSDE_ERR_*).  A flagged sequence gets defined outputs: accepted = 0
 *     and every token = pad_id; kld = NaN at its positions when its drafted
 *     pairs could not be evaluated (a bad token, temperature, uniform or a
 *     non-finite logit in a drafted pair; not written when the layout itself is
 *     invalid).  A non-finite bonus row only withholds the token: the KLD values
 *     stay.  NaN KLD makes the signal NaN, and such sequences are left out of
 *     the cap.
 *   - Finite logits are assumed to satisfy |z| <= 2^64 (any real logit does);
 *     larger magnitudes are outside the contract.
 *
 * Packed ragged layout (no padding rows): with N = sum_b SL_b and
 * cu_sl[b] = SL_0 + ... + SL_{b-1} (cu_sl[0] = 0, cu_sl[B] = N),
 *   drafted position (b, j), j < SL_b  ->  index cu_sl[b] + j      in [0, N)
 *   its target row                      ->  cu_sl[b] + b + j        in [0, N+B)
 *   the bonus row of b                  ->  cu_sl[b] + b + SL_b
 *   its draft row                       ->  cu_sl[b] + j            in [0, N)
 * Logits are row-major [rows, V], fp32 or bf16.
 */
#ifndef DSDE_H_
#define DSDE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DSDE_ABI_VERSION 3

/* status codes */
#define DSDE_OK 0
#define DSDE_INVALID_ARG 1
#define DSDE_WORKSPACE_TOO_SMALL 2
#define DSDE_DEVICE_ERROR 3

/* logit element types */
#define DSDE_FP32 0
#define DSDE_BF16 1

/* per-sequence device error bits */
#define DSDE_ERR_LAYOUT 1u   /* SL_b outside [0, k_max], or cu_sl not the prefix sums of sl with cu_sl[B] = N */
#define DSDE_ERR_TOKEN 2u    /* a drafted token outside [0, V) */
#define DSDE_ERR_LOGIT 4u    /* NaN or +-inf in a row the step reads (every drafted pair; the bonus row
                                only when it is sampled) */
#define DSDE_ERR_TEMP 8u     /* temperature neither 0 nor in [2^-16, 2^16] */
#define DSDE_ERR_UNIFORM 16u /* a uniform outside [0, 1) */
#define DSDE_ERR_SIGNAL 32u  /* non-finite KLD, SF, WVIR or SL_max, or SL_max < sl_min */
#define DSDE_ERR_STATE 64u   /* ring head outside [0, W) or count outside [0, W] */

/* Largest supported speculation length bound (one wavefront lane per drafted position). */
#define DSDE_MAX_K 63
/* Largest supported vocabulary (512 chunks of 8192 logits; the draw keeps one
 * total per chunk on chip). */
#define DSDE_MAX_VOCAB 4194304

/* The ABI version this library implements (DSDE_ABI_VERSION). */
int32_t dsde_abi_version(void);

/* A static description of a status code; never NULL. */
const char *dsde_status_string(int32_t status);

/* Workspace bytes dsde_verify needs for B sequences, N drafted positions,
 * vocabulary V and speculation bound k_max; 0 when the sizes are invalid. */
size_t dsde_verify_workspace_bytes(int32_t B, int64_t N, int64_t V, int32_t k_max);

/*
 * One batched verification step (speculative sampling, Sec. 2.1; ragged
 * per-sequence lengths and the bonus/pad handling of Sec. 3.2; per-token KLD of
 * Sec. 3.1.2).
 *
 *   target_logits [N+B, V]  dtype       target rows in the packed layout above
 *   draft_logits  [N, V]    dtype       draft rows (may be NULL when N = 0)
 *   dtype                               DSDE_FP32 or DSDE_BF16
 *   V, B, N, k_max                      vocabulary, sequences, drafted positions, SL bound
 *                                       (1 <= V <= DSDE_MAX_VOCAB, B >= 1, 0 <= N <= B*k_max,
 *                                        0 <= k_max <= DSDE_MAX_K)
 *   sl [B], cu_sl [B+1]     int32       per-sequence SL and its exclusive prefix sums
 *   draft_tokens [N]        int32       the drafted token at each position
 *   temperature [B]         float       per-sequence temperature T_b: in [2^-16, 2^16] for
 *                                       speculative sampling with p = softmax(z_target / T_b),
 *                                       q = softmax(z_draft / T_b); T_b = 0 selects greedy
 *                                       verification (below); anything else is DSDE_ERR_TEMP
 *   u_acc [N]               float       acceptance uniforms in [0, 1), one per position
 *   u_res [B]               float       draw uniforms in [0, 1), one per sequence
 *   pad_id                              token written into unused slots
 * Outputs:
 *   accepted [B]            int32       a_b: number of leading drafted tokens accepted
 *   tokens [B, k_max+1]     int32       x_0..x_{a_b-1}, the drawn token, then pad_id
 *   kld [N]                 float       KL(p || q) in nats per drafted position (>= 0)
 *   seq_err [B]             uint32      DSDE_ERR_* bits per sequence (0 when fine)
 *   row_lse [N, 2]          double      optional (may be NULL): natural-log normalisers
 *                                       log sum_v exp(z_v / T_b) of the target and draft rows
 *   draft_entropy [N]       float       optional (may be NULL): H(q) = -sum_v q_v ln q_v of
 *                                       each drafted position's draft distribution (nats),
 *                                       the draft-entropy signal of Sec. 4.2 / Table 2;
 *                                       NULL also skips its accumulation in the statistics
 *                                       pass (every other output is unchanged, bit for bit)
 * The draw walks token ids in ascending order and returns the smallest id whose
 * cumulative weight exceeds u_res[b] times the total weight.  Acceptance is
 * evaluated as u < p(x)/q(x) in double precision.
 * Greedy verification (T_b = 0; the temperature-0.0 setting of Sec. 4.2): a
 * drafted token is accepted iff it is the argmax of its target row (the
 * smallest token id among equal maxima), the argmax of the first rejected row
 * or of the bonus row is emitted, u_acc and u_res of the sequence are not read
 * for decisions (nor checked), and kld and row_lse are taken at T = 1.
 */
int32_t dsde_verify(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                    int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl,
                    const int32_t *draft_tokens, const float *temperature, const float *u_acc,
                    const float *u_res, int32_t pad_id, int32_t *accepted, int32_t *tokens, float *kld,
                    uint32_t *seq_err, double *row_lse, float *draft_entropy, void *workspace,
                    size_t workspace_bytes, void *stream);

/*
 * KLD stability signal (Sec. 3.1.2, Eqs. 3-7).
 *
 * For each sequence: if SL_b > 0, mu_last = mean of kld over its SL_b positions
 * and it is pushed into the sequence's ring (hist[b, head[b]] = mu_last,
 * head = (head + 1) mod W, count = min(count + 1, W)); if SL_b = 0 nothing is
 * pushed and mu_last is the newest entry (0 for an empty ring).  Then, over the
 * n_s = min(n_short, count) and n_l = min(n_long, count) newest entries h_1..h_n
 * (h_1 newest) with weights alpha_i = delta^(i-1):
 *   mu_w = sum alpha_i h_i / sum alpha_i,  Var_w = sum alpha_i (h_i - mu_w)^2 / sum alpha_i
 *   WVIR = Var_s / Var_l (Eq. 4),          SF = exp(2 mu_last) - 1.
 * The sums are taken over h_i - h_1 (Var_w does not change under a common
 * shift), so a window of equal entries has a variance of exactly 0.  Where
 * Var_l = 0 (the long window holds one value; its short window is constant
 * too) eps replaces it in the quotient, giving WVIR = 0.  An empty window
 * has variance 0.
 *
 *   B, N                     sequences and drafted positions (as in dsde_verify)
 *   sl [B], cu_sl [B+1]      int32   as in dsde_verify
 *   kld [N]                  float   per-token KLD (dsde_verify's output)
 *   hist [B, W]              float   ring of per-step mean KLD (in/out)
 *   head [B], count [B]      int32   next write slot, entries held (in/out)
 *   W                                ring capacity (>= 1)
 *   n_short, n_long                  window sizes, 1 <= n_short <= n_long (paper: 10, 30)
 *   delta                            recency decay in (0, 1] (paper: 0.85)
 *   eps                              > 0 and finite: divisor of WVIR where Var_l = 0 (1e-6)
 * Outputs [B] float: mu_last, var_short, var_long, wvir, sf; seq_err [B] uint32
 * (DSDE_ERR_LAYOUT, DSDE_ERR_SIGNAL, DSDE_ERR_STATE; a flagged ring is left unchanged).
 */
int32_t dsde_kld_signal(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const float *kld,
                        float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short,
                        int32_t n_long, float delta, float eps, float *mu_last, float *var_short,
                        float *var_long, float *wvir, float *sf, uint32_t *seq_err, void *stream);

/*
 * Next speculation length with the batch cap (Eqs. 2 and 8; Sec. 3.3, Eqs. 9-11).
 *
 *   pen_b   = sf[b] * wvir[b]
 *   SL_hat_b = (1 - pen_b)(sl_max[b] - sl_min) + sl_min   if pen_b <= 1, else sl_min
 *   SL_cap  = mean of SL_hat over the sequences without an error (the MSE-optimal cap)
 *   sl_next[b] = clamp(floor(min(SL_hat_b, SL_cap) + 1/2), ceil(sl_min), sl_hi)
 * A sequence with a non-finite sf, wvir or sl_max, or sl_max < sl_min, gets
 * DSDE_ERR_SIGNAL, sl_hat = NaN and sl_next = ceil(sl_min); with no valid
 * sequence SL_cap is NaN.
 *
 * Then the per-sequence token budget of the policy interface (Sec. 3.2: the
 * length is clamped under the remaining max_tokens and context capacity): a
 * step emits up to SL + 1 tokens, so sl_next[b] = min(sl_next[b],
 * max(budget[b] - 1, 0)).  The budget wins over sl_min; the cap is taken
 * before the budget.
 *
 *   sf [B], wvir [B], sl_max [B]   float
 *   sl_min                          finite; ceil(sl_min) <= sl_hi (paper: SL_min = 2)
 *   sl_hi                           upper bound of the next step's SL (its k_max)
 *   budget [B]                      int32, optional (may be NULL): tokens each sequence
 *                                   may still emit
 * Outputs: sl_hat [B] float, sl_cap [1] float, sl_next [B] int32, seq_err [B] uint32.
 */
int32_t dsde_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max, float sl_min,
                     int32_t sl_hi, const int32_t *budget, float *sl_hat, float *sl_cap, int32_t *sl_next,
                     uint32_t *seq_err, void *stream);

/*
 * The whole step fused: dsde_verify, then dsde_kld_signal on the KLD it
 * produces, then dsde_next_sl on the signal it produces, with the arguments
 * of those three calls (see them for meaning and layout), in four kernel
 * launches instead of five.  Outputs are bit-identical to the three calls made
 * in sequence; seq_err is the OR of their error bits, except that a layout
 * error (DSDE_ERR_LAYOUT) also skips the signal update.
 * For serving loops that run the complete verification step.
 */
int32_t dsde_step(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                  int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                  const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                  int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                  float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long,
                  float delta, float eps, float *mu_last, float *var_short, float *var_long, float *wvir, float *sf,
                  const float *sl_max, float sl_min, int32_t sl_hi, const int32_t *budget, float *sl_hat,
                  float *sl_cap, int32_t *sl_next, uint32_t *seq_err, void *workspace, size_t workspace_bytes,
                  void *stream);

/*
 * dsde_step without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels and bit-identical outputs, with the
 * scratch space in a device array of DSDE_STATIC_SCRATCH_BYTES that the
 * library holds, one copy per device, until the process ends.  The call
 * allocates nothing; its first call on a device looks up that device's copy.
 *
 * Arguments as in dsde_step, less workspace and workspace_bytes.  Returns
 * DSDE_WORKSPACE_TOO_SMALL when dsde_verify_workspace_bytes(B, N, V, k_max)
 * exceeds DSDE_STATIC_SCRATCH_BYTES (nothing is enqueued), and
 * DSDE_DEVICE_ERROR when the device copy cannot be found.  Every call on one
 * device uses the same array: calls that may overlap on one device (several
 * streams or threads) race and must be serialised by the caller.  No part of
 * the array has to start at any value: every region a call reads is written
 * earlier in that call.
 */
#define DSDE_STATIC_SCRATCH_BYTES (16u << 20)
int32_t dsde_step_static(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                         int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl,
                         const int32_t *draft_tokens, const float *temperature, const float *u_acc,
                         const float *u_res, int32_t pad_id, int32_t *accepted, int32_t *tokens, float *kld,
                         double *row_lse, float *draft_entropy, float *hist, int32_t *head, int32_t *count, int32_t W,
                         int32_t n_short, int32_t n_long, float delta, float eps, float *mu_last, float *var_short,
                         float *var_long, float *wvir, float *sf, const float *sl_max, float sl_min, int32_t sl_hi,
                         const int32_t *budget, float *sl_hat, float *sl_cap, int32_t *sl_next, uint32_t *seq_err,
                         void *stream);

/*
 * SL_max calibration (Sec. 3.1.1, Eq. 1):
 *   SL_max = SL_A,max * (1 + mu_KLD,pre / (KLD_pre,max + eps))
 * over a few preliminary steps: SL_A,max the largest number of drafts accepted
 * in one step, mu_KLD,pre the mean of every per-token KLD seen, KLD_pre,max
 * the largest one.
 *
 * dsde_calibration_update folds one verification step (its sl, cu_sl,
 * accepted, kld and seq_err, as dsde_verify produced them) into running
 * per-sequence statistics; sequences with error bits are skipped, and an
 * invalid layout skips the whole step.  The caller zeroes the statistics
 * before the first step:
 *   a_max [B] int32, kld_sum [B] double, kld_count [B] int64, kld_max [B] float  (in/out)
 * dsde_calibrate_sl_max evaluates Eq. 1 into sl_max [B] (float): per sequence
 * (pooled = 0) or, pooled = 1, from the statistics pooled over the batch (the
 * same value for every sequence).  A sequence without KLD values has mean 0.
 *   eps >= 0 (paper: 1e-6)
 */
int32_t dsde_calibration_update(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl,
                                const int32_t *accepted, const float *kld, const uint32_t *seq_err, int32_t *a_max,
                                double *kld_sum, int64_t *kld_count, float *kld_max, void *stream);
int32_t dsde_calibrate_sl_max(int32_t B, const int32_t *a_max, const double *kld_sum, const int64_t *kld_count,
                              const float *kld_max, float eps, int32_t pooled, float *sl_max, void *stream);

/*
 * Vocabulary-sharded verification, for logits that arrive split by vocabulary,
 * as a tensor-parallel LM head produces them when the target model spans
 * several GPUs (the paper's experiments run on one eight-GPU server, Sec. 4.1;
 * how the model is split there is not stated).  Shard g of G holds, for every row
 * of the packed layout above, the logits of one contiguous vocabulary slice
 * [v_begin_g, v_begin_g + V_g), as row-major [rows, V_g] arrays; the slices of
 * g = 0, 1, ..., G-1 tile [0, V) in ascending order.  A step is four calls on
 * every shard with two exchanges between them, which the caller makes (an
 * all-gather across the G GPUs, e.g. over RCCL):
 *
 *   1. dsde_shard_stats      this slice's statistics of every drafted pair:
 *                            part [N]                   -> gather parts [G][N]
 *   2. dsde_shard_accept     from parts: KLD, acceptance, the accepted drafts
 *                            and each sequence's draw job, jobs [B] (every
 *                            shard computes the same values)
 *   3. dsde_shard_draw_mass  this slice's share of each sequence's draw
 *                            weight: mass [B]           -> gather masses [G][B]
 *   4. dsde_shard_draw_pick  the emitted token: drawn[b] >= 0 on the shard
 *                            that determines it (the one whose slice holds
 *                            the inverse-CDF point, or every shard for greedy
 *                            rows), -1 elsewhere, so an all-reduce max gives
 *                            it to every shard; that shard also writes it into
 *                            tokens.
 *
 * The exchanges carry 64 bytes per drafted position and 32 bytes per sequence
 * from each shard.  Results are those of dsde_verify on the whole rows, with
 * the sums split at slice boundaries: accepted counts, tokens and error bits
 * outside the tie bands, KLD within the same tolerance.  dsde_kld_signal and
 * dsde_next_sl then run unchanged on every shard (their inputs are identical
 * there), or fused behind call 2 (dsde_shard_accept_step).  Every pointer,
 * layout and error rule of dsde_verify applies; the
 * calls of one shard share its workspace (dsde_shard_workspace_bytes), whose
 * contents pass from call 1 to 2 (none), 3 to 4 (the slice's chunk totals).
 */
typedef struct {
  float mt, md;      /* the slice's largest z c of the target and the draft row (log2 domain) */
  double sp, sq;     /* sum over the slice of 2^(z_t c - mt), of 2^(z_d c - md) */
  double a;          /* sum of 2^(z_t c - mt) ((z_t c - mt) - (z_d c - md)) */
  double h;          /* sum of 2^(z_d c - md) (z_d c - md) */
  float zt, zd;      /* target and draft logit at the drafted token, when the slice holds it */
  int32_t has_token; /* 1 when the drafted token lies in the slice */
  float zmax;        /* greedy rows (T_b = 0): the slice's largest target logit, */
  int32_t argmax;    /* and the smallest (global) token id holding it */
  int32_t bad;       /* 1: a NaN or infinite logit in the slice of either row */
} dsde_shard_partial; /* 64 bytes */

typedef struct {
  int32_t kind;      /* 0: residual of the first rejected pair, 1: bonus row, 2: greedy, token
                        known, 3: greedy, argmax of the bonus row, -1: nothing (flagged) */
  int32_t accepted;  /* a_b */
  int32_t target_row, draft_row; /* rows of the draw in the packed layout (draft_row -1: none) */
  float scale;       /* log2(e) / T_b */
  float mt, md;      /* kind 0: the whole rows' largest z c (target, draft) */
  float inv_sp, inv_sq; /* kind 0: 1 / their sums of 2^(z c - m) */
  float u;           /* u_res[b] */
  int32_t token;     /* kind 2: the emitted token */
} dsde_draw_job;     /* 44 bytes */

typedef struct {
  double mass;       /* the slice's total draw weight: max(0, p - q) (kind 0), or 2^(z c - ref)
                        of the bonus row (kind 1); 0 otherwise */
  double p_mass;     /* kind 0: the slice's mass of p, for the draw's fallback to p when no
                        slice holds residual mass */
  float ref;         /* kind 1: the slice's largest z c of the bonus row */
  float zmax;        /* kind 3: the slice's largest bonus-row logit, */
  int32_t argmax;    /* and the smallest (global) token id holding it */
  int32_t bad;       /* kinds 1 and 3: a NaN or infinite logit in the slice of the bonus row */
} dsde_shard_mass;   /* 32 bytes */

/* Workspace bytes of one shard's four calls: B sequences, N drafted positions,
 * slice width V_shard, bound k_max; 0 when the sizes are invalid. */
size_t dsde_shard_workspace_bytes(int32_t B, int64_t N, int64_t V_shard, int32_t k_max);

/*
 * Call 1: the slice statistics of every drafted pair.
 *   target_logits [N+B, V_shard], draft_logits [N, V_shard]   this shard's slices
 *   v_begin, V                  the slice's first token id and the whole vocabulary
 *                               (0 <= v_begin, 1 <= V_shard, v_begin + V_shard <= V <= DSDE_MAX_VOCAB)
 *   sl, cu_sl, draft_tokens (global ids), temperature, B, N, k_max   as in dsde_verify
 *   part [N]                    output, one per drafted position
 *   seq_err [B]                 output: DSDE_ERR_LAYOUT or 0 (the layout check of dsde_verify)
 */
int32_t dsde_shard_stats(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V_shard,
                         int64_t v_begin, int64_t V, int32_t B, int64_t N, int32_t k_max, const int32_t *sl,
                         const int32_t *cu_sl, const int32_t *draft_tokens, const float *temperature,
                         dsde_shard_partial *part, uint32_t *seq_err, void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * Call 2: acceptance and KLD from every shard's partials.
 *   G, parts [G][N]             the gathered partials in shard order (1 <= G <= 1024)
 *   V                           the whole vocabulary
 *   sl ... pad_id               as in dsde_verify
 *   accepted, tokens, kld, row_lse, draft_entropy   as in dsde_verify, except that the
 *                               drawn token is left to call 4 (greedy rows whose token is
 *                               known here get it now)
 *   jobs [B]                    output: the draw of every sequence, for calls 3 and 4
 *   seq_err [B]                 in/out: call 1's bits, OR this call's (a drafted token
 *                               held by no slice or by several is DSDE_ERR_TOKEN)
 */
int32_t dsde_shard_accept(int32_t G, const dsde_shard_partial *parts, int64_t V, int32_t B, int64_t N,
                          int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                          const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                          int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                          dsde_draw_job *jobs, uint32_t *seq_err, void *stream);

/*
 * Call 2 fused with the signal update and the SL rule (Sec. 3.1.2, Eqs. 2-11):
 * dsde_shard_accept, then dsde_kld_signal on the KLD it produces, then
 * dsde_next_sl, with the arguments of those calls (see them for meaning,
 * layout and ownership) in two launches instead of three; the outputs are
 * bit-identical to the three calls in sequence and seq_err is the OR of their
 * error bits, except that a layout error also skips the signal update (as in
 * dsde_step).  Every GPU of the split holds the same KLD after the exchange,
 * so each may run this on its own copy of the controller state.
 * For serving loops that run the complete sharded step.
 */
int32_t dsde_shard_accept_step(int32_t G, const dsde_shard_partial *parts, int64_t V, int32_t B, int64_t N,
                               int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                               const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                               int32_t *accepted, int32_t *tokens, float *kld, double *row_lse,
                               float *draft_entropy, dsde_draw_job *jobs, float *hist, int32_t *head, int32_t *count,
                               int32_t W, int32_t n_short, int32_t n_long, float delta, float eps, float *mu_last,
                               float *var_short, float *var_long, float *wvir, float *sf, const float *sl_max,
                               float sl_min, int32_t sl_hi, const int32_t *budget, float *sl_hat, float *sl_cap,
                               int32_t *sl_next, uint32_t *seq_err, void *stream);

/*
 * Call 3: this slice's share of each sequence's draw weight (it reads the
 * slice of the first rejected pair, or of the bonus row, once) into mass [B];
 * the slice's chunk totals stay in the workspace for call 4.
 *   part [N]                    this shard's call-1 output
 *   jobs [B]                    call 2's output
 */
int32_t dsde_shard_draw_mass(const void *target_logits, const void *draft_logits, int32_t dtype,
                             int64_t V_shard, int64_t v_begin, int32_t B, int64_t N, int32_t k_max,
                             const dsde_shard_partial *part, const dsde_draw_job *jobs, dsde_shard_mass *mass,
                             void *workspace, size_t workspace_bytes, void *stream);

/*
 * Call 4: the draw.  From the gathered masses [G][B] every shard finds the
 * slice holding u'_b Z_b (a fixed-order fp64 prefix over the slices, the rule
 * of dsde_verify's draw); that shard scans its slice (chunk totals from call
 * 3, the fallback to p computed here when it is needed).
 *   g                           this shard's index (0 <= g < G)
 *   drawn [B]                   output: the token, or -1 (see above)
 *   accepted, tokens, seq_err   updated when a sampled bonus row holds a NaN or infinite
 *                               logit: accepted = 0, pad_id tokens, DSDE_ERR_LOGIT (on every
 *                               shard alike)
 */
int32_t dsde_shard_draw_pick(int32_t G, int32_t g, const dsde_shard_mass *masses, const void *target_logits,
                             const void *draft_logits, int32_t dtype, int64_t V_shard, int64_t v_begin,
                             int32_t B, int64_t N, int32_t k_max, const dsde_draw_job *jobs, int32_t pad_id,
                             int32_t *accepted, int32_t *tokens, int32_t *drawn, uint32_t *seq_err,
                             void *workspace, size_t workspace_bytes, void *stream);

/*
 * Measurement utility, not part of the method: reads `bytes` bytes of device
 * memory at `buf` with the statistics pass's access pattern (one workgroup per
 * 32 KiB, 16-byte vector loads, 1 KiB contiguous per wavefront load) and
 * writes the XOR of every 32-bit word of 32 KiB unit u to out[u].  Timed over
 * a buffer much larger than the last-level cache it gives the streaming-read
 * ceiling the row statistics kernel is compared against.
 *   buf      device pointer, 16-byte aligned
 *   bytes    a positive multiple of 16
 *   out      device array of ceil(bytes / 32768) uint32
 * Returns DSDE_INVALID_ARG for a NULL or misaligned pointer or a bad size.
 */
int32_t dsde_stream_read(const void *buf, int64_t bytes, uint32_t *out, void *stream);

/*
 * Profiling hook: when both events are non-NULL (hipEvent_t, created with
 * timing enabled), every later dsde_verify or dsde_step with N > 0 attaches
 * `start` to the completion of its set-up kernel and `stop` to the completion
 * of its row statistics kernel (the pass that reads every drafted row pair
 * once), which runs right after it on the same stream; the elapsed time
 * between them is that kernel's execution time.  Events created with
 * hipEventDisableSystemFence add no gap to the stream.  Passing NULLs turns it
 * off.  Process-wide; not thread-safe.
 */
int32_t dsde_set_profile_events(void *start, void *stop);

#ifdef __cplusplus
}
#endif

#endif /* DSDE_H_ */
