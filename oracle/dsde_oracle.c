/*
 * DSDE oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU implementation of the speculative-verification step with
 * ragged per-sequence speculation lengths (SL), the per-token KL divergence,
 * the KLD-variance stability signal and the batch SL cap of DSDE
 * (arXiv 2509.01083).  Everything is computed in double precision with
 * straight loops in the order the definitions are written; there is no
 * blocking, fusion or reordering.  It shares no code, header, table or
 * constant with the HIP library; only tests, the smoke check and the CPU
 * baseline leg of the benchmark may load it.
 *
 * What each function follows:
 *   oracle_verify     -- speculative sampling as cited in Sec. 2.1 (accept a
 *                        drafted token while u < min(1, p/q); on the first
 *                        rejection draw from the normalised residual
 *                        max(0, p - q); if every drafted token is accepted draw
 *                        the bonus token from the extra target row), the
 *                        ragged per-sequence layout and pad id of Sec. 3.2, and
 *                        the per-token KLD used by the SL adapter (Sec. 3.1.2).
 *   oracle_kld_signal -- Sec. 3.1.2: mu_KLD,last (Eq. 3's argument), the
 *                        recency weights alpha_i = delta^(i-1) (Eq. 5), the
 *                        weighted mean and population variance (Eqs. 6-7) over
 *                        the short (N=10) and long (N=30) windows, WVIR (Eq. 4)
 *                        and SF (Eq. 3).
 *   oracle_next_sl    -- Eq. 2 with the lower bound of Eq. 8, and the batch cap
 *                        of Sec. 3.3 (Eqs. 9-11: the MSE-optimal cap is the mean
 *                        of the predicted lengths).
 *   oracle_calibrate_sl_max -- Eq. 1 (Sec. 3.1.1).
 *
 * Also: the entropy H(q) of every drafted position's tempered draft
 * distribution (the draft-entropy signal the paper compares against, Sec. 4.2
 * and Table 2), and a per-sequence token budget that bounds the next
 * speculation length (the clamp under remaining max_tokens and context
 * capacity of the policy interface, Sec. 3.2): a step emits up to SL + 1
 * tokens, so SL_next <= max(budget - 1, 0).
 *
 * Greedy verification (the temperature-0.0 setting of the experiments, Sec. 4.2
 * and Table 3(a)): a sequence with T_b = 0 accepts a drafted token iff it is
 * the argmax of its target row (the smallest token id among equal maxima) and
 * emits the argmax of the first rejected row, or of the bonus row; its KLD is
 * taken on the T = 1 softmaxes, and its uniforms are not used.
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   - KL direction KL(p_target || q_draft); both softmaxes use the sequence's
 *     temperature, the same p and q the acceptance test uses.
 *   - mu_KLD,last is the mean KLD over all SL_b drafted positions of the step;
 *     one history entry per (sequence, step); the entry is pushed before the
 *     windows are taken, so i = 1 is the step just verified.
 *   - Window sizes are min(n_short, count) and min(n_long, count); an empty
 *     window has mean 0 and variance 0; WVIR = Var_s / Var_l (Eq. 4), with
 *     eps > 0 in place of Var_l only when Var_l = 0 (then WVIR = 0).
 *   - Acceptance is strict (u < min(1, r)); the inverse-CDF draw walks token
 *     ids in ascending order and returns the smallest id whose cumulative
 *     weight exceeds u' * Z.
 *   - SL_next = clamp(floor(min(SL_hat, SL_cap) + 1/2), ceil(sl_min), sl_hi).
 *     The paper gives no rounding rule and no worked example, so this integer
 *     step is parity unpinned: the tests pin it to the reading above only
 *     (SL_hat and the cap themselves are pinned by closed forms).
 *
 * Ties: a decision that sits within 1e-6 of its threshold is flagged, not
 * resolved: |u - min(1, r)| <= 1e-6 for an acceptance test, and
 * |u' * Z - C| <= 1e-6 (probability mass) for either CDF boundary around the
 * drawn token.  Flagged sequences are left out of bit-exact comparisons.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* per-sequence error bits (mirrors the documented contract of the step) */
#define ORC_BAD_LAYOUT 1u   /* SL_b outside [0, k_max] or cu_sl inconsistent */
#define ORC_BAD_TOKEN 2u    /* drafted token outside [0, V) */
#define ORC_BAD_LOGIT 4u    /* non-finite logit in a row the step uses */
#define ORC_BAD_TEMP 8u     /* temperature not finite or outside [2^-16, 2^16] */
#define ORC_BAD_UNIFORM 16u /* uniform outside [0, 1) */
#define ORC_BAD_SIGNAL 32u  /* non-finite signal value */
#define ORC_BAD_STATE 64u   /* ring head/count outside their ranges */

#define ORC_TIE_BAND 1e-6

/* ------------------------------------------------------------------ */
/* compensated sums                                                    */
/* ------------------------------------------------------------------ */

/* Neumaier's compensated summation: the running sum s, and in c the
 * low-order part every addition rounded away (taken from whichever operand
 * is smaller in magnitude); the sum is s + c. */
typedef struct {
  double s, c;
} csum;

static void csum_add(csum *a, double x) {
  double t = a->s + x;
  if (fabs(a->s) >= fabs(x))
    a->c += (a->s - t) + x;
  else
    a->c += (x - t) + a->s;
  a->s = t;
}

static double csum_value(const csum *a) { return a->s + a->c; }

/* ------------------------------------------------------------------ */
/* logits                                                              */
/* ------------------------------------------------------------------ */

/* Exact decode of one logit: fp32 as is, bf16 as the top 16 bits of an fp32. */
static double logit(const void *base, int dtype, int64_t V, int64_t row, int64_t v) {
  int64_t k = row * V + v;
  if (dtype == 0) return (double)((const float *)base)[k];
  uint32_t bits = (uint32_t)((const uint16_t *)base)[k] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

static int row_is_finite(const void *base, int dtype, int64_t V, int64_t row) {
  for (int64_t v = 0; v < V; ++v)
    if (!isfinite(logit(base, dtype, V, row, v))) return 0;
  return 1;
}

/* log of the softmax normaliser of the tempered row s_v = z_v / T:
 * lse = m + log(sum_v exp(s_v - m)), m = max_v s_v. */
static double row_lse(const void *base, int dtype, int64_t V, int64_t row, double T) {
  double m = -INFINITY;
  for (int64_t v = 0; v < V; ++v) {
    double s = logit(base, dtype, V, row, v) / T;
    if (s > m) m = s;
  }
  csum S = {0.0, 0.0};
  for (int64_t v = 0; v < V; ++v) csum_add(&S, exp(logit(base, dtype, V, row, v) / T - m));
  return m + log(csum_value(&S));
}

/* The smallest token id holding the row's largest logit. */
static int64_t row_argmax(const void *base, int dtype, int64_t V, int64_t row) {
  int64_t best = 0;
  double m = logit(base, dtype, V, row, 0);
  for (int64_t v = 1; v < V; ++v) {
    double z = logit(base, dtype, V, row, v);
    if (z > m) {
      m = z;
      best = v;
    }
  }
  return best;
}

/* ------------------------------------------------------------------ */
/* verification step                                                   */
/* ------------------------------------------------------------------ */

typedef struct {
  const void *target, *draft;
  int dtype;
  int64_t V, N;
  int32_t B, k_max;
  const int32_t *sl, *cu_sl, *draft_tokens;
  const float *temperature, *u_acc, *u_res;
  int32_t pad_id;
  int layout_ok;
  /* outputs */
  int32_t *accepted, *tokens;
  double *kld, *lse; /* lse: [N, 2] (p, q), may be NULL */
  double *entropy;   /* [N] H(q) in nats, may be NULL */
  uint32_t *seq_err;
  int32_t *acc_tie, *cdf_tie;
  double *sample_mass; /* [B]: Z of the draw (probability mass), may be NULL */
  int n_threads, tid;
} verify_job;

static void verify_sequence(const verify_job *J, int32_t b) {
  const int64_t V = J->V;
  const int32_t width = J->k_max + 1;
  int32_t *tok = J->tokens + (int64_t)b * width;
  for (int32_t k = 0; k < width; ++k) tok[k] = J->pad_id;
  J->accepted[b] = 0;
  J->acc_tie[b] = 0;
  J->cdf_tie[b] = 0;
  if (J->sample_mass) J->sample_mass[b] = NAN;

  uint32_t err = 0;
  const int32_t SL = J->sl[b];
  if (!J->layout_ok) {
    J->seq_err[b] = ORC_BAD_LAYOUT;
    return;
  }
  const int64_t first = J->cu_sl[b];          /* first drafted position of b */
  const int64_t trow0 = first + b;            /* its first target row */
  /* T_b = 0: greedy verification, whose KLD is taken at T = 1 */
  const int greedy = J->temperature[b] == 0.0f;
  const double T = greedy ? 1.0 : (double)J->temperature[b];

  for (int32_t j = 0; j < SL; ++j) {
    int32_t x = J->draft_tokens[first + j];
    if (x < 0 || (int64_t)x >= V) err |= ORC_BAD_TOKEN;
    float u = J->u_acc[first + j];
    if (!greedy && !(u >= 0.0f && u < 1.0f)) err |= ORC_BAD_UNIFORM;
  }
  if (!greedy) {
    float u = J->u_res[b];
    if (!(u >= 0.0f && u < 1.0f)) err |= ORC_BAD_UNIFORM;
    /* the admissible temperature range of the boundary: [2^-16, 2^16] */
    if (!(T >= ldexp(1.0, -16) && T <= ldexp(1.0, 16))) err |= ORC_BAD_TEMP;
  }
  if (!err) {
    for (int32_t j = 0; j < SL; ++j)
      if (!row_is_finite(J->target, J->dtype, V, trow0 + j) ||
          !row_is_finite(J->draft, J->dtype, V, first + j))
        err |= ORC_BAD_LOGIT;
  }
  if (err) goto fail;

  /* row normalisers and the per-token KLD of every drafted pair */
  double *lse_p = (double *)malloc(sizeof(double) * (SL > 0 ? SL : 1));
  double *lse_q = (double *)malloc(sizeof(double) * (SL > 0 ? SL : 1));
  for (int32_t j = 0; j < SL; ++j) {
    const int64_t tr = trow0 + j, dr = first + j;
    lse_p[j] = row_lse(J->target, J->dtype, V, tr, T);
    lse_q[j] = row_lse(J->draft, J->dtype, V, dr, T);
    /* KL(p || q) = sum_v p_v (log p_v - log q_v); terms with p_v == 0 vanish */
    csum kls = {0.0, 0.0};
    for (int64_t v = 0; v < V; ++v) {
      double lp = logit(J->target, J->dtype, V, tr, v) / T - lse_p[j];
      double lq = logit(J->draft, J->dtype, V, dr, v) / T - lse_q[j];
      double p = exp(lp);
      if (p > 0.0) csum_add(&kls, p * (lp - lq));
    }
    const double kl = csum_value(&kls);
    J->kld[first + j] = kl > 0.0 ? kl : 0.0;
    if (J->entropy) {
      /* H(q) = -sum_v q_v log q_v of the same tempered draft distribution */
      csum h = {0.0, 0.0};
      for (int64_t v = 0; v < V; ++v) {
        double lq = logit(J->draft, J->dtype, V, dr, v) / T - lse_q[j];
        double q = exp(lq);
        if (q > 0.0) csum_add(&h, -q * lq);
      }
      J->entropy[first + j] = csum_value(&h);
    }
    if (J->lse) {
      J->lse[2 * (first + j)] = lse_p[j];
      J->lse[2 * (first + j) + 1] = lse_q[j];
    }
  }

  if (greedy) {
    /* accept x_j while it is the argmax of its target row; emit the argmax of
     * the first rejected row, or of the bonus row */
    int32_t a = 0;
    while (a < SL && (int64_t)J->draft_tokens[first + a] == row_argmax(J->target, J->dtype, V, trow0 + a)) ++a;
    free(lse_p);
    free(lse_q);
    if (a == SL && !row_is_finite(J->target, J->dtype, V, trow0 + SL)) {
      J->seq_err[b] = ORC_BAD_LOGIT;
      return;
    }
    for (int32_t j = 0; j < a; ++j) tok[j] = J->draft_tokens[first + j];
    tok[a] = (int32_t)row_argmax(J->target, J->dtype, V, trow0 + a);
    J->accepted[b] = a;
    J->seq_err[b] = 0;
    return;
  }

  /* acceptance scan: accept drafted token x_j while u_j < min(1, p(x_j)/q(x_j)) */
  int32_t a = 0;
  for (int32_t j = 0; j < SL; ++j) {
    const int32_t x = J->draft_tokens[first + j];
    double lp = logit(J->target, J->dtype, V, trow0 + j, x) / T - lse_p[j];
    double lq = logit(J->draft, J->dtype, V, first + j, x) / T - lse_q[j];
    double r = exp(lp - lq);
    double thr = r < 1.0 ? r : 1.0;
    double u = (double)J->u_acc[first + j];
    if (fabs(u - thr) <= ORC_TIE_BAND) J->acc_tie[b] = 1;
    if (u < thr) {
      ++a;
    } else {
      break;
    }
  }

  /* the draw: residual max(0, p - q) of the first rejected pair, or the
   * target distribution of the bonus row when every drafted token was accepted */
  int64_t tr, dr = -1;
  double lp_row, lq_row = 0.0;
  if (a < SL) {
    tr = trow0 + a;
    dr = first + a;
    lp_row = lse_p[a];
    lq_row = lse_q[a];
  } else {
    tr = trow0 + SL;
    if (!row_is_finite(J->target, J->dtype, V, tr)) {
      /* a non-finite bonus row withholds the token only: the KLD of the
       * drafted pairs stays defined */
      free(lse_p);
      free(lse_q);
      J->seq_err[b] = ORC_BAD_LOGIT;
      return;
    }
    lp_row = row_lse(J->target, J->dtype, V, tr, T);
  }
  double *w = (double *)malloc(sizeof(double) * (size_t)V);
  csum Zs = {0.0, 0.0};
  for (int64_t v = 0; v < V; ++v) {
    double p = exp(logit(J->target, J->dtype, V, tr, v) / T - lp_row);
    if (dr >= 0) {
      double q = exp(logit(J->draft, J->dtype, V, dr, v) / T - lq_row);
      w[v] = p - q > 0.0 ? p - q : 0.0;
    } else {
      w[v] = p;
    }
    csum_add(&Zs, w[v]);
  }
  if (csum_value(&Zs) == 0.0) { /* no residual mass left: draw from p of the same target row */
    for (int64_t v = 0; v < V; ++v) {
      w[v] = exp(logit(J->target, J->dtype, V, tr, v) / T - lp_row);
      csum_add(&Zs, w[v]);
    }
  }
  const double Z = csum_value(&Zs);
  const double target_mass = (double)J->u_res[b] * Z;
  /* the cumulative weight C(v) in ascending token id, compensated like Z */
  int64_t y = -1;
  csum Cs = {0.0, 0.0};
  double C = 0.0, C_prev = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    C_prev = C;
    csum_add(&Cs, w[v]);
    C = csum_value(&Cs);
    if (C > target_mass) {
      y = v;
      break;
    }
  }
  if (y < 0) { /* rounding left u' * Z at or past the total: last positive weight */
    y = V - 1;
    for (int64_t v = V - 1; v >= 0; --v)
      if (w[v] > 0.0) {
        y = v;
        break;
      }
    C_prev = Z - w[y];
    C = Z;
  }
  if (fabs(target_mass - C_prev) <= ORC_TIE_BAND || fabs(target_mass - C) <= ORC_TIE_BAND)
    J->cdf_tie[b] = 1;
  if (J->sample_mass) J->sample_mass[b] = Z;
  free(w);
  free(lse_p);
  free(lse_q);

  for (int32_t j = 0; j < a; ++j) tok[j] = J->draft_tokens[first + j];
  tok[a] = (int32_t)y;
  J->accepted[b] = a;
  J->seq_err[b] = 0;
  return;

fail:
  J->seq_err[b] = err;
  for (int32_t j = 0; j < SL; ++j) J->kld[first + j] = NAN;
  if (J->entropy)
    for (int32_t j = 0; j < SL; ++j) J->entropy[first + j] = NAN;
}

static void *verify_worker(void *arg) {
  const verify_job *J = (const verify_job *)arg;
  for (int32_t b = J->tid; b < J->B; b += J->n_threads) verify_sequence(J, b);
  return NULL;
}

/* Layout of the packed rows (Sec. 3.2, "Ragged Q"): sequence b owns drafted
 * positions [cu_sl[b], cu_sl[b+1]), target rows cu_sl[b] + b + j for
 * j = 0..SL_b (the last one is the bonus row) and draft rows cu_sl[b] + j for
 * j < SL_b.  Valid when cu_sl[0] = 0, cu_sl[B] = N, and every sequence has
 * 0 <= SL_b <= k_max and cu_sl[b+1] - cu_sl[b] = SL_b. */
static int layout_valid(int32_t B, int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl) {
  if (cu_sl[0] != 0 || (int64_t)cu_sl[B] != N) return 0;
  for (int32_t b = 0; b < B; ++b)
    if (sl[b] < 0 || sl[b] > k_max || cu_sl[b + 1] - cu_sl[b] != sl[b]) return 0;
  return 1;
}

int oracle_verify(const void *target, const void *draft, int32_t dtype, int64_t V, int32_t B, int32_t k_max,
                  int64_t N, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                  const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                  int32_t *accepted, int32_t *tokens, double *kld, double *lse, double *entropy,
                  uint32_t *seq_err, int32_t *acc_tie, int32_t *cdf_tie, double *sample_mass,
                  int32_t n_threads) {
  if (B < 1 || V < 1 || k_max < 0 || N < 0 || (dtype != 0 && dtype != 1)) return 1;
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 256) n_threads = 256;
  verify_job base = {target, draft, dtype, V, N, B, k_max, sl, cu_sl, draft_tokens, temperature, u_acc,
                     u_res, pad_id, layout_valid(B, N, k_max, sl, cu_sl), accepted, tokens, kld, lse,
                     entropy, seq_err, acc_tie, cdf_tie, sample_mass, n_threads, 0};
  verify_job jobs[256];
  pthread_t th[256];
  for (int t = 0; t < n_threads; ++t) {
    jobs[t] = base;
    jobs[t].tid = t;
  }
  for (int t = 1; t < n_threads; ++t) pthread_create(&th[t], NULL, verify_worker, &jobs[t]);
  verify_worker(&jobs[0]);
  for (int t = 1; t < n_threads; ++t) pthread_join(th[t], NULL);
  return 0;
}

/* ------------------------------------------------------------------ */
/* KLD stability signal                                                */
/* ------------------------------------------------------------------ */

/* Weighted mean and population variance (Eqs. 5-7) of the n newest entries
 * h_1..h_n (h_1 newest) with alpha_i = delta^(i-1).  The sums run over the
 * entries less h_1: a common shift leaves Eq. 7 unchanged, and with it a
 * window of equal entries has a variance of exactly 0 instead of a rounding
 * residue of its mean. */
static void weighted_stats(const double *newest_first, int32_t n, double delta, double *mean, double *var) {
  if (n <= 0) {
    *mean = 0.0;
    *var = 0.0;
    return;
  }
  const double h1 = newest_first[0];
  double sa = 0.0, sad = 0.0;
  for (int32_t i = 1; i <= n; ++i) {
    double alpha = pow(delta, (double)(i - 1));
    sa += alpha;
    sad += alpha * (newest_first[i - 1] - h1);
  }
  double mu_d = sad / sa; /* the weighted mean less h_1 */
  double sv = 0.0;
  for (int32_t i = 1; i <= n; ++i) {
    double alpha = pow(delta, (double)(i - 1));
    double d = (newest_first[i - 1] - h1) - mu_d;
    sv += alpha * d * d;
  }
  *mean = h1 + mu_d;
  *var = sv / sa;
}

/* One sequence of the signal update, on an explicit newest-first history
 * (count entries, after any push).  Exposed so the SL tie analysis can
 * re-evaluate it on perturbed histories. */
static void signal_from_history(const double *newest_first, int32_t count, double mu_last, int32_t n_short,
                                int32_t n_long, double delta, double eps, double *var_s, double *var_l,
                                double *wvir, double *sf) {
  int32_t ns = n_short < count ? n_short : count;
  int32_t nl = n_long < count ? n_long : count;
  double ms, ml;
  weighted_stats(newest_first, ns, delta, &ms, var_s);
  weighted_stats(newest_first, nl, delta, &ml, var_l);
  /* Eq. 4 as printed; eps stands in for the long-window variance only where
   * that is 0 (a window of equal entries, whose short window is constant
   * too, so WVIR = 0) */
  *wvir = *var_s / (*var_l > 0.0 ? *var_l : eps);
  *sf = exp(2.0 * mu_last) - 1.0;
}

int oracle_kld_signal(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const double *kld,
                      double *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long,
                      double delta, double eps, double *mu_last, double *var_short, double *var_long,
                      double *wvir, double *sf, uint32_t *seq_err) {
  if (B < 1 || N < 0 || W < 1 || n_short < 1 || n_short > n_long || !(delta > 0.0 && delta <= 1.0) ||
      !(eps > 0.0))
    return 1;
  int layout_ok = cu_sl[0] == 0 && (int64_t)cu_sl[B] == N;
  for (int32_t b = 0; b < B && layout_ok; ++b)
    if (sl[b] < 0 || cu_sl[b + 1] - cu_sl[b] != sl[b]) layout_ok = 0;
  double *h = (double *)malloc(sizeof(double) * (size_t)W);
  for (int32_t b = 0; b < B; ++b) {
    uint32_t err = 0;
    if (!layout_ok) err |= ORC_BAD_LAYOUT;
    if (head[b] < 0 || head[b] >= W || count[b] < 0 || count[b] > W) err |= ORC_BAD_STATE;
    double mu = 0.0;
    if (!err && sl[b] > 0) {
      double s = 0.0;
      for (int32_t j = 0; j < sl[b]; ++j) s += kld[cu_sl[b] + j];
      mu = s / (double)sl[b];
      if (!isfinite(mu)) err |= ORC_BAD_SIGNAL;
    }
    if (err) {
      seq_err[b] = err;
      mu_last[b] = var_short[b] = var_long[b] = wvir[b] = sf[b] = NAN;
      continue;
    }
    double *ring = hist + (int64_t)b * W;
    if (sl[b] > 0) { /* push the step's mean KLD */
      ring[head[b]] = mu;
      head[b] = (head[b] + 1) % W;
      if (count[b] < W) count[b] += 1;
    } else { /* nothing verified: the newest entry stands in, or 0 */
      mu = count[b] > 0 ? ring[(head[b] - 1 + W) % W] : 0.0;
    }
    for (int32_t i = 1; i <= count[b]; ++i) h[i - 1] = ring[((head[b] - i) % W + W) % W];
    signal_from_history(h, count[b], mu, n_short, n_long, delta, eps, &var_short[b], &var_long[b], &wvir[b],
                        &sf[b]);
    mu_last[b] = mu;
    seq_err[b] = 0;
  }
  free(h);
  return 0;
}

/* ------------------------------------------------------------------ */
/* SL rule and batch cap                                               */
/* ------------------------------------------------------------------ */

/* Eq. 2 with Eq. 8's lower bound: penalty SF * WVIR above 1 gives SL_min. */
static double sl_hat_of(double sf, double wvir, double sl_max, double sl_min) {
  double pen = sf * wvir;
  if (pen <= 1.0) return (1.0 - pen) * (sl_max - sl_min) + sl_min;
  return sl_min;
}

static int32_t round_clamp(double x, int32_t lo, int32_t hi) {
  double r = floor(x + 0.5);
  if (r < (double)lo) return lo;
  if (r > (double)hi) return hi;
  return (int32_t)r;
}

int oracle_next_sl(int32_t B, const double *sf, const double *wvir, const double *sl_max, double sl_min,
                   int32_t sl_hi, const int32_t *budget, double *sl_hat, double *sl_cap, int32_t *sl_next,
                   uint32_t *seq_err) {
  if (B < 1 || !isfinite(sl_min) || ceil(sl_min) > (double)sl_hi) return 1;
  const int32_t lo = (int32_t)ceil(sl_min);
  double sum = 0.0;
  int32_t n = 0;
  for (int32_t b = 0; b < B; ++b) {
    int ok = isfinite(sf[b]) && isfinite(wvir[b]) && isfinite(sl_max[b]) && sl_max[b] >= sl_min;
    seq_err[b] = ok ? 0u : ORC_BAD_SIGNAL;
    sl_hat[b] = ok ? sl_hat_of(sf[b], wvir[b], sl_max[b], sl_min) : NAN;
    if (ok) {
      sum += sl_hat[b];
      ++n;
    }
  }
  /* Eqs. 9-11: the cap minimising the mean squared distance to every
   * predicted length is their arithmetic mean */
  double cap = n > 0 ? sum / (double)n : NAN;
  *sl_cap = cap;
  for (int32_t b = 0; b < B; ++b) {
    if (seq_err[b]) {
      sl_next[b] = lo;
      continue;
    }
    double x = sl_hat[b] < cap ? sl_hat[b] : cap;
    sl_next[b] = round_clamp(x, lo, sl_hi);
  }
  if (budget) /* the step after this one may emit at most budget[b] tokens */
    for (int32_t b = 0; b < B; ++b) {
      int32_t room = budget[b] - 1 > 0 ? budget[b] - 1 : 0;
      if (sl_next[b] > room) sl_next[b] = room;
    }
  return 0;
}

/* Eq. 1: SL_max = SL_A,max * (1 + mu_KLD,pre / (KLD_pre,max + eps)), from the
 * accepted counts and the per-token KLD values of the calibration steps. */
double oracle_calibrate_sl_max(int32_t n_steps, const int32_t *accepted_per_step, int64_t n_kld,
                               const double *kld_values, double eps) {
  int32_t amax = 0;
  for (int32_t s = 0; s < n_steps; ++s)
    if (accepted_per_step[s] > amax) amax = accepted_per_step[s];
  double sum = 0.0, kmax = 0.0;
  for (int64_t i = 0; i < n_kld; ++i) {
    sum += kld_values[i];
    if (kld_values[i] > kmax) kmax = kld_values[i];
  }
  double mean = n_kld > 0 ? sum / (double)n_kld : 0.0;
  return (double)amax * (1.0 + mean / (kmax + eps));
}

/* ------------------------------------------------------------------ */
/* tie analysis of SL decisions                                        */
/* ------------------------------------------------------------------ */

/* First-order spread of the signal outputs under a relative uncertainty rho
 * on every history entry a sequence uses (including the one pushed this step,
 * which is also the mu_KLD,last of SF).  For each entry alone the signal is
 * re-evaluated with the entry scaled by (1 - rho) and (1 + rho); per output the
 * larger change is kept and the changes are summed over entries.  Inputs are
 * the post-step rings and sl_max; every output pointer may be NULL.  Eq. 8 is
 * continuous at SF * WVIR = 1, so SL_hat's spread bounds its decision. */
int oracle_signal_spread(int32_t B, const double *hist, const int32_t *head, const int32_t *count, int32_t W,
                         const double *sl_max, int32_t n_short, int32_t n_long, double delta, double eps,
                         double sl_min, double rho, const uint32_t *seq_err, double *hat, double *dhat,
                         double *dvar_s, double *dvar_l, double *dwvir, double *dsf) {
  double *h = (double *)malloc(sizeof(double) * (size_t)(W > 0 ? W : 1));
  for (int32_t b = 0; b < B; ++b) {
    double base[5] = {NAN, NAN, NAN, NAN, NAN}, spread[5] = {NAN, NAN, NAN, NAN, NAN};
    if (!seq_err[b]) {
      const int32_t cnt = count[b];
      for (int32_t i = 1; i <= cnt; ++i) h[i - 1] = hist[(int64_t)b * W + ((head[b] - i) % W + W) % W];
      double vs, vl, wv, sf;
      signal_from_history(h, cnt, cnt > 0 ? h[0] : 0.0, n_short, n_long, delta, eps, &vs, &vl, &wv, &sf);
      base[0] = vs;
      base[1] = vl;
      base[2] = wv;
      base[3] = sf;
      base[4] = sl_hat_of(sf, wv, sl_max[b], sl_min);
      for (int k = 0; k < 5; ++k) spread[k] = 0.0;
      const int32_t nuse = n_long < cnt ? n_long : cnt;
      for (int32_t i = 0; i < nuse; ++i) {
        const double keep = h[i];
        double worst[5] = {0.0, 0.0, 0.0, 0.0, 0.0};
        for (int sgn = -1; sgn <= 1; sgn += 2) {
          h[i] = keep * (1.0 + sgn * rho);
          double vs2, vl2, wv2, sf2;
          signal_from_history(h, cnt, h[0], n_short, n_long, delta, eps, &vs2, &vl2, &wv2, &sf2);
          const double now[5] = {vs2, vl2, wv2, sf2, sl_hat_of(sf2, wv2, sl_max[b], sl_min)};
          for (int k = 0; k < 5; ++k) {
            double d = fabs(now[k] - base[k]);
            if (d > worst[k]) worst[k] = d;
          }
        }
        h[i] = keep;
        for (int k = 0; k < 5; ++k) spread[k] += worst[k];
      }
    }
    if (dvar_s) dvar_s[b] = spread[0];
    if (dvar_l) dvar_l[b] = spread[1];
    if (dwvir) dwvir[b] = spread[2];
    if (dsf) dsf[b] = spread[3];
    if (hat) hat[b] = base[4];
    if (dhat) dhat[b] = spread[4];
  }
  free(h);
  return 0;
}

/* A sequence's SL decision is a tie when the interval of min(SL_hat, cap),
 * widened by tau, contains a rounding boundary k + 1/2 that separates two
 * results inside [ceil(sl_min), sl_hi].  The cap's spread is the mean of the
 * SL_hat spreads of the sequences it averages. */
int oracle_sl_round_ties(int32_t B, const double *hat, const double *dhat, const uint32_t *seq_err, double sl_min,
                         int32_t sl_hi, double tau, int32_t *tie) {
  const int32_t lo = (int32_t)ceil(sl_min);
  double cap = 0.0, dcap = 0.0;
  int32_t n = 0;
  for (int32_t b = 0; b < B; ++b)
    if (!seq_err[b]) {
      cap += hat[b];
      dcap += dhat[b];
      ++n;
    }
  if (n > 0) {
    cap /= n;
    dcap /= n;
  }
  for (int32_t b = 0; b < B; ++b) {
    tie[b] = 0;
    if (seq_err[b]) continue;
    double x, dx;
    if (fabs(hat[b] - cap) <= dhat[b] + dcap + tau) {
      x = hat[b] < cap ? hat[b] : cap;
      dx = (dhat[b] > dcap ? dhat[b] : dcap) + fabs(hat[b] - cap);
    } else if (hat[b] < cap) {
      x = hat[b];
      dx = dhat[b];
    } else {
      x = cap;
      dx = dcap;
    }
    for (int32_t k = lo; k < sl_hi; ++k)
      if (fabs(x - ((double)k + 0.5)) <= dx + tau) tie[b] = 1;
  }
  return 0;
}
