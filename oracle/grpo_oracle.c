/*
 * Plain double-precision CPU oracle for the GRPO scoring + loss hot path.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may call this library. It shares no code,
 * header, table or constant with the HIP path. Every input arrives already
 * decoded to double (bf16 and fp32 values are exactly representable).
 *
 * What it computes (AutoTriton, Sec. 3.3):
 *   - Eq. 2, group-normalised advantages, read as statistics over the G
 *     rollouts of one prompt (an all-equal group gives exactly 0);
 *   - the policy log-probability pi_theta(o_t | q, o_<t) of each sampled
 *     token: a softmax over the vocabulary of the LM-head logits
 *     z_v = <h_t, W_v>, taken at the sampled id;
 *   - Eq. 1, the clipped surrogate with the k3 KL estimator
 *     exp(ref - logp) - (ref - logp) - 1, averaged over the tokens of each
 *     rollout and then over the rollouts (loss = -J);
 *   - the exact analytic gradients of that loss with respect to the hidden
 *     states h and the LM-head weight W.
 *
 *   - the supervised stage before it (Sec. 3.2): the mean over supervised
 *     tokens of the next-token cross-entropy -log pi_theta(y_t), and its
 *     gradients through the same log-softmax.
 *
 * Everything is written the slow, direct way: logits rows are materialised
 * in full, sums run in index order, and nothing is blocked or fused.
 * Parallelism is OpenMP over independent tokens or vocabulary rows only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- Eq. 2 */
/* Advantage of rollout i of a prompt: (r_i - mean_g r) / (std_g r + eps).
 * std is the unbiased (G-1) estimate when unbiased != 0, else the population
 * one. A group whose rewards are all equal gets exactly 0 (the explicit test
 * keeps a rounding-level nonzero mean difference from leaking through). */
void oracle_group_advantages(const double* rewards, int64_t num_prompts, int64_t group,
                             double std_eps, int unbiased, double* adv) {
  for (int64_t p = 0; p < num_prompts; ++p) {
    const double* r = rewards + p * group;
    double* a = adv + p * group;
    double lo = r[0], hi = r[0];
    for (int64_t i = 1; i < group; ++i) {
      if (r[i] < lo) lo = r[i];
      if (r[i] > hi) hi = r[i];
    }
    if (lo == hi) {
      for (int64_t i = 0; i < group; ++i) a[i] = 0.0;
      continue;
    }
    double mean = 0.0;
    for (int64_t i = 0; i < group; ++i) mean += r[i];
    mean /= (double)group;
    double ss = 0.0;
    for (int64_t i = 0; i < group; ++i) ss += (r[i] - mean) * (r[i] - mean);
    double var = ss / (double)(unbiased ? group - 1 : group);
    double sd = sqrt(var);
    for (int64_t i = 0; i < group; ++i) a[i] = (r[i] - mean) / (sd + std_eps);
  }
}

/* --------------------------------------------------- valid-token packing */
/* Rows whose mask is set, in increasing order, and the count |o_b| of each
 * rollout b (rows cu[b] .. cu[b+1]-1). Returns the number of valid rows. */
int64_t oracle_pack_valid(const uint8_t* mask, const int64_t* cu_seqlens, int64_t num_seqs,
                          int64_t* rows, int64_t* counts, int64_t* seq_of_row) {
  int64_t n = 0;
  for (int64_t b = 0; b < num_seqs; ++b) {
    int64_t c = 0;
    for (int64_t t = cu_seqlens[b]; t < cu_seqlens[b + 1]; ++t) {
      if (seq_of_row) seq_of_row[t] = b;
      if (mask == NULL || mask[t]) {
        if (rows) rows[n] = t;
        ++n;
        ++c;
      }
    }
    counts[b] = c;
  }
  return n;
}

/* ------------------------------------------------- Eq. 1 normalisation */
/* Weight c_b of every valid token of rollout b in the loss sum.
 * agg 0 (Eq. 1 as written): 1/G per prompt mean, 1/|o_b| per rollout, and
 *   the expectation over prompts as a mean over the P prompts, so
 *   c_b = 1 / (B * |o_b|) with B = P*G.
 * agg 1 (one global token mean): c_b = 1 / sum_b |o_b|.
 * An empty rollout contributes nothing (c_b = 0) but still counts in B. */
void oracle_seq_weights(const int64_t* counts, int64_t num_seqs, int agg, double* c) {
  int64_t total = 0;
  for (int64_t b = 0; b < num_seqs; ++b) total += counts[b];
  for (int64_t b = 0; b < num_seqs; ++b) {
    if (counts[b] == 0) {
      c[b] = 0.0;
    } else if (agg == 0) {
      c[b] = 1.0 / ((double)num_seqs * (double)counts[b]);
    } else {
      c[b] = 1.0 / (double)total;
    }
  }
}

/* ------------------------------------------- policy log-prob of a token */
/* z_v = sum_k h_k W_{v,k} for every vocabulary entry v (the full row). */
static void logits_row(const double* h, const double* W, int64_t H, int64_t V, double* z) {
  for (int64_t v = 0; v < V; ++v) {
    const double* w = W + v * H;
    double s = 0.0;
    for (int64_t k = 0; k < H; ++k) s += h[k] * w[k];
    z[v] = s;
  }
}

/* log sum_v exp z_v, shifted by the maximum for range safety. */
static double logsumexp(const double* z, int64_t V) {
  double m = z[0];
  for (int64_t v = 1; v < V; ++v)
    if (z[v] > m) m = z[v];
  double s = 0.0;
  for (int64_t v = 0; v < V; ++v) s += exp(z[v] - m);
  return m + log(s);
}

/* For each of n tokens (hidden row h_i, sampled id y_i): lse_i and
 * logp_i = z_{i,y_i} - lse_i. Also returns z_{i,y_i} when zy != NULL. */
void oracle_score_rows(const double* h, const double* W, const int64_t* y, int64_t n,
                       int64_t H, int64_t V, double* lse, double* logp, double* zy) {
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)V);
#pragma omp for schedule(dynamic, 1)
    for (int64_t i = 0; i < n; ++i) {
      logits_row(h + i * H, W, H, V, z);
      double l = logsumexp(z, V);
      lse[i] = l;
      logp[i] = z[y[i]] - l;
      if (zy) zy[i] = z[y[i]];
    }
    free(z);
  }
}

/* ------------------------------------------------ Eq. 1, per token term */
/* rho = exp(logp - old); clip(rho) to [1-eps, 1+eps];
 * pg = -min(rho*A, clip(rho)*A); kl = exp(ref - logp) - (ref - logp) - 1;
 * ell = pg + beta*kl. The per-token gradient weight is
 *   g = d(c * ell)/d logp = c * (-A*rho*[rho*A <= clip(rho)*A] + beta*(1 - exp(ref - logp)))
 * where the clipped branch has zero slope (the clip is a constant there) and
 * a tie goes to the unclipped branch. clipped[i] = 1 when the clipped branch
 * was taken. A masked token (m = 0) gets ell = g = 0. */
void oracle_token_objective(const double* logp, const double* old_logp, const double* ref_logp,
                            const double* adv, const double* c, const uint8_t* m, int64_t n,
                            double eps, double beta, double* ell, double* g,
                            uint8_t* clipped) {
  for (int64_t i = 0; i < n; ++i) {
    if (m != NULL && !m[i]) {
      ell[i] = 0.0;
      g[i] = 0.0;
      if (clipped) clipped[i] = 0;
      continue;
    }
    double rho = exp(logp[i] - old_logp[i]);
    double rc = rho < 1.0 - eps ? 1.0 - eps : (rho > 1.0 + eps ? 1.0 + eps : rho);
    double u = rho * adv[i];
    double cl = rc * adv[i];
    double pg = -(u < cl ? u : cl);
    double d = ref_logp[i] - logp[i];
    double ed = exp(d);
    double kl = ed - d - 1.0;
    ell[i] = pg + beta * kl;
    int unclipped = (u <= cl);
    double dpg = unclipped ? -adv[i] * rho : 0.0;
    g[i] = c[i] * (dpg + beta * (1.0 - ed));
    if (clipped) clipped[i] = (uint8_t)(!unclipped);
  }
}

/* ---------------------------------------------------------- gradients */
/* dL/dz_{i,v} = g_i * (1[v = y_i] - exp(z_{i,v} - lse_i)), and
 * dL/dh_i = sum_v dL/dz_{i,v} W_v, for each of n tokens. */
void oracle_grad_hidden_rows(const double* h, const double* W, const int64_t* y,
                             const double* lse, const double* g, int64_t n, int64_t H, int64_t V,
                             double* dh) {
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)V);
#pragma omp for schedule(dynamic, 1)
    for (int64_t i = 0; i < n; ++i) {
      double* out = dh + i * H;
      for (int64_t k = 0; k < H; ++k) out[k] = 0.0;
      if (g[i] == 0.0) continue;
      logits_row(h + i * H, W, H, V, z);
      for (int64_t v = 0; v < V; ++v) {
        double dz = g[i] * ((v == y[i] ? 1.0 : 0.0) - exp(z[v] - lse[i]));
        const double* w = W + v * H;
        for (int64_t k = 0; k < H; ++k) out[k] += dz * w[k];
      }
    }
    free(z);
  }
}

/* dL/dW_v = sum_i dL/dz_{i,v} h_i over all n tokens, for the nv vocabulary
 * rows listed in vrows (all rows when vrows == NULL, nv = V). */
void oracle_grad_weight_rows(const double* h, const double* W, const int64_t* y,
                             const double* lse, const double* g, int64_t n, int64_t H, int64_t V,
                             const int64_t* vrows, int64_t nv, double* dW) {
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t j = 0; j < nv; ++j) {
    int64_t v = vrows ? vrows[j] : j;
    const double* w = W + v * H;
    double* out = dW + j * H;
    for (int64_t k = 0; k < H; ++k) out[k] = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      if (g[i] == 0.0) continue;
      const double* hi = h + i * H;
      double z = 0.0;
      for (int64_t k = 0; k < H; ++k) z += hi[k] * w[k];
      double dz = g[i] * ((v == y[i] ? 1.0 : 0.0) - exp(z - lse[i]));
      for (int64_t k = 0; k < H; ++k) out[k] += dz * hi[k];
    }
  }
}

/* --------------------------------------------- the whole loss, composed */
/* Full loss and gradients for a problem small enough to score every row.
 * Inputs are per padded row (N rows; h is [N,H], W is [V,H]); adv is one
 * value per rollout. Outputs (any may be NULL except loss): per-row lse,
 * logp, ell, g, clipped (zeros on masked rows), dh [N,H] (zero rows where
 * masked) and dW [V,H]. Returns the number of valid rows. */
int64_t oracle_grpo_loss(const double* h, const double* W, const int64_t* y, const uint8_t* mask,
                         const int64_t* cu_seqlens, int64_t num_seqs, int64_t N, int64_t H,
                         int64_t V, const double* old_logp, const double* ref_logp,
                         const double* adv_seq, double eps, double beta, int agg, double* loss,
                         double* lse_out, double* logp_out, double* ell_out, double* g_out,
                         uint8_t* clipped_out, double* dh, double* dW) {
  int64_t* counts = (int64_t*)malloc(sizeof(int64_t) * (size_t)num_seqs);
  int64_t* seq = (int64_t*)malloc(sizeof(int64_t) * (size_t)N);
  double* cseq = (double*)malloc(sizeof(double) * (size_t)num_seqs);
  double* lse = (double*)calloc((size_t)N, sizeof(double));
  double* logp = (double*)calloc((size_t)N, sizeof(double));
  double* ell = (double*)calloc((size_t)N, sizeof(double));
  double* g = (double*)calloc((size_t)N, sizeof(double));
  double* a_tok = (double*)calloc((size_t)N, sizeof(double));
  double* c_tok = (double*)calloc((size_t)N, sizeof(double));
  uint8_t* clipped = (uint8_t*)calloc((size_t)N, 1);
  int64_t nvalid = oracle_pack_valid(mask, cu_seqlens, num_seqs, NULL, counts, seq);
  oracle_seq_weights(counts, num_seqs, agg, cseq);

  /* every row is scored; masked rows are zeroed afterwards */
  oracle_score_rows(h, W, y, N, H, V, lse, logp, NULL);
  for (int64_t t = 0; t < N; ++t) {
    a_tok[t] = adv_seq[seq[t]];
    c_tok[t] = cseq[seq[t]];
  }
  oracle_token_objective(logp, old_logp, ref_logp, a_tok, c_tok, mask, N, eps, beta, ell, g,
                         clipped);
  double L = 0.0;
  for (int64_t b = 0; b < num_seqs; ++b) {
    double s = 0.0;
    for (int64_t t = cu_seqlens[b]; t < cu_seqlens[b + 1]; ++t)
      if (mask == NULL || mask[t]) s += ell[t];
    L += cseq[b] * s;
  }
  *loss = L;
  for (int64_t t = 0; t < N; ++t) {
    int valid = (mask == NULL || mask[t]);
    if (lse_out) lse_out[t] = valid ? lse[t] : 0.0;
    if (logp_out) logp_out[t] = valid ? logp[t] : 0.0;
    if (ell_out) ell_out[t] = ell[t];
    if (g_out) g_out[t] = g[t];
    if (clipped_out) clipped_out[t] = clipped[t];
  }
  if (dh) oracle_grad_hidden_rows(h, W, y, lse, g, N, H, V, dh);
  if (dW) oracle_grad_weight_rows(h, W, y, lse, g, N, H, V, NULL, V, dW);
  free(counts); free(seq); free(cseq); free(lse); free(logp); free(ell); free(g);
  free(a_tok); free(c_tok); free(clipped);
  return nvalid;
}

/* ------------------------------------------------------- SFT (Sec. 3.2) */
/* Supervised cross-entropy over the valid rows (mask NULL = all rows):
 * loss = -(1/n) sum_{valid t} logp_t, n = number of valid rows (loss 0 when
 * n = 0). dL/dlogp_t = -1/n on valid rows and 0 elsewhere; dh and dW follow
 * through the log-softmax with the row gradient functions above. Outputs
 * other than loss may be NULL. Returns n. */
int64_t oracle_sft_ce(const double* h, const double* W, const int64_t* y, const uint8_t* mask,
                      int64_t N, int64_t H, int64_t V, double* loss, double* lse_out,
                      double* logp_out, double* g_out, double* dh, double* dW) {
  double* lse = (double*)calloc((size_t)N, sizeof(double));
  double* logp = (double*)calloc((size_t)N, sizeof(double));
  double* g = (double*)calloc((size_t)N, sizeof(double));
  int64_t n = 0;
  for (int64_t t = 0; t < N; ++t)
    if (mask == NULL || mask[t]) ++n;
  oracle_score_rows(h, W, y, N, H, V, lse, logp, NULL);
  double s = 0.0;
  for (int64_t t = 0; t < N; ++t) {
    int valid = (mask == NULL || mask[t]);
    if (valid) {
      s += logp[t];
      g[t] = -1.0 / (double)n;
    } else {
      lse[t] = 0.0;
      logp[t] = 0.0;
      g[t] = 0.0;
    }
  }
  *loss = n > 0 ? -s / (double)n : 0.0;
  if (lse_out) memcpy(lse_out, lse, sizeof(double) * (size_t)N);
  if (logp_out) memcpy(logp_out, logp, sizeof(double) * (size_t)N);
  if (g_out) memcpy(g_out, g, sizeof(double) * (size_t)N);
  if (dh) oracle_grad_hidden_rows(h, W, y, lse, g, N, H, V, dh);
  if (dW) oracle_grad_weight_rows(h, W, y, lse, g, N, H, V, NULL, V, dW);
  free(lse); free(logp); free(g);
  return n;
}
