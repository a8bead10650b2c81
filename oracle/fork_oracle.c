/*
 * fork_oracle.c -- plain binary64 CPU oracle for one Fork-dLLM step.
 *
 * TEST INFRASTRUCTURE ONLY (see fork_oracle.h): used by the tests, the smoke
 * check and the CPU-baseline leg of the benchmark; never by the product path.
 *
 * The code is deliberately slow and direct: one row at a time, every logit
 * materialised, two plain passes for the normaliser, the entropy written as
 * its definition.  OpenMP only distributes independent rows.
 */
#include "fork_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Exact widening of one stored element to binary64.  A bf16 value is the top
 * 16 bits of a binary32 value, so shifting it into place is exact. */
static double widen(const void* base, int dtype, int64_t idx) {
  if (dtype == ORACLE_BF16) {
    uint16_t h = ((const uint16_t*)base)[idx];
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return (double)((const float*)base)[idx];
}

/* Logits of position r, z_v = <h_r, W_v>, accumulated with j ascending.
 * Returns 0, or -2 when a logit is not finite. */
static int logits(const void* hidden, const void* W, int dtype, int64_t d,
                  int64_t V, int64_t r, double* z) {
  for (int64_t v = 0; v < V; ++v) {
    double acc = 0.0;
    for (int64_t j = 0; j < d; ++j)
      acc += widen(hidden, dtype, r * d + j) * widen(W, dtype, v * d + j);
    if (!isfinite(acc)) return -2;
    z[v] = acc;
  }
  return 0;
}

/* log sum_v exp(z_v), shifted by the maximum so that exp() cannot overflow */
static double log_normaliser(const double* z, int64_t V) {
  double zmax = z[0];
  for (int64_t v = 1; v < V; ++v)
    if (z[v] > zmax) zmax = z[v];
  double sum = 0.0;
  for (int64_t v = 0; v < V; ++v) sum += exp(z[v] - zmax);
  return zmax + log(sum);
}

/* entropy -sum_v q_v log q_v with log q_v = z_v - log_norm (Section 3.1) */
static double entropy_of(const double* z, int64_t V, double log_norm) {
  double h = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double lq = z[v] - log_norm;
    h -= exp(lq) * lq;
  }
  return h;
}

/* Statistics of q(. | x_t) for one position, from the definitions in Section 2
 * (the model's per-position categorical, the greedy candidate and its
 * confidence) and Section 3.1 (token entropy).  Returns 0, or -2 when a logit
 * is not finite. */
static int one_row(const void* hidden, const void* W, int dtype, int64_t d,
                   int64_t V, int64_t r, double* z, double* conf,
                   double* entropy, double* logp, double* lse, int32_t* amax,
                   double* gap) {
  const int rc = logits(hidden, W, dtype, d, V, r, z);
  if (rc) return rc;
  /* greedy candidate: the lowest index attaining the maximum logit */
  int64_t a = 0;
  for (int64_t v = 1; v < V; ++v)
    if (z[v] > z[a]) a = v;
  double zmax = z[a];
  double log_norm = log_normaliser(z, V);
  double h = entropy_of(z, V, log_norm);
  /* gap to the runner-up (any index other than a) */
  double second = -INFINITY;
  for (int64_t v = 0; v < V; ++v)
    if (v != a && z[v] > second) second = z[v];
  if (conf) *conf = exp(z[a] - log_norm);
  if (logp) *logp = z[a] - log_norm;
  if (lse) *lse = log_norm;
  if (entropy) *entropy = h;
  if (amax) *amax = (int32_t)a;
  if (gap) *gap = (V > 1) ? (zmax - second) : 0.0;
  return 0;
}

int oracle_row_stats(const void* hidden, const void* W, int dtype, int64_t d,
                     int64_t V, const int64_t* rows, int64_t nrows,
                     double* conf, double* entropy, double* logp, double* lse,
                     int32_t* argmax, double* gap, int nthreads) {
  if (!hidden || !W || !rows || d <= 0 || V <= 0 || V > INT32_MAX || nrows < 0)
    return -1;
  if (dtype != ORACLE_BF16 && dtype != ORACLE_F32) return -1;
  int status = 0;
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc((size_t)V * sizeof(double));
    if (!z) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      status = -1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t i = 0; i < nrows; ++i) {
        int rc = one_row(hidden, W, dtype, d, V, rows[i], z,
                         conf ? conf + i : NULL, entropy ? entropy + i : NULL,
                         logp ? logp + i : NULL, lse ? lse + i : NULL,
                         argmax ? argmax + i : NULL, gap ? gap + i : NULL);
        if (rc) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
          status = rc;
        }
      }
      free(z);
    }
  }
  (void)nthreads;
  return status;
}

/* ---------------------------------------------------------------- sampling */

/* One Philox round: two 32x32 -> 64-bit products, their halves exchanged and
 * mixed with the other two counter words and the round key. */
static void philox_round(uint32_t c[4], const uint32_t k[2]) {
  const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
  const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
  const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  const uint32_t n0 = hi1 ^ c[1] ^ k[0];
  const uint32_t n2 = hi0 ^ c[3] ^ k[1];
  c[0] = n0;
  c[1] = lo1;
  c[2] = n2;
  c[3] = lo0;
}

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                          uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k[2] = {key[0], key[1]};
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {  /* Weyl sequence of round keys */
      k[0] += 0x9E3779B9u;
      k[1] += 0xBB67AE85u;
    }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof c);
}

double oracle_exp_draw(uint64_t seed, uint32_t counter, int64_t row, int64_t v,
                       double* u) {
  const uint32_t ctr[4] = {(uint32_t)(v / 4), (uint32_t)row, counter, 0u};
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  oracle_philox4x32_10(ctr, key, w);
  const double U = ldexp(2.0 * (double)(w[v % 4] >> 9) + 1.0, -24);
  if (u) *u = U;
  return -log1p(-U);
}

/* The drawn candidate of one position: the Gumbel-perturbed,
 * temperature-scaled logits and their maximiser. */
static int one_sample(const void* hidden, const void* W, int dtype, int64_t d,
                      int64_t V, int64_t r, double tau, uint64_t seed,
                      uint32_t counter, double* z, int32_t* cand, double* conf,
                      double* logp, double* keygap) {
  const int rc = logits(hidden, W, dtype, d, V, r, z);
  if (rc) return rc;
  const double log_norm = log_normaliser(z, V);
  /* keys z_v / tau + g_v with g_v = -log E_v; best and runner-up */
  int64_t a = -1;
  double best = -INFINITY, second = -INFINITY;
  for (int64_t v = 0; v < V; ++v) {
    const double key = z[v] / tau - log(oracle_exp_draw(seed, counter, r, v, NULL));
    if (a < 0 || key > best) {
      second = best;
      best = key;
      a = v;
    } else if (key > second) {
      second = key;
    }
  }
  const double log_q = z[a] - log_norm;  /* untempered log q of the draw */
  if (cand) *cand = (int32_t)a;
  if (conf) *conf = exp(log_q);
  if (logp) *logp = log_q;
  if (keygap) *keygap = (V > 1) ? (best - second) : 0.0;
  return 0;
}

int oracle_row_sample(const void* hidden, const void* W, int dtype, int64_t d,
                      int64_t V, const int64_t* rows, int64_t nrows,
                      double tau, uint64_t seed, uint32_t counter,
                      int32_t* cand, double* conf, double* logp,
                      double* keygap, int nthreads) {
  if (!hidden || !W || !rows || d <= 0 || V <= 0 || V > INT32_MAX || nrows < 0)
    return -1;
  if (dtype != ORACLE_BF16 && dtype != ORACLE_F32) return -1;
  if (!(tau > 0.0) || !isfinite(tau)) return -1;
  int status = 0;
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc((size_t)V * sizeof(double));
    if (!z) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      status = -1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t i = 0; i < nrows; ++i) {
        int rc = one_sample(hidden, W, dtype, d, V, rows[i], tau, seed, counter, z,
                            cand ? cand + i : NULL, conf ? conf + i : NULL,
                            logp ? logp + i : NULL, keygap ? keygap + i : NULL);
        if (rc) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
          status = rc;
        }
      }
      free(z);
    }
  }
  (void)nthreads;
  return status;
}

/* ---------------------------------------------------------------- selection */

/* The single position committed on a fallback step, among the masked
 * positions of [s, e) of sequence row `base`. */
static int32_t fallback_pick(int rule, const double* conf, const double* entropy,
                             const float* uniform, int32_t b, int64_t base,
                             const uint8_t* mask, int32_t s, int32_t e) {
  int32_t pick = -1;
  if (rule == ORACLE_RULE_RANDOM) {
    int32_t n = 0;
    for (int32_t k = s; k < e; ++k) n += mask[base + k] ? 1 : 0;
    float prod = uniform[b] * (float)n;  /* binary32, as the method's draw */
    int32_t j = (int32_t)prod;
    if (j > n - 1) j = n - 1;
    if (j < 0) j = 0;
    for (int32_t k = s; k < e; ++k)
      if (mask[base + k] && j-- == 0) return k;
    return -1;
  }
  for (int32_t k = s; k < e; ++k) {
    if (!mask[base + k]) continue;
    if (pick < 0) {
      pick = k;
      if (rule == ORACLE_RULE_LEFTMOST) break;
      continue;
    }
    const double* key = rule == ORACLE_RULE_MAXENT ? entropy : conf;
    const double cand = key[base + k], best = key[base + pick];
    const int better = rule == ORACLE_RULE_MINCONF ? (cand < best) : (cand > best);
    if (better) pick = k;
  }
  return pick;
}

/* Algorithm 2 (Fork-dLLM), Algorithm 1 (Fast-dLLM) and the fallback
 * ablations of Section 4.1, applied inside the active block of the
 * semi-autoregressive regime (Section 4.1, block length BL); the fallback
 * flag is membership of the step in F_i (Section 3.2). */
int oracle_select_ex(int32_t B, int32_t L, int32_t block_len, const double* conf,
                     const double* entropy, const float* uniform,
                     const int32_t* argmax_tok, double lambda, int rule,
                     int32_t* tokens, uint8_t* mask, int32_t* block_start,
                     int32_t* fallback, int32_t* ncommit) {
  if (B <= 0 || L <= 0 || block_len <= 0 || !conf || !argmax_tok || !tokens ||
      !mask || !block_start || !fallback)
    return -1;
  if (rule < ORACLE_RULE_LEFTMOST || rule > ORACLE_RULE_RANDOM) return -1;
  if (rule == ORACLE_RULE_MAXENT && !entropy) return -1;
  if (rule == ORACLE_RULE_RANDOM && !uniform) return -1;
  for (int32_t b = 0; b < B; ++b) {
    const int64_t base = (int64_t)b * L;
    if (block_start[b] < 0 || block_start[b] > L) return -1;
    /* find the active block: first block from block_start holding a mask */
    int32_t s = block_start[b];
    int found = 0;
    while (s < L) {
      int32_t e = s + block_len < L ? s + block_len : L;
      for (int32_t k = s; k < e; ++k)
        if (mask[base + k]) found = 1;
      if (found) break;
      s += block_len;
    }
    if (!found) {
      fallback[b] = -1;
      if (ncommit) ncommit[b] = 0;
      continue;
    }
    const int32_t e = s + block_len < L ? s + block_len : L;
    /* the threshold set U (strict comparison) */
    uint8_t* in_u = (uint8_t*)calloc((size_t)(e - s), 1);
    if (!in_u) return -1;
    int32_t n = 0;
    for (int32_t k = s; k < e; ++k)
      if (mask[base + k] && conf[base + k] > lambda) {
        in_u[k - s] = 1;
        ++n;
      }
    if (n == 0) {
      /* fallback: exactly one position */
      const int32_t pick = fallback_pick(rule, conf, entropy, uniform, b, base, mask, s, e);
      if (pick < s || pick >= e) {
        free(in_u);
        return -1;
      }
      in_u[pick - s] = 1;
      n = 1;
      fallback[b] = 1;
    } else {
      fallback[b] = 0;
    }
    for (int32_t k = s; k < e; ++k)
      if (in_u[k - s]) {
        tokens[base + k] = argmax_tok[base + k];
        mask[base + k] = 0;
      }
    free(in_u);
    block_start[b] = s;
    if (ncommit) ncommit[b] = n;
  }
  return 0;
}

int oracle_select(int32_t B, int32_t L, int32_t block_len, const double* conf,
                  const int32_t* argmax_tok, double lambda, int rule,
                  int32_t* tokens, uint8_t* mask, int32_t* block_start,
                  int32_t* fallback, int32_t* ncommit) {
  if (rule != ORACLE_RULE_LEFTMOST && rule != ORACLE_RULE_MAXCONF) return -1;
  return oracle_select_ex(B, L, block_len, conf, NULL, NULL, argmax_tok, lambda,
                          rule, tokens, mask, block_start, fallback, ncommit);
}

/* ------------------------------------------------------------ ForkGRPO */

int oracle_token_logprob(const void* hidden, const void* W, int dtype,
                         int64_t M, int64_t d, int64_t V, const int64_t* rows,
                         const int32_t* tokens, int64_t n, double* logp,
                         double* entropy, int nthreads) {
  if (!hidden || !W || (n > 0 && (!rows || !tokens || !logp)) || M <= 0 || d <= 0 ||
      V <= 0 || V > INT32_MAX || n < 0)
    return -1;
  if (dtype != ORACLE_BF16 && dtype != ORACLE_F32) return -1;
  for (int64_t e = 0; e < n; ++e)
    if (rows[e] < 0 || rows[e] >= M || tokens[e] < 0 || tokens[e] >= V) return -1;
  int status = 0;
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc((size_t)V * sizeof(double));
    if (!z) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      status = -1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t e = 0; e < n; ++e) {
        int rc = logits(hidden, W, dtype, d, V, rows[e], z);
        if (rc) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
          status = rc;
          continue;
        }
        const double log_norm = log_normaliser(z, V);
        /* log q of the given token: its logit against the normaliser */
        logp[e] = z[tokens[e]] - log_norm;
        if (entropy) entropy[e] = entropy_of(z, V, log_norm);
      }
      free(z);
    }
  }
  (void)nthreads;
  return status;
}

int oracle_grpo_objective(int32_t n_groups, int32_t G, const double* rewards,
                          const int32_t* offsets, const double* lp_new,
                          const double* lp_old, double eps, double* adv,
                          double* ratio, double* term, double* rollout_obj,
                          double* group_obj, uint8_t* skipped, double* J) {
  if (n_groups < 0 || G <= 0 || !rewards || !offsets || !(eps >= 0.0)) return -1;
  const int64_t R = (int64_t)n_groups * G;
  if (offsets[0] != 0) return -1;
  for (int64_t i = 0; i < R; ++i)
    if (offsets[i + 1] < offsets[i]) return -1;
  if (offsets[R] > 0 && (!lp_new || !lp_old)) return -1;
  double total = 0.0;
  int32_t kept = 0;
  for (int32_t g = 0; g < n_groups; ++g) {
    const double* r = rewards + (int64_t)g * G;
    /* group mean and standard deviation (divisor G) of the rewards */
    double mean = 0.0;
    for (int32_t j = 0; j < G; ++j) mean += r[j];
    mean /= G;
    double var = 0.0;
    for (int32_t j = 0; j < G; ++j) var += (r[j] - mean) * (r[j] - mean);
    const double sd = sqrt(var / G);
    const int skip = !(sd > 0.0);
    double gsum = 0.0;
    for (int32_t j = 0; j < G; ++j) {
      const int64_t i = (int64_t)g * G + j;
      const double A = skip ? 0.0 : (r[j] - mean) / sd;
      if (adv) adv[i] = A;
      double acc = 0.0;
      const int32_t nF = offsets[i + 1] - offsets[i];
      for (int32_t e = offsets[i]; e < offsets[i + 1]; ++e) {
        const double rho = exp(lp_new[e] - lp_old[e]);
        const double clipped = rho < 1.0 - eps ? 1.0 - eps : (rho > 1.0 + eps ? 1.0 + eps : rho);
        const double a = rho * A, b = clipped * A;
        const double tm = a < b ? a : b;
        if (ratio) ratio[e] = rho;
        if (term) term[e] = tm;
        acc += tm;
      }
      const double ro = nF > 0 ? acc / nF : 0.0;
      if (rollout_obj) rollout_obj[i] = ro;
      gsum += ro;
    }
    const double go = skip ? 0.0 : gsum / G;
    if (group_obj) group_obj[g] = go;
    if (skipped) skipped[g] = (uint8_t)skip;
    if (!skip) {
      total += go;
      ++kept;
    }
  }
  if (J) *J = kept > 0 ? total / kept : 0.0;
  return 0;
}

int oracle_top_entropy(int32_t R, int32_t Lg, int32_t k, const double* entropy,
                       uint8_t* sel) {
  if (R < 0 || Lg <= 0 || k < 0 || k > Lg || (R > 0 && (!entropy || !sel))) return -1;
  for (int32_t i = 0; i < R; ++i) {
    const double* h = entropy + (int64_t)i * Lg;
    uint8_t* out = sel + (int64_t)i * Lg;
    /* a position is chosen when fewer than k positions come before it in
       the order (higher entropy first, then lower position) */
    for (int32_t p = 0; p < Lg; ++p) {
      int32_t ahead = 0;
      for (int32_t q = 0; q < Lg; ++q)
        if (h[q] > h[p] || (h[q] == h[p] && q < p)) ++ahead;
      out[p] = (uint8_t)(ahead < k);
    }
  }
  return 0;
}
