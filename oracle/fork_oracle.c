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

/* Statistics of q(. | x_t) for one position, from the definitions in Section 2
 * (the model's per-position categorical, the greedy candidate and its
 * confidence) and Section 3.1 (token entropy).  Returns 0, or -2 when a logit
 * is not finite. */
static int one_row(const void* hidden, const void* W, int dtype, int64_t d,
                   int64_t V, int64_t r, double* z, double* conf,
                   double* entropy, double* logp, double* lse, int32_t* amax,
                   double* gap) {
  /* logits z_v = <h_r, W_v>, accumulated with j ascending */
  for (int64_t v = 0; v < V; ++v) {
    double acc = 0.0;
    for (int64_t j = 0; j < d; ++j)
      acc += widen(hidden, dtype, r * d + j) * widen(W, dtype, v * d + j);
    if (!isfinite(acc)) return -2;
    z[v] = acc;
  }
  /* greedy candidate: the lowest index attaining the maximum logit */
  int64_t a = 0;
  for (int64_t v = 1; v < V; ++v)
    if (z[v] > z[a]) a = v;
  double zmax = z[a];
  /* log-normaliser, shifted by the maximum so that exp() cannot overflow */
  double sum = 0.0;
  for (int64_t v = 0; v < V; ++v) sum += exp(z[v] - zmax);
  double log_norm = zmax + log(sum);
  /* entropy -sum q log q with log q_v = z_v - log_norm */
  double h = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double lq = z[v] - log_norm;
    h -= exp(lq) * lq;
  }
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
