/*
 * fork_oracle.h -- CPU reference (oracle) for one Fork-dLLM denoising step.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing on the product path links, loads or calls
 * this code; only the test suite, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant with the HIP
 * library, and it does not include any HIP header.
 *
 * Everything is computed in IEEE binary64 from the same input bits the GPU
 * path reads (bf16 or binary32 values are widened exactly).  No blocking,
 * fusion or re-ordering is applied beyond what the definitions state.
 *
 * Paper: "Fork-dLLM: Avoiding the Flexibility Trap in Diffusion Language
 * Models", Section 2 (Sampling in masked dLLMs), Algorithm 2 (Fork-dLLM),
 * Algorithm 1 (Fast-dLLM, for the differential tests), Section 3.2 (fallback
 * step set F_i and the ratio at k_{i,t}).
 */
#ifndef FORK_ORACLE_H
#define FORK_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_BF16 = 0, ORACLE_F32 = 1 };
enum { ORACLE_RULE_LEFTMOST = 0,   /* Fork-dLLM fallback (Algorithm 2)      */
       ORACLE_RULE_MAXCONF = 1,    /* Fast-dLLM fallback (Algorithm 1)      */
       ORACLE_RULE_MINCONF = 2,    /* ablations of Section 4.1: lowest      */
       ORACLE_RULE_MAXENT = 3,     /*   confidence, highest entropy,        */
       ORACLE_RULE_RANDOM = 4 };   /*   uniformly random masked position    */

/*
 * Per-position statistics of the model distribution q^k(. | x_t) for the
 * rows listed in `rows` (indices into the [M, d] hidden matrix).
 *
 *   z_v      = sum_j h_j * W[v, j]               (j ascending, binary64)
 *   argmax   = lowest v with z_v = max_u z_u      (greedy candidate x_0^k)
 *   lse      = log sum_v exp(z_v)
 *   conf     = q(argmax) = exp(z_argmax - lse)   (confidence c_t^k)
 *   logp     = log q(argmax) = z_argmax - lse    (numerator/denominator of rho)
 *   entropy  = -sum_v q_v log q_v                 (nats)
 *   gap      = z_argmax - max_{v != argmax} z_v  (0 if V == 1; tie diagnostics)
 *
 * Any output pointer may be NULL.  Outputs are indexed by position in `rows`.
 * nthreads <= 0 means "use OpenMP's default".  Returns 0, or -1 on bad
 * arguments, -2 if a logit is not finite.
 */
int oracle_row_stats(const void* hidden, const void* W, int dtype,
                     int64_t d, int64_t V,
                     const int64_t* rows, int64_t nrows,
                     double* conf, double* entropy, double* logp, double* lse,
                     int32_t* argmax, double* gap, int nthreads);

/*
 * One application of the unmasking rule to B sequences of length L, in place.
 *
 * Active block of sequence b: the first block [s, min(s+BL, L)) with
 * s = block_start[b] + j*BL (j = 0, 1, ...) that holds a masked position.
 * Inside it, with M the masked positions:
 *   U = { k in M : conf[k] > lambda }                       (strict)
 *   if U is empty:  U = { leftmost(M) }       (rule LEFTMOST, Algorithm 2)
 *                   U = { argmax_k conf[k] }  (rule MAXCONF,  Algorithm 1;
 *                                              ties -> lowest k)
 *   tokens[k] = argmax_tok[k], mask[k] = 0 for k in U.
 * fallback[b] = 1 if U was empty before the fallback, 0 otherwise, and -1
 * (nothing written, block_start unchanged) when no masked position exists at
 * or after block_start[b].  block_start[b] is set to the active block's start.
 * ncommit[b] (may be NULL) receives |U|.
 * Arrays conf / argmax_tok / tokens / mask are [B*L], row b*L + position.
 * Returns 0, or -1 on bad arguments.
 */
int oracle_select(int32_t B, int32_t L, int32_t block_len,
                  const double* conf, const int32_t* argmax_tok,
                  double lambda, int rule,
                  int32_t* tokens, uint8_t* mask, int32_t* block_start,
                  int32_t* fallback, int32_t* ncommit);

/*
 * oracle_select with the fallback ablations of Section 4.1 as well:
 *   MINCONF: the masked position of lowest confidence (lowest k on ties);
 *   MAXENT:  the masked position of highest entropy (lowest k on ties);
 *   RANDOM:  with n masked positions in the block and u = uniform[b] in
 *            [0, 1), the j-th of them in increasing order, j = (int)(u * n)
 *            evaluated in binary32 and capped at n - 1.
 * entropy ([B*L]) is read by MAXENT only, uniform ([B]) by RANDOM only; either
 * may be NULL when its rule is not used.
 */
int oracle_select_ex(int32_t B, int32_t L, int32_t block_len,
                     const double* conf, const double* entropy,
                     const float* uniform, const int32_t* argmax_tok,
                     double lambda, int rule,
                     int32_t* tokens, uint8_t* mask, int32_t* block_start,
                     int32_t* fallback, int32_t* ncommit);

/*
 * Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and
 * Shaw ("Parallel random numbers: as easy as 1, 2, 3", SC'11): ten rounds of
 * the 4x32 Philox S-box on the counter, the key bumped by the Weyl constants
 * between rounds.
 */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                          uint32_t out[4]);

/*
 * The random draw attached to vocabulary entry v of position `row` in the
 * sampled-candidate step (`counter` is the caller's step counter):
 *   w = Philox4x32-10(ctr = (v / 4, row, counter, 0),
 *                     key = (seed mod 2^32, seed / 2^32))[v mod 4]
 *   U = (2 * (w >> 9) + 1) * 2^-24        (uniform on an odd grid in (0, 1))
 *   E = -log(1 - U)                       (standard exponential)
 * Returns E; *u (may be NULL) receives U.
 */
double oracle_exp_draw(uint64_t seed, uint32_t counter, int64_t row, int64_t v,
                       double* u);

/*
 * Sampled candidates at temperature tau > 0 (Section 2: the candidate is
 * drawn from q^k(. | x_t; tau), the softmax of z / tau), by the Gumbel-max
 * property: -log E_v is a standard Gumbel variable, so
 *   cand   = argmax_v  z_v / tau - log E_v            (lowest v on ties)
 * is distributed as softmax(z / tau).  With lse = log sum_v exp(z_v):
 *   conf   = exp(z_cand - lse)      (untempered q of the drawn token)
 *   logp   = z_cand - lse
 *   keygap = key_cand - max_{v != cand} key_v          (0 if V == 1)
 * Rows, outputs and return codes as in oracle_row_stats; -1 also when tau is
 * not a positive finite number.
 */
int oracle_row_sample(const void* hidden, const void* W, int dtype,
                      int64_t d, int64_t V,
                      const int64_t* rows, int64_t nrows,
                      double tau, uint64_t seed, uint32_t counter,
                      int32_t* cand, double* conf, double* logp,
                      double* keygap, int nthreads);

/*
 * Teacher-forced log-probabilities (the numerator and denominator of the
 * ForkGRPO ratio, Section 3.2): for each entry e, with z the logits of
 * hidden row rows[e],
 *   logp[e]    = z_{tokens[e]} - log sum_v exp(z_v)
 *   entropy[e] = -sum_v q_v log q_v            (may be NULL)
 * Returns 0, -1 on bad arguments (a row outside [0, M) or a token outside
 * [0, V) included), -2 if a logit is not finite.
 */
int oracle_token_logprob(const void* hidden, const void* W, int dtype,
                         int64_t M, int64_t d, int64_t V,
                         const int64_t* rows, const int32_t* tokens, int64_t n,
                         double* logp, double* entropy, int nthreads);

/*
 * The ForkGRPO objective of Section 3.2 on one batch of n_groups prompts
 * with G rollouts each (rollout i = g * G + j).  Entries e of rollout i
 * (its fallback steps t in F_i) are [offsets[i], offsets[i+1]).
 *   A_i          = (r_i - mean_g) / std_g     (group-normalised advantage;
 *                  std over the G rewards of the group, divisor G)
 *   groups with std_g == 0 are skipped: their A_i = 0 and they are left out
 *   of the mean below (group_obj = 0, skipped[g] = 1)
 *   ratio[e]     = exp(lp_new[e] - lp_old[e])
 *   term[e]      = min(ratio * A_i, clip(ratio, 1 - eps, 1 + eps) * A_i)
 *   rollout_obj  = (1 / |F_i|) sum_{e in F_i} term[e]    (0 if F_i is empty)
 *   group_obj[g] = (1 / G) sum_{i in g} rollout_obj[i]
 *   *J           = mean of group_obj over the groups not skipped (0 if none)
 * Any output array may be NULL.  Returns 0, or -1 on bad arguments.
 */
int oracle_grpo_objective(int32_t n_groups, int32_t G, const double* rewards,
                          const int32_t* offsets, const double* lp_new,
                          const double* lp_old, double eps, double* adv,
                          double* ratio, double* term, double* rollout_obj,
                          double* group_obj, uint8_t* skipped, double* J);

/*
 * JustGRPO-Fast position selection (Section 3.2): in each of R rollouts of
 * Lg positions, the k positions of highest entropy (entropy[i * Lg + p]);
 * equal entropies are taken in increasing position.  sel[i * Lg + p] = 1 for
 * the chosen positions, 0 otherwise.  Returns 0, or -1 on bad arguments
 * (k outside [0, Lg] included).
 */
int oracle_top_entropy(int32_t R, int32_t Lg, int32_t k, const double* entropy,
                       uint8_t* sel);

#ifdef __cplusplus
}
#endif
#endif
