/*
 * fork_step.h -- C ABI of the MI355X (gfx950) Fork-dLLM denoising step.
 *
 * One call performs one denoising step of the Fork-dLLM sampler (Fork-dLLM
 * paper, Section 2 "Sampling in masked dLLMs" and Algorithm 2) for B
 * sequences of L positions:
 *
 *   1. logits z[r, v] = sum_j hidden[r, j] * W_head[v, j] for every position
 *      r < B*L and vocabulary entry v < V (the LM-head projection that yields
 *      the model's per-position categorical q^k(. | x_t));
 *   2. per position: greedy candidate x_0 = argmax_v z (lowest v on ties),
 *      confidence c = q(x_0) (Section 2), log q(x_0) (the quantity inside the
 *      ForkGRPO ratio, Section 3.2), entropy -sum q log q in nats (Section
 *      3.1) and, optionally, the log-normaliser;
 *   3. per sequence, inside its active block of the semi-autoregressive
 *      regime (Section 4.1): commit every masked position with c > tau
 *      (strict); if there is none, commit only the leftmost masked position
 *      (Algorithm 2) and report a fallback step (membership of the step in
 *      the set F_i of Section 3.2).
 *
 * `tau` is the paper's confidence threshold lambda.  Candidates are greedy
 * (sampling temperature 0).  The [B*L, V] logits are never written to memory.
 *
 * Conventions shared by every entry point
 *   - All array arguments are DEVICE pointers (HIP device memory of the
 *     current device) owned by the caller; the library never frees them.
 *   - Row-major layouts; position r of sequence b is row b*L + r.
 *   - The call is asynchronous: work is enqueued on `stream` (a hipStream_t,
 *     NULL = the legacy default stream) and the function returns without
 *     synchronising (unless the environment sets FORK_SYNC=1, a debugging aid
 *     that synchronises and reports launch-time errors).
 *   - Argument errors are detected on the host before anything is enqueued
 *     and return a negative status; fork_last_error() then describes them.
 *   - Output arrays must not alias inputs.  tokens, mask and block_start are
 *     updated in place.
 *   - Calls may come from several host threads and on several streams.
 *     Calls that pass no workspace of their own use the library-managed
 *     workspace of the (device, stream) pair they are enqueued on: calls on
 *     one stream share a buffer (their work runs in stream order), calls on
 *     different streams get different buffers and may overlap.  A buffer
 *     that must grow is replaced by a larger one without synchronising; the
 *     outgrown allocation is kept until fork_release, since work already
 *     queued may still read it.  Each stream that has used the managed
 *     workspace keeps its buffer until fork_release.
 *   - Graph capture: a call that would use the managed workspace returns
 *     FORK_EINVAL while its stream is being captured (the graph would keep
 *     the buffer's address beyond fork_release).  Captured calls pass a
 *     caller workspace, which must outlive the graph.
 */
#ifndef FORK_STEP_H
#define FORK_STEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
enum {
  FORK_OK = 0,
  FORK_EINVAL = -1,       /* bad argument (null pointer, size, alignment, tau)  */
  FORK_EUNSUPPORTED = -2, /* valid but unsupported (d not a multiple of 8 / 4) */
  FORK_EHIP = -3,         /* a HIP runtime call or launch failed               */
  FORK_ENOMEM = -4        /* the library-managed workspace could not grow      */
};

/* Element types of hidden and W_head (both the same). */
enum { FORK_BF16 = 0, FORK_F32 = 1 };

/* Fallback rules when no masked position of the active block passes tau.
   Ties go to the lowest position. */
enum {
  FORK_RULE_LEFTMOST = 0, /* Fork-dLLM, Algorithm 2: the leftmost masked position */
  FORK_RULE_MAXCONF = 1,  /* Fast-dLLM, Algorithm 1: the highest confidence       */
  FORK_RULE_MINCONF = 2,  /* ablations of Section 4.1: the lowest confidence,     */
  FORK_RULE_MAXENT = 3,   /*   the highest entropy,                               */
  FORK_RULE_RANDOM = 4    /*   or a uniformly random masked position: with n
                               masked positions and u = fallback_uniform[b], the
                               j-th in increasing order, j = (int)(u * n) in
                               binary32, capped at n - 1                          */
};

/* Which positions get statistics (fork_step_args.rows_mode). */
enum {
  FORK_ROWS_ALL = 0,    /* every one of the B*L positions                      */
  FORK_ROWS_ACTIVE = 1  /* only the positions of each sequence's active block:
                           the selection reads nothing else, so the decisions
                           are those of FORK_ROWS_ALL; out_conf, out_entropy,
                           out_logp, out_lse and out_argmax are written at
                           those positions only and left untouched elsewhere.
                           Needs B*L*d*element_size < 2^31.                    */
};

/* Values written to out_fallback[b]. */
enum {
  FORK_STEP_PARALLEL = 0, /* at least one position passed tau, all committed   */
  FORK_STEP_FALLBACK = 1, /* none passed; exactly one position committed       */
  FORK_STEP_IDLE = -1,    /* no masked position at or after block_start[b]     */
  FORK_STEP_BADSTATE = -2 /* block_start[b] outside [0, L]; nothing written    */
};

/*
 * fork_step -- one denoising step (Algorithm 2 with greedy candidates).
 *
 * hidden       [B*L, d]  FORK_BF16 or FORK_F32, row-major, 16-byte aligned.
 *                        Final hidden state of every position.
 * W_head       [V, d]    same element type, row-major (one row per
 *                        vocabulary entry), 16-byte aligned.
 * tokens       [B*L] int32, in/out.  Written only at committed positions,
 *                        with the candidate token.
 * mask         [B*L] uint8, in/out.  Nonzero = [MASK].  Cleared at committed
 *                        positions.  Only positions at or after block_start[b]
 *                        are considered.
 * block_start  [B] int32, in/out.  Start of the block to resume from; the
 *                        active block is the first block [s, min(s+block_len,
 *                        L)), s = block_start[b] + j*block_len, that holds a
 *                        masked position; its start is written back.
 * block_len    1 <= block_len <= L.
 * tau          the confidence threshold (lambda); finite.  Commit iff
 *                        conf > tau, compared in binary32.
 * out_conf     [B*L] float: q(candidate) for every position.
 * out_entropy  [B*L] float: entropy of q in nats for every position.
 * out_logp     [B*L] float: log q(candidate) for every position.
 * out_fallback [B] int32: FORK_STEP_* per sequence.
 * B, L, d, V   sizes: L, d, V >= 1, B >= 0, B*L < 2^31; d % 8 == 0 for
 *              FORK_BF16, d % 4 == 0 for FORK_F32, d <= 2^20 (else
 *              FORK_EUNSUPPORTED).  B == 0 (an empty batch) enqueues
 *              nothing and returns FORK_OK; the array pointers may then be
 *              NULL.
 * dtype        FORK_BF16 or FORK_F32.
 * stream       hipStream_t to enqueue on (NULL = default stream).
 *
 * Returns FORK_OK or a negative FORK_E* code (FORK_EUNSUPPORTED also when
 * the launch grid would exceed 2^32 work-items, i.e. when
 * ceil(positions/256) * ceil(V/256) * 512 >= 2^32; split such batches).
 * Uses the library-managed workspace of (device of `stream`, `stream`),
 * grown on demand with hipMalloc; fork_release frees it.  Returns FORK_EINVAL
 * while `stream` is being captured into a graph.
 */
int fork_step(const void* hidden, const void* W_head, int32_t* tokens,
              uint8_t* mask, int32_t* block_start, int32_t block_len,
              float tau, float* out_conf, float* out_entropy, float* out_logp,
              int32_t* out_fallback, int32_t B, int32_t L, int32_t d,
              int32_t V, int32_t dtype, void* stream);

/* Arguments of fork_step_ex: those of fork_step plus optional extras. */
typedef struct fork_step_args {
  const void* hidden;
  const void* W_head;
  int32_t* tokens;
  uint8_t* mask;
  int32_t* block_start;
  int32_t block_len;
  float tau;
  float* out_conf;
  float* out_entropy;
  float* out_logp;
  int32_t* out_fallback;
  int32_t B, L, d, V, dtype;
  void* stream;
  /* Optional outputs (NULL = not produced). */
  float* out_lse;          /* [B*L] log sum_v exp z_v (log-normaliser)        */
  int32_t* out_argmax;     /* [B*L] greedy candidate of every position        */
  int32_t* out_ncommit;    /* [B] number of positions committed this step     */
  int32_t* out_commit_pos; /* [B*block_len] committed positions of sequence b,
                              ascending, in row b, padded with -1             */
  int32_t rule;            /* FORK_RULE_*; fork_step uses FORK_RULE_LEFTMOST  */
  /* Caller-provided device workspace (NULL = library-managed).  Must hold
     fork_workspace_bytes(B, L, V) bytes and be 256-byte aligned. */
  void* workspace;
  size_t workspace_bytes;
  /* Optional profiling hooks (NULL = none): hipEvent_t handles recorded on
     `stream` immediately before and after the LM-head kernel, so a caller
     can time that kernel alone with hipEventElapsedTime. */
  void* ev_lmhead_begin;
  void* ev_lmhead_end;
  /* [B] float in [0, 1): the random draw of each sequence for
     FORK_RULE_RANDOM (required by that rule, ignored by the others). */
  const float* fallback_uniform;
  int32_t rows_mode;       /* FORK_ROWS_*; fork_step uses FORK_ROWS_ALL        */
  /* Drawn candidates (Section 2: the candidate of position k is drawn from
     q^k(. | x_t; tau), the softmax of the logits divided by the sampling
     temperature).  0 (fork_step's value) keeps the greedy candidate.  With
     sample_temperature > 0 the candidates of the active blocks' positions
     are drawn by the Gumbel-max property: cand = argmax_v z_v / tau - log E_v
     with E_v = -log(1 - U_v), U_v = (2 (w >> 9) + 1) 2^-24 and w word v % 4
     of Philox4x32-10 (Salmon et al., SC'11) at counter
     (v / 4, b * L + k, sample_counter, 0) under key (sample_seed mod 2^32,
     sample_seed / 2^32); ties go to the lower v.  out_conf and out_logp of
     such a position are q(cand) and log q(cand) of the untempered q (the
     confidence of Algorithm 2); out_entropy and out_lse are unchanged.
     Other positions keep the greedy candidate and its statistics.  Draws do
     not depend on rows_mode.  Must be 0 or in [1e-30, inf) (FORK_EINVAL). */
  float sample_temperature;
  uint32_t sample_counter; /* per-step counter of the draws (e.g. step index) */
  uint64_t sample_seed;    /* key of the draws                                 */
} fork_step_args;

/* fork_step with the extras above.  Same return codes. */
int fork_step_ex(const fork_step_args* args);

/* Maximum scratch of fork_step_noalloc: 64 MiB, enough for every mode at
   B*L = 4096 positions and V = 126464 (the LLaDA-8B shape). */
#define FORK_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* fork_step_ex for callers that cannot allocate device memory: code under
   HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
   Same arguments, semantics, outputs and kernels as fork_step_ex, but the
   step's scratch (per-tile partial statistics, candidates, row lists) lives
   in a static device array of FORK_NOALLOC_SCRATCH_BYTES that the library
   holds on each GPU it runs on until the process ends; nothing is allocated
   (no hipMalloc, hipFree or allocating library call).  The first call on a
   device looks up that device's copy of the array (hipGetSymbolAddress):
   make it outside graph capture.  Nothing in the scratch needs to start at
   zero; every call overwrites what it reads.
   args->workspace must be NULL and args->workspace_bytes 0 (FORK_EINVAL).
   Sizes whose scratch (fork_workspace_bytes without the drawn partials when
   sample_temperature == 0) exceeds FORK_NOALLOC_SCRATCH_BYTES return
   FORK_EUNSUPPORTED before anything is enqueued.
   All calls on one GPU share its array: calls whose GPU work overlaps (on
   different streams, or from threads not ordered with each other) race on
   it and give undefined results; serialise them, e.g. on one stream. */
int fork_step_noalloc(const fork_step_args* args);

/* Device workspace bytes a step with these sizes needs in any mode (per-tile
   partial statistics, the per-position candidates, the active-row list, and
   the per-tile drawn candidates when sample_temperature > 0); 0 if the sizes
   are invalid. */
size_t fork_workspace_bytes(int32_t B, int32_t L, int32_t V);

/* Layouts of the per-position arrays of fork_select (conf, entropy, argmax,
   tokens, mask). */
enum {
  FORK_LAYOUT_ROW_MAJOR = 0,      /* position k of sequence b at b*L + k (as
                                     everywhere else in this interface)       */
  FORK_LAYOUT_POSITION_MAJOR = 1  /* position k of sequence b at k*B + b: the
                                     sequences' entries for one position are
                                     adjacent, so a batch whose sequences sit
                                     at the same positions reads and commits
                                     whole cache lines (large batches)        */
};

/* The unmasking rule alone (Algorithm 2; the `rule` variants of
   fork_step_args), applied in place to B sequences from per-position
   confidences and candidates computed elsewhere: exactly the selection stage
   of fork_step_ex, with the same arguments, semantics and outputs
   (out_fallback per sequence; out_ncommit and out_commit_pos optional).
   entropy ([B*L]) is needed by FORK_RULE_MAXENT, uniform ([B]) by
   FORK_RULE_RANDOM.  `layout` (FORK_LAYOUT_*) orders conf, entropy, argmax,
   tokens and mask; block_start, out_fallback, out_ncommit and
   out_commit_pos ([B, block_len], row b for sequence b) do not depend on it,
   and neither do the decisions.  B == 0 enqueues nothing (array pointers may
   be NULL).  Returns FORK_OK, FORK_EINVAL or FORK_EHIP. */
typedef struct fork_select_args {
  const float* conf;       /* [B*L] confidence of each position's candidate    */
  const float* entropy;    /* [B*L] or NULL                                    */
  const float* uniform;    /* [B] or NULL                                      */
  const int32_t* argmax;   /* [B*L] candidate token of each position           */
  int32_t* tokens;         /* [B*L] in/out                                     */
  uint8_t* mask;           /* [B*L] in/out                                     */
  int32_t* block_start;    /* [B]   in/out                                     */
  int32_t* out_fallback;   /* [B]                                              */
  int32_t* out_ncommit;    /* [B] or NULL                                      */
  int32_t* out_commit_pos; /* [B*block_len] or NULL                            */
  int32_t B, L, block_len;
  float tau;
  int32_t rule;
  void* stream;
  int32_t layout;          /* FORK_LAYOUT_*                                    */
} fork_select_args;
int fork_select(const fork_select_args* args);

/* ------------------------------------------------------------ ForkGRPO
 *
 * Section 3.2 of the paper trains on the fallback steps of Fork-dLLM
 * rollouts: at each fallback step t of rollout i one token is committed at
 * k_{i,t} (the leftmost masked position), so the policy-likelihood ratio
 * rho_{i,t} = q_new(x^{k}|c, x_{i,t}) / q_old(x^{k}|c, x_{i,t}) is exact.
 * fork_step records log q_old (out_logp at the committed position).  The
 * calls below evaluate log q_new of the recorded tokens under another head
 * (teacher forcing), the clipped surrogate objective, and JustGRPO-Fast's
 * highest-entropy positions.
 */

/* Teacher-forced log-probabilities: for entry e, with z the logits of
   hidden row rows[e] against W_head,
     out_logp[e] = z_{tokens[e]} - log sum_v exp(z_v)     (log q of the token)
   and optionally out_q[e] = exp(out_logp[e]), out_entropy[e] (nats) and
   out_lse[e] = log sum_v exp(z_v).  A token outside [0, V) gives NaN; a row
   outside [0, M) gives unspecified values (it is never read out of bounds).
   Pointers are device pointers; the call is asynchronous on `stream`. */
typedef struct fork_logprob_args {
  const void* hidden;      /* [M, d], dtype                                    */
  const void* W_head;      /* [V, d], dtype                                    */
  const int32_t* rows;     /* [n] hidden row of each entry; NULL: row e        */
  const int32_t* tokens;   /* [n] token of each entry                          */
  float* out_logp;         /* [n]                                              */
  float* out_q;            /* [n] or NULL                                      */
  float* out_entropy;      /* [n] or NULL                                      */
  float* out_lse;          /* [n] or NULL                                      */
  int32_t n, M, d, V, dtype;
  void* stream;
  void* workspace;         /* NULL: library-managed, as for fork_step_ex       */
  size_t workspace_bytes;
  void* ev_lmhead_begin;   /* optional hipEvent_t pair around the LM head      */
  void* ev_lmhead_end;
} fork_logprob_args;

/* FORK_OK, or FORK_EINVAL / FORK_EUNSUPPORTED (same size and alignment rules
   as fork_step; with rows given, M*d*element_size < 2^31) / FORK_EHIP /
   FORK_ENOMEM.  n == 0 enqueues nothing. */
int fork_logprob(const fork_logprob_args* args);

/* Workspace bytes of fork_logprob for n entries over V words. */
size_t fork_logprob_workspace_bytes(int32_t n, int32_t V);

/* The ForkGRPO objective (Section 3.2) of one batch: n_groups prompts with
   G rollouts each, rollout i = g*G + j.  The fallback-step entries of
   rollout i are [offsets[i], offsets[i+1]) of lp_new / lp_old (n entries).
     A_i       = (r_i - mean_g) / std_g, std with divisor G; a group with
                 std_g == 0 is skipped (A = 0, group_obj = 0, skipped = 1)
     ratio[e]  = exp(lp_new[e] - lp_old[e])
     term[e]   = min(ratio A_i, clip(ratio, 1 - eps, 1 + eps) A_i)
     rollout_obj[i] = mean of term over the rollout's entries (0 if none)
     group_obj[g]   = mean of rollout_obj over the group
     J         = mean of group_obj over the groups not skipped (0 if none)
   fp32 arithmetic, fixed-order sums (bit-reproducible).  Offsets are
   clamped to [0, n].  Returns FORK_OK, FORK_EINVAL (sizes, G >
   1024, eps < 0 or not finite, a required pointer NULL) or FORK_EHIP. */
typedef struct fork_grpo_args {
  int32_t n_groups, G, n;
  const float* rewards;    /* [n_groups*G]                                     */
  const int32_t* offsets;  /* [n_groups*G + 1]                                 */
  const float* lp_new;     /* [n] log q under the policy being trained         */
  const float* lp_old;     /* [n] log q recorded at rollout time               */
  float eps;               /* clip range                                       */
  float* out_adv;          /* [n_groups*G] or NULL                             */
  float* out_ratio;        /* [n] or NULL                                      */
  float* out_term;         /* [n] or NULL                                      */
  float* out_rollout_obj;  /* [n_groups*G] or NULL                             */
  float* out_group_obj;    /* [n_groups], required                             */
  uint8_t* out_skipped;    /* [n_groups], required                             */
  float* out_J;            /* [1], required                                    */
  void* stream;
} fork_grpo_args;
int fork_grpo_objective(const fork_grpo_args* args);

/* JustGRPO-Fast's position selection (compared with ForkGRPO in Section
   3.2): in each of R rollouts of Lg positions (entropy[i*Lg + p], e.g. the
   out_entropy recorded when position p was committed), sel[i*Lg + p] = 1
   for the k positions of highest entropy, equal values taken in increasing
   position, 0 elsewhere.  Lg <= 16384, 0 <= k <= Lg.  Returns FORK_OK,
   FORK_EINVAL, FORK_EUNSUPPORTED (Lg too large) or FORK_EHIP. */
int fork_top_entropy(const float* entropy, int32_t R, int32_t Lg, int32_t k, uint8_t* sel,
                     void* stream);

/* Description of the last non-OK return on the calling thread ("" if none).
   The string stays valid until the thread's next call into the library. */
const char* fork_last_error(void);

/* Free the library-managed workspaces of every device and stream, outgrown
   allocations included.  Synchronises each device that holds one first, so
   work already queued finishes; must not race with calls still being
   issued by other threads. */
void fork_release(void);

/* Library version as major*10000 + minor*100 + patch. */
int fork_version(void);

#ifdef __cplusplus
}
#endif
#endif /* FORK_STEP_H */
