// Internal interface between the C-ABI host code and the HIP kernels of the
// Fork-dLLM step.  Not installed; the public interface is include/fork_step.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fork {

// Vocabulary rows and positions covered by one GEMM workgroup.
constexpr int kTileV = 256;
constexpr int kTileP = 256;

// Partial statistics of one position over one vocabulary tile, stored as a
// float4 {m, s, t, idx}: m = max logit, s = sum exp(z - m),
// t = sum exp(z - m) * (z - m), idx = lowest vocabulary index with z == m
// (bit pattern of an int32).  An empty partial has s == 0.
struct Partial {
  float m, s, t;
  int idx;
};

// Drawn candidates at a sampling temperature tau > 0 (Gumbel-max over
// Philox4x32-10 draws).  row[p] is the row index that keys the draws of
// LM-head position p, or -1 for a position that keeps the greedy candidate;
// a null `row` disables drawing.  partials[vt * M + p] receives, for each
// drawn position, {best key, its vocabulary index (int32 bits), its logit, 0}.
struct SampleArgs {
  const int32_t* row;
  float4* partials;
  float inv_tau;
  uint32_t key0, key1, counter;
};

// Teacher-forced mode: token[p] is a vocabulary index per LM-head position;
// the epilogue stores that entry's logit to z[p] (tokens outside [0, V)
// store nothing).
struct TargetArgs {
  const int32_t* token;
  float* z;
};

inline int num_vocab_tiles(int V) { return (V + kTileV - 1) / kTileV; }
inline int num_pos_tiles(int M) { return (M + kTileP - 1) / kTileP; }

// Logits of M positions against W (never stored) reduced to one Partial per
// (vocabulary tile, position): partials[vt * M + p].  Position p is hidden row
// p, or with a row list hidden row rowlist[p] (-1 = none) out of Mh rows.
// At most one of sample.row and target.token may be set.
hipError_t launch_gemm_stats(const void* hidden, const void* W, bool bf16,
                             int M, int d, int V, float4* partials,
                             const int32_t* rowlist, int Mh, const SampleArgs& sample,
                             const TargetArgs& target, hipStream_t stream);

// Merge the partials of each position over all vocabulary tiles into the
// per-position results (position p lands in row p, or rowlist[p] if a row
// list is given; -1 = dropped).  lse may be null.  Positions with
// sample_row[p] >= 0 (sample_row may be null) take the drawn candidate from
// spartials, with the untempered confidence and log-probability of it.
//
// Teacher-forced mode (token non-null): logp and conf are log q and q of
// token[p] from its logit ztoken[p] (NaN for a token outside [0, V)).  Any of
// conf, entropy, lse, argmax may be null.
hipError_t launch_merge(const float4* partials, int M, int nvt, float* conf,
                        float* entropy, float* logp, float* lse,
                        int32_t* argmax, const int32_t* rowlist,
                        const int32_t* sample_row, const float4* spartials,
                        const int32_t* token, const float* ztoken, int V,
                        hipStream_t stream);

// Rows of each sequence's active block (the same skip-forward as the
// selection): rowlist[b * block_len + i] = b * L + s_b + i, -1 past the block
// end or for sequences with nothing to commit.  rowmap (B * L entries) holds
// r for the rows of the active blocks and -1 elsewhere.  Either may be null.
hipError_t launch_active_rows(int B, int L, int block_len, const uint8_t* mask,
                              const int32_t* block_start, int32_t* rowlist,
                              int32_t* rowmap, hipStream_t stream);

// Unmasking rule per sequence, in place.  ncommit / commit_pos may be null;
// entropy is read by the highest-entropy rule, uniform by the random rule.
// Row-major state (element k of sequence b at b * L + k): batches of at
// least kLaneSelectMinB sequences with blocks of at most kLaneSelectMaxBL
// positions run one lane per sequence, others one wave per sequence.
// Position-major state (at k * B + b): one lane per four sequences from
// kPmWideMinB sequences on (B a multiple of 4, the arrays 16-byte aligned),
// one lane per sequence otherwise.  All give the same results.
constexpr int kLaneSelectMinB = 4096;
constexpr int kLaneSelectMaxBL = 64;
constexpr int kPmWideMinB = 1 << 18;
hipError_t launch_select(int B, int L, int block_len, float tau, int rule,
                         const float* conf, const float* entropy, const float* uniform,
                         const int32_t* argmax,
                         int32_t* tokens, uint8_t* mask, int32_t* block_start,
                         int32_t* fallback, int32_t* ncommit,
                         int32_t* commit_pos, bool position_major, hipStream_t stream);

// ForkGRPO objective over n_groups groups of G rollouts (G <=
// kMaxGroupSize); entries of rollout i are [offsets[i], offsets[i+1])
// clamped to [0, n).  adv, ratio, term, rollout_obj may be null; group_obj,
// skipped ([n_groups]) and J ([1]) are written.
constexpr int kMaxGroupSize = 1024;
hipError_t launch_grpo_objective(int n_groups, int G, int n, const float* rewards,
                                 const int32_t* offsets, const float* lp_new,
                                 const float* lp_old, float eps, float* adv, float* ratio,
                                 float* term, float* rollout_obj, float* group_obj,
                                 uint8_t* skipped, float* J, hipStream_t stream);

// Per rollout (R of them, Lg <= kMaxTopEntropyLen positions each) the k
// positions of highest entropy, ties in increasing position: sel = 1 there.
constexpr int kMaxTopEntropyLen = 16384;
hipError_t launch_top_entropy(int R, int Lg, int k, const float* entropy, uint8_t* sel,
                              hipStream_t stream);

}  // namespace fork
