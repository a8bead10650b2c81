// Cross-tile merge of the per-tile statistics, and the unmasking rule.
//
// Merge (per position, over vocabulary tiles j):
//   m = max_j m_j,  s = sum_j s_j e^(m_j - m),
//   t = sum_j e^(m_j - m) (t_j + (m_j - m) s_j)
// which is the exact re-basing of each tile's sums from its own maximum m_j to
// the global one.  With q_v = e^(z_v - m) / s this gives
//   confidence q(argmax) = 1/s,  log q(argmax) = -log s,
//   log-normaliser = m + log s,  entropy = -sum q log q = log s - t/s,
// the quantities of Section 2 (confidence), Section 3.1 (entropy) and
// Section 3.2 (log-probability inside the ForkGRPO ratio) of the Fork-dLLM
// paper.  For a drawn candidate x (sampling temperature > 0) the confidence
// and log-probability are those of x under the untempered q: e^(z_x - m)/s
// and (z_x - m) - log s.  The merge order is fixed, so results are
// bit-reproducible.
//
// Selection (Algorithm 2 of the paper, in the active block of the
// semi-autoregressive regime of Section 4.1): one wave64 per sequence; the
// threshold test is a ballot over the block's lanes, the fallback is the
// first set bit of the mask ballot (leftmost masked position), and committed
// positions are compacted with a lane-prefix count.  The other fallback rules
// (Algorithm 1's highest confidence; Section 4.1's ablations: lowest
// confidence, highest entropy, random position) are wave reductions.
#include "fork_kernels.h"

#include <math.h>

#include <type_traits>

namespace fork {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMergePositions = 16;  // positions per merge workgroup
constexpr int kMergeWaves = 16;      // waves per workgroup, 4 tile streams each
constexpr int kMergeThreads = 64 * kMergeWaves;

__device__ __forceinline__ float4 merge2(float4 a, float4 b) {
  if (b.y == 0.f) return a;
  if (a.y == 0.f) return b;
  const float m = fmaxf(a.x, b.x);
  const float ea = __builtin_amdgcn_exp2f((a.x - m) * kLog2e);
  const float eb = __builtin_amdgcn_exp2f((b.x - m) * kLog2e);
  float4 r;
  r.x = m;
  r.y = a.y * ea + b.y * eb;
  r.z = ea * (a.z + (a.x - m) * a.y) + eb * (b.z + (b.x - m) * b.y);
  const int ia = __float_as_int(a.w), ib = __float_as_int(b.w);
  const bool take_a = (a.x > b.x) || (a.x == b.x && ia < ib);
  r.w = __int_as_float(take_a ? ia : ib);
  return r;
}

// Drawn-candidate partials {key, idx bits, z, 0}: larger key wins, lower
// index on equal keys.
__device__ __forceinline__ float4 pick_drawn(float4 a, float4 b) {
  const bool take_a = a.x > b.x || (a.x == b.x && __float_as_int(a.y) < __float_as_int(b.y));
  return make_float4(take_a ? a.x : b.x, take_a ? a.y : b.y, take_a ? a.z : b.z, 0.f);
}

__device__ __forceinline__ float4 shfl_xor4(float4 v, int off) {
  return make_float4(__shfl_xor(v.x, off), __shfl_xor(v.y, off), __shfl_xor(v.z, off),
                     __shfl_xor(v.w, off));
}

// 16 positions per workgroup of 16 waves.  Lane l of wave w serves position
// l % 16 and tile stream c = 4 w + l / 16 (64 streams): it merges tiles
// c, c + 64, ... in increasing order, loads issued four at a time, so one
// load instruction reads four runs of 16 consecutive positions (256 B each).
// The 64 stream results of a position are then combined in a fixed tree —
// lanes l, l ^ 16, l ^ 32 by shuffles, then the 16 waves through LDS (four
// at a time, then pairwise) — each pair merged as (lower, higher).  The result depends only on
// the tile order, not on M, the grid or the row list.
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(
    const float4* __restrict__ partials, int M, int nvt, float* __restrict__ conf,
    float* __restrict__ entropy, float* __restrict__ logp, float* __restrict__ lse,
    int32_t* __restrict__ argmax, const int32_t* __restrict__ rowlist,
    const int32_t* __restrict__ sample_row, const float4* __restrict__ spartials,
    const int32_t* __restrict__ token, const float* __restrict__ ztoken, int V) {
  __shared__ float4 red[kMergeWaves][kMergePositions];
  __shared__ float4 sred[kMergeWaves][kMergePositions];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int pl = lane & 15;                  // position within the workgroup
  const int c = 4 * w + (lane >> 4);         // tile stream 0..63
  const int r = blockIdx.x * kMergePositions + pl;
  const bool live = r < M;
  float4 acc = make_float4(-INFINITY, 0.f, 0.f, __int_as_float(0x7fffffff));
  if (live) {
    const float4* col = partials + r;
    int j = c;
    for (; j + 192 < nvt; j += 256) {
      const float4 p0 = col[(size_t)j * M], p1 = col[(size_t)(j + 64) * M];
      const float4 p2 = col[(size_t)(j + 128) * M], p3 = col[(size_t)(j + 192) * M];
      acc = merge2(merge2(merge2(merge2(acc, p0), p1), p2), p3);
    }
    // the last (at most three) tiles of the stream: loads issued together,
    // merged in the same increasing order
    float4 q[3];
#pragma unroll
    for (int t = 0; t < 3; ++t)
      if (j + 64 * t < nvt) q[t] = col[(size_t)(j + 64 * t) * M];
#pragma unroll
    for (int t = 0; t < 3; ++t)
      if (j + 64 * t < nvt) acc = merge2(acc, q[t]);
  }
  // streams 4w + {0..3} of this position: lanes pl, pl + 16, pl + 32, pl + 48
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    const float4 o = shfl_xor4(acc, off);
    acc = (lane & off) ? merge2(o, acc) : merge2(acc, o);
  }
  if (lane < 16) red[w][pl] = acc;
  const bool drawn = sample_row && live && sample_row[r] >= 0;
  float4 sacc = make_float4(-INFINITY, __int_as_float(0x7fffffff), 0.f, 0.f);
  if (drawn) {
    // the winner does not depend on the order: loads eight at a time
    const float4* scol = spartials + r;
    for (int k0 = c; k0 < nvt; k0 += 512) {
      float4 q[8];
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (k0 + 64 * t < nvt) q[t] = scol[(size_t)(k0 + 64 * t) * M];
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (k0 + 64 * t < nvt) sacc = pick_drawn(sacc, q[t]);
    }
  }
  if (sample_row) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float4 o = shfl_xor4(sacc, off);
      sacc = (lane & off) ? pick_drawn(o, sacc) : pick_drawn(sacc, o);
    }
    if (lane < 16) sred[w][pl] = sacc;
  }
  __syncthreads();
  if (w != 0) return;
  // wave 0 combines the 16 wave results: lane group q = lane / 16 merges
  // waves 4q .. 4q + 3, then the four groups pairwise
  const int q = lane >> 4;
  acc = red[4 * q][pl];
#pragma unroll
  for (int k = 1; k < 4; ++k) acc = merge2(acc, red[4 * q + k][pl]);
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    const float4 o = shfl_xor4(acc, off);
    acc = (lane & off) ? merge2(o, acc) : merge2(acc, o);
  }
  if (sample_row) {
    sacc = sred[4 * q][pl];
#pragma unroll
    for (int k = 1; k < 4; ++k) sacc = pick_drawn(sacc, sred[4 * q + k][pl]);
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float4 o = shfl_xor4(sacc, off);
      sacc = (lane & off) ? pick_drawn(o, sacc) : pick_drawn(sacc, o);
    }
  }
  if (lane >= 16 || !live) return;
  const int dst = rowlist ? rowlist[r] : r;
  if (dst < 0) return;
  const float log_s = logf(acc.y);
  if (entropy) entropy[dst] = log_s - acc.z / acc.y;
  if (lse) lse[dst] = acc.x + log_s;
  if (argmax) argmax[dst] = __float_as_int(acc.w);
  if (token) {
    // teacher-forced: log q of the given token from its logit
    const int tk = token[r];
    const float lq = (tk >= 0 && tk < V) ? (ztoken[r] - acc.x) - log_s : __int_as_float(0x7fc00000);
    logp[dst] = lq;
    if (conf) conf[dst] = exp2f(lq * kLog2e);
  } else if (drawn) {
    // untempered q of the drawn token: exp(z - m) / s
    const float dz = sacc.z - acc.x;
    conf[dst] = exp2f(dz * kLog2e) / acc.y;
    logp[dst] = dz - log_s;
    argmax[dst] = __float_as_int(sacc.y);
  } else {
    if (conf) conf[dst] = 1.0f / acc.y;
    logp[dst] = -log_s;
  }
}

__device__ __forceinline__ unsigned long long ballot(bool p) { return __ballot(p); }

// rule values as in the C ABI
enum { kLeftmost = 0, kMaxConf = 1, kMinConf = 2, kMaxEnt = 3, kRandom = 4 };

__global__ __launch_bounds__(64) void select_kernel(
    int L, int BL, float tau, int rule, const float* __restrict__ conf,
    const float* __restrict__ entropy, const float* __restrict__ uniform,
    const int32_t* __restrict__ argmax, int32_t* __restrict__ tokens,
    uint8_t* __restrict__ mask, int32_t* __restrict__ block_start,
    int32_t* __restrict__ fallback, int32_t* __restrict__ ncommit,
    int32_t* __restrict__ commit_pos) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const size_t base = (size_t)b * L;
  int32_t* my_commits = commit_pos ? commit_pos + (size_t)b * BL : nullptr;

  if (BL <= 64) {
    // lane i <-> position s + i of a block: the block's mask byte,
    // confidence, candidate (and entropy) arrive together, and the rule is
    // decided from registers
    int s = block_start[b];
    int status = (s < 0 || s > L) ? -2 : -1;
    bool masked = false;
    float cf = 0.f;
    int cand = 0;
    unsigned long long mball = 0;
    while (status == -1 && s < L) {
      const int k = s + lane;
      const bool in = k < min(s + BL, L);
      const uint8_t m = in ? mask[base + k] : 0;
      cf = in ? conf[base + k] : 0.f;
      cand = in ? argmax[base + k] : 0;
      masked = m != 0;
      mball = ballot(masked);
      if (mball) status = 0;
      else s += BL;
    }
    if (status != 0) {
      if (lane == 0) {
        fallback[b] = status;
        if (ncommit) ncommit[b] = 0;
      }
      if (my_commits && lane < BL) my_commits[lane] = -1;
      return;
    }
    const int k = s + lane;
    const bool pass = masked && cf > tau;
    const unsigned long long pball = ballot(pass);
    const bool fb = pball == 0;
    int pick = -1;
    if (fb) {
      if (rule == kLeftmost) {
        pick = s + __ffsll((long long)mball) - 1;
      } else if (rule == kRandom) {
        const int n = __popcll(mball);
        int j = (int)(uniform[b] * (float)n);
        j = j > n - 1 ? n - 1 : (j < 0 ? 0 : j);
        const int below = __popcll(mball & ((1ull << lane) - 1ull));
        pick = s + __ffsll((long long)ballot(masked && below == j)) - 1;
      } else {
        // extreme of confidence (highest or lowest) or of entropy (highest),
        // lowest position on ties
        const bool lowest = rule == kMinConf;
        float best = masked ? (rule == kMaxEnt ? entropy[base + k] : cf) : 0.f;
        int bi = masked ? k : 0x7fffffff;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const float ob = __shfl_xor(best, off);
          const int oi = __shfl_xor(bi, off);
          const bool better = lowest ? ob < best : ob > best;
          const bool take =
              oi != 0x7fffffff && (bi == 0x7fffffff || better || (ob == best && oi < bi));
          best = take ? ob : best;
          bi = take ? oi : bi;
        }
        pick = bi;
      }
    }
    const bool commit = masked && (fb ? k == pick : pass);
    const unsigned long long cball = ballot(commit);
    if (commit) {
      tokens[base + k] = cand;
      mask[base + k] = 0;
      if (my_commits) my_commits[__popcll(cball & ((1ull << lane) - 1ull))] = k;
    }
    const int written = __popcll(cball);
    if (my_commits && lane >= written && lane < BL) my_commits[lane] = -1;
    if (lane == 0) {
      fallback[b] = fb ? 1 : 0;
      block_start[b] = s;
      if (ncommit) ncommit[b] = written;
    }
    return;
  }

  int s = block_start[b];
  int status = 0;
  if (s < 0 || s > L) {
    status = -2;
  } else {
    // skip forward to the first block holding a masked position
    bool found = false;
    while (s < L) {
      const int e = min(s + BL, L);
      for (int c = s; c < e; c += 64) {
        const int k = c + lane;
        if (ballot(k < e && mask[base + k] != 0)) {
          found = true;
          break;
        }
      }
      if (found) break;
      s += BL;
    }
    if (!found) status = -1;
  }
  if (status != 0) {
    if (lane == 0) {
      fallback[b] = status;
      if (ncommit) ncommit[b] = 0;
    }
    if (my_commits)
      for (int i = lane; i < BL; i += 64) my_commits[i] = -1;
    return;
  }

  const int e = min(s + BL, L);
  // threshold set U = { k masked : conf[k] > tau }
  int npass = 0;
  for (int c = s; c < e; c += 64) {
    const int k = c + lane;
    const bool pass = k < e && mask[base + k] != 0 && conf[base + k] > tau;
    npass += __popcll(ballot(pass));
  }
  const bool fb = npass == 0;
  int pick = -1;
  if (fb) {
    if (rule == kLeftmost) {
      // leftmost masked position of the block
      for (int c = s; c < e; c += 64) {
        const int k = c + lane;
        const unsigned long long bm = ballot(k < e && mask[base + k] != 0);
        if (bm) {
          pick = c + __ffsll((long long)bm) - 1;
          break;
        }
      }
    } else if (rule == kRandom) {
      // the j-th masked position, j = (int)(u * n) in binary32, capped
      int n = 0;
      for (int c = s; c < e; c += 64) n += __popcll(ballot(c + lane < e && mask[base + c + lane] != 0));
      int j = (int)(uniform[b] * (float)n);
      j = j > n - 1 ? n - 1 : (j < 0 ? 0 : j);
      for (int c = s; c < e; c += 64) {
        const int k = c + lane;
        const bool masked = k < e && mask[base + k] != 0;
        const unsigned long long bm = ballot(masked);
        const int cnt = __popcll(bm);
        if (j < cnt) {
          const int below = __popcll(bm & ((1ull << lane) - 1ull));
          const unsigned long long hit = ballot(masked && below == j);
          pick = c + __ffsll((long long)hit) - 1;
          break;
        }
        j -= cnt;
      }
    } else {
      // extreme of confidence (highest or lowest) or of entropy (highest),
      // lowest position on ties
      const float* key = rule == kMaxEnt ? entropy : conf;
      const bool lowest = rule == kMinConf;
      float best = 0.f;
      int bi = 0x7fffffff;
      for (int c = s; c < e; c += 64) {
        const int k = c + lane;
        if (k < e && mask[base + k] != 0) {
          const float v = key[base + k];
          if (bi == 0x7fffffff || (lowest ? v < best : v > best)) {
            best = v;
            bi = k;
          }
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float ob = __shfl_xor(best, off);
        const int oi = __shfl_xor(bi, off);
        const bool better = lowest ? ob < best : ob > best;
        if (oi != 0x7fffffff && (bi == 0x7fffffff || better || (ob == best && oi < bi))) {
          best = ob;
          bi = oi;
        }
      }
      pick = bi;
    }
  }
  // commit, compacting the committed positions in ascending order
  int written = 0;
  for (int c = s; c < e; c += 64) {
    const int k = c + lane;
    const bool masked = k < e && mask[base + k] != 0;
    const bool commit = masked && (fb ? (k == pick) : (conf[base + k] > tau));
    const unsigned long long bm = ballot(commit);
    if (commit) {
      tokens[base + k] = argmax[base + k];
      mask[base + k] = 0;
      if (my_commits) {
        const unsigned long long below = bm & ((1ull << lane) - 1ull);
        my_commits[written + __popcll(below)] = k;
      }
    }
    written += __popcll(bm);
  }
  if (my_commits)
    for (int i = written + lane; i < BL; i += 64) my_commits[i] = -1;
  if (lane == 0) {
    fallback[b] = fb ? 1 : 0;
    block_start[b] = s;
    if (ncommit) ncommit[b] = written;
  }
}

// Element k of sequence b: row-major (b * L + k) or position-major
// (k * B + b) state arrays.
struct RowMajor {
  int L;
  __device__ size_t operator()(int b, int k) const { return (size_t)b * L + k; }
};
struct PosMajor {
  int B;
  __device__ size_t operator()(int b, int k) const { return (size_t)k * B + b; }
};

// The unmasking rule for sequence b by one lane, visiting the positions one
// by one from block start s (already read from block_start[b]): skip
// forward to the first block holding a masked position, then the threshold
// set, the fallback pick and the commits.
template <class At>
__device__ void lane_rule(int b, int s, int L, int BL, float tau, int rule,
                          const float* __restrict__ conf, const float* __restrict__ entropy,
                          const float* __restrict__ uniform, const int32_t* __restrict__ argmax,
                          int32_t* __restrict__ tokens, uint8_t* __restrict__ mask,
                          int32_t* __restrict__ block_start, int32_t* __restrict__ fallback,
                          int32_t* __restrict__ ncommit, int32_t* __restrict__ my_commits,
                          At at) {
  if (s < 0 || s > L) {
    fallback[b] = -2;
    if (ncommit) ncommit[b] = 0;
    if (my_commits)
      for (int i = 0; i < BL; ++i) my_commits[i] = -1;
    return;
  }
  bool found = false;
  while (s < L) {
    const int e = min(s + BL, L);
    for (int k = s; k < e && !found; ++k) found = mask[at(b, k)] != 0;
    if (found) break;
    s += BL;
  }
  if (!found) {
    fallback[b] = -1;
    if (ncommit) ncommit[b] = 0;
    if (my_commits)
      for (int i = 0; i < BL; ++i) my_commits[i] = -1;
    return;
  }
  const int e = min(s + BL, L);
  // threshold count, masked count, leftmost masked, extreme of the key
  const float* key = rule == kMaxEnt ? entropy : conf;
  const bool extreme = rule == kMaxConf || rule == kMinConf || rule == kMaxEnt;
  const bool lowest = rule == kMinConf;
  int npass = 0, n = 0, first = -1, bi = -1;
  float best = 0.f;
  for (int k = s; k < e; ++k) {
    const size_t idx = at(b, k);
    if (!mask[idx]) continue;
    ++n;
    if (first < 0) first = k;
    if (conf[idx] > tau) ++npass;
    if (extreme) {
      const float v = key[idx];
      if (bi < 0 || (lowest ? v < best : v > best)) {
        best = v;
        bi = k;
      }
    }
  }
  const bool fb = npass == 0;
  int pick = -1;
  if (fb) {
    if (rule == kLeftmost) {
      pick = first;
    } else if (rule == kRandom) {
      int j = (int)(uniform[b] * (float)n);
      j = j > n - 1 ? n - 1 : (j < 0 ? 0 : j);
      for (int k = s; k < e; ++k)
        if (mask[at(b, k)] && j-- == 0) {
          pick = k;
          break;
        }
    } else {
      pick = bi;
    }
  }
  int written = 0;
  for (int k = s; k < e; ++k) {
    const size_t idx = at(b, k);
    if (!mask[idx]) continue;
    if (fb ? (k == pick) : (conf[idx] > tau)) {
      tokens[idx] = argmax[idx];
      mask[idx] = 0;
      if (my_commits) my_commits[written] = k;
      ++written;
    }
  }
  if (my_commits)
    for (int i = written; i < BL; ++i) my_commits[i] = -1;
  fallback[b] = fb ? 1 : 0;
  block_start[b] = s;
  if (ncommit) ncommit[b] = written;
}

// The same rule with one lane per sequence, for large batches of short
// blocks: each lane walks its block position by position, so a wave keeps
// the loads of 64 sequences in flight instead of one (the wave-per-sequence
// kernel is latency-bound once B reaches thousands).  Decisions are those of
// select_kernel: binary32 threshold test, lowest position on ties.
__global__ __launch_bounds__(256) void select_lanes_kernel(
    int B, int L, int BL, float tau, int rule, const float* __restrict__ conf,
    const float* __restrict__ entropy, const float* __restrict__ uniform,
    const int32_t* __restrict__ argmax, int32_t* __restrict__ tokens,
    uint8_t* __restrict__ mask, int32_t* __restrict__ block_start,
    int32_t* __restrict__ fallback, int32_t* __restrict__ ncommit,
    int32_t* __restrict__ commit_pos) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const size_t base = (size_t)b * L;
  int32_t* my_commits = commit_pos ? commit_pos + (size_t)b * BL : nullptr;
  int s = block_start[b];
  if (s < 0 || s > L) {
    fallback[b] = -2;
    if (ncommit) ncommit[b] = 0;
    if (my_commits)
      for (int i = 0; i < BL; ++i) my_commits[i] = -1;
    return;
  }
  // Blocks of at most 32 positions whose 32 entries from s stay in the row
  // and start 16-byte aligned: mask and confidences come in with wide loads
  // issued together and the decision is taken on a bitmask in registers.
  if (rule != kMaxEnt && BL <= 32 && s + 32 <= L &&
      ((reinterpret_cast<uintptr_t>(mask + base + s) | reinterpret_cast<uintptr_t>(conf + base + s)) &
       15) == 0) {
    const int cnt = min(BL, L - s);
    const uint4 mv0 = *reinterpret_cast<const uint4*>(mask + base + s);
    const uint4 mv1 = *reinterpret_cast<const uint4*>(mask + base + s + 16);
    float c[32];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 v = *reinterpret_cast<const float4*>(conf + base + s + 4 * q);
      c[4 * q] = v.x;
      c[4 * q + 1] = v.y;
      c[4 * q + 2] = v.z;
      c[4 * q + 3] = v.w;
    }
    const uint32_t mw[8] = {mv0.x, mv0.y, mv0.z, mv0.w, mv1.x, mv1.y, mv1.z, mv1.w};
    uint32_t mbits = 0, pbits = 0;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const bool m = i < cnt && ((mw[i >> 2] >> (8 * (i & 3))) & 0xffu) != 0;
      mbits |= (uint32_t)m << i;
      pbits |= (uint32_t)(m && c[i] > tau) << i;
    }
    if (mbits != 0) {  // the block at s is the active block
      const bool fb = pbits == 0;
      uint32_t commit = pbits;
      if (fb) {
        int pick = 0;
        if (rule == kLeftmost) {
          pick = __ffs(mbits) - 1;
        } else if (rule == kRandom) {
          const int n = __popc(mbits);
          int j = (int)(uniform[b] * (float)n);
          j = j > n - 1 ? n - 1 : (j < 0 ? 0 : j);
          uint32_t rest = mbits;
          for (int t = 0; t < j; ++t) rest &= rest - 1;  // drop the j lowest
          pick = __ffs(rest) - 1;
        } else {
          const bool lowest = rule == kMinConf;
          float best = 0.f;
          int bi = -1;
#pragma unroll
          for (int i = 0; i < 32; ++i)
            if (((mbits >> i) & 1u) && (bi < 0 || (lowest ? c[i] < best : c[i] > best))) {
              best = c[i];
              bi = i;
            }
          pick = bi;
        }
        commit = 1u << pick;
      }
      int written = 0;
      for (uint32_t rest = commit; rest; rest &= rest - 1) {
        const int k = s + __ffs(rest) - 1;
        tokens[base + k] = argmax[base + k];
        mask[base + k] = 0;
        if (my_commits) my_commits[written] = k;
        ++written;
      }
      if (my_commits)
        for (int i = written; i < BL; ++i) my_commits[i] = -1;
      fallback[b] = fb ? 1 : 0;
      block_start[b] = s;
      if (ncommit) ncommit[b] = written;
      return;
    }
    s += BL;  // nothing masked there: continue the skip-forward below
  }
  lane_rule(b, s, L, BL, tau, rule, conf, entropy, uniform, argmax, tokens, mask, block_start,
            fallback, ncommit, my_commits, RowMajor{L});
}

// Position-major state (element (b, k) at k * B + b): one lane per group of
// kS consecutive sequences (kS = 4 for large batches, 1 otherwise, so that
// small batches still spread over many waves).  When the group shares its
// block start and the block has at most 32 positions, each position of the
// block comes in as one load of the group's kS confidences (and keys) and
// one of its kS mask bytes, so a wave's loads cover whole cache lines.
// Loads are issued kChunk positions at a time, with the next batch in flight
// while one is decided when kDB; every load is unconditional (positions past
// the block re-read its last one and are ignored), so the compiler counts
// the loads in flight instead of waiting for all of them.  Confidences, keys
// and mask bytes are read once, with nontemporal loads.  The rule class is a
// template parameter: the threshold, leftmost and random rules load no keys.
// For kS = 4, when the group's four sequences each commit one position, the
// same one, the candidates, tokens and mask bytes move as one 16-byte and one
// 4-byte access, and the per-sequence outputs are stored as 16-byte vectors
// (the host launches kS = 4 only when every array is aligned for that).
// Sequences outside these cases take the position-by-position path.
// Decisions are those of the row-major kernels.
typedef float f32x4 __attribute__((ext_vector_type(4)));
template <int kS> struct PmVec;
template <> struct PmVec<1> {
  typedef float F;
  typedef uint8_t M;
  static __device__ float get(F v, int) { return v; }
};
template <> struct PmVec<4> {
  typedef f32x4 F;
  typedef uint32_t M;
  static __device__ float get(F v, int j) { return v[j]; }
};

template <int kS, int kChunk, bool kDB, bool kExtreme>
__global__ __launch_bounds__(256) void select_pm_kernel(
    int B, int L, int BL, float tau, int rule, const float* __restrict__ conf,
    const float* __restrict__ entropy, const float* __restrict__ uniform,
    const int32_t* __restrict__ argmax, int32_t* __restrict__ tokens,
    uint8_t* __restrict__ mask, int32_t* __restrict__ block_start,
    int32_t* __restrict__ fallback, int32_t* __restrict__ ncommit,
    int32_t* __restrict__ commit_pos) {
  typedef typename PmVec<kS>::F VF;
  typedef typename PmVec<kS>::M VM;
  static_assert(kS == 1 || kS == 4, "one or four sequences per lane");
  const int b0 = kS * (blockIdx.x * 256 + threadIdx.x);
  if (b0 >= B) return;
  const PosMajor at{B};
  const float* key = rule == kMaxEnt ? entropy : conf;
  const bool lowest = rule == kMinConf;
  // the group's block starts in one load (kS = 4: B % 4 == 0, 16-byte aligned)
  int sv[kS];
  if (kS == 4) {
    const int4 v = *reinterpret_cast<const int4*>(block_start + b0);
    sv[0] = v.x;
    sv[kS > 1 ? 1 : 0] = v.y;
    sv[kS > 2 ? 2 : 0] = v.z;
    sv[kS > 3 ? 3 : 0] = v.w;
  } else {
    sv[0] = block_start[b0];
  }
  const int s = sv[0];
  int differ = 0;
#pragma unroll
  for (int j = 1; j < kS; ++j) differ |= sv[j] ^ s;
  // no short-circuit: the compiler would otherwise split the load above
  const bool wide = (differ == 0) & (s >= 0) & (s + BL <= L) & (BL <= 32);
  if (!wide) {
#pragma unroll 1
    for (int j = 0; j < kS; ++j) {
      const int b = b0 + j;
      lane_rule(b, sv[j], L, BL, tau, rule, conf, entropy, uniform, argmax, tokens, mask,
                block_start, fallback, ncommit,
                commit_pos ? commit_pos + (size_t)b * BL : nullptr, at);
    }
    return;
  }
  uint32_t mb[kS], pb[kS];
  float best[kS];
  int bi[kS];
#pragma unroll
  for (int j = 0; j < kS; ++j) {
    mb[j] = pb[j] = 0;
    best[j] = 0.f;
    bi[j] = -1;
  }
  VM mv[2][kChunk];
  VF cv[2][kChunk], kv[2][kChunk];
  auto load = [&](auto bufc, int i0) {
    constexpr int buf = decltype(bufc)::value;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      // positions past the block re-read its last one (in bounds, ignored)
      const size_t row = (size_t)(s + min(i0 + u, BL - 1)) * B + b0;
      mv[buf][u] = __builtin_nontemporal_load(reinterpret_cast<const VM*>(mask + row));
      cv[buf][u] = __builtin_nontemporal_load(reinterpret_cast<const VF*>(conf + row));
      if (kExtreme) kv[buf][u] = __builtin_nontemporal_load(reinterpret_cast<const VF*>(key + row));
    }
  };
  auto decide = [&](auto bufc, int i0) {
    constexpr int buf = decltype(bufc)::value;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const int i = i0 + u;
      const bool in = i < BL;
#pragma unroll
      for (int j = 0; j < kS; ++j) {
        const bool m = in & ((((uint32_t)mv[buf][u] >> (8 * j)) & 0xffu) != 0);
        const float c = PmVec<kS>::get(cv[buf][u], j);
        mb[j] |= (uint32_t)m << (i & 31);
        pb[j] |= (uint32_t)(m & (c > tau)) << (i & 31);
        if (kExtreme) {
          // branch-free: a select per value (lowest position on equal keys)
          const float k = PmVec<kS>::get(kv[buf][u], j);
          const bool better = lowest ? k < best[j] : k > best[j];
          const bool take = m & ((bi[j] < 0) | better);
          best[j] = take ? k : best[j];
          bi[j] = take ? i : bi[j];
        }
      }
    }
  };
  using Buf0 = std::integral_constant<int, 0>;
  using Buf1 = std::integral_constant<int, 1>;
  if (kDB) {
    load(Buf0{}, 0);
    for (int i0 = 0; i0 < BL; i0 += 2 * kChunk) {
      load(Buf1{}, i0 + kChunk);
      decide(Buf0{}, i0);
      load(Buf0{}, i0 + 2 * kChunk);
      decide(Buf1{}, i0 + kChunk);
    }
  } else {
    for (int i0 = 0; i0 < BL; i0 += kChunk) {
      load(Buf0{}, i0);
      decide(Buf0{}, i0);
    }
  }
  // positions to commit and the fallback flag of each sequence
  uint32_t commit[kS];
  int fbv[kS];
  bool any_empty = false;
#pragma unroll
  for (int j = 0; j < kS; ++j) {
    any_empty = any_empty || mb[j] == 0;
    const bool fb = pb[j] == 0;
    commit[j] = pb[j];
    fbv[j] = fb ? 1 : 0;
    if (fb && mb[j] != 0) {
      int pick;
      if (rule == kLeftmost) {
        pick = __ffs(mb[j]) - 1;
      } else if (rule == kRandom) {
        const int n = __popc(mb[j]);
        int r = (int)(uniform[b0 + j] * (float)n);
        r = r > n - 1 ? n - 1 : (r < 0 ? 0 : r);
        uint32_t rest = mb[j];
        for (int t = 0; t < r; ++t) rest &= rest - 1;  // drop the r lowest
        pick = __ffs(rest) - 1;
      } else {
        pick = bi[j];
      }
      commit[j] = 1u << pick;
    }
  }
  if (kS == 4 && !any_empty && commit_pos == nullptr) {
    bool same1 = (commit[0] & (commit[0] - 1)) == 0;
#pragma unroll
    for (int j = 1; j < kS; ++j) same1 = same1 && commit[j] == commit[0];
    if (same1) {
      const size_t row = (size_t)(s + __ffs(commit[0]) - 1) * B + b0;
      *reinterpret_cast<int4*>(tokens + row) = *reinterpret_cast<const int4*>(argmax + row);
      *reinterpret_cast<uint32_t*>(mask + row) = 0u;
    } else {
#pragma unroll
      for (int j = 0; j < kS; ++j)
        for (uint32_t rest = commit[j]; rest; rest &= rest - 1) {
          const size_t idx = at(b0 + j, s + __ffs(rest) - 1);
          tokens[idx] = argmax[idx];
          mask[idx] = 0;
        }
    }
    *reinterpret_cast<int4*>(fallback + b0) =
        make_int4(fbv[0], fbv[kS > 1 ? 1 : 0], fbv[kS > 2 ? 2 : 0], fbv[kS > 3 ? 3 : 0]);
    *reinterpret_cast<int4*>(block_start + b0) = make_int4(s, s, s, s);
    if (ncommit)
      *reinterpret_cast<int4*>(ncommit + b0) =
          make_int4(__popc(commit[0]), __popc(commit[kS > 1 ? 1 : 0]),
                    __popc(commit[kS > 2 ? 2 : 0]), __popc(commit[kS > 3 ? 3 : 0]));
    return;
  }
#pragma unroll
  for (int j = 0; j < kS; ++j) {
    const int b = b0 + j;
    int32_t* my_commits = commit_pos ? commit_pos + (size_t)b * BL : nullptr;
    if (mb[j] == 0) {  // nothing masked in the block at s: skip forward
      lane_rule(b, s, L, BL, tau, rule, conf, entropy, uniform, argmax, tokens, mask,
                block_start, fallback, ncommit, my_commits, at);
      continue;
    }
    int written = 0;
    for (uint32_t rest = commit[j]; rest; rest &= rest - 1) {
      const int k = s + __ffs(rest) - 1;
      const size_t idx = at(b, k);
      tokens[idx] = argmax[idx];
      mask[idx] = 0;
      if (my_commits) my_commits[written] = k;
      ++written;
    }
    if (my_commits)
      for (int i = written; i < BL; ++i) my_commits[i] = -1;
    fallback[b] = fbv[j];
    block_start[b] = s;
    if (ncommit) ncommit[b] = written;
  }
}

// Active block of each sequence (first block from block_start holding a
// masked position, as in the selection) expanded to its rows.
__global__ __launch_bounds__(64) void active_rows_kernel(int L, int BL,
                                                        const uint8_t* __restrict__ mask,
                                                        const int32_t* __restrict__ block_start,
                                                        int32_t* __restrict__ rowlist,
                                                        int32_t* __restrict__ rowmap) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const size_t base = (size_t)b * L;
  int s = block_start[b];
  bool found = false;
  if (s >= 0 && s <= L) {
    while (s < L) {
      const int e = min(s + BL, L);
      for (int c = s; c < e; c += 64) {
        const int k = c + lane;
        if (ballot(k < e && mask[base + k] != 0)) {
          found = true;
          break;
        }
      }
      if (found) break;
      s += BL;
    }
  }
  const int e = found ? min(s + BL, L) : 0;
  if (rowlist)
    for (int i = lane; i < BL; i += 64)
      rowlist[(size_t)b * BL + i] = (found && s + i < e) ? (int32_t)(base + s + i) : -1;
  if (rowmap)
    for (int k = lane; k < L; k += 64)
      rowmap[base + k] = (found && k >= s && k < e) ? (int32_t)(base + k) : -1;
}

}  // namespace

hipError_t launch_active_rows(int B, int L, int block_len, const uint8_t* mask,
                              const int32_t* block_start, int32_t* rowlist, int32_t* rowmap,
                              hipStream_t stream) {
  hipLaunchKernelGGL(active_rows_kernel, dim3((unsigned)B), dim3(64), 0, stream, L, block_len,
                     mask, block_start, rowlist, rowmap);
  return hipGetLastError();
}

hipError_t launch_merge(const float4* partials, int M, int nvt, float* conf,
                        float* entropy, float* logp, float* lse, int32_t* argmax,
                        const int32_t* rowlist, const int32_t* sample_row,
                        const float4* spartials, const int32_t* token, const float* ztoken,
                        int V, hipStream_t stream) {
  const dim3 grid((unsigned)((M + kMergePositions - 1) / kMergePositions));
  const dim3 block(kMergeThreads);
  hipLaunchKernelGGL(merge_kernel, grid, block, 0, stream, partials, M, nvt, conf,
                     entropy, logp, lse, argmax, rowlist, sample_row, spartials, token, ztoken,
                     V);
  return hipGetLastError();
}

hipError_t launch_select(int B, int L, int block_len, float tau, int rule,
                         const float* conf, const float* entropy, const float* uniform,
                         const int32_t* argmax, int32_t* tokens, uint8_t* mask,
                         int32_t* block_start, int32_t* fallback, int32_t* ncommit,
                         int32_t* commit_pos, bool position_major, hipStream_t stream) {
  if (position_major) {
    const bool extreme = rule == kMaxConf || rule == kMinConf || rule == kMaxEnt;
    // four sequences per lane: whole 16-byte groups, every array aligned
    auto a16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    const bool four = B >= kPmWideMinB && B % 4 == 0 && a16(conf) && a16(argmax) &&
                      a16(tokens) && a16(block_start) && a16(fallback) &&
                      (ncommit == nullptr || a16(ncommit)) &&
                      (rule != kMaxEnt || a16(entropy)) &&
                      (reinterpret_cast<uintptr_t>(mask) & 3) == 0;
    const dim3 grid((unsigned)(((four ? B / 4 : B) + 255) / 256));
#define FORK_SELECT_PM(S, C, D, X)                                                          \
  hipLaunchKernelGGL((select_pm_kernel<S, C, D, X>), grid, dim3(256), 0, stream, B, L,       \
                     block_len, tau, rule, conf, entropy, uniform, argmax, tokens, mask,     \
                     block_start, fallback, ncommit, commit_pos)
    if (four && extreme) FORK_SELECT_PM(4, 1, true, true);
    else if (four) FORK_SELECT_PM(4, 1, true, false);
    else if (extreme) FORK_SELECT_PM(1, 16, false, true);
    else FORK_SELECT_PM(1, 16, false, false);
#undef FORK_SELECT_PM
  }
  else if (B >= kLaneSelectMinB && block_len <= kLaneSelectMaxBL)
    hipLaunchKernelGGL(select_lanes_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0,
                       stream, B, L, block_len, tau, rule, conf, entropy, uniform, argmax,
                       tokens, mask, block_start, fallback, ncommit, commit_pos);
  else
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)B), dim3(64), 0, stream, L,
                       block_len, tau, rule, conf, entropy, uniform, argmax, tokens, mask,
                       block_start, fallback, ncommit, commit_pos);
  return hipGetLastError();
}

}  // namespace fork
