// LM-head projection fused with the per-position vocabulary reductions.
//
// For every position r (a row of `hidden`) the model's categorical over the
// vocabulary is softmax(z) with z_v = <hidden_r, W_v> (Fork-dLLM paper,
// Section 2, "Sampling in masked dLLMs").  The step needs, per position, the
// greedy candidate, its probability (the confidence c_t^k), its log-
// probability (ForkGRPO's ratio, Section 3.2) and the entropy (Section 3.1).
// All of them follow from four numbers per (position, vocabulary tile) that
// this kernel produces straight from the MFMA accumulators, so the [M, V]
// logits never leave the registers:
//   m   = max_v z_v                 idx = lowest v attaining m
//   s   = sum_v exp(z_v - m)        t   = sum_v exp(z_v - m) * (z_v - m)
//
// Work decomposition (gfx950 / CDNA4), common to both element types:
//   * one workgroup = 256 vocabulary rows x 256 positions, 8 wave64s laid out
//     2 (vocabulary) x 4 (positions); each wave owns 128 x 64 outputs (fp32
//     accumulators): 8 x 4 blocks of 16 x 16 (v_mfma_f32_16x16x32_bf16) on
//     the bf16 path, 4 x 2 blocks of 32 x 32 (v_mfma_f32_32x32x2f32) on the
//     fp32 path;
//   * the MFMA "A" operand is W (vocabulary on the MFMA M axis) and "B" is
//     hidden, so each lane's accumulators hold vocabulary values of whole
//     positions: the vocabulary reduction is mostly in-lane (32 or 64 values
//     per position), plus shuffles between the lanes holding the same
//     position and one LDS exchange between the two vocabulary waves;
//   * K is staged through LDS in 128-byte slabs per row (whole cache lines),
//     the 16-byte chunk c of row r stored at chunk slot c ^ f(r) with
//     f(r) = (r & 7) ^ ((r >> 3) & 1): the fragment reads of 16 consecutive
//     lanes (16 rows, one chunk) then hit 16 distinct bank groups;
//   * workgroups are renumbered so that each XCD (private L2) walks a
//     contiguous range of tiles, sweeping groups of kGroupV vocabulary
//     stripes across all position tiles, so concurrently running workgroups
//     share W and hidden stripes in L2.
//
// bf16 path (the hot one): K is fed to LDS by buffer loads that write LDS
// directly (no register staging).  W gets a 3-slot ring (prefetched two
// stages ahead: it streams from HBM), hidden a 2-slot ring (one stage ahead:
// it stays in the last-level cache): 5 x 32 KiB = the whole 160 KiB of LDS.
// One barrier per 64-element K stage, placed after the first MFMAs of the
// stage's second 32-element step so that queued MFMAs cover it; the fragment
// reads of the next step are interleaved with the current MFMAs, and the
// buffer loads of later stages are spread over the stage one at a time so
// that no wave stalls its MFMA stream behind a burst of loads.  The 16x16x32
// MFMA shape moves the same bytes per flop as 32x32x16 and, on gfx950,
// sustains a higher clock under the same power limit.
// fp32 path (small problems): register-staged double buffer.
//
// Drawn candidates (sampling temperature tau > 0, Section 2): for the
// positions the caller marks, the epilogue also keeps the maximiser of the
// Gumbel-perturbed keys z_v / tau - log E_v, where E_v = -log(1 - U_v) is an
// exponential draw built from Philox4x32-10 (Salmon et al., SC'11) at
// counter (v / 4, row, step counter, 0): one generator call serves the four
// consecutive vocabulary entries a lane holds in one accumulator group.
#include "fork_kernels.h"

#include <math.h>

#include <type_traits>

namespace fork {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;
constexpr int kSlab = 128;                   // bytes of K per row per stage
constexpr int kOperandBytes = 256 * kSlab;   // 32 KiB: one operand, one stage
constexpr int kGroupV = 8;                   // vocab stripes per sweep group
constexpr int kXcds = 8;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Raw-buffer descriptor word 3 for gfx9-family buffers: 32-bit data format,
// offsets checked against the record count (out of range reads return 0).
constexpr int kBufferWord3 = 0x00020000;
constexpr unsigned kOutOfRange = 0x80000000u;

static_assert(kTileV == 256 && kTileP == 256, "tile layout assumes 256 x 256");

__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * kSlab + ((chunk ^ swz(row)) << 4);
}

// Maps the hardware workgroup id to (vocabulary tile, position tile).
__device__ __forceinline__ void map_tile(int bid, int nvt, int npt, int& vt, int& pt) {
  const int n = nvt * npt;
  // Workgroups are dealt to the XCDs round-robin: XCD x gets x, x+8, ...
  const int x = bid % kXcds, i = bid / kXcds;
  const int base = n / kXcds, rem = n % kXcds;
  const int logical = x * base + min(x, rem) + i;
  const int per_group = kGroupV * npt;
  const int group = logical / per_group;
  const int in = logical - group * per_group;
  const int gv0 = group * kGroupV;
  const int gvn = min(kGroupV, nvt - gv0);
  pt = in / gvn;
  vt = gv0 + (in - pt * gvn);
}

// Merge of two partials (either may be empty, s == 0).
__device__ __forceinline__ float4 merge2(float4 a, float4 b) {
  if (b.y == 0.f) return a;
  if (a.y == 0.f) return b;
  const float m = fmaxf(a.x, b.x);
  const float ea = exp2f((a.x - m) * kLog2e), eb = exp2f((b.x - m) * kLog2e);
  float4 r;
  r.x = m;
  r.y = a.y * ea + b.y * eb;
  r.z = ea * (a.z + (a.x - m) * a.y) + eb * (b.z + (b.x - m) * b.y);
  const int ia = __float_as_int(a.w), ib = __float_as_int(b.w);
  const bool take_a = (a.x > b.x) || (a.x == b.x && ia < ib);
  r.w = __int_as_float(take_a ? ia : ib);
  return r;
}

// Philox4x32-10: ten rounds of the 4x32 S-box (two 32 x 32 -> 64-bit
// products whose halves are exchanged and mixed with the other counter words
// and the round key), the key advanced by the Weyl constants between rounds.
// Each product is one 32 x 32 -> 64-bit multiply (v_mad_u64_u32).
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1,
                   (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Gumbel key of one logit: z / tau - log E with E = -log(1 - U) and U on the
// odd grid (2 (w >> 9) + 1) 2^-24 of (0, 1).  1 - U is exact in binary32, so
// E comes from the hardware base-2 logarithm, except below U = 2^-7, where
// the series U + U^2/2 + U^3/3 + U^4/4 (relative error < U^4/5 < 2^-30)
// avoids the cancellation of a logarithm near 1.  The key carries a relative
// error of about 1e-6 in E, far below the logit rounding.
__device__ __forceinline__ float gumbel_key(float z, float inv_tau, uint32_t w) {
  const float u = (float)(2u * (w >> 9) + 1u) * 0x1p-24f;
  const float series = u * fmaf(u, fmaf(u, fmaf(u, 0.25f, 1.0f / 3.0f), 0.5f), 1.0f);
  const float viaLog = -__builtin_amdgcn_logf(1.0f - u) * kLn2;
  const float e = u < 0x1p-7f ? series : viaLog;
  return fmaf(z, inv_tau, -__builtin_amdgcn_logf(e) * kLn2);
}

// Accumulator layouts.  In both, a lane's accumulators hold vocabulary values
// (MFMA rows) of whole positions (MFMA columns), so the reduction over the
// vocabulary is mostly in-lane.
//
// Acc16 (bf16 path, v_mfma_f32_16x16x32_bf16): a wave's 128 x 64 outputs are
// 8 x 4 blocks of 16 x 16; element e of block (i, j) in lane l is row
// 16 i + 4 (l / 16) + e, column 16 j + l % 16.  The four lanes l % 16 + 16 g
// (g = 0..3) hold the 128 rows of a column, 32 each.
struct Acc16 {
  typedef f32x4 Arr[8][4];
  static constexpr int kNI = 8, kNJ = 4, kNE = 4;
  static constexpr int kLeaders = 16;  // lanes 0..15 hold one copy of each column
  __device__ static float get(const Arr& a, int i, int j, int e) { return a[i][j][e]; }
  __device__ static void set(Arr& a, int i, int j, int e, float v) { a[i][j][e] = v; }
  __device__ static int row(int i, int e, int lane) { return i * 16 + (lane >> 4) * 4 + e; }
  __device__ static int col(int j, int lane) { return j * 16 + (lane & 15); }
  // combine the copies of a column: lanes 16 and 32 apart
  template <class F>
  __device__ static void across(F&& f) {
    f(16);
    f(32);
  }
};

// Acc32 (fp32 path, v_mfma_f32_32x32x2f32): 4 x 2 blocks of 32 x 32; element
// e of block (i, j) in lane l is row 32 i + 8 (e / 4) + 4 (l / 32) + e % 4,
// column 32 j + l % 32.  Lanes l and l ^ 32 hold the 128 rows of a column.
struct Acc32 {
  typedef f32x16 Arr[4][2];
  static constexpr int kNI = 4, kNJ = 2, kNE = 16;
  static constexpr int kLeaders = 32;
  __device__ static float get(const Arr& a, int i, int j, int e) { return a[i][j][e]; }
  __device__ static void set(Arr& a, int i, int j, int e, float v) { a[i][j][e] = v; }
  __device__ static int row(int i, int e, int lane) {
    return i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
  }
  __device__ static int col(int j, int lane) { return j * 32 + (lane & 31); }
  template <class F>
  __device__ static void across(F&& f) {
    f(32);
  }
};

// What the epilogue produces besides the per-tile statistics.
enum EpilogueMode { kGreedy = 0, kDrawn = 1, kTarget = 2 };

// Per-position inputs of the epilogue, loaded before the last MFMAs so that
// their latency is hidden: the given token (kTarget) or the draw's row index
// (kDrawn) of each column this lane holds.
template <class Lay>
struct ColIn {
  int col[Lay::kNJ];
};

// Launch position of column c (0..255) of position tile pt.  Contiguous:
// p0 + c.  Interleaved (M = 256 * npt, the drawing kernel over all rows):
// 16-column block k of tile pt is the 16-row chunk k * npt + (pt + k) mod
// npt, i.e. column c is row of that chunk's c % 16-th; chunk k * npt + s
// goes to tile (s - k) mod npt.  The active blocks, the only rows whose
// candidates are drawn, usually sit at a fixed offset in every sequence;
// the rotation by k spreads them over the position tiles instead of
// gathering them in a few (which a plain stride of npt chunks does whenever
// the sequence length is a multiple of 16 npt), so the tiles' epilogues
// cost about the same.
struct PosMap {
  int p0, pt, npt;
  bool ilv;
  __device__ int operator()(int c) const {
    const int k = c >> 4;
    return ilv ? ((k * npt + (pt + k) % npt) << 4) + (c & 15) : p0 + c;
  }
};

template <class Lay, int kMode>
__device__ __forceinline__ void load_col_inputs(ColIn<Lay>& ci, int tid, int lane, int wp,
                                                const PosMap& pos, int M, const SampleArgs& sa,
                                                const TargetArgs& ta) {
  if (kMode == kGreedy) return;
  const int32_t* src = kMode == kTarget ? ta.token : sa.row;
#pragma unroll
  for (int j = 0; j < Lay::kNJ; ++j) {
    const int p = pos(wp * 64 + Lay::col(j, lane));
    ci.col[j] = p < M ? src[p] : -1;
  }
}

// Statistics of the logits of column j that this lane holds (rows vbase +
// Lay::row(i, e, lane), increasing in (i, e)), combined with the lanes that
// hold the column's other rows: the maximum m, the lowest row holding it,
// s = sum e^(z-m) and t = sum e^(z-m)(z-m).  Branch-free.  Unless kFull
// (every row < V), rows past V are set to -inf in acc first, so that no pass
// needs a row test.
template <class Lay, bool kFull>
__device__ __forceinline__ void column_stats(typename Lay::Arr& acc, int j, int lane, int vbase,
                                             int V, float& m_out, int& idx_out, float& s_out,
                                             float& t_out) {
  if (!kFull) {
#pragma unroll
    for (int i = 0; i < Lay::kNI; ++i)
#pragma unroll
      for (int e = 0; e < Lay::kNE; ++e)
        if (vbase + Lay::row(i, e, lane) >= V) Lay::set(acc, i, j, e, -INFINITY);
  }
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < Lay::kNI; ++i)
#pragma unroll
    for (int e = 0; e < Lay::kNE; ++e) m = fmaxf(m, Lay::get(acc, i, j, e));
  // the lowest row holding m: scan from the highest row down
  int idx = 0x7fffffff;
#pragma unroll
  for (int i = Lay::kNI - 1; i >= 0; --i)
#pragma unroll
    for (int e = Lay::kNE - 1; e >= 0; --e)
      idx = Lay::get(acc, i, j, e) == m ? vbase + Lay::row(i, e, lane) : idx;
  Lay::across([&](int off) {
    const float mo = __shfl_xor(m, off);
    const int io = __shfl_xor(idx, off);
    const bool take = mo > m || (mo == m && io < idx);
    m = take ? mo : m;
    idx = take ? io : idx;
  });
  float s = 0.f, tl = 0.f;
  if (m > -INFINITY) {
    const float nml = -m * kLog2e;
#pragma unroll
    for (int i = 0; i < Lay::kNI; ++i)
#pragma unroll
      for (int e = 0; e < Lay::kNE; ++e) {
        // (z - m) * log2(e) with one rounding; the moment is summed in
        // these units and scaled by ln 2 once
        const float dl = fmaf(Lay::get(acc, i, j, e), kLog2e, nml);
        const float ex = __builtin_amdgcn_exp2f(dl);
        s += ex;
        // a -inf row has ex = 0: keep 0 * -inf out of the moment
        tl = fmaf(ex, kFull ? dl : fmaxf(dl, -1e30f), tl);
      }
  }
  // lanes holding the same column add in the same order: identical results
  Lay::across([&](int off) {
    s += __shfl_xor(s, off);
    tl += __shfl_xor(tl, off);
  });
  m_out = m;
  idx_out = idx;
  s_out = s;
  t_out = tl * kLn2;
}

// Per-(position, tile) statistics from the accumulators of one wave, combined
// across the two vocabulary waves through LDS, stored to partials.  Drawn
// candidates (kDrawn) go through a second LDS exchange and a second partials
// array (see SampleArgs); the logit of a given token (kTarget) is stored by
// the one lane that holds it.  kFull: the tile's 256 vocabulary rows are all
// < V (every tile but a ragged last one), so no row test is compiled in.
template <class Lay, int kMode, bool kFull>
__device__ __forceinline__ void epilogue_tile(typename Lay::Arr& acc, unsigned char* smem,
                                              int tid, int lane, int wv, int wp, int vt, int v0,
                                              const PosMap& pos, int M, int V,
                                              float4* __restrict__ partials, const SampleArgs& sa,
                                              const TargetArgs& ta, const ColIn<Lay>& ci) {
  constexpr bool kDraw = kMode == kDrawn;
  constexpr bool full = kFull;
  float4* red = reinterpret_cast<float4*>(smem);  // [2][kTileP]
  float4* sred = red + 2 * kTileP;                // [2][kTileP], drawn candidates
  const int vbase = v0 + wv * 128;
  const bool leader = lane < Lay::kLeaders;
  // the draw's row of this thread's position, for the store after the exchange
  const int own_pos = pos(tid < kTileP ? tid : 0);
  const int own_row = (kDraw && tid < kTileP && own_pos < M) ? sa.row[own_pos] : -1;
#pragma unroll
  for (int j = 0; j < Lay::kNJ; ++j) {
    float m, s, t;
    int idx;
    column_stats<Lay, kFull>(acc, j, lane, vbase, V, m, idx, s, t);
    const int col = wp * 64 + Lay::col(j, lane);
    if (leader) red[wv * kTileP + col] = make_float4(m, s, t, __int_as_float(idx));
    if (kMode == kTarget) {
      const int tk = ci.col[j];
      if (tk >= vbase && tk < vbase + 128 && tk < V) {
        float zt = 0.f;
        bool hit = false;
#pragma unroll
        for (int i = 0; i < Lay::kNI; ++i)
#pragma unroll
          for (int e = 0; e < Lay::kNE; ++e)
            if (vbase + Lay::row(i, e, lane) == tk) {
              zt = Lay::get(acc, i, j, e);
              hit = true;
            }
        if (hit) ta.z[pos(col)] = zt;
      }
    }
    if (kDraw) {
      const int srow = ci.col[j];
      if (__ballot(srow >= 0)) {
        float best = -INFINITY, bz = 0.f;
        int bidx = 0x7fffffff;
        if (srow >= 0) {
          // elements 4g .. 4g + 3 of a block are four consecutive rows from
          // a multiple of 4: one generator call yields their four words
#pragma unroll
          for (int i = 0; i < Lay::kNI; ++i)
#pragma unroll
            for (int g = 0; g < Lay::kNE / 4; ++g) {
              const int vq = vbase + Lay::row(i, 4 * g, lane);
              if (full || vq < V) {
                const uint4 w = philox4x32_10(make_uint4((uint32_t)vq >> 2, (uint32_t)srow,
                                                         sa.counter, 0u),
                                              sa.key0, sa.key1);
                const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                  const float z = Lay::get(acc, i, j, 4 * g + c);
                  const float key = gumbel_key(z, sa.inv_tau, words[c]);
                  if ((full || vq + c < V) && key > best) {
                    best = key;
                    bidx = vq + c;
                    bz = z;
                  }
                }
              }
            }
        }
        Lay::across([&](int off) {
          const float ob = __shfl_xor(best, off), oz = __shfl_xor(bz, off);
          const int oi = __shfl_xor(bidx, off);
          if (ob > best || (ob == best && oi < bidx)) {
            best = ob;
            bidx = oi;
            bz = oz;
          }
        });
        if (leader) sred[wv * kTileP + col] = make_float4(best, __int_as_float(bidx), bz, 0.f);
      }
    }
  }
  __syncthreads();
  if (tid < kTileP) {
    const int r = own_pos;
    if (r < M) {
      partials[(size_t)vt * M + r] = merge2(red[tid], red[kTileP + tid]);
      if (kDraw && own_row >= 0) {
        const float4 a = sred[tid], b = sred[kTileP + tid];
        const bool take_a = a.x > b.x || (a.x == b.x && __float_as_int(a.y) < __float_as_int(b.y));
        sa.partials[(size_t)vt * M + r] = make_float4(take_a ? a.x : b.x, take_a ? a.y : b.y,
                                                      take_a ? a.z : b.z, 0.f);
      }
    }
  }
}

template <class Lay, int kMode>
__device__ __forceinline__ void epilogue(typename Lay::Arr& acc, unsigned char* smem, int tid,
                                         int lane, int wv, int wp, int vt, int v0, const PosMap& pos, int M,
                                         int V, float4* __restrict__ partials,
                                         const SampleArgs& sa, const TargetArgs& ta,
                                         const ColIn<Lay>& ci) {
  if (v0 + kTileV <= V)
    epilogue_tile<Lay, kMode, true>(acc, smem, tid, lane, wv, wp, vt, v0, pos, M, V, partials, sa,
                                    ta, ci);
  else
    epilogue_tile<Lay, kMode, false>(acc, smem, tid, lane, wv, wp, vt, v0, pos, M, V, partials,
                                     sa, ta, ci);
}

__device__ __forceinline__ void barrier_nofence() {
  // s_barrier alone: the release fence of __syncthreads would also wait for
  // the loads still in flight for later stages.  The empty asm statements
  // keep the compiler from moving LDS accesses across the barrier.
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with vmcnt <= n and lgkmcnt == 0 (expcnt not waited on).
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

template <int kMode, bool kIlv = false>
__device__ __forceinline__ void gemm_stats_bf16_body(
    const unsigned char* __restrict__ hidden, const unsigned char* __restrict__ W, int M, int d,
    int V, int nvt, int npt, float4* __restrict__ partials, const int32_t* __restrict__ rowlist,
    int Mh, const SampleArgs& sa, const TargetArgs& ta) {
  // W ring: slots 0..2; hidden ring: slots 3..4
  __shared__ __attribute__((aligned(1024))) unsigned char smem[5 * kOperandBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1;   // vocabulary half: rows wv*128 .. +128
  const int wp = wave >> 1;  // position quarter: cols wp*64 .. +64

  int vt, pt;
  map_tile(blockIdx.x, nvt, npt, vt, pt);
  const int v0 = vt * kTileV;
  const int p0 = pt * kTileP;
  const PosMap pos{p0, pt, npt, kIlv};

  const int row_bytes = d * 2;
  const int kchunks = row_bytes >> 4;      // 16-byte chunks per row
  const int nk = (kchunks + 7) >> 3;       // 128-byte stages

  // Buffer descriptors rooted at this tile's first rows: rows past the end of
  // W / hidden are outside the record count and read as zero.
  const unsigned recW = (unsigned)(min(kTileV, V - v0) * row_bytes);
  // With a row list, position p of the tile is hidden row rowlist[p0 + p]
  // (outside [0, Mh): no row, reads as zero) and the descriptor spans all Mh
  // rows; interleaved positions (kIlv) span all M rows too.
  const bool whole = rowlist != nullptr || kIlv;
  const unsigned recH = whole ? (unsigned)((rowlist ? Mh : M) * row_bytes)
                              : (unsigned)(min(kTileP, M - p0) * row_bytes);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W + (size_t)v0 * row_bytes), (short)0, (int)recW, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rsH = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(hidden + (whole ? (size_t)0 : (size_t)p0 * row_bytes)), (short)0, (int)recH,
      kBufferWord3);

  // Each load instruction of a wave writes 1 KiB of LDS = 8 rows x 128 B;
  // lane i fills chunk slot i % 8 of row drow + 8q, so it loads the logical
  // chunk stored there.  Rows drow + 8q with odd q differ in bit 3, which
  // flips bit 0 of the swizzle.
  const int slot_in_row = lane & 7;
  const int drow = wave * 32 + (lane >> 3);
  const int dchunk0 = slot_in_row ^ swz(drow);
  const int dchunk1 = dchunk0 ^ 1;
  const unsigned off0 = (unsigned)(drow * row_bytes) + (unsigned)(dchunk0 << 4);
  const unsigned off1 = (unsigned)(drow * row_bytes) + (unsigned)(dchunk1 << 4);
  const unsigned qstride = (unsigned)(8 * row_bytes);
  unsigned qoff[4], hoff[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    qoff[q] = ((q & 1) ? off1 : off0) + (unsigned)q * qstride;
    hoff[q] = qoff[q];
    if (kIlv)
      hoff[q] = (unsigned)(pos(drow + 8 * q) * row_bytes) +
                (unsigned)(((q & 1) ? dchunk1 : dchunk0) << 4);
    if (rowlist) {
      const int p = p0 + drow + 8 * q;
      const int r = p < M ? rowlist[p] : -1;
      hoff[q] = (r >= 0 && r < Mh)
                    ? (unsigned)(r * row_bytes) + (unsigned)(((q & 1) ? dchunk1 : dchunk0) << 4)
                    : kOutOfRange;
    }
  }
  const int kfull = kchunks >> 3;  // stages whose chunks all lie inside d
  auto src_off = [&](const unsigned (&base)[4], int s, int q) -> unsigned {
    if (s < kfull) return base[q] + (unsigned)(s * kSlab);
    // chunks past d read as zero (the offset lies beyond every record count)
    const int c = (q & 1) ? dchunk1 : dchunk0;
    return (s * 8 + c < kchunks) ? base[q] + (unsigned)(s * kSlab) : kOutOfRange;
  };
  auto issue_W1 = [&](int s, int slot, int q) {  // sub-block q of W stage s
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsW, (__attribute__((address_space(3))) void*)(smem + slot * kOperandBytes + (wave * 4 + q) * 1024),
        16, src_off(qoff, s, q), 0, 0, 0);
  };
  auto issue_H1 = [&](int s, int slot, int q) {  // sub-block q of hidden stage s
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsH, (__attribute__((address_space(3))) void*)(smem + (3 + slot) * kOperandBytes + (wave * 4 + q) * 1024),
        16, src_off(hoff, s, q), 0, 0, 0);
  };
  auto issue_W = [&](int s, int slot) {
#pragma unroll
    for (int q = 0; q < 4; ++q) issue_W1(s, slot, q);
  };
  auto issue_H = [&](int s, int slot) {
#pragma unroll
    for (int q = 0; q < 4; ++q) issue_H1(s, slot, q);
  };

  Acc16::Arr acc;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.f;

  // Fragments of one 32-element K step: A fragment i = W rows arow + 16 i,
  // B fragment j = positions brow + 16 j.  Step kk of a stage takes the
  // stage's 16-byte chunks kk, kk + 2, kk + 4, kk + 6: lane group kq =
  // lane / 16 supplies chunk 2 kq + kk of both operands, so each MFMA sums
  // over the step's 32 K values and the two steps cover the stage.  With the
  // swizzle above, this assignment reads LDS without bank conflicts (four
  // consecutive chunks per step do not).  Rows 16 apart share a swizzle.
  const int arow = wv * 128 + (lane & 15);
  const int brow = wp * 64 + (lane & 15);
  const int kq = lane >> 4;
  const int fa = swz(arow), fb = swz(brow);
  auto rd_a = [&](int ws, int kk, int i) {
    const int chunk = 2 * kq + kk;
    return *reinterpret_cast<const bf16x8*>(smem + ws * kOperandBytes + (arow + 16 * i) * kSlab +
                                            ((chunk ^ fa) << 4));
  };
  auto rd_b = [&](int hs, int kk, int j) {
    const int chunk = 2 * kq + kk;
    return *reinterpret_cast<const bf16x8*>(smem + (3 + hs) * kOperandBytes +
                                            (brow + 16 * j) * kSlab + ((chunk ^ fb) << 4));
  };
  // One K step: 32 MFMAs on (a, bc), block row i at a time.  After the four
  // MFMAs of row i, a[i] is refilled with the fragment of step kkn (slots
  // wsn / hsn), and the four bn are read in between.  `dma` spreads four
  // buffer loads over the rows: 1 = W stage s_dma (rows 0..3), 2 = hidden
  // stage s_dma (rows 2..5, after the barrier), into slot slot_dma.
  // kSync >= 0: the stage barrier (with its wait for the next stage's data)
  // comes after the MFMAs of rows 0..kSync, so that queued MFMAs cover it;
  // every read of the step follows the barrier.
  // kLive: the wave's 64 positions include one below M.  A wave whose
  // positions all lie past M (a last position tile with fewer than 256
  // positions) issues no MFMAs and reads no fragments; it still loads its
  // share of every stage and takes every barrier.
  auto step = [&](auto live_tag, auto sync_tag, bf16x8 (&a)[8], const bf16x8 (&bc)[4],
                  bf16x8 (&bn)[4], int wsn, int hsn, int kkn, int dma, int s_dma, int slot_dma) {
    constexpr bool kLive = decltype(live_tag)::value;
    constexpr int kSync = decltype(sync_tag)::value;
    // Reads held back by the barrier (kSync >= 0), in this order: a[0..kSync],
    // then bn[0..3]; row kSync + 1 + r takes item r after its second MFMA
    // and, for r < kExtra, item kRows + r after its fourth.
    constexpr int kRows = 7 - kSync;
    constexpr int kItems = kSync + 5;
    constexpr int kExtra = kItems - kRows > 0 ? kItems - kRows : 0;
    auto held = [&](int item) {
      if (item <= kSync) a[item] = rd_a(wsn, kkn, item);
      else bn[item - kSync - 1] = rd_b(hsn, kkn, item - kSync - 1);
    };
    auto row = [&](int i) {
      const int r = i - kSync - 1;
      if (kLive) {
        acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bc[0], acc[i][0], 0, 0, 0);
        acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bc[1], acc[i][1], 0, 0, 0);
        if (kSync < 0) {
          if (i < 4) bn[i] = rd_b(hsn, kkn, i);
        } else if (r >= 0 && r < kItems) {
          held(r);
        }
        acc[i][2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bc[2], acc[i][2], 0, 0, 0);
        acc[i][3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bc[3], acc[i][3], 0, 0, 0);
        if (kSync < 0 || r >= 0) a[i] = rd_a(wsn, kkn, i);
        if (kSync >= 0 && r >= 0 && r < kExtra) held(kRows + r);
      }
      if (dma == 1 && i < 4) issue_W1(s_dma, slot_dma, i);
      if (dma == 2 && i >= 2 && i < 6) issue_H1(s_dma, slot_dma, i - 2);
    };
    auto order = [&](int i) {
      const int r = i - kSync - 1;
      const bool r1 = kSync < 0 ? i < 4 : (r >= 0 && r < kItems);
      const int n2 = (kSync < 0 || r >= 0 ? 1 : 0) + (kSync >= 0 && r >= 0 && r < kExtra ? 1 : 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
      if (r1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      if (n2 >= 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (n2 >= 2) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if ((dma == 1 && i < 4) || (dma == 2 && i >= 2 && i < 6))
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // buffer load
    };
    if (kSync >= 0) {
#pragma unroll
      for (int i = 0; i <= kSync; ++i) row(i);
#pragma unroll
      for (int i = 0; i <= kSync; ++i)
        if (kLive) order(i);
      __builtin_amdgcn_sched_barrier(0);
      // the next stage's hidden and W resident; all reads of this stage returned
      wait_vm_lgkm0<4>();
      barrier_nofence();
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kSync + 1; i < 8; ++i) row(i);
#pragma unroll
    for (int i = kSync + 1; i < 8; ++i)
      if (kLive) order(i);
  };
  using NoSync = std::integral_constant<int, -1>;
  using SyncAfterRow1 = std::integral_constant<int, 1>;

  ColIn<Acc16> ci;
  auto mainloop = [&](auto live_tag) {
  constexpr bool kLive = decltype(live_tag)::value;
  bf16x8 a[8], b0[4], b1[4];
  // Load order: H0 W0 W1 H1, then per stage k: W(k+2) during the stage's
  // first K step, H(k+2) during its second, after the stage's barrier (which
  // follows the second step's first eight MFMAs).
  // At the barrier of stage k only W(k+2), the 4 newest loads, may be in
  // flight, and every slot refilled after it belongs to a stage all waves
  // have finished reading.  Stages past the end read as zero into slots
  // nobody reads again.
  issue_H(0, 0);
  issue_W(0, 0);
  issue_W(1, 1);
  issue_H(1, 1);
  wait_vm_lgkm0<8>();  // H0 and W0 resident
  barrier_nofence();
  if (kLive) {
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = rd_a(0, 0, i);
#pragma unroll
    for (int j = 0; j < 4; ++j) b0[j] = rd_b(0, 0, j);
  }
  int ws = 0, hs = 0, ws2 = 2;  // W slots of stages k and k + 2, hidden slot of k
  for (int k = 0; k + 1 < nk; ++k) {
    const int ws1 = ws == 2 ? 0 : ws + 1, hs1 = hs ^ 1;
    step(live_tag, NoSync{}, a, b0, b1, ws, hs, 1, 1, k + 2, ws2);
    __builtin_amdgcn_sched_barrier(0);
    step(live_tag, SyncAfterRow1{}, a, b1, b0, ws1, hs1, 0, 2, k + 2, hs);
    __builtin_amdgcn_sched_barrier(0);
    ws = ws1;
    hs = hs1;
    ws2 = ws2 == 2 ? 0 : ws2 + 1;
  }
  load_col_inputs<Acc16, kMode>(ci, tid, lane, wp, pos, M, sa, ta);
  step(live_tag, NoSync{}, a, b0, b1, ws, hs, 1, 0, 0, 0);
  if (kLive) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b1[j], acc[i][j], 0, 0, 0);
  }
  };
  if (pos(wp * 64) < M)
    mainloop(std::true_type{});
  else
    mainloop(std::false_type{});
  __builtin_amdgcn_s_waitcnt(0);
  barrier_nofence();

  epilogue<Acc16, kMode>(acc, smem, tid, lane, wv, wp, vt, v0, pos, M, V, partials, sa, ta, ci);
}

// fp32 inputs: register-staged double buffer, two v_mfma_f32_32x32x2f32 per
// 16-byte chunk.
template <int kMode>
__device__ __forceinline__ void gemm_stats_f32_body(
    const unsigned char* __restrict__ hidden, const unsigned char* __restrict__ W, int M, int d,
    int V, int nvt, int npt, float4* __restrict__ partials, const int32_t* __restrict__ rowlist,
    int Mh, const SampleArgs& sa, const TargetArgs& ta) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[4 * kOperandBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wv = wave & 1;
  const int wp = wave >> 1;

  int vt, pt;
  map_tile(blockIdx.x, nvt, npt, vt, pt);
  const int v0 = vt * kTileV;
  const int p0 = pt * kTileP;

  const size_t row_bytes = (size_t)d * 4;
  const int kchunks = (int)(row_bytes >> 4);
  const int nk = (kchunks + 7) >> 3;

  // Global -> LDS copy assignment: thread owns chunk c of rows r0 + 64*i.
  const int c = tid & 7;
  const int r0 = tid >> 3;
  const unsigned char* ga[4];
  const unsigned char* gb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // Rows past the end re-read the last row; their results are discarded.
    const int vr = min(v0 + r0 + 64 * i, V - 1);
    int pr = min(p0 + r0 + 64 * i, M - 1);
    // positions without a valid row read row 0 (their results are dropped
    // or unspecified); rows stay inside hidden
    if (rowlist) pr = min(max(rowlist[pr], 0), Mh - 1);
    ga[i] = W + (size_t)vr * row_bytes + (c << 4);
    gb[i] = hidden + (size_t)pr * row_bytes + (c << 4);
  }
  uint4 ra[4], rb[4];
  auto gload = [&](int kt) {
    const bool ok = (kt * 8 + c) < kchunks;  // chunks past d are zero on both sides
    const size_t off = (size_t)kt * kSlab;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = ok ? *reinterpret_cast<const uint4*>(ga[i] + off) : make_uint4(0, 0, 0, 0);
      rb[i] = ok ? *reinterpret_cast<const uint4*>(gb[i] + off) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
    unsigned char* sa = smem + (buf * 2 + 0) * kOperandBytes;
    unsigned char* sb = smem + (buf * 2 + 1) * kOperandBytes;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(sa + lds_off(r0 + 64 * i, c)) = ra[i];
      *reinterpret_cast<uint4*>(sb + lds_off(r0 + 64 * i, c)) = rb[i];
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int arow = wv * 128 + (lane & 31);
  const int brow = wp * 64 + (lane & 31);
  const int khalf = lane >> 5;

  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const unsigned char* sa = smem + (buf * 2 + 0) * kOperandBytes;
    const unsigned char* sb = smem + (buf * 2 + 1) * kOperandBytes;
#pragma unroll 2
    for (int q = 0; q < 8; ++q) {  // 4 fp32 of K per chunk, two MFMAs of K=2
      float4 a[4], b[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const float4*>(sa + lds_off(arow + i * 32, q));
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = *reinterpret_cast<const float4*>(sb + lds_off(brow + j * 32, q));
      // lanes 0-31 supply K index 0 of each pair, lanes 32-63 index 1
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const float a0 = khalf ? a[i].y : a[i].x, b0 = khalf ? b[j].y : b[j].x;
          const float a1 = khalf ? a[i].w : a[i].z, b1 = khalf ? b[j].w : b[j].z;
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[i][j], 0, 0, 0);
        }
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  ColIn<Acc32> ci;
  const PosMap pos{p0, pt, npt, false};
  load_col_inputs<Acc32, kMode>(ci, tid, lane, wp, pos, M, sa, ta);
  epilogue<Acc32, kMode>(acc, smem, tid, lane, wv, wp, vt, v0, pos, M, V, partials, sa, ta, ci);
}

// Entry points: positions = hidden rows 0..M-1, or gathered through a row
// list; greedy candidates only, drawn candidates as well, or the logits of
// given tokens.  Separate symbols keep the row-list, drawing and target code
// out of the dense greedy kernel and the variants apart in kernel traces.
#define FORK_GEMM_ARGS                                                                         \
  const unsigned char *__restrict__ hidden, const unsigned char *__restrict__ W, int M, int d, \
      int V, int nvt, int npt, float4 *__restrict__ partials
#define FORK_GEMM_ENTRIES(T)                                                                   \
  __global__ __launch_bounds__(kThreads) void gemm_stats_##T##_kernel(FORK_GEMM_ARGS) {       \
    gemm_stats_##T##_body<kGreedy>(hidden, W, M, d, V, nvt, npt, partials, nullptr, M,         \
                                   SampleArgs{}, TargetArgs{});                                \
  }                                                                                            \
  __global__ __launch_bounds__(kThreads) void gemm_stats_##T##_rows_kernel(                   \
      FORK_GEMM_ARGS, const int32_t* __restrict__ rowlist, int Mh) {                           \
    gemm_stats_##T##_body<kGreedy>(hidden, W, M, d, V, nvt, npt, partials, rowlist, Mh,        \
                                   SampleArgs{}, TargetArgs{});                                \
  }                                                                                            \
  __global__ __launch_bounds__(kThreads) void gemm_stats_##T##_draw_kernel(FORK_GEMM_ARGS,    \
                                                                          SampleArgs sa) {     \
    gemm_stats_##T##_body<kDrawn>(hidden, W, M, d, V, nvt, npt, partials, nullptr, M, sa,      \
                                  TargetArgs{});                                               \
  }                                                                                            \
  __global__ __launch_bounds__(kThreads) void gemm_stats_##T##_rows_draw_kernel(              \
      FORK_GEMM_ARGS, const int32_t* __restrict__ rowlist, int Mh, SampleArgs sa) {            \
    gemm_stats_##T##_body<kDrawn>(hidden, W, M, d, V, nvt, npt, partials, rowlist, Mh, sa,     \
                                  TargetArgs{});                                               \
  }                                                                                            \
  __global__ __launch_bounds__(kThreads) void gemm_stats_##T##_target_kernel(FORK_GEMM_ARGS,  \
                                                                            TargetArgs ta) {   \
    gemm_stats_##T##_body<kTarget>(hidden, W, M, d, V, nvt, npt, partials, nullptr, M,         \
                                   SampleArgs{}, ta);                                          \
  }                                                                                            \
  __global__ __launch_bounds__(kThreads) void gemm_stats_##T##_rows_target_kernel(            \
      FORK_GEMM_ARGS, const int32_t* __restrict__ rowlist, int Mh, TargetArgs ta) {            \
    gemm_stats_##T##_body<kTarget>(hidden, W, M, d, V, nvt, npt, partials, rowlist, Mh,        \
                                   SampleArgs{}, ta);                                          \
  }
FORK_GEMM_ENTRIES(bf16)
FORK_GEMM_ENTRIES(f32)
// Drawing over all rows with interleaved positions (M = 256 * npt).
__global__ __launch_bounds__(kThreads) void gemm_stats_bf16_draw_ilv_kernel(FORK_GEMM_ARGS,
                                                                           SampleArgs sa) {
  gemm_stats_bf16_body<kDrawn, true>(hidden, W, M, d, V, nvt, npt, partials, nullptr, M, sa,
                                     TargetArgs{});
}
#undef FORK_GEMM_ARGS
#undef FORK_GEMM_ENTRIES

}  // namespace

hipError_t launch_gemm_stats(const void* hidden, const void* W, bool bf16, int M, int d, int V,
                             float4* partials, const int32_t* rowlist, int Mh,
                             const SampleArgs& sample, const TargetArgs& target,
                             hipStream_t stream) {
  const int nvt = num_vocab_tiles(V);
  const int npt = num_pos_tiles(M);
  const dim3 grid((unsigned)(nvt * npt)), block(kThreads);
  const auto* h = static_cast<const unsigned char*>(hidden);
  const auto* w = static_cast<const unsigned char*>(W);
  const bool draw = sample.row != nullptr;
  const bool tgt = target.token != nullptr;
#define FORK_LAUNCH(K, ...) hipLaunchKernelGGL(K, grid, block, 0, stream, h, w, M, d, V, nvt, npt, \
                                               partials, ##__VA_ARGS__)
  if (bf16 && rowlist && tgt)
    FORK_LAUNCH(gemm_stats_bf16_rows_target_kernel, rowlist, Mh, target);
  else if (bf16 && tgt)
    FORK_LAUNCH(gemm_stats_bf16_target_kernel, target);
  else if (!bf16 && rowlist && tgt)
    FORK_LAUNCH(gemm_stats_f32_rows_target_kernel, rowlist, Mh, target);
  else if (!bf16 && tgt)
    FORK_LAUNCH(gemm_stats_f32_target_kernel, target);
  else if (bf16 && rowlist && draw)
    FORK_LAUNCH(gemm_stats_bf16_rows_draw_kernel, rowlist, Mh, sample);
  else if (bf16 && draw && npt > 1 && M == npt * kTileP && (long long)M * d * 2 < (1LL << 31))
    FORK_LAUNCH(gemm_stats_bf16_draw_ilv_kernel, sample);
  else if (bf16 && rowlist)
    FORK_LAUNCH(gemm_stats_bf16_rows_kernel, rowlist, Mh);
  else if (bf16 && draw)
    FORK_LAUNCH(gemm_stats_bf16_draw_kernel, sample);
  else if (bf16)
    FORK_LAUNCH(gemm_stats_bf16_kernel);
  else if (rowlist && draw)
    FORK_LAUNCH(gemm_stats_f32_rows_draw_kernel, rowlist, Mh, sample);
  else if (rowlist)
    FORK_LAUNCH(gemm_stats_f32_rows_kernel, rowlist, Mh);
  else if (draw)
    FORK_LAUNCH(gemm_stats_f32_draw_kernel, sample);
  else
    FORK_LAUNCH(gemm_stats_f32_kernel);
#undef FORK_LAUNCH
  return hipGetLastError();
}

}  // namespace fork
