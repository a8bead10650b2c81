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
// Work decomposition (gfx950 / CDNA4):
//   * one workgroup = 256 vocabulary rows x 256 positions, 8 wave64s laid out
//     2 (vocabulary) x 4 (positions); each wave owns 128 x 64 outputs as
//     4 x 2 tiles of v_mfma_f32_32x32x16_bf16 (fp32 accumulate);
//   * the MFMA "A" operand is W (vocabulary on the MFMA M axis) and "B" is
//     hidden, so each lane's accumulators hold 16 vocabulary values of ONE
//     position: the vocabulary reduction is mostly in-lane, plus one
//     exchange with lane^32 and one LDS exchange between the two vocabulary
//     waves;
//   * K is staged through LDS in 128-byte slabs (64 bf16 / 32 fp32) per row,
//     double-buffered, with the 16-byte chunks of row r stored at chunk
//     position (c ^ (r & 7)) so that the fragment reads of 8 consecutive
//     lanes (8 different rows, same chunk) fall in 8 different bank groups;
//   * workgroups are renumbered so that each XCD (private L2) walks a
//     contiguous range of tiles, and inside it groups of kGroupV vocabulary
//     stripes are swept across all position tiles, so a W stripe is fetched
//     from HBM about once and re-read from L2 by the position tiles.
#include "fork_kernels.h"

#include <math.h>

namespace fork {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;
constexpr int kSlabBytes = 128;                       // bytes of K per row per stage
constexpr int kOperandBytes = kTileV * kSlabBytes;    // 32 KiB (kTileV == kTileP)
constexpr int kGroupV = 4;                            // vocab stripes per sweep group
constexpr int kXcds = 8;
constexpr float kLog2e = 1.4426950408889634f;

static_assert(kTileV == kTileP, "LDS layout assumes square tiles");

__device__ __forceinline__ int swz(int row, int chunk) {
  return row * kSlabBytes + ((chunk ^ (row & 7)) << 4);
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

// Vocabulary index held by accumulator element `e` of MFMA tile `i` in this
// lane (32x32 output layout: column = lane % 32, row = 8*(e/4) + 4*(lane/32)
// + e%4), relative to the wave's first vocabulary row.
__device__ __forceinline__ int acc_row(int i, int e, int lane) {
  return i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
}

template <bool kBF16>
__global__ __launch_bounds__(kThreads) void gemm_stats_kernel(
    const unsigned char* __restrict__ hidden, const unsigned char* __restrict__ W,
    int M, int d, int V, int nvt, int npt, float4* __restrict__ partials) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[4 * kOperandBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wv = wave & 1;   // vocabulary half: rows wv*128 .. +128
  const int wp = wave >> 1;  // position quarter: cols wp*64 .. +64

  int vt, pt;
  map_tile(blockIdx.x, nvt, npt, vt, pt);
  const int v0 = vt * kTileV;
  const int p0 = pt * kTileP;

  const size_t row_bytes = (size_t)d * (kBF16 ? 2 : 4);
  const int kchunks = (int)(row_bytes >> 4);       // 16-byte chunks per row
  const int nk = (kchunks + 7) >> 3;               // 128-byte stages

  // Global -> LDS copy assignment: thread owns chunk c of rows r0 + 64*i.
  const int c = tid & 7;
  const int r0 = tid >> 3;
  const unsigned char* ga[4];
  const unsigned char* gb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // Rows past the end re-read the last row; their results are discarded.
    const int vr = min(v0 + r0 + 64 * i, V - 1);
    const int pr = min(p0 + r0 + 64 * i, M - 1);
    ga[i] = W + (size_t)vr * row_bytes + (c << 4);
    gb[i] = hidden + (size_t)pr * row_bytes + (c << 4);
  }
  uint4 ra[4], rb[4];
  auto gload = [&](int kt) {
    const bool ok = (kt * 8 + c) < kchunks;  // chunks past d are zero on both sides
    const size_t off = (size_t)kt * kSlabBytes;
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
      *reinterpret_cast<uint4*>(sa + swz(r0 + 64 * i, c)) = ra[i];
      *reinterpret_cast<uint4*>(sb + swz(r0 + 64 * i, c)) = rb[i];
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int arow = wv * 128 + (lane & 31);  // + i*32
  const int brow = wp * 64 + (lane & 31);   // + j*32
  const int khalf = lane >> 5;

  gload(0);
  sstore(0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const unsigned char* sa = smem + (buf * 2 + 0) * kOperandBytes;
    const unsigned char* sb = smem + (buf * 2 + 1) * kOperandBytes;
    if constexpr (kBF16) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {  // 16 bf16 of K per MFMA
        const int chunk = kk * 2 + khalf;
        bf16x8 a[4], b[2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[i] = *reinterpret_cast<const bf16x8*>(sa + swz(arow + i * 32, chunk));
#pragma unroll
        for (int j = 0; j < 2; ++j)
          b[j] = *reinterpret_cast<const bf16x8*>(sb + swz(brow + j * 32, chunk));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    } else {
#pragma unroll 2
      for (int q = 0; q < 8; ++q) {  // 4 fp32 of K per chunk, two MFMAs of K=2
        float4 a[4], b[2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[i] = *reinterpret_cast<const float4*>(sa + swz(arow + i * 32, q));
#pragma unroll
        for (int j = 0; j < 2; ++j)
          b[j] = *reinterpret_cast<const float4*>(sb + swz(brow + j * 32, q));
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
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: per-position statistics over this workgroup's 256 rows of W
  float4* red = reinterpret_cast<float4*>(smem);  // [2][kTileP], LDS is free now
  const int vbase = v0 + wv * 128;                 // first vocabulary row of the wave
  const bool full = v0 + kTileV <= V;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    // maximum and its lowest index; values are visited in increasing v
    float m = -INFINITY;
    int idx = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int v = vbase + acc_row(i, e, lane);
        const float z = acc[i][j][e];
        if ((full || v < V) && z > m) {
          m = z;
          idx = v;
        }
      }
    {
      const float mo = __shfl_xor(m, 32);
      const int io = __shfl_xor(idx, 32);
      if (mo > m || (mo == m && io < idx)) {
        m = mo;
        idx = io;
      }
    }
    float s = 0.f, t = 0.f;
    if (m > -INFINITY) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int v = vbase + acc_row(i, e, lane);
          if (full || v < V) {
            const float dz = acc[i][j][e] - m;
            const float ex = __builtin_amdgcn_exp2f(dz * kLog2e);
            s += ex;
            t = fmaf(ex, dz, t);
          }
        }
    }
    s += __shfl_xor(s, 32);
    t += __shfl_xor(t, 32);
    if (lane < 32)
      red[wv * kTileP + wp * 64 + j * 32 + lane] =
          make_float4(m, s, t, __int_as_float(idx));
  }
  __syncthreads();
  if (tid < kTileP) {
    const int r = p0 + tid;
    if (r < M) {
      const float4 out = merge2(red[tid], red[kTileP + tid]);
      partials[(size_t)vt * M + r] = out;
    }
  }
}

}  // namespace

hipError_t launch_gemm_stats(const void* hidden, const void* W, bool bf16, int M,
                             int d, int V, float4* partials, hipStream_t stream) {
  const int nvt = num_vocab_tiles(V);
  const int npt = num_pos_tiles(M);
  const dim3 grid((unsigned)(nvt * npt)), block(kThreads);
  if (bf16)
    hipLaunchKernelGGL(gemm_stats_kernel<true>, grid, block, 0, stream,
                       static_cast<const unsigned char*>(hidden),
                       static_cast<const unsigned char*>(W), M, d, V, nvt, npt, partials);
  else
    hipLaunchKernelGGL(gemm_stats_kernel<false>, grid, block, 0, stream,
                       static_cast<const unsigned char*>(hidden),
                       static_cast<const unsigned char*>(W), M, d, V, nvt, npt, partials);
  return hipGetLastError();
}

}  // namespace fork
