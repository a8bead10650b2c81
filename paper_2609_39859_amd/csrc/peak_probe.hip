// Measurement probes for the benchmark (not part of the Fork-dLLM library):
// the achievable dense bf16 MFMA rate and HBM streaming rate of the GPU the
// benchmark runs on, against which its roofline fractions are also quoted.
// Built into its own small library (libforkprobe.so), loaded by bench.py.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Both MFMA probes issue the LM-head kernel's instruction,
// v_mfma_f32_16x16x32_bf16, on register-resident operands (no memory traffic
// inside the loop) into the same 8 x 4 blocks of 16 x 16 accumulators per
// wave; 512-thread workgroups put two waves on each SIMD, as the LM-head
// kernel does.  One round = 16 MFMAs = 262144 flops per wave; `iters` is a
// multiple of 4.

// Constant operands.
__global__ __launch_bounds__(512) void mfma_peak_kernel(int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)(lane + i));
    b[i] = (__bf16)(0.002f * (float)(lane - i));
  }
  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.f;
  for (int it = 0; it < iters; it += 2) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[i][j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) s += acc[i][j][e];
  out[blockIdx.x * 512 + threadIdx.x] = s;
}

// The same MFMA stream on operands with the statistics of the LM head's real
// data: each wave holds two sets of fragments loaded from `a_src` / `b_src`
// (random bf16 values drawn like W_head and the hidden rows), eight A and
// four B fragments per set as one 32-element K step of the LM-head kernel
// uses, and alternates between the sets every step, so consecutive MFMAs see
// changing operand bits as in the LM head.
__global__ __launch_bounds__(512) void mfma_data_kernel(int iters, const bf16x8* __restrict__ a_src,
                                                        const bf16x8* __restrict__ b_src, int nfrag,
                                                        float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * 8 + (threadIdx.x >> 6)) % nfrag;
  bf16x8 a0[8], b0[4], a1[8], b1[4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a0[i] = a_src[((size_t)wave * 16 + i) * 64 + lane];
    a1[i] = a_src[((size_t)wave * 16 + 8 + i) * 64 + lane];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    b0[j] = b_src[((size_t)wave * 8 + j) * 64 + lane];
    b1[j] = b_src[((size_t)wave * 8 + 4 + j) * 64 + lane];
  }
  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.f;
  for (int it = 0; it < iters; it += 4) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[i], b0[j], acc[i][j], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[i], b1[j], acc[i][j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) s += acc[i][j][e];
  out[blockIdx.x * 512 + threadIdx.x] = s;
}

// Streaming copy: one 16-byte element per thread over a grid that covers the
// buffer, nontemporal loads and stores (of the copy forms tried — several
// elements per thread, grid-stride loops, cached accesses — the fastest).
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256) void stream_copy_kernel(const u32x4* __restrict__ src,
                                                          u32x4* __restrict__ dst, size_t n) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace

extern "C" {

// Launches the MFMA probe: `blocks` workgroups of 512 threads, `iters`
// rounds each (a multiple of 4); out must hold blocks * 512 floats.  Returns
// a hipError_t.  Dense bf16 flops of one launch = blocks * 8 waves * iters *
// 16 * 16384.
int fork_probe_mfma(int blocks, int iters, float* out, void* stream) {
  hipLaunchKernelGGL(mfma_peak_kernel, dim3((unsigned)blocks), dim3(512), 0,
                     static_cast<hipStream_t>(stream), iters, out);
  return (int)hipGetLastError();
}

// Launches the MFMA probe on data operands: a_src holds nfrag x 16 x 64 and
// b_src nfrag x 8 x 64 fragments of 8 bf16 (wave w of the grid uses set
// w % nfrag); iters a multiple of 4.  Same flop count as fork_probe_mfma.
// Returns a hipError_t.
int fork_probe_mfma_data(int blocks, int iters, const void* a_src, const void* b_src, int nfrag,
                         float* out, void* stream) {
  hipLaunchKernelGGL(mfma_data_kernel, dim3((unsigned)blocks), dim3(512), 0,
                     static_cast<hipStream_t>(stream), iters,
                     static_cast<const bf16x8*>(a_src), static_cast<const bf16x8*>(b_src), nfrag,
                     out);
  return (int)hipGetLastError();
}

// Launches the copy probe on n 16-byte elements (src and dst 16-byte
// aligned, n * 16 bytes each, n < 2^39): ceil(n / 256) workgroups.  Returns
// a hipError_t.
int fork_probe_copy(const void* src, void* dst, size_t n, void* stream) {
  const size_t blocks = (n + 255) / 256;
  if (blocks == 0) return (int)hipSuccess;
  if (blocks > 0x7fffffffu) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(stream_copy_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(src),
                     static_cast<u32x4*>(dst), n);
  return (int)hipGetLastError();
}

}  // extern "C"
