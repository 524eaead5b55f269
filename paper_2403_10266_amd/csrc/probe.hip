// Measurement aid: the bf16 MFMA rate the chip sustains with every CU busy.
//
// The published dense bf16 figure assumes the peak engine clock.  Under a
// long all-CU MFMA load the clock settles lower, so a kernel's fraction of
// the published figure mixes two things: how busy it keeps the matrix cores
// and how fast they are clocked.  This kernel measures the second: each wave
// keeps 8 independent 32x32x16 accumulator chains (the MFMA pipe never waits
// on a result), two waves per SIMD, two work-groups per CU, operands from
// random bits that change every iteration (the matrix cores' power depends
// on the data).  Nothing else runs: no memory traffic inside the loop, no
// LDS, a few VALU ops per 8 MFMAs.
#include "dsp_internal.h"

namespace dsp {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr int kProbeBlocks = 256 * 2 * 4;  // four rounds of two work-groups per CU
constexpr int kProbeRegs = 6;              // operand registers (16 bytes) per lane

__global__ __launch_bounds__(kProbeThreads, 2) void mfma_probe_kernel(float* sink, int iters) {
  const int lane = threadIdx.x & 63;
  const int64_t base = ((int64_t)blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6)) * kProbeRegs * 64;
  // operand bits: a hash of the position (every exponent kept below 2^1)
  u32x4 a[kProbeRegs];
#pragma unroll
  for (int i = 0; i < kProbeRegs; ++i) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      uint32_t x = (uint32_t)((base + i * 64 + lane) * 4 + c) * 2654435761u;
      x ^= x >> 13;
      x *= 0x5bd1e995u;
      x ^= x >> 15;
      a[i][c] = x & 0xBFFFBFFFu;
    }
  }
  floatx16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;
  uint32_t salt = 0x9e3779b9u * (uint32_t)(lane + 1);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kProbeRegs; ++i) {
      a[i].x ^= salt;
      a[i].y ^= salt >> 3;
      a[i].z ^= salt << 5;
      a[i].w ^= salt >> 7;
      a[i] &= 0xBFFFBFFFu;
    }
    salt = salt * 1664525u + 1013904223u;
#pragma unroll
    for (int w = 0; w < 2; ++w)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        acc[w * 4 + b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[4 + w]),
                                                                 __builtin_bit_cast(bf16x8, a[b]), acc[w * 4 + b],
                                                                 0, 0, 0);
  }
  // keep the results live: one float per thread
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  sink[(int64_t)blockIdx.x * kProbeThreads + threadIdx.x] = s;
}

}  // namespace
}  // namespace dsp

extern "C" {

size_t dsp_probe_mfma_workspace_bytes(void) { return (size_t)dsp::kProbeBlocks * dsp::kProbeThreads * 4; }

double dsp_probe_mfma_flops(int iters) {
  if (iters < 1) return 0.0;
  return (double)dsp::kProbeBlocks * (dsp::kProbeThreads / 64) * iters * 8 * (2.0 * 32 * 32 * 16);
}

int dsp_probe_mfma(void* workspace, size_t ws_bytes, int iters, void* stream) {
  if (iters < 1) return DSP_ERR_ARG;
  if (!workspace) return DSP_ERR_NULL;
  if (ws_bytes < dsp_probe_mfma_workspace_bytes()) return DSP_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return DSP_ERR_ALIGN;
  hipLaunchKernelGGL(dsp::mfma_probe_kernel, dim3(dsp::kProbeBlocks), dim3(dsp::kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<float*>(workspace), iters);
  return dsp::last_launch_status();
}

}  // extern "C"
