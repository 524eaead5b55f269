// LayerNorm over the hidden size (Eq. 4 and Eq. 6 normalise every sublayer):
// y = (x - mean) / sqrt(var + eps), biased variance, no affine part.
// One wave per row; the row is held in registers (up to 64*VPL elements),
// statistics are computed in fp32 in two passes over the registers (mean,
// then centred sum of squares), and reductions use cross-lane adds.
// HBM-bound: one read of x and one write of y per row.
#include <math.h>

#include <algorithm>

#include "dsp_internal.h"

namespace dsp {
namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float load_elem(const void* p, int64_t i, int bf) {
  if (bf) {
    const uint16_t u = static_cast<const uint16_t*>(p)[i];
    return __uint_as_float(((uint32_t)u) << 16);
  }
  return static_cast<const float*>(p)[i];
}

__device__ __forceinline__ void store_elem(void* p, int64_t i, float v, int bf) {
  if (bf) {
    static_cast<__bf16*>(p)[i] = (__bf16)v;
  } else {
    static_cast<float*>(p)[i] = v;
  }
}

constexpr int kRowsPerBlock = 4;  // one wave per row

template <int VPL>
__global__ __launch_bounds__(64 * kRowsPerBlock) void layernorm_kernel(
    const void* __restrict__ x, int x_bf, void* __restrict__ y, int y_bf, int64_t rows, int C,
    float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t base = row * C;
  float v[VPL];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int c = lane + 64 * i;
    v[i] = c < C ? load_elem(x, base + c, x_bf) : 0.0f;
    s += v[i];
  }
  const float mean = wave_sum(s) / (float)C;
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int c = lane + 64 * i;
    const float d = c < C ? v[i] - mean : 0.0f;
    ss = fmaf(d, d, ss);
  }
  const float var = wave_sum(ss) / (float)C;
  const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int c = lane + 64 * i;
    if (c < C) store_elem(y, base + c, (v[i] - mean) * rstd, y_bf);
  }
}

// Rows longer than the register budget: three passes over global memory.
__global__ __launch_bounds__(64 * kRowsPerBlock) void layernorm_long_kernel(
    const void* __restrict__ x, int x_bf, void* __restrict__ y, int y_bf, int64_t rows, int C,
    float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t base = row * C;
  float s = 0.0f;
  for (int c = lane; c < C; c += 64) s += load_elem(x, base + c, x_bf);
  const float mean = wave_sum(s) / (float)C;
  float ss = 0.0f;
  for (int c = lane; c < C; c += 64) {
    const float d = load_elem(x, base + c, x_bf) - mean;
    ss = fmaf(d, d, ss);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)C + eps);
  for (int c = lane; c < C; c += 64) store_elem(y, base + c, (load_elem(x, base + c, x_bf) - mean) * rstd, y_bf);
}

// Backward: with y = (x - mean) / sigma, dx = dres + (dy - mean(dy) - y mean(dy y)) / sigma.
// One wave per row: x and dy held in registers, the statistics of x recomputed
// in fp32 as in the forward, then two row means of the upstream gradient.
template <int VPL>
__global__ __launch_bounds__(64 * kRowsPerBlock) void layernorm_bwd_kernel(
    const void* __restrict__ x, int x_bf, const void* __restrict__ dy, int dy_bf, const float* dres,
    float* dx, void* dx2, int dx2_bf, RowSwap rs, int64_t rows, int C, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t base = row * C;
  float v[VPL], g[VPL];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int c = lane + 64 * i;
    v[i] = c < C ? load_elem(x, base + c, x_bf) : 0.0f;
    g[i] = c < C ? load_elem(dy, base + c, dy_bf) : 0.0f;
    s += v[i];
  }
  const float mean = wave_sum(s) / (float)C;
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int c = lane + 64 * i;
    const float d = c < C ? v[i] - mean : 0.0f;
    ss = fmaf(d, d, ss);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)C + eps);
  float sg = 0.0f, sgy = 0.0f;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    v[i] = (v[i] - mean) * rstd;  // y (0 past C: g is 0 there too)
    sg += g[i];
    sgy = fmaf(g[i], v[i], sgy);
  }
  const float mg = wave_sum(sg) / (float)C, mgy = wave_sum(sgy) / (float)C;
  const int64_t obase = rs.outer ? rs.map((int)row) * C : base;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int c = lane + 64 * i;
    if (c < C) {
      float d = (g[i] - mg - v[i] * mgy) * rstd;
      if (dres) d += dres[base + c];
      dx[obase + c] = d;
      if (dx2) store_elem(dx2, obase + c, d, dx2_bf);
    }
  }
}

// Rows longer than the register budget: passes over global memory.
__global__ __launch_bounds__(64 * kRowsPerBlock) void layernorm_bwd_long_kernel(
    const void* __restrict__ x, int x_bf, const void* __restrict__ dy, int dy_bf, const float* dres,
    float* dx, void* dx2, int dx2_bf, RowSwap rs, int64_t rows, int C, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t base = row * C;
  float s = 0.0f;
  for (int c = lane; c < C; c += 64) s += load_elem(x, base + c, x_bf);
  const float mean = wave_sum(s) / (float)C;
  float ss = 0.0f;
  for (int c = lane; c < C; c += 64) {
    const float d = load_elem(x, base + c, x_bf) - mean;
    ss = fmaf(d, d, ss);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)C + eps);
  float sg = 0.0f, sgy = 0.0f;
  for (int c = lane; c < C; c += 64) {
    const float gv = load_elem(dy, base + c, dy_bf);
    sg += gv;
    sgy = fmaf(gv, (load_elem(x, base + c, x_bf) - mean) * rstd, sgy);
  }
  const float mg = wave_sum(sg) / (float)C, mgy = wave_sum(sgy) / (float)C;
  const int64_t obase = rs.outer ? rs.map((int)row) * C : base;
  for (int c = lane; c < C; c += 64) {
    const float yv = (load_elem(x, base + c, x_bf) - mean) * rstd;
    float d = (load_elem(dy, base + c, dy_bf) - mg - yv * mgy) * rstd;
    if (dres) d += dres[base + c];
    dx[obase + c] = d;
    if (dx2) store_elem(dx2, obase + c, d, dx2_bf);
  }
}

// fp32 -> bf16, eight elements per thread and iteration: two 16-byte loads,
// one 16-byte store (n a multiple of 8, 16-byte aligned buffers)
__global__ __launch_bounds__(256) void cast_f32_bf16_x8_kernel(const float4* __restrict__ x,
                                                               uint4* __restrict__ y, int64_t n8) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += stride) {
    const float4 a = x[2 * i], b = x[2 * i + 1];
    typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
    bf16x8_t v = {(__bf16)a.x, (__bf16)a.y, (__bf16)a.z, (__bf16)a.w,
                  (__bf16)b.x, (__bf16)b.y, (__bf16)b.z, (__bf16)b.w};
    y[i] = __builtin_bit_cast(uint4, v);
  }
}

__global__ __launch_bounds__(256) void cast_kernel(const void* __restrict__ x, int x_bf,
                                                   void* __restrict__ y, int y_bf, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    store_elem(y, i, load_elem(x, i, x_bf), y_bf);
}

}  // namespace

int launch_layernorm_bwd(const void* x, int x_bf16, const void* dy, int dy_bf16, const float* dres, float* dx,
                         int64_t rows, int C, float eps, hipStream_t s, RowSwap rs, void* dx2, int dx2_bf16) {
  if (rows == 0) return DSP_OK;
  if (rs.outer && (rs.inner == 0 || rows > INT32_MAX || rows % ((int64_t)rs.outer * rs.inner) ||
                   (const void*)dres == (const void*)dx || (dx2 && (const void*)dres == dx2)))
    return DSP_ERR_ARG;
  const int64_t blocks = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
  if (blocks >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  const dim3 grid((uint32_t)blocks), block(64 * kRowsPerBlock);
  const int vpl = (C + 63) / 64;
#define DSP_LN_BWD_ARGS x, x_bf16, dy, dy_bf16, dres, dx, dx2, dx2_bf16, rs, rows, C, eps
  if (vpl <= 4) {
    hipLaunchKernelGGL(layernorm_bwd_kernel<4>, grid, block, 0, s, DSP_LN_BWD_ARGS);
  } else if (vpl <= 8) {
    hipLaunchKernelGGL(layernorm_bwd_kernel<8>, grid, block, 0, s, DSP_LN_BWD_ARGS);
  } else if (vpl <= 18) {
    hipLaunchKernelGGL(layernorm_bwd_kernel<18>, grid, block, 0, s, DSP_LN_BWD_ARGS);
  } else {
    hipLaunchKernelGGL(layernorm_bwd_long_kernel, grid, block, 0, s, DSP_LN_BWD_ARGS);
  }
#undef DSP_LN_BWD_ARGS
  return last_launch_status();
}

// Element-wise format conversion (fp32 <-> bf16, round to nearest even).
int launch_cast(const void* x, int x_bf16, void* y, int y_bf16, int64_t n, hipStream_t s) {
  if (n == 0) return DSP_OK;
  if (!x_bf16 && y_bf16 && n % 8 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
      reinterpret_cast<uintptr_t>(y) % 16 == 0) {
    const int64_t n8 = n / 8;
    const int64_t blocks = std::min<int64_t>((n8 + 255) / 256, 16384);
    hipLaunchKernelGGL(cast_f32_bf16_x8_kernel, dim3((uint32_t)blocks), dim3(256), 0, s,
                       static_cast<const float4*>(x), static_cast<uint4*>(y), n8);
    return last_launch_status();
  }
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL(cast_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, x, x_bf16, y, y_bf16, n);
  return last_launch_status();
}

int launch_layernorm(const void* x, int x_bf16, void* y, int y_bf16, int64_t rows, int C, float eps,
                     hipStream_t s) {
  if (rows == 0) return DSP_OK;
  const int64_t blocks = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
  if (blocks >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  const dim3 grid((uint32_t)blocks), block(64 * kRowsPerBlock);
  const int vpl = (C + 63) / 64;
  if (vpl <= 4) {
    hipLaunchKernelGGL(layernorm_kernel<4>, grid, block, 0, s, x, x_bf16, y, y_bf16, rows, C, eps);
  } else if (vpl <= 8) {
    hipLaunchKernelGGL(layernorm_kernel<8>, grid, block, 0, s, x, x_bf16, y, y_bf16, rows, C, eps);
  } else if (vpl <= 18) {
    hipLaunchKernelGGL(layernorm_kernel<18>, grid, block, 0, s, x, x_bf16, y, y_bf16, rows, C, eps);
  } else if (vpl <= 32) {
    hipLaunchKernelGGL(layernorm_kernel<32>, grid, block, 0, s, x, x_bf16, y, y_bf16, rows, C, eps);
  } else {
    hipLaunchKernelGGL(layernorm_long_kernel, grid, block, 0, s, x, x_bf16, y, y_bf16, rows, C, eps);
  }
  return last_launch_status();
}

}  // namespace dsp
