// Linear maps of the block (Eq. 1 output projection W^O, the Q/K/V
// projections, Eq. 5 FFN W_1 and W_2): out = epilogue(a * W + bias) with a
// [M, K] row-major and W stored [N][K] (reduction index contiguous).
//
// bf16 path (gfx950 MFMA):
//  * 256 x 128 output tile per work-group, 4 waves of 128 x 64, K staged 64 at
//    a time through LDS (row pitch 144 bytes, an odd multiple of 16: the
//    16-byte fragment reads of 16 consecutive rows hit distinct banks), with
//    the next K slice prefetched into registers during the current slice's
//    MFMAs.
//  * v_mfma_f32_32x32x16_bf16 with the operands swapped (W rows on the MFMA
//    M side, activation rows on the N side), so each lane ends up owning one
//    output row and four consecutive output columns per register group: the
//    epilogue reads bias/residual and writes results as 8- or 16-byte
//    vectors.
//  * Epilogues: none, exact-erf GELU (bf16 out), fp32 output, residual add
//    (fp32 out, may be in place).
// fp32 path: LDS-tiled FMA kernel, 64 x 64 tile, 4 x 4 outputs per thread.
#include <math.h>

#include "dsp_internal.h"

namespace dsp {
namespace {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

constexpr int BM = 256, BN = 128, BK = 64;
constexpr int PITCH = BK + 8;                 // 144-byte rows
constexpr int NTHR = 256;
constexpr int A_CHUNKS = BM * BK / 8;         // 16-byte chunks per A slice
constexpr int W_CHUNKS = BN * BK / 8;
constexpr int NLOAD = (A_CHUNKS + W_CHUNKS) / NTHR;
static_assert((A_CHUNKS + W_CHUNKS) % NTHR == 0, "loader shape");

__device__ __forceinline__ float bf2f(bf16 v) { return (float)v; }

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

template <int EPI>
__global__ __launch_bounds__(NTHR, 2) void gemm_bf16_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ W, const bf16* __restrict__ bias,
    const float* resid, void* out, int M, int N, int K, int n_ntiles, int n_tiles) {
  __shared__ __attribute__((aligned(16))) bf16 As[BM * PITCH];
  __shared__ __attribute__((aligned(16))) bf16 Ws[BN * PITCH];

  // XCD-aware order: logical tiles are m-major (n fastest); each XCD takes a
  // contiguous range so the n-tiles sharing an A slice share that XCD's L2.
  uint32_t bid = blockIdx.x;
  if ((n_tiles & 7) == 0) bid = (bid & 7u) * ((uint32_t)n_tiles >> 3) + (bid >> 3);
  const int mt = bid / n_ntiles;
  const int nt = bid - mt * n_ntiles;
  const int m0 = mt * BM, n0 = nt * BN;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;

  uint4 pre[NLOAD];
  auto load_regs = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int c = threadIdx.x + i * NTHR;
      pre[i] = make_uint4(0, 0, 0, 0);
      if (c < A_CHUNKS) {
        const int row = c / (BK / 8), col = c % (BK / 8);
        const int gm = m0 + row, gk = k0 + col * 8;
        if (gm < M && gk < K) pre[i] = *reinterpret_cast<const uint4*>(A + (int64_t)gm * K + gk);
      } else {
        const int cc = c - A_CHUNKS;
        const int row = cc / (BK / 8), col = cc % (BK / 8);
        const int gn = n0 + row, gk = k0 + col * 8;
        if (gn < N && gk < K) pre[i] = *reinterpret_cast<const uint4*>(W + (int64_t)gn * K + gk);
      }
    }
  };
  auto store_lds = [&]() {
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int c = threadIdx.x + i * NTHR;
      if (c < A_CHUNKS) {
        const int row = c / (BK / 8), col = c % (BK / 8);
        *reinterpret_cast<uint4*>(As + row * PITCH + col * 8) = pre[i];
      } else {
        const int cc = c - A_CHUNKS;
        const int row = cc / (BK / 8), col = cc % (BK / 8);
        *reinterpret_cast<uint4*>(Ws + row * PITCH + col * 8) = pre[i];
      }
    }
  };

  floatx16 acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  const int nk = (K + BK - 1) / BK;
  load_regs(0);
  store_lds();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) load_regs((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[4], wf[2];
#pragma unroll
      for (int b = 0; b < 4; ++b)
        af[b] = *reinterpret_cast<const bf16x8*>(As + (wm * 128 + 32 * b + l32) * PITCH + 16 * ks + 8 * g);
#pragma unroll
      for (int a = 0; a < 2; ++a)
        wf[a] = *reinterpret_cast<const bf16x8*>(Ws + (wn * 64 + 32 * a + l32) * PITCH + 16 * ks + 8 * g);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[a], af[b], acc[a][b], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      __syncthreads();
      store_lds();
      __syncthreads();
    }
  }

  // epilogue: lane owns row m = .. + l32 and columns n = .. + 8*r4 + 4g + {0..3}
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int m = m0 + wm * 128 + 32 * b + l32;
    if (m >= M) continue;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int n = n0 + wn * 64 + 32 * a + 8 * r4 + 4 * g;
        if (n >= N) continue;
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = acc[a][b][4 * r4 + i];
        const bool full = (n + 3 < N) && ((N & 3) == 0);
        if (bias) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (n + i < N) v[i] += bf2f(bias[n + i]);
        }
        if (EPI == DSP_EPI_GELU) {
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = gelu_erf(v[i]);
        }
        const int64_t off = (int64_t)m * N + n;
        if (EPI == DSP_EPI_RESID || EPI == DSP_EPI_F32) {
          float* o = static_cast<float*>(out);
          if (EPI == DSP_EPI_RESID) {
            if (full) {
              const float4 rv = *reinterpret_cast<const float4*>(resid + off);
              v[0] += rv.x; v[1] += rv.y; v[2] += rv.z; v[3] += rv.w;
            } else {
              for (int i = 0; i < 4; ++i)
                if (n + i < N) v[i] += resid[off + i];
            }
          }
          if (full) {
            *reinterpret_cast<float4*>(o + off) = make_float4(v[0], v[1], v[2], v[3]);
          } else {
            for (int i = 0; i < 4; ++i)
              if (n + i < N) o[off + i] = v[i];
          }
        } else {
          bf16* o = static_cast<bf16*>(out);
          if (full) {
            bf16x2 lo = {(bf16)v[0], (bf16)v[1]};
            bf16x2 hi = {(bf16)v[2], (bf16)v[3]};
            uint2 w;
            w.x = __builtin_bit_cast(uint32_t, lo);
            w.y = __builtin_bit_cast(uint32_t, hi);
            *reinterpret_cast<uint2*>(o + off) = w;
          } else {
            for (int i = 0; i < 4; ++i)
              if (n + i < N) o[off + i] = (bf16)v[i];
          }
        }
      }
  }
}

// ---------------------------------------------------------------- fp32 path
constexpr int FT = 64, FK = 16;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                        const float* __restrict__ W,
                                                        const float* __restrict__ bias,
                                                        const float* resid, float* out, int M,
                                                        int N, int K) {
  __shared__ float As[FK][FT + 1];
  __shared__ float Bs[FK][FT + 1];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FK) {
    for (int e = threadIdx.x; e < FT * FK; e += 256) {
      const int r = e / FK, kk = e % FK;
      const int gm = m0 + r, gn = n0 + r, gk = k0 + kk;
      As[kk][r] = (gm < M && gk < K) ? A[(int64_t)gm * K + gk] : 0.0f;
      Bs[kk][r] = (gn < N && gk < K) ? W[(int64_t)gn * K + gk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty + 16 * i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx + 16 * j;
      if (n >= N) continue;
      float v = acc[i][j];
      if (bias) v += bias[n];
      if (EPI == DSP_EPI_GELU) v = 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
      const int64_t off = (int64_t)m * N + n;
      if (EPI == DSP_EPI_RESID) v += resid[off];
      out[off] = v;
    }
  }
}

}  // namespace

int launch_linear_bf16(const void* a, const void* w, const void* bias, const float* residual,
                       void* out, int64_t M, int N, int K, int epilogue, hipStream_t s) {
  if (M == 0) return DSP_OK;
  const int64_t n_mt = (M + BM - 1) / BM, n_nt = (N + BN - 1) / BN;
  const int64_t tiles = n_mt * n_nt;
  if (tiles >= (int64_t(1) << 31) || M >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  const dim3 grid((uint32_t)tiles), block(NTHR);
  const bf16* A = static_cast<const bf16*>(a);
  const bf16* Wt = static_cast<const bf16*>(w);
  const bf16* bs = static_cast<const bf16*>(bias);
  switch (epilogue) {
    case DSP_EPI_NONE:
      hipLaunchKernelGGL(gemm_bf16_kernel<DSP_EPI_NONE>, grid, block, 0, s, A, Wt, bs, residual,
                         out, (int)M, N, K, (int)n_nt, (int)tiles);
      break;
    case DSP_EPI_GELU:
      hipLaunchKernelGGL(gemm_bf16_kernel<DSP_EPI_GELU>, grid, block, 0, s, A, Wt, bs, residual,
                         out, (int)M, N, K, (int)n_nt, (int)tiles);
      break;
    case DSP_EPI_RESID:
      hipLaunchKernelGGL(gemm_bf16_kernel<DSP_EPI_RESID>, grid, block, 0, s, A, Wt, bs, residual,
                         out, (int)M, N, K, (int)n_nt, (int)tiles);
      break;
    case DSP_EPI_F32:
      hipLaunchKernelGGL(gemm_bf16_kernel<DSP_EPI_F32>, grid, block, 0, s, A, Wt, bs, residual,
                         out, (int)M, N, K, (int)n_nt, (int)tiles);
      break;
    default:
      return DSP_ERR_ARG;
  }
  return last_launch_status();
}

int launch_linear_f32(const float* a, const float* w, const float* bias, const float* residual,
                      float* out, int64_t M, int N, int K, int epilogue, hipStream_t s) {
  if (M == 0) return DSP_OK;
  const int64_t gy = (M + FT - 1) / FT;
  if (gy >= 65536 * 1024) return DSP_ERR_SHAPE;
  const dim3 grid((uint32_t)((N + FT - 1) / FT), (uint32_t)gy), block(256);
  switch (epilogue) {
    case DSP_EPI_NONE:
      hipLaunchKernelGGL(gemm_f32_kernel<DSP_EPI_NONE>, grid, block, 0, s, a, w, bias, residual, out,
                         (int)M, N, K);
      break;
    case DSP_EPI_GELU:
      hipLaunchKernelGGL(gemm_f32_kernel<DSP_EPI_GELU>, grid, block, 0, s, a, w, bias, residual, out,
                         (int)M, N, K);
      break;
    case DSP_EPI_RESID:
      hipLaunchKernelGGL(gemm_f32_kernel<DSP_EPI_RESID>, grid, block, 0, s, a, w, bias, residual, out,
                         (int)M, N, K);
      break;
    case DSP_EPI_F32:
      hipLaunchKernelGGL(gemm_f32_kernel<DSP_EPI_NONE>, grid, block, 0, s, a, w, bias, residual, out,
                         (int)M, N, K);
      break;
    default:
      return DSP_ERR_ARG;
  }
  return last_launch_status();
}

}  // namespace dsp
