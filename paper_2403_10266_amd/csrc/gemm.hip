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
//  * Epilogues: none, erf GELU (bf16 out; erf evaluated by Abramowitz-Stegun
//    7.1.26, abs. error <= 1.5e-7), ReLU (Eq. 5), fp32 output, residual add
//    (fp32 out, may be in place); for training, GELU / ReLU that also keep the
//    pre-activation (or GELU' there), and the activation's backward (the sum
//    times act'(u), or times a kept GELU').
//  * A batched bf16 transpose for the block backward's weights.
// fp32 path: LDS-tiled FMA kernel, 64 x 64 tile, 4 x 4 outputs per thread.
#include <math.h>

#include <type_traits>

#include "dsp_internal.h"

// Large-tile kernel for problems of at least one full round of 256 x 192/256 tiles.
#ifndef DSP_GEMM_BIG
#define DSP_GEMM_BIG 1
#endif

namespace dsp {
namespace {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = 256, BN = 128, BK = 64;
constexpr int PITCH = BK + 8;                 // 144-byte rows
constexpr int NTHR = 256;
constexpr int A_CHUNKS = BM * BK / 8;         // 16-byte chunks per A slice
constexpr int W_CHUNKS = BN * BK / 8;
constexpr int NLOAD = (A_CHUNKS + W_CHUNKS) / NTHR;
static_assert((A_CHUNKS + W_CHUNKS) % NTHR == 0, "loader shape");

__device__ __forceinline__ float bf2f(bf16 v) { return (float)v; }

// Buffer resource over [base, base + bytes) built from wave-uniform values in
// scalar registers; out-of-range loads return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const uint32_t n = __builtin_amdgcn_readfirstlane(bytes);
  void* p = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)n, 0x00020000);
}

// erf(z) by Abramowitz and Stegun, Handbook of Mathematical Functions, 7.1.26:
// 1 - (a1 t + ... + a5 t^5) exp(-z^2) with t = 1 / (1 + p |z|), |error| <=
// 1.5e-7 -- far below the bf16 rounding of the GEMM output, and a reciprocal,
// an exp2 and five FMAs instead of a general erf.
constexpr float AS_P = 0.3275911f, AS_A1 = 0.254829592f, AS_A2 = -0.284496736f, AS_A3 = 1.421413741f,
                AS_A4 = -1.453152027f, AS_A5 = 1.061405429f;

// GELU x Phi(x) for the bf16 path (output rounded to bf16).  Phi(x) is
// 1 - erfc(|x| / sqrt 2) / 2 for x >= 0 and erfc(|x| / sqrt 2) / 2 for x < 0, so
// x Phi(x) = max(x, 0) - |x| erfc(|x| / sqrt 2) / 2, with erfc(a) = 1 - erf(a)
// from 7.1.26 above.  The 1 / sqrt 2 of the argument and the 1 / 2 are folded
// into the constants, and the negative tail keeps its relative accuracy (no
// 1 + erf cancellation).
__device__ __forceinline__ float gelu_bf16out(float v) {
  const float av = fabsf(v);
  const float t = __builtin_amdgcn_rcpf(fmaf(AS_P * 0.70710678118654752f, av, 1.0f));
  float poly = fmaf(0.5f * AS_A5, t, 0.5f * AS_A4);
  poly = fmaf(poly, t, 0.5f * AS_A3);
  poly = fmaf(poly, t, 0.5f * AS_A2);
  poly = fmaf(poly, t, 0.5f * AS_A1);
  // exp(-x^2 / 2) = exp2(-x^2 log2(e) / 2); the raw exp2 flushes tiny results to 0
  const float e = __builtin_amdgcn_exp2f(av * (av * (-0.5f * 1.4426950408889634f)));
  return fmaf(-(av * t) * poly, e, fmaxf(v, 0.0f));
}

// its derivative Phi(u) + u phi(u), for the backward epilogue.  The
// exp(-z^2) of erf's tail at z = u / sqrt(2) is exp(-u^2 / 2) = sqrt(2 pi)
// phi(u), so one exponential serves both terms.
__device__ __forceinline__ float gelu_grad_bf16(float u) {
  const float z = u * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(AS_P, fabsf(z), 1.0f));
  float poly = fmaf(AS_A5, t, AS_A4);
  poly = fmaf(poly, t, AS_A3);
  poly = fmaf(poly, t, AS_A2);
  poly = fmaf(poly, t, AS_A1);
  poly *= t;
  const float e = __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);
  const float erf = copysignf(1.0f - poly * e, z);
  return fmaf(0.5f, erf, 0.5f) + u * (0.3989422804014327f * e);
}

// GELU'(v) = Phi(v) + v phi(v) at the fp32 pre-activation, from the same
// terms as gelu_bf16out (for a forward that keeps the derivative): with
// q = erfc(|v| / sqrt 2) / 2, Phi(v) is 1 - q for v >= 0 and q for v < 0, and
// phi(v) = exp(-v^2 / 2) / sqrt(2 pi).
__device__ __forceinline__ float gelu_grad_fwd(float v) {
  const float av = fabsf(v);
  const float t = __builtin_amdgcn_rcpf(fmaf(AS_P * 0.70710678118654752f, av, 1.0f));
  float poly = fmaf(0.5f * AS_A5, t, 0.5f * AS_A4);
  poly = fmaf(poly, t, 0.5f * AS_A3);
  poly = fmaf(poly, t, 0.5f * AS_A2);
  poly = fmaf(poly, t, 0.5f * AS_A1);
  const float e = __builtin_amdgcn_exp2f(av * (av * (-0.5f * 1.4426950408889634f)));
  const float q = (t * poly) * e;
  return fmaf(v, 0.3989422804014327f * e, v >= 0.0f ? 1.0f - q : q);
}

// the factor of a backward epilogue (the output is the GEMM sum times it) from
// the saved value u: the activation's derivative at the pre-activation u, or
// u itself when the forward kept the derivative
template <int EPI>
__device__ __forceinline__ float act_grad(float u) {
  if constexpr (EPI == DSP_EPI_SCALE_BWD) return u;
  return EPI == DSP_EPI_GELU_BWD ? gelu_grad_bf16(u) : (u > 0.0f ? 1.0f : 0.0f);
}

template <int EPI>
constexpr bool epi_is_bwd() {
  return EPI == DSP_EPI_GELU_BWD || EPI == DSP_EPI_RELU_BWD || EPI == DSP_EPI_SCALE_BWD;
}
template <int EPI>
constexpr bool epi_is_gelu() {
  return EPI == DSP_EPI_GELU || EPI == DSP_EPI_GELU_KEEP_GRAD;
}
// what a keeping forward stores beside the activation
template <int EPI>
__device__ __forceinline__ float kept(float v) {
  if constexpr (EPI == DSP_EPI_GELU_KEEP_GRAD) return gelu_grad_fwd(v);
  return v;
}

__device__ __forceinline__ uint2 pack_bf16x4(const float v[4]) {
  bf16x2 lo = {(bf16)v[0], (bf16)v[1]};
  bf16x2 hi = {(bf16)v[2], (bf16)v[3]};
  uint2 w;
  w.x = __builtin_bit_cast(uint32_t, lo);
  w.y = __builtin_bit_cast(uint32_t, hi);
  return w;
}

// Epilogue of four consecutive outputs (row m, columns n .. n+3, n < N) held by
// one lane: bias, optional pre-activation copy, activation or residual, store.
// KEEP (GELU/ReLU only): also store the pre-activation a W + bias, rounded to
// bf16, into `keep_out` at the output's offsets -- what a training forward keeps
// for the activation's backward.  The activation itself still reads the fp32
// sum, so `out` has the bits of the plain epilogue.
// The residual is read at row m, the outputs are written at row om (m itself,
// or its place after a row swap, see RowSwap).
template <int EPI, bool KEEP>
__device__ __forceinline__ void epilogue4(float v[4], int m, int64_t om, int n, int N,
                                          const bf16* __restrict__ bias, const float* resid, void* out,
                                          bf16* keep_out) {
  const bool full = (n + 3 < N) && ((N & 3) == 0);
  if (epi_is_bwd<EPI>()) {
    // keep_out holds the saved value u, read at the output's offsets
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (n + i < N) v[i] *= act_grad<EPI>(bf2f(keep_out[om * N + n + i]));
  }
  if (bias) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (n + i < N) v[i] += bf2f(bias[n + i]);
  }
  const int64_t roff = (int64_t)m * N + n;
  const int64_t off = om * N + n;
  if (KEEP) {
    float k[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) k[i] = kept<EPI>(v[i]);
    if (full) {
      *reinterpret_cast<uint2*>(keep_out + off) = pack_bf16x4(k);
    } else {
      for (int i = 0; i < 4; ++i)
        if (n + i < N) keep_out[off + i] = (bf16)k[i];
    }
  }
  if (epi_is_gelu<EPI>()) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = gelu_bf16out(v[i]);
  }
  if (EPI == DSP_EPI_RELU) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = fmaxf(v[i], 0.0f);
  }
  if (EPI == DSP_EPI_RESID || EPI == DSP_EPI_F32) {
    float* o = static_cast<float*>(out);
    if (EPI == DSP_EPI_RESID) {
      if (full) {
        const float4 rv = *reinterpret_cast<const float4*>(resid + roff);
        v[0] += rv.x; v[1] += rv.y; v[2] += rv.z; v[3] += rv.w;
      } else {
        for (int i = 0; i < 4; ++i)
          if (n + i < N) v[i] += resid[roff + i];
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
      *reinterpret_cast<uint2*>(o + off) = pack_bf16x4(v);
    } else {
      for (int i = 0; i < 4; ++i)
        if (n + i < N) o[off + i] = (bf16)v[i];
    }
  }
}

template <int EPI, bool KEEP>
__global__ __launch_bounds__(NTHR, 2) void gemm_bf16_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ W, const bf16* __restrict__ bias,
    const float* resid, void* out, bf16* keep_out, int M, int N, int K, int n_ntiles, int n_tiles,
    RowSwap rs) {
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

  // Loader: thread t moves 16-byte chunk (row t/8 + 32 i, column 8 (t % 8)) of
  // the A slice (i < 8) and of the W slice (i < 4), through buffer resources
  // whose range ends at the last valid row (rows past M or N read as zero).
  // The per-thread offsets are fixed; a slice only adds its K offset.
  const int lrow = threadIdx.x >> 3, lcol = threadIdx.x & 7;
  const uint32_t row_bytes = (uint32_t)K * 2u;
  const uint32_t a_rows = (uint32_t)min(BM, M - m0), w_rows = (uint32_t)min(BN, N - n0);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + (int64_t)m0 * K, a_rows * row_bytes);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(W + (int64_t)n0 * K, w_rows * row_bytes);
  const uint32_t off0 = (uint32_t)lrow * row_bytes + (uint32_t)lcol * 16u;
  const uint32_t step32 = 32u * row_bytes;            // 32 rows further
  constexpr int A_LOADS = A_CHUNKS / NTHR, W_LOADS = W_CHUNKS / NTHR;
  u32x4 pre[NLOAD];
  auto load_regs = [&](int k0) {
    // columns past K: an offset past every range reads zero
    const bool kin = k0 + 8 * lcol < K;
    const uint32_t off = off0 + (uint32_t)k0 * 2u;
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i)
      pre[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, kin ? off + i * step32 : 0xFFFFFFF0u, 0, 0);
#pragma unroll
    for (int i = 0; i < W_LOADS; ++i)
      pre[A_LOADS + i] =
          __builtin_amdgcn_raw_buffer_load_b128(rw, kin ? off + i * step32 : 0xFFFFFFF0u, 0, 0);
  };
  auto store_lds = [&]() {
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i)
      *reinterpret_cast<u32x4*>(As + (lrow + 32 * i) * PITCH + lcol * 8) = pre[i];
#pragma unroll
    for (int i = 0; i < W_LOADS; ++i)
      *reinterpret_cast<u32x4*>(Ws + (lrow + 32 * i) * PITCH + lcol * 8) = pre[A_LOADS + i];
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
        epilogue4<EPI, KEEP>(v, m, rs.map(m), n, N, bias, resid, out, keep_out);
      }
  }
}

// Large-tile variant for problems with many tiles: 256 x (64 TN) output tile,
// 4 waves of 128 x (32 TN), one work-group per CU (one wave per SIMD) with the
// accumulators in AGPRs.  Two LDS buffers, so one barrier per 64-wide K slice;
// the next slice's LDS stores, each followed by the global load that refills
// its register, are spread between the MFMAs of the current slice's first
// three steps, and each 16-wide K step's fragments are read from LDS during
// the previous step's MFMAs.  The barrier sits before the slice's last step: by
// then every wave has stored the next slice (steps 0-2) and read this slice's
// last fragments, so the next slice's first fragments are read during the
// last step's MFMAs instead of after a barrier at the slice's end.  The MFMAs
// and their k order are those of gemm_bf16_kernel, so both kernels give the
// same bits.
#ifndef DSP_GEMM_BIG_GROUP
#define DSP_GEMM_BIG_GROUP 4
#endif
constexpr int BIG_BM = 256, BIG_GROUP = DSP_GEMM_BIG_GROUP;

template <int EPI, bool KEEP, int TN>
__global__ __launch_bounds__(NTHR, 1) void gemm_bf16_big_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ W, const bf16* __restrict__ bias,
    const float* resid, void* out, bf16* keep_out, int M, int N, int K, int n_ntiles, int n_tiles,
    RowSwap rs) {
  constexpr int TM = 4;
  constexpr int BNB = 2 * TN * 32;
  constexpr int STAGE = (BIG_BM + BNB) * PITCH;
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * STAGE];

  // tile order: contiguous ranges per XCD, then groups of BIG_GROUP m-tiles
  // with m fastest, so that the A and W slices of the tiles running together
  // on one XCD fit its L2
  uint32_t bid = blockIdx.x;
  if ((n_tiles & 7) == 0) bid = (bid & 7u) * ((uint32_t)n_tiles >> 3) + (bid >> 3);
  const int n_mt = n_tiles / n_ntiles;
  const int per_group = BIG_GROUP * n_ntiles;
  const int grp = (int)bid / per_group;
  const int first_m = grp * BIG_GROUP;
  const int gm = min(BIG_GROUP, n_mt - first_m);
  const int rem = (int)bid - grp * per_group;
  const int m0 = (first_m + rem % gm) * BIG_BM, n0 = (rem / gm) * BNB;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;

  // loader: thread t moves 16-byte chunk (row t/8 + 32 i, column 8 (t % 8))
  constexpr int A_LOADS = BIG_BM / 32, W_LOADS = BNB / 32, NL = A_LOADS + W_LOADS;
  const int lrow = threadIdx.x >> 3, lcol = threadIdx.x & 7;
  const uint32_t row_bytes = (uint32_t)K * 2u;
  const uint32_t a_rows = (uint32_t)min(BIG_BM, M - m0), w_rows = (uint32_t)min(BNB, N - n0);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + (int64_t)m0 * K, a_rows * row_bytes);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(W + (int64_t)n0 * K, w_rows * row_bytes);
  const uint32_t off0 = (uint32_t)lrow * row_bytes + (uint32_t)lcol * 16u;
  const uint32_t step32 = 32u * row_bytes;
  u32x4 pre[NL];
  auto gload = [&](int i, int k0) {
    // columns past K: an offset past every range reads zero
    const bool kin = k0 + 8 * lcol < K;
    const uint32_t off = off0 + (uint32_t)k0 * 2u;
    if (i < A_LOADS)
      pre[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, kin ? off + i * step32 : 0xFFFFFFF0u, 0, 0);
    else
      pre[i] = __builtin_amdgcn_raw_buffer_load_b128(rw, kin ? off + (i - A_LOADS) * step32 : 0xFFFFFFF0u, 0, 0);
  };
  auto lstore = [&](int i, int buf) {
    bf16* As = lds + buf * STAGE;
    bf16* Ws = As + BIG_BM * PITCH;
    if (i < A_LOADS)
      *reinterpret_cast<u32x4*>(As + (lrow + 32 * i) * PITCH + lcol * 8) = pre[i];
    else
      *reinterpret_cast<u32x4*>(Ws + (lrow + 32 * (i - A_LOADS)) * PITCH + lcol * 8) = pre[i];
  };

  floatx16 acc[TN][TM];
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  bf16x8 af[2][TM], wf[2][TN];
  auto fread = [&](int slot, int buf, int ks) {
    const bf16* As = lds + buf * STAGE;
    const bf16* Ws = As + BIG_BM * PITCH;
#pragma unroll
    for (int b = 0; b < TM; ++b)
      af[slot][b] = *reinterpret_cast<const bf16x8*>(As + (wm * TM * 32 + 32 * b + l32) * PITCH + 16 * ks + 8 * g);
#pragma unroll
    for (int a = 0; a < TN; ++a)
      wf[slot][a] = *reinterpret_cast<const bf16x8*>(Ws + (wn * TN * 32 + 32 * a + l32) * PITCH + 16 * ks + 8 * g);
  };

  // One K slice from LDS buffer kt & 1.  ST: store the prefetched slice kt + 1
  // into the other buffer; LD: reload each prefetch register with its part of
  // slice kt + 2 right after its store, which gives the loads a slice of MFMAs
  // before their store.  The stores are spread over the MFMAs of the first
  // three steps: in one step, they and the next step's fragment reads
  // together needed more LDS bandwidth than the CU has (~190 of 128 B/clk).
  auto slice = [&](int kt, auto st_c, auto ld_c) {
    constexpr bool ST = decltype(st_c)::value, LD = decltype(ld_c)::value;
    constexpr int NMF = TM * TN;
    constexpr int NSPREAD = 3;  // steps that carry the next slice's LDS stores
    const int b = kt & 1;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < BK / 16) {
        fread(cur ^ 1, b, ks + 1);
      } else if (ST) {
        __syncthreads();
        fread(cur ^ 1, b ^ 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < NMF; ++j) {
        const int a = j / TM, bb = j % TM;
        acc[a][bb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[cur][a], af[cur][bb], acc[a][bb], 0, 0, 0);
        if (ks < NSPREAD && ST) {
#pragma unroll
          for (int i = (ks * NMF + j) * NL / (NSPREAD * NMF); i < (ks * NMF + j + 1) * NL / (NSPREAD * NMF); ++i) {
            lstore(i, b ^ 1);
            if (LD) gload(i, (kt + 2) * BK);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  const int nk = (K + BK - 1) / BK;
#pragma unroll
  for (int i = 0; i < NL; ++i) gload(i, 0);
#pragma unroll
  for (int i = 0; i < NL; ++i) lstore(i, 0);
  if (nk > 1) {
#pragma unroll
    for (int i = 0; i < NL; ++i) gload(i, BK);
  }
  __syncthreads();
  fread(0, 0, 0);
  using yes = std::true_type;
  using no = std::false_type;
  int kt = 0;
  for (; kt + 2 < nk; ++kt) slice(kt, yes{}, yes{});
  if (kt + 1 < nk) {
    slice(kt, yes{}, no{});
    ++kt;
  }
  // Epilogue layout of the fp32-staged results (fp32 output, backward
  // epilogues, pre-activation copy): NP passes of RPP rows (pass p: rows
  // HR p + [0, HR) of each wave row half), 16-byte chunks of 4 columns, PER
  // chunks per thread and pass.  Four passes where two would hold more
  // residual or pre-activation reads than the registers do.
  constexpr bool BWD = epi_is_bwd<EPI>();
  constexpr bool F32OUT = EPI == DSP_EPI_RESID || EPI == DSP_EPI_F32;
  constexpr int NP = (TN == 4 && (EPI == DSP_EPI_RESID || BWD)) ? 4 : 2;
  constexpr int RPP = BIG_BM / NP, HR = RPP / 2, BPP = TM / NP;
  constexpr int CPR4 = BNB / 4;
  constexpr int PER = RPP * CPR4 / NTHR;
  const uint32_t rrow = (uint32_t)N * 4u, urow = (uint32_t)N * 2u;
  __amdgpu_buffer_rsrc_t rr, ru;
  if constexpr (EPI == DSP_EPI_RESID) rr = make_rsrc(resid + (int64_t)m0 * N, a_rows * rrow);
  if constexpr (BWD) ru = make_rsrc(keep_out + (int64_t)m0 * N, a_rows * urow);
  constexpr int NRV = EPI == DSP_EPI_RESID ? PER : 1, NUV = BWD ? PER : 1;
  // the residual or saved pre-activation chunks of pass p
  auto side_loads = [&](int p, u32x4 (&rv)[NRV], u32x2 (&uv)[NUV]) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int c = (int)threadIdx.x + NTHR * q;
      const int sr = c / CPR4, cc = c % CPR4;
      const uint32_t tr = (uint32_t)((sr / HR) * 128 + HR * p + sr % HR);
      const int n = n0 + 4 * cc;
      if constexpr (EPI == DSP_EPI_RESID)
        rv[q] = __builtin_amdgcn_raw_buffer_load_b128(rr, n < N ? tr * rrow + (uint32_t)n * 4u : 0xFFFFFFF0u, 0, 0);
      if constexpr (BWD)
        uv[q] = __builtin_amdgcn_raw_buffer_load_b64(ru, n < N ? tr * urow + (uint32_t)n * 2u : 0xFFFFFFF0u, 0, 0);
    }
  };
  // the first pass's reads go out before the last slice, whose MFMAs then
  // hide their latency
  u32x4 rv0[NRV];
  u32x2 uv0[NUV];
  if constexpr (EPI == DSP_EPI_RESID || BWD) side_loads(0, rv0, uv0);
  slice(kt, no{}, no{});

  // Epilogue (N is a multiple of 8 here).  The accumulators hold, per lane,
  // rows m = .. + 32 bb + l32 and in each the column groups
  // n = .. + 32 a + 8 r4 + 4 g + {0..3}: stored from there, one store
  // instruction would write 16-byte pieces of 32 rows, and the L2 would take
  // a request per piece.  So the tile goes through LDS (free once every wave
  // has read its last fragments) and leaves in whole rows: 64 lanes write
  // consecutive 16-byte chunks of one or two rows.
  constexpr int NG = TN * 4;  // column groups of 4 per lane and row
  // Bias of each column group, kept as bf16 pairs until used.  Without a
  // bias the loads read nothing (empty range) and the pairs become -0, the
  // one addend that leaves every value, -0 included, unchanged: the adds stay
  // unconditional, with no branch for the accumulators to be copied across.
  u32x2 braw[NG];
  {
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(bias, bias ? (uint32_t)N * 2u : 0u);
    const uint32_t neg0 = bias ? 0u : 0x80008000u;
#pragma unroll
    for (int j = 0; j < NG; ++j) {
      const int n = n0 + wn * TN * 32 + 32 * (j / 4) + 8 * (j % 4) + 4 * g;
      braw[j] = __builtin_amdgcn_raw_buffer_load_b64(rb, n < N ? (uint32_t)n * 2u : 0xFFFFFFF0u, 0, 0);
      braw[j][0] |= neg0;
      braw[j][1] |= neg0;
    }
  }
  // a W + bias of accumulator row block bb, column group j
  auto sum4 = [&](int bb, int j, float v[4]) {
    const int a = j / 4, r4 = j % 4;
    v[0] = acc[a][bb][4 * r4 + 0] + __uint_as_float(braw[j][0] << 16);
    v[1] = acc[a][bb][4 * r4 + 1] + __uint_as_float(braw[j][0] & 0xFFFF0000u);
    v[2] = acc[a][bb][4 * r4 + 2] + __uint_as_float(braw[j][1] << 16);
    v[3] = acc[a][bb][4 * r4 + 3] + __uint_as_float(braw[j][1] & 0xFFFF0000u);
  };
  // output row of each tile row (the row swap evaluated once per row), at
  // the end of the LDS buffers, past every staged row
  uint32_t* orows = reinterpret_cast<uint32_t*>(lds + 2 * STAGE) - BIG_BM;
  auto put_orow = [&]() {
    const int m = m0 + (int)threadIdx.x;
    orows[threadIdx.x] = (uint32_t)rs.map(m < M ? m : 0);
  };
  if constexpr (!F32OUT && !BWD) {
    // bf16 results, activation applied in registers, staged as bf16 and
    // stored in 16-byte chunks of 8 columns.  Two halves (accumulator row
    // blocks 0-1, then 2-3, i.e. tile rows 64 h + [0, 64) of each wave row
    // half): the first half's stores are in flight while the second half's
    // activation is computed.  KEEP: the pre-activation copy of a half is
    // staged in the other half's rows (tile row r ^ 64), free at that time.
    constexpr int SP = BNB + 8;  // staged row pitch (bf16): a 16-byte pad
    static_assert(BIG_BM * SP * 2 + BIG_BM * 4 <= 2 * STAGE * 2, "bf16 staging fits the LDS buffers");
    constexpr int CPR = BNB / 8;  // chunks per row
    bf16* st = lds;
    __syncthreads();
    put_orow();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (KEEP && h == 1) __syncthreads();  // the first half's copies are read
#pragma unroll
      for (int bb = 2 * h; bb < 2 * h + 2; ++bb)
#pragma unroll
        for (int j = 0; j < NG; ++j) {
          float v[4];
          sum4(bb, j, v);
          const int col = wn * TN * 32 + 32 * (j / 4) + 8 * (j % 4) + 4 * g;
          const int row = wm * TM * 32 + 32 * bb + l32;
          if (KEEP) {
            float k[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) k[i] = kept<EPI>(v[i]);
            *reinterpret_cast<uint2*>(st + (row ^ 64) * SP + col) = pack_bf16x4(k);
          }
          if (epi_is_gelu<EPI>()) {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = gelu_bf16out(v[i]);
          }
          if (EPI == DSP_EPI_RELU) {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = fmaxf(v[i], 0.0f);
          }
          *reinterpret_cast<uint2*>(st + row * SP + col) = pack_bf16x4(v);
        }
      __syncthreads();
#pragma unroll 4
      for (int q = 0; q < CPR / 2; ++q) {
        const int c = (int)threadIdx.x + NTHR * q;
        const int sr = c / CPR, cc = c % CPR;
        const int tr = (sr / 64) * 128 + 64 * h + sr % 64;
        const int m = m0 + tr, n = n0 + 8 * cc;
        const u32x4 w = *reinterpret_cast<const u32x4*>(st + tr * SP + 8 * cc);
        const int64_t o = (int64_t)orows[tr] * N + n;
        if (m < M && n < N) {
          *reinterpret_cast<u32x4*>(static_cast<bf16*>(out) + o) = w;
          if (KEEP)
            *reinterpret_cast<u32x4*>(keep_out + o) = *reinterpret_cast<const u32x4*>(st + (tr ^ 64) * SP + 8 * cc);
        }
      }
    }
  } else {
    // fp32 staging: the reads of pass p > 0 are issued before its staging
    constexpr int SPF = BNB + 4;  // staged row pitch (fp32): a 16-byte pad
    static_assert(RPP * SPF * 4 + BIG_BM * 4 <= 2 * STAGE * 2, "fp32 staging fits the LDS buffers");
    constexpr int CPR = CPR4;
    float* sf = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      u32x4 rv[NRV];
      u32x2 uv[NUV];
      if (p == 0) {
#pragma unroll
        for (int q = 0; q < NRV; ++q) rv[q] = rv0[q];
#pragma unroll
        for (int q = 0; q < NUV; ++q) uv[q] = uv0[q];
      } else if constexpr (EPI == DSP_EPI_RESID || BWD) {
        side_loads(p, rv, uv);
      }
      __syncthreads();  // p = 0: last fragments read; p > 0: the previous pass's rows read
      if (p == 0) put_orow();
#pragma unroll
      for (int h = 0; h < BPP; ++h)
#pragma unroll
        for (int j = 0; j < NG; ++j) {
          float v[4];
          sum4(BPP * p + h, j, v);
          const int col = wn * TN * 32 + 32 * (j / 4) + 8 * (j % 4) + 4 * g;
          *reinterpret_cast<float4*>(sf + (wm * HR + 32 * h + l32) * SPF + col) = make_float4(v[0], v[1], v[2], v[3]);
        }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int c = (int)threadIdx.x + NTHR * q;
        const int sr = c / CPR, cc = c % CPR;
        const int tr = (sr / HR) * 128 + HR * p + sr % HR;
        const int m = m0 + tr, n = n0 + 4 * cc;
        const float4 s4 = *reinterpret_cast<const float4*>(sf + sr * SPF + 4 * cc);
        if (m >= M || n >= N) continue;
        float v[4] = {s4.x, s4.y, s4.z, s4.w};
        const int64_t orow = (int64_t)orows[tr] * N;
        if (KEEP) {
          float k[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) k[i] = kept<EPI>(v[i]);
          *reinterpret_cast<uint2*>(keep_out + orow + n) = pack_bf16x4(k);
        }
        if constexpr (BWD) {
          const uint32_t w0 = uv[q][0], w1 = uv[q][1];
          v[0] *= act_grad<EPI>(__uint_as_float(w0 << 16));
          v[1] *= act_grad<EPI>(__uint_as_float(w0 & 0xFFFF0000u));
          v[2] *= act_grad<EPI>(__uint_as_float(w1 << 16));
          v[3] *= act_grad<EPI>(__uint_as_float(w1 & 0xFFFF0000u));
        }
        if (epi_is_gelu<EPI>()) {
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = gelu_bf16out(v[i]);
        }
        if (EPI == DSP_EPI_RELU) {
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = fmaxf(v[i], 0.0f);
        }
        if constexpr (EPI == DSP_EPI_RESID) {
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] += __uint_as_float(rv[q][i]);
        }
        if (F32OUT)
          *reinterpret_cast<float4*>(static_cast<float*>(out) + orow + n) = make_float4(v[0], v[1], v[2], v[3]);
        else
          *reinterpret_cast<uint2*>(static_cast<bf16*>(out) + orow + n) = pack_bf16x4(v);
      }
    }
  }
}

// ---------------------------------------------------------------- fp32 path
constexpr int FT = 64, FK = 64;  // one global round trip per 64-wide K slice

// `pre` (GELU/ReLU, may be null): also store the pre-activation there.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                        const float* __restrict__ W,
                                                        const float* __restrict__ bias,
                                                        const float* resid, float* out, float* pre,
                                                        int M, int N, int K, RowSwap rs) {
  __shared__ float As[FK][FT + 1];
  __shared__ float Bs[FK][FT + 1];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FK) {
    // all loads of the slice first (one round trip), then the LDS stores
    constexpr int PER = FT * FK / 256;
    float la[PER], lb[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + 256 * i;
      const int r = e / FK, kk = e % FK;
      const int gm = m0 + r, gn = n0 + r, gk = k0 + kk;
      la[i] = (gm < M && gk < K) ? A[(int64_t)gm * K + gk] : 0.0f;
      lb[i] = (gn < N && gk < K) ? W[(int64_t)gn * K + gk] : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + 256 * i;
      As[e % FK][e / FK] = la[i];
      Bs[e % FK][e / FK] = lb[i];
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
      const int64_t off = rs.map(m) * N + n;
      if ((EPI == DSP_EPI_GELU || EPI == DSP_EPI_RELU) && pre) pre[off] = v;
      if (EPI == DSP_EPI_GELU) v = 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
      if (EPI == DSP_EPI_RELU) v = fmaxf(v, 0.0f);
      if (EPI == DSP_EPI_RESID) v += resid[(int64_t)m * N + n];
      out[off] = v;
    }
  }
}

// bf16 transposes of up to kMaxTranspose matrices in one launch (the weights
// of the block backward), one 64 x 64 tile per work-group: 16-byte chunks of
// 8 elements in, through LDS, 16-byte chunks out.  Rows and columns are
// multiples of 8, so a chunk is either wholly inside a matrix or outside.
constexpr int kMaxTranspose = 6;
struct TransposeBatch {
  const uint16_t* x[kMaxTranspose];
  uint16_t* y[kMaxTranspose];
  int rows[kMaxTranspose], cols[kMaxTranspose], col_tiles[kMaxTranspose];
  int first[kMaxTranspose + 1];  // first tile of each matrix; first[n] = all tiles
  int n;
};

__global__ __launch_bounds__(256) void transpose_bf16_batch_kernel(TransposeBatch b) {
  __shared__ __attribute__((aligned(16))) uint16_t t[64][72];
  int m = 0;
  while (m + 1 < b.n && (int)blockIdx.x >= b.first[m + 1]) ++m;
  const int tile = (int)blockIdx.x - b.first[m];
  const int R = b.rows[m], C = b.cols[m];
  const int c0 = (tile % b.col_tiles[m]) * 64, r0 = (tile / b.col_tiles[m]) * 64;
  const uint16_t* x = b.x[m];
  uint16_t* y = b.y[m];
#pragma unroll
  for (int i = threadIdx.x; i < 512; i += 256) {
    const int r = i / 8, c = (i % 8) * 8;
    if (r0 + r < R && c0 + c < C)
      *reinterpret_cast<u32x4*>(&t[r][c]) = *reinterpret_cast<const u32x4*>(x + (int64_t)(r0 + r) * C + c0 + c);
  }
  __syncthreads();
#pragma unroll
  for (int i = threadIdx.x; i < 512; i += 256) {
    const int c = i / 8, r = (i % 8) * 8;
    if (c0 + c < C && r0 + r < R) {
      u32x4 v;
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = (uint32_t)t[r + 2 * j][c] | ((uint32_t)t[r + 2 * j + 1][c] << 16);
      *reinterpret_cast<u32x4*>(y + (int64_t)(c0 + c) * R + r0 + r) = v;
    }
  }
}

}  // namespace

int launch_transpose_bf16_batch(const void* const* x, void* const* y, const int64_t* rows, const int64_t* cols,
                                int n, hipStream_t s) {
  if (n < 1 || n > kMaxTranspose) return DSP_ERR_ARG;
  TransposeBatch b = {};
  b.n = n;
  int64_t tiles = 0;
  for (int i = 0; i < n; ++i) {
    if (rows[i] < 1 || cols[i] < 1 || rows[i] % 8 || cols[i] % 8 || rows[i] * cols[i] >= (int64_t(1) << 31))
      return DSP_ERR_SHAPE;
    b.x[i] = static_cast<const uint16_t*>(x[i]);
    b.y[i] = static_cast<uint16_t*>(y[i]);
    b.rows[i] = (int)rows[i];
    b.cols[i] = (int)cols[i];
    b.col_tiles[i] = (int)((cols[i] + 63) / 64);
    b.first[i] = (int)tiles;
    tiles += ((rows[i] + 63) / 64) * b.col_tiles[i];
  }
  b.first[n] = (int)tiles;
  hipLaunchKernelGGL(transpose_bf16_batch_kernel, dim3((uint32_t)tiles), dim3(256), 0, s, b);
  return last_launch_status();
}

bool linear_bf16_large_tiles(int64_t M, int N) {
  const int big_bn = N >= 2048 ? 256 : 192;
  const int64_t big_tiles = ((M + BIG_BM - 1) / BIG_BM) * ((N + big_bn - 1) / big_bn);
  return DSP_GEMM_BIG && big_tiles >= 256 && N % 8 == 0 && (int64_t)BIG_BM * N * 4 < (int64_t(1) << 31);
}

int launch_linear_bf16(const void* a, const void* w, const void* bias, const float* residual,
                       void* out, int64_t M, int N, int K, int epilogue, hipStream_t s, void* pre, RowSwap rs) {
  if (M == 0) return DSP_OK;
  // backward epilogues: `pre` is the saved value, read (not written)
  const bool bwd = epilogue == DSP_EPI_GELU_BWD || epilogue == DSP_EPI_RELU_BWD || epilogue == DSP_EPI_SCALE_BWD;
  if (bwd && (!pre || rs.outer != 0)) return DSP_ERR_ARG;
  const int64_t n_mt = (M + BM - 1) / BM, n_nt = (N + BN - 1) / BN;
  const int64_t tiles = n_mt * n_nt;
  // a tile's buffer resources address BM rows of K bf16 with 32-bit offsets
  if (tiles >= (int64_t(1) << 31) || M >= (int64_t(1) << 31) || (int64_t)BM * K * 2 >= (int64_t(1) << 31))
    return DSP_ERR_SHAPE;
  const bool keep = pre != nullptr && !bwd;
  if (keep && epilogue != DSP_EPI_GELU && epilogue != DSP_EPI_RELU && epilogue != DSP_EPI_GELU_KEEP_GRAD)
    return DSP_ERR_ARG;
  if (epilogue == DSP_EPI_GELU_KEEP_GRAD && !keep) return DSP_ERR_ARG;
  const bf16* A = static_cast<const bf16*>(a);
  const bf16* Wt = static_cast<const bf16*>(w);
  const bf16* bs = static_cast<const bf16*>(bias);
  bf16* pb = static_cast<bf16*>(pre);
  // Large tiles when they still fill every CU at least once: 256 x 256 for
  // wide outputs, 256 x 192 otherwise (N = 1152 is six of them).
  const int big_bn = N >= 2048 ? 256 : 192;
  const int64_t big_nt = (N + big_bn - 1) / big_bn;
  const int64_t big_tiles = ((M + BIG_BM - 1) / BIG_BM) * big_nt;
  // (the large-tile epilogue addresses a tile's 256 rows of fp32 residual
  // with 32-bit offsets)
  const bool big = linear_bf16_large_tiles(M, N);
#define DSP_GEMM_LAUNCH(E, KP)                                                                                  \
  do {                                                                                                        \
    if (!big) {                                                                                               \
      hipLaunchKernelGGL((gemm_bf16_kernel<E, KP>), dim3((uint32_t)tiles), dim3(NTHR), 0, s, A, Wt, bs, residual, \
                         out, pb, (int)M, N, K, (int)n_nt, (int)tiles, rs);                                        \
    } else if (big_bn == 256) {                                                                               \
      hipLaunchKernelGGL((gemm_bf16_big_kernel<E, KP, 4>), dim3((uint32_t)big_tiles), dim3(NTHR), 0, s, A, Wt,  \
                         bs, residual, out, pb, (int)M, N, K, (int)big_nt, (int)big_tiles, rs);                    \
    } else {                                                                                                  \
      hipLaunchKernelGGL((gemm_bf16_big_kernel<E, KP, 3>), dim3((uint32_t)big_tiles), dim3(NTHR), 0, s, A, Wt,  \
                         bs, residual, out, pb, (int)M, N, K, (int)big_nt, (int)big_tiles, rs);                    \
    }                                                                                                         \
  } while (0)
  switch (epilogue) {
    case DSP_EPI_NONE: DSP_GEMM_LAUNCH(DSP_EPI_NONE, false); break;
    case DSP_EPI_RESID: DSP_GEMM_LAUNCH(DSP_EPI_RESID, false); break;
    case DSP_EPI_F32: DSP_GEMM_LAUNCH(DSP_EPI_F32, false); break;
    case DSP_EPI_GELU:
      if (keep) DSP_GEMM_LAUNCH(DSP_EPI_GELU, true); else DSP_GEMM_LAUNCH(DSP_EPI_GELU, false);
      break;
    case DSP_EPI_RELU:
      if (keep) DSP_GEMM_LAUNCH(DSP_EPI_RELU, true); else DSP_GEMM_LAUNCH(DSP_EPI_RELU, false);
      break;
    case DSP_EPI_GELU_KEEP_GRAD: DSP_GEMM_LAUNCH(DSP_EPI_GELU_KEEP_GRAD, true); break;
    case DSP_EPI_GELU_BWD: DSP_GEMM_LAUNCH(DSP_EPI_GELU_BWD, false); break;
    case DSP_EPI_SCALE_BWD: DSP_GEMM_LAUNCH(DSP_EPI_SCALE_BWD, false); break;
    case DSP_EPI_RELU_BWD: DSP_GEMM_LAUNCH(DSP_EPI_RELU_BWD, false); break;
    default:
      return DSP_ERR_ARG;
  }
#undef DSP_GEMM_LAUNCH
  return last_launch_status();
}

int launch_linear_f32(const float* a, const float* w, const float* bias, const float* residual,
                      float* out, int64_t M, int N, int K, int epilogue, hipStream_t s, float* pre, RowSwap rs) {
  if (M == 0) return DSP_OK;
  const int64_t gy = (M + FT - 1) / FT;
  if (gy >= 65536 * 1024) return DSP_ERR_SHAPE;
  if (pre && epilogue != DSP_EPI_GELU && epilogue != DSP_EPI_RELU) return DSP_ERR_ARG;
  const dim3 grid((uint32_t)((N + FT - 1) / FT), (uint32_t)gy), block(256);
#define DSP_GEMM_LAUNCH(E) \
  hipLaunchKernelGGL(gemm_f32_kernel<E>, grid, block, 0, s, a, w, bias, residual, out, pre, (int)M, N, K, rs)
  switch (epilogue) {
    case DSP_EPI_NONE: DSP_GEMM_LAUNCH(DSP_EPI_NONE); break;
    case DSP_EPI_GELU: DSP_GEMM_LAUNCH(DSP_EPI_GELU); break;
    case DSP_EPI_RESID: DSP_GEMM_LAUNCH(DSP_EPI_RESID); break;
    case DSP_EPI_F32: DSP_GEMM_LAUNCH(DSP_EPI_NONE); break;
    case DSP_EPI_RELU: DSP_GEMM_LAUNCH(DSP_EPI_RELU); break;
    default:
      return DSP_ERR_ARG;
  }
#undef DSP_GEMM_LAUNCH
  return last_launch_status();
}

}  // namespace dsp
