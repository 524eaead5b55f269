// One attention sublayer of the projection-only fp32 chain in one kernel, for
// small shapes: for a group of L consecutive token rows (a frame for the
// spatial half, a spatial location for the temporal half -- the reshape of
// Eq. 7-8),
//     out_rows = Attn(x_rows W_qkv + b_qkv) W_o + b_o
// with Attn the per-head softmax attention of Eq. 3 (heads as in Eq. 1-2).
// At these sizes the separate GEMM and attention launches are bound by their
// fixed costs (dispatch and one global round trip each), not by work; here one
// work-group loads its rows and the weights in one round trip, keeps every
// intermediate in LDS, and writes the sublayer's output rows -- in (B, S, T)
// order for the spatial half, which performs the Switch on the way out.
// Arithmetic is fp32 FMA with expf (as the fp32 path's kernels), the softmax
// two-pass with the exact row maximum.
#include <math.h>

#include "dsp_internal.h"

namespace dsp {
namespace {

constexpr int CH_CMAX = 64, CH_LMAX = 64;
// LDS floats for the largest shape: rows, W_qkv (pitch C + 4), qkv (pitch 3C + 4)
constexpr int CH_LDS = CH_LMAX * CH_CMAX + 3 * CH_CMAX * (CH_CMAX + 4) + CH_LMAX * (3 * CH_CMAX + 4);

struct ChainParams {
  const float* x;  // group g's row r at x + (g * L + r) * C
  const float* wqkv;  // [3C][C], stored [out][in]
  const float* bqkv;  // [3C] or null
  const float* wo;    // [C][C]
  const float* bo;    // [C] or null
  float* y;           // row rs.map(g * L + r); may alias x (each group reads its rows before writing them)
                      // x, y and the weights 16-byte aligned
  int L, C, H, D;
  float scale;
  RowSwap rs;
};

// out[m][n] = b[n] + sum_k a[m][k] w[n][k] for rows [m0, m1) of one output
// column n: float4 chunks of the weight row and of four activation rows at a
// time (the activation reads are broadcasts), four independent accumulators
template <typename Store>
__device__ __forceinline__ void chain_gemm_col(const float* a, int C, const float* wrow, float b, int m0, int m1,
                                               Store store) {
  for (int m = m0; m < m1; m += 4) {
    const int mr[4] = {m, min(m + 1, m1 - 1), min(m + 2, m1 - 1), min(m + 3, m1 - 1)};
    float acc[4] = {b, b, b, b};
#pragma unroll 2
    for (int k = 0; k < C; k += 4) {
      const float4 w = *reinterpret_cast<const float4*>(wrow + k);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float4 xv = *reinterpret_cast<const float4*>(a + mr[r] * C + k);
        acc[r] = fmaf(xv.x, w.x, acc[r]);
        acc[r] = fmaf(xv.y, w.y, acc[r]);
        acc[r] = fmaf(xv.z, w.z, acc[r]);
        acc[r] = fmaf(xv.w, w.w, acc[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (m + r < m1) store(m + r, acc[r]);  // rows past m1 recomputed the last one
  }
}

// NTH threads: 1024 for head widths up to 32 (more threads for the two
// GEMMs' output columns and row bands; the attention's per-thread registers
// still fit), 256 for 64
template <int DT, int NTH>
__global__ __launch_bounds__(NTH) void chain_sublayer_f32_kernel(ChainParams p) {
  const int L = p.L, C = p.C, H = p.H;
  constexpr int D = DT;
  constexpr int CH_NT = NTH;
  const int C3 = 3 * C;
  const int WP = C + 4;     // weight row pitch (floats): float4 rows
  const int QP = C3 + 4;    // qkv row pitch: float4 rows
  __shared__ __attribute__((aligned(16))) float smem[CH_LDS];
  float* xs = smem;                 // [L][C]: the input rows, later the attention output
  float* ws = xs + L * C;           // [3C][WP]: W_qkv, later W_o
  float* qs = ws + C3 * WP;         // [L][QP]: q | k | v
  const int t = threadIdx.x;
  const int64_t row0 = (int64_t)blockIdx.x * L;

  // ---- one round trip: every load of the group's rows, W_qkv and W_o is
  // issued before any is used (float4 chunks; rows are multiples of 4 floats)
  constexpr int X4 = CH_LMAX * CH_CMAX / 4 / CH_NT, WQ4 = 3 * CH_CMAX * CH_CMAX / 4 / CH_NT,
                WO4 = CH_CMAX * CH_CMAX / 4 / CH_NT;
  // chunks past the end re-read the last one (always in bounds, so every
  // load is one unconditional 16-byte load); the stores below skip them
  const int nx = L * C, nq = C3 * C, no = C * C;
  float4 xr[X4], wq[WQ4], wo4[WO4];
#pragma unroll
  for (int i = 0; i < X4; ++i)
    xr[i] = *reinterpret_cast<const float4*>(p.x + row0 * C + min(4 * (t + i * CH_NT), nx - 4));
#pragma unroll
  for (int i = 0; i < WQ4; ++i)
    wq[i] = *reinterpret_cast<const float4*>(p.wqkv + min(4 * (t + i * CH_NT), nq - 4));
#pragma unroll
  for (int i = 0; i < WO4; ++i)
    wo4[i] = *reinterpret_cast<const float4*>(p.wo + min(4 * (t + i * CH_NT), no - 4));
  // weight chunk at element e (4 floats of one row) into LDS row e / C
  auto wstore = [&](int e, float4 v) { *reinterpret_cast<float4*>(ws + (e / C) * WP + e % C) = v; };
#pragma unroll
  for (int i = 0; i < X4; ++i) {
    const int e = 4 * (t + i * CH_NT);
    if (e < nx) *reinterpret_cast<float4*>(xs + e) = xr[i];
  }
#pragma unroll
  for (int i = 0; i < WQ4; ++i) {
    const int e = 4 * (t + i * CH_NT);
    if (e < nq) wstore(e, wq[i]);
  }
  __syncthreads();

  // ---- qkv = x W_qkv + b_qkv: thread -> one output column for a band of rows
  {
    const int bands = CH_NT / C3;
    const int n = t % C3, band = t / C3;
    if (band < bands) {
      const int rows = (L + bands - 1) / bands;
      chain_gemm_col(xs, C, ws + n * WP, p.bqkv ? p.bqkv[n] : 0.0f, band * rows, min(L, (band + 1) * rows),
                     [&](int m, float v) { qs[m * QP + n] = v; });
    }
  }
  __syncthreads();

  // ---- W_o into LDS (the W_qkv rows are no longer read)
#pragma unroll
  for (int i = 0; i < WO4; ++i) {
    const int e = 4 * (t + i * CH_NT);
    if (e < no) wstore(e, wo4[i]);
  }
  // ---- attention per (head, query) task: scores against the L keys, exact
  // row maximum, exp, row sum, probability-weighted values; output into xs
  for (int task = t; task < H * L; task += CH_NT) {
    const int h = task / L, i = task - h * L;
    float qr[D];
#pragma unroll
    for (int d = 0; d < D; d += 4) {
      const float4 v = *reinterpret_cast<const float4*>(qs + i * QP + h * D + d);
      qr[d] = v.x; qr[d + 1] = v.y; qr[d + 2] = v.z; qr[d + 3] = v.w;
    }
    // the scores are recomputed in the second pass rather than kept: a loop
    // over the keys instead of a register array unrolled to the largest L
    // keeps the code small (a short kernel run once pays for every
    // instruction-cache line it touches)
    auto score = [&](int j) {
      const float* kr = qs + j * QP + C + h * D;
      float acc = 0.0f;
#pragma unroll
      for (int d = 0; d < D; d += 4) {
        const float4 v = *reinterpret_cast<const float4*>(kr + d);
        acc = fmaf(qr[d], v.x, acc);
        acc = fmaf(qr[d + 1], v.y, acc);
        acc = fmaf(qr[d + 2], v.z, acc);
        acc = fmaf(qr[d + 3], v.w, acc);
      }
      return acc * p.scale;
    };
    float mx = -INFINITY;
#pragma unroll 2
    for (int j = 0; j < L; ++j) mx = fmaxf(mx, score(j));
    float l = 0.0f;
    float o[D];
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] = 0.0f;
#pragma unroll 2
    for (int j = 0; j < L; ++j) {
      const float e = expf(score(j) - mx);
      l += e;
      const float* vr = qs + j * QP + 2 * C + h * D;
#pragma unroll
      for (int d = 0; d < D; d += 4) {
        const float4 v = *reinterpret_cast<const float4*>(vr + d);
        o[d] = fmaf(e, v.x, o[d]);
        o[d + 1] = fmaf(e, v.y, o[d + 1]);
        o[d + 2] = fmaf(e, v.z, o[d + 2]);
        o[d + 3] = fmaf(e, v.w, o[d + 3]);
      }
    }
    const float inv = 1.0f / l;
#pragma unroll
    for (int d = 0; d < D; d += 4)
      *reinterpret_cast<float4*>(xs + i * C + h * D + d) =
          make_float4(o[d] * inv, o[d + 1] * inv, o[d + 2] * inv, o[d + 3] * inv);
  }
  __syncthreads();

  // ---- out = o W_o + b_o, rows written at rs.map(global row)
  {
    const RowSwap rs = p.rs;
    float* const y = p.y;
    const int bands = CH_NT / C;
    const int n = t % C, band = t / C;
    if (band < bands) {
      const int rows = (L + bands - 1) / bands;
      chain_gemm_col(xs, C, ws + n * WP, p.bo ? p.bo[n] : 0.0f, band * rows, min(L, (band + 1) * rows),
                     [=](int m, float v) { y[rs.map((int)(row0 + m)) * C + n] = v; });
    }
  }
}

}  // namespace

bool chain_sublayer_f32_fits(int64_t L, int C, int H) {
  // float4 rows of x, q, k, v; head widths with an instance of the kernel
  if (L < 1 || L > CH_LMAX || C < 4 || C > CH_CMAX || H < 1 || C % H) return false;
  const int D = C / H;
  return D == 8 || D == 16 || D == 32 || D == 64;
}

int launch_chain_sublayer_f32(const float* x, const float* wqkv, const float* bqkv, const float* wo, const float* bo,
                              float* y, int64_t groups, int L, int C, int H, float scale, RowSwap rs, hipStream_t s) {
  if (groups == 0) return DSP_OK;
  if (!chain_sublayer_f32_fits(L, C, H) || groups >= (int64_t(1) << 31) || groups * L >= (int64_t(1) << 31))
    return DSP_ERR_SHAPE;
  ChainParams p;
  p.x = x;
  p.wqkv = wqkv;
  p.bqkv = bqkv;
  p.wo = wo;
  p.bo = bo;
  p.y = y;
  p.L = L;
  p.C = C;
  p.H = H;
  p.D = C / H;
  p.scale = scale;
  p.rs = rs;
  switch (p.D) {
    case 8: hipLaunchKernelGGL((chain_sublayer_f32_kernel<8, 1024>), dim3((uint32_t)groups), dim3(1024), 0, s, p); break;
    case 16: hipLaunchKernelGGL((chain_sublayer_f32_kernel<16, 1024>), dim3((uint32_t)groups), dim3(1024), 0, s, p); break;
    case 32: hipLaunchKernelGGL((chain_sublayer_f32_kernel<32, 1024>), dim3((uint32_t)groups), dim3(1024), 0, s, p); break;
    case 64: hipLaunchKernelGGL((chain_sublayer_f32_kernel<64, 256>), dim3((uint32_t)groups), dim3(256), 0, s, p); break;
    default: return DSP_ERR_SHAPE;
  }
  return last_launch_status();
}

}  // namespace dsp
