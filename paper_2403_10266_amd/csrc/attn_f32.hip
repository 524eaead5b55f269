// fp32 attention along one sequence dimension (Eq. 3 per head; also grouped
// key/value heads and a key length of its own for cross-attention), the exact
// path: fp32 storage, fp32 FMA arithmetic, no reduced-precision operand
// anywhere.  Head widths 16, 32, 64, 72, 80 and 96 run one wave per unit
// (attn_f32_unit_kernel below); any other width runs the general kernel, in
// which one thread owns one (unit, query, 32-column slice of the output):
// a first pass over the keys finds the row maximum of the scaled scores, a
// second pass accumulates exp(score - max) and the weighted values of its
// slice.  Meant for small problems and for checking; the bf16 MFMA kernel is
// the fast path.
#include <math.h>

#include "dsp_internal.h"

namespace dsp {
namespace {

constexpr int DC = 32;  // output columns per thread

struct ParamsF {
  const float* q;
  const float* k;
  const float* v;
  float* o;
  float* lse;  // optional row log-sum-exp output
  int64_t b_in, x_in, r_in, b_out, x_out, r_out;
  int64_t b_kv, x_kv, r_kv, Lk, grp;  // keys/values: layout, count, query heads per kv head
  int64_t X, H, L, D, n_dc, total;
  float scale;
};

__global__ __launch_bounds__(256) void attn_f32_kernel(ParamsF p) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= p.total) return;
  // tid -> (unit, query, column slice), slice fastest
  const int64_t dc = tid % p.n_dc;
  const int64_t uq = tid / p.n_dc;
  const int64_t qi = uq % p.L;
  const int64_t unit = uq / p.L;
  const int64_t h = unit % p.H;
  const int64_t bx = unit / p.H;
  const int64_t xx = bx % p.X;
  const int64_t bb = bx / p.X;
  const int64_t in_base = bb * p.b_in + xx * p.x_in + h * p.D;
  const float* qrow = p.q + in_base + qi * p.r_in;
  const int64_t kv_base = bb * p.b_kv + xx * p.x_kv + (h / p.grp) * p.D;
  const float* kb = p.k + kv_base;
  const float* vb = p.v + kv_base;
  float m = -INFINITY;
  for (int64_t j = 0; j < p.Lk; ++j) {
    const float* krow = kb + j * p.r_kv;
    float s = 0.0f;
    for (int64_t d = 0; d < p.D; ++d) s = fmaf(qrow[d], krow[d], s);
    m = fmaxf(m, s * p.scale);
  }
  const int64_t c0 = dc * DC;
  const int64_t nc = min((int64_t)DC, p.D - c0);
  float acc[DC];
#pragma unroll
  for (int c = 0; c < DC; ++c) acc[c] = 0.0f;
  float l = 0.0f;
  for (int64_t j = 0; j < p.Lk; ++j) {
    const float* krow = kb + j * p.r_kv;
    float s = 0.0f;
    for (int64_t d = 0; d < p.D; ++d) s = fmaf(qrow[d], krow[d], s);
    const float e = expf(s * p.scale - m);
    l += e;
    const float* vrow = vb + j * p.r_kv + c0;
#pragma unroll
    for (int c = 0; c < DC; ++c)
      if (c < nc) acc[c] = fmaf(e, vrow[c], acc[c]);
  }
  float* orow = p.o + bb * p.b_out + xx * p.x_out + h * p.D + qi * p.r_out + c0;
  const float inv = 1.0f / l;
  if (p.lse && dc == 0) p.lse[unit * p.L + qi] = m + logf(l);
#pragma unroll
  for (int c = 0; c < DC; ++c)
    if (c < nc) orow[c] = acc[c] * inv;
}

// One wave per unit for common head widths: the unit's keys and values pass
// through LDS in chunks of KC rows (every lane reads the same row: an LDS
// broadcast), each lane owns queries lane, lane + 64, ... with its query row
// and its D output columns in registers, and the softmax runs online (the
// reference maximum moves when a larger score arrives, rescaling the
// accumulator and the row sum by exp of the difference).  Same arithmetic
// type (fp32 FMAs, expf) as the kernel above, but no loop waits on global
// memory per key.
template <int D>
__global__ __launch_bounds__(64) void attn_f32_unit_kernel(ParamsF p) {
  constexpr int KC = 32;
  __shared__ __attribute__((aligned(16))) float ks[KC * D];
  __shared__ __attribute__((aligned(16))) float vs[KC * D];
  const int lane = threadIdx.x;
  const int64_t unit = blockIdx.x;
  const int64_t h = unit % p.H;
  const int64_t bx = unit / p.H;
  const int64_t xx = bx % p.X;
  const int64_t bb = bx / p.X;
  const float* qg = p.q + bb * p.b_in + xx * p.x_in + h * D;
  const int64_t kv_base = bb * p.b_kv + xx * p.x_kv + (h / p.grp) * D;
  const float* kg = p.k + kv_base;
  const float* vg = p.v + kv_base;
  float* og = p.o + bb * p.b_out + xx * p.x_out + h * D;
  for (int64_t q0 = 0; q0 < p.L; q0 += 64) {
    const int64_t qi = q0 + lane;
    const bool valid = qi < p.L;
    float qr[D], acc[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
      qr[d] = valid ? qg[qi * p.r_in + d] : 0.0f;
      acc[d] = 0.0f;
    }
    float m = -INFINITY, l = 0.0f;
    for (int64_t k0 = 0; k0 < p.Lk; k0 += KC) {
      const int nk = (int)min((int64_t)KC, p.Lk - k0);
      __syncthreads();  // the previous chunk is consumed
      for (int e = lane; e < nk * D; e += 64) {
        const int r = e / D, c = e - r * D;
        ks[e] = kg[(k0 + r) * p.r_kv + c];
        vs[e] = vg[(k0 + r) * p.r_kv + c];
      }
      __syncthreads();
      for (int j = 0; j < nk; ++j) {
        float sc = 0.0f;
#pragma unroll
        for (int d = 0; d < D; ++d) sc = fmaf(qr[d], ks[j * D + d], sc);
        sc *= p.scale;
        if (sc > m) {
          const float corr = expf(m - sc);  // 0 for the first key
          l *= corr;
#pragma unroll
          for (int d = 0; d < D; ++d) acc[d] *= corr;
          m = sc;
        }
        const float e = expf(sc - m);
        l += e;
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] = fmaf(e, vs[j * D + d], acc[d]);
      }
    }
    if (valid) {
      const float inv = 1.0f / l;
      float* orow = og + qi * p.r_out;
#pragma unroll
      for (int d = 0; d < D; ++d) orow[d] = acc[d] * inv;
      if (p.lse) p.lse[unit * p.L + qi] = m + logf(l);
    }
  }
}

}  // namespace

int launch_attn_f32(const AttnArgs& a, hipStream_t s) {
  ParamsF p;
  p.q = static_cast<const float*>(a.q);
  p.k = static_cast<const float*>(a.k);
  p.v = static_cast<const float*>(a.v);
  p.o = static_cast<float*>(a.o);
  p.lse = a.lse;
  p.b_in = a.b_stride_in;
  p.x_in = a.x_stride_in;
  p.r_in = a.r_stride_in;
  p.b_out = a.b_stride_out;
  p.x_out = a.x_stride_out;
  p.r_out = a.r_stride_out;
  p.b_kv = a.b_stride_kv;
  p.x_kv = a.x_stride_kv;
  p.r_kv = a.r_stride_kv;
  p.Lk = a.Lk;
  p.grp = a.H / a.Hkv;
  p.X = a.X;
  p.H = a.H;
  p.L = a.L;
  p.D = a.D;
  p.n_dc = (a.D + DC - 1) / DC;
  p.total = a.B * a.X * a.H * a.L * p.n_dc;
  p.scale = a.scale;
  if (p.total == 0) return DSP_OK;
  const int64_t units = a.B * a.X * a.H;
  if (units < (int64_t(1) << 31)) {
    const dim3 g((uint32_t)units), b(64);
    switch (a.D) {
      case 16: hipLaunchKernelGGL(attn_f32_unit_kernel<16>, g, b, 0, s, p); return last_launch_status();
      case 32: hipLaunchKernelGGL(attn_f32_unit_kernel<32>, g, b, 0, s, p); return last_launch_status();
      case 64: hipLaunchKernelGGL(attn_f32_unit_kernel<64>, g, b, 0, s, p); return last_launch_status();
      case 72: hipLaunchKernelGGL(attn_f32_unit_kernel<72>, g, b, 0, s, p); return last_launch_status();
      case 80: hipLaunchKernelGGL(attn_f32_unit_kernel<80>, g, b, 0, s, p); return last_launch_status();
      case 96: hipLaunchKernelGGL(attn_f32_unit_kernel<96>, g, b, 0, s, p); return last_launch_status();
      default: break;
    }
  }
  const int64_t blocks = (p.total + 255) / 256;
  if (blocks >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  hipLaunchKernelGGL(attn_f32_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, p);
  return last_launch_status();
}

}  // namespace dsp
