// Internal declarations shared by the libdsp translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dsp.h"

namespace dsp {

// Launch wrappers implemented in the kernel translation units.  Arguments have
// been validated by the ABI layer; each returns a dsp_status_t.
// N-rank exchange + unpack (exchange.hip); N <= kMaxExchangeRanks.
constexpr int kMaxExchangeRanks = 64;
int launch_exchange_unpack(const void* const* packed, void* const* out, int64_t N, int64_t B,
                           int64_t P, int64_t run_bytes, hipStream_t s);
// Strided row copy (rowcopy.hip): rows of row_bytes bytes; the row at
// multi-index (i_0, .., i_{nd-1}) moves from row sum(i_d * src_stride[d]) of
// src[p] to row sum(i_d * dst_stride[d]) of dst[p], for each pair p.
constexpr int kMaxCopyDims = 6;
constexpr int kMaxCopyPairs = 64;
struct RowCopyDesc {
  int nd;
  int64_t size[kMaxCopyDims];
  int64_t src_stride[kMaxCopyDims];
  int64_t dst_stride[kMaxCopyDims];
  int64_t row_bytes;
};
int launch_rowcopy(const void* const* src, void* const* dst, int n_pairs, const RowCopyDesc& desc,
                   hipStream_t s);
int launch_switch_rows(const void* x, void* y, int64_t B, int64_t D1, int64_t D2, int64_t row_bytes,
                       int from_dim, int to_dim, int64_t n_chunks, hipStream_t s);
int launch_switch_tiles(const void* x, void* y, int64_t B, int64_t D1, int64_t D2, int64_t C,
                        int elem_bytes, int from_dim, int to_dim, int64_t n_chunks, hipStream_t s);

// Attention over units of L consecutive sequence positions.  Unit u decomposes
// as u = (b * X + x) * H + h; position r of unit (b, x, h) sits at element
//   b * b_stride + x * x_stride + r * r_stride + h * D
// of q/k/v (strides *_in) and of o (strides *_out).
// Cross-attention and grouped key/value heads: the unit's keys and values are
// Lk positions of key/value head h / (H / Hkv), at b * b_stride_kv + x *
// x_stride_kv + r * r_stride_kv + (h / (H / Hkv)) * D of k and v (self-attention:
// Lk = L, Hkv = H and the kv strides equal the in strides).
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int64_t B, X, L;
  int H, D;
  int64_t b_stride_in, x_stride_in, r_stride_in;
  int64_t b_stride_out, x_stride_out, r_stride_out;
  int64_t Lk;
  int Hkv;
  int64_t b_stride_kv, x_stride_kv, r_stride_kv;
  float scale;
  // optional (may be null): fp32 [B * X * H][L], the natural-log row
  // log-sum-exp of the scaled scores of each query (the backward's statistic)
  float* lse;
};
int launch_attn_bf16(const AttnArgs& a, hipStream_t s);

// Backward of attention (attn_bwd.hip).  Units and positions as in AttnArgs
// (L queries, Lk keys, Hkv key/value heads): q and dq use q_strides, k, v, dk
// and dv kv_strides, o and dout o_strides; lse and delta are fp32
// [B * X * H][L] (delta is written by the first kernel).
struct AttnBwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dout;
  const float* lse;
  void* dq;
  void* dk;
  void* dv;
  float* delta;
  int64_t B, X, L, Lk;
  int H, Hkv, D;
  int64_t q_strides[3], kv_strides[3], o_strides[3];
  float scale;
};
bool attn_bwd_bf16_fits(const AttnBwdArgs& a);
int launch_attn_bwd_bf16(const AttnBwdArgs& a, hipStream_t s);
int launch_attn_bwd_f32(const AttnBwdArgs& a, hipStream_t s);
int launch_attn_f32(const AttnArgs& a, hipStream_t s);
bool attn_bf16_supports(int D);
// Persistent kernel for short units, L <= kShortAttnMaxL (attn_short.hip);
// attn_bf16_short_fits() tells whether the shape is in its 32-bit range.
constexpr int kShortAttnMaxL = 128;
bool attn_bf16_short_fits(const AttnArgs& a);
int launch_attn_bf16_short(const AttnArgs& a, hipStream_t s);

int launch_layernorm(const void* x, int x_bf16, void* y, int y_bf16, int64_t rows, int C, float eps,
                     hipStream_t s);

// Gradient GEMMs (gemm_grad.hip): out[m][n] = sum_k A(m, k) B(n, k) with
// A(m, k) = a[m * lda + k] (ta = 0) or a[k * lda + m] (ta = 1), B likewise.
// epi: DSP_GRAD_EPI_*.  splits > 1 (fp32 output only) uses ws, fp32
// [splits][M][N].  bf16 needs M, N, K multiples of 8 (checked by the ABI).
int grad_splits(int64_t M, int64_t N, int64_t K);
bool grad_gemm_fits(int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb);
int launch_gemm_grad(const void* a, int ta, int64_t lda, const void* b, int tb, int64_t ldb, const void* aux,
                     void* out, int64_t M, int64_t N, int64_t K, int epi, int splits, float* ws, hipStream_t s);
int launch_gemm_grad_f32(const float* a, int ta, int64_t lda, const float* b, int tb, int64_t ldb,
                         const float* aux, float* out, int64_t M, int64_t N, int64_t K, int epi, hipStream_t s);
int launch_add_f32(const float* a, const float* b, float* out, int64_t n, hipStream_t s);
int launch_colsum_bf16(const void* dy, float* db, int64_t M, int N, hipStream_t s);
int launch_colsum_f32(const float* dy, float* db, int64_t M, int N, hipStream_t s);


int launch_cast(const void* x, int x_bf16, void* y, int y_bf16, int64_t n, hipStream_t s);

// Output row of GEMM row m when the rows are (b, t, s) tokens of a (B, T, S)
// sequence and the output is wanted in (B, S, T) order: the switch T -> S
// folded into the epilogue (outer = T, inner = S; outer = 0: no swap).
struct RowSwap {
  uint32_t outer = 0, inner = 0;
  __host__ __device__ int64_t map(int m) const {
    if (outer == 0) return m;
    const uint32_t per = outer * inner, r = (uint32_t)m % per;
    return (int64_t)((uint32_t)m - r) + (int64_t)(r % inner) * outer + r / inner;
  }
};

// dx = dres (if not null) + the LayerNorm backward of dy at x (layernorm.hip).
// x, dy and dres are read at row r, dx (and dx2, a second copy in fp32 or
// bf16, if not null) written at row rs.map(r); with a swap, dres may not
// alias an output.
int launch_layernorm_bwd(const void* x, int x_bf16, const void* dy, int dy_bf16, const float* dres, float* dx,
                         int64_t rows, int C, float eps, hipStream_t s, RowSwap rs = RowSwap(),
                         void* dx2 = nullptr, int dx2_bf16 = 0);

// out = epilogue(a W^T + bias) (gemm.hip).  pre (GELU or ReLU epilogue only,
// else null): also receives the pre-activation, in the output's dtype.  rs:
// output rows permuted as above (the residual is read in the input's order).
int launch_linear_bf16(const void* a, const void* w, const void* bias, const float* residual,
                       void* out, int64_t M, int N, int K, int epilogue, hipStream_t s, void* pre = nullptr,
                       RowSwap rs = RowSwap());
// Internal epilogues of launch_linear_bf16 (not in the public header): the
// backward of an activation, out = (a W^T) * act'(u), u the saved
// pre-activation passed as `pre` (read, at the output's offsets; no row swap).
constexpr int DSP_EPI_GELU_BWD = 5, DSP_EPI_RELU_BWD = 6;
// DSP_EPI_GELU_KEEP_GRAD: GELU whose `pre` receives GELU'(v), the derivative
// at the fp32 pre-activation v (rounded to the output dtype), instead of v.
// DSP_EPI_SCALE_BWD: the backward through such a kept derivative,
// out = (a W^T) * f with f read from `pre`.  Together they turn the
// activation's backward epilogue into one multiply.
constexpr int DSP_EPI_GELU_KEEP_GRAD = 7, DSP_EPI_SCALE_BWD = 8;
// Whether launch_linear_bf16 runs (M, N) on its large-tile kernel.
bool linear_bf16_large_tiles(int64_t M, int N);
// y_i[c][r] = x_i[r][c] for n <= 6 bf16 matrices of rows_i x cols_i (multiples
// of 8, 16-byte aligned), in one launch (gemm.hip).
int launch_transpose_bf16_batch(const void* const* x, void* const* y, const int64_t* rows, const int64_t* cols,
                                int n, hipStream_t s);
int launch_linear_f32(const float* a, const float* w, const float* bias, const float* residual,
                      float* out, int64_t M, int N, int K, int epilogue, hipStream_t s, float* pre = nullptr,
                      RowSwap rs = RowSwap());

// One attention sublayer of the fp32 projection-only chain in one kernel
// (chain_f32.hip), for groups of L <= 64 rows and C <= 64:
//   y[rs.map(g L + r)] = (Attn(x[g L + r] Wqkv^T + bqkv)) Wo^T + bo
// per group g (the heads' softmax attention over the group's rows); y may
// alias x.  fits() tells whether the shape is in range.
bool chain_sublayer_f32_fits(int64_t L, int C, int H);
int launch_chain_sublayer_f32(const float* x, const float* wqkv, const float* bqkv, const float* wo, const float* bo,
                              float* y, int64_t groups, int L, int C, int H, float scale, RowSwap rs, hipStream_t s);

inline int hip_status(hipError_t e) { return e == hipSuccess ? DSP_OK : DSP_ERR_HIP; }
inline int last_launch_status() { return hip_status(hipGetLastError()); }

}  // namespace dsp
