// C ABI of libdsp: host-side argument validation and launches on the caller's
// stream.  Every entry point validates all of its arguments before it enqueues
// anything, so a nonzero status means nothing was launched (except
// DSP_ERR_HIP from a launch, or from a later step of the block composite).
#include <math.h>
#include <string.h>

#include <mutex>
#include <utility>

#include "dsp_internal.h"

using namespace dsp;

namespace {

constexpr int kVersion = 1 * 10000 + 0 * 100 + 0;

bool valid_dtype(int dt) { return dt == DSP_F32 || dt == DSP_BF16; }
int elem_size(int dt) { return dt == DSP_F32 ? 4 : 2; }
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return na && nb && pa < pb + nb && pb < pa + na;
}

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

// Sequence tensors [B, S_1, .., S_K, C] with K = 2 or 3: checks ndim and the
// sizes, and returns the element count (via *elems) and the row strides of
// dims 0..K (row = C elements).
int seq_shape(const int64_t* shape, int ndim, int64_t* elems, int64_t* row_st) {
  if (!shape) return DSP_ERR_NULL;
  if (ndim != 4 && ndim != 5) return DSP_ERR_DIM;
  for (int k = 0; k < ndim; ++k)
    if (shape[k] < 0) return DSP_ERR_SHAPE;
  const int K = ndim - 2;
  int64_t rows = 1;
  row_st[K] = 1;
  for (int k = K; k >= 0; --k) {
    if (!mul_ok(rows, shape[k], &rows)) return DSP_ERR_SHAPE;
    if (k > 0) row_st[k - 1] = rows;
  }
  if (!mul_ok(rows, shape[K + 1], elems)) return DSP_ERR_SHAPE;
  return DSP_OK;
}

// Fills d with dense destination strides for its sizes.
void dense_dst(RowCopyDesc* d) {
  d->dst_stride[d->nd - 1] = 1;
  for (int i = d->nd - 2; i >= 0; --i) d->dst_stride[i] = d->dst_stride[i + 1] * d->size[i + 1];
}

// One GPU's Switch for K = 3 as a row copy: output rows enumerated
// (n, b, the other sequence dims in order with the to-dim sliced, from-dim).
int switch_k3(const void* x, void* y, const int64_t* shape, const int64_t* row_st, int from, int to,
              int64_t n_chunks, int64_t es, hipStream_t s) {
  const int K = 3;
  RowCopyDesc d = {};
  if (from == to) {
    d.nd = 1;
    d.size[0] = row_st[0] * shape[0];
    d.src_stride[0] = 1;
  } else {
    const int64_t per = shape[to] / n_chunks;
    d.size[d.nd] = n_chunks;  d.src_stride[d.nd++] = per * row_st[to];
    d.size[d.nd] = shape[0];  d.src_stride[d.nd++] = row_st[0];
    for (int k = 1; k <= K; ++k) {
      if (k == from) continue;
      d.size[d.nd] = k == to ? per : shape[k];
      d.src_stride[d.nd++] = row_st[k];
    }
    d.size[d.nd] = shape[from];
    d.src_stride[d.nd++] = row_st[from];
  }
  dense_dst(&d);
  d.row_bytes = shape[K + 1] * es;
  return launch_rowcopy(&x, &y, 1, d, s);
}

int switch_impl(const void* x, void* y, const int64_t* shape, int ndim, int from_dim, int to_dim,
                int n_chunks, int dtype, int variant, void* stream) {
  if (!shape) return DSP_ERR_NULL;
  if (ndim != 4 && ndim != 5) return DSP_ERR_DIM;
  if (from_dim < 1 || from_dim > ndim - 2 || to_dim < 1 || to_dim > ndim - 2) return DSP_ERR_DIM;
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (variant < 0 || variant > 2 || (ndim == 5 && variant != 0)) return DSP_ERR_ARG;
  if (ndim == 5) {
    int64_t elems, row_st[4];
    int st = seq_shape(shape, ndim, &elems, row_st);
    if (st != DSP_OK) return st;
    if (n_chunks < 1 || (from_dim != to_dim && shape[to_dim] % n_chunks)) return DSP_ERR_SHAPE;
    if (elems > INT64_MAX / 4) return DSP_ERR_SHAPE;
    const int64_t bytes = elems * elem_size(dtype);
    if (bytes == 0) return DSP_OK;
    if (!x || !y) return DSP_ERR_NULL;
    if (overlap(x, (size_t)bytes, y, (size_t)bytes)) return DSP_ERR_ARG;
    return switch_k3(x, y, shape, row_st, from_dim, to_dim, n_chunks, elem_size(dtype),
                     as_stream(stream));
  }
  const int64_t B = shape[0], D1 = shape[1], D2 = shape[2], C = shape[3];
  if (B < 0 || D1 < 0 || D2 < 0 || C < 0 || n_chunks < 1) return DSP_ERR_SHAPE;
  const int64_t d_to = to_dim == 2 ? D2 : D1;
  if (from_dim != to_dim && d_to % n_chunks != 0) return DSP_ERR_SHAPE;
  int64_t rows, elems, bytes;
  if (!mul_ok(B, D1, &rows) || !mul_ok(rows, D2, &rows) || !mul_ok(rows, C, &elems) ||
      !mul_ok(elems, elem_size(dtype), &bytes))
    return DSP_ERR_SHAPE;
  if (bytes == 0) return DSP_OK;  // empty: NULL pointers allowed, nothing launched
  if (!x || !y) return DSP_ERR_NULL;
  if (overlap(x, (size_t)bytes, y, (size_t)bytes)) return DSP_ERR_ARG;
  const int64_t row_bytes = C * elem_size(dtype);
  const bool rows_ok = row_bytes % 16 == 0 && aligned(x, 16) && aligned(y, 16);
  if (variant == 1 && !rows_ok) return DSP_ERR_ALIGN;
  const bool use_rows = variant == 1 || (variant == 0 && rows_ok && row_bytes >= 64);
  hipStream_t s = as_stream(stream);
  if (use_rows) return launch_switch_rows(x, y, B, D1, D2, row_bytes, from_dim, to_dim, n_chunks, s);
  return launch_switch_tiles(x, y, B, D1, D2, C, elem_size(dtype), from_dim, to_dim, n_chunks, s);
}

// Rows of a (B, X, L) grid with element strides st = {b, x, l}, each `width`
// elements wide, do not overlap when, taking the dimensions of extent > 1 by
// increasing stride, every stride is at least the span of the smaller ones.
bool rows_disjoint(int64_t B, int64_t X, int64_t L, const int64_t* st, int64_t width) {
  int64_t e[3] = {B, X, L}, s[3] = {st[0], st[1], st[2]};
  for (int i = 0; i < 3; ++i)
    for (int j = i + 1; j < 3; ++j)
      if (s[j] < s[i]) { std::swap(s[i], s[j]); std::swap(e[i], e[j]); }
  int64_t span = width;
  for (int i = 0; i < 3; ++i) {
    if (e[i] <= 1) continue;
    if (s[i] < span) return false;
    if (!mul_ok(s[i], e[i] - 1, &span) || span > INT64_MAX - width) return false;
    span += width;
  }
  return true;
}

// Attention over general layouts: queries (B, X, Lq) of H heads with q_st,
// keys/values (B, X, Lk) of Hkv heads with kv_st, output with o_st.
int attn_general_impl(const void* q, const void* k, const void* v, void* o, float* lse, int64_t B,
                      int64_t X, int64_t Lq, int64_t Lk, int H, int Hkv, int D, const int64_t* q_st,
                      const int64_t* kv_st, const int64_t* o_st, float scale, int dtype, void* stream) {
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (!q_st || !kv_st || !o_st) return DSP_ERR_NULL;
  if (B < 0 || X < 0 || Lq < 0 || Lk < 0 || H < 1 || D < 1 || Hkv < 1 || H % Hkv) return DSP_ERR_SHAPE;
  const bool empty = B == 0 || X == 0 || Lq == 0;
  if (!empty && Lk == 0) return DSP_ERR_SHAPE;  // a softmax over no keys
  if ((!q || !k || !v || !o) && !empty) return DSP_ERR_NULL;
  for (int i = 0; i < 3; ++i)
    if (q_st[i] < 0 || kv_st[i] < 0 || o_st[i] < 0) return DSP_ERR_SHAPE;
  if (isnan(scale) || isinf(scale)) return DSP_ERR_ARG;
  if (lse && !aligned(lse, 4)) return DSP_ERR_ALIGN;
  int64_t width;
  if (!mul_ok(H, D, &width)) return DSP_ERR_SHAPE;
  if (dtype == DSP_BF16) {
    if (!attn_bf16_supports(D)) return DSP_ERR_SHAPE;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16)) return DSP_ERR_ALIGN;
    for (int i = 0; i < 3; ++i)
      if (q_st[i] % 8 || kv_st[i] % 8 || o_st[i] % 8) return DSP_ERR_ALIGN;
  } else if (D > 256) {
    return DSP_ERR_SHAPE;
  }
  if (empty) return DSP_OK;
  // every output row is written by exactly one unit
  if (!rows_disjoint(B, X, Lq, o_st, width)) return DSP_ERR_ARG;
  // the largest element offset of each side must be addressable
  const int64_t* sts[3] = {q_st, kv_st, o_st};
  const int64_t lens[3] = {Lq, Lk, Lq};
  for (int i = 0; i < 3; ++i) {
    int64_t tb, tx, tl;
    if (!mul_ok(B - 1, sts[i][0], &tb) || !mul_ok(X - 1, sts[i][1], &tx) || !mul_ok(lens[i] - 1, sts[i][2], &tl) ||
        tb > INT64_MAX / 4 || tx > INT64_MAX / 4 || tl > INT64_MAX / 4)
      return DSP_ERR_SHAPE;
  }
  AttnArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.B = B; a.X = X; a.L = Lq; a.H = H; a.D = D;
  a.b_stride_in = q_st[0];
  a.x_stride_in = q_st[1];
  a.r_stride_in = q_st[2];
  a.b_stride_out = o_st[0];
  a.x_stride_out = o_st[1];
  a.r_stride_out = o_st[2];
  a.Lk = Lk;
  a.Hkv = Hkv;
  a.b_stride_kv = kv_st[0];
  a.x_stride_kv = kv_st[1];
  a.r_stride_kv = kv_st[2];
  a.scale = scale > 0.0f ? scale : (float)(1.0 / sqrt((double)D));
  a.lse = lse;
  hipStream_t s = as_stream(stream);
  return dtype == DSP_BF16 ? launch_attn_bf16(a, s) : launch_attn_f32(a, s);
}

int attn_impl_strided(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t X,
                      int64_t L, int H, int D, const int64_t* in_st, const int64_t* out_st,
                      float scale, int dtype, void* stream, float* lse = nullptr) {
  return attn_general_impl(q, k, v, o, lse, B, X, L, L, H, H, D, in_st, in_st, out_st, scale, dtype, stream);
}

// The largest element offset of a (B, X, L) grid of rows with strides st is
// addressable (each term well inside int64).
bool offsets_ok(int64_t B, int64_t X, int64_t L, const int64_t* st) {
  int64_t tb, tx, tl;
  return mul_ok(B - 1, st[0], &tb) && mul_ok(X - 1, st[1], &tx) && mul_ok(L - 1, st[2], &tl) &&
         tb <= INT64_MAX / 4 && tx <= INT64_MAX / 4 && tl <= INT64_MAX / 4;
}

int attn_bwd_general_impl(const void* q, const void* k, const void* v, const void* o, const void* dout,
                          const float* lse, void* dq, void* dk, void* dv, float* delta, int64_t B, int64_t X,
                          int64_t Lq, int64_t Lk, int H, int Hkv, int D, const int64_t* q_st,
                          const int64_t* kv_st, const int64_t* o_st, float scale, int dtype, void* stream) {
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (!q_st || !kv_st || !o_st) return DSP_ERR_NULL;
  if (B < 0 || X < 0 || Lq < 0 || Lk < 0 || H < 1 || D < 1 || Hkv < 1 || H % Hkv) return DSP_ERR_SHAPE;
  const bool empty = B == 0 || X == 0 || (Lq == 0 && Lk == 0);
  if (!empty && (Lq == 0) != (Lk == 0)) return DSP_ERR_SHAPE;  // queries without keys, or keys without queries
  if (!empty && (!q || !k || !v || !o || !dout || !lse || !dq || !dk || !dv || !delta))
    return DSP_ERR_NULL;
  for (int i = 0; i < 3; ++i)
    if (q_st[i] < 0 || kv_st[i] < 0 || o_st[i] < 0) return DSP_ERR_SHAPE;
  if (isnan(scale) || isinf(scale)) return DSP_ERR_ARG;
  int64_t width, kv_width, units, stat_elems;
  if (!mul_ok(H, D, &width) || !mul_ok(Hkv, D, &kv_width) || !mul_ok(B, X, &units) || !mul_ok(units, H, &units) ||
      !mul_ok(units, Lq, &stat_elems))
    return DSP_ERR_SHAPE;
  if (dtype == DSP_BF16) {
    if (!attn_bf16_supports(D) || D % 32 > 16) return DSP_ERR_SHAPE;
    for (const void* ptr : {q, k, v, o, dout, (const void*)dq, (const void*)dk, (const void*)dv})
      if (!aligned(ptr, 16)) return DSP_ERR_ALIGN;
    for (int i = 0; i < 3; ++i)
      if (q_st[i] % 8 || kv_st[i] % 8 || o_st[i] % 8) return DSP_ERR_ALIGN;
  } else if (D > 256) {
    return DSP_ERR_SHAPE;
  }
  if (!aligned(lse, 4) || !aligned(delta, 4)) return DSP_ERR_ALIGN;
  if (empty) return DSP_OK;
  // every gradient row is written by exactly one (unit, position): key/value
  // rows shared by several units (a broadcast layout) have no single owner
  if (!rows_disjoint(B, X, Lq, q_st, width) || !rows_disjoint(B, X, Lk, kv_st, kv_width)) return DSP_ERR_ARG;
  if (!offsets_ok(B, X, Lq, q_st) || !offsets_ok(B, X, Lk, kv_st) || !offsets_ok(B, X, Lq, o_st))
    return DSP_ERR_SHAPE;
  if (stat_elems > INT64_MAX / 8) return DSP_ERR_SHAPE;
  if (overlap(delta, (size_t)stat_elems * 4, lse, (size_t)stat_elems * 4)) return DSP_ERR_ARG;
  AttnBwdArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.dout = dout; a.lse = lse;
  a.dq = dq; a.dk = dk; a.dv = dv; a.delta = delta;
  a.B = B; a.X = X; a.L = Lq; a.Lk = Lk; a.H = H; a.Hkv = Hkv; a.D = D;
  for (int i = 0; i < 3; ++i) {
    a.q_strides[i] = q_st[i];
    a.kv_strides[i] = kv_st[i];
    a.o_strides[i] = o_st[i];
  }
  a.scale = scale > 0.0f ? scale : (float)(1.0 / sqrt((double)D));
  hipStream_t s = as_stream(stream);
  if (dtype == DSP_BF16) {
    if (!attn_bwd_bf16_fits(a)) return DSP_ERR_SHAPE;
    return launch_attn_bwd_bf16(a, s);
  }
  return launch_attn_bwd_f32(a, s);
}

int attn_bwd_impl(const void* q, const void* k, const void* v, const void* o, const void* dout,
                  const float* lse, void* dq, void* dk, void* dv, float* delta, int64_t B, int64_t X,
                  int64_t L, int H, int D, const int64_t* qkv_st, const int64_t* o_st, float scale,
                  int dtype, void* stream) {
  return attn_bwd_general_impl(q, k, v, o, dout, lse, dq, dk, dv, delta, B, X, L, L, H, H, D, qkv_st, qkv_st, o_st,
                               scale, dtype, stream);
}

// Spatial (B,T,S,*): unit (b, t), positions s.  Temporal (B,S,T,*): unit
// (b, s), positions t.  Both: position r of unit (b, x) is row (b*X + x)*L + r.
int attn_impl(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t X, int64_t L,
              int H, int D, int64_t ld_in, int64_t ld_out, float scale, int dtype, void* stream) {
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (B < 0 || X < 0 || L < 0 || H < 1 || D < 1) return DSP_ERR_SHAPE;
  if ((int64_t)H * D > ld_in || (int64_t)H * D > ld_out) return DSP_ERR_SHAPE;
  int64_t tokens, xl_in, xl_out, bl_in, bl_out;
  if (!mul_ok(B, X, &tokens) || !mul_ok(tokens, L, &tokens)) return DSP_ERR_SHAPE;
  int64_t span_in, span_out;
  if (!mul_ok(tokens, ld_in, &span_in) || !mul_ok(tokens, ld_out, &span_out)) return DSP_ERR_SHAPE;
  if (!mul_ok(L, ld_in, &xl_in) || !mul_ok(L, ld_out, &xl_out) || !mul_ok(X, xl_in, &bl_in) ||
      !mul_ok(X, xl_out, &bl_out))
    return DSP_ERR_SHAPE;
  const int64_t in_st[3] = {bl_in, xl_in, ld_in}, out_st[3] = {bl_out, xl_out, ld_out};
  return attn_impl_strided(q, k, v, o, B, X, L, H, D, in_st, out_st, scale, dtype, stream);
}

// pre (GELU/ReLU epilogue, may be null): also receives the pre-activation.
// rs (optional): the output rows permuted from (B, T, S) to (B, S, T) token order
// (the switch T -> S in the epilogue); the residual is read in the input's order,
// so out must not alias it.
int linear_impl(const void* a, const void* w, const void* bias, const float* residual, void* out,
                int64_t M, int N, int K, int epilogue, int dtype, hipStream_t s, void* pre = nullptr,
                RowSwap rs = RowSwap()) {
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (M < 0 || N < 1 || K < 1) return DSP_ERR_SHAPE;
  if (rs.outer && (rs.inner == 0 || M % ((int64_t)rs.outer * rs.inner) || residual == out)) return DSP_ERR_ARG;
  // the public epilogues, and (bf16 only, with `pre`) GELU keeping its derivative
  const bool keep_grad = epilogue == DSP_EPI_GELU_KEEP_GRAD;
  if ((epilogue < DSP_EPI_NONE || epilogue > DSP_EPI_RELU) && !keep_grad) return DSP_ERR_ARG;
  if (keep_grad && (dtype != DSP_BF16 || !pre)) return DSP_ERR_ARG;
  if (!w) return DSP_ERR_NULL;
  if (M == 0) return DSP_OK;
  if (!a || !out) return DSP_ERR_NULL;
  if (epilogue == DSP_EPI_RESID && !residual) return DSP_ERR_NULL;
  int64_t mk, mn;
  if (!mul_ok(M, K, &mk) || !mul_ok(M, N, &mn)) return DSP_ERR_SHAPE;
  const int es = elem_size(dtype);
  const int out_es = (epilogue == DSP_EPI_RESID || epilogue == DSP_EPI_F32) ? 4 : es;
  const size_t out_bytes = (size_t)mn * out_es;
  if (overlap(out, out_bytes, a, (size_t)mk * es) || overlap(out, out_bytes, w, (size_t)N * K * es) ||
      (bias && overlap(out, out_bytes, bias, (size_t)N * es)))
    return DSP_ERR_ARG;
  if (residual && epilogue == DSP_EPI_RESID && residual != out &&
      overlap(out, out_bytes, residual, (size_t)mn * 4))
    return DSP_ERR_ARG;
  if (pre && ((epilogue != DSP_EPI_GELU && epilogue != DSP_EPI_RELU && !keep_grad) ||
              overlap(pre, out_bytes, out, out_bytes) ||
              overlap(pre, out_bytes, a, (size_t)mk * es)))
    return DSP_ERR_ARG;
  if (dtype == DSP_BF16) {
    if (K % 8 || !aligned(a, 16) || !aligned(w, 16) || !aligned(out, 16)) return DSP_ERR_ALIGN;
    if (epilogue == DSP_EPI_RESID && !aligned(residual, 16)) return DSP_ERR_ALIGN;
    if (pre && !aligned(pre, 16)) return DSP_ERR_ALIGN;
    return launch_linear_bf16(a, w, bias, epilogue == DSP_EPI_RESID ? residual : nullptr, out, M, N,
                              K, epilogue, s, pre, rs);
  }
  return launch_linear_f32(static_cast<const float*>(a), static_cast<const float*>(w),
                           static_cast<const float*>(bias),
                           epilogue == DSP_EPI_RESID ? residual : nullptr,
                           static_cast<float*>(out), M, N, K, epilogue, s, static_cast<float*>(pre), rs);
}

// Workspace regions of the block (each 256-byte aligned).
struct BlockWs {
  size_t h, qkv, o, f, x1, total;
};

bool block_ws_layout(int64_t B, int64_t T, int64_t S, int C, int F, int dtype, BlockWs* ws) {
  int64_t tokens;
  if (!mul_ok(B, T, &tokens) || !mul_ok(tokens, S, &tokens)) return false;
  const int es = elem_size(dtype);
  auto up = [](size_t v) { return (v + 255) & ~size_t(255); };
  int64_t tc, t3c, tf;
  if (!mul_ok(tokens, C, &tc) || !mul_ok(tokens, 3 * (int64_t)C, &t3c) || !mul_ok(tokens, F, &tf))
    return false;
  size_t off = 0;
  ws->h = off;   off += up((size_t)tc * es);
  ws->qkv = off; off += up((size_t)t3c * es);
  ws->o = off;   off += up((size_t)tc * es);
  ws->f = off;   off += up((size_t)tf * es);
  ws->x1 = off;  off += up((size_t)tc * 4);
  ws->total = off;
  return true;
}

// Activations a training forward keeps for the backward (offsets into the
// caller's `saved` buffer, each 256-byte aligned).  Residual streams in fp32,
// operands in the block dtype, log-sum-exps in fp32 ([units][L] = tokens * H).
// Pre-LN: y0 and y1 hold the streams entering the temporal half and the MLP
// (the inputs of their LayerNorms).  Post-LN: y0 and y1 hold the sums r1
// (switched to (B, S, T, C)) and r2 that the first two LayerNorms normalise,
// and r3, the sum the MLP's LayerNorm normalises, gets a slot of its own.
// u is what the MLP activation's backward needs: the pre-activation, or with
// GELU in bf16 at sizes whose backward runs on the large-tile GEMM, GELU' at
// the fp32 pre-activation (block_keeps_act_grad), so that the backward's
// epilogue is one multiply instead of the derivative's evaluation.
struct BlockSaved {
  size_t y0, y1, h1, qkv1, a1, lse1, h2, qkv2, a2, lse2, h3, u, g, r3, total;
};

bool block_keeps_act_grad(int64_t tokens, int F, int dtype, int flags) {
  return dtype == DSP_BF16 && !(flags & DSP_BLOCK_RELU) && linear_bf16_large_tiles(tokens, F);
}

bool block_saved_layout(int64_t B, int64_t T, int64_t S, int C, int H, int F, int flags, int dtype,
                        BlockSaved* sv) {
  int64_t tokens, tc, t3c, tf, th;
  if (!mul_ok(B, T, &tokens) || !mul_ok(tokens, S, &tokens) || !mul_ok(tokens, C, &tc) ||
      !mul_ok(tokens, 3 * (int64_t)C, &t3c) || !mul_ok(tokens, F, &tf) || !mul_ok(tokens, H, &th))
    return false;
  if (tc > INT64_MAX / 64 || tf > INT64_MAX / 64) return false;
  const size_t es = elem_size(dtype);
  auto up = [](size_t v) { return (v + 255) & ~size_t(255); };
  size_t off = 0;
  sv->y0 = off;   off += up((size_t)tc * 4);
  sv->y1 = off;   off += up((size_t)tc * 4);
  sv->h1 = off;   off += up((size_t)tc * es);
  sv->qkv1 = off; off += up((size_t)t3c * es);
  sv->a1 = off;   off += up((size_t)tc * es);
  sv->lse1 = off; off += up((size_t)th * 4);
  sv->h2 = off;   off += up((size_t)tc * es);
  sv->qkv2 = off; off += up((size_t)t3c * es);
  sv->a2 = off;   off += up((size_t)tc * es);
  sv->lse2 = off; off += up((size_t)th * 4);
  sv->h3 = off;   off += up((size_t)tc * es);
  sv->u = off;    off += up((size_t)tf * es);
  sv->g = off;    off += up((size_t)tf * es);
  sv->r3 = off;
  if ((flags & DSP_BLOCK_POST_LN) && !(flags & DSP_BLOCK_NO_MLP_LN)) off += up((size_t)tc * 4);
  sv->total = off;
  return true;
}

// Scratch of the block backward.
struct BlockBwdWs {
  size_t dyb, du, dh, dcur, dx1, da, dqkv, delta, wg, wg_bytes, wt, total;
};

bool block_bwd_ws_layout(int64_t B, int64_t T, int64_t S, int C, int H, int F, int dtype, BlockBwdWs* ws) {
  int64_t tokens, tc, t3c, tf, th;
  if (!mul_ok(B, T, &tokens) || !mul_ok(tokens, S, &tokens) || !mul_ok(tokens, C, &tc) ||
      !mul_ok(tokens, 3 * (int64_t)C, &t3c) || !mul_ok(tokens, F, &tf) || !mul_ok(tokens, H, &th))
    return false;
  if (tc > INT64_MAX / 64 || tf > INT64_MAX / 64) return false;
  const size_t es = elem_size(dtype);
  auto up = [](size_t v) { return (v + 255) & ~size_t(255); };
  size_t wg = 0;
  const int64_t shapes[4][2] = {{3 * (int64_t)C, C}, {C, C}, {F, C}, {C, F}};
  for (const auto& nk : shapes)
    wg = std::max(wg, dsp_linear_bwd_weight_workspace_bytes(tokens, (int)nk[0], (int)nk[1], dtype));
  size_t off = 0;
  ws->dyb = off;   off += up((size_t)tc * es);
  ws->du = off;    off += up((size_t)tf * es);
  ws->dh = off;    off += up((size_t)tc * 4);
  ws->dcur = off;  off += up((size_t)tc * 4);
  ws->dx1 = off;   off += up((size_t)tc * 4);
  ws->da = off;    off += up((size_t)tc * es);
  ws->dqkv = off;  off += up((size_t)t3c * es);
  ws->delta = off; off += up((size_t)th * 4);
  ws->wg = off;    off += up(wg);
  ws->wg_bytes = wg;
  // bf16: the six weight matrices transposed, for the input gradients on the
  // forward's GEMM
  ws->wt = off;
  if (dtype == DSP_BF16)
    off += 2 * up((size_t)3 * C * C * es) + 2 * up((size_t)C * C * es) + 2 * up((size_t)F * C * es);
  ws->total = off;
  return true;
}

// ---- dsp_attn_bwd_noalloc: the attention backward with its Delta rows in a
// library-owned device array instead of a caller workspace.  Each device holds
// its own copy of `scratch` (loaded with the code object, kept until the
// process ends); host code must never pass the array's name to a kernel or a
// copy (in host code it is a host-side stand-in), only the device address
// hipGetSymbolAddress returns for the device that is current.
constexpr int64_t kNoallocDeltaRows = int64_t(1) << 22;  // fp32 Delta values: 16 MiB
__device__ __align__(256) float scratch[kNoallocDeltaRows];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the device the stream belongs to, looked
// up once per device with that device current; nullptr if HIP fails.
float* noalloc_scratch(hipStream_t s) {
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) return nullptr;
  int dev = cur;
  if (s && hipStreamGetDevice(s, &dev) != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return nullptr;
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (dev != cur && hipSetDevice(cur) != hipSuccess) return nullptr;
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();  // leave no error behind for the next launch check
      return nullptr;
    }
    g_scratch_ptr[dev] = static_cast<float*>(ptr);
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

const char* dsp_status_str(int status) {
  switch (status) {
    case DSP_OK: return "DSP_OK";
    case DSP_ERR_NULL: return "DSP_ERR_NULL: a required pointer is NULL";
    case DSP_ERR_DIM: return "DSP_ERR_DIM: bad ndim or dimension index";
    case DSP_ERR_SHAPE: return "DSP_ERR_SHAPE: invalid or unsupported size";
    case DSP_ERR_DTYPE: return "DSP_ERR_DTYPE: unknown or unsupported dtype";
    case DSP_ERR_ALIGN: return "DSP_ERR_ALIGN: pointer or stride alignment not met";
    case DSP_ERR_HIP: return "DSP_ERR_HIP: HIP runtime or launch failure";
    case DSP_ERR_WORKSPACE: return "DSP_ERR_WORKSPACE: workspace missing or too small";
    case DSP_ERR_ARG: return "DSP_ERR_ARG: invalid argument";
    default: return "unknown dsp status";
  }
}

int dsp_version(void) { return kVersion; }

int dsp_switch(const void* x, void* y, const int64_t* shape, int ndim, int from_dim, int to_dim,
               int n_chunks, int dtype, void* stream) {
  return switch_impl(x, y, shape, ndim, from_dim, to_dim, n_chunks, dtype, 0, stream);
}

int dsp_switch_variant(const void* x, void* y, const int64_t* shape, int ndim, int from_dim,
                       int to_dim, int n_chunks, int dtype, int variant, void* stream) {
  return switch_impl(x, y, shape, ndim, from_dim, to_dim, n_chunks, dtype, variant, stream);
}

int dsp_exchange_unpack(const void* const* packed, void* const* out, const int64_t* shape,
                        int dtype, void* stream) {
  if (!shape) return DSP_ERR_NULL;
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  const int64_t N = shape[0], B = shape[1], P = shape[2], F = shape[3], C = shape[4];
  if (N < 1 || N > kMaxExchangeRanks || B < 0 || P < 0 || F < 0 || C < 0) return DSP_ERR_SHAPE;
  int64_t run, per_rank, run_bytes;
  if (!mul_ok(F, C, &run) || !mul_ok(run, elem_size(dtype), &run_bytes) ||
      !mul_ok(N, B, &per_rank) || !mul_ok(per_rank, P, &per_rank) ||
      !mul_ok(per_rank, run_bytes, &per_rank))
    return DSP_ERR_SHAPE;
  if (per_rank == 0) return DSP_OK;
  if (!packed || !out) return DSP_ERR_NULL;
  for (int64_t i = 0; i < N; ++i)
    if (!packed[i] || !out[i]) return DSP_ERR_NULL;
  // every destination is written by N sources: it must not overlap a source or
  // another destination (sources may alias each other: they are only read)
  for (int64_t i = 0; i < N; ++i) {
    for (int64_t j = 0; j < N; ++j) {
      if (overlap(out[i], (size_t)per_rank, packed[j], (size_t)per_rank)) return DSP_ERR_ARG;
      if (j != i && overlap(out[i], (size_t)per_rank, out[j], (size_t)per_rank)) return DSP_ERR_ARG;
    }
  }
  return launch_exchange_unpack(packed, out, N, B, P, run_bytes, static_cast<hipStream_t>(stream));
}

int dsp_split(const void* x, void* y, const int64_t* shape, int ndim, int dim, int n_chunks,
              int rank, int dtype, void* stream) {
  int64_t elems, row_st[4];
  if (!shape) return DSP_ERR_NULL;
  int st = seq_shape(shape, ndim, &elems, row_st);
  if (st != DSP_OK) return st;
  if (dim < 1 || dim > ndim - 2) return DSP_ERR_DIM;
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (n_chunks < 1 || shape[dim] % n_chunks) return DSP_ERR_SHAPE;
  if (rank < 0 || rank >= n_chunks) return DSP_ERR_ARG;
  if (elems > INT64_MAX / 4) return DSP_ERR_SHAPE;
  const int64_t es = elem_size(dtype), in_bytes = elems * es, out_bytes = in_bytes / n_chunks;
  if (out_bytes == 0) return DSP_OK;
  if (!x || !y) return DSP_ERR_NULL;
  if (overlap(x, (size_t)in_bytes, y, (size_t)out_bytes)) return DSP_ERR_ARG;
  const int K = ndim - 2;
  const int64_t per = shape[dim] / n_chunks;
  RowCopyDesc d = {};
  for (int k = 0; k <= K; ++k) {
    d.size[d.nd] = k == dim ? per : shape[k];
    d.src_stride[d.nd++] = row_st[k];
  }
  dense_dst(&d);
  d.row_bytes = shape[K + 1] * es;
  const void* src = static_cast<const char*>(x) + rank * per * row_st[dim] * d.row_bytes;
  return launch_rowcopy(&src, &y, 1, d, as_stream(stream));
}

int dsp_gather(const void* const* shards, void* y, const int64_t* shard_shape, int ndim, int dim,
               int n_shards, int dtype, void* stream) {
  int64_t elems, row_st[4];
  if (!shard_shape) return DSP_ERR_NULL;
  int st = seq_shape(shard_shape, ndim, &elems, row_st);
  if (st != DSP_OK) return st;
  if (dim < 1 || dim > ndim - 2) return DSP_ERR_DIM;
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (n_shards < 1 || n_shards > kMaxCopyPairs) return DSP_ERR_SHAPE;
  int64_t out_elems;
  if (!mul_ok(elems, n_shards, &out_elems) || out_elems > INT64_MAX / 4) return DSP_ERR_SHAPE;
  const int64_t es = elem_size(dtype), shard_bytes = elems * es, out_bytes = out_elems * es;
  if (out_bytes == 0) return DSP_OK;
  if (!shards || !y) return DSP_ERR_NULL;
  for (int m = 0; m < n_shards; ++m) {
    if (!shards[m]) return DSP_ERR_NULL;
    if (overlap(shards[m], (size_t)shard_bytes, y, (size_t)out_bytes)) return DSP_ERR_ARG;
  }
  // destination row strides: the shard's with dim grown n_shards times
  const int K = ndim - 2;
  int64_t out_st[4];
  out_st[K] = 1;
  for (int k = K - 1; k >= 0; --k) out_st[k] = out_st[k + 1] * shard_shape[k + 1] * (k + 1 == dim ? n_shards : 1);
  RowCopyDesc d = {};
  for (int k = 0; k <= K; ++k) {
    d.size[d.nd] = shard_shape[k];
    d.src_stride[d.nd] = row_st[k];
    d.dst_stride[d.nd++] = out_st[k];
  }
  d.row_bytes = shard_shape[K + 1] * es;
  void* dst[kMaxCopyPairs];
  for (int m = 0; m < n_shards; ++m)
    dst[m] = static_cast<char*>(y) + m * shard_shape[dim] * out_st[dim] * d.row_bytes;
  return launch_rowcopy(shards, dst, n_shards, d, as_stream(stream));
}

int dsp_spatial_attn(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t T,
                     int64_t S, int H, int D, int64_t ld_in, int64_t ld_out, float scale,
                     int dtype, void* stream) {
  return attn_impl(q, k, v, o, B, T, S, H, D, ld_in, ld_out, scale, dtype, stream);
}

int dsp_temporal_attn(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t S,
                      int64_t T, int H, int D, int64_t ld_in, int64_t ld_out, float scale,
                      int dtype, void* stream) {
  return attn_impl(q, k, v, o, B, S, T, H, D, ld_in, ld_out, scale, dtype, stream);
}

int dsp_attn_strided(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t X,
                     int64_t L, int H, int D, const int64_t* in_strides, const int64_t* out_strides,
                     float scale, int dtype, void* stream) {
  return attn_impl_strided(q, k, v, o, B, X, L, H, D, in_strides, out_strides, scale, dtype, stream);
}

int dsp_attn_fwd_lse(const void* q, const void* k, const void* v, void* o, float* lse, int64_t B,
                     int64_t X, int64_t L, int H, int D, const int64_t* in_strides,
                     const int64_t* out_strides, float scale, int dtype, void* stream) {
  if (B > 0 && X > 0 && L > 0 && !lse) return DSP_ERR_NULL;
  if (lse && !aligned(lse, 4)) return DSP_ERR_ALIGN;
  return attn_impl_strided(q, k, v, o, B, X, L, H, D, in_strides, out_strides, scale, dtype, stream,
                           lse);
}

int dsp_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                 const float* lse, void* dq, void* dk, void* dv, float* delta, int64_t B, int64_t X,
                 int64_t L, int H, int D, const int64_t* qkv_strides, const int64_t* o_strides,
                 float scale, int dtype, void* stream) {
  return attn_bwd_impl(q, k, v, o, dout, lse, dq, dk, dv, delta, B, X, L, H, D, qkv_strides, o_strides,
                       scale, dtype, stream);
}

int64_t dsp_attn_bwd_noalloc_max_rows(void) { return kNoallocDeltaRows; }

int dsp_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dout,
                         const float* lse, void* dq, void* dk, void* dv, int64_t B, int64_t X, int64_t L, int H,
                         int D, const int64_t* qkv_strides, const int64_t* o_strides, float scale, int dtype,
                         void* stream) {
  int64_t rows;
  if (B < 0 || X < 0 || L < 0 || H < 1 || !mul_ok(B, X, &rows) || !mul_ok(rows, H, &rows) ||
      !mul_ok(rows, L, &rows))
    return DSP_ERR_SHAPE;
  if (rows > kNoallocDeltaRows) return DSP_ERR_WORKSPACE;
  if (rows == 0)  // nothing to compute: validate without touching the device
    return attn_bwd_impl(q, k, v, o, dout, lse, dq, dk, dv, nullptr, B, X, L, H, D, qkv_strides, o_strides,
                         scale, dtype, stream);
  float* delta = noalloc_scratch(as_stream(stream));
  if (!delta) return DSP_ERR_HIP;
  return attn_bwd_impl(q, k, v, o, dout, lse, dq, dk, dv, delta, B, X, L, H, D, qkv_strides, o_strides, scale,
                       dtype, stream);
}

int dsp_attn_general(const void* q, const void* k, const void* v, void* o, float* lse, int64_t B, int64_t X,
                     int64_t Lq, int64_t Lk, int H, int Hkv, int D, const int64_t* q_strides,
                     const int64_t* kv_strides, const int64_t* o_strides, float scale, int dtype, void* stream) {
  return attn_general_impl(q, k, v, o, lse, B, X, Lq, Lk, H, Hkv, D, q_strides, kv_strides, o_strides, scale, dtype,
                           stream);
}

int dsp_attn_general_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                         const float* lse, void* dq, void* dk, void* dv, float* delta, int64_t B, int64_t X,
                         int64_t Lq, int64_t Lk, int H, int Hkv, int D, const int64_t* q_strides,
                         const int64_t* kv_strides, const int64_t* o_strides, float scale, int dtype,
                         void* stream) {
  return attn_bwd_general_impl(q, k, v, o, dout, lse, dq, dk, dv, delta, B, X, Lq, Lk, H, Hkv, D, q_strides,
                               kv_strides, o_strides, scale, dtype, stream);
}

int dsp_linear_bwd_data(const void* dy, const void* w, const void* u, void* dx, int64_t M, int N, int K,
                        int epilogue, int dtype, void* stream) {
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (M < 0 || N < 1 || K < 1) return DSP_ERR_SHAPE;
  if (epilogue < DSP_GRAD_EPI_F32 || epilogue > DSP_GRAD_EPI_RELU_BWD) return DSP_ERR_ARG;
  const bool act = epilogue == DSP_GRAD_EPI_GELU_BWD || epilogue == DSP_GRAD_EPI_RELU_BWD;
  if (!w) return DSP_ERR_NULL;
  if (M == 0) return DSP_OK;
  if (!dy || !dx || (act && !u)) return DSP_ERR_NULL;
  int64_t mn, mk, nk;
  if (!mul_ok(M, N, &mn) || !mul_ok(M, K, &mk) || !mul_ok(N, K, &nk)) return DSP_ERR_SHAPE;
  const int es = elem_size(dtype);
  const size_t out_bytes = (size_t)mk * (epilogue == DSP_GRAD_EPI_F32 ? 4 : es);
  if (overlap(dx, out_bytes, dy, (size_t)mn * es) || overlap(dx, out_bytes, w, (size_t)nk * es) ||
      (act && overlap(dx, out_bytes, u, (size_t)mk * es)))
    return DSP_ERR_ARG;
  hipStream_t s = as_stream(stream);
  if (dtype == DSP_BF16) {
    if (N % 8 || K % 8) return DSP_ERR_ALIGN;
    for (const void* ptr : {dy, w, (const void*)dx, act ? u : w})
      if (!aligned(ptr, 16)) return DSP_ERR_ALIGN;
    if (!grad_gemm_fits(M, K, N, N, K)) return DSP_ERR_SHAPE;
    // dx[m][k] = sum_n dy[m][n] W[n][k]: A = dy as stored, B(k, n) = W[n][k] transposed
    return launch_gemm_grad(dy, 0, N, w, 1, K, act ? u : nullptr, dx, M, K, N, epilogue, 1, nullptr, s);
  }
  if (epilogue == DSP_GRAD_EPI_BF16) return DSP_ERR_ARG;  // fp32 path: fp32 output only
  return launch_gemm_grad_f32(static_cast<const float*>(dy), 0, N, static_cast<const float*>(w), 1, K,
                              static_cast<const float*>(act ? u : nullptr), static_cast<float*>(dx), M, K, N,
                              epilogue, s);
}

size_t dsp_linear_bwd_weight_workspace_bytes(int64_t M, int N, int K, int dtype) {
  if (dtype != DSP_BF16 || M <= 0 || N < 1 || K < 1) return 0;
  const int splits = grad_splits(N, K, M);
  return splits > 1 ? (size_t)splits * (size_t)N * (size_t)K * 4 : 0;
}

int dsp_linear_bwd_weight(const void* dy, const void* x, float* dw, float* db, void* workspace,
                          size_t ws_bytes, int64_t M, int N, int K, int dtype, void* stream) {
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (M < 0 || N < 1 || K < 1) return DSP_ERR_SHAPE;
  if (!dw || (M > 0 && (!dy || !x))) return DSP_ERR_NULL;
  int64_t mn, mk, nk;
  if (!mul_ok(M, N, &mn) || !mul_ok(M, K, &mk) || !mul_ok(N, K, &nk)) return DSP_ERR_SHAPE;
  const int es = elem_size(dtype);
  if (overlap(dw, (size_t)nk * 4, dy, (size_t)mn * es) || overlap(dw, (size_t)nk * 4, x, (size_t)mk * es) ||
      (db && (overlap(db, (size_t)N * 4, dy, (size_t)mn * es) || overlap(db, (size_t)N * 4, dw, (size_t)nk * 4))))
    return DSP_ERR_ARG;
  if (!aligned(dw, 16) || (db && !aligned(db, 16))) return DSP_ERR_ALIGN;
  hipStream_t s = as_stream(stream);
  if (dtype == DSP_BF16) {
    if (N % 8 || K % 8) return DSP_ERR_ALIGN;
    if ((M > 0 && (!aligned(dy, 16) || !aligned(x, 16)))) return DSP_ERR_ALIGN;
    if (!grad_gemm_fits(N, K, M, N, K)) return DSP_ERR_SHAPE;
    const size_t need = dsp_linear_bwd_weight_workspace_bytes(M, N, K, dtype);
    if (need && (!workspace || ws_bytes < need || !aligned(workspace, 16))) return DSP_ERR_WORKSPACE;
    if (need && (overlap(workspace, need, dw, (size_t)nk * 4) || overlap(workspace, need, dy, (size_t)mn * es) ||
                 overlap(workspace, need, x, (size_t)mk * es)))
      return DSP_ERR_ARG;
    // dw[n][k] = sum_m dy[m][n] x[m][k]: A(n, m) = dy[m][n] and B(k, m) = x[m][k], both transposed
    const int splits = need ? grad_splits(N, K, M) : 1;
    int st = launch_gemm_grad(dy, 1, N, x, 1, K, nullptr, dw, N, K, M, DSP_GRAD_EPI_F32, splits,
                              static_cast<float*>(workspace), s);
    if (st != DSP_OK || !db) return st;
    return launch_colsum_bf16(dy, db, M, N, s);
  }
  int st = launch_gemm_grad_f32(static_cast<const float*>(dy), 1, N, static_cast<const float*>(x), 1, K, nullptr,
                                dw, N, K, M, DSP_GRAD_EPI_F32, s);
  if (st != DSP_OK || !db) return st;
  return launch_colsum_f32(static_cast<const float*>(dy), db, M, N, s);
}

int dsp_layernorm_bwd(const void* x, int x_dtype, const void* dy, int dy_dtype, const float* dres, float* dx,
                      int64_t rows, int C, float eps, void* stream) {
  if (!valid_dtype(x_dtype) || !valid_dtype(dy_dtype)) return DSP_ERR_DTYPE;
  if (rows < 0 || C < 1) return DSP_ERR_SHAPE;
  if (!(eps >= 0.0f) || isinf(eps)) return DSP_ERR_ARG;
  if (rows == 0) return DSP_OK;
  if (!x || !dy || !dx) return DSP_ERR_NULL;
  int64_t n;
  if (!mul_ok(rows, C, &n) || n > INT64_MAX / 8) return DSP_ERR_SHAPE;
  const size_t out = (size_t)n * 4;
  if (overlap(dx, out, x, (size_t)n * elem_size(x_dtype)) || overlap(dx, out, dy, (size_t)n * elem_size(dy_dtype)))
    return DSP_ERR_ARG;
  if (dres && dres != dx && overlap(dx, out, dres, out)) return DSP_ERR_ARG;
  return launch_layernorm_bwd(x, x_dtype == DSP_BF16, dy, dy_dtype == DSP_BF16, dres, dx, rows, C, eps,
                              as_stream(stream));
}

int dsp_layernorm(const void* x, int x_dtype, void* y, int y_dtype, int64_t rows, int C, float eps,
                  void* stream) {
  if (!valid_dtype(x_dtype) || !valid_dtype(y_dtype)) return DSP_ERR_DTYPE;
  if (rows < 0 || C < 1) return DSP_ERR_SHAPE;
  if (rows == 0) return DSP_OK;
  if (!x || !y) return DSP_ERR_NULL;
  if (!(eps >= 0.0f) || isinf(eps)) return DSP_ERR_ARG;
  int64_t n;
  if (!mul_ok(rows, C, &n)) return DSP_ERR_SHAPE;
  if (overlap(x, (size_t)n * elem_size(x_dtype), y, (size_t)n * elem_size(y_dtype))) return DSP_ERR_ARG;
  return launch_layernorm(x, x_dtype == DSP_BF16, y, y_dtype == DSP_BF16, rows, C, eps,
                          as_stream(stream));
}

int dsp_linear(const void* a, const void* w, const void* bias, const float* residual, void* out,
               int64_t M, int N, int K, int epilogue, int dtype, void* stream) {
  if (epilogue < DSP_EPI_NONE || epilogue > DSP_EPI_RELU) return DSP_ERR_ARG;
  return linear_impl(a, w, bias, residual, out, M, N, K, epilogue, dtype, as_stream(stream));
}

size_t dsp_st_block_workspace_bytes(int64_t B, int64_t T, int64_t S, int C, int H, int F,
                                    int dtype) {
  if (!valid_dtype(dtype) || B < 0 || T < 0 || S < 0 || C < 1 || H < 1 || F < 0 || C % H)
    return 0;
  BlockWs ws;
  if (!block_ws_layout(B, T, S, C, F, dtype, &ws)) return 0;
  return ws.total;
}

int dsp_st_block_forward(const float* x_BTSC, float* y_BSTC, const dsp_block_weights_t* w,
                         void* workspace, size_t ws_bytes, int64_t B, int64_t T, int64_t S, int C,
                         int H, int F, float ln_eps, int flags, int dtype, void* stream) {
  if (!x_BTSC || !y_BSTC || !w) return DSP_ERR_NULL;
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  if (flags & ~(DSP_BLOCK_NO_MLP_LN | DSP_BLOCK_ATTN_ONLY | DSP_BLOCK_POST_LN | DSP_BLOCK_RELU))
    return DSP_ERR_ARG;
  const bool attn_only = (flags & DSP_BLOCK_ATTN_ONLY) != 0;
  if (B < 0 || T < 0 || S < 0 || C < 1 || H < 1 || C % H || F < 0) return DSP_ERR_SHAPE;
  if (!attn_only && F < 1) return DSP_ERR_SHAPE;
  const int D = C / H;
  if (dtype == DSP_BF16 && (!attn_bf16_supports(D) || C % 8 || F % 8)) return DSP_ERR_SHAPE;
  if (!(ln_eps >= 0.0f) || isinf(ln_eps)) return DSP_ERR_ARG;
  if (!w->wqkv_s || !w->wo_s || !w->wqkv_t || !w->wo_t) return DSP_ERR_NULL;
  if (!attn_only && (!w->w1 || !w->w2)) return DSP_ERR_NULL;
  BlockWs ws;
  if (!block_ws_layout(B, T, S, C, F, dtype, &ws)) return DSP_ERR_SHAPE;
  if (!workspace || ws_bytes < ws.total) return DSP_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return DSP_ERR_ALIGN;
  const int64_t tokens = B * T * S;
  const size_t act_bytes = (size_t)tokens * C * 4;
  if (overlap(x_BTSC, act_bytes, y_BSTC, act_bytes) ||
      overlap(x_BTSC, act_bytes, workspace, ws_bytes) ||
      overlap(y_BSTC, act_bytes, workspace, ws_bytes))
    return DSP_ERR_ARG;
  if (dtype == DSP_BF16) {
    const void* ws_[] = {w->wqkv_s, w->wo_s, w->wqkv_t, w->wo_t, w->w1, w->w2};
    for (const void* p : ws_)
      if (p && !aligned(p, 16)) return DSP_ERR_ALIGN;
    if (!aligned(x_BTSC, 16) || !aligned(y_BSTC, 16)) return DSP_ERR_ALIGN;
  }
  if (tokens == 0) return DSP_OK;

  hipStream_t s = as_stream(stream);
  char* base = static_cast<char*>(workspace);
  void* h = base + ws.h;
  void* qkv = base + ws.qkv;
  void* o = base + ws.o;
  void* f = base + ws.f;
  float* x1 = reinterpret_cast<float*>(base + ws.x1);
  const int bf = dtype == DSP_BF16;
  const int es = elem_size(dtype);
  const int64_t ld3 = 3 * (int64_t)C;
  char* qkvc = static_cast<char*>(qkv);
  int st;
#define DSP_TRY(expr)            \
  do {                           \
    st = (expr);                 \
    if (st != DSP_OK) return st; \
  } while (0)

  const bool post = (flags & DSP_BLOCK_POST_LN) != 0 && !attn_only;
  const int act = (flags & DSP_BLOCK_RELU) ? DSP_EPI_RELU : DSP_EPI_GELU;
  RowSwap swap;  // (B, T, S) token rows -> (B, S, T)
  swap.outer = (uint32_t)T;
  swap.inner = (uint32_t)S;
  // the bf16 (or fp32) operand of a projection: LN of the residual stream, or
  // (post-LN, projection-only chain) the stream itself
  // (fp32 without LN: the stream itself, no copy)
  const void* hin = h;
  auto operand = [&](const float* r, bool norm) {
    hin = h;
    if (norm) return launch_layernorm(r, 0, h, bf, tokens, C, ln_eps, s);
    if (!bf) {
      hin = r;
      return (int)DSP_OK;
    }
    return launch_cast(r, 0, h, bf, tokens * C, s);
  };
  auto attn_sublayer = [&](const void* wqkv, const void* bqkv, int64_t X, int64_t L) {
    int r = linear_impl(hin, wqkv, bqkv, nullptr, qkv, tokens, 3 * C, C, DSP_EPI_NONE, dtype, s);
    if (r != DSP_OK) return r;
    return attn_impl(qkvc, qkvc + (size_t)C * es, qkvc + (size_t)2 * C * es, o, B, X, L, H, D, ld3, C,
                     0.0f, dtype, s);
  };
  if (attn_only) {
    // y = Wo_t * TemporalAttn(Switch(Wo_s * SpatialAttn(x * Wqkv_s)) * Wqkv_t)
    if (!bf && chain_sublayer_f32_fits(S, C, H) && chain_sublayer_f32_fits(T, C, H) && aligned(x_BTSC, 16) &&
        aligned(y_BSTC, 16) && aligned(w->wqkv_s, 16) && aligned(w->wo_s, 16) && aligned(w->wqkv_t, 16) &&
        aligned(w->wo_t, 16)) {
      // small fp32 shapes: each sublayer in one kernel (one work-group per frame,
      // then per location); the spatial one writes its rows in (B, S, T) order
      const float scl = (float)(1.0 / sqrt((double)D));
      DSP_TRY(launch_chain_sublayer_f32(x_BTSC, static_cast<const float*>(w->wqkv_s),
                                        static_cast<const float*>(w->bqkv_s), static_cast<const float*>(w->wo_s),
                                        static_cast<const float*>(w->bo_s), y_BSTC, B * T, (int)S, C, H, scl, swap, s));
      DSP_TRY(launch_chain_sublayer_f32(y_BSTC, static_cast<const float*>(w->wqkv_t),
                                        static_cast<const float*>(w->bqkv_t), static_cast<const float*>(w->wo_t),
                                        static_cast<const float*>(w->bo_t), y_BSTC, B * S, (int)T, C, H, scl,
                                        RowSwap(), s));
      return DSP_OK;
    }
    DSP_TRY(operand(x_BTSC, false));
    DSP_TRY(attn_sublayer(w->wqkv_s, w->bqkv_s, T, S));
    // the Switch T -> S folded into the out-projection's epilogue (rows written in (B, S, T) order)
    DSP_TRY(linear_impl(o, w->wo_s, w->bo_s, nullptr, y_BSTC, tokens, C, C, DSP_EPI_F32, dtype, s, nullptr, swap));
    DSP_TRY(operand(y_BSTC, false));
    DSP_TRY(attn_sublayer(w->wqkv_t, w->bqkv_t, S, T));
    DSP_TRY(linear_impl(o, w->wo_t, w->bo_t, nullptr, y_BSTC, tokens, C, C, DSP_EPI_F32, dtype, s));
    return DSP_OK;
  }
  if (!post) {
    // pre-LN: x += F(LN(x)) for each sublayer
    // ---- spatial half on (B, T, S, C): attention over S inside each frame
    DSP_TRY(operand(x_BTSC, true));
    DSP_TRY(attn_sublayer(w->wqkv_s, w->bqkv_s, T, S));
    // ---- the Switch T -> S on one GPU, (B, T, S, C) -> (B, S, T, C), folded into the
    // out-projection's epilogue: row (b, t, s) of x + o Wo is written at (b, s, t)
    DSP_TRY(linear_impl(o, w->wo_s, w->bo_s, x_BTSC, y_BSTC, tokens, C, C, DSP_EPI_RESID, dtype, s, nullptr,
                        swap));
    // ---- temporal half on (B, S, T, C): attention over T at each location
    DSP_TRY(operand(y_BSTC, true));
    DSP_TRY(attn_sublayer(w->wqkv_t, w->bqkv_t, S, T));
    DSP_TRY(linear_impl(o, w->wo_t, w->bo_t, y_BSTC, y_BSTC, tokens, C, C, DSP_EPI_RESID, dtype, s));
    // ---- MLP (Eq. 5 with GELU or ReLU), residual
    DSP_TRY(operand(y_BSTC, !(flags & DSP_BLOCK_NO_MLP_LN)));
    DSP_TRY(linear_impl(hin, w->w1, w->b1, nullptr, f, tokens, F, C, act, dtype, s));
    DSP_TRY(linear_impl(f, w->w2, w->b2, y_BSTC, y_BSTC, tokens, C, F, DSP_EPI_RESID, dtype, s));
    return DSP_OK;
  }
  // post-LN (Eq. 4, 6): x = LN(x + F(x)) for each sublayer.  The residual
  // stream alternates between x1 and y_BSTC (LN is never run in place).
  DSP_TRY(operand(x_BTSC, false));
  DSP_TRY(attn_sublayer(w->wqkv_s, w->bqkv_s, T, S));
  // switch first (in the out-projection's epilogue), then LN: LN acts per token,
  // so LN(Switch(v)) = Switch(LN(v))
  DSP_TRY(linear_impl(o, w->wo_s, w->bo_s, x_BTSC, y_BSTC, tokens, C, C, DSP_EPI_RESID, dtype, s, nullptr, swap));
  DSP_TRY(launch_layernorm(y_BSTC, 0, x1, 0, tokens, C, ln_eps, s));           // x1 = r1 (B,S,T,C)
  DSP_TRY(operand(x1, false));
  DSP_TRY(attn_sublayer(w->wqkv_t, w->bqkv_t, S, T));
  DSP_TRY(linear_impl(o, w->wo_t, w->bo_t, x1, y_BSTC, tokens, C, C, DSP_EPI_RESID, dtype, s));
  DSP_TRY(launch_layernorm(y_BSTC, 0, x1, 0, tokens, C, ln_eps, s));           // x1 = r2
  DSP_TRY(operand(x1, false));
  DSP_TRY(linear_impl(hin, w->w1, w->b1, nullptr, f, tokens, F, C, act, dtype, s));
  if (flags & DSP_BLOCK_NO_MLP_LN) {
    DSP_TRY(linear_impl(f, w->w2, w->b2, x1, y_BSTC, tokens, C, F, DSP_EPI_RESID, dtype, s));
    return DSP_OK;
  }
  DSP_TRY(linear_impl(f, w->w2, w->b2, x1, x1, tokens, C, F, DSP_EPI_RESID, dtype, s));
  DSP_TRY(launch_layernorm(x1, 0, y_BSTC, 0, tokens, C, ln_eps, s));
  return DSP_OK;
#undef DSP_TRY
}

size_t dsp_st_block_train_saved_bytes(int64_t B, int64_t T, int64_t S, int C, int H, int F, int flags,
                                      int dtype) {
  if (!valid_dtype(dtype) || B < 0 || T < 0 || S < 0 || C < 1 || H < 1 || F < 1 || C % H) return 0;
  BlockSaved sv;
  return block_saved_layout(B, T, S, C, H, F, flags, dtype, &sv) ? sv.total : 0;
}

size_t dsp_st_block_backward_workspace_bytes(int64_t B, int64_t T, int64_t S, int C, int H, int F, int dtype) {
  if (!valid_dtype(dtype) || B < 0 || T < 0 || S < 0 || C < 1 || H < 1 || F < 1 || C % H) return 0;
  BlockBwdWs ws;
  return block_bwd_ws_layout(B, T, S, C, H, F, dtype, &ws) ? ws.total : 0;
}

namespace {

// Checks shared by the training forward and the backward.
int block_train_check(const dsp_block_weights_t* w, int64_t B, int64_t T, int64_t S, int C, int H, int F,
                      float ln_eps, int flags, int dtype) {
  if (!w) return DSP_ERR_NULL;
  if (!valid_dtype(dtype)) return DSP_ERR_DTYPE;
  // training covers the pre- and post-LN blocks (GELU or ReLU, with or
  // without the MLP's LN); the projection-only chain has no training path
  if (flags & ~(DSP_BLOCK_NO_MLP_LN | DSP_BLOCK_POST_LN | DSP_BLOCK_RELU)) return DSP_ERR_ARG;
  if (B < 0 || T < 0 || S < 0 || C < 1 || H < 1 || C % H || F < 1) return DSP_ERR_SHAPE;
  const int D = C / H;
  if (dtype == DSP_BF16 && (!attn_bf16_supports(D) || D % 32 > 16 || C % 8 || F % 8)) return DSP_ERR_SHAPE;
  if (!(ln_eps >= 0.0f) || isinf(ln_eps)) return DSP_ERR_ARG;
  if (!w->wqkv_s || !w->wo_s || !w->wqkv_t || !w->wo_t || !w->w1 || !w->w2) return DSP_ERR_NULL;
  if (dtype == DSP_BF16) {
    const void* all[] = {w->wqkv_s, w->bqkv_s, w->wo_s, w->bo_s, w->wqkv_t, w->bqkv_t,
                         w->wo_t, w->bo_t, w->w1, w->b1, w->w2, w->b2};
    for (const void* p : all)
      if (p && !aligned(p, 16)) return DSP_ERR_ALIGN;
  }
  return DSP_OK;
}

}  // namespace

int dsp_st_block_forward_train(const float* x_BTSC, float* y_BSTC, const dsp_block_weights_t* w, void* saved,
                               size_t saved_bytes, int64_t B, int64_t T, int64_t S, int C, int H, int F,
                               float ln_eps, int flags, int dtype, void* stream) {
  int st = block_train_check(w, B, T, S, C, H, F, ln_eps, flags, dtype);
  if (st != DSP_OK) return st;
  if (!x_BTSC || !y_BSTC) return DSP_ERR_NULL;
  BlockSaved sv;
  if (!block_saved_layout(B, T, S, C, H, F, flags, dtype, &sv)) return DSP_ERR_SHAPE;
  if (!saved || saved_bytes < sv.total) return DSP_ERR_WORKSPACE;
  if (!aligned(saved, 256)) return DSP_ERR_ALIGN;
  if (!aligned(x_BTSC, 16) || !aligned(y_BSTC, 16)) return DSP_ERR_ALIGN;
  const int64_t tokens = B * T * S;
  const size_t act_bytes = (size_t)tokens * C * 4;
  if (overlap(x_BTSC, act_bytes, y_BSTC, act_bytes) || overlap(x_BTSC, act_bytes, saved, saved_bytes) ||
      overlap(y_BSTC, act_bytes, saved, saved_bytes))
    return DSP_ERR_ARG;
  if (tokens == 0) return DSP_OK;
  hipStream_t s = as_stream(stream);
  char* base = static_cast<char*>(saved);
  float* y0 = reinterpret_cast<float*>(base + sv.y0);
  float* y1 = reinterpret_cast<float*>(base + sv.y1);
  char *h1 = base + sv.h1, *qkv1 = base + sv.qkv1, *a1 = base + sv.a1, *h2 = base + sv.h2, *qkv2 = base + sv.qkv2,
       *a2 = base + sv.a2, *h3 = base + sv.h3, *u = base + sv.u, *g = base + sv.g;
  float* lse1 = reinterpret_cast<float*>(base + sv.lse1);
  float* lse2 = reinterpret_cast<float*>(base + sv.lse2);
  const int bf = dtype == DSP_BF16;
  const size_t es = elem_size(dtype);
  const int D = C / H;
  const int act = (flags & DSP_BLOCK_RELU) ? DSP_EPI_RELU : DSP_EPI_GELU;
  // what the MLP's first GEMM keeps in `u` (see block_keeps_act_grad)
  const int act_keep = block_keeps_act_grad(tokens, F, dtype, flags) ? DSP_EPI_GELU_KEEP_GRAD : act;
  RowSwap swap;  // (B, T, S) token rows -> (B, S, T)
  swap.outer = (uint32_t)T;
  swap.inner = (uint32_t)S;
#define DSP_TRY(expr)            \
  do {                           \
    st = (expr);                 \
    if (st != DSP_OK) return st; \
  } while (0)
  // an attention sublayer's projection and attention over L, positions of
  // unit (b, x) at rows (b X + x) L + l, saving q/k/v, the output and lse
  auto attn_sub = [&](const void* h, const void* wqkv, const void* bqkv, char* qkv, char* a, float* lse,
                      int64_t X, int64_t L) {
    int r = linear_impl(h, wqkv, bqkv, nullptr, qkv, tokens, 3 * C, C, DSP_EPI_NONE, dtype, s);
    if (r != DSP_OK) return r;
    const int64_t in_st[3] = {X * L * 3 * C, L * 3 * C, 3 * (int64_t)C}, out_st[3] = {X * L * C, L * C, C};
    return attn_impl_strided(qkv, qkv + (size_t)C * es, qkv + (size_t)2 * C * es, a, B, X, L, H, D, in_st, out_st,
                             0.0f, dtype, stream, lse);
  };
  if (flags & DSP_BLOCK_POST_LN) {
    // post-LN (Eq. 4, 6): each sublayer reads the stream itself and LN follows
    // the residual add.  y_BSTC holds the fp32 streams y0 and y1 until the
    // output is written; the ops are those of dsp_st_block_forward, in its order.
    float* r3 = reinterpret_cast<float*>(base + sv.r3);
    DSP_TRY(launch_cast(x_BTSC, 0, h1, bf, tokens * C, s));
    DSP_TRY(attn_sub(h1, w->wqkv_s, w->bqkv_s, qkv1, a1, lse1, T, S));
    DSP_TRY(linear_impl(a1, w->wo_s, w->bo_s, x_BTSC, y0, tokens, C, C, DSP_EPI_RESID, dtype, s, nullptr,
                        swap));                                                  // y0 slot: r1 (B,S,T,C)
    DSP_TRY(launch_layernorm(y0, 0, y_BSTC, 0, tokens, C, ln_eps, s));           // stream y0 = LN(r1)
    DSP_TRY(launch_cast(y_BSTC, 0, h2, bf, tokens * C, s));
    DSP_TRY(attn_sub(h2, w->wqkv_t, w->bqkv_t, qkv2, a2, lse2, S, T));
    DSP_TRY(linear_impl(a2, w->wo_t, w->bo_t, y_BSTC, y1, tokens, C, C, DSP_EPI_RESID, dtype, s));  // r2
    DSP_TRY(launch_layernorm(y1, 0, y_BSTC, 0, tokens, C, ln_eps, s));           // stream y1 = LN(r2)
    DSP_TRY(launch_cast(y_BSTC, 0, h3, bf, tokens * C, s));
    DSP_TRY(linear_impl(h3, w->w1, w->b1, nullptr, g, tokens, F, C, act_keep, dtype, s, u));
    if (flags & DSP_BLOCK_NO_MLP_LN) {
      DSP_TRY(linear_impl(g, w->w2, w->b2, y_BSTC, y_BSTC, tokens, C, F, DSP_EPI_RESID, dtype, s));
    } else {
      DSP_TRY(linear_impl(g, w->w2, w->b2, y_BSTC, r3, tokens, C, F, DSP_EPI_RESID, dtype, s));
      DSP_TRY(launch_layernorm(r3, 0, y_BSTC, 0, tokens, C, ln_eps, s));
    }
    return DSP_OK;
  }
  // spatial half on (B, T, S, C); y1's slot holds the pre-switch stream x1
  DSP_TRY(launch_layernorm(x_BTSC, 0, h1, bf, tokens, C, ln_eps, s));
  DSP_TRY(attn_sub(h1, w->wqkv_s, w->bqkv_s, qkv1, a1, lse1, T, S));
  // the Switch T -> S in the out-projection's epilogue: y0 = Switch(x + a1 Wo_s)
  DSP_TRY(linear_impl(a1, w->wo_s, w->bo_s, x_BTSC, y0, tokens, C, C, DSP_EPI_RESID, dtype, s, nullptr, swap));
  // temporal half on (B, S, T, C)
  DSP_TRY(launch_layernorm(y0, 0, h2, bf, tokens, C, ln_eps, s));
  DSP_TRY(attn_sub(h2, w->wqkv_t, w->bqkv_t, qkv2, a2, lse2, S, T));
  DSP_TRY(linear_impl(a2, w->wo_t, w->bo_t, y0, y1, tokens, C, C, DSP_EPI_RESID, dtype, s));
  // MLP: u = h3 W1 + b1 and g = act(u) from one GEMM (both kept; g from the
  // fp32 sum, as in the forward), y = y1 + g W2 + b2
  if (flags & DSP_BLOCK_NO_MLP_LN) {
    DSP_TRY(launch_cast(y1, 0, h3, bf, tokens * C, s));
  } else {
    DSP_TRY(launch_layernorm(y1, 0, h3, bf, tokens, C, ln_eps, s));
  }
  DSP_TRY(linear_impl(h3, w->w1, w->b1, nullptr, g, tokens, F, C, act_keep, dtype, s, u));
  DSP_TRY(linear_impl(g, w->w2, w->b2, y1, y_BSTC, tokens, C, F, DSP_EPI_RESID, dtype, s));
  return DSP_OK;
#undef DSP_TRY
}

int dsp_st_block_backward(const float* x_BTSC, const float* dy_BSTC, const dsp_block_weights_t* w,
                          const void* saved, size_t saved_bytes, void* workspace, size_t ws_bytes, float* dx_BTSC,
                          const dsp_block_grads_t* grads, int64_t B, int64_t T, int64_t S, int C, int H, int F,
                          float ln_eps, int flags, int dtype, void* stream) {
  int st = block_train_check(w, B, T, S, C, H, F, ln_eps, flags, dtype);
  if (st != DSP_OK) return st;
  if (!x_BTSC || !dy_BSTC || !dx_BTSC || !grads) return DSP_ERR_NULL;
  if (!grads->wqkv_s || !grads->wo_s || !grads->wqkv_t || !grads->wo_t || !grads->w1 || !grads->w2)
    return DSP_ERR_NULL;
  BlockSaved sv;
  BlockBwdWs bw;
  if (!block_saved_layout(B, T, S, C, H, F, flags, dtype, &sv) ||
      !block_bwd_ws_layout(B, T, S, C, H, F, dtype, &bw))
    return DSP_ERR_SHAPE;
  if (!saved || saved_bytes < sv.total || !workspace || ws_bytes < bw.total) return DSP_ERR_WORKSPACE;
  if (!aligned(saved, 256) || !aligned(workspace, 256)) return DSP_ERR_ALIGN;
  const float* gp[] = {grads->wqkv_s, grads->bqkv_s, grads->wo_s, grads->bo_s, grads->wqkv_t, grads->bqkv_t,
                       grads->wo_t, grads->bo_t, grads->w1, grads->b1, grads->w2, grads->b2};
  for (const float* p : gp)
    if (p && !aligned(p, 16)) return DSP_ERR_ALIGN;
  if (!aligned(x_BTSC, 16) || !aligned(dy_BSTC, 16) || !aligned(dx_BTSC, 16)) return DSP_ERR_ALIGN;
  const int64_t tokens = B * T * S;
  const size_t act_bytes = (size_t)tokens * C * 4;
  if (overlap(dx_BTSC, act_bytes, x_BTSC, act_bytes) || overlap(dx_BTSC, act_bytes, dy_BSTC, act_bytes) ||
      overlap(dx_BTSC, act_bytes, saved, saved_bytes) || overlap(dx_BTSC, act_bytes, workspace, ws_bytes) ||
      overlap(workspace, ws_bytes, saved, saved_bytes))
    return DSP_ERR_ARG;
  if (tokens == 0) return DSP_OK;
  hipStream_t s = as_stream(stream);
  const char* sb = static_cast<const char*>(saved);
  const float* y0 = reinterpret_cast<const float*>(sb + sv.y0);
  const float* y1 = reinterpret_cast<const float*>(sb + sv.y1);
  const char *h1 = sb + sv.h1, *qkv1 = sb + sv.qkv1, *a1 = sb + sv.a1, *h2 = sb + sv.h2, *qkv2 = sb + sv.qkv2,
             *a2 = sb + sv.a2, *h3 = sb + sv.h3, *u = sb + sv.u, *g = sb + sv.g;
  const float* lse1 = reinterpret_cast<const float*>(sb + sv.lse1);
  const float* lse2 = reinterpret_cast<const float*>(sb + sv.lse2);
  char* wb = static_cast<char*>(workspace);
  char *dyb = wb + bw.dyb, *du = wb + bw.du, *da = wb + bw.da, *dqkv = wb + bw.dqkv;
  float* dh = reinterpret_cast<float*>(wb + bw.dh);
  float* dcur = reinterpret_cast<float*>(wb + bw.dcur);
  float* dx1 = reinterpret_cast<float*>(wb + bw.dx1);
  float* delta = reinterpret_cast<float*>(wb + bw.delta);
  void* wg = bw.wg_bytes ? wb + bw.wg : nullptr;
  void* wt = wb + bw.wt;
  const int bf = dtype == DSP_BF16;
  const size_t es = elem_size(dtype);
  const int D = C / H;
  const int act_epi = bf ? DSP_GRAD_EPI_BF16 : DSP_GRAD_EPI_F32;   // gradients fed to bf16 / fp32 operands
  const int act_bwd = (flags & DSP_BLOCK_RELU) ? DSP_GRAD_EPI_RELU_BWD : DSP_GRAD_EPI_GELU_BWD;
  const bool kept_grad = block_keeps_act_grad(tokens, F, dtype, flags);
  RowSwap back;  // (B, S, T) token rows -> (B, T, S): the Switch's adjoint
  back.outer = (uint32_t)S;
  back.inner = (uint32_t)T;
#define DSP_TRY(expr)            \
  do {                           \
    st = (expr);                 \
    if (st != DSP_OK) return st; \
  } while (0)
  // the upstream fp32 gradient as an operand of the block dtype
  auto operand = [&](const float* d) { return launch_cast(d, 0, dyb, bf, tokens * C, s); };
  // dx = dy W (+ the activation's derivative) for W stored [N][K]: in bf16 at
  // sizes the forward's large-tile GEMM takes, dx = dy (W^T)^T runs on that
  // GEMM with W^T from the workspace; else the gradient GEMM.  The weights
  // taking the large tiles are transposed first, all in one launch.
  struct Transposed {
    const void* w;
    int N, K;
    const void* wt;
  };
  Transposed tw[6];
  int n_tw = 0;
  if (bf) {
    const void* src[6] = {w->wqkv_s, w->wo_s, w->wqkv_t, w->wo_t, w->w1, w->w2};
    const int nk[6][2] = {{3 * C, C}, {C, C}, {3 * C, C}, {C, C}, {F, C}, {C, F}};
    const void* xs[6];
    void* ys[6];
    int64_t rows[6], cols[6];
    size_t off = 0;
    for (int i = 0; i < 6; ++i) {
      if (!linear_bf16_large_tiles(tokens, nk[i][1])) continue;
      void* dst = static_cast<char*>(wt) + off;
      off += ((size_t)nk[i][0] * nk[i][1] * es + 255) & ~size_t(255);
      tw[n_tw] = {src[i], nk[i][0], nk[i][1], dst};
      xs[n_tw] = src[i];
      ys[n_tw] = dst;
      rows[n_tw] = nk[i][0];
      cols[n_tw] = nk[i][1];
      ++n_tw;
    }
    if (n_tw) DSP_TRY(launch_transpose_bf16_batch(xs, ys, rows, cols, n_tw, s));
  }
  auto bwd_data = [&](const void* dyp, const void* wp, const void* up, void* dxp, int N, int K, int epi) -> int {
    if (bf && linear_bf16_large_tiles(tokens, K)) {
      const void* wtp = nullptr;
      for (int i = 0; i < n_tw; ++i)
        if (tw[i].w == wp && tw[i].N == N && tw[i].K == K) wtp = tw[i].wt;
      if (!wtp) return DSP_ERR_ARG;  // every large-tile weight was transposed above
      const int e = epi == DSP_GRAD_EPI_F32 ? DSP_EPI_F32
                    : epi == DSP_GRAD_EPI_BF16 ? DSP_EPI_NONE
                    : epi == DSP_GRAD_EPI_GELU_BWD ? (kept_grad ? DSP_EPI_SCALE_BWD : DSP_EPI_GELU_BWD)
                                                   : DSP_EPI_RELU_BWD;
      return launch_linear_bf16(dyp, wtp, nullptr, nullptr, dxp, tokens, K, N, e, s, const_cast<void*>(up));
    }
    return dsp_linear_bwd_data(dyp, wp, up, dxp, tokens, N, K, epi, dtype, stream);
  };
  // backward of one attention sublayer: d_out (in dyb) -> dh (fp32), weight gradients
  auto attn_sub_bwd = [&](const char* h, const char* qkv, const char* a, const float* lse, const void* wqkv,
                          const void* wo, float* g_wqkv, float* g_bqkv, float* g_wo, float* g_bo, int64_t X,
                          int64_t L) {
    int r = dsp_linear_bwd_weight(dyb, a, g_wo, g_bo, wg, bw.wg_bytes, tokens, C, C, dtype, stream);
    if (r != DSP_OK) return r;
    r = bwd_data(dyb, wo, nullptr, da, C, C, act_epi);
    if (r != DSP_OK) return r;
    const int64_t q_st[3] = {X * L * 3 * C, L * 3 * C, 3 * (int64_t)C}, o_st[3] = {X * L * C, L * C, C};
    r = attn_bwd_impl(qkv, qkv + (size_t)C * es, qkv + (size_t)2 * C * es, a, da, lse, dqkv, dqkv + (size_t)C * es,
                      dqkv + (size_t)2 * C * es, delta, B, X, L, H, D, q_st, o_st, 0.0f, dtype, stream);
    if (r != DSP_OK) return r;
    r = dsp_linear_bwd_weight(dqkv, h, g_wqkv, g_bqkv, wg, bw.wg_bytes, tokens, 3 * C, C, dtype, stream);
    if (r != DSP_OK) return r;
    return bwd_data(dqkv, wqkv, nullptr, dh, 3 * C, C, DSP_GRAD_EPI_F32);
  };
  if (flags & DSP_BLOCK_POST_LN) {
    // post-LN: the gradient passes each LayerNorm before its sublayer, and the
    // sublayer's input gradient adds to the stream's (the residual branch).
    const float* r1 = y0;   // (B, S, T, C)
    const float* r2 = y1;
    const float* dr3 = dy_BSTC;
    // ---- MLP: r3 = y1 + act(y1 W1 + b1) W2 + b2
    if (!(flags & DSP_BLOCK_NO_MLP_LN)) {
      DSP_TRY(launch_layernorm_bwd(sb + sv.r3, 0, dy_BSTC, 0, nullptr, dcur, tokens, C, ln_eps, s, RowSwap(),
                                   dyb, bf));
      dr3 = dcur;
    } else {
      DSP_TRY(operand(dr3));
    }
    DSP_TRY(dsp_linear_bwd_weight(dyb, g, grads->w2, grads->b2, wg, bw.wg_bytes, tokens, C, F, dtype, stream));
    DSP_TRY(bwd_data(dyb, w->w2, u, du, C, F, act_bwd));
    DSP_TRY(dsp_linear_bwd_weight(du, h3, grads->w1, grads->b1, wg, bw.wg_bytes, tokens, F, C, dtype, stream));
    DSP_TRY(bwd_data(du, w->w1, nullptr, dh, F, C, DSP_GRAD_EPI_F32));
    DSP_TRY(launch_add_f32(dr3, dh, dcur, tokens * C, s));                           // dy1
    // ---- temporal half: r2 = y0 + Attn_T(y0 Wqkv_t) Wo_t, y1 = LN(r2)
    DSP_TRY(launch_layernorm_bwd(r2, 0, dcur, 0, nullptr, dx1, tokens, C, ln_eps, s, RowSwap(), dyb, bf));  // dr2
    DSP_TRY(attn_sub_bwd(h2, qkv2, a2, lse2, w->wqkv_t, w->wo_t, grads->wqkv_t, grads->bqkv_t, grads->wo_t,
                         grads->bo_t, S, T));
    DSP_TRY(launch_add_f32(dx1, dh, dcur, tokens * C, s));                           // dy0
    // ---- spatial half: r1 = x + Attn_S(x Wqkv_s) Wo_s, y0 = LN(Switch(r1))
    // dr1, written back in (B, T, S, C) order (the Switch's adjoint) with its operand copy
    DSP_TRY(launch_layernorm_bwd(r1, 0, dcur, 0, nullptr, dx1, tokens, C, ln_eps, s, back, dyb, bf));
    DSP_TRY(attn_sub_bwd(h1, qkv1, a1, lse1, w->wqkv_s, w->wo_s, grads->wqkv_s, grads->bqkv_s, grads->wo_s,
                         grads->bo_s, T, S));
    DSP_TRY(launch_add_f32(dx1, dh, dx_BTSC, tokens * C, s));
    return DSP_OK;
  }
  // ---- MLP: y = y1 + act(h3 W1 + b1) W2 + b2
  DSP_TRY(operand(dy_BSTC));
  DSP_TRY(dsp_linear_bwd_weight(dyb, g, grads->w2, grads->b2, wg, bw.wg_bytes, tokens, C, F, dtype, stream));
  DSP_TRY(bwd_data(dyb, w->w2, u, du, C, F, act_bwd));
  DSP_TRY(dsp_linear_bwd_weight(du, h3, grads->w1, grads->b1, wg, bw.wg_bytes, tokens, F, C, dtype, stream));
  DSP_TRY(bwd_data(du, w->w1, nullptr, dh, F, C, DSP_GRAD_EPI_F32));
  if (flags & DSP_BLOCK_NO_MLP_LN) {
    DSP_TRY(launch_add_f32(dy_BSTC, dh, dcur, tokens * C, s));
    DSP_TRY(operand(dcur));
  } else {
    DSP_TRY(launch_layernorm_bwd(y1, 0, dh, 0, dy_BSTC, dcur, tokens, C, ln_eps, s, RowSwap(), dyb, bf));
  }
  // ---- temporal half: y1 = y0 + Attn_T(LN(y0) Wqkv_t) Wo_t
  DSP_TRY(attn_sub_bwd(h2, qkv2, a2, lse2, w->wqkv_t, w->wo_t, grads->wqkv_t, grads->bqkv_t, grads->wo_t,
                       grads->bo_t, S, T));
  // dy0, written back in (B, T, S, C) order (the Switch's adjoint) with its operand copy
  DSP_TRY(launch_layernorm_bwd(y0, 0, dh, 0, dcur, dx1, tokens, C, ln_eps, s, back, dyb, bf));
  // ---- spatial half: x1 = x + Attn_S(LN(x) Wqkv_s) Wo_s
  DSP_TRY(attn_sub_bwd(h1, qkv1, a1, lse1, w->wqkv_s, w->wo_s, grads->wqkv_s, grads->bqkv_s, grads->wo_s,
                       grads->bo_s, T, S));
  DSP_TRY(launch_layernorm_bwd(x_BTSC, 0, dh, 0, dx1, dx_BTSC, tokens, C, ln_eps, s));
  return DSP_OK;
#undef DSP_TRY
}

}  // extern "C"
