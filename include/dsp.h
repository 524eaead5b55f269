/*
 * dsp.h -- C ABI of libdsp: one GPU's share of a Dynamic Sequence Parallelism
 * (DSP) spatial-temporal transformer block on AMD MI355X (gfx950).
 *
 * The operations follow "DSP: Dynamic Sequence Parallelism for
 * Multi-Dimensional Transformers" (Zhao et al., ICML 2025):
 *   - the Switch primitive (primitive table, row s_i -> s_j; Eq. 10), here
 *     the local permute + pack of one GPU's shard that precedes the exchange;
 *   - scaled dot-product attention (Eq. 3), per head (Eq. 1-2), run along one
 *     sequence dimension of a multi-dimensional sequence (Eq. 7-8): spatial
 *     attention over S inside each frame, temporal attention over T at each
 *     spatial location;
 *   - the LayerNorm (Eq. 4, 6), linear maps and MLP (Eq. 5) of the block.
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers owned by the caller.  The
 *     library allocates nothing, keeps no pointer after returning and holds no
 *     mutable global state; calls are thread-safe.  The one exception is
 *     dsp_attn_bwd_noalloc, whose scratch is a static per-device array (calls
 *     that overlap on one GPU race on it).
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t passed as an
 *     opaque pointer; NULL means the default stream).  Device faults surface at
 *     the caller's next synchronisation.
 *   - Arguments are validated on the host before anything is launched; a
 *     failed check returns a nonzero dsp_status_t and launches nothing.  A
 *     launch failure returns DSP_ERR_HIP.  No C++ exception crosses the ABI.
 *   - Tensors are dense row-major.  Sequence tensors are [B, S_1, S_2, C]
 *     (C innermost); dimension numbers follow that order: 0 = batch,
 *     1 and 2 = the two sequence dimensions, 3 = hidden.
 *   - Weights of linear maps are stored [out][in] (row-major, the reduction
 *     index contiguous), i.e. y = x * W with W = stored^T.
 */
#ifndef DSP_H_
#define DSP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DSP_OK = 0,
  DSP_ERR_NULL = 1,      /* a required pointer is NULL */
  DSP_ERR_DIM = 2,       /* bad ndim or dimension index */
  DSP_ERR_SHAPE = 3,     /* nonpositive / non-divisible / unsupported size */
  DSP_ERR_DTYPE = 4,     /* unknown or unsupported dtype */
  DSP_ERR_ALIGN = 5,     /* pointer or stride alignment the kernel requires */
  DSP_ERR_HIP = 6,       /* a HIP runtime call or kernel launch failed */
  DSP_ERR_WORKSPACE = 7, /* workspace missing or too small */
  DSP_ERR_ARG = 8        /* any other invalid argument (flags, eps, ...) */
} dsp_status_t;

typedef enum { DSP_F32 = 0, DSP_BF16 = 1 } dsp_dtype_t;

/* Human-readable name of a status code (static string, never NULL). */
const char* dsp_status_str(int status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int dsp_version(void);

/* ------------------------------------------------------------------------
 * dsp_switch -- one GPU's share of DynamicSwitch(X, i, j)
 * (primitive table, row s_i -> s_j; Eq. 10; system overview figure).
 *
 * x:      [B, D1, D2, C] (ndim 4: K = 2 sequence dimensions) or
 *         [B, D1, D2, D3, C] (ndim 5: K = 3, the multi-dimensional form of
 *         Eq. 7), the local shard, currently sharded on `from_dim`.
 * y:      output, same number of elements as x, written as `n_chunks`
 *         contiguous per-destination chunks.  With from_dim=1, to_dim=2:
 *             y[n][b][j'][i][c] = x[b][i][n*D2/n_chunks + j'][c]
 *         (chunk n has shape [B, D2/n_chunks, D1, C]: the to-dim slice
 *         outermost, the from-dim -- the dimension the next stage computes
 *         over -- innermost before C).  With from_dim=2, to_dim=1:
 *             y[n][b][i'][j][c] = x[b][n*D1/n_chunks + i'][j][c].
 *         For (B,T,S,C) with T sharded, from=1 (T), to=2 (S) and n_chunks=1
 *         this is the permute to (B,S,T,C).  Chunk n is what rank n receives
 *         in the all-to-all; the exchange itself is not part of this call.
 *         For K = 3 the chunk keeps the other two sequence dimensions in
 *         their order (the to-dim cut to D_to/n_chunks) and puts the from-dim
 *         next to C, e.g. from=1, to=3:
 *             y[n][b][j][k'][i][c] = x[b][i][j][n*D3/n_chunks + k'][c].
 * from_dim == to_dim is the "no primitive" row of the table: y = copy of x.
 * Errors: DSP_ERR_NULL (shape NULL, or x / y NULL for a non-empty tensor;
 *   an empty tensor may come with NULL pointers), DSP_ERR_DIM (ndim not 4 or 5,
 *   or a dim not in 1..K), DSP_ERR_SHAPE (a size < 0, n_chunks < 1, the to-dim not
 *   divisible by n_chunks, or more than 2^31 rows / 16-byte vectors),
 *   DSP_ERR_DTYPE, DSP_ERR_ARG (x and y overlap).  A tensor with a zero size
 *   is accepted and launches nothing.
 * The data are moved as raw bits (bit-exact for any payload, NaNs included).
 * ------------------------------------------------------------------------ */
int dsp_switch(const void* x, void* y, const int64_t* shape, int ndim, int from_dim, int to_dim,
               int n_chunks, int dtype, void* stream);

/* Same as dsp_switch with an explicit kernel choice: 0 = automatic,
 * 1 = direct 128-bit row copy (requires 16-byte aligned pointers and rows),
 * 2 = LDS-staged tile transpose.  Any other value -> DSP_ERR_ARG.  K = 3
 * tensors (ndim 5) have one kernel: only variant 0 is accepted. */
int dsp_switch_variant(const void* x, void* y, const int64_t* shape, int ndim, int from_dim,
                       int to_dim, int n_chunks, int dtype, int variant, void* stream);

/* ------------------------------------------------------------------------
 * dsp_split -- the Split row of the primitive table (s^ -> s_i): a tensor
 * replicated on every rank becomes sharded on sequence dimension `dim`, with
 * no communication; rank `rank` keeps its slice.
 *
 * x:      [B, S_1, .., S_K, C] (ndim = K + 2, K = 2 or 3), replicated.
 * y:      [B, .., S_dim / n_chunks, .., C], dense:
 *             y[b][..][i'][..][c] = x[b][..][rank * S_dim/n_chunks + i'][..][c].
 * Errors: DSP_ERR_NULL, DSP_ERR_DIM (ndim not 4 or 5, dim not in 1..K),
 *   DSP_ERR_SHAPE (a negative size, n_chunks < 1, S_dim not divisible),
 *   DSP_ERR_DTYPE, DSP_ERR_ARG (rank not in [0, n_chunks), x and y overlap).
 * A bit copy; an empty result launches nothing.
 * ------------------------------------------------------------------------ */
int dsp_split(const void* x, void* y, const int64_t* shape, int ndim, int dim, int n_chunks,
              int rank, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * dsp_gather -- the Gather row of the primitive table (s_i -> s^, an
 * all-gather): the receiver's concatenation of every rank's shard, run on
 * one GPU with one buffer per rank.
 *
 * shards:      host array of n_shards device pointers, each a dense
 *              [B, S_1, .., S_K, C] shard with the size shard_shape
 *              (ndim = K + 2, K = 2 or 3); they may alias each other.
 * y:           [B, .., n_shards * S_dim, .., C], dense:
 *                  y[b][..][m * S_dim + i][..][c] = shards[m][b][..][i][..][c].
 * n_shards:    1..64.
 * Errors: DSP_ERR_NULL, DSP_ERR_DIM, DSP_ERR_SHAPE (a negative size, n_shards
 *   out of range), DSP_ERR_DTYPE, DSP_ERR_ARG (y overlaps a shard).
 * A bit copy; an empty result launches nothing.
 * ------------------------------------------------------------------------ */
int dsp_gather(const void* const* shards, void* y, const int64_t* shard_shape, int ndim, int dim,
               int n_shards, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * dsp_exchange_unpack -- the exchange of DynamicSwitch among N ranks (the
 * all-to-all of the primitive table's row s_i -> s_j, Eq. 10), run on one GPU
 * with one buffer per rank, fused with every receiver's unpack.
 *
 * packed: host array of N device pointers; packed[m] is rank m's dsp_switch
 *         output, shape [N][B][P][F][C] (P = D_to / N, F = rank m's length of
 *         the from-dimension; for K = 3, P is the product of the two other
 *         sequence dimensions of a chunk).  Read only; the N buffers may alias
 *         each other.
 * out:    host array of N device pointers; out[n] receives rank n's result,
 *         shape [B][P][N*F][C]:
 *             out[n][b][p][m*F + f][c] = packed[m][n][b][p][f][c]
 *         i.e. chunk n of every rank, concatenated along the from-dimension
 *         in rank order.  For the (B,T,S,C) -> (B,S,T,C) switch of T-shards
 *         this is S-shard n of the permuted tensor (Eq. 7-8, i = T).
 * shape:  {N, B, P, F, C}.  dtype: element type (only its size matters; the
 *         data move as raw bits).
 * The caller owns all buffers; N*(B*P*F*C) elements per buffer.
 * Errors: DSP_ERR_NULL (shape NULL, or a pointer array / pointer NULL for a
 *   non-empty exchange), DSP_ERR_SHAPE (N < 1, N > 64, a negative size, or a
 *   size overflow), DSP_ERR_DTYPE, DSP_ERR_ARG (an output buffer overlaps a
 *   packed buffer or another output buffer).  An empty exchange launches
 *   nothing.
 * ------------------------------------------------------------------------ */
int dsp_exchange_unpack(const void* const* packed, void* const* out, const int64_t* shape,
                        int dtype, void* stream);

/* ------------------------------------------------------------------------
 * Attention along one sequence dimension (Eq. 3 per head, Eq. 1-2; the
 * per-dimension reshape of Eq. 7-8).  Non-causal softmax(q k^T * scale) v.
 *
 * dsp_spatial_attn:  q, k, v, o laid out (B, T, S, *), attention over L = S
 *   inside each (b, t) frame, independently per head h.
 * dsp_temporal_attn: q, k, v, o laid out (B, S, T, *), attention over L = T at
 *   each (b, s) location, independently per head.
 *
 * Head h of a token occupies elements [h*D, (h+1)*D) of that token's row.
 * ld_in:  elements between consecutive token rows of q, k and v (C = H*D for
 *         separate tensors, 3C when q/k/v point into one packed [Q|K|V] buffer).
 * ld_out: elements between consecutive token rows of o (>= H*D).
 * scale:  softmax scale; scale <= 0 selects 1/sqrt(D) with the true D.
 * dtype:  DSP_BF16 (bf16 storage, bf16 MFMA, fp32 softmax and accumulation)
 *         or DSP_F32 (fp32 storage and fp32 arithmetic throughout).
 * Supported D: DSP_BF16 -- D in {16, 32, 64, 72, 80, 96}; DSP_F32 --
 *   1 <= D <= 256.  bf16 needs 16-byte aligned q/k/v/o and ld_in, ld_out
 *   multiples of 8 (DSP_ERR_ALIGN otherwise).
 * Errors: DSP_ERR_NULL, DSP_ERR_SHAPE (a size < 0, H < 1, D < 1, H*D > ld,
 *   unsupported D), DSP_ERR_DTYPE, DSP_ERR_ALIGN, DSP_ERR_ARG (scale NaN or
 *   infinite), DSP_ERR_HIP.  An empty input (B, T or S equal to 0) is
 *   accepted, may come with NULL pointers, and launches nothing.
 * ------------------------------------------------------------------------ */
int dsp_spatial_attn(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t T,
                     int64_t S, int H, int D, int64_t ld_in, int64_t ld_out, float scale,
                     int dtype, void* stream);
int dsp_temporal_attn(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t S,
                      int64_t T, int H, int D, int64_t ld_in, int64_t ld_out, float scale,
                      int dtype, void* stream);

/* Attention with explicit layouts: the same operation over L positions of
 * each (b, x, h) unit, element (b, x, l, h*D + d) of q/k/v at
 *     b*in_strides[0] + x*in_strides[1] + l*in_strides[2] + h*D + d
 * and of o at the same offsets with out_strides (strides in elements).  This
 * reads a layout the previous stage left behind without a switch, e.g.
 * temporal attention straight from (B, T, S, C): X = S, L = T, in_strides =
 * {T*S*C, C, S*C} (Eq. 7-8 with i = T, computed on the unswitched tensor).
 * dsp_spatial_attn and dsp_temporal_attn are this call with the strides of
 * their dense layouts.  Requirements and errors as for dsp_spatial_attn, plus:
 * strides must be >= 0 (DSP_ERR_SHAPE), the output rows must not overlap
 * (checked: DSP_ERR_ARG), and for DSP_BF16 every stride a multiple of 8
 * elements and min(L, 64) * in_strides[2] * 2 < 2^31 (DSP_ERR_ALIGN /
 * DSP_ERR_SHAPE).  o must not overlap q, k or v. */
int dsp_attn_strided(const void* q, const void* k, const void* v, void* o, int64_t B, int64_t X,
                     int64_t L, int H, int D, const int64_t* in_strides, const int64_t* out_strides,
                     float scale, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * dsp_attn_fwd_lse -- dsp_attn_strided that also saves, for every query, the
 * natural-log log-sum-exp of its scaled scores,
 *     lse[u][i] = log sum_j exp(scale * q_i . k_j),
 * the row statistic of the softmax in Eq. 3 that the backward pass needs to
 * recompute the probabilities.  Used for training, which the paper's models
 * undergo (its weak-scaling runs are a training stage, with ZeRO-2).
 * lse: DEVICE fp32 [B * X * H][L], unit u = (b * X + x) * H + h, caller-owned,
 *   4-byte aligned (DSP_ERR_ALIGN), required unless the input is empty
 *   (DSP_ERR_NULL).  The bf16 kernels compute it from the same bf16-rounded
 *   scores and probabilities that produce o.
 * Everything else, including errors, as for dsp_attn_strided.
 * ------------------------------------------------------------------------ */
int dsp_attn_fwd_lse(const void* q, const void* k, const void* v, void* o, float* lse, int64_t B,
                     int64_t X, int64_t L, int H, int D, const int64_t* in_strides,
                     const int64_t* out_strides, float scale, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * dsp_attn_bwd -- gradient of attention along one sequence dimension (Eq. 3
 * per head, Eq. 1-2; any layout as in dsp_attn_strided) by the chain rule
 * through the softmax.  With z = scale * q.k, P = softmax(z) per row and
 * Delta_i = sum_d dout[i][d] * o[i][d]:
 *     dv = P^T dout,  dz = P * (dout v^T - Delta),
 *     dq = scale * dz k,  dk = scale * dz^T q.
 * q, k, v: the forward's inputs; o, lse: its outputs (dsp_attn_fwd_lse);
 *   dout: the gradient of the loss with respect to o.
 * dq, dk, dv: outputs, same shapes and strides as q, k, v (qkv_strides), so
 *   gradients of a packed [Q|K|V] buffer land in a packed buffer.
 * o, dout: element (b, x, l, h*D + d) at b*o_strides[0] + x*o_strides[1] +
 *   l*o_strides[2] + h*D + d.
 * delta: DEVICE fp32 workspace [B * X * H][L]; on return it holds Delta.
 * All pointers are DEVICE pointers owned by the caller; dq, dk, dv must not
 *   overlap each other or any input, and delta must not overlap lse
 *   (checked: DSP_ERR_ARG).
 * dtype DSP_BF16: bf16 tensors, fp32 accumulation on the matrix cores; D in
 *   {16, 32, 64, 72, 80, 96}; 16-byte aligned tensors and strides that are
 *   multiples of 8 (DSP_ERR_ALIGN); 64 * qkv_strides[2] * 2 and
 *   64 * o_strides[2] * 2 below 2^31 (DSP_ERR_SHAPE).  Deterministic: no
 *   atomics, so repeated calls give identical bits.
 * dtype DSP_F32: fp32 FMA throughout; 1 <= D <= 256.
 * scale <= 0 selects 1/sqrt(D).  An empty input launches nothing.
 * Errors: DSP_ERR_NULL, DSP_ERR_SHAPE, DSP_ERR_DTYPE, DSP_ERR_ALIGN,
 *   DSP_ERR_ARG (scale not finite, overlapping gradient rows), DSP_ERR_HIP.
 * ------------------------------------------------------------------------ */
int dsp_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                 const float* lse, void* dq, void* dk, void* dv, float* delta, int64_t B, int64_t X,
                 int64_t L, int H, int D, const int64_t* qkv_strides, const int64_t* o_strides,
                 float scale, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * dsp_attn_bwd_noalloc -- dsp_attn_bwd for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  It takes no `delta` workspace: the Delta rows live in
 * a library-owned static device array of dsp_attn_bwd_noalloc_max_rows()
 * fp32 values (4194304 values, 16 MiB), one copy per GPU, loaded with the
 * library's code and held until the process ends.  The call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine); its first call on a
 * device looks up that device's copy (hipGetSymbolAddress).
 * Every call on one GPU uses that GPU's array, and its contents are those of
 * the last call: calls that overlap on one GPU (several streams or host
 * threads) race and must be serialised by the caller.  Delta is not returned.
 * B * X * H * L above the maximum: DSP_ERR_WORKSPACE, nothing launched.
 * Everything else -- arguments, layouts, dtypes, errors and the bits of dq,
 * dk, dv -- as dsp_attn_bwd.
 * ------------------------------------------------------------------------ */
int64_t dsp_attn_bwd_noalloc_max_rows(void);
int dsp_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dout,
                         const float* lse, void* dq, void* dk, void* dv, int64_t B, int64_t X, int64_t L, int H,
                         int D, const int64_t* qkv_strides, const int64_t* o_strides, float scale, int dtype,
                         void* stream);

/* ------------------------------------------------------------------------
 * dsp_attn_general / dsp_attn_general_bwd -- the attention variants the
 * paper states DSP is compatible with: multi-query and grouped-query attention
 * (Hkv key/value heads shared by H / Hkv query heads each) and cross-attention
 * (keys and values from another sequence, of their own length), on the same
 * per-(b, x) units as dsp_attn_strided.  For unit (b, x, h):
 *   queries: Lq positions, element (b, x, l, h*D + d) of q at
 *            b*q_strides[0] + x*q_strides[1] + l*q_strides[2] + h*D + d;
 *   keys, values: Lk positions of head h / (H / Hkv), at
 *            b*kv_strides[0] + x*kv_strides[1] + l*kv_strides[2] + (h/(H/Hkv))*D + d;
 *   output (and dout): o_strides, H heads, Lq positions.
 * Hkv == H, Lq == Lk and kv_strides == q_strides is dsp_attn_strided.  A
 * kv stride of 0 broadcasts keys and values (e.g. one text sequence shared
 * by every frame: kv_strides[1] = 0); the backward rejects it (its key and
 * value gradients would have no single owner: DSP_ERR_ARG).
 * lse (forward, optional: NULL skips it): fp32 [B * X * H][Lq].  The
 * backward's contract (lse, delta [B*X*H][Lq], dq with q's strides, dk and dv
 * with kv_strides -- the sums over each group's query heads) is otherwise
 * dsp_attn_bwd's.  H % Hkv != 0, or Lk == 0 with Lq > 0: DSP_ERR_SHAPE.
 * Everything else, including dtypes, alignment and errors, as for
 * dsp_attn_strided / dsp_attn_bwd.
 * ------------------------------------------------------------------------ */
int dsp_attn_general(const void* q, const void* k, const void* v, void* o, float* lse, int64_t B, int64_t X,
                     int64_t Lq, int64_t Lk, int H, int Hkv, int D, const int64_t* q_strides,
                     const int64_t* kv_strides, const int64_t* o_strides, float scale, int dtype, void* stream);
int dsp_attn_general_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                         const float* lse, void* dq, void* dk, void* dv, float* delta, int64_t B, int64_t X,
                         int64_t Lq, int64_t Lk, int H, int Hkv, int D, const int64_t* q_strides,
                         const int64_t* kv_strides, const int64_t* o_strides, float scale, int dtype,
                         void* stream);

/* ------------------------------------------------------------------------
 * dsp_layernorm -- per-row normalisation over C (Eq. 4, 6):
 *   y = (x - mean) / sqrt(var + eps), biased variance, no affine part,
 *   statistics in fp32.
 * x: [rows, C] of x_dtype; y: [rows, C] of y_dtype (DSP_F32 or DSP_BF16).
 * Errors: DSP_ERR_NULL, DSP_ERR_SHAPE (rows < 0, C < 1), DSP_ERR_DTYPE,
 *   DSP_ERR_ARG (eps < 0 or not finite).
 * ------------------------------------------------------------------------ */
int dsp_layernorm(const void* x, int x_dtype, void* y, int y_dtype, int64_t rows, int C, float eps,
                  void* stream);

/* ------------------------------------------------------------------------
 * dsp_layernorm_bwd -- gradient of dsp_layernorm with respect to its input
 * (Eq. 4, 6; used to train the block):
 *   dx = dres + (dy - mean(dy) - y * mean(dy * y)) / sqrt(var + eps),
 *   y = (x - mean) / sqrt(var + eps), statistics of x recomputed in fp32.
 * x: [rows, C] of x_dtype (the forward's input); dy: [rows, C] of dy_dtype;
 * dres: [rows, C] fp32 gradient already flowing into x (e.g. through a
 *   residual connection), or NULL; may equal dx (accumulate in place);
 * dx: [rows, C] fp32.  DEVICE pointers owned by the caller.
 * Errors: DSP_ERR_NULL, DSP_ERR_SHAPE, DSP_ERR_DTYPE, DSP_ERR_ARG (eps < 0
 *   or not finite; dx overlapping x, dy, or dres other than in place).
 * ------------------------------------------------------------------------ */
int dsp_layernorm_bwd(const void* x, int x_dtype, const void* dy, int dy_dtype, const float* dres, float* dx,
                      int64_t rows, int C, float eps, void* stream);

/* ------------------------------------------------------------------------
 * dsp_linear -- out = epilogue(a * W + bias)  (Eq. 1 W^O, Eq. 5 W_1/W_2)
 *
 * a:        [M, K] of dtype.
 * w:        [N, K] of dtype (stored [out][in]).
 * bias:     [N] of dtype, or NULL.
 * residual: [M, N] fp32 or NULL; required iff DSP_EPI_RESID.  May equal out.
 * out:      [M, N]; dtype for DSP_EPI_NONE / DSP_EPI_GELU / DSP_EPI_RELU,
 *           fp32 for DSP_EPI_F32 (out = a*W + bias) and DSP_EPI_RESID
 *           (out = residual + a*W + bias).
 * epilogue: DSP_EPI_NONE, DSP_EPI_GELU (erf GELU: x*Phi(x)), DSP_EPI_RESID,
 *           DSP_EPI_F32, DSP_EPI_RELU (max(0, x): the FFN activation of Eq. 5).
 * dtype:    DSP_BF16 (bf16 MFMA, fp32 accumulation) or DSP_F32 (fp32 FMA).
 * bf16 needs K % 8 == 0 and 16-byte aligned a, w, out and residual
 * (DSP_ERR_ALIGN).  out must not overlap a, w or bias.
 * Errors: DSP_ERR_NULL, DSP_ERR_SHAPE (M < 0, N < 1, K < 1), DSP_ERR_DTYPE,
 *   DSP_ERR_ALIGN, DSP_ERR_ARG (unknown epilogue, residual missing).
 * ------------------------------------------------------------------------ */
enum { DSP_EPI_NONE = 0, DSP_EPI_GELU = 1, DSP_EPI_RESID = 2, DSP_EPI_F32 = 3, DSP_EPI_RELU = 4 };
int dsp_linear(const void* a, const void* w, const void* bias, const float* residual, void* out,
               int64_t M, int N, int K, int epilogue, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * Gradients of dsp_linear, y = a * W + bias (W stored [N][K] = [out][in]),
 * for training the block (the paper trains its models; weak scaling is a
 * training stage with ZeRO-2).  Chain rule: da = dy * W^T-stored = dy W,
 * dW = dy^T a, dbias = the column sums of dy.
 *
 * dsp_linear_bwd_data -- dx[M][K] = epilogue(dy[M][N] * W[N][K]).
 *   dy: [M, N] of dtype;  w: [N, K] of dtype (the forward's weight);
 *   u:  [M, K] of dtype, the saved pre-activation for DSP_GRAD_EPI_GELU_BWD
 *       (dx = (dy W) * GELU'(u), GELU'(u) = Phi(u) + u phi(u): the backward
 *       through the MLP's activation, Eq. 5) and DSP_GRAD_EPI_RELU_BWD
 *       (dx = (dy W) where u > 0, else 0); NULL otherwise;
 *   dx: [M, K], fp32 for DSP_GRAD_EPI_F32, dtype otherwise.
 * dsp_linear_bwd_weight -- dw[N][K] = dy^T[N][M] * x[M][K] (fp32) and, when
 *   db is not NULL, db[N] = sum over m of dy[m][n] (fp32).
 *   dy: [M, N] of dtype; x: [M, K] of dtype (the forward's input).
 *   workspace: device memory of at least
 *   dsp_linear_bwd_weight_workspace_bytes(M, N, K, dtype) bytes (may be NULL
 *   when that is 0).  The reduction over M is split across work-groups, and
 *   their fp32 partial sums are added in a fixed order: the result is
 *   deterministic.
 * dtype DSP_BF16: bf16 operands on the matrix cores, fp32 accumulation;
 *   N % 8 == 0 and K % 8 == 0 and 16-byte aligned tensors (DSP_ERR_ALIGN).
 * dtype DSP_F32: fp32 FMA.
 * All pointers are DEVICE pointers owned by the caller; outputs must not
 * overlap inputs (DSP_ERR_ARG).  M == 0: dsp_linear_bwd_data launches
 * nothing; dsp_linear_bwd_weight writes dw = 0 (and db = 0).
 * Errors: DSP_ERR_NULL, DSP_ERR_SHAPE (M < 0, N < 1, K < 1, sizes past the
 *   32-bit tile range), DSP_ERR_DTYPE, DSP_ERR_ALIGN, DSP_ERR_ARG (unknown
 *   epilogue, overlap), DSP_ERR_WORKSPACE, DSP_ERR_HIP.
 * ------------------------------------------------------------------------ */
enum { DSP_GRAD_EPI_F32 = 0, DSP_GRAD_EPI_BF16 = 1, DSP_GRAD_EPI_GELU_BWD = 2, DSP_GRAD_EPI_RELU_BWD = 3 };
int dsp_linear_bwd_data(const void* dy, const void* w, const void* u, void* dx, int64_t M, int N, int K,
                        int epilogue, int dtype, void* stream);
size_t dsp_linear_bwd_weight_workspace_bytes(int64_t M, int N, int K, int dtype);
int dsp_linear_bwd_weight(const void* dy, const void* x, float* dw, float* db, void* workspace,
                          size_t ws_bytes, int64_t M, int N, int K, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * The spatial-temporal block: one GPU's share of one layer of the 2D
 * transformer of the model-details appendix (a spatial block, then a temporal
 * block), with one Switch between them.
 *
 *   x  += Wo_s * SpatialAttn(LN(x) * Wqkv_s)          x in (B,T,S,C)
 *   y   = Switch_{T->S}(x)                             y in (B,S,T,C)
 *   y  += Wo_t * TemporalAttn(LN(y) * Wqkv_t)
 *   y  += W2 * GELU(LN(y) * W1)
 *
 * Weights (dtype, stored [out][in]): wqkv_* [3C][C] with output columns
 * [Q | K | V], wo_* [C][C], w1 [F][C], w2 [C][F]; biases ([out], dtype) may be
 * NULL.  x_BTSC and y_BSTC are fp32 (the residual stream); they must not
 * overlap.  Flags:
 *   DSP_BLOCK_NO_MLP_LN -- no LayerNorm for the MLP;
 *   DSP_BLOCK_ATTN_ONLY -- projections and attention only: no LayerNorm, no
 *     residual adds and no MLP (w1/w2 unused):
 *       y = Wo_t * TemporalAttn(Switch(Wo_s * SpatialAttn(x * Wqkv_s)) * Wqkv_t);
 *   DSP_BLOCK_POST_LN -- every LayerNorm after its residual add, the form of
 *     Eq. 4 and Eq. 6:  x = LN(x + Wo_s * SpatialAttn(x * Wqkv_s)), ...,
 *     y = LN(y + W2 * act(y * W1));
 *   DSP_BLOCK_RELU -- the FFN activation is ReLU (Eq. 5) instead of GELU.
 *   DSP_BLOCK_POST_LN | DSP_BLOCK_RELU is the paper's own block.
 * workspace: device buffer of at least dsp_st_block_workspace_bytes(...)
 * bytes, 256-byte aligned, owned by the caller; contents are scratch.
 * dsp_st_block_workspace_bytes returns 0 for invalid sizes.
 * Errors: those of the pieces plus DSP_ERR_WORKSPACE and DSP_ERR_ARG.
 * ------------------------------------------------------------------------ */
typedef struct {
  const void *wqkv_s, *bqkv_s, *wo_s, *bo_s;
  const void *wqkv_t, *bqkv_t, *wo_t, *bo_t;
  const void *w1, *b1, *w2, *b2;
} dsp_block_weights_t;

enum { DSP_BLOCK_NO_MLP_LN = 1, DSP_BLOCK_ATTN_ONLY = 2, DSP_BLOCK_POST_LN = 4, DSP_BLOCK_RELU = 8 };

size_t dsp_st_block_workspace_bytes(int64_t B, int64_t T, int64_t S, int C, int H, int F,
                                    int dtype);
int dsp_st_block_forward(const float* x_BTSC, float* y_BSTC, const dsp_block_weights_t* w,
                         void* workspace, size_t ws_bytes, int64_t B, int64_t T, int64_t S, int C,
                         int H, int F, float ln_eps, int flags, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * Training the block: a forward that keeps its activations, and the backward.
 * The paper trains its models (weak scaling as a training stage, ZeRO-2), so
 * every step of the block has a gradient: the chain rule through LayerNorm,
 * the linear maps and the MLP activation, attention along each sequence
 * dimension (Eq. 3 per head), and the Switch, whose adjoint is the switch
 * back (S -> T).
 *
 * dsp_st_block_forward_train -- dsp_st_block_forward (same x, y, w, sizes,
 *   eps and dtype) that writes the activations the backward needs into
 *   `saved`: DEVICE memory of at least dsp_st_block_train_saved_bytes(...)
 *   bytes for the same sizes, flags and dtype, 256-byte aligned, owned by the
 *   caller (1.7 GB at B1 T32 S1024 C1152 F4608 in bf16, pre-LN; post-LN with
 *   the MLP's LayerNorm keeps one more fp32 stream).  Flags: any combination
 *   of DSP_BLOCK_NO_MLP_LN, DSP_BLOCK_POST_LN (Eq. 4, 6: LN after each
 *   residual add) and DSP_BLOCK_RELU; the projection-only chain
 *   (DSP_BLOCK_ATTN_ONLY) gives DSP_ERR_ARG.  y has the bits
 *   dsp_st_block_forward writes for the same arguments (the MLP's first GEMM
 *   stores, from the same fp32 sum as the activation, what the activation's
 *   backward needs: the pre-activation, or GELU' there when the block is
 *   bf16 with GELU at sizes whose backward runs on the large-tile GEMM).
 * dsp_st_block_backward -- given the forward's x (B,T,S,C), its saved
 *   activations, and dy (B,S,T,C) = dL/dy, writes dx = dL/dx (B,T,S,C, fp32)
 *   and the weight gradients into `grads`: fp32 arrays shaped like the weights
 *   (stored [out][in]), required for the six weights; bias gradients are
 *   written where the pointer is not NULL (whether or not the forward used a
 *   bias).  workspace: DEVICE scratch of at least
 *   dsp_st_block_backward_workspace_bytes(...) bytes, 256-byte aligned.
 *   Gradients are deterministic (no atomics).  bf16: the operands of every
 *   product are bf16 (gradients rounded to bf16 where they enter a product),
 *   accumulation and the residual-stream gradient are fp32.
 * Errors: as dsp_st_block_forward, plus DSP_ERR_WORKSPACE (saved or
 *   workspace missing or too small) and DSP_ERR_ARG (unsupported flags,
 *   overlapping buffers).
 * ------------------------------------------------------------------------ */
typedef struct {
  float *wqkv_s, *bqkv_s, *wo_s, *bo_s, *wqkv_t, *bqkv_t, *wo_t, *bo_t, *w1, *b1, *w2, *b2;
} dsp_block_grads_t;
size_t dsp_st_block_train_saved_bytes(int64_t B, int64_t T, int64_t S, int C, int H, int F, int flags,
                                      int dtype);
size_t dsp_st_block_backward_workspace_bytes(int64_t B, int64_t T, int64_t S, int C, int H, int F, int dtype);
int dsp_st_block_forward_train(const float* x_BTSC, float* y_BSTC, const dsp_block_weights_t* w, void* saved,
                               size_t saved_bytes, int64_t B, int64_t T, int64_t S, int C, int H, int F,
                               float ln_eps, int flags, int dtype, void* stream);
int dsp_st_block_backward(const float* x_BTSC, const float* dy_BSTC, const dsp_block_weights_t* w,
                          const void* saved, size_t saved_bytes, void* workspace, size_t ws_bytes, float* dx_BTSC,
                          const dsp_block_grads_t* grads, int64_t B, int64_t T, int64_t S, int C, int H, int F,
                          float ln_eps, int flags, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * Measurement aid (not a step of the method): the bf16 MFMA rate the chip
 * sustains with every CU busy.  The published dense bf16 figure assumes the
 * peak engine clock; under a long all-CU MFMA load the clock settles lower.
 * A benchmark reports a kernel's fraction of the published peak, and this
 * rate beside it, measured in the same process and conditions.
 *
 * dsp_probe_mfma -- launches 2048 work-groups of 4 waves (two per SIMD), each
 *   wave issuing 8 * iters independent v_mfma_f32_32x32x16_bf16 on operands
 *   whose bits change every iteration; nothing else runs in its loop.  The
 *   caller times it (events on `stream`) and divides
 *   dsp_probe_mfma_flops(iters) by the time.  workspace: DEVICE memory of at
 *   least dsp_probe_mfma_workspace_bytes() bytes, 16-byte aligned (receives
 *   one float per thread, meaningless).  Errors: DSP_ERR_ARG (iters < 1),
 *   DSP_ERR_NULL, DSP_ERR_WORKSPACE, DSP_ERR_ALIGN.
 * ------------------------------------------------------------------------ */
size_t dsp_probe_mfma_workspace_bytes(void);
double dsp_probe_mfma_flops(int iters);
int dsp_probe_mfma(void* workspace, size_t ws_bytes, int iters, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DSP_H_ */
