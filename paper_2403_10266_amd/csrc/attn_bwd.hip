// Backward of attention along one sequence dimension: the gradient of
// softmax(Q K^T * scale) V (Eq. 3, per head as in Eq. 1-2) by the chain rule
// through the softmax.  With z = scale * q.k, P = softmax(z) row by row and
// Delta_i = sum_d dO[i][d] O[i][d] (= sum_j dP[i][j] P[i][j]):
//   dV = P^T dO,  dP = dO V^T,  dZ = P * (dP - Delta),
//   dQ = scale * dZ K,  dK = scale * dZ^T Q.
// P is recomputed from the forward's row log-sum-exp, so nothing of size
// L x L is ever stored.
//
// bf16 path, on v_mfma_f32_32x32x16_bf16 like the forward:
//  * Two deterministic kernels, no atomics: the first owns a block of queries
//    and loops over key tiles (dQ, and Delta for its queries); the second owns
//    a block of keys and loops over query tiles (dK and dV).  Each recomputes
//    the scores it needs.  Units of at most 128 queries and keys (temporal
//    attention) run a third kernel that holds the whole unit in LDS and does
//    both loops, so its rows are read from HBM once.
//  * The head width is padded to a multiple of 16 with three spare columns.
//    They carry the per-row statistics into the score products as three bf16
//    terms whose sum is the fp32 value exactly (8 significant bits each): the
//    query side holds -lse and the key side 1.0, so the MFMA yields z' - lse
//    directly and P = exp2 of the accumulator, at any magnitude of lse.  In
//    the same way the dO side holds -Delta and the V side 1.0, so the dP
//    product yields dP - Delta.
//  * Scores use Q' = Q * scale * log2(e), rounded to bf16 exactly as in the
//    forward, so P matches the probabilities whose log-sum-exp was saved.
//  * The d-row products (dQ^T = K^T dZ^T, dV^T = dO^T P, dK^T = Q'^T dZ) take
//    their A operand transposed from row-major LDS tiles (ds_read_b64_tr_b16)
//    and their B operand straight from the score accumulators converted to
//    bf16, with the same permuted row order on both sides.  The last 16 rows
//    of a head width that is not a multiple of 32 run on 16x16x32 MFMAs.
//
// fp32 path: plain FMA loops, one thread per (unit, row, 32-column slice).
#include <math.h>

#include <algorithm>

#include "attn_bf16_common.h"
#include "dsp_internal.h"

// Units of at most 128 queries and keys (no grouped heads) run the fused
// single-pass kernel.
#ifndef DSP_ATTN_BWD_SHORT
#define DSP_ATTN_BWD_SHORT 1
#endif
// Row pad (elements) of the backward's LDS tiles.
#ifndef DSP_ATTN_BWD_PAD
#define DSP_ATTN_BWD_PAD 24
#endif

namespace dsp {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int D>
struct BGeo {
  static constexpr int NDK = (D + 3 + 15) / 16;  // 16-wide d steps of the score products
  static constexpr int NT32 = D / 32;            // 32-row tiles of the d-row products
  static constexpr bool SLAB = (D % 32) != 0;    // rows 32 NT32 .. + 15 on 16x16x32
  static constexpr int P = NDK * 16 + DSP_ATTN_BWD_PAD;  // LDS row pitch (elements): an odd multiple of 16 B
  static constexpr int CH = D / 8;               // 16-byte chunks of a row
  static constexpr int SB = D / 16;              // d step holding the bias columns D .. D + 2
  static constexpr int GB = (D % 16) / 8;        // ... in lanes with g == GB, elements 0 .. 2
  static_assert(D % 8 == 0 && D % 32 <= 16, "head width");
};

struct BwdParams {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  const bf16* o;
  const bf16* dout;
  const float* lse;
  bf16* dq;
  bf16* dk;
  bf16* dv;
  float* delta;
  int64_t b_q, x_q, r_q;     // q and dq
  int64_t b_kv, x_kv, r_kv;  // k, v and dk, dv
  int64_t b_o, x_o, r_o;     // o and dout
  uint32_t X, H, L, Lk, grp, n_blk, n_blocks;  // L queries, Lk keys; grp query heads per kv head
  float c;      // scale * log2(e)
  float scale;
};

// Work-group -> (unit, block) with an XCD-aware order; units are (b, x, head)
// over `heads` heads per (b, x).  Also the (b, x) index for the bases.
struct BwdMap {
  uint32_t unit, blk, bx, head;
};

__device__ __forceinline__ BwdMap bwd_map(const BwdParams& p, uint32_t heads) {
  uint32_t bid = blockIdx.x;
  // hardware places block i on XCD i % 8; give each XCD a contiguous range
  if ((p.n_blocks & 7u) == 0) bid = (bid & 7u) * (p.n_blocks >> 3) + (bid >> 3);
  BwdMap m;
  m.unit = bid / p.n_blk;
  m.blk = bid - m.unit * p.n_blk;
  m.head = m.unit % heads;
  m.bx = m.unit / heads;
  return m;
}

__device__ __forceinline__ int64_t bx_base(const BwdParams& p, uint32_t bx, int64_t bs, int64_t xs) {
  return (int64_t)(bx / p.X) * bs + (int64_t)(bx % p.X) * xs;
}

// A operand of a 32x32x16 MFMA read transposed from a row-major LDS tile:
// lane (m + 32g) gets column col0 + m at rows row0 + 4g + {0..3, 8..11}, the
// row order of the registers 8kk .. 8kk + 7 of a 32x32 accumulator.
__device__ __forceinline__ bf16x8 tr_frag32(const bf16* t, int pitch, int row0, int col0, int lane) {
  const int j16 = lane & 15, g = lane >> 5, mbase = 16 * ((lane >> 4) & 1);
  const int row = row0 + 4 * g + (j16 >> 2);
  const int col = col0 + mbase + 4 * (j16 & 3);
  const shortx4 lo = lds_read_tr(t + row * pitch + col);
  const shortx4 hi = lds_read_tr(t + (row + 8) * pitch + col);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// A operand of the 16x16x32 slab (16 columns col0 .. col0 + 15, 32 rows of a
// 32x32 tile starting at row0), in the row order that one permlane16 swap
// gives the B operand (see slab_b).
__device__ __forceinline__ bf16x8 tr_slab(const bf16* t, int pitch, int row0, int col0, int lane) {
  const int j16 = lane & 15, c = lane >> 4;
  const int kbase = ((c & 1) ? 16 : 0) + ((c & 2) ? 4 : 0);
  const int row = row0 + kbase + (j16 >> 2);
  const int col = col0 + 4 * (j16 & 3);
  const shortx4 lo = lds_read_tr(t + row * pitch + col);
  const shortx4 hi = lds_read_tr(t + (row + 8) * pitch + col);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// B operands of the slab from the two bf16 halves (registers 0-7, 8-15) of a
// 32x32 accumulator: b0 for its columns 0-15, b1 for 16-31.
__device__ __forceinline__ void slab_b(const bf16x8& x8, const bf16x8& y8, bf16x8& b0, bf16x8& b1) {
  const u32x4 x = __builtin_bit_cast(u32x4, x8), y = __builtin_bit_cast(u32x4, y8);
  u32x4 r0, r1;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const auto r = __builtin_amdgcn_permlane16_swap(x[w], y[w], false, false);
    r0[w] = r[0];
    r1[w] = r[1];
  }
  b0 = __builtin_bit_cast(bf16x8, r0);
  b1 = __builtin_bit_cast(bf16x8, r1);
}

// -x as three bf16 terms t0 + t1 + t2 == -x exactly for any normal fp32 x:
// each round to nearest leaves an exact residual of at most 16, then 8,
// significant bits, and the last term holds the final 8.
struct Bf16x3 {
  bf16 t[3];
};
__device__ __forceinline__ Bf16x3 neg_split3(float x) {
  const bf16 hi = (bf16)x;
  const float r1 = x - (float)hi;
  const bf16 mid = (bf16)r1;
  return {{(bf16)(-(float)hi), (bf16)(-(float)mid), (bf16)(-(r1 - (float)mid))}};
}

// Row fragment (B operand of a score product) of one row of a bf16 tensor:
// lane (n + 32g) gets elements 16s + 8g .. + 7 for every d step s; columns
// >= D are 0.  `row` may be null (rows past L): all zero.
template <int D>
__device__ __forceinline__ void row_frags(const bf16* row, int g, bf16x8 (&f)[BGeo<D>::NDK]) {
#pragma unroll
  for (int s = 0; s < BGeo<D>::NDK; ++s) {
    const int d = 16 * s + 8 * g;
    if (row && d < D) {
      f[s] = *reinterpret_cast<const bf16x8*>(row + d);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) f[s][e] = (bf16)0.0f;
    }
  }
}

// Stores the 32x32 accumulator tiles (and slab) of a d-row product: lane
// (n + 32g) owns row `row` of the output, t-th tile holding d = 32t + 8(r/4) +
// 4g + r%4; slab h (16x16) holds d = 32 NT32 + 4 (lane / 16) + r of output
// row 16h + lane % 16 of the wave's 32.
template <int D>
__device__ __forceinline__ void store_rows(bf16* base, int64_t r_st, uint32_t row0, uint32_t L, int lane,
                                           const floatx16 (&t32)[BGeo<D>::NT32 > 0 ? BGeo<D>::NT32 : 1],
                                           const floatx4 (&sl)[2], float mul) {
  using G = BGeo<D>;
  const int l32 = lane & 31, g = lane >> 5;
  const uint32_t row = row0 + l32;
  if (row < L) {
    bf16* orow = base + (int64_t)row * r_st;
#pragma unroll
    for (int t = 0; t < G::NT32; ++t)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = 32 * t + 8 * r4 + 4 * g;
        bf16x2 lo = {(bf16)(t32[t][4 * r4 + 0] * mul), (bf16)(t32[t][4 * r4 + 1] * mul)};
        bf16x2 hi = {(bf16)(t32[t][4 * r4 + 2] * mul), (bf16)(t32[t][4 * r4 + 3] * mul)};
        uint2 w;
        w.x = __builtin_bit_cast(uint32_t, lo);
        w.y = __builtin_bit_cast(uint32_t, hi);
        *reinterpret_cast<uint2*>(orow + d0) = w;
      }
  }
  if constexpr (G::SLAB) {
    const int d0 = 32 * G::NT32 + 4 * (lane >> 4);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t rs = row0 + 16 * h + (lane & 15);
      if (d0 < D && rs < L) {
        bf16x2 lo = {(bf16)(sl[h][0] * mul), (bf16)(sl[h][1] * mul)};
        bf16x2 hi = {(bf16)(sl[h][2] * mul), (bf16)(sl[h][3] * mul)};
        uint2 w;
        w.x = __builtin_bit_cast(uint32_t, lo);
        w.y = __builtin_bit_cast(uint32_t, hi);
        *reinterpret_cast<uint2*>(base + (int64_t)rs * r_st + d0) = w;
      }
    }
  }
}

// store_rows through LDS: the wave's 32 rows are staged (bf16, row pitch SP)
// in `so`, a region only this wave touches, and leave as whole 16-byte
// chunks, D / 8 consecutive lanes per row.  From the accumulator layout a
// store instruction would write 8-byte pieces of 32 rows, one L2 request
// each.  One wave's LDS accesses complete in order, so no barrier separates
// the staging from the reads.
template <int D, int SP>
__device__ __forceinline__ void store_rows_lds(bf16* so, bf16* base, int64_t r_st, uint32_t row0, uint32_t L,
                                               int lane,
                                               const floatx16 (&t32)[BGeo<D>::NT32 > 0 ? BGeo<D>::NT32 : 1],
                                               const floatx4 (&sl)[2], float mul) {
  using G = BGeo<D>;
  static_assert(D % 8 == 0, "rows leave in 16-byte chunks");
  const int l32 = lane & 31, g = lane >> 5;
#pragma unroll
  for (int t = 0; t < G::NT32; ++t)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d0 = 32 * t + 8 * r4 + 4 * g;
      bf16x2 lo = {(bf16)(t32[t][4 * r4 + 0] * mul), (bf16)(t32[t][4 * r4 + 1] * mul)};
      bf16x2 hi = {(bf16)(t32[t][4 * r4 + 2] * mul), (bf16)(t32[t][4 * r4 + 3] * mul)};
      uint2 w;
      w.x = __builtin_bit_cast(uint32_t, lo);
      w.y = __builtin_bit_cast(uint32_t, hi);
      *reinterpret_cast<uint2*>(so + l32 * SP + d0) = w;
    }
  if constexpr (G::SLAB) {
    const int d0 = 32 * G::NT32 + 4 * (lane >> 4);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (d0 < D) {
        bf16x2 lo = {(bf16)(sl[h][0] * mul), (bf16)(sl[h][1] * mul)};
        bf16x2 hi = {(bf16)(sl[h][2] * mul), (bf16)(sl[h][3] * mul)};
        uint2 w;
        w.x = __builtin_bit_cast(uint32_t, lo);
        w.y = __builtin_bit_cast(uint32_t, hi);
        *reinterpret_cast<uint2*>(so + (16 * h + (lane & 15)) * SP + d0) = w;
      }
    }
  }
  constexpr int CH = D / 8, OCH = 32 * CH;
#pragma unroll
  for (int i = 0; i < (OCH + 63) / 64; ++i) {
    const int c = lane + 64 * i;
    const int row = c / CH, col = c - row * CH;
    if (c < OCH && row0 + (uint32_t)row < L)
      *reinterpret_cast<u32x4*>(base + (int64_t)(row0 + row) * r_st + col * 8) =
          *reinterpret_cast<const u32x4*>(so + row * SP + col * 8);
  }
}

// staged output row pitch (elements) for NW waves within `elems` of LDS:
// padded so that the rows of 16 consecutive lanes start on distinct banks,
// where the padded rows fit
template <int D, int NW>
constexpr int staged_pitch(int elems) {
  return NW * 32 * ((D % 16 == 8) ? D : D + 8) <= elems ? ((D % 16 == 8) ? D : D + 8) : D;
}

// ---------------------------------------------------------------------------
// dQ (and Delta): a work-group owns 32 NW queries of one unit and loops over
// the unit's keys in LDS tiles of 64 (K and V, double-buffered, the next tile
// prefetched into registers).  Per wave and 32-key step:
//   S^T = K Q'^T - lse2   (bias columns)     -> P^T = exp2(S^T)
//   dP^T = V dO^T - Delta (bias columns)     -> dZ^T = P^T * dP^T
//   dQ^T += K^T dZ^T
template <int D, int NW>
__global__ __launch_bounds__(NW * 64, 2) void attn_bwd_dq_kernel(BwdParams p) {
  using G = BGeo<D>;
  constexpr int KB = 64, NKT = KB / 32, NT = NW * 64, FT = NT / 2;
  constexpr int TCH = KB * G::CH;
  constexpr int NLOAD = (TCH + FT - 1) / FT;
  constexpr int TILE = 2 * KB * G::P;  // K then V
  static_assert(NW % 2 == 0, "K/V fetch split needs an even wave count");
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * TILE];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const BwdMap um = bwd_map(p, p.H);  // unit = a query head's (b, x, h)
  const uint32_t L = p.L, Lk = p.Lk;
  const int64_t q_base = bx_base(p, um.bx, p.b_q, p.x_q) + (int64_t)um.head * D;
  const int64_t o_base = bx_base(p, um.bx, p.b_o, p.x_o) + (int64_t)um.head * D;
  const int64_t kv_base = bx_base(p, um.bx, p.b_kv, p.x_kv) + (int64_t)(um.head / p.grp) * D;

  // padding columns of both buffers: D .. D + 2 are 1.0 (they multiply the
  // bias columns of the query side), the rest 0
  for (int e = threadIdx.x; e < 4 * KB; e += NT) {
    bf16* row = lds + (e / (2 * KB)) * TILE + (e % (2 * KB)) * G::P;
    for (int c = D; c < G::P; ++c) row[c] = (bf16)(c < D + 3 ? 1.0f : 0.0f);
  }

  // this wave's 32 queries: Q' and dO row fragments with the bias columns,
  // and Delta = rowsum(dO * O)
  const uint32_t q = um.blk * 32 * NW + 32 * wave + l32;
  const bool qv = q < L;
  bf16x8 qf[G::NDK], df[G::NDK], of[G::NDK];
  row_frags<D>(qv ? p.q + q_base + (int64_t)q * p.r_q : nullptr, g, qf);
  row_frags<D>(qv ? p.dout + o_base + (int64_t)q * p.r_o : nullptr, g, df);
  row_frags<D>(qv ? p.o + o_base + (int64_t)q * p.r_o : nullptr, g, of);
  float dl = 0.0f;
#pragma unroll
  for (int s = 0; s < G::NDK; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      dl += (float)df[s][e] * (float)of[s][e];
      qf[s][e] = (bf16)((float)qf[s][e] * p.c);
    }
  const float delta = dl + swap_halves(dl);
  const float lse2 = qv ? p.lse[(int64_t)um.unit * L + q] * kLog2e : 0.0f;
  if (qv && g == 0) p.delta[(int64_t)um.unit * L + q] = delta;
  if (g == G::GB) {
    const Bf16x3 nl = neg_split3(lse2), nd = neg_split3(delta);
#pragma unroll
    for (int e = 0; e < 3; ++e) {
      qf[G::SB][e] = nl.t[e];
      df[G::SB][e] = nd.t[e];
    }
  }

  // tile fetch: waves [0, NW/2) K, the others V; rows past L read as zero
  const bool fetch_v = wave >= NW / 2;
  const int ft = threadIdx.x % FT;
  const uint32_t row_bytes = (uint32_t)p.r_kv * 2u;
  uint32_t voff[NLOAD];
  int lofs[NLOAD];
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int c = ft + i * FT;
    const int row = c / G::CH, col = c - row * G::CH;
    voff[i] = (uint32_t)row * row_bytes + (uint32_t)col * 16u;
    lofs[i] = (fetch_v ? KB * G::P : 0) + row * G::P + col * 8;
  }
  u32x4 pre[NLOAD];
  auto fetch = [&](uint32_t kb) {
    const uint32_t rows = kb < Lk ? min(Lk - kb, (uint32_t)KB) : 0u;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc((fetch_v ? p.v : p.k) + kv_base + (int64_t)kb * p.r_kv, rows * row_bytes);
#pragma unroll
    for (int i = 0; i < NLOAD; ++i)
      if (ft + i * FT < TCH) pre[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i], 0, 0);
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NLOAD; ++i)
      if (ft + i * FT < TCH) *reinterpret_cast<u32x4*>(lds + buf * TILE + lofs[i]) = pre[i];
  };

  floatx16 dqt[G::NT32 > 0 ? G::NT32 : 1];
  floatx4 dqs[2];
#pragma unroll
  for (int t = 0; t < G::NT32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqt[t][r] = 0.0f;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int r = 0; r < 4; ++r) dqs[h][r] = 0.0f;

  const uint32_t n_kb = (Lk + KB - 1) / KB;
  fetch(0);
  stash(0);
  __syncthreads();
  for (uint32_t it = 0; it < n_kb; ++it) {
    const uint32_t kb = it * KB;
    const bool more = it + 1 < n_kb;
    if (more) fetch(kb + KB);
    const bf16* k_lds = lds + (it & 1) * TILE;
    const bf16* v_lds = k_lds + KB * G::P;

    floatx16 s[NKT], dp[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] = dp[kt][r] = 0.0f;
#pragma unroll
    for (int st = 0; st < G::NDK; ++st)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(k_lds + (32 * kt + l32) * G::P + 16 * st + 8 * g);
        const bf16x8 va = *reinterpret_cast<const bf16x8*>(v_lds + (32 * kt + l32) * G::P + 16 * st + 8 * g);
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[st], s[kt], 0, 0, 0);
        dp[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, df[st], dp[kt], 0, 0, 0);
      }
    // lane (n + 32g) holds keys kb + 32kt + 8(r/4) + 4g + r%4 of query n.
    // Keys past Lk (only the last tile holds any) get score -inf, so P = +0
    // there; the branch keeps the key compares out of every other tile.
    if (kb + KB > Lk) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kb + 32 * kt + (r / 4) * 8 + 4 * g + (r % 4) >= Lk) s[kt][r] = -INFINITY;
    }
    bf16x8 zb[NKT][2];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) zb[kt][r / 8][r % 8] = (bf16)(__builtin_amdgcn_exp2f(s[kt][r]) * dp[kt][r]);
    // dQ^T += K^T dZ^T
#pragma unroll
    for (int t = 0; t < G::NT32; ++t)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
          dqt[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              tr_frag32(k_lds, G::P, 32 * kt + 16 * kk, 32 * t, lane), zb[kt][kk], dqt[t], 0, 0, 0);
    if constexpr (G::SLAB) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const bf16x8 a = tr_slab(k_lds, G::P, 32 * kt, 32 * G::NT32, lane);
        bf16x8 b0, b1;
        slab_b(zb[kt][0], zb[kt][1], b0, b1);
        dqs[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b0, dqs[0], 0, 0, 0);
        dqs[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b1, dqs[1], 0, 0, 0);
      }
    }
    if (more) stash((it + 1) & 1);
    __syncthreads();
  }
  constexpr int SP = staged_pitch<D, NW>(2 * TILE);
  static_assert(NW * 32 * SP <= 2 * TILE, "the output staging fits the LDS tiles");
  store_rows_lds<D, SP>(lds + wave * 32 * SP, p.dq + q_base, p.r_q, um.blk * 32 * NW + 32 * wave, L, lane, dqt,
                        dqs, p.scale);
}

// ---------------------------------------------------------------------------
// dK and dV: a work-group owns 32 NW keys of one unit and loops over the
// unit's queries in LDS tiles of 64 (Q' and dO, with their bias columns,
// double-buffered, the next tile prefetched into registers).  Per wave and
// 32-query step:
//   S = Q' K^T - lse2  -> P = exp2(S);   dP = dO V^T - Delta -> dZ = P * dP
//   dV^T += dO^T P;    dK^T += Q'^T dZ
// With grouped key/value heads the keys belong to a key/value head, and the
// query tiles of every query head of its group are visited in turn, so dK and
// dV are the sums over the group (in a fixed order).
// Query rows past L are zero with zero bias, so they contribute nothing.
template <int D, int NW>
__global__ __launch_bounds__(NW * 64, 2) void attn_bwd_dkv_kernel(BwdParams p) {
  using G = BGeo<D>;
  constexpr int QB = 64, NT = NW * 64, FT = NT / 2;
  constexpr int TCH = QB * G::CH;
  constexpr int NLOAD = (TCH + FT - 1) / FT;
  constexpr int TILE = 2 * QB * G::P;  // Q' then dO
  static_assert(NW % 2 == 0 && FT >= QB, "fetch split");
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * TILE];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const BwdMap um = bwd_map(p, p.H / p.grp);  // unit = a key/value head's (b, x, h_kv)
  const uint32_t L = p.L, Lk = p.Lk;
  const int64_t kv_base = bx_base(p, um.bx, p.b_kv, p.x_kv) + (int64_t)um.head * D;
  const int64_t q_bx = bx_base(p, um.bx, p.b_q, p.x_q), o_bx = bx_base(p, um.bx, p.b_o, p.x_o);
  const uint32_t hq0 = um.head * p.grp;                 // first query head of the group

  // padding columns past the bias terms: 0 (the bias columns are rewritten per tile)
  for (int e = threadIdx.x; e < 4 * QB; e += NT) {
    bf16* row = lds + (e / (2 * QB)) * TILE + (e % (2 * QB)) * G::P;
    for (int c = D + 3; c < G::P; ++c) row[c] = (bf16)0.0f;
  }

  // this wave's 32 keys: K and V row fragments, bias columns 1.0
  const uint32_t key0 = um.blk * 32 * NW + 32 * wave;
  const uint32_t key = key0 + l32;
  const bool kv = key < Lk;
  bf16x8 kf[G::NDK], vf[G::NDK];
  row_frags<D>(kv ? p.k + kv_base + (int64_t)key * p.r_kv : nullptr, g, kf);
  row_frags<D>(kv ? p.v + kv_base + (int64_t)key * p.r_kv : nullptr, g, vf);
  if (g == G::GB) {
    kf[G::SB][0] = kf[G::SB][1] = kf[G::SB][2] = (bf16)1.0f;
    vf[G::SB][0] = vf[G::SB][1] = vf[G::SB][2] = (bf16)1.0f;
  }

  // tile fetch: waves [0, NW/2) Q (scaled to Q' when stashed), the others dO;
  // threads ft < QB of each half also fetch the row's lse or Delta
  const bool fetch_do = wave >= NW / 2;
  const int ft = threadIdx.x % FT;
  const uint32_t qrow_bytes = (uint32_t)p.r_q * 2u, orow_bytes = (uint32_t)p.r_o * 2u;
  const uint32_t row_bytes = fetch_do ? orow_bytes : qrow_bytes;
  uint32_t voff[NLOAD];
  int lofs[NLOAD];
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int c = ft + i * FT;
    const int row = c / G::CH, col = c - row * G::CH;
    voff[i] = (uint32_t)row * row_bytes + (uint32_t)col * 16u;
    lofs[i] = (fetch_do ? QB * G::P : 0) + row * G::P + col * 8;
  }
  const float* stat = fetch_do ? p.delta : p.lse;
  u32x4 pre[NLOAD];
  float pstat = 0.0f;
  // tile `it` of the group's query heads: head hq0 + it / n_qt, queries from (it % n_qt) QB
  const uint32_t n_qt = (L + QB - 1) / QB;
  auto fetch = [&](uint32_t it) {
    const uint32_t hq = hq0 + it / n_qt, qb = (it % n_qt) * QB;
    const uint32_t rows = qb < L ? min(L - qb, (uint32_t)QB) : 0u;
    const bf16* base = fetch_do ? p.dout + o_bx + (int64_t)hq * D + (int64_t)qb * p.r_o
                                : p.q + q_bx + (int64_t)hq * D + (int64_t)qb * p.r_q;
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(base, rows * row_bytes);
#pragma unroll
    for (int i = 0; i < NLOAD; ++i)
      if (ft + i * FT < TCH) pre[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i], 0, 0);
    const uint32_t unit_q = um.bx * p.H + hq;
    pstat = (ft < QB && qb + ft < L) ? stat[(int64_t)unit_q * L + qb + ft] : 0.0f;
  };
  auto stash = [&](int buf) {
    bf16* t = lds + buf * TILE;
#pragma unroll
    for (int i = 0; i < NLOAD; ++i)
      if (ft + i * FT < TCH) {
        u32x4 v = pre[i];
        if (!fetch_do) {  // Q' = Q * scale * log2(e), rounded as in the forward
          bf16x8 x = __builtin_bit_cast(bf16x8, v);
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = (bf16)((float)x[e] * p.c);
          v = __builtin_bit_cast(u32x4, x);
        }
        *reinterpret_cast<u32x4*>(t + lofs[i]) = v;
      }
    if (ft < QB) {  // bias terms of row ft: -(lse * log2 e) for Q', -Delta for dO
      const float x = fetch_do ? pstat : pstat * kLog2e;
      bf16* row = t + (fetch_do ? QB * G::P : 0) + ft * G::P;
      const Bf16x3 nx = neg_split3(x);
      row[D] = nx.t[0];
      row[D + 1] = nx.t[1];
      row[D + 2] = nx.t[2];
    }
  };

  floatx16 dvt[G::NT32 > 0 ? G::NT32 : 1], dkt[G::NT32 > 0 ? G::NT32 : 1];
  floatx4 dvs[2], dks[2];
#pragma unroll
  for (int t = 0; t < G::NT32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dvt[t][r] = dkt[t][r] = 0.0f;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int r = 0; r < 4; ++r) dvs[h][r] = dks[h][r] = 0.0f;

  const uint32_t n_it = n_qt * p.grp;
  fetch(0);
  stash(0);
  __syncthreads();
  for (uint32_t it = 0; it < n_it; ++it) {
    const bool more = it + 1 < n_it;
    if (more) fetch(it + 1);
    const bf16* q_lds = lds + (it & 1) * TILE;
    const bf16* o_lds = q_lds + QB * G::P;
    if (key0 < Lk) {  // wave-uniform: waves whose keys are all past Lk only fetch
#pragma unroll
      for (int sub = 0; sub < QB / 32; ++sub) {
        const int q0 = 32 * sub;
        floatx16 s, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.0f;
#pragma unroll
        for (int st = 0; st < G::NDK; ++st) {
          const bf16x8 qa = *reinterpret_cast<const bf16x8*>(q_lds + (q0 + l32) * G::P + 16 * st + 8 * g);
          const bf16x8 da = *reinterpret_cast<const bf16x8*>(o_lds + (q0 + l32) * G::P + 16 * st + 8 * g);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kf[st], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vf[st], dp, 0, 0, 0);
        }
        // lane (n + 32g) holds queries q0 + 8(r/4) + 4g + r%4 of key n
        bf16x8 pb[2], zb[2];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pr = __builtin_amdgcn_exp2f(s[r]);
          pb[r / 8][r % 8] = (bf16)pr;
          zb[r / 8][r % 8] = (bf16)(pr * dp[r]);
        }
#pragma unroll
        for (int t = 0; t < G::NT32; ++t)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            dvt[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                tr_frag32(o_lds, G::P, q0 + 16 * kk, 32 * t, lane), pb[kk], dvt[t], 0, 0, 0);
            dkt[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                tr_frag32(q_lds, G::P, q0 + 16 * kk, 32 * t, lane), zb[kk], dkt[t], 0, 0, 0);
          }
        if constexpr (G::SLAB) {
          bf16x8 b0, b1;
          const bf16x8 ao = tr_slab(o_lds, G::P, q0, 32 * G::NT32, lane);
          slab_b(pb[0], pb[1], b0, b1);
          dvs[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ao, b0, dvs[0], 0, 0, 0);
          dvs[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ao, b1, dvs[1], 0, 0, 0);
          const bf16x8 aq = tr_slab(q_lds, G::P, q0, 32 * G::NT32, lane);
          slab_b(zb[0], zb[1], b0, b1);
          dks[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, b0, dks[0], 0, 0, 0);
          dks[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, b1, dks[1], 0, 0, 0);
        }
      }
    }
    if (more) stash((it + 1) & 1);
    __syncthreads();
  }
  // dK = scale * dZ^T Q = ln 2 * dZ^T Q'
  constexpr int SP = staged_pitch<D, NW>(2 * TILE);
  static_assert(NW * 32 * SP <= 2 * TILE, "the output staging fits the LDS tiles");
  bf16* so = lds + wave * 32 * SP;
  store_rows_lds<D, SP>(so, p.dv + kv_base, p.r_kv, key0, Lk, lane, dvt, dvs, 1.0f);
  store_rows_lds<D, SP>(so, p.dk + kv_base, p.r_kv, key0, Lk, lane, dkt, dks, kLn2);
}

// ---------------------------------------------------------------------------
// Short units (L, Lk <= 32 NW, one query head per key/value head): one
// work-group owns a whole unit.  Q', dO, K and V (and dO * O for Delta) are
// read from global memory once, with coalesced 16-byte loads, into LDS tiles
// whose bias columns are set as in the two kernels above (K, V: 1.0 on rows
// below Lk, 0 past it -- so keys past Lk get dZ = 0 without a mask; Q', dO:
// -lse2 and -Delta on rows below L, 0 past it).  Then, from LDS only, wave w
// runs the dQ loop for queries 32w .. 32w + 31 over all keys, and the dK/dV
// loop for keys 32w .. 32w + 31 over all queries (see the wave roles below).  The scores are computed
// twice, as in the two-kernel path, but the unit's rows cross HBM once.  The
// grid is persistent: while a unit is computed from LDS, the next unit's rows
// are already in flight in registers.
// 2 NW waves: waves [0, NW) run the dQ loops, waves [NW, 2 NW) the dK/dV loops.
template <int D, int NW>
__global__ __launch_bounds__(NW * 128, 1) void attn_bwd_short_kernel(BwdParams p) {
  using G = BGeo<D>;
  constexpr int R = 32 * NW, NT = NW * 128;
  constexpr int TILE = R * G::P;
  constexpr int NCH = R * G::CH;                 // 16-byte chunks of one tensor's rows
  constexpr int NLOAD = (NCH + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) bf16 lds[4 * TILE];
  __shared__ float dpart[NCH];
  bf16* qs = lds;             // Q'
  bf16* os = lds + TILE;      // dO
  bf16* ks = lds + 2 * TILE;  // K
  bf16* vs = lds + 3 * TILE;  // V

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const uint32_t L = p.L, Lk = p.Lk;

  // Persistent: this work-group's units are 8 contiguous ranges, one per XCD
  // (work-group i runs on XCD i % 8), the work-groups of an XCD interleaved
  // over its range, so neighbouring heads of a token row share an L2.  While
  // one unit is computed from LDS, the next unit's rows are in flight in
  // registers.
  const uint32_t nb = gridDim.x, n_units = p.n_blocks;
  uint32_t u, u_end, u_step;
  if ((nb & 7u) == 0) {
    const uint32_t xcd = blockIdx.x & 7u;
    u = (uint32_t)(((uint64_t)n_units * xcd) >> 3) + (blockIdx.x >> 3);
    u_end = (uint32_t)(((uint64_t)n_units * (xcd + 1)) >> 3);
    u_step = nb >> 3;
  } else {
    u = blockIdx.x;
    u_end = n_units;
    u_step = nb;
  }

  // padding columns, the same for every unit (the bias terms of Q' and dO are
  // written per unit): K, V columns D .. D + 2 are 1.0 on rows below Lk
  for (int r = threadIdx.x; r < R; r += NT) {
    const bf16 kb = (bf16)((uint32_t)r < Lk ? 1.0f : 0.0f);
    ks[r * G::P + D] = ks[r * G::P + D + 1] = ks[r * G::P + D + 2] = kb;
    vs[r * G::P + D] = vs[r * G::P + D + 1] = vs[r * G::P + D + 2] = kb;
    for (int c = D + 3; c < G::P; ++c)
      qs[r * G::P + c] = os[r * G::P + c] = ks[r * G::P + c] = vs[r * G::P + c] = (bf16)0.0f;
  }

  // ---- a unit's rows: chunk c = row c / CH, 16 bytes at column 8 (c % CH);
  // rows past L (Lk) fall outside the buffer ranges and read as zero
  u32x4 cq[NLOAD], cd[NLOAD], co[NLOAD], ck[NLOAD], cv[NLOAD];
  auto issue = [&](uint32_t unit) {
    const uint32_t head = unit % p.H, bx = unit / p.H;  // (b, x, h): query head = key/value head
    const int64_t qb = bx_base(p, bx, p.b_q, p.x_q) + (int64_t)head * D;
    const int64_t ob = bx_base(p, bx, p.b_o, p.x_o) + (int64_t)head * D;
    const int64_t kb = bx_base(p, bx, p.b_kv, p.x_kv) + (int64_t)head * D;
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(p.q + qb, L * (uint32_t)p.r_q * 2u);
    const __amdgpu_buffer_rsrc_t rd = make_rsrc(p.dout + ob, L * (uint32_t)p.r_o * 2u);
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(p.o + ob, L * (uint32_t)p.r_o * 2u);
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(p.k + kb, Lk * (uint32_t)p.r_kv * 2u);
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.v + kb, Lk * (uint32_t)p.r_kv * 2u);
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int c = threadIdx.x + i * NT;
      if (c < NCH) {
        const uint32_t row = c / G::CH, col = c - row * G::CH;
        const uint32_t oq = row * (uint32_t)p.r_q * 2u + col * 16u;
        const uint32_t oo = row * (uint32_t)p.r_o * 2u + col * 16u;
        const uint32_t okv = row * (uint32_t)p.r_kv * 2u + col * 16u;
        cq[i] = __builtin_amdgcn_raw_buffer_load_b128(rq, oq, 0, 0);
        cd[i] = __builtin_amdgcn_raw_buffer_load_b128(rd, oo, 0, 0);
        co[i] = __builtin_amdgcn_raw_buffer_load_b128(ro, oo, 0, 0);
        ck[i] = __builtin_amdgcn_raw_buffer_load_b128(rk, okv, 0, 0);
        cv[i] = __builtin_amdgcn_raw_buffer_load_b128(rv, okv, 0, 0);
      }
    }
  };
  if (u < u_end) issue(u);
  for (; u < u_end; u += u_step) {
    const uint32_t unit = u;
    const uint32_t head = unit % p.H, bx = unit / p.H;
    const int64_t q_base = bx_base(p, bx, p.b_q, p.x_q) + (int64_t)head * D;
    const int64_t o_base = bx_base(p, bx, p.b_o, p.x_o) + (int64_t)head * D;
    const int64_t kv_base = bx_base(p, bx, p.b_kv, p.x_kv) + (int64_t)head * D;
    __syncthreads();  // the previous unit's LDS reads are done (and the padding is written)
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int c = threadIdx.x + i * NT;
      if (c < NCH) {
        const int row = c / G::CH, col = c - row * G::CH;
        const int off = row * G::P + col * 8;
        bf16x8 x = __builtin_bit_cast(bf16x8, cq[i]);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = (bf16)((float)x[e] * p.c);  // Q' as in the forward
        *reinterpret_cast<bf16x8*>(qs + off) = x;
        *reinterpret_cast<u32x4*>(os + off) = cd[i];
        *reinterpret_cast<u32x4*>(ks + off) = ck[i];
        *reinterpret_cast<u32x4*>(vs + off) = cv[i];
        const bf16x8 dv8 = __builtin_bit_cast(bf16x8, cd[i]), ov8 = __builtin_bit_cast(bf16x8, co[i]);
        float d = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d += (float)dv8[e] * (float)ov8[e];
        dpart[c] = d;
      }
    }
    __syncthreads();
    // Delta = rowsum(dO * O) and the bias terms: -(lse * log2 e) on Q', -Delta on dO
    for (int r = threadIdx.x; r < R; r += NT) {
      float delta = 0.0f, lse2 = 0.0f;
      if ((uint32_t)r < L) {
#pragma unroll
        for (int col = 0; col < G::CH; ++col) delta += dpart[r * G::CH + col];
        lse2 = p.lse[(int64_t)unit * L + r] * kLog2e;
        p.delta[(int64_t)unit * L + r] = delta;
      }
      const Bf16x3 nl = neg_split3(lse2), nd = neg_split3(delta);
#pragma unroll
      for (int e = 0; e < 3; ++e) {
        qs[r * G::P + D + e] = nl.t[e];
        os[r * G::P + D + e] = nd.t[e];
      }
    }
    __syncthreads();
    if (u + u_step < u_end) issue(u + u_step);

    const int row0 = 32 * (wave % NW);
    // ---- dQ for queries row0 .. row0 + 31 over all keys:
    //   S^T = K Q'^T - lse2 -> P^T;  dP^T = V dO^T - Delta;  dZ^T = P^T * dP^T;  dQ^T += K^T dZ^T
    if (wave < NW && (uint32_t)row0 < L) {
      bf16x8 qf[G::NDK], df[G::NDK];
#pragma unroll
      for (int st = 0; st < G::NDK; ++st) {
        qf[st] = *reinterpret_cast<const bf16x8*>(qs + (row0 + l32) * G::P + 16 * st + 8 * g);
        df[st] = *reinterpret_cast<const bf16x8*>(os + (row0 + l32) * G::P + 16 * st + 8 * g);
      }
      floatx16 dqt[G::NT32 > 0 ? G::NT32 : 1];
      floatx4 dqs[2];
#pragma unroll
      for (int t = 0; t < G::NT32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) dqt[t][r] = 0.0f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) dqs[h][r] = 0.0f;
      for (uint32_t k0 = 0; k0 < Lk; k0 += 32) {
        floatx16 sc, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] = dp[r] = 0.0f;
#pragma unroll
        for (int st = 0; st < G::NDK; ++st) {
          const bf16x8 ka = *reinterpret_cast<const bf16x8*>(ks + (k0 + l32) * G::P + 16 * st + 8 * g);
          const bf16x8 va = *reinterpret_cast<const bf16x8*>(vs + (k0 + l32) * G::P + 16 * st + 8 * g);
          sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[st], sc, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, df[st], dp, 0, 0, 0);
        }
        bf16x8 zb[2];
#pragma unroll
        for (int r = 0; r < 16; ++r) zb[r / 8][r % 8] = (bf16)(__builtin_amdgcn_exp2f(sc[r]) * dp[r]);
#pragma unroll
        for (int t = 0; t < G::NT32; ++t)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
            dqt[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag32(ks, G::P, k0 + 16 * kk, 32 * t, lane),
                                                             zb[kk], dqt[t], 0, 0, 0);
        if constexpr (G::SLAB) {
          const bf16x8 a = tr_slab(ks, G::P, k0, 32 * G::NT32, lane);
          bf16x8 b0, b1;
          slab_b(zb[0], zb[1], b0, b1);
          dqs[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b0, dqs[0], 0, 0, 0);
          dqs[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b1, dqs[1], 0, 0, 0);
        }
      }
      store_rows<D>(p.dq + q_base, p.r_q, row0, L, lane, dqt, dqs, p.scale);
    }

    // ---- dK, dV for keys row0 .. row0 + 31 over all queries:
    //   S = Q' K^T - lse2 -> P;  dP = dO V^T - Delta;  dZ = P * dP;  dV^T += dO^T P;  dK^T += Q'^T dZ
    if (wave >= NW && (uint32_t)row0 < Lk) {
      bf16x8 kf[G::NDK], vf[G::NDK];
#pragma unroll
      for (int st = 0; st < G::NDK; ++st) {
        kf[st] = *reinterpret_cast<const bf16x8*>(ks + (row0 + l32) * G::P + 16 * st + 8 * g);
        vf[st] = *reinterpret_cast<const bf16x8*>(vs + (row0 + l32) * G::P + 16 * st + 8 * g);
      }
      floatx16 dvt[G::NT32 > 0 ? G::NT32 : 1], dkt[G::NT32 > 0 ? G::NT32 : 1];
      floatx4 dvs[2], dks[2];
#pragma unroll
      for (int t = 0; t < G::NT32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) dvt[t][r] = dkt[t][r] = 0.0f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) dvs[h][r] = dks[h][r] = 0.0f;
      for (uint32_t q0 = 0; q0 < L; q0 += 32) {
        floatx16 sc, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] = dp[r] = 0.0f;
#pragma unroll
        for (int st = 0; st < G::NDK; ++st) {
          const bf16x8 qa = *reinterpret_cast<const bf16x8*>(qs + (q0 + l32) * G::P + 16 * st + 8 * g);
          const bf16x8 da = *reinterpret_cast<const bf16x8*>(os + (q0 + l32) * G::P + 16 * st + 8 * g);
          sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kf[st], sc, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vf[st], dp, 0, 0, 0);
        }
        bf16x8 pb[2], zb[2];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pr = __builtin_amdgcn_exp2f(sc[r]);
          pb[r / 8][r % 8] = (bf16)pr;
          zb[r / 8][r % 8] = (bf16)(pr * dp[r]);
        }
#pragma unroll
        for (int t = 0; t < G::NT32; ++t)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            dvt[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag32(os, G::P, q0 + 16 * kk, 32 * t, lane),
                                                             pb[kk], dvt[t], 0, 0, 0);
            dkt[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag32(qs, G::P, q0 + 16 * kk, 32 * t, lane),
                                                             zb[kk], dkt[t], 0, 0, 0);
          }
        if constexpr (G::SLAB) {
          bf16x8 b0, b1;
          const bf16x8 ao = tr_slab(os, G::P, q0, 32 * G::NT32, lane);
          slab_b(pb[0], pb[1], b0, b1);
          dvs[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ao, b0, dvs[0], 0, 0, 0);
          dvs[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ao, b1, dvs[1], 0, 0, 0);
          const bf16x8 aq = tr_slab(qs, G::P, q0, 32 * G::NT32, lane);
          slab_b(zb[0], zb[1], b0, b1);
          dks[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, b0, dks[0], 0, 0, 0);
          dks[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, b1, dks[1], 0, 0, 0);
        }
      }
      store_rows<D>(p.dv + kv_base, p.r_kv, row0, Lk, lane, dvt, dvs, 1.0f);
      store_rows<D>(p.dk + kv_base, p.r_kv, row0, Lk, lane, dkt, dks, kLn2);
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 path: plain FMA loops.  One thread per (unit, row, 32-column slice):
// the dQ kernel's units are query heads (rows: queries), the dK/dV kernel's
// key/value heads (rows: keys; it visits every query head of the group).
constexpr int DC = 32;

struct BwdParamsF {
  const float* q;
  const float* k;
  const float* v;
  const float* o;
  const float* dout;
  const float* lse;
  float* dq;
  float* dk;
  float* dv;
  float* delta;
  int64_t b_q, x_q, r_q, b_kv, x_kv, r_kv, b_o, x_o, r_o;
  int64_t X, H, L, Lk, grp, D, n_dc;
  float scale;
};

__device__ __forceinline__ float dotf(const float* a, const float* b, int64_t n) {
  float s = 0.0f;
  for (int64_t d = 0; d < n; ++d) s = fmaf(a[d], b[d], s);
  return s;
}

__global__ __launch_bounds__(256) void attn_bwd_f32_dq_kernel(BwdParamsF p, int64_t total) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= total) return;
  const int64_t c0 = (tid % p.n_dc) * DC, ur = tid / p.n_dc;
  const int64_t nc = min((int64_t)DC, p.D - c0);
  const int64_t row = ur % p.L, unit = ur / p.L;
  const int64_t h = unit % p.H, bx = unit / p.H, xx = bx % p.X, bb = bx / p.X;
  const float* qrow = p.q + bb * p.b_q + xx * p.x_q + h * p.D + row * p.r_q;
  const int64_t ob = bb * p.b_o + xx * p.x_o + h * p.D + row * p.r_o;
  const int64_t kvb = bb * p.b_kv + xx * p.x_kv + (h / p.grp) * p.D;
  const float* drow = p.dout + ob;
  const float delta = dotf(drow, p.o + ob, p.D);
  const float lse = p.lse[unit * p.L + row];
  if (c0 == 0) p.delta[unit * p.L + row] = delta;
  float acc[DC];
#pragma unroll
  for (int c = 0; c < DC; ++c) acc[c] = 0.0f;
  for (int64_t j = 0; j < p.Lk; ++j) {
    const float* krow = p.k + kvb + j * p.r_kv;
    const float pr = expf(dotf(qrow, krow, p.D) * p.scale - lse);
    const float dz = pr * (dotf(drow, p.v + kvb + j * p.r_kv, p.D) - delta);
#pragma unroll
    for (int c = 0; c < DC; ++c)
      if (c < nc) acc[c] = fmaf(dz, krow[c0 + c], acc[c]);
  }
  float* out = p.dq + bb * p.b_q + xx * p.x_q + h * p.D + row * p.r_q + c0;
#pragma unroll
  for (int c = 0; c < DC; ++c)
    if (c < nc) out[c] = acc[c] * p.scale;
}

__global__ __launch_bounds__(256) void attn_bwd_f32_dkv_kernel(BwdParamsF p, int64_t total) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= total) return;
  const int64_t Hkv = p.H / p.grp;
  const int64_t c0 = (tid % p.n_dc) * DC, ur = tid / p.n_dc;
  const int64_t nc = min((int64_t)DC, p.D - c0);
  const int64_t key = ur % p.Lk, unit = ur / p.Lk;
  const int64_t hk = unit % Hkv, bx = unit / Hkv, xx = bx % p.X, bb = bx / p.X;
  const int64_t kvb = bb * p.b_kv + xx * p.x_kv + hk * p.D + key * p.r_kv;
  const float* krow = p.k + kvb;
  const float* vrow = p.v + kvb;
  float ak[DC], av[DC];
#pragma unroll
  for (int c = 0; c < DC; ++c) ak[c] = av[c] = 0.0f;
  for (int64_t hq = hk * p.grp; hq < (hk + 1) * p.grp; ++hq) {
    const int64_t uq = bx * p.H + hq;
    for (int64_t i = 0; i < p.L; ++i) {
      const float* qrow = p.q + bb * p.b_q + xx * p.x_q + hq * p.D + i * p.r_q;
      const float* drow = p.dout + bb * p.b_o + xx * p.x_o + hq * p.D + i * p.r_o;
      const float pr = expf(dotf(qrow, krow, p.D) * p.scale - p.lse[uq * p.L + i]);
      const float dz = pr * (dotf(drow, vrow, p.D) - p.delta[uq * p.L + i]);
#pragma unroll
      for (int c = 0; c < DC; ++c)
        if (c < nc) {
          ak[c] = fmaf(dz, qrow[c0 + c], ak[c]);
          av[c] = fmaf(pr, drow[c0 + c], av[c]);
        }
    }
  }
  float* ok = p.dk + kvb + c0;
  float* ov = p.dv + kvb + c0;
#pragma unroll
  for (int c = 0; c < DC; ++c)
    if (c < nc) {
      ok[c] = ak[c] * p.scale;
      ov[c] = av[c];
    }
}

template <typename P>
void fill_common(P& p, const AttnBwdArgs& a) {
  p.b_q = a.q_strides[0];
  p.x_q = a.q_strides[1];
  p.r_q = a.q_strides[2];
  p.b_kv = a.kv_strides[0];
  p.x_kv = a.kv_strides[1];
  p.r_kv = a.kv_strides[2];
  p.b_o = a.o_strides[0];
  p.x_o = a.o_strides[1];
  p.r_o = a.o_strides[2];
  p.lse = a.lse;
  p.delta = a.delta;
}

template <int D, int NW>
int launch_bwd_nw(const AttnBwdArgs& a, hipStream_t s) {
  BwdParams p;
  p.q = static_cast<const bf16*>(a.q);
  p.k = static_cast<const bf16*>(a.k);
  p.v = static_cast<const bf16*>(a.v);
  p.o = static_cast<const bf16*>(a.o);
  p.dout = static_cast<const bf16*>(a.dout);
  p.dq = static_cast<bf16*>(a.dq);
  p.dk = static_cast<bf16*>(a.dk);
  p.dv = static_cast<bf16*>(a.dv);
  fill_common(p, a);
  p.X = (uint32_t)a.X;
  p.H = (uint32_t)a.H;
  p.L = (uint32_t)a.L;
  p.Lk = (uint32_t)a.Lk;
  p.grp = (uint32_t)(a.H / a.Hkv);
  p.c = a.scale * kLog2e;
  p.scale = a.scale;
  // dQ: query heads x blocks of 32 NW queries
  const int64_t nq = (a.L + 32 * NW - 1) / (32 * NW);
  const int64_t bq = a.B * a.X * a.H * nq;
  if (bq == 0) return DSP_OK;
  p.n_blk = (uint32_t)nq;
  p.n_blocks = (uint32_t)bq;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, NW>), dim3((uint32_t)bq), dim3(NW * 64), 0, s, p);
  int st = last_launch_status();
  if (st != DSP_OK) return st;
  // dK, dV: key/value heads x blocks of 32 NW keys
  const int64_t nk = (a.Lk + 32 * NW - 1) / (32 * NW);
  const int64_t bk = a.B * a.X * a.Hkv * nk;
  if (bk == 0) return DSP_OK;
  p.n_blk = (uint32_t)nk;
  p.n_blocks = (uint32_t)bk;
  hipLaunchKernelGGL((attn_bwd_dkv_kernel<D, NW>), dim3((uint32_t)bk), dim3(NW * 64), 0, s, p);
  return last_launch_status();
}

template <int D, int NW>
int launch_bwd_short(const AttnBwdArgs& a, hipStream_t s) {
  BwdParams p;
  p.q = static_cast<const bf16*>(a.q);
  p.k = static_cast<const bf16*>(a.k);
  p.v = static_cast<const bf16*>(a.v);
  p.o = static_cast<const bf16*>(a.o);
  p.dout = static_cast<const bf16*>(a.dout);
  p.dq = static_cast<bf16*>(a.dq);
  p.dk = static_cast<bf16*>(a.dk);
  p.dv = static_cast<bf16*>(a.dv);
  fill_common(p, a);
  p.X = (uint32_t)a.X;
  p.H = (uint32_t)a.H;
  p.L = (uint32_t)a.L;
  p.Lk = (uint32_t)a.Lk;
  p.grp = 1;
  p.c = a.scale * kLog2e;
  p.scale = a.scale;
  const int64_t units = a.B * a.X * a.H;
  if (units == 0) return DSP_OK;
  p.n_blk = 1;
  p.n_blocks = (uint32_t)units;
  // persistent grid: as many work-groups as are resident at once (the
  // runtime's occupancy for this kernel: registers and LDS), a multiple of 8
  // (whole XCD ranges)
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1 ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_bwd_short_kernel<D, NW>, NW * 128, 0) !=
          hipSuccess ||
      per_cu < 1)
    return DSP_ERR_HIP;
  int64_t blocks = std::min<int64_t>(units, (int64_t)cus * per_cu);
  if (blocks >= 8) blocks &= ~int64_t(7);
  hipLaunchKernelGGL((attn_bwd_short_kernel<D, NW>), dim3((uint32_t)blocks), dim3(NW * 128), 0, s, p);
  return last_launch_status();
}

template <int D>
int launch_bwd_d(const AttnBwdArgs& a, hipStream_t s) {
  const int64_t L = std::max(a.L, a.Lk);
#if DSP_ATTN_BWD_SHORT
  // short units with one query head per key/value head: one work-group per unit
  if (a.H == a.Hkv && L <= 128 && a.L > 0 && a.Lk > 0) {
    if (L <= 32) return launch_bwd_short<D, 1>(a, s);
    if (L <= 64) return launch_bwd_short<D, 2>(a, s);
    return launch_bwd_short<D, 4>(a, s);
  }
#endif
  if (L <= 64) return launch_bwd_nw<D, 2>(a, s);
  if (L <= 128) return launch_bwd_nw<D, 4>(a, s);
  return launch_bwd_nw<D, 8>(a, s);
}

}  // namespace

bool attn_bwd_bf16_fits(const AttnBwdArgs& a) {
  // block indices, and the byte ranges of a 64-row tile, are 32-bit
  const int64_t L = std::max(a.L, a.Lk);
  const int64_t blocks = a.B * a.X * a.H * ((L + 63) / 64);
  return blocks < (int64_t(1) << 31) && L < (int64_t(1) << 31) &&
         64 * a.q_strides[2] * 2 < (int64_t(1) << 31) && 64 * a.kv_strides[2] * 2 < (int64_t(1) << 31) &&
         64 * a.o_strides[2] * 2 < (int64_t(1) << 31) && (int64_t)(a.H / a.Hkv) * ((a.L + 63) / 64) < (int64_t(1) << 31);
}

int launch_attn_bwd_bf16(const AttnBwdArgs& a, hipStream_t s) {
  if (!attn_bwd_bf16_fits(a)) return DSP_ERR_SHAPE;
  switch (a.D) {
    case 16: return launch_bwd_d<16>(a, s);
    case 32: return launch_bwd_d<32>(a, s);
    case 64: return launch_bwd_d<64>(a, s);
    case 72: return launch_bwd_d<72>(a, s);
    case 80: return launch_bwd_d<80>(a, s);
    case 96: return launch_bwd_d<96>(a, s);
    default: return DSP_ERR_SHAPE;
  }
}

int launch_attn_bwd_f32(const AttnBwdArgs& a, hipStream_t s) {
  BwdParamsF p;
  p.q = static_cast<const float*>(a.q);
  p.k = static_cast<const float*>(a.k);
  p.v = static_cast<const float*>(a.v);
  p.o = static_cast<const float*>(a.o);
  p.dout = static_cast<const float*>(a.dout);
  p.dq = static_cast<float*>(a.dq);
  p.dk = static_cast<float*>(a.dk);
  p.dv = static_cast<float*>(a.dv);
  fill_common(p, a);
  p.X = a.X;
  p.H = a.H;
  p.L = a.L;
  p.Lk = a.Lk;
  p.grp = a.H / a.Hkv;
  p.D = a.D;
  p.n_dc = (a.D + DC - 1) / DC;
  p.scale = a.scale;
  const int64_t tq = a.B * a.X * a.H * a.L * p.n_dc, tk = a.B * a.X * a.Hkv * a.Lk * p.n_dc;
  if (tq == 0) return DSP_OK;
  if ((tq + 255) / 256 >= (int64_t(1) << 31) || (tk + 255) / 256 >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  hipLaunchKernelGGL(attn_bwd_f32_dq_kernel, dim3((uint32_t)((tq + 255) / 256)), dim3(256), 0, s, p, tq);
  int st = last_launch_status();
  if (st != DSP_OK || tk == 0) return st;
  hipLaunchKernelGGL(attn_bwd_f32_dkv_kernel, dim3((uint32_t)((tk + 255) / 256)), dim3(256), 0, s, p, tk);
  return last_launch_status();
}

}  // namespace dsp
