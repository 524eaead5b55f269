// Fused bf16 attention along one sequence dimension (Eq. 3 per head, Eq. 1-2),
// applied to the per-dimension reshape of a multi-dimensional sequence
// (Eq. 7-8): every (batch, other-dimension index, head) triple is an
// independent problem over L consecutive sequence positions.  Spatial
// attention (L = S) and temporal attention (L = T) are the same kernel with
// different L, strides and tiling.
//
// Design for gfx950 (CDNA4):
//  * Both products run on v_mfma_f32_32x32x16_bf16 and are computed
//    transposed: S^T = K Q^T (keys on MFMA rows, queries on columns) and
//    O^T = V^T P^T.  In the 32x32 accumulator layout a lane owns one query
//    column, so the softmax row statistics are per-lane scalars (one
//    cross-half swap per reduction) and the rescale of O is a per-lane
//    multiply.  The S^T accumulator registers are, after conversion to bf16,
//    exactly the B operand of the P V product (the key order inside a
//    16-key step is permuted identically on both operands), so P never goes
//    through LDS.
//  * Head width D is padded to 16 for Q K^T (D=72 -> 80, 90% useful) and to
//    32 for P V (72 -> 96).  For D not a multiple of 32, padding column D of
//    V is 1.0 in LDS, so the P V product also yields the softmax row sum from
//    the bf16 probabilities actually used.
//  * The softmax scale and log2(e) are folded into Q once (Q' = Q * scale *
//    log2 e, rounded to bf16), so the MFMA produces scores in the exp2
//    domain.  When D leaves spare columns in the Q K^T contraction (D % 16
//    == 8, e.g. 72), K's padding columns D and D + 1 are 1.0 and Q's hold
//    -m as a bf16 pair (-hi, -lo) with m = hi + lo exactly in fp32 (the
//    running reference maximum, within 2^-17 |m| of the tile maximum it was
//    taken from): the MFMA then also subtracts the maximum and the VALU only
//    evaluates exp2 -- no per-score FMA.
//  * Online softmax with a lazily moved reference: the bias subtracted from
//    the scores is the first tile's maximum plus 64, and the exponentials are
//    clamped to 1.  A later score above the bias shows as a row sum above
//    1/2 (probabilities below the bias sum to far less); only then is the
//    bias moved, O rescaled and the clamped probabilities corrected, after
//    the tile's P V product.  The result does not depend on the reference
//    point (the row sum uses the same one).
//  * K and V tiles of 64 keys are staged in LDS, double-buffered, with the
//    next tile prefetched into registers during the current tile's math.
//    Tiles are fetched with buffer loads through a per-tile buffer resource:
//    rows past L fall outside the resource's range and read as zero, so there
//    are no per-lane bounds checks or address computations in the loop.  Half
//    of the work-group's waves fetch K, the other half V (the resource is
//    wave-uniform).  K rows are read as 16-byte MFMA A fragments (row pitch
//    an odd multiple of 16 bytes: conflict-free); V fragments come straight
//    from row-major LDS through ds_read_b64_tr_b16, so V is never transposed.
//  * Work-group index -> (unit, query block) is remapped so that consecutive
//    units land on the same XCD: the query blocks of a unit, and neighbouring
//    heads of a token row, then share that XCD's L2.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "attn_bf16_common.h"
#include "dsp_internal.h"

// Compile-time tiling of the long-sequence (spatial) and short-sequence
// (temporal) launches: waves per work-group, 32-query tiles per wave, keys per
// LDS tile, minimum waves per SIMD the register allocation must allow.
#ifndef DSP_SATTN_NW
#define DSP_SATTN_NW 8
#endif
#ifndef DSP_SATTN_QT
#define DSP_SATTN_QT 2
#endif
#ifndef DSP_SATTN_KB
#define DSP_SATTN_KB 64
#endif
#ifndef DSP_SATTN_MINW
#define DSP_SATTN_MINW 2
#endif
#ifndef DSP_TATTN_NW
#define DSP_TATTN_NW 4
#endif
#ifndef DSP_TATTN_QT
#define DSP_TATTN_QT 1
#endif
#ifndef DSP_TATTN_KB
#define DSP_TATTN_KB 64
#endif
#ifndef DSP_TATTN_MINW
#define DSP_TATTN_MINW 2
#endif
// D % 32 == 8 (e.g. 72): the last 16 rows of O^T = V^T P^T (d = D - 8 .. D + 7,
// holding the row-sum column) on 16x16x32 MFMAs instead of a padded 32-row tile.
#ifndef DSP_ATTN_PV_SLAB
#define DSP_ATTN_PV_SLAB 1
#endif
// Q K^T with the d step outer and the next step's K fragments read ahead.
#ifndef DSP_ATTN_QK_PIPELINE
#define DSP_ATTN_QK_PIPELINE 1
#endif
// Units of L <= 128 go to the persistent single-tile kernel (attn_short.hip).
#ifndef DSP_ATTN_SHORT_PERSISTENT
#define DSP_ATTN_SHORT_PERSISTENT 1
#endif
// Fold the running maximum into the Q K^T contraction when D allows it.
#ifndef DSP_ATTN_BIAS_COLUMN
#define DSP_ATTN_BIAS_COLUMN 1
#endif

// Row padding (elements) of the K and V tiles in LDS.
#ifndef DSP_ATTN_KP_PAD
#define DSP_ATTN_KP_PAD 8
#endif
#ifndef DSP_ATTN_VP_PAD
#define DSP_ATTN_VP_PAD 16
#endif
#ifndef DSP_ATTN_VP_PAD_WIDE
#define DSP_ATTN_VP_PAD_WIDE 0
#endif

namespace dsp {
namespace {

// log2 headroom of the bias over the reference maximum: probabilities stay at
// most 2^-64 of the reference's (still normal in bf16 and fp32) until a score
// beats the bias, so the reference rarely moves
constexpr float kLazyRescale = 64.0f;

template <int D, int KB>
struct Geo {
  static constexpr int NDK = (D + 15) / 16;       // 16-wide d steps of Q K^T
  static constexpr int NDV = (D + 31) / 32;       // 32-row d tiles of P V
  static constexpr bool ONES = (D % 32) != 0;     // spare V column carries the row sum
  static constexpr bool BIAS = DSP_ATTN_BIAS_COLUMN && (D % 16) == 8;  // spare Q K^T column
  static constexpr int KP = NDK * 16 + DSP_ATTN_KP_PAD;  // K row pitch (elements)
  // V row pitch (elements): 192 bytes for three or more 32-row d tiles (measured:
  // half the LDS bank conflicts of 224), else padded by 16
  static constexpr int VP = NDV * 32 + (NDV >= 3 ? DSP_ATTN_VP_PAD_WIDE : DSP_ATTN_VP_PAD);
  static constexpr int CH = D / 8;                // 16-byte chunks per row
  static constexpr int TILE_ELEMS = KB * (KP + VP);
  static constexpr int NKT = KB / 32;             // 32-key MFMA tiles per LDS tile
};

struct Params {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  bf16* o;
  float* lse;  // optional row log-sum-exp output
  int64_t b_in, x_in, r_in, b_out, x_out, r_out;
  int64_t b_kv, x_kv, r_kv;  // k and v
  uint32_t X, H, L, n_units, n_qb, n_blocks;
  uint32_t Lk, grp;          // keys per unit; query heads per key/value head
  float c;  // scale * log2(e)
};

// Work-group -> unit and query block (XCD-aware), and the unit's base offsets.
struct UnitMap {
  uint32_t unit, qb;
  int64_t in_base, out_base, kv_base;
};

__device__ __forceinline__ UnitMap map_unit(const Params& p, int D) {
  uint32_t bid = blockIdx.x;
  // hardware places block i on XCD i % 8; give each XCD a contiguous range
  if ((p.n_blocks & 7u) == 0) bid = (bid & 7u) * (p.n_blocks >> 3) + (bid >> 3);
  const uint32_t unit = bid / p.n_qb;
  UnitMap m;
  m.unit = unit;
  m.qb = bid - unit * p.n_qb;
  const uint32_t h = unit % p.H;
  const uint32_t bx = unit / p.H;
  const uint32_t xx = bx % p.X;
  const uint32_t bb = bx / p.X;
  m.in_base = (int64_t)bb * p.b_in + (int64_t)xx * p.x_in + (int64_t)h * D;
  m.out_base = (int64_t)bb * p.b_out + (int64_t)xx * p.x_out + (int64_t)h * D;
  m.kv_base = (int64_t)bb * p.b_kv + (int64_t)xx * p.x_kv + (int64_t)(h / p.grp) * D;
  return m;
}

template <int D, int NW, int QT, int KB, int MINW, int NBUF>
__global__ __launch_bounds__(NW * 64, MINW) void attn_fwd_kernel(Params p) {
  // NBUF == 1: the launcher guarantees L <= KB (one tile, nothing to prefetch)
  using G = Geo<D, KB>;
  constexpr int NT = NW * 64;
  constexpr int QB = NW * 32 * QT;
  constexpr int NKT = G::NKT;
  constexpr bool SPLIT = NW > 1;                       // K and V fetched by separate waves
  constexpr int FT = SPLIT ? NT / 2 : NT;              // threads fetching one tensor
  constexpr int TCH = KB * G::CH;                      // 16-byte chunks of one tensor tile
  constexpr int NLOAD = (TCH + FT - 1) / FT;
  static_assert(NW == 1 || NW % 2 == 0, "K/V fetch split needs an even wave count");
  __shared__ __attribute__((aligned(16))) bf16 lds[NBUF * G::TILE_ELEMS];

  const int lane = threadIdx.x & 63;
  // wave index as a scalar: the K/V choice of the tile fetch must be provably
  // wave-uniform, or the buffer resource would need a waterfall loop
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31;
  const int g = lane >> 5;
  const UnitMap um = map_unit(p, D);
  const uint32_t L = p.L;     // queries of the unit
  const uint32_t Lk = p.Lk;   // keys and values of the unit

  // ---- tile fetch through buffer resources covering rows [kb, L) of the
  // unit (rows past L read as zero).  With several waves, waves [0, NW/2)
  // fetch K and the others V; a single wave fetches both.
  const bool fetch_v = SPLIT && wave >= NW / 2;
  const int ft = SPLIT ? threadIdx.x % FT : threadIdx.x;
  const uint32_t row_bytes = (uint32_t)p.r_kv * 2u;
  uint32_t voff[NLOAD];
  int lofs[NLOAD];
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int c = ft + i * FT;
    const int row = c / G::CH, col = c - row * G::CH;
    voff[i] = (uint32_t)row * row_bytes + (uint32_t)col * 16u;
    lofs[i] = row * G::KP + col * 8;                 // K layout; V adds its own base/pitch
    if (fetch_v) lofs[i] = KB * G::KP + row * G::VP + col * 8;
  }
  // the range covers the tile's own rows only, so that widely strided rows
  // (a row stride of many megabytes) still fit a 32-bit byte range
  auto rsrc = [&](const bf16* tensor, uint32_t kb) {
    const uint32_t rows_left = kb < Lk ? min(Lk - kb, (uint32_t)KB) : 0u;
    return make_rsrc(tensor + um.kv_base + (int64_t)kb * p.r_kv, rows_left * row_bytes);
  };
  u32x4 pre[SPLIT ? NLOAD : 1];
  auto fetch = [&](uint32_t kb) {  // SPLIT: one tensor into registers
    const __amdgpu_buffer_rsrc_t rs = rsrc(fetch_v ? p.v : p.k, kb);
#pragma unroll
    for (int i = 0; i < NLOAD; ++i)
      if (ft + i * FT < TCH) pre[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i], 0, 0);
  };
  auto stash = [&](int buf) {  // SPLIT: registers into LDS buffer `buf`
    bf16* t = lds + buf * G::TILE_ELEMS;
#pragma unroll
    for (int i = 0; i < NLOAD; ++i)
      if (ft + i * FT < TCH) *reinterpret_cast<u32x4*>(t + lofs[i]) = pre[i];
  };
  auto fetch_single = [&](uint32_t kb, int buf) {  // one wave: both tensors straight to LDS
    bf16* t = lds + buf * G::TILE_ELEMS;
#pragma unroll
    for (int tsr = 0; tsr < 2; ++tsr) {
      const __amdgpu_buffer_rsrc_t rs = rsrc(tsr ? p.v : p.k, kb);
#pragma unroll
      for (int i = 0; i < NLOAD; ++i) {
        const int c = ft + i * FT;
        if (c < TCH) {
          const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i], 0, 0);
          const int row = c / G::CH, col = c - row * G::CH;
          bf16* dst = tsr ? t + KB * G::KP + row * G::VP + col * 8 : t + lofs[i];
          *reinterpret_cast<u32x4*>(dst) = v;
        }
      }
    }
  };

  // O^T accumulators: NT32 tiles of 32 rows of d (32x32 MFMA layout), plus
  // with SLAB the last 16 rows per 16-query half (16x16 MFMA layout)
  constexpr bool SLAB = DSP_ATTN_PV_SLAB && (D % 32) == 8;
  constexpr int NT32 = SLAB ? D / 32 : G::NDV;
  floatx16 o[NT32 > 0 ? NT32 : 1][QT];
  floatx4 os[QT][2];
#pragma unroll
  for (int t = 0; t < NT32; ++t)
#pragma unroll
    for (int j = 0; j < QT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][j][r] = 0.0f;
#pragma unroll
  for (int j = 0; j < QT; ++j)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) os[j][h][r] = 0.0f;
  // b_ref: the bias subtracted from every score of a query (exp2 domain): the
  // reference maximum plus kLazyRescale, as the exact sum of the bf16 pair
  // (b_hi, b_lo) when the Q K^T MFMA applies it.  Probabilities are
  // exp2(s - b_ref) clamped to 1: at most 2^-kLazyRescale of the reference
  // maximum's until a score beats the bias.
  float b_ref[QT], l_run[QT];
#pragma unroll
  for (int j = 0; j < QT; ++j) { b_ref[j] = 0.0f; l_run[j] = 0.0f; }

  const uint32_t n_kb = (Lk + KB - 1) / KB;
  // the first tile's fetch goes out first: the padding columns and the Q
  // fragments (a global round trip of their own) are prepared while it is in
  // flight
  if (SPLIT) fetch(0);

  // ---- padding columns of the LDS buffers.  K: columns D and D + 1 are 1.0
  // when they carry the bias pair, the rest 0.  V: column D is 1.0 (row sum),
  // the rest 0.
  for (int e = threadIdx.x; e < NBUF * KB; e += NT) {
    bf16* t = lds + (e / KB) * G::TILE_ELEMS;
    const int r = e % KB;
    for (int c = D; c < G::KP; ++c) t[r * G::KP + c] = (bf16)((G::BIAS && c <= D + 1) ? 1.0f : 0.0f);
    bf16* vt = t + KB * G::KP;
    for (int c = D; c < G::VP; ++c) vt[r * G::VP + c] = (bf16)((G::ONES && c == D) ? 1.0f : 0.0f);
  }

  // ---- Q' = Q * scale * log2(e) as bf16 B fragments: lane (n + 32g) holds
  // Q'[q][16s + 8g .. +7].  With the bias columns, elements D and D + 1 of Q'
  // are the negated reference maximum as a hi/lo pair (0 until the first tile
  // sets it).
  const uint32_t q_wave = um.qb * QB + wave * 32 * QT;
  // Loaded through a buffer resource over this work-group's query rows: rows
  // past L and columns past D read as zero, so every load goes out at once
  // (no per-lane branch, no wait between them).
  const uint32_t q_first = um.qb * QB;
  const uint32_t q_rows = L > q_first ? min(L - q_first, (uint32_t)QB) : 0u;
  const __amdgpu_buffer_rsrc_t rq =
      make_rsrc(p.q + um.in_base + (int64_t)q_first * p.r_in, q_rows * (uint32_t)p.r_in * 2u);
  u32x4 qraw[QT][G::NDK];
#pragma unroll
  for (int j = 0; j < QT; ++j) {
    const uint32_t qr = (uint32_t)(wave * 32 * QT + 32 * j + l32);  // row within the work-group's
#pragma unroll
    for (int s = 0; s < G::NDK; ++s) {
      const int d = 16 * s + 8 * g;
      qraw[j][s] = __builtin_amdgcn_raw_buffer_load_b128(
          rq, d < D ? (qr * (uint32_t)p.r_in + (uint32_t)d) * 2u : 0xFFFFFFF0u, 0, 0);
    }
  }
  bf16x8 qf[QT][G::NDK];
#pragma unroll
  for (int j = 0; j < QT; ++j)
#pragma unroll
    for (int s = 0; s < G::NDK; ++s) {
      bf16x8 v = __builtin_bit_cast(bf16x8, qraw[j][s]);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (bf16)((float)v[e] * p.c);
      qf[j][s] = v;
    }
  constexpr int BS = G::NDK - 1;  // the d step holding column D (lanes g == 1)

  if (SPLIT) {
    stash(0);
  } else {
    fetch_single(0, 0);
  }
  __syncthreads();

  // ---- O^T += V^T F^T for bf16 probability fragments F (the P V product, and
  // the correction of a moved reference)
  const int j16 = lane & 15;
  const int mbase = 16 * ((lane >> 4) & 1);
  auto pv = [&](const bf16* v_lds, const bf16x8 (&f)[NKT][2][QT]) {
#pragma unroll
    for (int t = 0; t < NT32; ++t) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int row = 32 * kt + 16 * kk + 4 * g + (j16 >> 2);
          const int col = 32 * t + mbase + 4 * (j16 & 3);
          const shortx4 lo = lds_read_tr(v_lds + row * G::VP + col);
          const shortx4 hi = lds_read_tr(v_lds + (row + 8) * G::VP + col);
          const shortx8 both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          const bf16x8 a = __builtin_bit_cast(bf16x8, both);
#pragma unroll
          for (int j = 0; j < QT; ++j)
            o[t][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, f[kt][kk][j], o[t][j], 0, 0, 0);
        }
    }
    if constexpr (SLAB) {
      // rows d = 32 NT32 .. + 15 over each 32-key tile with 16x16x32 MFMAs.
      // B operand (keys x 16 queries): lane group c = lane / 16 holds 8 keys
      // for queries lane % 16.  One permlane16 swap of the two 16-key halves
      // of a 32x32 probability tile yields it: group c then holds keys
      // kb(c) + {0..3, 8..11} with kb = {0, 16, 4, 20}, for queries 0-15 of
      // the tile in the first register and 16-31 in the second.
      const int c = lane >> 4;
      const int kbase = ((c & 1) ? 16 : 0) + ((c & 2) ? 4 : 0);
      const int col = 32 * NT32 + 4 * (j16 & 3);
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        // A operand: lane (d + 16 c) holds V^T[d][keys of group c]
        const int row = 32 * kt + kbase + (j16 >> 2);
        const shortx4 lo = lds_read_tr(v_lds + row * G::VP + col);
        const shortx4 hi = lds_read_tr(v_lds + (row + 8) * G::VP + col);
        const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int j = 0; j < QT; ++j) {
          u32x4 x = __builtin_bit_cast(u32x4, f[kt][0][j]);
          u32x4 y = __builtin_bit_cast(u32x4, f[kt][1][j]);
          u32x4 b0, b1;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const auto r = __builtin_amdgcn_permlane16_swap(x[w], y[w], false, false);
            b0[w] = r[0];
            b1[w] = r[1];
          }
          os[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, b0), os[j][0], 0, 0, 0);
          os[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, b1), os[j][1], 0, 0, 0);
        }
      }
    }
  };

  // ---- S'^T = K Q'^T (exp2-domain scores, minus the bias with BIAS) for the
  // key tile at kb, keys past Lk at -inf
  auto qk = [&](const bf16* k_lds, uint32_t kb, floatx16 (&s)[NKT][QT]) {
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int j = 0; j < QT; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kt][j][r] = 0.0f;
#if DSP_ATTN_QK_PIPELINE
    // d step outer: the K fragments of step st + 1 are read from LDS while the
    // NKT * QT independent MFMAs of step st run
    auto k_frag = [&](int kt, int st) {
      return *reinterpret_cast<const bf16x8*>(k_lds + (32 * kt + l32) * G::KP + 16 * st + 8 * g);
    };
    bf16x8 ka[2][NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) ka[0][kt] = k_frag(kt, 0);
#pragma unroll
    for (int st = 0; st < G::NDK; ++st) {
      if (st + 1 < G::NDK) {
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt) ka[(st + 1) & 1][kt] = k_frag(kt, st + 1);
      }
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int j = 0; j < QT; ++j)
          s[kt][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[st & 1][kt], qf[j][st], s[kt][j], 0, 0, 0);
    }
#else
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int st = 0; st < G::NDK; ++st) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(k_lds + (32 * kt + l32) * G::KP + 16 * st + 8 * g);
#pragma unroll
        for (int j = 0; j < QT; ++j)
          s[kt][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[j][st], s[kt][j], 0, 0, 0);
      }
#endif
    if (kb + KB > Lk) {  // keys past Lk: score -inf (only the last tile can hold any)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t key = kb + 32 * kt + (r / 4) * 8 + 4 * g + (r % 4);
          if (key >= Lk) {
#pragma unroll
            for (int j = 0; j < QT; ++j) s[kt][j][r] = -INFINITY;
          }
        }
    }
  };

  // the maximum of query j's scores in a tile (the lane's query, both halves)
  auto tile_max = [&](const floatx16 (&s)[NKT][QT], int j) {
    float m = s[0][j][0];
#pragma unroll
    for (int r = 1; r < 16; ++r) m = fmaxf(m, s[0][j][r]);
#pragma unroll
    for (int kt = 1; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) m = fmaxf(m, s[kt][j][r]);
    return fmaxf(m, swap_halves(m));
  };
  // whether this lane holds the running row sum of a query of tile j and it
  // exceeds thr (the lanes and registers the normalisation reads it from)
  auto row_sum_over = [&](int j, float thr) -> bool {
    if constexpr (SLAB) {
      return lane >= 32 && lane < 48 && (os[j][0][0] > thr || os[j][1][0] > thr);
    } else if constexpr (G::ONES) {
      constexpr int tl = D / 32, ml = D % 32;
      constexpr int gl = (ml / 4) % 2, rl = (ml / 8) * 4 + ml % 4;
      return g == gl && o[tl][j][rl] > thr;
    } else {
      return l_run[j] > thr;
    }
  };

  // One key tile, up to (not including) its barrier.  FIRST: the first tile
  // sets the reference from its exact maximum (nothing is applied in the MFMA
  // yet).  Later tiles take their probabilities against the current bias and
  // return whether, afterwards, some query's row sum shows a clamped
  // probability (a score at or above the bias): then fix() moves the reference
  // before the tile's barrier.  The fix runs outside the loop of ordinary
  // tiles, so its code does not weigh on that loop.
  auto tile = [&](uint32_t it, auto first_c) -> bool {
    constexpr bool FIRST = decltype(first_c)::value;
    const uint32_t kb = it * KB;
    const bool more = NBUF > 1 && it + 1 < n_kb;
    if (SPLIT && more) fetch(kb + KB);
    const bf16* k_lds = lds + (NBUF > 1 ? (it & 1) : 0) * G::TILE_ELEMS;

    // ---- S'^T = K Q'^T (exp2-domain scores, minus the bias with BIAS)
    floatx16 s[NKT][QT];
    qk(k_lds, kb, s);

    if constexpr (FIRST) {
      // the bias: the exact maximum plus the headroom, as a bf16 pair whose sum
      // (exact in fp32, within 2^-17 of its size) is what the MFMA subtracts
#pragma unroll
      for (int j = 0; j < QT; ++j) {
        const float bt = tile_max(s, j) + kLazyRescale;
        const bf16 hi = (bf16)bt;
        const bf16 lo = (bf16)(bt - (float)hi);
        b_ref[j] = (float)hi + (float)lo;
        if (G::BIAS && g == 1) {
          qf[j][BS][0] = (bf16)(-(float)hi);
          qf[j][BS][1] = (bf16)(-(float)lo);
        }
      }
    }

    // ---- probabilities exp2(s - bias) clamped to 1 (the clamp only acts when
    // a score reached the bias; fix() then restores it), as bf16 B fragments
    // of the P V product
    bf16x8 pf[NKT][2][QT];
#pragma unroll
    for (int j = 0; j < QT; ++j) {
      float ls = 0.0f;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float x = (FIRST || !G::BIAS) ? s[kt][j][r] - b_ref[j] : s[kt][j][r];
          const float e = __builtin_amdgcn_fmed3f(__builtin_amdgcn_exp2f(x), 0.0f, 1.0f);
          if (!G::ONES) ls += e;
          pf[kt][r / 8][j][r % 8] = (bf16)e;
        }
      if (!G::ONES) l_run[j] += ls;
    }

    // the next tile's prefetched rows into the other LDS buffer (no wave reads
    // it during this tile), so the registers are free for the rest of it
    if (more) {
      if (SPLIT) {
        stash((it + 1) & 1);
      } else {
        fetch_single(kb + KB, (it + 1) & 1);
      }
    }

    // ---- O^T += V^T P^T, V fragments read transposed from row-major LDS
    pv(k_lds + KB * G::KP, pf);

    // a clamped probability puts its query's row sum at 1 or more, while
    // probabilities below the bias sum to far less than 1/2 (each is under
    // 2^-kLazyRescale of the reference maximum's, unless scores crept up to
    // within ~kLazyRescale of the bias: then the reference moves early, which
    // is harmless)
    bool need = false;
    if constexpr (!FIRST) {
#pragma unroll
      for (int j = 0; j < QT; ++j) need |= row_sum_over(j, 0.5f);
    }
    return __any(need);
  };

  // The rare move of the reference in tile it, after its P V product: the
  // scores again (against the bias still in place), the tile maximum; for
  // each query with a score above its bias, the bias becomes that maximum
  // plus the headroom (d higher), O and the row sum are rescaled by 2^-d, and
  // every key gets, in a second P V pass, the difference between its exact
  // probability against the new bias and the clamped one already summed:
  // exp2(x - d) - exp2(min(x, 0) - d), x the score minus the old bias (0 for
  // keys below the old bias and for queries that keep theirs).
  auto fix = [&](uint32_t it) {
    const uint32_t kb = it * KB;
    const bf16* k_lds = lds + (NBUF > 1 ? (it & 1) : 0) * G::TILE_ELEMS;
    floatx16 s[NKT][QT];
    qk(k_lds, kb, s);
    bf16x8 pf[NKT][2][QT];
#pragma unroll
    for (int j = 0; j < QT; ++j) {
      const float mrel = G::BIAS ? tile_max(s, j) : tile_max(s, j) - b_ref[j];
      const bool mv = mrel > 0.0f;
      float d = 0.0f;
      if (mv) {
        const float bt = b_ref[j] + mrel + kLazyRescale;
        const bf16 hi = (bf16)bt;
        const bf16 lo = (bf16)(bt - (float)hi);
        const float bn = (float)hi + (float)lo;
        d = bn - b_ref[j];
        b_ref[j] = bn;
        if (G::BIAS && g == 1) {
          qf[j][BS][0] = (bf16)(-(float)hi);
          qf[j][BS][1] = (bf16)(-(float)lo);
        }
      }
      const float alpha = __builtin_amdgcn_exp2f(-d);
      l_run[j] *= alpha;
#pragma unroll
      for (int t = 0; t < NT32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][j][r] *= alpha;
      if (SLAB) {
        // the 16x16 slab of half h holds query 16 h + lane % 16 in every
        // lane, not the lane's own query lane % 32: take that query's factor
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float alpha_h = __shfl(alpha, 16 * h + (lane & 15));
#pragma unroll
          for (int r = 0; r < 4; ++r) os[j][h][r] *= alpha_h;
        }
      }
      float ls = 0.0f;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float x = G::BIAS ? s[kt][j][r] : s[kt][j][r] - (b_ref[j] - d);
          const float cx = __builtin_amdgcn_exp2f(x - d) - __builtin_amdgcn_exp2f(fminf(x, 0.0f) - d);
          if (!G::ONES) ls += cx;
          pf[kt][r / 8][j][r % 8] = (bf16)cx;
        }
      if (!G::ONES) l_run[j] += ls;
    }
    pv(k_lds + KB * G::KP, pf);
  };

  tile(0, std::true_type{});
  __syncthreads();
  uint32_t it = 1;
  while (it < n_kb) {
    bool moved = false;
    for (; it < n_kb; ++it) {
      if (tile(it, std::false_type{})) {
        moved = true;
        break;
      }
      __syncthreads();
    }
    if (!moved) break;
    fix(it);
    __syncthreads();
    ++it;
  }

  // ---- normalise and store: lane (n + 32g) holds O^T[32t + 8(r/4) + 4g + r%4][q]
  bf16* og = p.o + um.out_base;
  // staged output row pitch (elements): padded so that the rows of 16
  // consecutive queries start on distinct banks for the 8-byte staging writes,
  // where the padded rows fit the tile buffers
  constexpr int SOP_PAD = (D % 16 == 8) ? D : D + 8;
  constexpr int SOP = NW * 32 * SOP_PAD <= NBUF * G::TILE_ELEMS ? SOP_PAD : D;
  static_assert(NW * 32 * SOP <= NBUF * G::TILE_ELEMS, "the output staging fits the LDS tile buffers");
  __syncthreads();  // every wave is done with the K and V tiles
#pragma unroll
  for (int j = 0; j < QT; ++j) {
    float l;
    if constexpr (SLAB) {
      // row sum (d = D) of query l32: 16x16 slab of half l32 / 16, lane
      // 32 + l32 % 16 (rows 8..11 of the slab), register 0
      const int src_lane = 32 + (l32 & 15);
      const float s0 = __shfl(os[j][0][0], src_lane);
      const float s1 = __shfl(os[j][1][0], src_lane);
      l = (l32 & 16) ? s1 : s0;
    } else if constexpr (G::ONES) {
      constexpr int tl = D / 32, ml = D % 32;
      constexpr int gl = (ml / 4) % 2, rl = (ml / 8) * 4 + ml % 4;
      const float vsum = o[tl][j][rl];
      const float other = swap_halves(vsum);
      l = (g == gl) ? vsum : other;
    } else {
      l = l_run[j] + swap_halves(l_run[j]);
    }
    const float inv = 1.0f / l;
    if (p.lse && g == 0) {
      // natural-log row log-sum-exp: the probabilities were exp2(s' - b_ref)
      // with s' the log2-domain score, summing to l
      const uint32_t q = q_wave + 32 * j + l32;
      if (q < L) p.lse[(int64_t)um.unit * L + q] = 0.6931471805599453f * (b_ref[j] + log2f(l));
    }
    // The output rows leave through LDS: this wave's 32 rows of query tile j
    // are staged (bf16, row pitch SOP) in its own LDS region and stored as
    // whole 16-byte chunks, CH consecutive lanes per row.  From the
    // accumulator layout a store instruction would write 8-byte pieces of 32
    // rows, one L2 request each.  Only this wave touches its region, and one
    // wave's LDS accesses complete in order, so no barrier is needed between
    // the staging and the reads.
    bf16* so = lds + wave * 32 * SOP;
    if constexpr (SLAB) {
      // slab rows d < D: lanes 0-31 hold d = 32 NT32 + 4 (lane / 16) + r for
      // query 16 h + lane % 16; their row sum is that query's
      const int sl = (lane & 15);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float inv_h = __shfl(inv, 16 * h + sl);
        if (lane < 32) {
          const int d0 = 32 * NT32 + 4 * (lane >> 4);
          bf16x2 lo = {(bf16)(os[j][h][0] * inv_h), (bf16)(os[j][h][1] * inv_h)};
          bf16x2 hi = {(bf16)(os[j][h][2] * inv_h), (bf16)(os[j][h][3] * inv_h)};
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, lo);
          w.y = __builtin_bit_cast(uint32_t, hi);
          *reinterpret_cast<uint2*>(so + (16 * h + sl) * SOP + d0) = w;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NT32; ++t)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = 32 * t + 8 * r4 + 4 * g;
        if (d0 < D) {
          bf16x2 lo = {(bf16)(o[t][j][4 * r4 + 0] * inv), (bf16)(o[t][j][4 * r4 + 1] * inv)};
          bf16x2 hi = {(bf16)(o[t][j][4 * r4 + 2] * inv), (bf16)(o[t][j][4 * r4 + 3] * inv)};
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, lo);
          w.y = __builtin_bit_cast(uint32_t, hi);
          *reinterpret_cast<uint2*>(so + l32 * SOP + d0) = w;
        }
      }
    constexpr int OCH = 32 * G::CH;  // 16-byte chunks of the 32 rows
#pragma unroll
    for (int i = 0; i < (OCH + 63) / 64; ++i) {
      const int c = lane + 64 * i;
      const int row = c / G::CH, col = c - row * G::CH;
      const uint32_t q = q_wave + 32 * j + row;
      if (c < OCH && q < L)
        *reinterpret_cast<u32x4*>(og + (int64_t)q * p.r_out + col * 8) =
            *reinterpret_cast<const u32x4*>(so + row * SOP + col * 8);
    }
  }
}

// Kernel parameters for a launch with QB queries per work-group and KB keys
// per tile; returns the number of work-groups (0: nothing to do) or -1 when
// the shape is out of range.
int64_t make_params(const AttnArgs& a, int QB, int KB, Params& p) {
  p.q = static_cast<const bf16*>(a.q);
  p.k = static_cast<const bf16*>(a.k);
  p.v = static_cast<const bf16*>(a.v);
  p.o = static_cast<bf16*>(a.o);
  p.lse = a.lse;
  p.b_in = a.b_stride_in;
  p.x_in = a.x_stride_in;
  p.r_in = a.r_stride_in;
  p.b_kv = a.b_stride_kv;
  p.x_kv = a.x_stride_kv;
  p.r_kv = a.r_stride_kv;
  p.Lk = (uint32_t)a.Lk;
  p.grp = (uint32_t)(a.H / a.Hkv);
  p.b_out = a.b_stride_out;
  p.x_out = a.x_stride_out;
  p.r_out = a.r_stride_out;
  p.X = (uint32_t)a.X;
  p.H = (uint32_t)a.H;
  p.L = (uint32_t)a.L;
  const int64_t units = a.B * a.X * a.H;
  const int64_t n_qb = (a.L + QB - 1) / QB;
  const int64_t blocks = units * n_qb;
  if (blocks == 0) return 0;
  // a tile's buffer resource addresses its rows with 32-bit byte offsets
  if (blocks >= (int64_t(1) << 31) || std::min<int64_t>(a.Lk, KB) * a.r_stride_kv * 2 >= (int64_t(1) << 31) ||
      std::min<int64_t>(a.L, QB) * a.r_stride_in * 2 >= (int64_t(1) << 31))
    return -1;
  p.n_units = (uint32_t)units;
  p.n_qb = (uint32_t)n_qb;
  p.n_blocks = (uint32_t)blocks;
  p.c = a.scale * 1.4426950408889634f;
  return blocks;
}

template <int D, int NW, int QT, int KB, int MINW, int NBUF = 2>
int launch_cfg(const AttnArgs& a, hipStream_t s) {
  if (NBUF == 1 && a.Lk > KB) return DSP_ERR_SHAPE;
  Params p;
  const int64_t blocks = make_params(a, NW * 32 * QT, KB, p);
  if (blocks <= 0) return blocks == 0 ? DSP_OK : DSP_ERR_SHAPE;
  hipLaunchKernelGGL((attn_fwd_kernel<D, NW, QT, KB, MINW, NBUF>), dim3((uint32_t)blocks),
                     dim3(NW * 64), 0, s, p);
  return last_launch_status();
}

template <int D>
int launch_d(const AttnArgs& a, hipStream_t s) {
  // few keys: all of a unit's keys are one tile, fetched at once (the tiling
  // is chosen by the key count; any number of queries runs in query blocks)
  if (a.Lk <= 32) return launch_cfg<D, 1, 1, 32, 1, 1>(a, s);
  if (a.Lk <= 64) return launch_cfg<D, 2, 1, 64, 2, 1>(a, s);
  if (a.Lk <= 128) {
    if constexpr (DSP_TATTN_KB >= 128)
      return launch_cfg<D, DSP_TATTN_NW, DSP_TATTN_QT, 128, DSP_TATTN_MINW, 1>(a, s);
    else
      return launch_cfg<D, DSP_TATTN_NW, DSP_TATTN_QT, DSP_TATTN_KB, DSP_TATTN_MINW>(a, s);
  }
  return launch_cfg<D, DSP_SATTN_NW, DSP_SATTN_QT, DSP_SATTN_KB, DSP_SATTN_MINW>(a, s);
}

}  // namespace

bool attn_bf16_supports(int D) {
  switch (D) {
    case 16: case 32: case 64: case 72: case 80: case 96: return true;
    default: return false;
  }
}

int launch_attn_bf16(const AttnArgs& a, hipStream_t s) {
#if DSP_ATTN_SHORT_PERSISTENT
  if (attn_bf16_short_fits(a)) return launch_attn_bf16_short(a, s);
#endif
  switch (a.D) {
    case 16: return launch_d<16>(a, s);
    case 32: return launch_d<32>(a, s);
    case 64: return launch_d<64>(a, s);
    case 72: return launch_d<72>(a, s);
    case 80: return launch_d<80>(a, s);
    case 96: return launch_d<96>(a, s);
    default: return DSP_ERR_SHAPE;
  }
}

}  // namespace dsp
