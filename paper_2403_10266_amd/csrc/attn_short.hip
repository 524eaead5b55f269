// Persistent bf16 attention for short units (L <= 128): temporal attention
// over the T frames at each spatial location (Eq. 3 per head, Eq. 1-2, on the
// temporal reshape of Eq. 7-8).  The same arithmetic as the tiled kernel in
// attn_bf16.hip -- S^T = K Q'^T and O^T = V^T P^T on v_mfma_f32_32x32x16_bf16,
// one lane per query, Q' = Q * scale * log2(e) rounded to bf16, probabilities
// rounded to bf16, fp32 accumulation -- organised for a problem that is bound
// by HBM rather than by the matrix cores:
//  * A unit is one LDS tile: all of its keys and values (L <= KB) are staged
//    at once, so the softmax maximum is exact before the first exponential and
//    there is no online rescaling.
//  * The kernel is persistent: a grid of two waves per SIMD loops over units,
//    and while it computes one unit it already holds the loads of the next
//    one (K, V and this lane's Q fragments) in flight in registers (for
//    128-key units, K and V of the next two).  Every work-group therefore
//    keeps one to two units' reads outstanding at all times, instead of
//    paying a full HBM round trip between a unit's fetch and its
//    math.
//  * Units are cut into 8 contiguous ranges, one per XCD, so the 16 heads of
//    a token row (neighbouring 144-byte segments of one 2304-byte row) are
//    fetched by work-groups sharing one L2.
//  * Rows past L fall outside the per-unit buffer resource and read as zero;
//    their scores are set to -inf before the maximum.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "attn_bf16_common.h"
#include "dsp_internal.h"

namespace dsp {
namespace {

// Cache hints, chosen per unit length by measurement (every byte is read or
// written once): 32-key units store O non-temporally (54-58 -> 49 us on
// (1, 1024, 32) x 16 heads), 64-key units load K, V and Q with the nt policy
// (124-126 -> 116-118 us on (2, 512, 64) x 16 heads); 128-key units gain from
// neither and lose 12-15% with the non-temporal store.
template <int KB>
struct ShortHints {
  static constexpr int kLoadCpol = KB == 64 ? 2 : 0;  // buffer aux: 2 = nt
  static constexpr bool kNtStore = KB == 32;
};

template <int D, int KB, int HG>
struct ShortGeo {
  static constexpr int NWH = KB / 32;                // waves per head, 32 queries each
  static constexpr int NW = HG * NWH;                // waves per work-group
  static constexpr int NT = NW * 64;
  static constexpr int NDK = (D + 15) / 16;          // 16-wide d steps of Q K^T
  static constexpr int NDV = (D + 31) / 32;          // 32-row d tiles of P V
  static constexpr int NKT = KB / 32;                // 32-key MFMA tiles
  static constexpr bool SLAB = (D % 32) == 8;        // last 16 rows of O^T on 16x16x32
  static constexpr int NT32 = SLAB ? D / 32 : NDV;   // 32-row tiles of O^T
  static constexpr bool ONES = (D % 32) != 0;        // spare V column D carries the row sum
  static constexpr int KP = NDK * 16 + 8;            // K row pitch (elements): odd multiple of 16 B
  static constexpr int VP = NDV * 32 + 16;           // V row pitch (elements)
  static constexpr int CH = D / 8;                   // 16-byte chunks per row
  static constexpr int HEAD_ELEMS = KB * (2 * KP + VP);  // per head: K, V, Q (Q rows later stage O)
  static constexpr int LDS_ELEMS = HG * HEAD_ELEMS;
};

struct ShortParams {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  bf16* o;
  float* lse;  // optional row log-sum-exp output
  int64_t b_in, x_in, r_in, b_out, x_out, r_out;
  uint32_t X, H, L, n_units;
  float c;  // scale * log2(e)
};

template <int D, int KB, int HG>
__global__ __launch_bounds__(HG * KB / 32 * 64, 2) void attn_short_kernel(ShortParams p) {
  using G = ShortGeo<D, KB, HG>;
  constexpr int NW = G::NW, NT = G::NT, NKT = G::NKT, NT32 = G::NT32;
  constexpr int RCH = HG * G::CH;                    // 16-byte chunks of a row's head group
  constexpr bool SPLIT = NW > 1;                     // K and V fetched by separate waves
  constexpr int FT = SPLIT ? NT / 2 : NT;            // threads fetching one tensor
  constexpr int NTS = SPLIT ? 1 : 2;                 // tensors fetched by one thread
  constexpr int TCH = KB * RCH;                      // 16-byte chunks of one tensor
  constexpr int NLOAD = (TCH + FT - 1) / FT;
  constexpr int NLQ = (TCH + NT - 1) / NT;           // Q chunks per thread (all threads)
  __shared__ __attribute__((aligned(16))) bf16 lds[G::LDS_ELEMS];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31;
  const int g = lane >> 5;
  const uint32_t L = p.L;

  // LDS per head of the group: K [KB][KP], V [KB][VP], Q [KB][KP]
  auto k_of = [&](int hh) { return lds + hh * G::HEAD_ELEMS; };
  auto v_of = [&](int hh) { return lds + hh * G::HEAD_ELEMS + KB * G::KP; };
  auto q_of = [&](int hh) { return lds + hh * G::HEAD_ELEMS + KB * (G::KP + G::VP); };
  // padding columns, written once (the fetches only write columns < D): K and
  // Q are 0 there; V's column D is 1.0 when it carries the row sum, the rest 0
  for (int e = threadIdx.x; e < HG * KB; e += NT) {
    const int hh = e / KB, r = e % KB;
    for (int c = D; c < G::KP; ++c) k_of(hh)[r * G::KP + c] = q_of(hh)[r * G::KP + c] = (bf16)0.0f;
    for (int c = D; c < G::VP; ++c) v_of(hh)[r * G::VP + c] = (bf16)((G::ONES && c == D) ? 1.0f : 0.0f);
  }

  // this work-group's units: 8 contiguous ranges, one per XCD (work-group i
  // runs on XCD i % 8); the work-groups of an XCD interleave over its range
  const uint32_t nb = gridDim.x;
  uint32_t u, u_end, u_step;
  if ((nb & 7u) == 0) {
    const uint32_t xcd = blockIdx.x & 7u;
    u = (uint32_t)(((uint64_t)p.n_units * xcd) >> 3) + (blockIdx.x >> 3);
    u_end = (uint32_t)(((uint64_t)p.n_units * (xcd + 1)) >> 3);
    u_step = nb >> 3;
  } else {
    u = blockIdx.x;
    u_end = p.n_units;
    u_step = nb;
  }
  // a unit is a group of HG consecutive heads of one (b, x) position
  const uint32_t n_groups = p.H / HG;
  auto unit_base = [&](uint32_t unit, int64_t bs, int64_t xs) {
    const uint32_t h = (unit % n_groups) * HG;
    const uint32_t bx = unit / n_groups;
    const uint32_t xx = bx % p.X;
    const uint32_t bb = bx / p.X;
    return (int64_t)bb * bs + (int64_t)xx * xs + (int64_t)h * D;
  };

  // fixed per-thread byte offsets of the tile fetches and LDS destinations:
  // every fetch reads whole 16-byte chunks, CH consecutive lanes per row
  const bool fetch_v = SPLIT && wave >= NW / 2;
  const int ft = SPLIT ? threadIdx.x % FT : threadIdx.x;
  const uint32_t row_bytes = (uint32_t)p.r_in * 2u;
  const uint32_t unit_bytes = L * row_bytes;
  uint32_t voff[NLOAD], qoff[NLQ];
  int kofs[NLOAD], vofs[NLOAD], qofs[NLQ];
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int c = ft + i * FT;
    const int row = c / RCH, rc = c - row * RCH, hh = rc / G::CH, col = rc - hh * G::CH;
    voff[i] = (uint32_t)row * row_bytes + (uint32_t)rc * 16u;
    kofs[i] = hh * G::HEAD_ELEMS + row * G::KP + col * 8;
    vofs[i] = hh * G::HEAD_ELEMS + KB * G::KP + row * G::VP + col * 8;
  }
#pragma unroll
  for (int i = 0; i < NLQ; ++i) {
    const int c = threadIdx.x + i * NT;
    const int row = c / RCH, rc = c - row * RCH, hh = rc / G::CH, col = rc - hh * G::CH;
    qoff[i] = (uint32_t)row * row_bytes + (uint32_t)rc * 16u;
    qofs[i] = hh * G::HEAD_ELEMS + KB * (G::KP + G::VP) + row * G::KP + col * 8;
  }

  // K/V chunks of the next units, in registers.  128-key units keep two sets:
  // set S holds the unit after next while the other set's unit is computed,
  // so two units' K and V are in flight at a time (266-279 against 273-287 us
  // on the temporal workload; shorter units measured no gain).  Q's chunks
  // (one set) are fetched one unit ahead.
  constexpr int NSET = KB == 128 ? 2 : 1;
  u32x4 pk[NSET][NTS][NLOAD];
  u32x4 pq[NLQ];
  auto issue_kv = [&](int S, uint32_t unit) {
    const int64_t ib = unit_base(unit, p.b_in, p.x_in);
#pragma unroll
    for (int t = 0; t < NTS; ++t) {
      const bf16* ten = SPLIT ? (fetch_v ? p.v : p.k) : (t ? p.v : p.k);
      const __amdgpu_buffer_rsrc_t rs = make_rsrc(ten + ib, unit_bytes);
#pragma unroll
      for (int i = 0; i < NLOAD; ++i)
        if (ft + i * FT < TCH)
          pk[S][t][i] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i], 0, ShortHints<KB>::kLoadCpol);
    }
  };
  auto issue_q = [&](uint32_t unit) {
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(p.q + unit_base(unit, p.b_in, p.x_in), unit_bytes);
#pragma unroll
    for (int i = 0; i < NLQ; ++i)
      if ((int)threadIdx.x + i * NT < TCH)
        pq[i] = __builtin_amdgcn_raw_buffer_load_b128(rq, qoff[i], 0, ShortHints<KB>::kLoadCpol);
  };

  // this wave's head of the group and its 32 queries
  const int hw = wave / G::NWH;
  const int qw = wave - hw * G::NWH;
  const bf16* const k_lds = k_of(hw);
  const bf16* const v_lds = v_of(hw);
  bf16* const q_lds = q_of(hw);
  const uint32_t q_row = 32 * qw + l32;
  // one unit from register set S (compile-time, so the two sets never move
  // between registers)
  auto unit_body = [&](auto s_c, uint32_t u) {
    constexpr int S = decltype(s_c)::value;
    __syncthreads();  // the previous unit's LDS reads are done (and the padding is written)
#pragma unroll
    for (int t = 0; t < NTS; ++t)
#pragma unroll
      for (int i = 0; i < NLOAD; ++i)
        if (ft + i * FT < TCH) {
          bf16* dst = lds + ((SPLIT ? fetch_v : t == 1) ? vofs[i] : kofs[i]);
          *reinterpret_cast<u32x4*>(dst) = pk[S][t][i];
        }
#pragma unroll
    for (int i = 0; i < NLQ; ++i)
      if ((int)threadIdx.x + i * NT < TCH) *reinterpret_cast<u32x4*>(lds + qofs[i]) = pq[i];
    __syncthreads();
    const int64_t ob = unit_base(u, p.b_out, p.x_out) + hw * D;
    if (u + NSET * u_step < u_end) issue_kv(S, u + NSET * u_step);
    if (u + u_step < u_end) issue_q(u + u_step);
    if (32 * (uint32_t)qw >= L) return;  // no queries for this wave (wave-uniform)

    // Q' = Q * scale * log2(e) as bf16 B fragments: lane (n + 32g) holds
    // Q'[32 wave + n][16s + 8g .. +7] (columns >= D are LDS padding, 0)
    bf16x8 qf[G::NDK];
#pragma unroll
    for (int s = 0; s < G::NDK; ++s) {
      const bf16x8 raw = *reinterpret_cast<const bf16x8*>(q_lds + q_row * G::KP + 16 * s + 8 * g);
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[s][e] = (bf16)((float)raw[e] * p.c);
    }

    // ---- S'^T = K Q'^T over all keys of the unit
    floatx16 s[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] = 0.0f;
#pragma unroll
      for (int st = 0; st < G::NDK; ++st) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(k_lds + (32 * kt + l32) * G::KP + 16 * st + 8 * g);
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], s[kt], 0, 0, 0);
      }
    }
    // lane (n + 32g) holds keys 32kt + 8(r/4) + 4g + r%4 of query n
    if (L < (uint32_t)KB) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if ((uint32_t)(32 * kt + (r / 4) * 8 + 4 * g + (r % 4)) >= L) s[kt][r] = -INFINITY;
    }
    float m = s[0][0];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) m = fmaxf(m, s[kt][r]);
    m = fmaxf(m, swap_halves(m));  // the other 16 keys of each group live in lane n ^ 32

    // probabilities as bf16 B fragments of the P V product
    bf16x8 pf[NKT][2];
    float ls = 0.0f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(s[kt][r] - m);
        if (!G::ONES) ls += e;
        pf[kt][r / 8][r % 8] = (bf16)e;
      }

    // ---- O^T = V^T P^T, V fragments read transposed from row-major LDS
    floatx16 o[NT32 > 0 ? NT32 : 1];
    floatx4 os[2];
#pragma unroll
    for (int t = 0; t < NT32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) os[h][r] = 0.0f;
    const int j16 = lane & 15;
    const int mbase = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int t = 0; t < NT32; ++t)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int row = 32 * kt + 16 * kk + 4 * g + (j16 >> 2);
          const int col = 32 * t + mbase + 4 * (j16 & 3);
          const shortx4 lo = lds_read_tr(v_lds + row * G::VP + col);
          const shortx4 hi = lds_read_tr(v_lds + (row + 8) * G::VP + col);
          const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kt][kk], o[t], 0, 0, 0);
        }
    if constexpr (G::SLAB) {
      // rows d = 32 NT32 .. + 15 (holding the row-sum column D) on 16x16x32
      // MFMAs.  B operand (32 keys x 16 queries): lane group c = lane / 16
      // holds 8 keys; one permlane16 swap of the two 16-key halves of a 32x32
      // probability tile gives group c the keys kb(c) + {0..3, 8..11},
      // kb = {0, 16, 4, 20}, for queries 0-15 in the first register and 16-31
      // in the second.  The A operand (V^T) is read at matching key rows.
      const int c = lane >> 4;
      const int kbase = ((c & 1) ? 16 : 0) + ((c & 2) ? 4 : 0);
      const int col = 32 * NT32 + 4 * (j16 & 3);
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const int row = 32 * kt + kbase + (j16 >> 2);
        const shortx4 lo = lds_read_tr(v_lds + row * G::VP + col);
        const shortx4 hi = lds_read_tr(v_lds + (row + 8) * G::VP + col);
        const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        const u32x4 x = __builtin_bit_cast(u32x4, pf[kt][0]);
        const u32x4 y = __builtin_bit_cast(u32x4, pf[kt][1]);
        u32x4 b0, b1;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const auto r = __builtin_amdgcn_permlane16_swap(x[w], y[w], false, false);
          b0[w] = r[0];
          b1[w] = r[1];
        }
        os[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, b0), os[0], 0, 0, 0);
        os[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, b1), os[1], 0, 0, 0);
      }
    }

    // ---- normalise and store: lane (n + 32g) holds O^T[32t + 8(r/4) + 4g + r%4][n]
    float l;
    if constexpr (G::SLAB) {
      // row sum (d = D) of query l32: slab l32 / 16, lane 32 + l32 % 16, register 0
      const int src_lane = 32 + (l32 & 15);
      const float s0 = __shfl(os[0][0], src_lane);
      const float s1 = __shfl(os[1][0], src_lane);
      l = (l32 & 16) ? s1 : s0;
    } else if constexpr (G::ONES) {
      constexpr int tl = D / 32, ml = D % 32;
      constexpr int gl = (ml / 4) % 2, rl = (ml / 8) * 4 + ml % 4;
      const float vsum = o[tl][rl];
      const float other = swap_halves(vsum);
      l = (g == gl) ? vsum : other;
    } else {
      l = ls + swap_halves(ls);
    }
    const float inv = 1.0f / l;
    if (p.lse && g == 0 && q_row < L) {
      // natural-log row log-sum-exp (exact maximum m, row sum l of exp2(s' - m))
      const uint32_t unit = (u / n_groups) * p.H + (u % n_groups) * HG + hw;
      p.lse[(int64_t)unit * L + q_row] = 0.6931471805599453f * (m + log2f(l));
    }
    // stage this wave's 32 output rows in its own Q rows of LDS (only this
    // wave reads them), then store whole 16-byte chunks, CH lanes per row
    if constexpr (G::SLAB) {
      // slab rows d < D: lanes 0-31 hold d = 32 NT32 + 4 (lane / 16) + r for
      // query 16 h + lane % 16
      const int sl = lane & 15;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float inv_h = __shfl(inv, 16 * h + sl);
        if (lane < 32) {
          const int d0 = 32 * NT32 + 4 * (lane >> 4);
          bf16x2 lo = {(bf16)(os[h][0] * inv_h), (bf16)(os[h][1] * inv_h)};
          bf16x2 hi = {(bf16)(os[h][2] * inv_h), (bf16)(os[h][3] * inv_h)};
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, lo);
          w.y = __builtin_bit_cast(uint32_t, hi);
          *reinterpret_cast<uint2*>(q_lds + (32 * qw + 16 * h + sl) * G::KP + d0) = w;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NT32; ++t)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = 32 * t + 8 * r4 + 4 * g;
        if (d0 < D) {
          bf16x2 lo = {(bf16)(o[t][4 * r4 + 0] * inv), (bf16)(o[t][4 * r4 + 1] * inv)};
          bf16x2 hi = {(bf16)(o[t][4 * r4 + 2] * inv), (bf16)(o[t][4 * r4 + 3] * inv)};
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, lo);
          w.y = __builtin_bit_cast(uint32_t, hi);
          *reinterpret_cast<uint2*>(q_lds + q_row * G::KP + d0) = w;
        }
      }
    bf16* og = p.o + ob;
    constexpr int OCH = 32 * G::CH;  // 16-byte chunks of this wave's rows
#pragma unroll
    for (int i = 0; i < (OCH + 63) / 64; ++i) {
      const int c = lane + 64 * i;
      const int row = c / G::CH, col = c - row * G::CH;
      const uint32_t q = 32 * qw + row;
      if (c < OCH && q < L) {
        const u32x4 val = *reinterpret_cast<const u32x4*>(q_lds + q * G::KP + col * 8);
        u32x4* dst = reinterpret_cast<u32x4*>(og + (int64_t)q * p.r_out + col * 8);
        if constexpr (ShortHints<KB>::kNtStore) __builtin_nontemporal_store(val, dst);
        else *dst = val;
      }
    }
  };
  using set0 = std::integral_constant<int, 0>;
  using set1 = std::integral_constant<int, 1>;
  if (u < u_end) {
    issue_kv(0, u);
    issue_q(u);
  }
  if constexpr (NSET == 2) {
    if (u + u_step < u_end) issue_kv(1, u + u_step);
  }
  for (; u < u_end; u += NSET * u_step) {
    unit_body(set0{}, u);
    if constexpr (NSET == 2) {
      if (u + u_step < u_end) unit_body(set1{}, u + u_step);
    }
  }
}

template <int D, int KB, int HG>
int launch_short_kb(const AttnArgs& a, hipStream_t s) {
  using G = ShortGeo<D, KB, HG>;
  ShortParams p;
  p.q = static_cast<const bf16*>(a.q);
  p.k = static_cast<const bf16*>(a.k);
  p.v = static_cast<const bf16*>(a.v);
  p.o = static_cast<bf16*>(a.o);
  p.lse = a.lse;
  p.b_in = a.b_stride_in;
  p.x_in = a.x_stride_in;
  p.r_in = a.r_stride_in;
  p.b_out = a.b_stride_out;
  p.x_out = a.x_stride_out;
  p.r_out = a.r_stride_out;
  p.X = (uint32_t)a.X;
  p.H = (uint32_t)a.H;
  p.L = (uint32_t)a.L;
  const int64_t units = a.B * a.X * (a.H / HG);
  p.n_units = (uint32_t)units;
  p.c = a.scale * 1.4426950408889634f;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return DSP_ERR_HIP;
  // resident work-groups per CU: two waves per SIMD (four SIMDs), within 160 KB of LDS
  constexpr int per_cu = std::max(1, std::min(8 / G::NW, 163840 / (G::LDS_ELEMS * 2)));
  int64_t blocks = std::min<int64_t>(units, (int64_t)cus * per_cu);
  if (blocks >= 8) blocks &= ~int64_t(7);
  hipLaunchKernelGGL((attn_short_kernel<D, KB, HG>), dim3((uint32_t)blocks), dim3(G::NT), 0, s, p);
  return last_launch_status();
}

// Heads per work-group: a group's rows are fetched as runs of HG * D elements,
// which the memory system serves more efficiently than single 144-byte heads.
// Bounded by LDS (each head of a 128-key unit holds 72 KB at D = 72).
#ifndef DSP_TATTN_HG128
#define DSP_TATTN_HG128 2
#endif
#ifndef DSP_TATTN_HG64
#define DSP_TATTN_HG64 4
#endif
#ifndef DSP_TATTN_HG32
#define DSP_TATTN_HG32 4
#endif

template <int D, int KB, int HG>
int launch_short_hg(const AttnArgs& a, hipStream_t s) {
  if (HG > 1 && a.H % HG == 0) return launch_short_kb<D, KB, HG>(a, s);
  return launch_short_kb<D, KB, 1>(a, s);
}

template <int D>
int launch_short_d(const AttnArgs& a, hipStream_t s) {
  if (a.L <= 32) return launch_short_hg<D, 32, DSP_TATTN_HG32>(a, s);
  if (a.L <= 64) return launch_short_hg<D, 64, DSP_TATTN_HG64>(a, s);
  return launch_short_hg<D, 128, DSP_TATTN_HG128>(a, s);
}

}  // namespace

bool attn_bf16_short_fits(const AttnArgs& a) {
  // self-attention only (queries, keys and values of one layout and length);
  // unit indices and the byte offsets of a unit's rows (up to the padded
  // tile of 128) are 32-bit in the kernel
  if (a.Lk != a.L || a.Hkv != a.H || a.b_stride_kv != a.b_stride_in || a.x_stride_kv != a.x_stride_in ||
      a.r_stride_kv != a.r_stride_in)
    return false;
  return a.L >= 1 && a.L <= kShortAttnMaxL && a.B * a.X * a.H < (int64_t(1) << 32) &&
         (int64_t)kShortAttnMaxL * a.r_stride_in * 2 < (int64_t(1) << 31);
}

int launch_attn_bf16_short(const AttnArgs& a, hipStream_t s) {
  if (!attn_bf16_short_fits(a)) return DSP_ERR_SHAPE;
  if (a.B * a.X == 0) return DSP_OK;
  switch (a.D) {
    case 16: return launch_short_d<16>(a, s);
    case 32: return launch_short_d<32>(a, s);
    case 64: return launch_short_d<64>(a, s);
    case 72: return launch_short_d<72>(a, s);
    case 80: return launch_short_d<80>(a, s);
    case 96: return launch_short_d<96>(a, s);
    default: return DSP_ERR_SHAPE;
  }
}

}  // namespace dsp
