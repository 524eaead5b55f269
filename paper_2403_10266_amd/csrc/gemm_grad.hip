// Gradient GEMMs of the block's linear maps (the backward of Eq. 1's W^O, the
// Q/K/V projections and Eq. 5's W_1, W_2).  With y = x W^T (W stored [out][in],
// as in the forward), the gradients are
//   dx = dy W          -- [tokens, in]  = [tokens, out] x [out, in]
//   dW = dy^T x        -- [out, in]     = [out, tokens] x [tokens, in]
// so one operand, or both, has its reduction index strided in memory.  This
// kernel computes out[m][n] = sum_k A(m, k) B(n, k) for either storage of each
// operand:  A(m, k) = a[m * lda + k] (TA = 0) or a[k * lda + m] (TA = 1), and
// the same for B with TB.
//
// Design for gfx950, on v_mfma_f32_32x32x16_bf16 like the forward GEMM
// (256 x 128 tiles, 4 waves of 128 x 64, 64-wide k slices through LDS, the next
// slice prefetched into registers, B rows on the MFMA M side so a lane owns one
// output row):
//  * An operand stored with the reduction contiguous keeps the forward's LDS
//    layout [rows][k] (144-byte rows).  One stored transposed is copied as it
//    lies, [k][rows] (rows contiguous, 16-byte chunks), and its MFMA fragments
//    are read with ds_read_b64_tr_b16, which gives each lane 8 k values of one
//    row in the order {4g..4g+3, 8+4g..8+4g+3} of a 16-k step.  The natural
//    operand is read in the same k order (two 8-byte reads), so the two sides
//    of every MFMA agree.
//  * Split-K: the reduction range is cut into `splits` parts, one per grid z;
//    each writes fp32 partial sums to its own slab of a workspace and a second
//    kernel adds the slabs in a fixed order (no atomics: deterministic).  The
//    weight gradients reduce over all tokens (32768 at the block's size) onto
//    few output tiles, which is what this is for.
//  * Epilogues: fp32 output; bf16 output; the GELU / ReLU backward, out =
//    acc * act'(u) with u the saved pre-activation (bf16), rounded to bf16.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "attn_bf16_common.h"
#include "dsp_internal.h"

namespace dsp {
namespace {

constexpr int GBM = 256, GBN = 128, GBK = 64;
constexpr int GNTHR = 256;
constexpr int NPITCH = GBK + 8;   // natural tiles: 144-byte rows

template <int ROWS>
struct TPitch {
  static constexpr int P = ROWS + 8;  // transposed tiles: an odd multiple of 16 bytes
};

// d/du (u Phi(u)) = Phi(u) + u phi(u), with erf by Abramowitz and Stegun
// 7.1.26 (|error| <= 1.5e-7).  The exp(-z^2) of erf's tail at z = u / sqrt(2)
// is exp(-u^2 / 2) = sqrt(2 pi) phi(u): one exponential serves both terms.
__device__ __forceinline__ float gelu_grad(float u) {
  const float z = u * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, fabsf(z), 1.0f));
  float poly = fmaf(1.061405429f, t, -1.453152027f);
  poly = fmaf(poly, t, 1.421413741f);
  poly = fmaf(poly, t, -0.284496736f);
  poly = fmaf(poly, t, 0.254829592f);
  poly *= t;
  const float e = __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);
  const float erf = copysignf(1.0f - poly * e, z);
  return fmaf(0.5f, erf, 0.5f) + u * (0.3989422804014327f * e);
}

struct GradArgs {
  const bf16* a;
  const bf16* b;
  const bf16* aux;  // saved pre-activation for the activation backward epilogues
  void* out;        // [M][N] (or, with splits > 1, the fp32 workspace [splits][M][N])
  int64_t lda, ldb;
  int M, N, K, n_ntiles, n_tiles, k_per_split;
};

// One operand's tile of one k slice: global -> registers -> LDS, and its MFMA
// fragments.  ROWS = tile rows on the M or N side (256 or 128).
template <int ROWS, bool TRANS>
struct Operand {
  static constexpr int CHUNKS = ROWS * GBK / 8;    // 16-byte chunks per slice
  static constexpr int LOADS = CHUNKS / GNTHR;
  static constexpr int ELEMS = TRANS ? GBK * TPitch<ROWS>::P : ROWS * NPITCH;
  static_assert(CHUNKS % GNTHR == 0, "loader shape");

  const bf16* base;
  int64_t ld;
  int r0, rows_valid, k_total;
  u32x4 pre[LOADS];
  uint32_t off[LOADS];
  int lds_off[LOADS];
  bool col_ok[LOADS];

  __device__ void init(const bf16* p, int64_t ld_, int r0_, int rows_total, int k_total_) {
    base = p;
    ld = ld_;
    r0 = r0_;
    rows_valid = min(ROWS, rows_total - r0_);
    k_total = k_total_;
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      if (!TRANS) {
        // chunk (row t/8 + 32 i, k columns 8 (t % 8) .. + 7)
        const int row = (t >> 3) + 32 * i, kc = t & 7;
        off[i] = (uint32_t)row * (uint32_t)(ld * 2) + (uint32_t)kc * 16u;
        lds_off[i] = row * NPITCH + kc * 8;
        col_ok[i] = true;
      } else {
        // chunk (k row r, columns 8 c .. + 7), ROWS / 8 chunks per k row
        constexpr int CPR = ROWS / 8;
        const int c = t % CPR, r = t / CPR + (GNTHR / CPR) * i;
        off[i] = (uint32_t)r * (uint32_t)(ld * 2) + (uint32_t)c * 16u;
        lds_off[i] = r * TPitch<ROWS>::P + c * 8;
        col_ok[i] = 8 * c < rows_valid;
      }
    }
  }

  // loads the slice starting at reduction index k0 (rows / k past the end read zero)
  __device__ void load(int k0) {
    if (!TRANS) {
      const __amdgpu_buffer_rsrc_t rs =
          make_rsrc(base + (int64_t)r0 * ld, (uint32_t)max(rows_valid, 0) * (uint32_t)(ld * 2));
      const bool kin = k0 + 8 * (int)(threadIdx.x & 7) < k_total;
#pragma unroll
      for (int i = 0; i < LOADS; ++i)
        pre[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, kin ? off[i] + (uint32_t)k0 * 2u : 0xFFFFFFF0u, 0, 0);
    } else {
      const int krows = max(0, min(GBK, k_total - k0));
      const __amdgpu_buffer_rsrc_t rs =
          make_rsrc(base + (int64_t)k0 * ld + r0, (uint32_t)krows * (uint32_t)(ld * 2));
#pragma unroll
      for (int i = 0; i < LOADS; ++i)
        pre[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, col_ok[i] ? off[i] : 0xFFFFFFF0u, 0, 0);
    }
  }

  __device__ void store(bf16* lds) const {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) *reinterpret_cast<u32x4*>(lds + lds_off[i]) = pre[i];
  }

  // fragment of tile rows rbase .. rbase + 31 for 16-k step ks: lane
  // (l32 + 32g) gets row rbase + l32 at k = 16 ks + {4g..4g+3, 8+4g..8+4g+3}
  __device__ static bf16x8 frag(const bf16* lds, int rbase, int ks, int lane) {
    const int l32 = lane & 31, g = lane >> 5;
    if (!TRANS) {
      const bf16* row = lds + (rbase + l32) * NPITCH + 16 * ks + 4 * g;
      const shortx4 lo = *reinterpret_cast<const shortx4*>(row);
      const shortx4 hi = *reinterpret_cast<const shortx4*>(row + 8);
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    } else {
      constexpr int P = TPitch<ROWS>::P;
      const int j16 = lane & 15, mbase = 16 * ((lane >> 4) & 1);
      const int row = 16 * ks + 4 * g + (j16 >> 2);
      const int col = rbase + mbase + 4 * (j16 & 3);
      const shortx4 lo = lds_read_tr(lds + row * P + col);
      const shortx4 hi = lds_read_tr(lds + (row + 8) * P + col);
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
  }
};

template <bool TA, bool TB, int EPI>
__global__ __launch_bounds__(GNTHR, 2) void gemm_grad_kernel(GradArgs p) {
  using OA = Operand<GBM, TA>;
  using OB = Operand<GBN, TB>;
  __shared__ __attribute__((aligned(16))) bf16 As[OA::ELEMS];
  __shared__ __attribute__((aligned(16))) bf16 Bs[OB::ELEMS];

  // XCD-aware order (tiles m-major, n fastest; each XCD a contiguous range)
  uint32_t bid = blockIdx.x;
  if ((p.n_tiles & 7) == 0) bid = (bid & 7u) * ((uint32_t)p.n_tiles >> 3) + (bid >> 3);
  const int mt = bid / p.n_ntiles;
  const int nt = bid - mt * p.n_ntiles;
  const int m0 = mt * GBM, n0 = nt * GBN;
  const int kb = blockIdx.z * p.k_per_split;
  const int ke = min(p.K, kb + p.k_per_split);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;

  OA a;
  OB b;
  a.init(p.a, p.lda, m0, p.M, ke);
  b.init(p.b, p.ldb, n0, p.N, ke);

  floatx16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (ke - kb + GBK - 1) / GBK;
  if (nk > 0) {
    a.load(kb);
    b.load(kb);
    a.store(As);
    b.store(Bs);
  }
  __syncthreads();
  for (int it = 0; it < nk; ++it) {
    const bool more = it + 1 < nk;
    if (more) {
      a.load(kb + (it + 1) * GBK);
      b.load(kb + (it + 1) * GBK);
    }
#pragma unroll
    for (int ks = 0; ks < GBK / 16; ++ks) {
      bf16x8 af[4], bfr[2];
#pragma unroll
      for (int j = 0; j < 4; ++j) af[j] = OA::frag(As, wm * 128 + 32 * j, ks, lane);
#pragma unroll
      for (int i = 0; i < 2; ++i) bfr[i] = OB::frag(Bs, wn * 64 + 32 * i, ks, lane);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[i], af[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      __syncthreads();
      a.store(As);
      b.store(Bs);
      __syncthreads();
    }
  }

  // epilogue: lane owns row m = .. + l32 and columns n = .. + 8 r4 + 4g + {0..3}
  const int64_t slab = (int64_t)blockIdx.z * p.M * p.N;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + wm * 128 + 32 * j + l32;
    if (m >= p.M) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int n = n0 + wn * 64 + 32 * i + 8 * r4 + 4 * g;
        if (n >= p.N) continue;   // N % 4 == 0: the group of 4 is whole
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * r4 + e];
        const int64_t off = (int64_t)m * p.N + n;
        if (EPI == DSP_GRAD_EPI_F32) {
          *reinterpret_cast<float4*>(static_cast<float*>(p.out) + slab + off) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          if (EPI == DSP_GRAD_EPI_GELU_BWD || EPI == DSP_GRAD_EPI_RELU_BWD) {
            const uint2 uw = *reinterpret_cast<const uint2*>(p.aux + off);
            const bf16x2 u01 = __builtin_bit_cast(bf16x2, uw.x), u23 = __builtin_bit_cast(bf16x2, uw.y);
            const float u[4] = {(float)u01[0], (float)u01[1], (float)u23[0], (float)u23[1]};
#pragma unroll
            for (int e = 0; e < 4; ++e)
              v[e] *= EPI == DSP_GRAD_EPI_GELU_BWD ? gelu_grad(u[e]) : (u[e] > 0.0f ? 1.0f : 0.0f);
          }
          bf16x2 lo = {(bf16)v[0], (bf16)v[1]};
          bf16x2 hi = {(bf16)v[2], (bf16)v[3]};
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, lo);
          w.y = __builtin_bit_cast(uint32_t, hi);
          *reinterpret_cast<uint2*>(static_cast<bf16*>(p.out) + off) = w;
        }
      }
  }
}

// out[i] = sum over z of ws[z][i], z in order (deterministic)
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float4* __restrict__ ws, float4* out,
                                                            int64_t n4, int splits) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 s = ws[i];
  for (int z = 1; z < splits; ++z) {
    const float4 v = ws[(int64_t)z * n4 + i];
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  out[i] = s;
}

// db[n] = sum over rows m of dy[m][n] (fp32), one thread per column group of 4,
// rows in order (deterministic)
__global__ __launch_bounds__(256) void colsum_bf16_kernel(const bf16* __restrict__ dy, float* db, int64_t M,
                                                          int N) {
  const int n4 = blockIdx.x * blockDim.x + threadIdx.x;
  if (4 * n4 >= N) return;
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t m = 0; m < M; ++m) {
    const uint2 w = *reinterpret_cast<const uint2*>(dy + m * N + 4 * n4);
    const bf16x2 a = __builtin_bit_cast(bf16x2, w.x), b = __builtin_bit_cast(bf16x2, w.y);
    s[0] += (float)a[0];
    s[1] += (float)a[1];
    s[2] += (float)b[0];
    s[3] += (float)b[1];
  }
  *reinterpret_cast<float4*>(db + 4 * n4) = make_float4(s[0], s[1], s[2], s[3]);
}

// ---------------------------------------------------------------------------
// Large-tile weight gradient: out[M][N] = sum over k of a[k][m] b[k][n] (both
// operands stored with the reduction index as rows: dW = dy^T x), fp32, with
// the reduction split over blockIdx.z into fp32 partials.  The schedule of
// gemm_bf16_big_kernel (gemm.hip): 256 x (64 TN) output tiles, 4 waves of
// 128 x (32 TN) on one SIMD each with the accumulators in AGPRs, two LDS
// buffers and one barrier per 64-wide k slice (before its last 16-wide step),
// the next slice's LDS stores and the loads after them spread over the MFMAs
// of steps 0-2, each step's fragments read during the previous step's MFMAs.  Tiles
// hold k rows of the tile's columns as they lie in memory; fragments are read
// with ds_read_b64_tr_b16 (k order {4g..4g+3, 8+4g..8+4g+3} on both sides).
constexpr int GB_BM = 256;
#ifndef DSP_GRAD_BIG
#define DSP_GRAD_BIG 1
#endif

template <int TN>
__global__ __launch_bounds__(GNTHR, 1) void gemm_grad_tt_big_kernel(GradArgs p) {
  constexpr int TM = 4;
  constexpr int BNB = 2 * TN * 32;
  constexpr int PA = GB_BM + 8, PB = BNB + 8;   // k-row pitches: odd multiples of 16 bytes
  constexpr int A_EL = GBK * PA, STAGE = A_EL + GBK * PB;
  constexpr int CA = GB_BM / 8, CB = BNB / 8;   // 16-byte chunks per k row
  constexpr int A_LOADS = GBK * CA / GNTHR, B_LOADS = GBK * CB / GNTHR, NL = A_LOADS + B_LOADS;
  static_assert(GBK * CA % GNTHR == 0 && GBK * CB % GNTHR == 0, "loader shape");
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * STAGE];

  // tile order: contiguous ranges per XCD, then groups of 4 m-tiles (m fastest)
  uint32_t bid = blockIdx.x;
  if ((p.n_tiles & 7) == 0) bid = (bid & 7u) * ((uint32_t)p.n_tiles >> 3) + (bid >> 3);
  const int n_mt = p.n_tiles / p.n_ntiles;
  const int per_group = 4 * p.n_ntiles;
  const int grp = (int)bid / per_group;
  const int first_m = grp * 4;
  const int gm = min(4, n_mt - first_m);
  const int rem = (int)bid - grp * per_group;
  const int m0 = (first_m + rem % gm) * GB_BM, n0 = (rem / gm) * BNB;
  const int kb = blockIdx.z * p.k_per_split;
  const int ke = min(p.K, kb + p.k_per_split);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;
  const int j16 = lane & 15, mbase = 16 * ((lane >> 4) & 1);

  // loader: chunk e = t + 256 i of a tensor's slice is k row e / C, columns
  // 8 (e % C) .. + 7 of the tile; columns past M (N) read zero
  uint32_t off[NL];
  int lofs[NL];
  bool ok[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const bool is_a = i < A_LOADS;
    const int e = threadIdx.x + GNTHR * (is_a ? i : i - A_LOADS);
    const int C = is_a ? CA : CB;
    const int r = e / C, c = e % C;
    off[i] = (uint32_t)r * (uint32_t)((is_a ? p.lda : p.ldb) * 2) + (uint32_t)c * 16u;
    lofs[i] = is_a ? r * PA + c * 8 : A_EL + r * PB + c * 8;
    ok[i] = is_a ? m0 + 8 * c < p.M : n0 + 8 * c < p.N;
  }
  u32x4 pre[NL];
  __amdgpu_buffer_rsrc_t ra, rb;
  auto rsrcs = [&](int k0) {  // the slice's k rows below ke (rows past it read zero)
    const uint32_t krows = (uint32_t)max(0, min(GBK, ke - k0));
    ra = make_rsrc(p.a + (int64_t)k0 * p.lda + m0, krows * (uint32_t)(p.lda * 2));
    rb = make_rsrc(p.b + (int64_t)k0 * p.ldb + n0, krows * (uint32_t)(p.ldb * 2));
  };
  auto gload = [&](int i) {
    pre[i] = __builtin_amdgcn_raw_buffer_load_b128(i < A_LOADS ? ra : rb, ok[i] ? off[i] : 0xFFFFFFF0u, 0, 0);
  };
  auto lstore = [&](int i, int buf) { *reinterpret_cast<u32x4*>(lds + buf * STAGE + lofs[i]) = pre[i]; };

  floatx16 acc[TN][TM];
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  auto frag = [&](const bf16* t, int P, int rbase, int ks) {
    const int row = 16 * ks + 4 * g + (j16 >> 2);
    const int col = rbase + mbase + 4 * (j16 & 3);
    const shortx4 lo = lds_read_tr(t + row * P + col);
    const shortx4 hi = lds_read_tr(t + (row + 8) * P + col);
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  bf16x8 af[2][TM], wf[2][TN];
  auto fread = [&](int slot, int buf, int ks) {
    const bf16* As = lds + buf * STAGE;
    const bf16* Bs = As + A_EL;
#pragma unroll
    for (int b = 0; b < TM; ++b) af[slot][b] = frag(As, PA, wm * TM * 32 + 32 * b, ks);
#pragma unroll
    for (int a = 0; a < TN; ++a) wf[slot][a] = frag(Bs, PB, wn * TN * 32 + 32 * a, ks);
  };

  auto slice = [&](int kt, auto st_c, auto ld_c) {
    constexpr bool ST = decltype(st_c)::value, LD = decltype(ld_c)::value;
    constexpr int NMF = TM * TN;
    constexpr int NSPREAD = 3;  // steps that carry the next slice's LDS stores
    const int b = kt & 1;
    if (LD) rsrcs(kb + (kt + 2) * GBK);
#pragma unroll
    for (int ks = 0; ks < GBK / 16; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < GBK / 16) {
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
            if (LD) gload(i);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  const int nk = (ke - kb + GBK - 1) / GBK;
  if (nk > 0) {
    rsrcs(kb);
#pragma unroll
    for (int i = 0; i < NL; ++i) gload(i);
#pragma unroll
    for (int i = 0; i < NL; ++i) lstore(i, 0);
    if (nk > 1) {
      rsrcs(kb + GBK);
#pragma unroll
      for (int i = 0; i < NL; ++i) gload(i);
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
    slice(kt, no{}, no{});
  }

  // fp32 partial (or the result, unsplit).  The lane holds rows
  // m = .. + 32 bb + l32 and column groups n = .. + 32 a + 8 r4 + 4 g + {0..3};
  // stored from there, a store instruction would write 16-byte pieces of 32
  // rows.  So the tile goes through LDS in two passes of 128 rows (rows
  // 64 p + [0, 64) of each wave row half) and leaves in whole 16-byte row
  // chunks, consecutive lanes on consecutive chunks.
  float* out = static_cast<float*>(p.out) + (int64_t)blockIdx.z * p.M * p.N;
  constexpr int SPF = BNB + 4;  // staged row pitch (fp32): a 16-byte pad
  static_assert(128 * SPF * 4 <= 2 * STAGE * 2, "the staging fits the LDS buffers");
  constexpr int CPR = BNB / 4, PER = 128 * CPR / GNTHR;
  float* sf = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    __syncthreads();  // pass 0: the last fragments are read; pass 1: pass 0's rows are read
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int a = 0; a < TN; ++a)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const floatx16& t = acc[a][2 * pass + h];
          *reinterpret_cast<float4*>(sf + (wm * 64 + 32 * h + l32) * SPF + wn * TN * 32 + 32 * a + 8 * r4 + 4 * g) =
              make_float4(t[4 * r4], t[4 * r4 + 1], t[4 * r4 + 2], t[4 * r4 + 3]);
        }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int c = (int)threadIdx.x + GNTHR * q;
      const int sr = c / CPR, cc = c % CPR;
      const int m = m0 + (sr / 64) * 128 + 64 * pass + sr % 64, n = n0 + 4 * cc;
      if (m < p.M && n < p.N)
        *reinterpret_cast<float4*>(out + (int64_t)m * p.N + n) =
            *reinterpret_cast<const float4*>(sf + sr * SPF + 4 * cc);
    }
  }
}

// Whether the weight gradient out[M][N] (reduction K, row strides lda, ldb)
// runs on the large-tile kernel, and with which tile width.
bool grad_big_ok(int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb) {
  return DSP_GRAD_BIG && M >= 512 && N >= 512 && M % 8 == 0 && N % 8 == 0 && K >= 2048 &&
         (int64_t)GBK * lda * 2 < (int64_t(1) << 31) && (int64_t)GBK * ldb * 2 < (int64_t(1) << 31) &&
         M * N < (int64_t(1) << 31);
}
int grad_big_tn(int64_t N) { return N >= 2048 ? 4 : 3; }

template <bool TA, bool TB, int EPI>
int launch_grad(const GradArgs& p0, int splits, float* ws, hipStream_t s) {
  GradArgs p = p0;
  const int64_t n_mt = (p.M + GBM - 1) / GBM, n_nt = (p.N + GBN - 1) / GBN;
  const int64_t tiles = n_mt * n_nt;
  p.n_ntiles = (int)n_nt;
  p.n_tiles = (int)tiles;
  p.k_per_split = ((p.K + splits - 1) / splits + GBK - 1) / GBK * GBK;
  void* final_out = p.out;
  if (splits > 1) p.out = ws;
  hipLaunchKernelGGL((gemm_grad_kernel<TA, TB, EPI>), dim3((uint32_t)tiles, 1, (uint32_t)splits), dim3(GNTHR),
                     0, s, p);
  int st = last_launch_status();
  if (st != DSP_OK || splits == 1) return st;
  const int64_t n4 = (int64_t)p.M * p.N / 4;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((uint32_t)((n4 + 255) / 256)), dim3(256), 0, s,
                     reinterpret_cast<const float4*>(ws), reinterpret_cast<float4*>(final_out), n4, splits);
  return last_launch_status();
}

// fp32 path: out[m][n] = sum_k A(m, k) B(n, k) with the same storage choices,
// plain FMA, one thread per output (small problems and checks)
__global__ __launch_bounds__(256) void gemm_grad_f32_kernel(const float* a, int ta, int64_t lda, const float* b,
                                                            int tb, int64_t ldb, const float* aux, float* out,
                                                            int64_t M, int64_t N, int64_t K, int epi) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M * N) return;
  const int64_t m = i / N, n = i % N;
  float s = 0.0f;
  for (int64_t k = 0; k < K; ++k) {
    const float av = ta ? a[k * lda + m] : a[m * lda + k];
    const float bv = tb ? b[k * ldb + n] : b[n * ldb + k];
    s = fmaf(av, bv, s);
  }
  if (epi == DSP_GRAD_EPI_GELU_BWD) {
    const float u = aux[i];
    s *= 0.5f * (1.0f + erff(u * 0.70710678118654752f)) + u * 0.3989422804014327f * expf(-0.5f * u * u);
  } else if (epi == DSP_GRAD_EPI_RELU_BWD) {
    s = aux[i] > 0.0f ? s : 0.0f;
  }
  out[i] = s;
}

__global__ __launch_bounds__(256) void colsum_f32_kernel(const float* __restrict__ dy, float* db, int64_t M,
                                                         int N) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  float s = 0.0f;
  for (int64_t m = 0; m < M; ++m) s += dy[m * N + n];
  db[n] = s;
}

// out = a + b (fp32); out may alias a or b
__global__ __launch_bounds__(256) void add_f32_kernel(const float* a, const float* b, float* out, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) out[i] = a[i] + b[i];
}

}  // namespace

int launch_add_f32(const float* a, const float* b, float* out, int64_t n, hipStream_t s) {
  if (n == 0) return DSP_OK;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL(add_f32_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, a, b, out, n);
  return last_launch_status();
}

int launch_gemm_grad_f32(const float* a, int ta, int64_t lda, const float* b, int tb, int64_t ldb,
                         const float* aux, float* out, int64_t M, int64_t N, int64_t K, int epi, hipStream_t s) {
  const int64_t total = M * N;
  if (total == 0) return DSP_OK;
  const int64_t blocks = (total + 255) / 256;
  if (blocks >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  hipLaunchKernelGGL(gemm_grad_f32_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, a, ta, lda, b, tb, ldb, aux,
                     out, M, N, K, epi);
  return last_launch_status();
}

int launch_colsum_f32(const float* dy, float* db, int64_t M, int N, hipStream_t s) {
  if (N == 0) return DSP_OK;
  hipLaunchKernelGGL(colsum_f32_kernel, dim3((uint32_t)((N + 255) / 256)), dim3(256), 0, s, dy, db, M, N);
  return last_launch_status();
}

int grad_splits(int64_t M, int64_t N, int64_t K) {
  if (grad_big_ok(M, N, K, M, N)) {
    // the large-tile kernel: one work-group per CU (256 slots), in units of
    // one 64-wide slice of a tile on a full round; a split's extra fp32
    // partial (8 M N bytes at 5 TB/s) against ~2 us per slice round
    const int bnb = grad_big_tn(N) * 64;
    const int64_t tiles = ((M + GB_BM - 1) / GB_BM) * ((N + bnb - 1) / bnb);
    const int64_t slices = (K + GBK - 1) / GBK;
    const double per_split = (double)M * (double)N * 8e-7;
    int best = 1;
    double best_cost = 0.0;
    for (int s = 1; s <= 16; ++s) {
      const int64_t per = (slices + s - 1) / s;
      if (per < 32 || per * (s - 1) >= slices) break;
      const int64_t rounds = (tiles * s + 255) / 256;
      const double cost = (double)rounds * (double)(per + 2) + (s > 1 ? s * per_split : 0.0);
      if (s == 1 || cost < best_cost) {
        best = s;
        best_cost = cost;
      }
    }
    return best;
  }
  // The split count minimising a cost model, in units of one 64-wide K slice
  // of one tile on a full round of work-groups (two per CU, 256 CUs):
  //   rounds * (slices per split + 2 for the work-group's set-up and fp32
  //   store) + s * (the extra write and read of an M x N fp32 partial,
  //   about 8 M N bytes at 5 TB/s against 2.9 us per slice round).
  // Splits keep at least 32 slices (a reduction of 2048), so small problems
  // run unsplit.
  const int64_t tiles = ((M + GBM - 1) / GBM) * ((N + GBN - 1) / GBN);
  const int64_t slices = (K + GBK - 1) / GBK;
  const double per_split = (double)M * (double)N * 5.5e-7;
  int best = 1;
  double best_cost = 0.0;
  for (int s = 1; s <= 16; ++s) {
    const int64_t per = (slices + s - 1) / s;
    if (per < 32 || per * (s - 1) >= slices) break;  // too short, or the last split empty
    const int64_t rounds = (tiles * s + 511) / 512;
    const double cost = (double)rounds * (double)(per + 2) + (s > 1 ? s * per_split : 0.0);
    if (s == 1 || cost < best_cost) {
      best = s;
      best_cost = cost;
    }
  }
  return best;
}

bool grad_gemm_fits(int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb) {
  // 32-bit tile offsets: GBM (or GBK) rows of a row stride in bytes
  return M < (int64_t(1) << 31) && N < (int64_t(1) << 31) && K < (int64_t(1) << 31) &&
         (int64_t)GBM * lda * 2 < (int64_t(1) << 31) && (int64_t)GBM * ldb * 2 < (int64_t(1) << 31) &&
         ((M + GBM - 1) / GBM) * ((N + GBN - 1) / GBN) < (int64_t(1) << 31);
}

int launch_gemm_grad(const void* a, int ta, int64_t lda, const void* b, int tb, int64_t ldb, const void* aux,
                     void* out, int64_t M, int64_t N, int64_t K, int epi, int splits, float* ws, hipStream_t s) {
  if (M == 0 || N == 0) return DSP_OK;
  GradArgs p;
  p.a = static_cast<const bf16*>(a);
  p.b = static_cast<const bf16*>(b);
  p.aux = static_cast<const bf16*>(aux);
  p.out = out;
  p.lda = lda;
  p.ldb = ldb;
  p.M = (int)M;
  p.N = (int)N;
  p.K = (int)K;
  if (ta == 1 && tb == 1 && epi == DSP_GRAD_EPI_F32 && grad_big_ok(M, N, K, lda, ldb) &&
      (splits == 1 || ws)) {
    const int tn = grad_big_tn(N);
    const int bnb = tn * 64;
    const int64_t n_nt = (N + bnb - 1) / bnb;
    const int64_t tiles = ((M + GB_BM - 1) / GB_BM) * n_nt;
    p.n_ntiles = (int)n_nt;
    p.n_tiles = (int)tiles;
    p.k_per_split = ((p.K + splits - 1) / splits + GBK - 1) / GBK * GBK;
    if (splits > 1) p.out = ws;
    if (tn == 4)
      hipLaunchKernelGGL((gemm_grad_tt_big_kernel<4>), dim3((uint32_t)tiles, 1, (uint32_t)splits), dim3(GNTHR), 0, s,
                         p);
    else
      hipLaunchKernelGGL((gemm_grad_tt_big_kernel<3>), dim3((uint32_t)tiles, 1, (uint32_t)splits), dim3(GNTHR), 0, s,
                         p);
    int st = last_launch_status();
    if (st != DSP_OK || splits == 1) return st;
    const int64_t n4 = M * N / 4;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((uint32_t)((n4 + 255) / 256)), dim3(256), 0, s,
                       reinterpret_cast<const float4*>(ws), reinterpret_cast<float4*>(out), n4, splits);
    return last_launch_status();
  }
#define DSP_GRAD_CASE(TA_, TB_)                                                                    \
  if (ta == TA_ && tb == TB_) {                                                                   \
    switch (epi) {                                                                                \
      case DSP_GRAD_EPI_F32: return launch_grad<TA_, TB_, DSP_GRAD_EPI_F32>(p, splits, ws, s);    \
      case DSP_GRAD_EPI_BF16: return launch_grad<TA_, TB_, DSP_GRAD_EPI_BF16>(p, 1, ws, s);       \
      case DSP_GRAD_EPI_GELU_BWD: return launch_grad<TA_, TB_, DSP_GRAD_EPI_GELU_BWD>(p, 1, ws, s); \
      case DSP_GRAD_EPI_RELU_BWD: return launch_grad<TA_, TB_, DSP_GRAD_EPI_RELU_BWD>(p, 1, ws, s); \
      default: return DSP_ERR_ARG;                                                                \
    }                                                                                             \
  }
  DSP_GRAD_CASE(0, 1)
  DSP_GRAD_CASE(1, 1)
  DSP_GRAD_CASE(0, 0)
  DSP_GRAD_CASE(1, 0)
#undef DSP_GRAD_CASE
  return DSP_ERR_ARG;
}

int launch_colsum_bf16(const void* dy, float* db, int64_t M, int N, hipStream_t s) {
  if (N == 0) return DSP_OK;
  const int groups = (N + 3) / 4;
  hipLaunchKernelGGL(colsum_bf16_kernel, dim3((uint32_t)((groups + 255) / 256)), dim3(256), 0, s,
                     static_cast<const bf16*>(dy), db, M, N);
  return last_launch_status();
}

}  // namespace dsp
