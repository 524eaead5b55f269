// Fused bf16 attention along one sequence dimension (Eq. 3 per head, Eq. 1-2),
// applied to the per-dimension reshape of a multi-dimensional sequence
// (Eq. 7-8): every (batch, other-dimension index, head) triple is an
// independent problem over L consecutive sequence positions.  Spatial
// attention (L = S) and temporal attention (L = T) are the same kernel with
// different L and strides.
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
//    32 for P V (72 -> 96).  Padding columns of K in LDS are zero; for D not
//    a multiple of 32, padding column D of V is 1.0, so the P V product also
//    yields the softmax row sum from the bf16 probabilities actually used.
//  * K and V tiles of 64 keys are staged in LDS, double-buffered, with
//    register prefetch of the next tile overlapping the current tile's math.
//    K rows are read as 16-byte MFMA A fragments (row pitch an odd multiple
//    of 16 bytes: conflict-free); V fragments come straight from row-major
//    LDS through ds_read_b64_tr_b16, so V is never transposed in memory.
//  * Online softmax in the exp2 domain with the running maximum updated
//    lazily: a wave only rescales its O accumulators when some query's block
//    maximum exceeds its running maximum by more than 2^8, which after the
//    first blocks is rare; exactness does not depend on the reference point.
//  * Work-group index -> (unit, query block) is remapped so that consecutive
//    units land on the same XCD: the query blocks of a unit, and neighbouring
//    heads of a token row, then share that XCD's L2.
#include <math.h>

#include "dsp_internal.h"

namespace dsp {
namespace {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short shortx4;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short shortx8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

constexpr int KB = 64;          // keys per LDS tile (two 32-key MFMA tiles)
constexpr float kLazyRescale = 8.0f;  // log2 headroom before the running max is moved

__device__ __forceinline__ float swap_halves(float v) {
  // value held by lane (l ^ 32)
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(threadIdx.x & 32 ? r[0] : r[1]);
}

__device__ __forceinline__ shortx4 lds_read_tr(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) shortx4*)(p));
}

template <int D>
struct Geo {
  static constexpr int NDK = (D + 15) / 16;       // 16-wide d steps of Q K^T
  static constexpr int NDV = (D + 31) / 32;       // 32-row d tiles of P V
  static constexpr bool ONES = (D % 32) != 0;     // spare V column carries the row sum
  static constexpr int KP = NDK * 16 + 8;         // K row pitch (elements)
  static constexpr int VP = NDV * 32 + 16;        // V row pitch (elements)
  static constexpr int CH = D / 8;                // 16-byte chunks per row
  static constexpr int TILE_ELEMS = KB * (KP + VP);
};

struct Params {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  bf16* o;
  int64_t b_in, x_in, r_in, b_out, x_out, r_out;
  uint32_t X, H, L, n_units, n_qb, n_blocks;
  float c;  // scale * log2(e)
};

template <int D, int NW, int QT>
__global__ __launch_bounds__(NW * 64) void attn_fwd_kernel(Params p) {
  using G = Geo<D>;
  constexpr int NT = NW * 64;
  constexpr int QW = 32 * QT;                      // queries per wave
  constexpr int QB = NW * QW;                      // queries per work-group
  constexpr int NCHUNK = 2 * KB * G::CH;           // 16-byte chunks per K+V tile
  constexpr int NLOAD = (NCHUNK + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * G::TILE_ELEMS];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31;
  const int g = lane >> 5;

  // XCD-aware block order: hardware places block i on XCD i % 8.
  uint32_t bid = blockIdx.x;
  if ((p.n_blocks & 7u) == 0) bid = (bid & 7u) * (p.n_blocks >> 3) + (bid >> 3);
  const uint32_t unit = bid / p.n_qb;
  const uint32_t qb = bid - unit * p.n_qb;
  const uint32_t h = unit % p.H;
  const uint32_t bx = unit / p.H;
  const uint32_t xx = bx % p.X;
  const uint32_t bb = bx / p.X;
  const int64_t in_base = (int64_t)bb * p.b_in + (int64_t)xx * p.x_in + (int64_t)h * D;
  const int64_t out_base = (int64_t)bb * p.b_out + (int64_t)xx * p.x_out + (int64_t)h * D;
  const bf16* __restrict__ qg = p.q + in_base;
  const bf16* __restrict__ kg = p.k + in_base;
  const bf16* __restrict__ vg = p.v + in_base;
  const uint32_t L = p.L;

  // ---- padding columns of both LDS buffers: K pad = 0, V pad = [1 (row sum), 0...]
  for (int e = threadIdx.x; e < 2 * KB; e += NT) {
    bf16* t = lds + (e / KB) * G::TILE_ELEMS;
    const int r = e % KB;
    for (int c = D; c < G::KP; ++c) t[r * G::KP + c] = (bf16)0.0f;
    bf16* vt = t + KB * G::KP;
    for (int c = D; c < G::VP; ++c) vt[r * G::VP + c] = (bf16)((G::ONES && c == D) ? 1.0f : 0.0f);
  }

  // ---- Q fragments (B operand of S^T = K Q^T): lane (n + 32g) holds Q[q][16s + 8g .. +7]
  const uint32_t q_wave = qb * QB + wave * QW;
  bf16x8 qf[QT][G::NDK];
#pragma unroll
  for (int j = 0; j < QT; ++j) {
    const uint32_t q = q_wave + 32 * j + l32;
#pragma unroll
    for (int s = 0; s < G::NDK; ++s) {
      const int d = 16 * s + 8 * g;
      if (q < L && d < D) {
        qf[j][s] = *reinterpret_cast<const bf16x8*>(qg + (int64_t)q * p.r_in + d);
      } else {
        for (int e = 0; e < 8; ++e) qf[j][s][e] = (bf16)0.0f;
      }
    }
  }

  // ---- tile loader: chunk c -> (tensor, row, column chunk)
  uint4 pre[NLOAD];
  auto load_tile = [&](uint32_t kb) {
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int c = threadIdx.x + i * NT;
      pre[i] = make_uint4(0, 0, 0, 0);
      if (c < NCHUNK) {
        const int tsr = c / (KB * G::CH);
        const int rc = c - tsr * (KB * G::CH);
        const int row = rc / G::CH;
        const int col = rc - row * G::CH;
        if (kb + row < L) {
          const bf16* src = (tsr ? vg : kg) + (int64_t)(kb + row) * p.r_in + col * 8;
          pre[i] = *reinterpret_cast<const uint4*>(src);
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
    bf16* t = lds + buf * G::TILE_ELEMS;
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int c = threadIdx.x + i * NT;
      if (c < NCHUNK) {
        const int tsr = c / (KB * G::CH);
        const int rc = c - tsr * (KB * G::CH);
        const int row = rc / G::CH;
        const int col = rc - row * G::CH;
        bf16* dst = tsr ? (t + KB * G::KP + row * G::VP + col * 8) : (t + row * G::KP + col * 8);
        *reinterpret_cast<uint4*>(dst) = pre[i];
      }
    }
  };

  floatx16 o[G::NDV][QT];
#pragma unroll
  for (int t = 0; t < G::NDV; ++t)
#pragma unroll
    for (int j = 0; j < QT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][j][r] = 0.0f;
  float m_run[QT], l_run[QT];
#pragma unroll
  for (int j = 0; j < QT; ++j) { m_run[j] = -INFINITY; l_run[j] = 0.0f; }

  const uint32_t n_kb = (L + KB - 1) / KB;
  load_tile(0);
  __syncthreads();  // padding columns written before tile rows land beside them
  store_tile(0);
  __syncthreads();

  for (uint32_t it = 0; it < n_kb; ++it) {
    const uint32_t kb = it * KB;
    if (it + 1 < n_kb) load_tile(kb + KB);
    const bf16* kt_lds = lds + (it & 1) * G::TILE_ELEMS;
    const bf16* vt_lds = kt_lds + KB * G::KP;

    // S^T = K Q^T for two 32-key tiles
    floatx16 sacc[2][QT];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int j = 0; j < QT; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kt][j][r] = 0.0f;
#pragma unroll
      for (int s = 0; s < G::NDK; ++s) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(kt_lds + (32 * kt + l32) * G::KP + 16 * s + 8 * g);
#pragma unroll
        for (int j = 0; j < QT; ++j)
          sacc[kt][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[j][s], sacc[kt][j], 0, 0, 0);
      }
    }

    // mask keys past L (only the last tile can hold any)
    if (kb + KB > L) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t key = kb + 32 * kt + (r / 4) * 8 + 4 * g + (r % 4);
          if (key >= L) {
#pragma unroll
            for (int j = 0; j < QT; ++j) sacc[kt][j][r] = -INFINITY;
          }
        }
    }

    // online softmax (exp2 domain), lazily moved reference maximum
    float mblk[QT];
    bool need = false;
#pragma unroll
    for (int j = 0; j < QT; ++j) {
      float mx = sacc[0][j][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sacc[0][j][r]);
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[1][j][r]);
      mx = fmaxf(mx, swap_halves(mx));
      mblk[j] = mx * p.c;
      need |= mblk[j] > m_run[j] + kLazyRescale;
    }
    if (__any(need)) {
#pragma unroll
      for (int j = 0; j < QT; ++j) {
        const float mnew = fmaxf(m_run[j], mblk[j]);
        const float alpha = __builtin_amdgcn_exp2f(m_run[j] - mnew);
        m_run[j] = mnew;
        l_run[j] *= alpha;
#pragma unroll
        for (int t = 0; t < G::NDV; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[t][j][r] *= alpha;
      }
    }
    bf16x8 pf[2][2][QT];  // [key tile][16-key step][query tile]
#pragma unroll
    for (int j = 0; j < QT; ++j) {
      const float mc = m_run[j];
      float ls = 0.0f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = __builtin_amdgcn_exp2f(fmaf(sacc[kt][j][r], p.c, -mc));
          if (!G::ONES) ls += e;
          pf[kt][r / 8][j][r % 8] = (bf16)e;
        }
      if (!G::ONES) l_run[j] += ls;
    }

    // O^T += V^T P^T: A fragment of V^T via transposing LDS reads
    const int j16 = lane & 15;
    const int mbase = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int t = 0; t < G::NDV; ++t) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int row = 32 * kt + 16 * kk + 4 * g + (j16 >> 2);
          const int col = 32 * t + mbase + 4 * (j16 & 3);
          const shortx4 lo = lds_read_tr(vt_lds + row * G::VP + col);
          const shortx4 hi = lds_read_tr(vt_lds + (row + 8) * G::VP + col);
          const shortx8 both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          const bf16x8 a = __builtin_bit_cast(bf16x8, both);
#pragma unroll
          for (int j = 0; j < QT; ++j)
            o[t][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kt][kk][j], o[t][j], 0, 0, 0);
        }
    }

    if (it + 1 < n_kb) store_tile((it + 1) & 1);
    __syncthreads();
  }

  // ---- normalise and store: lane (n + 32g) holds O^T[32t + 8(r/4) + 4g + r%4][q]
  bf16* __restrict__ og = p.o + out_base;
#pragma unroll
  for (int j = 0; j < QT; ++j) {
    float l;
    if (G::ONES) {
      constexpr int tl = D / 32, ml = D % 32;
      constexpr int gl = (ml / 4) % 2, rl = (ml / 8) * 4 + ml % 4;
      const float vsum = o[tl][j][rl];
      const float other = swap_halves(vsum);
      l = (g == gl) ? vsum : other;
    } else {
      l = l_run[j] + swap_halves(l_run[j]);
    }
    const float inv = 1.0f / l;
    const uint32_t q = q_wave + 32 * j + l32;
    if (q < L) {
      bf16* orow = og + (int64_t)q * p.r_out;
#pragma unroll
      for (int t = 0; t < G::NDV; ++t)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int d0 = 32 * t + 8 * r4 + 4 * g;
          if (d0 < D) {
            bf16x2 lo = {(bf16)(o[t][j][4 * r4 + 0] * inv), (bf16)(o[t][j][4 * r4 + 1] * inv)};
            bf16x2 hi = {(bf16)(o[t][j][4 * r4 + 2] * inv), (bf16)(o[t][j][4 * r4 + 3] * inv)};
            uint2 w;
            w.x = __builtin_bit_cast(uint32_t, lo);
            w.y = __builtin_bit_cast(uint32_t, hi);
            *reinterpret_cast<uint2*>(orow + d0) = w;
          }
        }
    }
  }
}

template <int D, int NW, int QT>
int launch_cfg(const AttnArgs& a, hipStream_t s) {
  constexpr int QB = NW * 32 * QT;
  Params p;
  p.q = static_cast<const bf16*>(a.q);
  p.k = static_cast<const bf16*>(a.k);
  p.v = static_cast<const bf16*>(a.v);
  p.o = static_cast<bf16*>(a.o);
  p.b_in = a.b_stride_in;
  p.x_in = a.x_stride_in;
  p.r_in = a.r_stride_in;
  p.b_out = a.b_stride_out;
  p.x_out = a.x_stride_out;
  p.r_out = a.r_stride_out;
  p.X = (uint32_t)a.X;
  p.H = (uint32_t)a.H;
  p.L = (uint32_t)a.L;
  const int64_t units = a.B * a.X * a.H;
  const int64_t n_qb = (a.L + QB - 1) / QB;
  const int64_t blocks = units * n_qb;
  if (blocks == 0) return DSP_OK;
  if (blocks >= (int64_t(1) << 31) || a.L >= (int64_t(1) << 30)) return DSP_ERR_SHAPE;
  p.n_units = (uint32_t)units;
  p.n_qb = (uint32_t)n_qb;
  p.n_blocks = (uint32_t)blocks;
  p.c = a.scale * 1.4426950408889634f;
  hipLaunchKernelGGL((attn_fwd_kernel<D, NW, QT>), dim3((uint32_t)blocks), dim3(NW * 64), 0, s, p);
  return last_launch_status();
}

template <int D>
int launch_d(const AttnArgs& a, hipStream_t s) {
  if (a.L <= 32) return launch_cfg<D, 1, 1>(a, s);
  if (a.L <= 64) return launch_cfg<D, 2, 1>(a, s);
  if (a.L <= 128) return launch_cfg<D, 2, 2>(a, s);
  return launch_cfg<D, 4, 2>(a, s);
}

}  // namespace

bool attn_bf16_supports(int D) {
  switch (D) {
    case 16: case 32: case 64: case 72: case 80: case 96: return true;
    default: return false;
  }
}

int launch_attn_bf16(const AttnArgs& a, hipStream_t s) {
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
