// DSP Switch, one GPU's share: permute + pack into per-destination chunks.
//
// The Switch primitive (primitive table, row s_i -> s_j; Eq. 10) reshards a
// sequence tensor from dimension i to dimension j with one all-to-all.  Before
// the exchange each GPU lays its shard out as n_chunks contiguous chunks, chunk
// n holding slice n of the to-dimension with the from-dimension innermost
// (the layout the next stage computes on, Eq. 7).  For [B, D1, D2, C] with
// from=1, to=2:  y[n][b][j'][i][c] = x[b][i][n*D2/N + j'][c].
//
// The operation is a pure data movement: every output row (C elements) is an
// input row.  Two kernels:
//  * rows  -- each thread moves 16-byte vectors of whole rows.  With rows of
//             >= 64 bytes (2304 B for C=1152 bf16) both the reads and the
//             writes are full 128-bit accesses, contiguous within a row, so no
//             staging is needed; loads are batched ahead of stores for memory
//             level parallelism and stores bypass the cache hierarchy's
//             allocation (non-temporal), since the output is not re-read here.
//             Output rows are visited in tiles of 4 from-indices x 16 local
//             to-indices (from-index fastest), so a work-group's reads come in
//             runs of 16 consecutive input rows instead of rows one whole
//             from-plane apart (+2-4% on a 604 MB shard, both directions).
//  * tiles -- for short rows: a (from x to) tile of rows is read with the
//             to-index fastest (contiguous in x), staged in LDS, and written
//             with the from-index fastest (contiguous in y), so both global
//             sides stay coalesced when rows are only a few bytes long.
#include <algorithm>

#include "dsp_internal.h"

namespace dsp {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Unsigned division by a run-time constant for numerators below 2^31:
// q = (umulhi(n, m) + n) >> s with s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1
// (the multiply-shift method of Granlund and Montgomery, 1994).
struct FastDiv {
  uint32_t m, s;
  FastDiv() : m(0), s(0) {}
  explicit FastDiv(uint32_t d) {
    s = 0;
    while ((1ull << s) < d) ++s;
    m = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
  }
  __device__ __forceinline__ uint32_t div(uint32_t n) const { return (__umulhi(n, m) + n) >> s; }
};

// Tuning knobs (compile time): 16-byte vectors per thread, and whether loads
// and stores carry the non-temporal hint.
#ifndef DSP_SWITCH_VPT
#define DSP_SWITCH_VPT 4
#endif
#ifndef DSP_SWITCH_NT_LOAD
#define DSP_SWITCH_NT_LOAD 1
#endif
#ifndef DSP_SWITCH_NT_STORE
#define DSP_SWITCH_NT_STORE 1
#endif
#ifndef DSP_SWITCH_TILE_F
#define DSP_SWITCH_TILE_F 4
#endif
#ifndef DSP_SWITCH_TILE_J
#define DSP_SWITCH_TILE_J 16
#endif
#ifndef DSP_SWITCH_TILED
#define DSP_SWITCH_TILED 1
#endif
#ifndef DSP_SWITCH_THREADS
#define DSP_SWITCH_THREADS 512
#endif

// Row mapping of the switch.  Output rows are enumerated (n, b, jt', if):
// chunk, batch, local to-dim index, from-dim index.  The matching input row
// index is b*D1*D2 + (to==2 ? if*D2 + jt : jt*D2 + if) with jt = n*per + jt'.
struct RowMap {
  FastDiv f_from, f_per, f_B;
  uint32_t per, d_from, B, D2, plane;  // plane = D1*D2
  uint32_t to_is_2;
  // Tiled order (when kTileRows divides both dims): output rows are taken in
  // tiles of kTileF from-indices x kTileJ local to-indices, from-index
  // fastest, so a tile reads kTileF runs of kTileJ consecutive input rows and
  // writes kTileJ runs of kTileF consecutive output rows.
  uint32_t tiled;
  FastDiv f_ft, f_jt;  // tiles along the from-dim, along the local to-dim
  uint32_t n_ft, n_jt;
  static constexpr uint32_t kTileF = DSP_SWITCH_TILE_F, kTileJ = DSP_SWITCH_TILE_J;
  // tile-order index -> (output row, input row)
  __device__ __forceinline__ void rows_tiled(uint32_t ro, uint32_t& dst, uint32_t& src) const {
    const uint32_t tile = ro / (kTileF * kTileJ), k = ro % (kTileF * kTileJ);
    const uint32_t q1 = f_ft.div(tile);
    const uint32_t i_from = (tile - q1 * n_ft) * kTileF + k % kTileF;
    const uint32_t q2 = f_jt.div(q1);
    const uint32_t jl = (q1 - q2 * n_jt) * kTileJ + k / kTileF;
    const uint32_t n = f_B.div(q2);
    const uint32_t b = q2 - n * B;
    const uint32_t jt = n * per + jl;
    dst = (q2 * per + jl) * d_from + i_from;
    src = b * plane + (to_is_2 ? (i_from * D2 + jt) : (jt * D2 + i_from));
  }
  __device__ __forceinline__ uint32_t src_row(uint32_t ro) const {
    uint32_t q1 = f_from.div(ro);
    uint32_t i_from = ro - q1 * d_from;
    uint32_t q2 = f_per.div(q1);
    uint32_t jl = q1 - q2 * per;
    uint32_t n = f_B.div(q2);
    uint32_t b = q2 - n * B;
    uint32_t jt = n * per + jl;
    uint32_t in_plane = to_is_2 ? (i_from * D2 + jt) : (jt * D2 + i_from);
    return b * plane + in_plane;
  }
};

constexpr int kRowThreads = DSP_SWITCH_THREADS;
constexpr int kRowVecPerThread = DSP_SWITCH_VPT;

// Moves 16-byte vectors.  Vector v of the output is (row ro = v / V, column
// c = v % V) and comes from vector src_row(ro) * V + c of the input.
__global__ __launch_bounds__(kRowThreads) void switch_rows_kernel(
    const u32x4* __restrict__ x, u32x4* __restrict__ y, RowMap map, FastDiv f_vec, uint32_t V,
    uint32_t n_vec, uint32_t identity) {
  const uint32_t base = blockIdx.x * (kRowThreads * kRowVecPerThread) + threadIdx.x;
  u32x4 buf[kRowVecPerThread];
  uint32_t dst[kRowVecPerThread];
#pragma unroll
  for (int u = 0; u < kRowVecPerThread; ++u) {
    const uint32_t v = base + u * kRowThreads;
    dst[u] = v;
    if (v < n_vec) {
      uint32_t src = v;
      if (!identity) {
        const uint32_t ro = f_vec.div(v);
        const uint32_t c = v - ro * V;
        if (map.tiled) {
          uint32_t d, r;
          map.rows_tiled(ro, d, r);
          dst[u] = d * V + c;
          src = r * V + c;
        } else {
          src = map.src_row(ro) * V + c;
        }
      }
      if (DSP_SWITCH_NT_LOAD) buf[u] = __builtin_nontemporal_load(x + src);
      else buf[u] = x[src];
    }
  }
#pragma unroll
  for (int u = 0; u < kRowVecPerThread; ++u) {
    if (dst[u] < n_vec) {
      if (DSP_SWITCH_NT_STORE) __builtin_nontemporal_store(buf[u], y + dst[u]);
      else y[dst[u]] = buf[u];
    }
  }
}

// Tile kernel: a tile of kTileF from-indices x kTileT to-indices of one (b),
// each entry a row of `row_units` units of `Unit` (2 or 4 bytes).  Input rows
// (b, i, j) for fixed i are contiguous along j when to==2; output rows are
// contiguous along i.  Staged through LDS so both sides are read/written with
// consecutive threads on consecutive addresses.
constexpr int kTileF = 32;
constexpr int kTileT = 32;
constexpr int kTileThreads = 256;
constexpr int kTileLdsBytes = 32 * 1024;

template <typename Unit>
__global__ __launch_bounds__(kTileThreads) void switch_tiles_kernel(
    const Unit* __restrict__ x, Unit* __restrict__ y, uint32_t B, uint32_t D1, uint32_t D2,
    uint32_t row_units, uint32_t per, uint32_t to_is_2, uint32_t tf, uint32_t tt) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  Unit* lds = reinterpret_cast<Unit*>(lds_raw);
  const uint32_t d_from = to_is_2 ? D1 : D2;
  const uint32_t d_to = to_is_2 ? D2 : D1;
  // blockIdx.x -> (b, from tile, to tile)
  const uint32_t n_ft = (d_from + tf - 1) / tf;
  const uint32_t n_tt = (d_to + tt - 1) / tt;
  uint32_t blk = blockIdx.x;
  const uint32_t t_tile = blk % n_tt;
  blk /= n_tt;
  const uint32_t f_tile = blk % n_ft;
  const uint32_t b = blk / n_ft;
  const uint32_t f0 = f_tile * tf, t0 = t_tile * tt;
  const uint32_t nf = min(tf, d_from - f0), nt = min(tt, d_to - t0);
  const uint32_t plane = D1 * D2;
  // load: entries ordered (f, t, unit), t fastest among rows -> contiguous in x when to==2
  const uint32_t tile_units = nf * nt * row_units;
  for (uint32_t e = threadIdx.x; e < tile_units; e += kTileThreads) {
    const uint32_t u = e % row_units;
    const uint32_t r = e / row_units;
    const uint32_t tl = r % nt, fl = r / nt;
    const uint32_t i_from = f0 + fl, jt = t0 + tl;
    const uint32_t in_row = b * plane + (to_is_2 ? (i_from * D2 + jt) : (jt * D2 + i_from));
    lds[(tl * tf + fl) * row_units + u] = x[(size_t)in_row * row_units + u];
  }
  __syncthreads();
  // store: entries ordered (t, f, unit), f fastest -> contiguous in y
  for (uint32_t e = threadIdx.x; e < tile_units; e += kTileThreads) {
    const uint32_t u = e % row_units;
    const uint32_t r = e / row_units;
    const uint32_t fl = r % nf, tl = r / nf;
    const uint32_t jt = t0 + tl;
    const uint32_t n = jt / per, jl = jt - n * per;
    const uint32_t out_row = ((n * B + b) * per + jl) * d_from + (f0 + fl);
    y[(size_t)out_row * row_units + u] = lds[(tl * tf + fl) * row_units + u];
  }
}

}  // namespace

int launch_switch_rows(const void* x, void* y, int64_t B, int64_t D1, int64_t D2, int64_t row_bytes,
                       int from_dim, int to_dim, int64_t n_chunks, hipStream_t s) {
  const int64_t rows = B * D1 * D2;
  const int64_t V = row_bytes / 16;
  const int64_t n_vec = rows * V;
  if (n_vec == 0) return DSP_OK;
  if (n_vec >= (int64_t(1) << 31) || rows >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  RowMap map;
  const bool identity = from_dim == to_dim;
  const int64_t d_to = to_dim == 2 ? D2 : D1;
  const int64_t d_from = to_dim == 2 ? D1 : D2;
  map.per = (uint32_t)(identity ? 1 : d_to / n_chunks);
  map.d_from = (uint32_t)d_from;
  map.B = (uint32_t)B;
  map.D2 = (uint32_t)D2;
  map.plane = (uint32_t)(D1 * D2);
  map.to_is_2 = to_dim == 2;
  map.f_from = FastDiv(map.d_from);
  map.f_per = FastDiv(map.per);
  map.f_B = FastDiv(map.B);
  map.tiled = DSP_SWITCH_TILED && !identity && map.per % RowMap::kTileJ == 0 && map.d_from % RowMap::kTileF == 0;
  map.n_ft = map.d_from / RowMap::kTileF;
  map.n_jt = std::max<uint32_t>(1, map.per / RowMap::kTileJ);
  map.f_ft = FastDiv(std::max<uint32_t>(1, map.n_ft));
  map.f_jt = FastDiv(map.n_jt);
  const uint32_t per_block = kRowThreads * kRowVecPerThread;
  const uint32_t blocks = (uint32_t)((n_vec + per_block - 1) / per_block);
  hipLaunchKernelGGL(switch_rows_kernel, dim3(blocks), dim3(kRowThreads), 0, s,
                     static_cast<const u32x4*>(x), static_cast<u32x4*>(y), map,
                     FastDiv((uint32_t)V), (uint32_t)V, (uint32_t)n_vec, identity ? 1u : 0u);
  return last_launch_status();
}

int launch_switch_tiles(const void* x, void* y, int64_t B, int64_t D1, int64_t D2, int64_t C,
                        int elem_bytes, int from_dim, int to_dim, int64_t n_chunks, hipStream_t s) {
  const int64_t rows = B * D1 * D2;
  if (rows == 0) return DSP_OK;
  // from == to is a copy: treat it as a tile pass with a single chunk over a
  // layout whose from-dim is dim 2 and to-dim dim 1 (no transpose).
  int to = to_dim, from = from_dim;
  int64_t nc = n_chunks;
  if (from == to) { from = 2; to = 1; nc = 1; }
  // rows as units of 4 bytes when possible, else 2 bytes
  const int64_t row_bytes = C * elem_bytes;
  const bool u4 = (row_bytes % 4) == 0 && ((uintptr_t)x % 4) == 0 && ((uintptr_t)y % 4) == 0;
  const int unit = u4 ? 4 : 2;
  const int64_t row_units = row_bytes / unit;
  if (rows * row_units >= (int64_t(1) << 32)) return DSP_ERR_SHAPE;
  // tile sizes: keep kTileF*kTileT rows unless rows are long, then shrink
  int64_t tf = kTileF, tt = kTileT;
  while (tf * tt * row_bytes > kTileLdsBytes && (tf > 1 || tt > 1)) {
    if (tt >= tf) tt = (tt + 1) / 2; else tf = (tf + 1) / 2;
  }
  if (tf * tt * row_bytes > kTileLdsBytes) return DSP_ERR_SHAPE;  // a single row exceeds the tile
  const int64_t d_to = to == 2 ? D2 : D1;
  const int64_t d_from = to == 2 ? D1 : D2;
  const int64_t per = d_to / nc;
  const int64_t blocks = B * ((d_from + tf - 1) / tf) * ((d_to + tt - 1) / tt);
  if (blocks >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  const size_t lds = (size_t)(tf * tt * row_bytes);
  if (u4) {
    hipLaunchKernelGGL(switch_tiles_kernel<uint32_t>, dim3((uint32_t)blocks), dim3(kTileThreads),
                       lds, s, static_cast<const uint32_t*>(x), static_cast<uint32_t*>(y),
                       (uint32_t)B, (uint32_t)D1, (uint32_t)D2, (uint32_t)row_units, (uint32_t)per,
                       to == 2 ? 1u : 0u, (uint32_t)tf, (uint32_t)tt);
  } else {
    hipLaunchKernelGGL(switch_tiles_kernel<uint16_t>, dim3((uint32_t)blocks), dim3(kTileThreads),
                       lds, s, static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y),
                       (uint32_t)B, (uint32_t)D1, (uint32_t)D2, (uint32_t)row_units, (uint32_t)per,
                       to == 2 ? 1u : 0u, (uint32_t)tf, (uint32_t)tt);
  }
  return last_launch_status();
}

}  // namespace dsp
