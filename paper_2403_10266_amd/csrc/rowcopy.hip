// Strided row copy: the data movement behind the Switch for K = 3 sequence
// dimensions and the table's Split and Gather rows (primitive table; Eq. 7).
//
// Every one of these operations moves whole rows of C elements: the output is
// an index space of up to kMaxCopyDims dimensions, and the row at multi-index
// (i_0, .., i_{nd-1}) is copied from source row sum(i_d * src_stride[d]) to
// destination row sum(i_d * dst_stride[d]).  Several (source, destination)
// buffer pairs share one index space (the N shards of a Gather); blockIdx.y
// picks the pair, so the pointers are uniform per work-group.
//
// The host first simplifies the index space: unit dimensions are dropped,
// neighbours that are contiguous on both sides are merged, and an innermost
// dimension that is contiguous on both sides is folded into the row itself, so
// that a Split along an outer dimension, for instance, becomes a few long
// contiguous runs.  Each thread then moves kCopyUnroll units (16 bytes when the
// row length and every pointer allow it), all loads issued before the stores,
// non-temporal on both sides: nothing is re-read by this kernel.
#include "dsp_internal.h"

namespace dsp {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 4;

// q = floor(n / d) for n < 2^31 by multiply and shift (Granlund and
// Montgomery, 1994): s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1.
struct Div32 {
  uint32_t m, s;
  Div32() : m(0), s(0) {}
  explicit Div32(uint32_t d) {
    s = 0;
    while ((1ull << s) < d) ++s;
    m = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
  }
  __device__ __forceinline__ uint32_t div(uint32_t n) const { return (__umulhi(n, m) + n) >> s; }
};

struct CopyArgs {
  const unsigned char* src[kMaxCopyPairs];
  unsigned char* dst[kMaxCopyPairs];
  uint32_t size[kMaxCopyDims];
  Div32 fdiv[kMaxCopyDims];
  uint32_t sst[kMaxCopyDims];   // source row strides
  uint32_t dstr[kMaxCopyDims];  // destination row strides
  Div32 fV;
  uint32_t V;                   // units per row
  uint32_t total;               // units per pair
  int nd;
};

template <typename Unit>
__global__ __launch_bounds__(kCopyThreads) void rowcopy_kernel(CopyArgs a) {
  const Unit* __restrict__ src = reinterpret_cast<const Unit*>(a.src[blockIdx.y]);
  Unit* __restrict__ dst = reinterpret_cast<Unit*>(a.dst[blockIdx.y]);
  const uint32_t base = blockIdx.x * (kCopyThreads * kCopyUnroll) + threadIdx.x;
  Unit buf[kCopyUnroll];
  uint32_t doff[kCopyUnroll];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u) {
    const uint32_t v = base + u * kCopyThreads;
    doff[u] = 0xFFFFFFFFu;
    if (v < a.total) {
      const uint32_t row = a.fV.div(v);
      const uint32_t c = v - row * a.V;
      uint32_t q = row, so = 0, dso = 0;
#pragma unroll
      for (int d = kMaxCopyDims - 1; d >= 0; --d) {
        if (d < a.nd) {
          const uint32_t qn = a.fdiv[d].div(q);
          const uint32_t i = q - qn * a.size[d];
          q = qn;
          so += i * a.sst[d];
          dso += i * a.dstr[d];
        }
      }
      buf[u] = __builtin_nontemporal_load(src + (uint64_t)so * a.V + c);
      doff[u] = dso * a.V + c;
    }
  }
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u)
    if (doff[u] != 0xFFFFFFFFu) __builtin_nontemporal_store(buf[u], dst + doff[u]);
}

template <typename Unit>
int launch_unit(const CopyArgs& a, int n_pairs, hipStream_t s) {
  const uint32_t per_block = kCopyThreads * kCopyUnroll;
  const dim3 grid((a.total + per_block - 1) / per_block, (uint32_t)n_pairs);
  hipLaunchKernelGGL(rowcopy_kernel<Unit>, grid, dim3(kCopyThreads), 0, s, a);
  return last_launch_status();
}

}  // namespace

int launch_rowcopy(const void* const* src, void* const* dst, int n_pairs, const RowCopyDesc& desc,
                   hipStream_t s) {
  if (n_pairs < 1 || n_pairs > kMaxCopyPairs || desc.nd < 0 || desc.nd > kMaxCopyDims)
    return DSP_ERR_ARG;
  // simplify: drop unit dims, merge neighbours contiguous on both sides
  int64_t size[kMaxCopyDims], sst[kMaxCopyDims], dsst[kMaxCopyDims];
  int nd = 0;
  for (int d = 0; d < desc.nd; ++d) {
    if (desc.size[d] == 0) return DSP_OK;
    if (desc.size[d] == 1) continue;
    if (nd > 0 && sst[nd - 1] == desc.size[d] * desc.src_stride[d] &&
        dsst[nd - 1] == desc.size[d] * desc.dst_stride[d]) {
      size[nd - 1] *= desc.size[d];
      sst[nd - 1] = desc.src_stride[d];
      dsst[nd - 1] = desc.dst_stride[d];
      continue;
    }
    size[nd] = desc.size[d];
    sst[nd] = desc.src_stride[d];
    dsst[nd] = desc.dst_stride[d];
    ++nd;
  }
  int64_t row_bytes = desc.row_bytes;
  if (row_bytes == 0) return DSP_OK;
  // an innermost dimension contiguous on both sides becomes part of the row
  // (when every other stride is a whole number of such longer rows)
  if (nd > 0 && sst[nd - 1] == 1 && dsst[nd - 1] == 1) {
    const int64_t z = size[nd - 1];
    bool whole = true;
    for (int d = 0; d + 1 < nd; ++d) whole = whole && sst[d] % z == 0 && dsst[d] % z == 0;
    if (whole) {
      row_bytes *= z;
      --nd;
      for (int d = 0; d < nd; ++d) {
        sst[d] /= z;
        dsst[d] /= z;
      }
    }
  }
  // widest unit dividing the row and every buffer address
  uintptr_t align = (uintptr_t)row_bytes;
  for (int p = 0; p < n_pairs; ++p) align |= (uintptr_t)src[p] | (uintptr_t)dst[p];
  const int unit = align % 16 == 0 ? 16 : align % 4 == 0 ? 4 : align % 2 == 0 ? 2 : 1;
  const int64_t V = row_bytes / unit;
  // 32-bit index arithmetic: units per pair below 2^31, row offsets below 2^32 / V
  int64_t rows = 1, src_max = 0, dst_max = 0;
  for (int d = 0; d < nd; ++d) {
    rows *= size[d];
    src_max += (size[d] - 1) * sst[d];
    dst_max += (size[d] - 1) * dsst[d];
  }
  if (rows >= (int64_t(1) << 31) / V || (src_max + 1) >= (int64_t(1) << 32) / V ||
      (dst_max + 1) >= (int64_t(1) << 32) / V)
    return DSP_ERR_SHAPE;
  CopyArgs a = {};
  for (int p = 0; p < n_pairs; ++p) {
    a.src[p] = static_cast<const unsigned char*>(src[p]);
    a.dst[p] = static_cast<unsigned char*>(dst[p]);
  }
  for (int d = 0; d < nd; ++d) {
    a.size[d] = (uint32_t)size[d];
    a.fdiv[d] = Div32((uint32_t)size[d]);
    a.sst[d] = (uint32_t)sst[d];
    a.dstr[d] = (uint32_t)dsst[d];
  }
  a.nd = nd;
  a.V = (uint32_t)V;
  a.fV = Div32((uint32_t)V);
  a.total = (uint32_t)(rows * V);
  switch (unit) {
    case 16: return launch_unit<u32x4>(a, n_pairs, s);
    case 4: return launch_unit<uint32_t>(a, n_pairs, s);
    case 2: return launch_unit<uint16_t>(a, n_pairs, s);
    default: return launch_unit<uint8_t>(a, n_pairs, s);
  }
}

}  // namespace dsp
