// The exchange step of the Switch primitive among N ranks, run on one GPU with
// one buffer per rank, fused with the receivers' unpack.
//
// In the primitive table's row s_i -> s_j every rank m splits its shard into N
// chunks (dsp_switch writes them contiguously) and sends chunk n to rank n;
// rank n then holds the to-dimension slice n of the whole tensor once it
// places the chunk received from rank m at from-dimension offset m * F (the
// from-dimension is what was sharded before the switch).  With packed[m] of
// shape [N][B][P][F][C]:
//     out[n][b][p][m*F + f][c] = packed[m][n][b][p][f][c].
// On one GPU the "send" is the read of another rank's buffer.  Every
// (n, m, b, p) is a contiguous run of F*C elements on both sides, so the
// kernel is a row copy: one work-group per run, 16-byte vectors when the run
// length and all pointers allow it (non-temporal: nothing is re-read here),
// narrower units otherwise.
#include "dsp_internal.h"

namespace dsp {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kExThreads = 256;
constexpr int kExUnroll = 4;

struct RankPtrs {
  const unsigned char* src[kMaxExchangeRanks];
  unsigned char* dst[kMaxExchangeRanks];
};

// Work-group r copies run (n, m, b, p), enumerated in destination order (m
// fastest, then p, b, n) so that consecutive work-groups write consecutive
// memory of one destination buffer.
template <typename Unit>
__global__ __launch_bounds__(kExThreads) void exchange_unpack_kernel(RankPtrs ptr, uint32_t N,
                                                                     uint32_t B, uint32_t P,
                                                                     uint64_t run_units) {
  uint32_t r = blockIdx.x;
  const uint32_t m = r % N;
  r /= N;
  const uint32_t p = r % P;
  r /= P;
  const uint32_t b = r % B;
  const uint32_t n = r / B;
  const Unit* src = reinterpret_cast<const Unit*>(ptr.src[m]) +
                    (((uint64_t)n * B + b) * P + p) * run_units;
  Unit* dst = reinterpret_cast<Unit*>(ptr.dst[n]) + (((uint64_t)b * P + p) * N + m) * run_units;
  for (uint64_t base = threadIdx.x; base < run_units; base += kExThreads * kExUnroll) {
    Unit v[kExUnroll];
#pragma unroll
    for (int u = 0; u < kExUnroll; ++u) {
      const uint64_t i = base + (uint64_t)u * kExThreads;
      if (i < run_units) v[u] = __builtin_nontemporal_load(src + i);
    }
#pragma unroll
    for (int u = 0; u < kExUnroll; ++u) {
      const uint64_t i = base + (uint64_t)u * kExThreads;
      if (i < run_units) __builtin_nontemporal_store(v[u], dst + i);
    }
  }
}

template <typename Unit>
int launch_unit(const RankPtrs& ptr, uint32_t N, uint32_t B, uint32_t P, uint64_t run_bytes,
                uint64_t runs, hipStream_t s) {
  hipLaunchKernelGGL(exchange_unpack_kernel<Unit>, dim3((uint32_t)runs), dim3(kExThreads), 0, s, ptr,
                     N, B, P, (uint64_t)(run_bytes / sizeof(Unit)));
  return last_launch_status();
}

}  // namespace

int launch_exchange_unpack(const void* const* packed, void* const* out, int64_t N, int64_t B,
                           int64_t P, int64_t run_bytes, hipStream_t s) {
  const int64_t runs = N * N * B * P;
  if (runs == 0 || run_bytes == 0) return DSP_OK;
  if (runs >= (int64_t(1) << 31)) return DSP_ERR_SHAPE;
  RankPtrs ptr = {};
  uintptr_t align = (uintptr_t)run_bytes;
  for (int64_t i = 0; i < N; ++i) {
    ptr.src[i] = static_cast<const unsigned char*>(packed[i]);
    ptr.dst[i] = static_cast<unsigned char*>(out[i]);
    align |= (uintptr_t)packed[i] | (uintptr_t)out[i];
  }
  // widest unit that divides the run length and every buffer address
  if (align % 16 == 0) return launch_unit<u32x4>(ptr, (uint32_t)N, (uint32_t)B, (uint32_t)P, run_bytes, runs, s);
  if (align % 4 == 0) return launch_unit<uint32_t>(ptr, (uint32_t)N, (uint32_t)B, (uint32_t)P, run_bytes, runs, s);
  if (align % 2 == 0) return launch_unit<uint16_t>(ptr, (uint32_t)N, (uint32_t)B, (uint32_t)P, run_bytes, runs, s);
  return launch_unit<uint8_t>(ptr, (uint32_t)N, (uint32_t)B, (uint32_t)P, run_bytes, runs, s);
}

}  // namespace dsp
