// Device-to-device copy of the link emulation (the payload crossing from the
// prefill to the decode side, Sec. 4.2, on one GPU): 16-byte units with
// non-temporal loads and stores, sixteen units in flight per thread, so that
// the copy streams like the codec's own kernels instead of going through the
// runtime's generic copy.
#include "device_util.h"
#include "skv_internal.h"

namespace skv {
namespace {

constexpr int kCopyThreads = 256;
constexpr int kCopyUnits = 16;  // 16-byte units per thread

// grid: ceil(units / (kCopyThreads * kCopyUnits)); unit i of a workgroup's
// range is handled by thread i % kCopyThreads, units past the end by nobody
__global__ __launch_bounds__(kCopyThreads) void link_copy(uint8_t* __restrict__ dst, const uint8_t* __restrict__ src,
                                                          uint64_t units) {
  const uint64_t base = static_cast<uint64_t>(blockIdx.x) * (kCopyThreads * kCopyUnits) + threadIdx.x;
  u32x4 x[kCopyUnits];
#pragma unroll
  for (int u = 0; u < kCopyUnits; ++u) {
    const uint64_t i = base + static_cast<uint64_t>(u) * kCopyThreads;
    x[u] = u32x4{0u, 0u, 0u, 0u};
    if (i < units) x[u] = ld_nt16(src + 16 * i);
  }
#pragma unroll
  for (int u = 0; u < kCopyUnits; ++u) {
    const uint64_t i = base + static_cast<uint64_t>(u) * kCopyThreads;
    if (i < units) st_nt16(dst + 16 * i, x[u]);
  }
}

}  // namespace

hipError_t launch_link_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream) {
  const uint64_t units = bytes / 16;
  const uint64_t per = static_cast<uint64_t>(kCopyThreads) * kCopyUnits;
  const uint64_t blocks = (units + per - 1) / per;
  if (bytes % 16 != 0 || blocks > 0x7FFFFFFFull) return hipErrorInvalidValue;
  if (blocks == 0) return hipSuccess;
  link_copy<<<static_cast<uint32_t>(blocks), kCopyThreads, 0, stream>>>(static_cast<uint8_t*>(dst),
                                                                        static_cast<const uint8_t*>(src), units);
  return hipGetLastError();
}

}  // namespace skv
