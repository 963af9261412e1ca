// Streaming reference kernels: the achievable HBM bandwidth of plain access
// patterns on this GPU, measured next to the codec's kernels so that their
// rates can be read against what the memory system delivers for the same
// mix of reads and writes.  None of this is part of the codec: it moves
// bytes and computes nothing.
//
// Every kernel runs 256 threads per workgroup; a thread moves 16-byte units
// with F = 4, 8 or 16 loads in flight (issued before any of them is used),
// as the codec's row kernels do with their rows.  Stores are non-temporal
// (the codec's policy) unless noted.
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "../../include/skv_ceiling.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kSteps = 16;                          // 16-byte units per thread
constexpr uint64_t kTile = kThreads * kSteps * 16;  // bytes per workgroup: 64 KiB

__device__ __forceinline__ u32x4 ld16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x2 ld8(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
}
template <bool NT>
__device__ __forceinline__ void st16(void* p, u32x4 v) {
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
  else *reinterpret_cast<u32x4*>(p) = v;
}

// Read-only: every 16-byte unit of the workgroup's tile is loaded; the xor of
// everything read is stored only if it equals a value no input here holds,
// which the compiler cannot know, so no load is dropped.
template <int F>
__global__ __launch_bounds__(kThreads) void read_only(const uint8_t* __restrict__ src, uint32_t* __restrict__ sink) {
  const uint8_t* base = src + blockIdx.x * kTile + threadIdx.x * 16;
  u32x4 acc{0u, 0u, 0u, 0u};
#pragma unroll
  for (int s = 0; s < kSteps; s += F) {
    u32x4 x[F];
#pragma unroll
    for (int u = 0; u < F; ++u) x[u] = ld16(base + (s + u) * kThreads * 16);
#pragma unroll
    for (int u = 0; u < F; ++u) acc ^= x[u];
  }
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[blockIdx.x & 1023] = acc.x;
}

template <bool NT>
__global__ __launch_bounds__(kThreads) void write_only(uint8_t* __restrict__ dst) {
  uint8_t* base = dst + blockIdx.x * kTile + threadIdx.x * 16;
  const u32x4 v{blockIdx.x, threadIdx.x, 0x3C003C00u, 0u};
#pragma unroll
  for (int s = 0; s < kSteps; ++s) st16<NT>(base + s * kThreads * 16, v);
}

// Write-only through buffer stores whose cache-policy bits are CPOL (bit 0
// sc0, bit 1 nt, bit 4 sc1: the instruction's own modifiers).  Each
// workgroup's buffer descriptor covers its own 64 KiB tile, so the hardware's
// range check also bounds every store.
template <int CPOL>
__global__ __launch_bounds__(kThreads) void write_cpol(uint8_t* __restrict__ dst) {
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(dst + blockIdx.x * kTile, 0, static_cast<int>(kTile), 0x00020000);
  const u32x4 v{blockIdx.x, threadIdx.x, 0x3C003C00u, 0u};
#pragma unroll
  for (int s = 0; s < kSteps; ++s)
    __builtin_amdgcn_raw_buffer_store_b128(v, r, (s * kThreads + static_cast<int>(threadIdx.x)) * 16, 0, CPOL);
}

// Copy: the tile read and written once.
template <int F>
__global__ __launch_bounds__(kThreads) void copy_1to1(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst) {
  const uint64_t off = blockIdx.x * kTile + threadIdx.x * 16;
#pragma unroll
  for (int s = 0; s < kSteps; s += F) {
    u32x4 x[F];
#pragma unroll
    for (int u = 0; u < F; ++u) x[u] = ld16(src + off + (s + u) * kThreads * 16);
#pragma unroll
    for (int u = 0; u < F; ++u) st16<true>(dst + off + (s + u) * kThreads * 16, x[u]);
  }
}

// Two bytes read per byte written (pack's mix): a 128 KiB read tile, a
// 64 KiB write tile.
template <int F>
__global__ __launch_bounds__(kThreads) void read2_write1(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst) {
  const uint8_t* in = src + 2 * blockIdx.x * kTile + threadIdx.x * 16;
  uint8_t* out = dst + blockIdx.x * kTile + threadIdx.x * 16;
#pragma unroll
  for (int s = 0; s < kSteps; s += F / 2) {
    u32x4 x[F];
#pragma unroll
    for (int u = 0; u < F; ++u) x[u] = ld16(in + (2 * s + u) * kThreads * 16);
#pragma unroll
    for (int u = 0; u < F / 2; ++u) st16<true>(out + (s + u) * kThreads * 16, x[2 * u] ^ x[2 * u + 1]);
  }
}

// One byte read per two written (unpack's mix), contiguous on both sides: a
// thread reads 8 bytes and writes the 16 bytes that follow from them, like an
// INT8 row slice decoded to binary16.  RB = 8: 8-byte reads (a 32 KiB read
// tile per workgroup); RB = 16: 16-byte reads, 32 bytes written per read.
template <int RB, int F>
__global__ __launch_bounds__(kThreads) void read1_write2(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst) {
  if constexpr (RB == 8) {
    const uint8_t* in = src + blockIdx.x * (kTile / 2) + threadIdx.x * 8;
    uint8_t* out = dst + blockIdx.x * kTile + threadIdx.x * 16;
#pragma unroll
    for (int s = 0; s < kSteps; s += F) {
      u32x2 x[F];
#pragma unroll
      for (int u = 0; u < F; ++u) x[u] = ld8(in + (s + u) * kThreads * 8);
#pragma unroll
      for (int u = 0; u < F; ++u) st16<true>(out + (s + u) * kThreads * 16, u32x4{x[u].x, x[u].y, x[u].x, x[u].y});
    }
  } else {
    constexpr int G = F < kSteps / 2 ? F : kSteps / 2;
    const uint8_t* in = src + blockIdx.x * (kTile / 2) + threadIdx.x * 16;
    uint8_t* out = dst + blockIdx.x * kTile + threadIdx.x * 32;
#pragma unroll
    for (int s = 0; s < kSteps / 2; s += G) {
      u32x4 x[G];
#pragma unroll
      for (int u = 0; u < G; ++u) x[u] = ld16(in + (s + u) * kThreads * 16);
#pragma unroll
      for (int u = 0; u < G; ++u) {
        st16<true>(out + (s + u) * kThreads * 32, x[u]);
        st16<true>(out + (s + u) * kThreads * 32 + 16, x[u] ^ u32x4{1u, 1u, 1u, 1u});
      }
    }
  }
}

// One byte read per four written (unpack's mix when most rows are INT4): a
// thread reads 4 bytes and writes 16, both contiguous; default-policy stores
// (the codec's d = 256 unpack), 16 KiB read and 64 KiB written per workgroup.
template <int F>
__global__ __launch_bounds__(kThreads) void read1_write4(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst) {
  const uint8_t* in = src + blockIdx.x * (kTile / 4) + threadIdx.x * 4;
  uint8_t* out = dst + blockIdx.x * kTile + threadIdx.x * 16;
#pragma unroll
  for (int s = 0; s < kSteps; s += F) {
    uint32_t x[F];
#pragma unroll
    for (int u = 0; u < F; ++u) x[u] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(in + (s + u) * kThreads * 4));
#pragma unroll
    for (int u = 0; u < F; ++u) st16<false>(out + (s + u) * kThreads * 16, u32x4{x[u], x[u] ^ 1u, x[u] ^ 2u, x[u] ^ 3u});
  }
}

// Unpack's access pattern without the decode: one workgroup per 256-token
// chunk of one of H = 8 head segments (segment-major workgroup order, as in
// the codec), each token's row of 128 bytes (an INT8 row at d = 128) read
// contiguously by 16 lanes x 8 bytes and written as 256 bytes (16 lanes x
// 16 bytes) into the token's slot of a [token][H][128] binary16 cache, so the
// pieces of one workgroup land 2 KiB apart.
constexpr int kNhdHeads = 8;
constexpr int kNhdRow = 128;  // bytes read per token row
template <int F>
__global__ __launch_bounds__(kThreads) void nhd_scatter(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                        uint32_t tokens) {
  const uint32_t nchunks = tokens / 256;
  const uint32_t h = blockIdx.x / nchunks, chunk = blockIdx.x % nchunks;
  const int lane = threadIdx.x % 16, rsub = threadIdx.x / 16;
  const uint8_t* seg = src + (static_cast<uint64_t>(h) * tokens + chunk * 256) * kNhdRow;
#pragma unroll
  for (int s = 0; s < 16; s += F) {
    u32x2 x[F];
#pragma unroll
    for (int u = 0; u < F; ++u) x[u] = ld8(seg + ((s + u) * 16 + rsub) * kNhdRow + lane * 8);
#pragma unroll
    for (int u = 0; u < F; ++u) {
      const uint64_t t = chunk * 256 + (s + u) * 16 + rsub;
      st16<true>(dst + (t * kNhdHeads + h) * (2 * kNhdRow) + lane * 16, u32x4{x[u].x, x[u].y, x[u].x, x[u].y});
    }
  }
}

// The attention score's key stream: each workgroup reads 256 KiB in 16 KiB
// stages into shared memory, the 256 threads filling a stage as consecutive
// 16-byte pieces (thread i: pieces i, i + 256, i + 512, i + 768), with a
// workgroup barrier per stage.  stage_direct uses gfx950's direct
// global-to-LDS loads with NB stage buffers (NB - 1 stages in flight),
// non-temporal (NT) or with the default cache policy; stage_regs loads RS
// stages ahead into registers (non-temporal) and writes each stage into one
// of two buffers once the previous one is done.  One 32-bit word per
// thread and stage is read back from shared memory, so every stage is used.
constexpr int kStageBytes = 16 << 10, kStreamBytes = 256 << 10, kStagePieces = kStageBytes / (kThreads * 16);
constexpr int kStreamStages = kStreamBytes / kStageBytes;

__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Waits until at most N of this wave's vector memory loads are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
  asm volatile("" ::: "memory");
}

template <int NB, bool NT>
__global__ __launch_bounds__(kThreads) void stage_direct(const uint8_t* __restrict__ src, uint32_t* __restrict__ sink) {
  static_assert(NB >= 2 && NB <= 4, "two to four stage buffers");
  __shared__ __align__(16) uint8_t buf[NB * kStageBytes];
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const uint8_t* blk = src + static_cast<uint64_t>(blockIdx.x) * kStreamBytes;
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)buf));
  auto issue = [&](int st) {
#pragma unroll
    for (int u = 0; u < kStagePieces; ++u) {
      // the wave's 64 lanes land 16 bytes each at consecutive LDS addresses from m0
      const uint32_t m0 = lds + (st % NB) * kStageBytes + (u * kThreads + wave * 64) * 16;
      const uint8_t* p = blk + st * kStageBytes + (u * kThreads + threadIdx.x) * 16;
      if (NT)
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(p), "s"(__builtin_amdgcn_readfirstlane(m0))
                     : "memory", "m0");
      else
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(p), "s"(__builtin_amdgcn_readfirstlane(m0))
                     : "memory", "m0");
    }
  };
  uint32_t acc = 0;
  for (int st = 0; st < NB - 1; ++st) issue(st);
  for (int st = 0; st < kStreamStages; ++st) {
    const int later = min(NB - 2, kStreamStages - 1 - st);  // stages issued after st
    if (later >= 2) wait_vm<2 * kStagePieces>();
    else if (later == 1) wait_vm<kStagePieces>();
    else wait_vm<0>();
    lds_barrier();
    if (st + NB - 1 < kStreamStages) issue(st + NB - 1);
    acc ^= *reinterpret_cast<const uint32_t*>(buf + (st % NB) * kStageBytes + threadIdx.x * 64);
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x & 1023] = acc;
}

template <int RS>
__global__ __launch_bounds__(kThreads) void stage_regs(const uint8_t* __restrict__ src, uint32_t* __restrict__ sink) {
  __shared__ __align__(16) uint8_t buf[2 * kStageBytes];
  const uint8_t* blk = src + static_cast<uint64_t>(blockIdx.x) * kStreamBytes + threadIdx.x * 16;
  u32x4 r[RS][kStagePieces];
#pragma unroll
  for (int a = 0; a < RS; ++a)
#pragma unroll
    for (int u = 0; u < kStagePieces; ++u) r[a][u] = ld16(blk + a * kStageBytes + u * kThreads * 16);
  uint32_t acc = 0;
  for (int st0 = 0; st0 < kStreamStages; st0 += RS) {
#pragma unroll
    for (int a = 0; a < RS; ++a) {
      const int st = st0 + a;
      if (st >= kStreamStages) break;
      // every thread is done reading the buffer this stage overwrites (stage st - 2)
      lds_barrier();
#pragma unroll
      for (int u = 0; u < kStagePieces; ++u)
        *reinterpret_cast<u32x4*>(buf + (st & 1) * kStageBytes + (u * kThreads + threadIdx.x) * 16) = r[a][u];
      if (st + RS < kStreamStages) {
#pragma unroll
        for (int u = 0; u < kStagePieces; ++u) r[a][u] = ld16(blk + (st + RS) * kStageBytes + u * kThreads * 16);
      }
      lds_barrier();
      acc ^= *reinterpret_cast<const uint32_t*>(buf + (st & 1) * kStageBytes + ((threadIdx.x * 67) & 1023) * 16);
    }
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x & 1023] = acc;
}

template <int F>
int run_pattern(int32_t pattern, uint8_t* out, const uint8_t* in, uint64_t bytes, uint64_t tiles, uint32_t* sink,
                hipStream_t stream) {
  switch (pattern) {
    case SKV_CEIL_READ:
      if (sink == nullptr) return 1;
      read_only<F><<<tiles, kThreads, 0, stream>>>(in, sink);
      break;
    case SKV_CEIL_WRITE: write_only<true><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_DEFAULT: write_only<false><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_COPY: copy_1to1<F><<<tiles, kThreads, 0, stream>>>(in, out); break;
    case SKV_CEIL_READ2_WRITE1: read2_write1<F><<<tiles / 2, kThreads, 0, stream>>>(in, out); break;
    case SKV_CEIL_READ1_WRITE2_8B: read1_write2<8, F><<<tiles, kThreads, 0, stream>>>(in, out); break;
    case SKV_CEIL_READ1_WRITE2_16B: read1_write2<16, F><<<tiles, kThreads, 0, stream>>>(in, out); break;
    case SKV_CEIL_READ1_WRITE4: read1_write4<F><<<tiles, kThreads, 0, stream>>>(in, out); break;
    case SKV_CEIL_WRITE_CPOL + 0: write_cpol<0><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 1: write_cpol<1><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 2: write_cpol<2><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 3: write_cpol<3><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 4: write_cpol<16><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 5: write_cpol<17><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 6: write_cpol<18><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_WRITE_CPOL + 7: write_cpol<19><<<tiles, kThreads, 0, stream>>>(out); break;
    case SKV_CEIL_NHD_SCATTER: {
      // bytes written = tokens * 8 heads * 256 B; tokens a multiple of 256
      const uint64_t tokens = bytes / (kNhdHeads * 2 * kNhdRow);
      if (tokens % 256 != 0 || tokens > 0xFFFFFFFFu) return 1;
      nhd_scatter<F><<<(tokens / 256) * kNhdHeads, kThreads, 0, stream>>>(in, out, static_cast<uint32_t>(tokens));
      break;
    }
    case SKV_CEIL_STAGE_DIRECT:
    case SKV_CEIL_STAGE_DIRECT_CACHED:
    case SKV_CEIL_STAGE_REGS: {
      // F = 4, 8, 16: one, two or three stages in flight
      const uint64_t blocks = bytes / kStreamBytes;
      if (sink == nullptr || blocks == 0) return 1;
      constexpr int ahead = F == 4 ? 1 : F == 8 ? 2 : 3;
      if (pattern == SKV_CEIL_STAGE_DIRECT) stage_direct<ahead + 1, true><<<blocks, kThreads, 0, stream>>>(in, sink);
      else if (pattern == SKV_CEIL_STAGE_DIRECT_CACHED)
        stage_direct<ahead + 1, false><<<blocks, kThreads, 0, stream>>>(in, sink);
      else stage_regs<ahead><<<blocks, kThreads, 0, stream>>>(in, sink);
      break;
    }
    default: return 1;
  }
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // namespace

extern "C" {

int skv_ceiling_run(int32_t pattern, int32_t inflight, void* dst, const void* src, uint64_t bytes, void* sink,
                    hipStream_t stream) {
  if (bytes == 0 || bytes % (2 * kTile) != 0 || dst == nullptr) return 1;
  const uint8_t* in = static_cast<const uint8_t*>(src);
  uint8_t* out = static_cast<uint8_t*>(dst);
  const uint64_t tiles = bytes / kTile;
  if (tiles > 0x7FFFFFFFu) return 1;
  const bool reads = pattern != SKV_CEIL_WRITE && pattern != SKV_CEIL_WRITE_DEFAULT &&
                     !(pattern >= SKV_CEIL_WRITE_CPOL && pattern < SKV_CEIL_WRITE_CPOL + 8);
  if ((pattern == SKV_CEIL_STAGE_DIRECT || pattern == SKV_CEIL_STAGE_DIRECT_CACHED || pattern == SKV_CEIL_STAGE_REGS) &&
      bytes / kStreamBytes > 0x7FFFFFFFu)
    return 1;
  if (reads && src == nullptr) return 1;
  uint32_t* sk = static_cast<uint32_t*>(sink);
  switch (inflight) {
    case 4: return run_pattern<4>(pattern, out, in, bytes, tiles, sk, stream);
    case 8: return run_pattern<8>(pattern, out, in, bytes, tiles, sk, stream);
    case 16: return run_pattern<16>(pattern, out, in, bytes, tiles, sk, stream);
    default: return 1;
  }
}

uint64_t skv_ceiling_bytes(int32_t pattern, uint64_t bytes, int32_t which) {
  // which 0: bytes read, 1: bytes written, for a call of skv_ceiling_run
  switch (pattern) {
    case SKV_CEIL_READ: return which == 0 ? bytes : 0;
    case SKV_CEIL_WRITE:
    case SKV_CEIL_WRITE_DEFAULT: return which == 0 ? 0 : bytes;
    case SKV_CEIL_COPY: return bytes;
    case SKV_CEIL_READ2_WRITE1: return which == 0 ? bytes : bytes / 2;
    case SKV_CEIL_READ1_WRITE2_8B:
    case SKV_CEIL_READ1_WRITE2_16B:
    case SKV_CEIL_NHD_SCATTER: return which == 0 ? bytes / 2 : bytes;
    case SKV_CEIL_READ1_WRITE4: return which == 0 ? bytes / 4 : bytes;
    case SKV_CEIL_STAGE_DIRECT:
    case SKV_CEIL_STAGE_DIRECT_CACHED:
    case SKV_CEIL_STAGE_REGS: return which == 0 ? bytes / kStreamBytes * kStreamBytes : 0;
    default:
      if (pattern >= SKV_CEIL_WRITE_CPOL && pattern < SKV_CEIL_WRITE_CPOL + 8) return which == 0 ? 0 : bytes;
      return 0;
  }
}

}  // extern "C"
