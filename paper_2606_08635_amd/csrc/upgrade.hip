// Cold-tier precision upgrade (Sec. 4.2 and Fig. "sysarch": an on-demand fetch
// that upgrades tokens the decoder already holds at low precision; Sec. 8,
// "cold-tier fetch design").
//
// The prefill side, which still has the fp16 K/V and the tier map, packs for
// a list of tokens either their fp16 rows (FP16 mode: exact, 2 bytes per
// element) or the INT8 residual between each fp16 row and the row the
// decoder reconstructed (RESIDUAL8 mode: 1 byte per element plus a scale per
// row; the decoder's error drops to half a residual step).  The decoder
// applies the upgrade in place in its paged cache.
//   upg_prep   (one workgroup)  checks the token list, writes header, token
//                               list, tiers and padding;
//   upg_rows   (one workgroup per 256 listed tokens of one (layer, K/V, head))
//                               gathers the rows, recomputes the held row with
//                               the pack quantizer, quantizes the residual;
//   upg_check  (one workgroup)  checks an upgrade payload against the
//                               configuration and the block table;
//   upg_apply  (one workgroup per 256 listed tokens of one segment) adds the
//                               residual to (or overwrites) the cached rows.
#include <type_traits>

#include "device_util.h"
#include "row_codec.h"
#include "skv_internal.h"

namespace skv {
namespace {

#ifndef SKV_UPG_ROWS_IN_FLIGHT
#define SKV_UPG_ROWS_IN_FLIGHT 4  // listed rows whose loads a thread issues before it processes any
#endif

constexpr int kUpgThreads = 256;  // listed tokens per row workgroup
constexpr int kUpgCheckThreads = 1024;
constexpr uint32_t kUpgMagic = 0x55564B53u;  // "SKVU"
constexpr int kUpgHdrStatus = 18;

struct UpgArgs {
  const uint16_t* k;
  const uint16_t* v;
  const uint8_t* tier;
  const int32_t* tokens;  // pack: the caller's list
  uint8_t* up;            // the upgrade payload
  uint32_t* status;
  uint16_t* k_cache;
  uint16_t* v_cache;
  const int32_t* block_table;
  int32_t num_blocks, block_size;
  int32_t L, H, d, n, m, mode;
  uint64_t tokens_off, tiers_off, scales_off, data_off, total, row_bytes;
};

__device__ __forceinline__ uint32_t upg_header_word(const UpgArgs& a, int i) {
  switch (i) {
    case 0: return kUpgMagic;
    case 1: return 1u;
    case 2: return static_cast<uint32_t>(a.L);
    case 3: return static_cast<uint32_t>(a.H);
    case 4: return static_cast<uint32_t>(a.d);
    case 5: return static_cast<uint32_t>(a.n);
    case 6: return static_cast<uint32_t>(a.m);
    case 7: return static_cast<uint32_t>(a.mode);
    case 8: return static_cast<uint32_t>(a.tokens_off);
    case 9: return static_cast<uint32_t>(a.tokens_off >> 32);
    case 10: return static_cast<uint32_t>(a.tiers_off);
    case 11: return static_cast<uint32_t>(a.tiers_off >> 32);
    case 12: return static_cast<uint32_t>(a.scales_off);
    case 13: return static_cast<uint32_t>(a.scales_off >> 32);
    case 14: return static_cast<uint32_t>(a.data_off);
    case 15: return static_cast<uint32_t>(a.data_off >> 32);
    case 16: return static_cast<uint32_t>(a.total);
    case 17: return static_cast<uint32_t>(a.total >> 32);
    default: return 0u;  // 18: status
  }
}

// The token list check shared by upg_prep and upg_check: every token in
// [0, n), strictly ascending, and (tier != null) its tier at most 3.  Loads are
// issued kListBatch at a time so the single workgroup keeps many in flight.
constexpr int kListBatch = 8;

__device__ __forceinline__ bool token_list_bad(const int32_t* tok, int m, int n, const uint8_t* tier_of_token,
                                               const uint8_t* tier_of_entry) {
  bool bad = false;
  for (int base = threadIdx.x; base < m; base += kListBatch * kUpgCheckThreads) {
    int t[kListBatch], prev[kListBatch];
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) {
      const int i = base + u * kUpgCheckThreads;
      t[u] = i < m ? tok[i] : 0;
      prev[u] = (i > 0 && i < m) ? tok[i - 1] : -1;
    }
    uint32_t tr[kListBatch];
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) {
      const int i = base + u * kUpgCheckThreads;
      const bool in = t[u] >= 0 && t[u] < n;
      bad |= !in || prev[u] >= t[u];
      tr[u] = 0;
      if (i < m && tier_of_token != nullptr && in) tr[u] = tier_of_token[t[u]];
      if (i < m && tier_of_entry != nullptr) tr[u] = tier_of_entry[i];
    }
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) bad |= tr[u] > 3u;
  }
  return bad;
}

__global__ __launch_bounds__(kUpgCheckThreads) void upg_prep(const UpgArgs a) {
  __shared__ uint32_t s_bad;
  const int tid = threadIdx.x;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  if (token_list_bad(a.tokens, a.m, a.n, a.tier, nullptr)) atomicOr(&s_bad, 1u);
  __syncthreads();
  const uint32_t status = s_bad ? static_cast<uint32_t>(SKV_ERR_INVALID_ARG) : 0u;
  uint8_t* up = a.up;
  if (tid < 64) reinterpret_cast<uint32_t*>(up)[tid] = tid == kUpgHdrStatus ? status : upg_header_word(a, tid);
  if (tid == 0 && a.status) *a.status = status;
  if (status) return;  // block-uniform
  int32_t* out_tok = reinterpret_cast<int32_t*>(up + a.tokens_off);
  uint8_t* out_tier = up + a.tiers_off;
  for (int base = tid; base < a.m; base += kListBatch * kUpgCheckThreads) {
    int t[kListBatch];
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) {
      const int i = base + u * kUpgCheckThreads;
      t[u] = i < a.m ? a.tokens[i] : 0;
    }
    uint8_t tr[kListBatch];
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) tr[u] = a.tier[t[u]];  // t in range: checked above
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) {
      const int i = base + u * kUpgCheckThreads;
      if (i < a.m) {
        out_tok[i] = t[u];
        out_tier[i] = tr[u];
      }
    }
  }
  for (uint64_t b = a.tokens_off + 4ull * a.m + tid; b < a.tiers_off; b += kUpgCheckThreads) up[b] = 0;
  for (uint64_t b = a.tiers_off + static_cast<uint64_t>(a.m) + tid; b < a.scales_off; b += kUpgCheckThreads) up[b] = 0;
  const uint64_t scales_end = a.scales_off + (a.mode == 1 ? 8ull * a.L * a.H * a.m : 0ull);
  for (uint64_t b = scales_end + tid; b < a.data_off; b += kUpgCheckThreads) up[b] = 0;
}

// INT8 codes of the lane's 8 residuals e (fp32) for a row whose largest
// |e| pattern is emax (bits & 0x7FFFFFFF, reduced over the row).
__device__ __forceinline__ u32x2 quantize_residual(const float (&e)[8], uint32_t emax, float* scale) {
  LaneCodes q;
  if (emax >= 0x7F800000u) {
    *scale = __builtin_bit_cast(float, 0x7FC00000u);
  } else if (emax == 0u) {
    *scale = 0.0f;
  } else {
    // RN32(a/127) and RN32(127/a) for the binary32 residual maximum a without
    // a division, and no clamp: both sequences are correctly rounded and
    // RN32(a RN32(127/a)) < 127.5 for every binary32 a (checked
    // exhaustively), so |e| <= a never codes beyond +-127
    const float amag = __builtin_bit_cast(float, emax);
    *scale = scale_of(amag, 127.0f, 1.0f / 127.0f);
    const float rcp = recip_scale_of_f32(amag, 127.0f);
#pragma unroll
    for (int i = 0; i < 8; ++i) q.c[i] = __builtin_bit_cast(uint32_t, e[i] * rcp + 12582912.0f);
    return pack_int8(q);
  }
  return u32x2{0u, 0u};
}

// The upgrade row of one lane: mode 0 the fp16 values themselves; mode 1 the
// INT8 residual codes against the held row (all lanes of a row take part in
// the two row reductions).
template <int LPR>
__device__ __forceinline__ u32x2 residual_lane(int tr, u32x4 x, float* scale) {
  const uint32_t amax = group_max<LPR>(absmax_bits8(x));
  const u32x4 held = held_lane(tr, x, amax);
  const uint32_t xs[4] = {x.x, x.y, x.z, x.w}, hs[4] = {held.x, held.y, held.z, held.w};
  float e[8];
  uint32_t emax = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    e[2 * j] = half_lo(xs[j]) - half_lo(hs[j]);
    e[2 * j + 1] = half_hi(xs[j]) - half_hi(hs[j]);
    emax = max(emax, __builtin_bit_cast(uint32_t, e[2 * j]) & 0x7FFFFFFFu);
    emax = max(emax, __builtin_bit_cast(uint32_t, e[2 * j + 1]) & 0x7FFFFFFFu);
  }
  emax = group_max<LPR>(emax);
  return quantize_residual(e, emax, scale);
}

// grid: ceil(m / 256) * 2 * L * H workgroups, chunk fastest
template <int D, int MODE>
__global__ __launch_bounds__(kUpgThreads) void upg_rows(const UpgArgs a) {
  constexpr int LPR = D / 8;                 // lanes per row, 16 bytes each
  constexpr int RPI = kUpgThreads / LPR;     // rows per block-wide iteration
  constexpr int ITERS = kUpgThreads / RPI;
  constexpr int U = ITERS < SKV_UPG_ROWS_IN_FLIGHT ? ITERS : SKV_UPG_ROWS_IN_FLIGHT;  // rows in flight per thread
  static_assert(ITERS % U == 0, "rows in flight must divide a thread's rows of the chunk");
  __shared__ int32_t s_tok[kUpgThreads];
  __shared__ uint8_t s_tier[kUpgThreads];
  uint8_t* up = a.up;
  const int nch = (a.m + kUpgThreads - 1) / kUpgThreads;
  const int chunk = blockIdx.x % nch, seg = blockIdx.x / nch;
  const int h = seg % a.H, kv = (seg / a.H) & 1, l = seg / (2 * a.H);
  const int i0 = chunk * kUpgThreads;
  const uint16_t* src = (kv ? a.v : a.k) + (static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(a.n) * D;
  const int lane = threadIdx.x % LPR, rsub = threadIdx.x / LPR;
  // The thread's first rows are loaded before the header check, the tier
  // gather and the barrier, with their token ids read straight from the list
  // and clamped into [0, n): the reads stay inside K/V even for a list the
  // check refuses (then nothing is written), and the clamp changes nothing
  // for a valid list.
  u32x4 first[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int i = i0 + u * RPI + rsub;
    first[u] = u32x4{0u, 0u, 0u, 0u};
    if (i < a.m) {
      const int t = min(max(a.tokens[i], 0), a.n - 1);
      first[u] = ld_nt16(src + static_cast<size_t>(t) * D + lane * 8);
    }
  }
  if (reinterpret_cast<const uint32_t*>(up)[kUpgHdrStatus] != 0u) return;
  {
    const int i = i0 + threadIdx.x;
    const int t = i < a.m ? a.tokens[i] : 0;
    s_tok[threadIdx.x] = t;
    s_tier[threadIdx.x] = i < a.m ? a.tier[t] : kDROP;
  }
  __syncthreads();
  const uint64_t seg_rows = static_cast<uint64_t>(seg) * a.m;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      if (it == 0) x[u] = first[u];
      else x[u] = i0 + r < a.m ? ld_nt16(src + static_cast<size_t>(s_tok[r]) * D + lane * 8) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int i = i0 + r;
      if constexpr (MODE == 0) {
        if (i < a.m) st_nt16(up + a.data_off + (seg_rows + i) * (2 * D) + lane * 16, x[u]);
      } else {
        float scale;
        const u32x2 codes = residual_lane<LPR>(s_tier[r], x[u], &scale);
        if (i < a.m) {
          st_nt8(up + a.data_off + (seg_rows + i) * D + lane * 8, codes);
          if (lane == 0) reinterpret_cast<float*>(up + a.scales_off)[seg_rows + i] = scale;
        }
      }
    }
  }
}

__global__ __launch_bounds__(kUpgCheckThreads) void upg_check(const UpgArgs a) {
  __shared__ uint32_t s_bad;
  const int tid = threadIdx.x;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  const uint8_t* up = a.up;
  if (tid <= kUpgHdrStatus && reinterpret_cast<const uint32_t*>(up)[tid] != upg_header_word(a, tid))
    atomicOr(&s_bad, 1u);
  __syncthreads();
  if (s_bad) {
    if (tid == 0) *a.status = static_cast<uint32_t>(SKV_ERR_FORMAT);
    return;
  }
  bool bad = token_list_bad(reinterpret_cast<const int32_t*>(up + a.tokens_off), a.m, a.n, nullptr,
                            up + a.tiers_off);
  const int nbt = (a.n + a.block_size - 1) / a.block_size;
  for (int base = tid; base < nbt; base += kListBatch * kUpgCheckThreads) {
    int b[kListBatch];
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) {
      const int i = base + u * kUpgCheckThreads;
      b[u] = i < nbt ? a.block_table[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < kListBatch; ++u) bad |= b[u] < 0 || b[u] >= a.num_blocks;
  }
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  if (tid == 0) *a.status = s_bad ? static_cast<uint32_t>(SKV_ERR_FORMAT) : 0u;
}

// out = RN16(RN32(held + RN32(code * scale))) for the lane's 8 elements.
__device__ __forceinline__ u32x4 add_residual(u32x4 held, u32x2 c, float scale) {
  const uint32_t hs[4] = {held.x, held.y, held.z, held.w};
  const uint32_t cw[2] = {c.x, c.y};
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t w = cw[j >> 1];
    const int sh = 16 * (j & 1);
    const float c0 = static_cast<float>(static_cast<int32_t>(w << (24 - sh)) >> 24) * scale;
    const float c1 = static_cast<float>(static_cast<int32_t>(w << (16 - sh)) >> 24) * scale;
    o[j] = pack_half2(half_lo(hs[j]) + c0, half_hi(hs[j]) + c1);
  }
  const u32x4 out{o[0], o[1], o[2], o[3]};
  // only an infinite scale makes a NaN (code 0, or an infinity of the other
  // sign): written as 0x7E00
  return __builtin_isinf(scale) ? canon_nan_lane(out) : out;
}

template <int D, int MODE>
__global__ __launch_bounds__(kUpgThreads) void upg_apply(const UpgArgs a) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kUpgThreads / LPR;
  constexpr int ITERS = kUpgThreads / RPI;
  constexpr int U = ITERS < 4 ? ITERS : 4;
  static_assert(ITERS % U == 0, "rows in flight must divide a thread's rows of the chunk");
  __shared__ uint32_t s_pos[kUpgThreads];
  if (*a.status != 0u) return;
  const uint8_t* up = a.up;
  const int nch = (a.m + kUpgThreads - 1) / kUpgThreads;
  const int chunk = blockIdx.x % nch, seg = blockIdx.x / nch;
  const int h = seg % a.H, kv = (seg / a.H) & 1, l = seg / (2 * a.H);
  const int i0 = chunk * kUpgThreads;
  {
    const int i = i0 + threadIdx.x;
    uint32_t pos = 0;
    if (i < a.m) {
      const int t = reinterpret_cast<const int32_t*>(up + a.tokens_off)[i];
      pos = static_cast<uint32_t>(a.block_table[t / a.block_size]) * static_cast<uint32_t>(a.block_size) +
            static_cast<uint32_t>(t % a.block_size);
    }
    s_pos[threadIdx.x] = pos;
  }
  __syncthreads();
  uint16_t* cache = (kv ? a.v_cache : a.k_cache) + static_cast<size_t>(l) * a.num_blocks * a.block_size * a.H * D +
                    static_cast<size_t>(h) * D;
  const uint64_t seg_rows = static_cast<uint64_t>(seg) * a.m;
  const int lane = threadIdx.x % LPR, rsub = threadIdx.x / LPR;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    if constexpr (MODE == 0) {
      u32x4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + (it + u) * RPI + rsub;
        if (i < a.m) x[u] = ld_nt16(up + a.data_off + (seg_rows + i) * (2 * D) + lane * 16);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = (it + u) * RPI + rsub;
        if (i0 + r < a.m) st_nt16(cache + static_cast<size_t>(s_pos[r]) * a.H * D + lane * 8, x[u]);
      }
    } else {
      u32x2 c[U];
      u32x4 held[U];
      float scale[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = (it + u) * RPI + rsub;
        const int i = i0 + r;
        scale[u] = __builtin_bit_cast(float, 0x7FC00000u);
        if (i < a.m) {
          scale[u] = reinterpret_cast<const float*>(up + a.scales_off)[seg_rows + i];
          c[u] = ld_nt8(up + a.data_off + (seg_rows + i) * D + lane * 8);
          held[u] = *reinterpret_cast<const u32x4*>(cache + static_cast<size_t>(s_pos[r]) * a.H * D + lane * 8);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = (it + u) * RPI + rsub;
        // a NaN scale (also set for rows past m) keeps the held row
        if (!__builtin_isnan(scale[u]))
          *reinterpret_cast<u32x4*>(cache + static_cast<size_t>(s_pos[r]) * a.H * D + lane * 8) =
              add_residual(held[u], c[u], scale[u]);
      }
    }
  }
}

inline uint64_t up256(uint64_t x) { return (x + 255u) / 256u * 256u; }

template <int MODE, typename F>
hipError_t dispatch_d(int d, F&& f) {
  switch (d) {
    case 32: return f(std::integral_constant<int, 32>{}, std::integral_constant<int, MODE>{});
    case 64: return f(std::integral_constant<int, 64>{}, std::integral_constant<int, MODE>{});
    case 128: return f(std::integral_constant<int, 128>{}, std::integral_constant<int, MODE>{});
    case 256: return f(std::integral_constant<int, 256>{}, std::integral_constant<int, MODE>{});
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

uint64_t upgrade_bytes(int32_t L, int32_t H, int32_t d, int32_t m, int32_t mode, uint64_t* offsets) {
  const uint64_t rows = 2ull * L * H * static_cast<uint64_t>(m);
  const uint64_t tokens_off = 256, tiers_off = tokens_off + up256(4ull * m);
  const uint64_t scales_off = tiers_off + up256(static_cast<uint64_t>(m));
  const uint64_t data_off = scales_off + (mode == 1 ? up256(rows * 4) : 0);
  const uint64_t row_bytes = mode == 0 ? 2ull * d : static_cast<uint64_t>(d);
  const uint64_t total = data_off + rows * row_bytes;
  if (offsets) {
    offsets[0] = tokens_off;
    offsets[1] = tiers_off;
    offsets[2] = scales_off;
    offsets[3] = data_off;
    offsets[4] = total;
    offsets[5] = row_bytes;
  }
  return total;
}

static UpgArgs upg_args(const Geometry& g, int32_t m, int32_t mode) {
  UpgArgs a{};
  a.L = g.L;
  a.H = g.H;
  a.d = g.d;
  a.n = g.n;
  a.m = m;
  a.mode = mode;
  uint64_t off[6];
  upgrade_bytes(g.L, g.H, g.d, m, mode, off);
  a.tokens_off = off[0];
  a.tiers_off = off[1];
  a.scales_off = off[2];
  a.data_off = off[3];
  a.total = off[4];
  a.row_bytes = off[5];
  return a;
}

hipError_t launch_pack_upgrade(const Geometry& g, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
                               const int32_t* tokens, int32_t m, int32_t mode, uint8_t* out, uint32_t* status,
                               hipStream_t stream) {
  UpgArgs a = upg_args(g, m, mode);
  a.k = k;
  a.v = v;
  a.tier = tier;
  a.tokens = tokens;
  a.up = out;
  a.status = status;
  upg_prep<<<1, kUpgCheckThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint64_t blocks = static_cast<uint64_t>((m + kUpgThreads - 1) / kUpgThreads) * 2u * g.L * g.H;
  auto run = [&](auto D, auto M) {
    upg_rows<decltype(D)::value, decltype(M)::value><<<blocks, kUpgThreads, 0, stream>>>(a);
    return hipGetLastError();
  };
  return mode == 0 ? dispatch_d<0>(g.d, run) : dispatch_d<1>(g.d, run);
}

hipError_t launch_unpack_upgrade(const Geometry& g, const uint8_t* up, int32_t m, int32_t mode, uint16_t* k_cache,
                                 uint16_t* v_cache, const int32_t* block_table, int32_t num_blocks,
                                 int32_t block_size, uint32_t* status, hipStream_t stream) {
  UpgArgs a = upg_args(g, m, mode);
  a.up = const_cast<uint8_t*>(up);
  a.status = status;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_table = block_table;
  a.num_blocks = num_blocks;
  a.block_size = block_size;
  upg_check<<<1, kUpgCheckThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint64_t blocks = static_cast<uint64_t>((m + kUpgThreads - 1) / kUpgThreads) * 2u * g.L * g.H;
  auto run = [&](auto D, auto M) {
    upg_apply<decltype(D)::value, decltype(M)::value><<<blocks, kUpgThreads, 0, stream>>>(a);
    return hipGetLastError();
  };
  return mode == 0 ? dispatch_d<0>(g.d, run) : dispatch_d<1>(g.d, run);
}

}  // namespace skv
