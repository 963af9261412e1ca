// Tier-map bookkeeping shared by pack (which writes the map and the chunk
// index) and unpack (which checks them): one thread reads the codes of a
// group of 16 consecutive tokens; the 16 groups of a 256-token chunk sit in
// 16 consecutive lanes, so chunk sums are a 16-lane reduction.
#pragma once

#include "device_util.h"
#include "skv_internal.h"

namespace skv {

constexpr int kGroupTokens = 16;
constexpr int kGroupsPerChunk = kChunkTokens / kGroupTokens;  // 16

struct TierGroup {
  uint32_t units;  // sum of row widths in units of d/2 bytes
  uint32_t quant;  // number of INT8/INT4 rows
  uint32_t map2;   // the 16 codes, 2 bits each (token 16g+j at bits 2j..2j+1)
  uint32_t cnt4;   // tokens per tier, one byte per tier (at most 16 each)
  bool bad;        // a code outside 0..3 (byte input only)

  __device__ __forceinline__ uint32_t count(int tier) const { return (cnt4 >> (8 * tier)) & 0xFFu; }
};

// Branch-free: a code outside 0..3 sets bad, keeps its low two bits in the
// map and is not counted.
__device__ __forceinline__ void tally(TierGroup& gi, uint32_t code, int j) {
  const uint32_t c = code & 3u;
  const uint32_t ok = code <= 3u ? 1u : 0u;
  gi.map2 |= c << (2 * j);
  gi.bad |= ok == 0u;
  gi.cnt4 += ok << (8 * c);
  gi.units += ok * ((0x124u >> (4 * c)) & 0xFu);  // 4, 2, 1, 0 for FP16, INT8, INT4, DROP
  gi.quant += ok & (0x6u >> c);                   // INT8 and INT4 carry a scale
}

__device__ __forceinline__ TierGroup empty_group() {
  TierGroup gi;
  gi.units = gi.quant = gi.map2 = gi.cnt4 = 0;
  gi.bad = false;
  return gi;
}

// Codes from a uint8[n] tier array (16-byte loads where the group is
// 16-byte aligned, as it always is for an aligned array; bytes otherwise).
__device__ __forceinline__ TierGroup group_from_bytes(const uint8_t* __restrict__ tier, int n, int g) {
  TierGroup gi = empty_group();
  const int t0 = g * kGroupTokens;
  if (t0 + kGroupTokens <= n && (reinterpret_cast<uintptr_t>(tier + t0) & 15u) == 0) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(tier + t0);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int j = 0; j < 16; ++j) tally(gi, (ws[j >> 2] >> (8 * (j & 3))) & 0xFFu, j);
  } else {
    for (int j = 0; j < kGroupTokens && t0 + j < n; ++j) tally(gi, tier[t0 + j], j);
  }
  return gi;
}

// Codes of group g from its 16 tier bytes already loaded as w (a whole,
// 16-byte-aligned group).
__device__ __forceinline__ TierGroup group_from_tier_words(u32x4 w) {
  TierGroup gi = empty_group();
  const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int j = 0; j < 16; ++j) tally(gi, (ws[j >> 2] >> (8 * (j & 3))) & 0xFFu, j);
  return gi;
}

// Whether group g of a uint8[n] tier array is whole and 16-byte aligned (then
// its 16 bytes are one load).
__device__ __forceinline__ bool tier_group_is_word(const uint8_t* tier, int n, int g) {
  const int t0 = g * kGroupTokens;
  return t0 + kGroupTokens <= n && (reinterpret_cast<uintptr_t>(tier + t0) & 15u) == 0;
}

// Codes of group g from its map word w (the payload's 2-bit tier map); codes
// of tokens >= n are ignored.
__device__ __forceinline__ TierGroup group_from_map_word(uint32_t w, int n, int g) {
  TierGroup gi = empty_group();
  const int t0 = g * kGroupTokens;
#pragma unroll
  for (int j = 0; j < kGroupTokens; ++j)
    if (t0 + j < n) tally(gi, (w >> (2 * j)) & 3u, j);
  return gi;
}

// Codes from the payload's 2-bit tier map; codes of tokens >= n are ignored.
__device__ __forceinline__ TierGroup group_from_map(const uint8_t* __restrict__ map, int n, int g) {
  return group_from_map_word(*reinterpret_cast<const uint32_t*>(map + 4 * g), n, g);
}

// Sum over aligned 16-lane groups (the DPP rows); every lane gets its group's
// sum: quad swaps leave each lane its quad's sum, then the half-row mirror
// (lane i <-> 7 - i) pairs the quads of each half and the row mirror
// (i <-> 15 - i) the halves.  Every lane of the row must be active.
__device__ __forceinline__ uint32_t sum16(uint32_t v) {
  v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  v += dpp_mov<0x140>(v);  // row_mirror
  return v;
}

// Exclusive prefix sum of one 64-bit value per thread over a 1024-thread
// block.  `scratch` holds at least 16 words of shared memory.  Every thread
// must call it; contains __syncthreads().
__device__ __forceinline__ uint64_t block_exclusive_scan_1024(uint64_t x, uint64_t* scratch) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  uint64_t base = 0;
  for (int w = 0; w < wave; ++w) base += scratch[w];
  __syncthreads();
  return base + inc - x;
}

// Word i (0..63) of the 256-byte payload header of request r, as pack writes it
// (non-finite row count and status zero).  Layout: 0 magic, 1 version, 2..5
// L, H, d, n, 6 sinks, 7 tiers, 8..10 budget / first-ratio / decay bits,
// 11 score mode, 12..15 tier counts, 16..35 u64 budget units, used units,
// tier-map, chunk-index and layer-0 offsets, segment bytes, segment stride,
// scale bytes, layer stride, total bytes; 36 non-finite rows, 37 status,
// 38 tokens per chunk.
__device__ __forceinline__ uint32_t header_word(const BatchArgs& a, const ReqDesc& r, int i) {
  auto lo = [](uint64_t x) { return static_cast<uint32_t>(x); };
  auto hi = [](uint64_t x) { return static_cast<uint32_t>(x >> 32); };
  switch (i) {
    case 0: return kMagic;
    case 1: return kVersion;
    case 2: return static_cast<uint32_t>(a.L);
    case 3: return static_cast<uint32_t>(a.H);
    case 4: return static_cast<uint32_t>(a.d);
    case 5: return static_cast<uint32_t>(r.n);
    case 6: return static_cast<uint32_t>(r.n_sink);
    case 7: return static_cast<uint32_t>(a.num_tiers);
    case 8: return a.budget_bits;
    case 9: return a.rho_bits;
    case 10: return a.decay_bits;
    case 11: return static_cast<uint32_t>(a.score_mode);
    case 12: return static_cast<uint32_t>(r.n16);
    case 13: return static_cast<uint32_t>(r.n8);
    case 14: return static_cast<uint32_t>(r.n4);
    case 15: return static_cast<uint32_t>(r.nd);
    case 16: return lo(static_cast<uint64_t>(r.budget_units));
    case 17: return hi(static_cast<uint64_t>(r.budget_units));
    case 18: return lo(static_cast<uint64_t>(r.used_units));
    case 19: return hi(static_cast<uint64_t>(r.used_units));
    case 20: return 256u;  // tier map right after the header
    case 21: return 0u;
    case 22: return lo(r.chunkidx_off);
    case 23: return hi(r.chunkidx_off);
    case 24: return lo(r.layers_off);
    case 25: return hi(r.layers_off);
    case 26: return lo(r.seg_bytes);
    case 27: return hi(r.seg_bytes);
    case 28: return lo(r.seg_stride);
    case 29: return hi(r.seg_stride);
    case 30: return lo(r.scales_bytes);
    case 31: return hi(r.scales_bytes);
    case 32: return lo(r.layer_stride);
    case 33: return hi(r.layer_stride);
    case 34: return lo(r.total);
    case 35: return hi(r.total);
    case 38: return static_cast<uint32_t>(kChunkTokens);
    case 39: return static_cast<uint32_t>(a.q8);
    case 40: return static_cast<uint32_t>(a.q4);
    case 42: return lo(r.channel_bytes);
    case 43: return hi(r.channel_bytes);
    default: return 0u;
  }
}
constexpr int kHdrNonfinite = 36;
constexpr int kHdrStatus = 37;

// The request that owns flat workgroup `bid` of a batched row launch.
__device__ __forceinline__ int request_of_block(const BatchArgs& a, uint64_t bid) {
  int r = 0;
  for (int i = 1; i < a.count; ++i)
    if (a.r[i].block_begin <= bid) r = i;
  return r;
}

}  // namespace skv
