// Per-layer and per-head tier maps (the extension named in Sec. 2.6,
// Sec. 6.10, Sec. 7.5 and Sec. 9 (iii)): the (layer, head) pairs are split
// into G groups, one per layer or one per (layer, head), and each group has
// its own budget, plan and tier map.  The grouped payload carries a group
// table, G tier maps and G chunk indexes, and a segment table with the
// offsets of every segment's scales and rows (segment sizes differ between
// groups).  Row work is the per-token codec's (row_stream.h); only the
// lookups of a segment's group, map, chunk index and offsets differ.
//   gpack_init    zeroes the header's non-finite counter and status words
//                 and the caller's status word;
//   gpack_prep    one workgroup per group checks the group's tier map against
//                 its plan and writes its 2-bit map and chunk index; one more
//                 workgroup writes the header, group table and segment table;
//   gpack_rows    one workgroup per (segment, 256-token chunk);
//   gunpack_init, gunpack_check (one workgroup per group + one for header
//                 and tables), gunpack_rows: the decode side.
#include "device_util.h"
#include "row_codec.h"
#include "row_stream.h"
#include "skv_internal.h"
#include "tier_groups.h"

namespace skv {
namespace {

constexpr int kPrepThreads = 1024;
constexpr int kMaxChunks = kMaxTokens / kChunkTokens;
constexpr uint32_t kGroupMagic = 0x47564B53u;  // "SKVG"
constexpr int kGHdrNonfinite = 32;
constexpr int kGHdrStatus = 33;

struct GroupArgs {
  const uint16_t* k;
  const uint16_t* v;
  const uint8_t* tier;          // pack: uint8 [G][n]
  uint8_t* payload;
  uint32_t* status;             // pack: optional; unpack: required
  const uint32_t* group_table;  // workspace: G x 8 words
  const uint64_t* segtab;       // workspace: 2LH x {scales offset, rows offset}
  const int32_t* block_table;
  int32_t num_blocks, block_size;
  int32_t L, H, d, n, gran, G, nchunks, num_tiers, score_mode, num_sink;
  uint32_t budget_bits, rho_bits, decay_bits;
  uint64_t group_off, tiermaps_off, tiermap_stride, chunkidx_off, chunkidx_stride, segtab_off, layers_off, total;
};

__device__ __forceinline__ int group_of(const GroupArgs& a, int l, int h) {
  return a.gran == SKV_GROUP_TOKEN ? 0 : a.gran == SKV_GROUP_LAYER ? l : l * a.H + h;
}

__device__ __forceinline__ uint32_t lo32(uint64_t x) { return static_cast<uint32_t>(x); }
__device__ __forceinline__ uint32_t hi32(uint64_t x) { return static_cast<uint32_t>(x >> 32); }

__device__ __forceinline__ uint32_t gheader_word(const GroupArgs& a, int i) {
  switch (i) {
    case 0: return kGroupMagic;
    case 1: return kVersion;
    case 2: return static_cast<uint32_t>(a.L);
    case 3: return static_cast<uint32_t>(a.H);
    case 4: return static_cast<uint32_t>(a.d);
    case 5: return static_cast<uint32_t>(a.n);
    case 6: return static_cast<uint32_t>(a.gran);
    case 7: return static_cast<uint32_t>(a.G);
    case 8: return static_cast<uint32_t>(a.num_tiers);
    case 9: return static_cast<uint32_t>(a.score_mode);
    case 10: return a.budget_bits;
    case 11: return a.rho_bits;
    case 12: return a.decay_bits;
    case 13: return static_cast<uint32_t>(a.num_sink);
    case 14: return static_cast<uint32_t>(kChunkTokens);
    case 16: return lo32(a.group_off);
    case 17: return hi32(a.group_off);
    case 18: return lo32(a.tiermaps_off);
    case 19: return hi32(a.tiermaps_off);
    case 20: return lo32(a.tiermap_stride);
    case 21: return hi32(a.tiermap_stride);
    case 22: return lo32(a.chunkidx_off);
    case 23: return hi32(a.chunkidx_off);
    case 24: return lo32(a.chunkidx_stride);
    case 25: return hi32(a.chunkidx_stride);
    case 26: return lo32(a.segtab_off);
    case 27: return hi32(a.segtab_off);
    case 28: return lo32(a.layers_off);
    case 29: return hi32(a.layers_off);
    case 30: return lo32(a.total);
    case 31: return hi32(a.total);
    default: return 0u;  // 15, the counters (32, 33) and the reserved words
  }
}

// Bytes of a group's segment rows (before padding).
__device__ __forceinline__ uint64_t group_seg_bytes(const uint32_t* e, int D) {
  return static_cast<uint64_t>(e[0] + e[1]) * (2 * D) + static_cast<uint64_t>(e[2]) * D +
         static_cast<uint64_t>(e[3]) * (D / 2);
}

__global__ void gpack_init(const GroupArgs a) {
  uint32_t* hdr = reinterpret_cast<uint32_t*>(a.payload);
  if (threadIdx.x == 0) {
    hdr[kGHdrNonfinite] = 0u;
    hdr[kGHdrStatus] = 0u;
    if (a.status) *a.status = 0u;
  }
}

// Zero-fills payload bytes [b0, b1), 4 bytes per store (both multiples of 4).
__device__ __forceinline__ void zero_range(uint8_t* p, uint64_t b0, uint64_t b1, int tid, int nthreads) {
  for (uint64_t b = b0 + 4ull * tid; b < b1; b += 4ull * nthreads) *reinterpret_cast<uint32_t*>(p + b) = 0u;
}

// grid: G + 1 workgroups
__global__ __launch_bounds__(kPrepThreads) void gpack_prep(const GroupArgs a) {
  __shared__ uint32_t s_chunk[kMaxChunks];
  __shared__ uint32_t s_cnt[4];
  __shared__ uint32_t s_bad;
  __shared__ uint64_t s_scan[16];
  uint8_t* __restrict__ payload = a.payload;
  const int tid = threadIdx.x;
  if (blockIdx.x == static_cast<unsigned>(a.G)) {
    // header (but the two counters), group table, segment table and their padding
    uint32_t* hdr = reinterpret_cast<uint32_t*>(payload);
    if (tid < 64 && tid != kGHdrNonfinite && tid != kGHdrStatus) hdr[tid] = gheader_word(a, tid);
    uint32_t* gt = reinterpret_cast<uint32_t*>(payload + a.group_off);
    for (int i = tid; i < 8 * a.G; i += kPrepThreads) gt[i] = a.group_table[i];
    zero_range(payload, a.group_off + 32ull * a.G, a.tiermaps_off, tid, kPrepThreads);
    uint64_t* st = reinterpret_cast<uint64_t*>(payload + a.segtab_off);
    const int nseg = 2 * a.L * a.H;
    for (int i = tid; i < 2 * nseg; i += kPrepThreads) st[i] = a.segtab[i];
    zero_range(payload, a.segtab_off + 16ull * nseg, a.layers_off, tid, kPrepThreads);
    return;
  }
  const int g = blockIdx.x;
  const uint32_t* e = a.group_table + 8 * g;
  const uint8_t* __restrict__ tier = a.tier + static_cast<size_t>(g) * a.n;
  const int n = a.n, nchunks = a.nchunks;
  const int ngroups = (n + kGroupTokens - 1) / kGroupTokens;
  if (tid < 4) s_cnt[tid] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  uint32_t cnt[4] = {0, 0, 0, 0};
  bool bad = false;
  for (int base = 0; base < ngroups; base += kPrepThreads) {  // block-uniform trip count
    const int q = base + tid;
    const TierGroup gi = q < ngroups ? group_from_bytes(tier, n, q) : empty_group();
#pragma unroll
    for (int i = 0; i < 4; ++i) cnt[i] += gi.count(i);
    bad |= gi.bad;
    const uint32_t u = sum16(gi.units), qs = sum16(gi.quant);
    if ((tid % kGroupsPerChunk) == 0 && q < ngroups) s_chunk[q / kGroupsPerChunk] = u | (qs << 16);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (cnt[i]) atomicAdd(&s_cnt[i], cnt[i]);
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  const bool ok = !s_bad && s_cnt[0] == e[0] + e[1] && s_cnt[1] == e[2] && s_cnt[2] == e[3] && s_cnt[3] == e[4];
  if (!ok) {  // block-uniform
    if (tid == 0) {
      atomicOr(reinterpret_cast<uint32_t*>(payload) + kGHdrStatus, static_cast<uint32_t>(SKV_ERR_INVALID_ARG));
      if (a.status) atomicOr(a.status, static_cast<uint32_t>(SKV_ERR_INVALID_ARG));
    }
    return;
  }
  // chunk index of the group (running sums at every chunk start) and padding
  const int per = (nchunks + kPrepThreads - 1) / kPrepThreads;
  const int c0 = min(nchunks, tid * per), c1 = min(nchunks, c0 + per);
  uint64_t run = 0;
  for (int c = c0; c < c1; ++c) run += (s_chunk[c] & 0xFFFFu) | (static_cast<uint64_t>(s_chunk[c] >> 16) << 32);
  const uint64_t ex = block_exclusive_scan_1024(run, s_scan);
  uint32_t ru = static_cast<uint32_t>(ex), rq = static_cast<uint32_t>(ex >> 32);
  const uint64_t ci_off = a.chunkidx_off + static_cast<uint64_t>(g) * a.chunkidx_stride;
  uint32_t* cidx = reinterpret_cast<uint32_t*>(payload + ci_off);
  for (int c = c0; c < c1; ++c) {
    cidx[2 * c] = ru;
    cidx[2 * c + 1] = rq;
    ru += s_chunk[c] & 0xFFFFu;
    rq += s_chunk[c] >> 16;
  }
  zero_range(payload, ci_off + 8ull * nchunks, ci_off + a.chunkidx_stride, tid, kPrepThreads);
  // the group's 2-bit map (4 bytes per 16 tokens) and padding
  const uint64_t map_off = a.tiermaps_off + static_cast<uint64_t>(g) * a.tiermap_stride;
  for (int q = tid; q < ngroups; q += kPrepThreads)
    *reinterpret_cast<uint32_t*>(payload + map_off + 4ull * q) = group_from_bytes(tier, n, q).map2;
  zero_range(payload, map_off + 4ull * ngroups, map_off + a.tiermap_stride, tid, kPrepThreads);
}

// grid: 2 * L * H * nchunks workgroups, chunk fastest
template <int D>
__global__ __launch_bounds__(kRowThreads) void gpack_rows(const GroupArgs a) {
  __shared__ ChunkLds s;
  uint8_t* __restrict__ payload = a.payload;
  uint32_t* hdr = reinterpret_cast<uint32_t*>(payload);
  const int n = a.n, H = a.H, nchunks = a.nchunks;
  const int chunk = static_cast<int>(blockIdx.x % static_cast<unsigned>(nchunks));
  const int seg = static_cast<int>(blockIdx.x / static_cast<unsigned>(nchunks));  // (l * 2 + kv) * H + h
  const int h = seg % H, kv = (seg / H) & 1, l = seg / (2 * H);
  const int g = group_of(a, l, h);
  const int t0 = chunk * kChunkTokens;
  const uint8_t* tier = a.tier + static_cast<size_t>(g) * n;
  const uint16_t* src = (kv ? a.v : a.k) + (static_cast<size_t>(l) * H + h) * static_cast<size_t>(n) * D;
  // the first rows are loaded before the status check and the layout scan
  RowBatch<D, pack_rows_in_flight<D>()> first;
  pack_first_batch<D, pack_rows_in_flight<D>()>(first, src, tier, t0, n);
  if (hdr[kGHdrStatus] != 0u) return;  // a tier map is off its plan: nothing to pack
  {
    const int t = t0 + threadIdx.x;
    chunk_layout<D>(s, t < n ? tier[t] : kDROP,
                    reinterpret_cast<const uint32_t*>(payload + a.chunkidx_off +
                                                      static_cast<uint64_t>(g) * a.chunkidx_stride) +
                        2 * chunk);
  }
  __syncthreads();
  const uint64_t sc_off = a.segtab[2 * seg], row_off = a.segtab[2 * seg + 1];
  uint8_t* dst = payload + row_off;
  pack_chunk<D, pack_rows_in_flight<D>(), pack_nt_store<D>()>(s, first, src, dst,
                                                            reinterpret_cast<float*>(payload + sc_off),
                                                            hdr + kGHdrNonfinite, t0, n);
  const uint32_t* e = a.group_table + 8 * g;
  if (chunk == nchunks - 1) {  // segment tail
    const uint64_t used = group_seg_bytes(e, D);
    const uint64_t stride = (used + 255u) / 256u * 256u;
    for (uint64_t b = used + 16ull * threadIdx.x; b < stride; b += 16ull * kRowThreads)
      st_nt16(dst + b, u32x4{0u, 0u, 0u, 0u});
  }
  if (chunk == 0 && kv == 1 && h == H - 1) {  // the layer's scale-section tail
    const uint64_t end = sc_off + 4ull * e[6];
    const uint64_t first_rows = a.segtab[2 * (l * 2 * H) + 1];
    zero_range(payload, end, first_rows, threadIdx.x, kRowThreads);
  }
}

__global__ void gunpack_init(const GroupArgs a) {
  if (threadIdx.x == 0) *a.status = 0u;
}

// grid: G + 1 workgroups.  Every metadata byte must be what the
// configuration, the group plans and the payload's own tier maps imply (the
// non-finite counter excepted); a failure sets the status to SKV_ERR_FORMAT.
__global__ __launch_bounds__(kPrepThreads) void gunpack_check(const GroupArgs a) {
  __shared__ uint32_t s_chunk[kMaxChunks];
  __shared__ uint32_t s_cnt[4];
  __shared__ uint32_t s_bad;
  __shared__ uint64_t s_scan[16];
  const uint8_t* __restrict__ payload = a.payload;
  const int tid = threadIdx.x;
  if (tid < 4) s_cnt[tid] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  bool bad = false;
  if (blockIdx.x == static_cast<unsigned>(a.G)) {
    const uint32_t* hdr = reinterpret_cast<const uint32_t*>(payload);
    if (tid < 64 && tid != kGHdrNonfinite) bad |= hdr[tid] != gheader_word(a, tid);
    const uint32_t* gt = reinterpret_cast<const uint32_t*>(payload + a.group_off);
    for (int i = tid; i < 8 * a.G; i += kPrepThreads) bad |= gt[i] != a.group_table[i];
    for (uint64_t b = a.group_off + 32ull * a.G + 4ull * tid; b < a.tiermaps_off; b += 4ull * kPrepThreads)
      bad |= *reinterpret_cast<const uint32_t*>(payload + b) != 0u;
    const uint64_t* st = reinterpret_cast<const uint64_t*>(payload + a.segtab_off);
    const int nseg = 2 * a.L * a.H;
    for (int i = tid; i < 2 * nseg; i += kPrepThreads) bad |= st[i] != a.segtab[i];
    for (uint64_t b = a.segtab_off + 16ull * nseg + 4ull * tid; b < a.layers_off; b += 4ull * kPrepThreads)
      bad |= *reinterpret_cast<const uint32_t*>(payload + b) != 0u;
    const int nbt = (a.n + a.block_size - 1) / a.block_size;
    for (int i = tid; i < nbt; i += kPrepThreads) {
      const int b = a.block_table[i];
      bad |= b < 0 || b >= a.num_blocks;
    }
    if (bad) atomicOr(&s_bad, 1u);
    __syncthreads();
    if (tid == 0 && s_bad) atomicOr(a.status, static_cast<uint32_t>(SKV_ERR_FORMAT));
    return;
  }
  const int g = blockIdx.x;
  const uint32_t* e = a.group_table + 8 * g;
  const int n = a.n, nchunks = a.nchunks;
  const int ngroups = (n + kGroupTokens - 1) / kGroupTokens;
  const uint64_t map_off = a.tiermaps_off + static_cast<uint64_t>(g) * a.tiermap_stride;
  const uint8_t* map = payload + map_off;
  uint32_t cnt[4] = {0, 0, 0, 0};
  for (int base = 0; base < ngroups; base += kPrepThreads) {
    const int q = base + tid;
    const TierGroup gi = q < ngroups ? group_from_map(map, n, q) : empty_group();
#pragma unroll
    for (int i = 0; i < 4; ++i) cnt[i] += gi.count(i);
    const uint32_t u = sum16(gi.units), qs = sum16(gi.quant);
    if ((tid % kGroupsPerChunk) == 0 && q < ngroups) s_chunk[q / kGroupsPerChunk] = u | (qs << 16);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (cnt[i]) atomicAdd(&s_cnt[i], cnt[i]);
  // codes of tokens >= n in the last word, and the map's padding, are zero
  if (tid == 0 && (n % kGroupTokens) != 0) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(map + 4ull * (ngroups - 1));
    bad |= (w >> (2 * (n % kGroupTokens))) != 0u;
  }
  for (uint64_t b = 4ull * ngroups + 4ull * tid; b < a.tiermap_stride; b += 4ull * kPrepThreads)
    bad |= *reinterpret_cast<const uint32_t*>(map + b) != 0u;
  __syncthreads();
  bad |= s_cnt[0] != e[0] + e[1] || s_cnt[1] != e[2] || s_cnt[2] != e[3] || s_cnt[3] != e[4];
  // the chunk index equals the running sums; its padding is zero
  const int per = (nchunks + kPrepThreads - 1) / kPrepThreads;
  const int c0 = min(nchunks, tid * per), c1 = min(nchunks, c0 + per);
  uint64_t run = 0;
  for (int c = c0; c < c1; ++c) run += (s_chunk[c] & 0xFFFFu) | (static_cast<uint64_t>(s_chunk[c] >> 16) << 32);
  const uint64_t ex = block_exclusive_scan_1024(run, s_scan);
  uint32_t ru = static_cast<uint32_t>(ex), rq = static_cast<uint32_t>(ex >> 32);
  const uint64_t ci_off = a.chunkidx_off + static_cast<uint64_t>(g) * a.chunkidx_stride;
  const uint32_t* cidx = reinterpret_cast<const uint32_t*>(payload + ci_off);
  for (int c = c0; c < c1; ++c) {
    bad |= cidx[2 * c] != ru || cidx[2 * c + 1] != rq;
    ru += s_chunk[c] & 0xFFFFu;
    rq += s_chunk[c] >> 16;
  }
  for (uint64_t b = 8ull * nchunks + 4ull * tid; b < a.chunkidx_stride; b += 4ull * kPrepThreads)
    bad |= *reinterpret_cast<const uint32_t*>(payload + ci_off + b) != 0u;
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  if (tid == 0 && s_bad) atomicOr(a.status, static_cast<uint32_t>(SKV_ERR_FORMAT));
}

// grid: 2 * L * H * nchunks workgroups, chunk fastest
template <int D>
__global__ __launch_bounds__(kRowThreads) void gunpack_rows(const GroupArgs a, uint16_t* __restrict__ k_cache,
                                                            uint16_t* __restrict__ v_cache) {
  __shared__ ChunkLds s;
  if (*a.status != 0u) return;  // payload rejected: write nothing
  const uint8_t* __restrict__ payload = a.payload;
  const int n = a.n, H = a.H, nchunks = a.nchunks, block_size = a.block_size;
  const int chunk = static_cast<int>(blockIdx.x % static_cast<unsigned>(nchunks));
  const int seg = static_cast<int>(blockIdx.x / static_cast<unsigned>(nchunks));
  const int h = seg % H, kv = (seg / H) & 1, l = seg / (2 * H);
  const int g = group_of(a, l, h);
  const int t0 = chunk * kChunkTokens;
  {
    const int t = t0 + threadIdx.x;
    int tr = kAbsent;
    uint32_t pos = 0;
    if (t < n) {
      const uint8_t* map = payload + a.tiermaps_off + static_cast<uint64_t>(g) * a.tiermap_stride;
      tr = (map[t >> 2] >> (2 * (t & 3))) & 3;
      pos = static_cast<uint32_t>(a.block_table[t / block_size]) * static_cast<uint32_t>(block_size) +
            static_cast<uint32_t>(t % block_size);
    }
    chunk_layout<D>(s, tr,
                    reinterpret_cast<const uint32_t*>(payload + a.chunkidx_off +
                                                      static_cast<uint64_t>(g) * a.chunkidx_stride) +
                        2 * chunk);
    stage_scale(s, tr, reinterpret_cast<const float*>(payload + a.segtab[2 * seg]));
    s.pos[threadIdx.x] = pos;
  }
  __syncthreads();
  const uint8_t* src = payload + a.segtab[2 * seg + 1];
  uint16_t* cache = (kv ? v_cache : k_cache) + static_cast<size_t>(l) * a.num_blocks * block_size * H * D +
                    static_cast<size_t>(h) * D;
  unpack_chunk<D, unpack_rows_in_flight<D>(), unpack_nt_store<D>()>(s, src, cache, H);
}

GroupArgs group_args(const GroupLaunch& gl) {
  GroupArgs a{};
  a.group_table = gl.group_table;
  a.segtab = gl.segtab;
  a.L = gl.L;
  a.H = gl.H;
  a.d = gl.d;
  a.n = gl.n;
  a.gran = gl.gran;
  a.G = gl.G;
  a.nchunks = gl.nchunks;
  a.num_tiers = gl.num_tiers;
  a.score_mode = gl.score_mode;
  a.num_sink = gl.num_sink;
  a.budget_bits = gl.budget_bits;
  a.rho_bits = gl.rho_bits;
  a.decay_bits = gl.decay_bits;
  a.group_off = gl.group_off;
  a.tiermaps_off = gl.tiermaps_off;
  a.tiermap_stride = gl.tiermap_stride;
  a.chunkidx_off = gl.chunkidx_off;
  a.chunkidx_stride = gl.chunkidx_stride;
  a.segtab_off = gl.segtab_off;
  a.layers_off = gl.layers_off;
  a.total = gl.total;
  return a;
}

}  // namespace

hipError_t launch_pack_groups(const GroupLaunch& gl, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
                              uint8_t* payload, uint32_t* status, hipStream_t stream) {
  GroupArgs a = group_args(gl);
  a.k = k;
  a.v = v;
  a.tier = tier;
  a.payload = payload;
  a.status = status;
  gpack_init<<<1, 64, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  gpack_prep<<<a.G + 1, kPrepThreads, 0, stream>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint64_t blocks = 2ull * a.L * a.H * static_cast<uint64_t>(a.nchunks);
  switch (a.d) {
    case 32: gpack_rows<32><<<blocks, kRowThreads, 0, stream>>>(a); break;
    case 64: gpack_rows<64><<<blocks, kRowThreads, 0, stream>>>(a); break;
    case 128: gpack_rows<128><<<blocks, kRowThreads, 0, stream>>>(a); break;
    case 256: gpack_rows<256><<<blocks, kRowThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_unpack_groups(const GroupLaunch& gl, const uint8_t* payload, uint16_t* k_cache, uint16_t* v_cache,
                                const int32_t* block_table, int32_t num_blocks, int32_t block_size,
                                uint32_t* status, hipStream_t stream) {
  GroupArgs a = group_args(gl);
  a.payload = const_cast<uint8_t*>(payload);
  a.status = status;
  a.block_table = block_table;
  a.num_blocks = num_blocks;
  a.block_size = block_size;
  gunpack_init<<<1, 64, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  gunpack_check<<<a.G + 1, kPrepThreads, 0, stream>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint64_t blocks = 2ull * a.L * a.H * static_cast<uint64_t>(a.nchunks);
  switch (a.d) {
    case 32: gunpack_rows<32><<<blocks, kRowThreads, 0, stream>>>(a, k_cache, v_cache); break;
    case 64: gunpack_rows<64><<<blocks, kRowThreads, 0, stream>>>(a, k_cache, v_cache); break;
    case 128: gunpack_rows<128><<<blocks, kRowThreads, 0, stream>>>(a, k_cache, v_cache); break;
    case 256: gunpack_rows<256><<<blocks, kRowThreads, 0, stream>>>(a, k_cache, v_cache); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace skv
