// Decode-side dequantization into the fp16 paged cache (Sec. 4.2: only a
// lightweight per-tier dequantization runs after receipt).
//
// unpack_check (one workgroup per request) compares the payload header with
// the one the configuration implies, recounts the 2-bit tier map, re-derives
// the chunk index and range-checks the block table; it writes the verdict to
// the request's status word.  unpack_rows (one workgroup per 256-token chunk
// of one (layer, K/V, head) segment of one request) does nothing unless the
// verdict is 0; it rebuilds the chunk's row offsets with a block scan, loads
// each row at its tier's width, dequantizes in registers
// (RN16(RN32(code * scale))) and writes 16 bytes per lane into the token's
// paged slot.  Requests of a launch share the paged cache (each has its own
// block table); a launch may cover a range of layers.
#include "device_util.h"
#include "row_codec.h"
#include "row_stream.h"
#include "row_variants.h"
#include "skv_internal.h"
#include "tier_groups.h"

namespace skv {
namespace {

constexpr int kCheckThreads = 1024;
constexpr int kMaxChunks = kMaxTokens / kChunkTokens;

// grid: one workgroup per request
__global__ __launch_bounds__(kCheckThreads) void unpack_check(const BatchArgs a, int num_blocks,
                                                              int block_size) {
  __shared__ uint32_t s_chunk[kMaxChunks];
  __shared__ uint32_t s_meta[kMaxChunks];  // per chunk: V-side | K-side << 16 metadata bytes (variants)
  __shared__ uint32_t s_cnt[4];
  __shared__ uint32_t s_bad;
  __shared__ uint64_t s_scan[16];
  __shared__ uint64_t s_scan2[16];
  const ReqDesc& r = a.r[blockIdx.x];
  const bool variant = (a.q8 | a.q4) != 0;  // launch-uniform
  const uint8_t* __restrict__ payload = r.payload;
  const int n = r.n, nchunks = r.nchunks;
  const int tid = threadIdx.x;
  const int nbt = (n + block_size - 1) / block_size;
  const int ngroups = (n + kGroupTokens - 1) / kGroupTokens;
  const uint8_t* map = payload + 256;
  const uint32_t* cidx = reinterpret_cast<const uint32_t*>(payload + r.chunkidx_off);
  const int entry = variant ? 4 : 2;  // chunk-index words per chunk
  const int per = (nchunks + kCheckThreads - 1) / kCheckThreads;
  const int c0 = min(nchunks, tid * per), c1 = min(nchunks, c0 + per);
  // The first pass of every check loads up front, so that one memory latency
  // covers them all: the header word, two block-table entries, two map words
  // and the first chunk-index entry of this thread.  Every address lies in
  // the payload's metadata or the block table whatever their contents.
  const uint32_t hword = tid < 64 ? reinterpret_cast<const uint32_t*>(payload)[tid] : 0u;
  int bt_first[2];
  uint32_t map_first[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = k * kCheckThreads + tid;
    bt_first[k] = i < nbt ? r.block_table[i] : 0;
    map_first[k] = i < ngroups ? reinterpret_cast<const uint32_t*>(map)[i] : 0u;
  }
  uint32_t cidx_first[4] = {0u, 0u, 0u, 0u};
  if (c0 < c1) {
#pragma unroll
    for (int w = 0; w < 4; ++w)
      if (w < entry) cidx_first[w] = cidx[entry * c0 + w];
  }
  if (tid < 4) s_cnt[tid] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  bool bad = false;
  // header: every word but the non-finite row counter must match
  if (tid < 64 && tid != kHdrNonfinite) bad |= hword != header_word(a, r, tid);
  // block table entries in range
#pragma unroll
  for (int k = 0; k < 2; ++k)
    if (k * kCheckThreads + tid < nbt) bad |= bt_first[k] < 0 || bt_first[k] >= num_blocks;
  for (int i = 2 * kCheckThreads + tid; i < nbt; i += kCheckThreads) {
    const int b = r.block_table[i];
    bad |= b < 0 || b >= num_blocks;
  }
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  if (s_bad) {  // header or table wrong: do not interpret the rest
    if (tid == 0) *r.status = static_cast<uint32_t>(SKV_ERR_FORMAT);
    return;
  }
  // tier counts and chunk sums from the 2-bit map (a chunk's 16 groups sit
  // in 16 lanes)
  uint32_t cnt[4] = {0, 0, 0, 0};
  for (int base = 0; base < ngroups; base += kCheckThreads) {  // block-uniform trip count
    const int g = base + tid;
    const int pass = base / kCheckThreads;
    TierGroup gi = empty_group();
    if (g < ngroups) gi = pass < 2 ? group_from_map_word(map_first[pass & 1], n, g) : group_from_map(map, n, g);
#pragma unroll
    for (int i = 0; i < 4; ++i) cnt[i] += gi.count(i);
    const uint32_t u = sum16(gi.units), q = sum16(gi.quant);
    const uint32_t m = sum16(gi.count(kINT8) * a.e8 + gi.count(kINT4) * a.e4);
    const uint32_t mk = sum16(gi.count(kINT8) * a.ek8 + gi.count(kINT4) * a.ek4);
    if ((tid % kGroupsPerChunk) == 0 && g < ngroups) {
      s_chunk[g / kGroupsPerChunk] = u | (q << 16);
      s_meta[g / kGroupsPerChunk] = m | (mk << 16);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (cnt[i]) atomicAdd(&s_cnt[i], cnt[i]);
  __syncthreads();
  bad = s_cnt[0] != static_cast<uint32_t>(r.n_sink + r.n16) || s_cnt[1] != static_cast<uint32_t>(r.n8) ||
        s_cnt[2] != static_cast<uint32_t>(r.n4) || s_cnt[3] != static_cast<uint32_t>(r.nd);
  // chunk index must equal the running sums
  uint64_t run = 0;
  for (int c = c0; c < c1; ++c) run += (s_chunk[c] & 0xFFFFu) | (static_cast<uint64_t>(s_chunk[c] >> 16) << 32);
  const uint64_t ex = block_exclusive_scan_1024(run, s_scan);
  uint32_t ru = static_cast<uint32_t>(ex), rq = static_cast<uint32_t>(ex >> 32);
  if (!variant) {
    for (int c = c0; c < c1; ++c) {
      const uint32_t w0 = c == c0 ? cidx_first[0] : cidx[2 * c], w1 = c == c0 ? cidx_first[1] : cidx[2 * c + 1];
      bad |= w0 != ru || w1 != rq;
      ru += s_chunk[c] & 0xFFFFu;
      rq += s_chunk[c] >> 16;
    }
  } else {
    const bool chan = ((a.q8 | a.q4) & kQuantChannel) != 0;
    uint64_t mrun = 0;
    for (int c = c0; c < c1; ++c) mrun += (s_meta[c] & 0xFFFFu) | (static_cast<uint64_t>(s_meta[c] >> 16) << 32);
    const uint64_t mex = block_exclusive_scan_1024(mrun, s_scan2);
    uint32_t rm = static_cast<uint32_t>(mex), rmk = static_cast<uint32_t>(mex >> 32);
    for (int c = c0; c < c1; ++c) {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = c == c0 ? cidx_first[i] : cidx[4 * c + i];
      bad |= w[0] != ru || w[1] != rq || w[2] != rm || w[3] != (chan ? rmk : 0u);
      ru += s_chunk[c] & 0xFFFFu;
      rq += s_chunk[c] >> 16;
      rm += s_meta[c] & 0xFFFFu;
      rmk += s_meta[c] >> 16;
    }
  }
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  if (tid == 0) *r.status = s_bad ? static_cast<uint32_t>(SKV_ERR_FORMAT) : 0u;
}

// grid: sum over requests of nchunks * 2 * H * layer_count workgroups.
// VARIANT: some tier uses a quantizer variant (row_variants.h); CHAN: some
// tier has per-channel keys (its own instantiation).
template <int D, bool VARIANT, bool CHAN = false>
__global__ __launch_bounds__(kRowThreads) void unpack_rows(const BatchArgs a, uint16_t* __restrict__ k_cache,
                                                           uint16_t* __restrict__ v_cache, int num_blocks,
                                                           int block_size) {
  __shared__ ChunkLds s;
  const uint64_t bid = blockIdx.x;
  const ReqDesc& r = a.r[request_of_block(a, bid)];
  if (*r.status != 0u) return;  // payload rejected: write nothing

  const uint8_t* __restrict__ payload = r.payload;
  const int n = r.n, H = a.H, nchunks = r.nchunks;
  // a launch has fewer than 2^32 workgroups: 32-bit index arithmetic
  const uint32_t local = static_cast<uint32_t>(bid - r.block_begin);
  const int chunk = static_cast<int>(local % static_cast<uint32_t>(nchunks));
  const int seg = static_cast<int>(local / static_cast<uint32_t>(nchunks));
  const int h = seg % H;
  const int kv = (seg / H) & 1;
  const int l = a.layer_begin + seg / (2 * H);
  const int t0 = chunk * kChunkTokens;
  // per-channel K tiers: K rows of those tiers decode with the chunk's channel
  // entries and use the K-side metadata offsets of the chunk index
  const bool chan_k = CHAN && kv == 0;
  const VarCfg var{a.q8, a.q4, kv == 0 ? a.ek8 : a.e8, kv == 0 ? a.ek4 : a.e4};
  {
    const int t = t0 + threadIdx.x;
    int tr = kAbsent;
    uint32_t pos = 0;
    if (t < n) {
      tr = (payload[256 + (t >> 2)] >> (2 * (t & 3))) & 3;
      pos = static_cast<uint32_t>(r.block_table[t / block_size]) * static_cast<uint32_t>(block_size) +
            static_cast<uint32_t>(t % block_size);
    }
    const uint32_t* cidx = reinterpret_cast<const uint32_t*>(payload + r.chunkidx_off);
    if constexpr (VARIANT) {
      chunk_layout_var<D>(s, tr, cidx + 4 * chunk, chan_k ? 3 : 2, var);
    } else {
      chunk_layout<D>(s, tr, cidx + 2 * chunk);
      // the layer's scales of this segment (descriptor 0: one fp32 per quantized row)
      const uint8_t* lay0 = payload + r.layers_off + static_cast<uint64_t>(l) * r.layer_stride;
      stage_scale(s, tr, reinterpret_cast<const float*>(lay0 + static_cast<uint64_t>(kv * H + h) * r.seg_scale_bytes));
    }
    s.pos[threadIdx.x] = pos;
  }
  __syncthreads();

  const uint8_t* lay = payload + r.layers_off + static_cast<uint64_t>(l) * r.layer_stride;
  const uint8_t* src = lay + r.scales_bytes + r.channel_bytes + static_cast<uint64_t>(kv * H + h) * r.seg_stride;
  const uint8_t* meta = lay + (kv == 0 ? static_cast<uint64_t>(h) * r.seg_scale_bytes_k
                                       : static_cast<uint64_t>(H) * r.seg_scale_bytes_k +
                                             static_cast<uint64_t>(h) * r.seg_scale_bytes);
  uint16_t* cache = (kv ? v_cache : k_cache) + static_cast<size_t>(l) * num_blocks * block_size * H * D +
                    static_cast<size_t>(h) * D;
  if constexpr (CHAN) {
    if (chan_k) {
      __shared__ ChanDecLds<D> c;
      const uint8_t* blk = lay + r.scales_bytes + (static_cast<uint64_t>(h) * nchunks + chunk) * (a.cb8 + a.cb4);
      const bool finite = load_channel_params<D>(c, blk, blk + a.cb8, var);
      unpack_chunk_var<D, SKV_VAR_ROWS_IN_FLIGHT, unpack_nt_store<D>(), true>(s, &c, finite, src, meta, cache, H,
                                                                                 var);
    } else {
      unpack_chunk_var<D, SKV_VAR_ROWS_IN_FLIGHT, unpack_nt_store<D>(), false>(s, nullptr, true, src, meta, cache, H,
                                                                                  var);
    }
  } else if constexpr (VARIANT) {
    unpack_chunk_var<D, SKV_VAR_ROWS_IN_FLIGHT, unpack_nt_store<D>(), false>(s, nullptr, true, src, meta, cache, H,
                                                                                var);
  } else {
    unpack_chunk<D, unpack_rows_in_flight<D>(), unpack_nt_store<D>()>(s, src, cache, H);
  }
}

}  // namespace

hipError_t launch_unpack(const BatchArgs& a, uint64_t rows, uint16_t* k_cache, uint16_t* v_cache,
                         int32_t num_blocks, int32_t block_size, hipStream_t stream) {
  if (a.layer_begin == 0) {
    unpack_check<<<a.count, kCheckThreads, 0, stream>>>(a, num_blocks, block_size);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const bool variant = (a.q8 | a.q4) != 0;
  const bool chan = ((a.q8 | a.q4) & kQuantChannel) != 0;
#define SKV_UNPACK_LAUNCH(D, V, C) \
  unpack_rows<D, V, C><<<rows, kRowThreads, 0, stream>>>(a, k_cache, v_cache, num_blocks, block_size)
  switch (a.d * 4 + (chan ? 2 : variant ? 1 : 0)) {
    case 128: SKV_UNPACK_LAUNCH(32, false, false); break;
    case 256: SKV_UNPACK_LAUNCH(64, false, false); break;
    case 512: SKV_UNPACK_LAUNCH(128, false, false); break;
    case 1024: SKV_UNPACK_LAUNCH(256, false, false); break;
    case 129: SKV_UNPACK_LAUNCH(32, true, false); break;
    case 257: SKV_UNPACK_LAUNCH(64, true, false); break;
    case 513: SKV_UNPACK_LAUNCH(128, true, false); break;
    case 1025: SKV_UNPACK_LAUNCH(256, true, false); break;
    case 130: SKV_UNPACK_LAUNCH(32, true, true); break;
    case 258: SKV_UNPACK_LAUNCH(64, true, true); break;
    case 514: SKV_UNPACK_LAUNCH(128, true, true); break;
    case 1026: SKV_UNPACK_LAUNCH(256, true, true); break;
    default: return hipErrorInvalidValue;
  }
#undef SKV_UNPACK_LAUNCH
  return hipGetLastError();
}

}  // namespace skv
