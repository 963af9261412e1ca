// Quantize-and-pack (Algorithm 1, transfer; "standard symmetric" quantizer of
// Sec. 8), batched over requests of different lengths.
//
// pack_prep (one workgroup per request) checks the tier map against the plan,
// then writes the header, the 2-bit tier map and the chunk index; pack_rows
// (one workgroup per 256-token chunk of one (layer, K/V, head) segment of one
// request) rebuilds its chunk's row offsets with a block scan, reads each row
// with 16-byte loads (d/8 lanes per row), takes the row's absmax with a DPP
// lane reduction, quantizes in registers and stores the row at its offset.
// A launch may cover a range of layers: the payload is layer-major, so the
// layers of a request can be packed (and sent) in pieces.
#include "device_util.h"
#include "row_codec.h"
#include "row_stream.h"
#include "row_variants.h"
#include "skv_internal.h"
#include "tier_groups.h"

namespace skv {
namespace {

constexpr int kPrepThreads = 1024;
constexpr int kMaxChunks = kMaxTokens / kChunkTokens;

// grid: one workgroup per request
__global__ __launch_bounds__(kPrepThreads) void pack_prep(const BatchArgs a) {
  __shared__ uint32_t s_chunk[kMaxChunks];  // per chunk: units | quant << 16
  __shared__ uint32_t s_meta[kMaxChunks];   // per chunk: V-side | K-side << 16 metadata bytes (variants)
  __shared__ uint32_t s_cnt[4];
  __shared__ uint32_t s_bad;
  __shared__ uint64_t s_scan[16];
  __shared__ uint64_t s_scan2[16];
  const ReqDesc& r = a.r[blockIdx.x];
  const uint8_t* __restrict__ tier = r.tier;
  uint8_t* __restrict__ payload = r.payload;
  const int n = r.n, nchunks = r.nchunks;
  const int tid = threadIdx.x;
  const int ngroups = (n + kGroupTokens - 1) / kGroupTokens;
  const bool variant = (a.q8 | a.q4) != 0;  // launch-uniform
  if (tid < 4) s_cnt[tid] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();

  // 1. tier counts and per-chunk sums (a chunk's 16 groups sit in 16 lanes).
  //    A pass takes two groups per thread, both loaded before either is
  //    tallied; the first pass's 2-bit map words stay in registers for step 4.
  uint32_t cnt[4] = {0, 0, 0, 0};
  bool bad = false;
  uint32_t map_first[2] = {0u, 0u};
  for (int base = 0; base < ngroups; base += 2 * kPrepThreads) {  // block-uniform trip count
    int gs[2];
    bool word[2];
    u32x4 w[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      gs[k] = base + k * kPrepThreads + tid;
      word[k] = gs[k] < ngroups && tier_group_is_word(tier, n, gs[k]);
      w[k] = word[k] ? *reinterpret_cast<const u32x4*>(tier + static_cast<size_t>(gs[k]) * kGroupTokens)
                     : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int g = gs[k];
      const TierGroup gi = word[k] ? group_from_tier_words(w[k])
                                   : g < ngroups ? group_from_bytes(tier, n, g) : empty_group();
#pragma unroll
      for (int i = 0; i < 4; ++i) cnt[i] += gi.count(i);
      bad |= gi.bad;
      const uint32_t u = sum16(gi.units), q = sum16(gi.quant);
      // a chunk's metadata is at most 256 rows x 64 bytes: 16 bits per side
      const uint32_t m = sum16(gi.count(kINT8) * a.e8 + gi.count(kINT4) * a.e4);
      const uint32_t mk = sum16(gi.count(kINT8) * a.ek8 + gi.count(kINT4) * a.ek4);
      if ((tid % kGroupsPerChunk) == 0 && g < ngroups) {
        s_chunk[g / kGroupsPerChunk] = u | (q << 16);
        s_meta[g / kGroupsPerChunk] = m | (mk << 16);
      }
      if (base == 0) map_first[k] = gi.map2;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (cnt[i]) atomicAdd(&s_cnt[i], cnt[i]);
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  const bool ok = !s_bad && s_cnt[0] == static_cast<uint32_t>(r.n_sink + r.n16) &&
                  s_cnt[1] == static_cast<uint32_t>(r.n8) && s_cnt[2] == static_cast<uint32_t>(r.n4) &&
                  s_cnt[3] == static_cast<uint32_t>(r.nd);
  const uint32_t status = ok ? 0u : static_cast<uint32_t>(SKV_ERR_INVALID_ARG);

  // 2. header (status recorded; the non-finite counter starts at zero)
  if (tid < 64) reinterpret_cast<uint32_t*>(payload)[tid] = tid == kHdrStatus ? status : header_word(a, r, tid);
  if (tid == 0 && r.status) *r.status = status;
  if (!ok) return;  // block-uniform

  // 3. chunk index: exclusive sums of row units and quantized rows at each
  //    chunk start; each thread owns a run of consecutive chunks
  const int per = (nchunks + kPrepThreads - 1) / kPrepThreads;
  const int c0 = min(nchunks, tid * per), c1 = min(nchunks, c0 + per);
  uint64_t run = 0;
  for (int c = c0; c < c1; ++c) run += (s_chunk[c] & 0xFFFFu) | (static_cast<uint64_t>(s_chunk[c] >> 16) << 32);
  const uint64_t ex = block_exclusive_scan_1024(run, s_scan);
  uint32_t ru = static_cast<uint32_t>(ex), rq = static_cast<uint32_t>(ex >> 32);
  uint32_t* cidx = reinterpret_cast<uint32_t*>(payload + r.chunkidx_off);
  if (!variant) {
    for (int c = c0; c < c1; ++c) {
      cidx[2 * c] = ru;
      cidx[2 * c + 1] = rq;
      ru += s_chunk[c] & 0xFFFFu;
      rq += s_chunk[c] >> 16;
    }
  } else {  // 16-byte entries {units, quantized rows, V-side metadata bytes, K-side metadata bytes or 0}
    const bool chan = ((a.q8 | a.q4) & kQuantChannel) != 0;
    uint64_t mrun = 0;
    for (int c = c0; c < c1; ++c) mrun += (s_meta[c] & 0xFFFFu) | (static_cast<uint64_t>(s_meta[c] >> 16) << 32);
    const uint64_t mex = block_exclusive_scan_1024(mrun, s_scan2);
    uint32_t rm = static_cast<uint32_t>(mex), rmk = static_cast<uint32_t>(mex >> 32);
    for (int c = c0; c < c1; ++c) {
      cidx[4 * c] = ru;
      cidx[4 * c + 1] = rq;
      cidx[4 * c + 2] = rm;
      cidx[4 * c + 3] = chan ? rmk : 0u;
      ru += s_chunk[c] & 0xFFFFu;
      rq += s_chunk[c] >> 16;
      rm += s_meta[c] & 0xFFFFu;
      rmk += s_meta[c] >> 16;
    }
  }
  const uint64_t entry = variant ? 16u : 8u;
  for (uint64_t b = r.chunkidx_off + entry * nchunks + 4ull * tid; b < r.layers_off; b += 4ull * kPrepThreads)
    *reinterpret_cast<uint32_t*>(payload + b) = 0u;

  // 4. the 2-bit tier map (4 bytes per group of 16 tokens), then its padding;
  //    up to two groups per thread the words are still in registers
  if (ngroups <= 2 * kPrepThreads) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int g = k * kPrepThreads + tid;
      if (g < ngroups) *reinterpret_cast<uint32_t*>(payload + 256 + 4ull * g) = map_first[k];
    }
  } else {
    for (int g = tid; g < ngroups; g += kPrepThreads)
      *reinterpret_cast<uint32_t*>(payload + 256 + 4ull * g) = group_from_bytes(tier, n, g).map2;
  }
  for (uint64_t b = 256 + 4ull * ngroups + 4ull * tid; b < r.chunkidx_off; b += 4ull * kPrepThreads)
    *reinterpret_cast<uint32_t*>(payload + b) = 0u;
}

// grid: sum over requests of nchunks * 2 * H * layer_count workgroups.
// VARIANT: some tier uses a quantizer variant (row_variants.h); CHAN: some
// tier has per-channel keys (its own instantiation, so the register budget of
// the other paths is unaffected).
template <int D, bool VARIANT, bool CHAN = false>
__global__ __launch_bounds__(kRowThreads) void pack_rows(const BatchArgs a) {
  __shared__ ChunkLds s;
  const uint64_t bid = blockIdx.x;
  const ReqDesc& r = a.r[request_of_block(a, bid)];
  uint8_t* __restrict__ payload = r.payload;
  const uint32_t* hdr = reinterpret_cast<const uint32_t*>(payload);

  const int n = r.n, H = a.H, nchunks = r.nchunks;
  // a launch has fewer than 2^32 workgroups: 32-bit index arithmetic
  const uint32_t local = static_cast<uint32_t>(bid - r.block_begin);
  const int chunk = static_cast<int>(local % static_cast<uint32_t>(nchunks));
  const int seg = static_cast<int>(local / static_cast<uint32_t>(nchunks));  // ((l - layer_begin) * 2 + kv) * H + h
  const int h = seg % H;
  const int kv = (seg / H) & 1;
  const int l = a.layer_begin + seg / (2 * H);
  const int t0 = chunk * kChunkTokens;
  const uint16_t* src = (kv ? r.v : r.k) + (static_cast<size_t>(l) * H + h) * static_cast<size_t>(n) * D;
  // default quantizer: the first rows are loaded before the status check and
  // the layout scan (the reads stay inside K/V whatever the status)
  constexpr int kRows = pack_rows_in_flight<D>();
  constexpr bool kNT = pack_nt_store<D>();
  RowBatch<D, kRows> first;
  if constexpr (!VARIANT) pack_first_batch<D, kRows>(first, src, r.tier, t0, n);
  if (hdr[kHdrStatus] != 0u) return;  // tier map off plan: nothing to pack
  // per-channel K tiers: their K rows carry no per-row metadata and use the
  // K-side metadata offsets of the chunk index
  const bool chan_k = CHAN && kv == 0;

  // row offsets of this chunk: chunk-index base + block exclusive scan
  const VarCfg var{a.q8, a.q4, kv == 0 ? a.ek8 : a.e8, kv == 0 ? a.ek4 : a.e4};
  {
    const int t = t0 + threadIdx.x;
    const int tr = t < n ? r.tier[t] : kDROP;
    const uint32_t* cidx = reinterpret_cast<const uint32_t*>(payload + r.chunkidx_off);
    if constexpr (VARIANT) chunk_layout_var<D>(s, tr, cidx + 4 * chunk, chan_k ? 3 : 2, var);
    else chunk_layout<D>(s, tr, cidx + 2 * chunk);
  }
  __syncthreads();

  uint8_t* lay = payload + r.layers_off + static_cast<uint64_t>(l) * r.layer_stride;
  uint8_t* dst = lay + r.scales_bytes + r.channel_bytes + static_cast<uint64_t>(kv * H + h) * r.seg_stride;
  uint8_t* meta = lay + (kv == 0 ? static_cast<uint64_t>(h) * r.seg_scale_bytes_k
                                 : static_cast<uint64_t>(H) * r.seg_scale_bytes_k + static_cast<uint64_t>(h) * r.seg_scale_bytes);
  uint32_t* nonfinite = reinterpret_cast<uint32_t*>(payload) + kHdrNonfinite;
  if constexpr (CHAN) {
    if (chan_k) {
      __shared__ __align__(16) ChanLds<D> c;
      uint8_t* blk = lay + r.scales_bytes + (static_cast<uint64_t>(h) * nchunks + chunk) * (a.cb8 + a.cb4);
      if constexpr (D <= 128) {  // the thread's rows fit in registers: one read of the chunk
        pack_chunk_chan<D, kNT>(s, c, src, dst, meta, nonfinite, t0, n, var, blk, blk + a.cb8);
      } else {
        channel_params<D>(s, c, src, t0, var, blk, blk + a.cb8);
        pack_chunk_var<D, SKV_VAR_ROWS_IN_FLIGHT, kNT, true>(s, &c, src, dst, meta, nonfinite, t0, n,
                                                                            var);
      }
    } else {
      pack_chunk_var<D, SKV_VAR_ROWS_IN_FLIGHT, kNT, false>(s, nullptr, src, dst, meta, nonfinite, t0, n,
                                                                           var);
    }
  } else if constexpr (VARIANT) {
    pack_chunk_var<D, SKV_VAR_ROWS_IN_FLIGHT, kNT, false>(s, nullptr, src, dst, meta, nonfinite, t0, n,
                                                                         var);
  } else {
    pack_chunk<D, kRows, kNT>(s, first, src, dst, reinterpret_cast<float*>(meta),
                                                              nonfinite, t0, n);
  }

  // padding: segment tail (last chunk), the layer's per-row metadata tail and
  // per-channel area tail
  if (chunk == nchunks - 1) {
    for (uint64_t b = r.seg_bytes + 16ull * threadIdx.x; b < r.seg_stride; b += 16ull * kRowThreads)
      st_nt16(dst + b, u32x4{0u, 0u, 0u, 0u});
  }
  if (chunk == 0 && kv == 0 && h == 0) {
    // every metadata entry is 2, 4 or 8 bytes, so the used sizes are only
    // 2-byte aligned (the K and V halves differ with per-channel tiers):
    // 16-bit stores end exactly at each section boundary
    const uint64_t used = static_cast<uint64_t>(H) * (r.seg_scale_bytes_k + r.seg_scale_bytes);
    for (uint64_t b = used + 2ull * threadIdx.x; b < r.scales_bytes; b += 2ull * kRowThreads)
      *reinterpret_cast<uint16_t*>(lay + b) = 0u;
    const uint64_t cused = static_cast<uint64_t>(H) * nchunks * (a.cb8 + a.cb4);
    for (uint64_t b = cused + 2ull * threadIdx.x; b < r.channel_bytes; b += 2ull * kRowThreads)
      *reinterpret_cast<uint16_t*>(lay + r.scales_bytes + b) = 0u;
  }
}

}  // namespace

hipError_t launch_pack(const BatchArgs& a, uint64_t rows, hipStream_t stream) {
  if (a.layer_begin == 0) {
    pack_prep<<<a.count, kPrepThreads, 0, stream>>>(a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const bool variant = (a.q8 | a.q4) != 0;
  const bool chan = ((a.q8 | a.q4) & kQuantChannel) != 0;
  switch (a.d * 4 + (chan ? 2 : variant ? 1 : 0)) {
    case 128: pack_rows<32, false><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 256: pack_rows<64, false><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 512: pack_rows<128, false><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 1024: pack_rows<256, false><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 129: pack_rows<32, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 257: pack_rows<64, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 513: pack_rows<128, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 1025: pack_rows<256, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 130: pack_rows<32, true, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 258: pack_rows<64, true, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 514: pack_rows<128, true, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    case 1026: pack_rows<256, true, true><<<rows, kRowThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace skv
