// Quantize-and-pack (Algorithm 1 step 4; "standard symmetric" quantizer of
// Sec. 8) and the shared tier-map helpers.
//
// pack_prep (one workgroup) checks the tier map against the plan, then writes
// the header, the 2-bit tier map and the chunk index; pack_rows (one
// workgroup per 256-token chunk of one (layer, K/V, head) segment) rebuilds
// its chunk's row offsets with a block scan, reads each row with 16-byte
// loads (d/8 lanes per row), takes the row's absmax with a DPP lane
// reduction, quantizes in registers and stores the row at its offset.
#include "device_util.h"
#include "skv_internal.h"
#include "tier_groups.h"

namespace skv {
namespace {

// Build-time tuning knobs (defaults are the measured best on MI355X).
#ifndef SKV_PACK_ROWS_IN_FLIGHT
#define SKV_PACK_ROWS_IN_FLIGHT 4
#endif
#ifndef SKV_PACK_NT_STORE
#define SKV_PACK_NT_STORE 1
#endif

constexpr int kPrepThreads = 1024;
constexpr int kRowThreads = 256;  // == kChunkTokens: one token per thread in the scan
constexpr int kMaxChunks = kMaxTokens / kChunkTokens;
static_assert(kRowThreads == kChunkTokens, "one scan slot per token of a chunk");

// Header words that pack fills in at run time.
constexpr int kHdrNonfinite = 144 / 4;
constexpr int kHdrStatus = 148 / 4;

__global__ __launch_bounds__(kPrepThreads) void pack_prep(const uint8_t* __restrict__ tier, int n,
                                                          int nchunks, int want16, int want8,
                                                          int want4, int wantd, HeaderImage hdr,
                                                          uint8_t* __restrict__ payload,
                                                          uint64_t tiermap_off,
                                                          uint64_t chunkidx_off,
                                                          uint64_t layers_off,
                                                          uint32_t* dev_status) {
  __shared__ uint32_t s_chunk[kMaxChunks];  // per chunk: units | quant << 16
  __shared__ uint32_t s_cnt[4];
  __shared__ uint32_t s_bad;
  __shared__ uint64_t s_scan[16];
  const int tid = threadIdx.x;
  const int ngroups = (n + kGroupTokens - 1) / kGroupTokens;
  if (tid < 4) s_cnt[tid] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();

  // 1. tier counts and per-chunk sums (a chunk's 16 groups sit in 16 lanes)
  uint32_t cnt[4] = {0, 0, 0, 0};
  bool bad = false;
  for (int base = 0; base < ngroups; base += kPrepThreads) {  // block-uniform trip count
    const int g = base + tid;
    const TierGroup gi = g < ngroups ? group_from_bytes(tier, n, g) : empty_group();
#pragma unroll
    for (int i = 0; i < 4; ++i) cnt[i] += gi.cnt[i];
    bad |= gi.bad;
    const uint32_t u = sum16(gi.units), q = sum16(gi.quant);
    if ((tid % kGroupsPerChunk) == 0 && g < ngroups) s_chunk[g / kGroupsPerChunk] = u | (q << 16);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (cnt[i]) atomicAdd(&s_cnt[i], cnt[i]);
  if (bad) atomicOr(&s_bad, 1u);
  __syncthreads();
  const bool ok = !s_bad && s_cnt[0] == static_cast<uint32_t>(want16) &&
                  s_cnt[1] == static_cast<uint32_t>(want8) &&
                  s_cnt[2] == static_cast<uint32_t>(want4) && s_cnt[3] == static_cast<uint32_t>(wantd);
  const uint32_t status = ok ? 0u : static_cast<uint32_t>(SKV_ERR_INVALID_ARG);

  // 2. header (status recorded; the non-finite counter starts at zero)
  if (tid < 64) {
    uint32_t w = hdr.w[tid];
    if (tid == kHdrStatus) w = status;
    if (tid == kHdrNonfinite) w = 0;
    reinterpret_cast<uint32_t*>(payload)[tid] = w;
  }
  if (tid == 0 && dev_status) *dev_status = status;
  if (!ok) return;  // block-uniform

  // 3. chunk index: exclusive sums of row units and quantized rows at each
  //    chunk start; each thread owns a run of consecutive chunks
  const int per = (nchunks + kPrepThreads - 1) / kPrepThreads;
  const int c0 = min(nchunks, tid * per), c1 = min(nchunks, c0 + per);
  uint64_t run = 0;
  for (int c = c0; c < c1; ++c) run += (s_chunk[c] & 0xFFFFu) | (static_cast<uint64_t>(s_chunk[c] >> 16) << 32);
  const uint64_t ex = block_exclusive_scan_1024(run, s_scan);
  uint32_t ru = static_cast<uint32_t>(ex), rq = static_cast<uint32_t>(ex >> 32);
  uint32_t* cidx = reinterpret_cast<uint32_t*>(payload + chunkidx_off);
  for (int c = c0; c < c1; ++c) {
    cidx[2 * c] = ru;
    cidx[2 * c + 1] = rq;
    ru += s_chunk[c] & 0xFFFFu;
    rq += s_chunk[c] >> 16;
  }
  for (uint64_t b = chunkidx_off + 8ull * nchunks + 4ull * tid; b < layers_off; b += 4ull * kPrepThreads)
    *reinterpret_cast<uint32_t*>(payload + b) = 0u;

  // 4. the 2-bit tier map (4 bytes per group of 16 tokens), then its padding
  for (int g = tid; g < ngroups; g += kPrepThreads)
    *reinterpret_cast<uint32_t*>(payload + tiermap_off + 4ull * g) = group_from_bytes(tier, n, g).map2;
  for (uint64_t b = tiermap_off + 4ull * ngroups + 4ull * tid; b < chunkidx_off; b += 4ull * kPrepThreads)
    *reinterpret_cast<uint32_t*>(payload + b) = 0u;
}

template <int D>
__global__ __launch_bounds__(kRowThreads) void pack_rows(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, const uint8_t* __restrict__ tier,
    uint8_t* __restrict__ payload, int n, int H, int nchunks, int64_t nq, uint64_t chunkidx_off,
    uint64_t layers_off, uint64_t seg_bytes, uint64_t seg_stride, uint64_t scales_bytes,
    uint64_t layer_stride) {
  constexpr int LPR = D / 8;                // lanes per row, 16 bytes each
  constexpr int RPI = kRowThreads / LPR;    // rows per block-wide iteration
  constexpr int ITERS = kChunkTokens / RPI;
  constexpr int U = ITERS < SKV_PACK_ROWS_IN_FLIGHT ? ITERS : SKV_PACK_ROWS_IN_FLIGHT;  // rows in flight per thread
  __shared__ uint8_t s_tier[kChunkTokens];
  __shared__ uint32_t s_off[kChunkTokens];  // byte offset of the row inside its segment
  __shared__ uint32_t s_q[kChunkTokens];    // index of the row's scale
  __shared__ uint32_t s_scan[4];

  const uint32_t* hdr = reinterpret_cast<const uint32_t*>(payload);
  if (hdr[kHdrStatus] != 0u) return;  // tier map off plan: nothing to pack

  const int chunk = blockIdx.x % nchunks;
  const int seg = blockIdx.x / nchunks;  // (l * 2 + kv) * H + h
  const int h = seg % H;
  const int kv = (seg / H) & 1;
  const int l = seg / (2 * H);
  const int t0 = chunk * kChunkTokens;

  // row offsets of this chunk: chunk-index base + block exclusive scan
  {
    const int t = t0 + threadIdx.x;
    const int tr = t < n ? tier[t] : kDROP;
    const uint32_t packed = tier_units(tr) | (tier_quant(tr) << 16);
    uint32_t total;
    const uint32_t ex = block_exclusive_scan_256(packed, s_scan, &total);
    const uint32_t* cidx = reinterpret_cast<const uint32_t*>(payload + chunkidx_off) + 2 * chunk;
    s_tier[threadIdx.x] = static_cast<uint8_t>(tr);
    s_off[threadIdx.x] = (cidx[0] + (ex & 0xFFFFu)) * static_cast<uint32_t>(D / 2);
    s_q[threadIdx.x] = cidx[1] + (ex >> 16);
  }
  __syncthreads();

  const uint16_t* src = (kv ? v : k) + (static_cast<size_t>(l) * H + h) * static_cast<size_t>(n) * D;
  uint8_t* lay = payload + layers_off + static_cast<uint64_t>(l) * layer_stride;
  uint8_t* dst = lay + scales_bytes + static_cast<uint64_t>(kv * H + h) * seg_stride;
  float* scales = reinterpret_cast<float*>(lay) + static_cast<uint64_t>(kv * H + h) * nq;
  uint32_t* nonfinite = reinterpret_cast<uint32_t*>(payload) + kHdrNonfinite;

  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int t = t0 + r;
      x[u] = u32x4{0u, 0u, 0u, 0u};
      if (t < n && s_tier[r] != kDROP) x[u] = ld_nt16(src + static_cast<size_t>(t) * D + lane * 8);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int tr = s_tier[r];
      const uint32_t amax = group_max<LPR>(absmax_bits8(x[u]));  // all lanes take part
      if (tr == kFP16) {
        store16<SKV_PACK_NT_STORE>(dst + s_off[r] + lane * 16, x[u]);
      } else if (tr == kINT8 || tr == kINT4) {
        const int Q = tr == kINT8 ? 127 : 7;
        const float Qf = static_cast<float>(Q);
        float scale;
        int32_t lo = 0x4B400000, hi = 0x4B400000;  // clamp window around 1.5 * 2^23
        uint32_t codes[8];
        if (amax >= 0x7C00u) {  // an infinity or NaN in the row
          scale = __builtin_bit_cast(float, 0x7FC00000u);
#pragma unroll
          for (int i = 0; i < 8; ++i) codes[i] = 0;
          if (lane == 0) atomicAdd(nonfinite, 1u);
        } else if (amax == 0u) {
          scale = 0.0f;
#pragma unroll
          for (int i = 0; i < 8; ++i) codes[i] = 0;
        } else {
          const float a = half_lo(amax);
          scale = a / Qf;          // correctly rounded binary32 division
          const float rcp = Qf / a;
          lo -= Q;
          hi += Q;
          const uint32_t w[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // RN32(x * r), then round to an integer (nearest-even) by adding
            // 1.5 * 2^23: the low mantissa bits of the sum are the code
            const float y0 = half_lo(w[i]) * rcp;
            const float y1 = half_hi(w[i]) * rcp;
            const int32_t b0 = __builtin_bit_cast(int32_t, y0 + 12582912.0f);
            const int32_t b1 = __builtin_bit_cast(int32_t, y1 + 12582912.0f);
            codes[2 * i] = static_cast<uint32_t>(min(max(b0, lo), hi));
            codes[2 * i + 1] = static_cast<uint32_t>(min(max(b1, lo), hi));
          }
        }
        uint8_t* row = dst + s_off[r];
        if (tr == kINT8) {
          u32x2 out;
          out.x = (codes[0] & 0xFFu) | ((codes[1] & 0xFFu) << 8) | ((codes[2] & 0xFFu) << 16) | (codes[3] << 24);
          out.y = (codes[4] & 0xFFu) | ((codes[5] & 0xFFu) << 8) | ((codes[6] & 0xFFu) << 16) | (codes[7] << 24);
          store8<SKV_PACK_NT_STORE>(row + lane * 8, out);
        } else {
          uint32_t out = 0;
#pragma unroll
          for (int i = 0; i < 8; ++i) out |= (codes[i] & 0xFu) << (4 * i);
          store4<SKV_PACK_NT_STORE>(row + lane * 4, out);
        }
        if (lane == 0) scales[s_q[r]] = scale;
      }
    }
  }

  // padding: segment tail (last chunk) and the layer's scale-section tail
  if (chunk == nchunks - 1) {
    for (uint64_t b = seg_bytes + 16ull * threadIdx.x; b < seg_stride; b += 16ull * kRowThreads)
      st_nt16(dst + b, u32x4{0u, 0u, 0u, 0u});
  }
  if (chunk == 0 && kv == 0 && h == 0) {
    const uint64_t used = 2ull * H * static_cast<uint64_t>(nq) * 4u;
    for (uint64_t b = used + 4ull * threadIdx.x; b < scales_bytes; b += 4ull * kRowThreads)
      *reinterpret_cast<uint32_t*>(lay + b) = 0u;
  }
}

}  // namespace

hipError_t launch_pack(const Geometry& g, const HeaderImage& hdr, const uint16_t* k,
                       const uint16_t* v, const uint8_t* tier, uint8_t* payload,
                       uint32_t* dev_status, hipStream_t stream) {
  pack_prep<<<1, kPrepThreads, 0, stream>>>(tier, g.n, static_cast<int>(g.nchunks), g.n_sink + g.n16,
                                            g.n8, g.n4, g.nd, hdr, payload, g.tiermap_off,
                                            g.chunkidx_off, g.layers_off, dev_status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint64_t blocks = static_cast<uint64_t>(g.nchunks) * 2u * g.L * g.H;
  const int nch = static_cast<int>(g.nchunks);
#define SKV_PACK_ARGS k, v, tier, payload, g.n, g.H, nch, g.nq, g.chunkidx_off, g.layers_off, \
                      g.seg_bytes, g.seg_stride, g.scales_bytes, g.layer_stride
  switch (g.d) {
    case 32: pack_rows<32><<<blocks, kRowThreads, 0, stream>>>(SKV_PACK_ARGS); break;
    case 64: pack_rows<64><<<blocks, kRowThreads, 0, stream>>>(SKV_PACK_ARGS); break;
    case 128: pack_rows<128><<<blocks, kRowThreads, 0, stream>>>(SKV_PACK_ARGS); break;
    case 256: pack_rows<256><<<blocks, kRowThreads, 0, stream>>>(SKV_PACK_ARGS); break;
    default: return hipErrorInvalidValue;
  }
#undef SKV_PACK_ARGS
  return hipGetLastError();
}

}  // namespace skv
