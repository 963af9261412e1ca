// The per-chunk bodies of the row kernels, shared by the per-token codec
// (pack.hip, unpack.hip) and the grouped codec (groups.hip): a workgroup of
// 256 threads owns one 256-token chunk of one (layer, K/V, head) segment.
//   chunk_layout_*  give every token of the chunk its tier, the byte offset
//                   of its row inside the segment and the index of its scale
//                   (chunk-index base + a block scan of the row widths);
//   pack_first_batch / pack_chunk
//                   read the chunk's rows (d/8 lanes per row, 16 bytes each,
//                   several rows in flight; the first batch is issued before
//                   the layout scan), quantize and store them;
//   unpack_chunk    loads the rows at their tier widths, dequantizes and
//                   writes them into their paged slots.
#pragma once

#include "device_util.h"
#include "row_codec.h"
#include "skv_internal.h"

namespace skv {

// Tuning of the default-quantizer row kernels, per head dim (measured on
// MI355X; the macros override them for sweeps): rows whose loads each thread
// issues before it processes any of them, and non-temporal or default-policy
// stores.  More rows in flight cover HBM latency (8 rows: pack 6.7 % and
// unpack 1 % faster than 4 at d = 128); at d = 256 a thread's quantized rows
// are narrow (4 or 8 bytes per lane), so unpack keeps 16 in flight.  Both
// kernels store non-temporally: default-policy stores leave up to the caches'
// size of dirty lines behind when the kernel ends, and the kernels after it
// pay their write-back (pack + unpack back to back: 2.7 % slower at d = 128,
// 1.7-2.9 % at d = 256).
#ifndef SKV_PACK_ROWS_IN_FLIGHT
#define SKV_PACK_ROWS_IN_FLIGHT 8
#endif
#ifndef SKV_PACK_ROWS_IN_FLIGHT_D256
#define SKV_PACK_ROWS_IN_FLIGHT_D256 8
#endif
#ifndef SKV_PACK_NT_STORE
#define SKV_PACK_NT_STORE 1
#endif
#ifndef SKV_UNPACK_ROWS_IN_FLIGHT
#define SKV_UNPACK_ROWS_IN_FLIGHT 8
#endif
#ifndef SKV_UNPACK_ROWS_IN_FLIGHT_D256
#define SKV_UNPACK_ROWS_IN_FLIGHT_D256 16
#endif
#ifndef SKV_UNPACK_NT_STORE
#define SKV_UNPACK_NT_STORE 1
#endif
// The quantizer-variant kernels hold more per row (group metadata): 4 rows.
#ifndef SKV_VAR_ROWS_IN_FLIGHT
#define SKV_VAR_ROWS_IN_FLIGHT 4
#endif

template <int D>
constexpr int pack_rows_in_flight() { return D >= 256 ? SKV_PACK_ROWS_IN_FLIGHT_D256 : SKV_PACK_ROWS_IN_FLIGHT; }
template <int D>
constexpr bool pack_nt_store() { return SKV_PACK_NT_STORE != 0; }
template <int D>
constexpr int unpack_rows_in_flight() { return D >= 256 ? SKV_UNPACK_ROWS_IN_FLIGHT_D256 : SKV_UNPACK_ROWS_IN_FLIGHT; }
template <int D>
constexpr bool unpack_nt_store() { return SKV_UNPACK_NT_STORE != 0; }

constexpr int kRowThreads = 256;  // == kChunkTokens: one token per thread in the scan
static_assert(kRowThreads == kChunkTokens, "one scan slot per token of a chunk");
constexpr int kAbsent = 4;  // unpack: a slot past the end of the request

struct ChunkLds {
  uint8_t tier[kChunkTokens];
  uint32_t off[kChunkTokens];  // byte offset of the row inside its segment
  uint32_t q[kChunkTokens];    // index of the row's scale
  uint32_t pos[kChunkTokens];  // unpack: physical block * block_size + slot
  float scale[kChunkTokens];   // unpack: the row's scale (quantized rows)
  uint32_t scan[4];
};

// Unpack: stages the scale of the chunk's row of this thread's scan slot
// (tier code tr) in shared memory, read with one load per quantized row
// rather than one per lane of each row.  The scale index is this thread's
// own s.q entry; the caller's barrier after chunk_layout publishes it.
__device__ __forceinline__ void stage_scale(ChunkLds& s, int tr, const float* __restrict__ scales) {
  s.scale[threadIdx.x] = (tr == kINT8 || tr == kINT4) ? scales[s.q[threadIdx.x]] : 0.0f;
}

// Fills s.tier/off/q of the chunk starting at t0 from the token's tier code
// tr (kDROP for pack slots past n, kAbsent for unpack slots past n) and the
// chunk's index entry {units, quantized rows}.  Contains __syncthreads().
template <int D>
__device__ __forceinline__ void chunk_layout(ChunkLds& s, int tr, const uint32_t* cidx_entry) {
  const uint32_t packed = (tr == kAbsent) ? 0u : (tier_units(tr) | (tier_quant(tr) << 16));
  uint32_t total;
  const uint32_t ex = block_exclusive_scan_256(packed, s.scan, &total);
  s.tier[threadIdx.x] = static_cast<uint8_t>(tr);
  s.off[threadIdx.x] = (cidx_entry[0] + (ex & 0xFFFFu)) * static_cast<uint32_t>(D / 2);
  s.q[threadIdx.x] = cidx_entry[1] + (ex >> 16);
}

// The rows a thread quantizes in one batch: lanes per row (16 bytes each),
// rows per block-wide iteration, iterations per chunk, rows in flight.
template <int D, int ROWS_IN_FLIGHT>
struct RowBatch {
  static constexpr int LPR = D / 8;
  static constexpr int RPI = kRowThreads / LPR;
  static constexpr int ITERS = kChunkTokens / RPI;
  static constexpr int U = ITERS < ROWS_IN_FLIGHT ? ITERS : ROWS_IN_FLIGHT;
  static_assert(ITERS % U == 0, "rows in flight must divide a thread's rows of the chunk");
  u32x4 x[U];
};

// Issues the loads of a thread's first batch of rows of the chunk at t0,
// taking their tiers from the caller's tier map (tier[t], t < n) rather than
// from the chunk layout: the loads are then in flight while the layout is
// scanned.  Reads only rows t < n of tiers other than DROP.
template <int D, int ROWS_IN_FLIGHT>
__device__ __forceinline__ void pack_first_batch(RowBatch<D, ROWS_IN_FLIGHT>& b, const uint16_t* __restrict__ src,
                                                 const uint8_t* __restrict__ tier, int t0, int n) {
  using B = RowBatch<D, ROWS_IN_FLIGHT>;
  const int lane = threadIdx.x % B::LPR;
  const int rsub = threadIdx.x / B::LPR;
#pragma unroll
  for (int u = 0; u < B::U; ++u) {
    const int t = t0 + u * B::RPI + rsub;
    b.x[u] = u32x4{0u, 0u, 0u, 0u};
    if (t < n && tier[t] != kDROP) b.x[u] = ld_nt16(src + static_cast<size_t>(t) * D + lane * 8);
  }
}

// Quantizes and stores the rows of one chunk.  first: the thread's first
// batch (pack_first_batch); src: the segment's plane [n][D]; dst: the
// segment's rows; scales: the segment's scales.
template <int D, int ROWS_IN_FLIGHT, bool NT>
__device__ __forceinline__ void pack_chunk(const ChunkLds& s, const RowBatch<D, ROWS_IN_FLIGHT>& first,
                                           const uint16_t* __restrict__ src, uint8_t* __restrict__ dst,
                                           float* __restrict__ scales, uint32_t* nonfinite, int t0, int n) {
  using B = RowBatch<D, ROWS_IN_FLIGHT>;
  constexpr int LPR = B::LPR, RPI = B::RPI, ITERS = B::ITERS, U = B::U;
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = (it + u) * RPI + rsub;
      const int t = t0 + row;
      if (it == 0) {
        x[u] = first.x[u];
      } else {
        x[u] = u32x4{0u, 0u, 0u, 0u};
        if (t < n && s.tier[row] != kDROP) x[u] = ld_nt16(src + static_cast<size_t>(t) * D + lane * 8);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = (it + u) * RPI + rsub;
      const int tr = s.tier[row];
      const uint32_t amax = group_max<LPR>(absmax_bits8(x[u]));  // all lanes take part
      if (tr == kFP16) {
        store16<NT>(dst + s.off[row] + lane * 16, x[u]);
      } else if (tr == kINT8 || tr == kINT4) {
        const LaneCodes q = quantize_lane(x[u], amax, tr == kINT8 ? 127 : 7);
        if (q.nonfinite && lane == 0) atomicAdd(nonfinite, 1u);
        uint8_t* out_row = dst + s.off[row];
        if (tr == kINT8) store8<NT>(out_row + lane * 8, pack_int8(q));
        else store4<NT>(out_row + lane * 4, pack_int4(q));
        if (lane == 0) scales[s.q[row]] = q.scale;
      }
    }
  }
}

// Loads one row slice of a lane: 16 B of FP16, 8 B of INT8 codes or 4 B of
// INT4 codes.
__device__ __forceinline__ void load_row(int tr, const uint8_t* row, int lane, u32x4& raw) {
  raw = u32x4{0u, 0u, 0u, 0u};
  if (tr == kFP16) {
    raw = ld_nt16(row + lane * 16);
  } else if (tr == kINT8) {
    const u32x2 c = ld_nt8(row + lane * 8);
    raw.x = c.x;
    raw.y = c.y;
  } else if (tr == kINT4) {
    raw.x = ld_nt4(row + lane * 4);
  }
}

// The lane's 8 output elements of a row: FP16 verbatim, DROP zeros, INT8/INT4
// dequantized, a NaN scale giving 0x7E00 (and any NaN product, 0x7E00).
__device__ __forceinline__ u32x4 decode_row(int tr, u32x4 raw, float sc) {
  if (tr == kINT8 || tr == kINT4) {
    if (__builtin_isnan(sc)) return u32x4{kNaNHalf2, kNaNHalf2, kNaNHalf2, kNaNHalf2};
    const u32x4 o = tr == kINT8 ? dequant_int8(u32x2{raw.x, raw.y}, sc) : dequant_int4(raw.x, sc);
    // only an infinite scale makes a NaN product (code 0): written as 0x7E00
    return __builtin_isinf(sc) ? canon_nan_lane(o) : o;
  }
  return raw;
}

// Dequantizes the rows of one chunk into their paged slots.  src: the
// segment's rows; the scales are staged in s.scale (stage_scale); cache: the
// (layer, head) column of the paged cache (slot stride H * D elements).
template <int D, int ROWS_IN_FLIGHT, bool NT>
__device__ __forceinline__ void unpack_chunk(const ChunkLds& s, const uint8_t* __restrict__ src,
                                             uint16_t* __restrict__ cache, int H) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  constexpr int U = ITERS < ROWS_IN_FLIGHT ? ITERS : ROWS_IN_FLIGHT;
  static_assert(ITERS % U == 0, "rows in flight must divide a thread's rows of the chunk");
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 raw[U];
    float sc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      load_row(s.tier[r], src + s.off[r], lane, raw[u]);
      sc[u] = s.scale[r];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int tr = s.tier[r];
      if (tr == kAbsent) continue;
      store16<NT>(cache + static_cast<size_t>(s.pos[r]) * H * D + lane * 8, decode_row(tr, raw[u], sc[u]));
    }
  }
}

}  // namespace skv
