// Library-internal declarations shared by the host API and the kernel files.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

#include "../../include/skv.h"

namespace skv {

constexpr int kChunkTokens = 256;         // tokens per chunk-index entry
constexpr uint32_t kMagic = 0x31564B53u;  // "SKV1"
constexpr uint32_t kVersion = 1u;
constexpr int kMaxTokens = 1 << 21;

// Everything the kernels need to know about one request: shape, tier counts
// and the payload geometry derived from them (sizes known before scoring).
struct Geometry {
  int32_t L, H, d, n;
  int32_t n_sink, n16, n8, n4, nd;
  int64_t budget_units, used_units;
  int64_t nq;       // quantized rows per segment (n8 + n4)
  int32_t q8, q4;    // quantizer variant descriptors (0: row-wise symmetric, fp32 scale)
  uint32_t e8, e4;   // per-row metadata bytes of an INT8 / INT4 V row
  uint32_t ek8, ek4; // the same for a K row (0 for a per-channel tier)
  uint32_t cb8, cb4; // per-channel entries of one (head, chunk): INT8 / INT4 tier (0 unless per-channel)
  uint64_t seg_scale_bytes, seg_scale_bytes_k;  // per-row metadata of a V / K segment
  uint64_t channel_bytes;  // the layer's per-channel area (256-aligned)
  uint64_t cidx_entry;     // chunk-index entry bytes (8 or 16)
  int64_t nchunks;  // ceil(n / 256)
  uint64_t tiermap_off, chunkidx_off, layers_off;
  uint64_t seg_bytes, seg_stride, scales_bytes, layer_stride, total;
};

skv_status make_geometry(const skv_config* cfg, Geometry* g, skv_plan* plan_out);

// One request of a pack/unpack launch: its buffers and payload geometry.
struct ReqDesc {
  const uint16_t* k;
  const uint16_t* v;
  const uint8_t* tier;
  uint8_t* payload;
  uint32_t* status;             // may be null for pack
  const int32_t* block_table;   // unpack only
  uint64_t block_begin;         // first flat workgroup of this request in the row launch
  uint64_t chunkidx_off, layers_off, seg_bytes, seg_stride, scales_bytes, layer_stride, total;
  uint64_t seg_scale_bytes;    // per-row metadata bytes of one V segment (4 * nq for descriptor 0)
  uint64_t seg_scale_bytes_k;  // the same for a K segment (differs only with per-channel tiers)
  uint64_t channel_bytes;      // per-channel area of a layer, after the per-row metadata
  int64_t nq, budget_units, used_units;
  int32_t n, nchunks, n_sink, n16, n8, n4, nd, pad;
};

constexpr int kMaxBatch = 16;  // requests per launch (descriptors travel as kernel arguments)

// Everything a batched launch needs; fits the 4 KiB kernel-argument limit.
struct BatchArgs {
  int32_t count, L, H, d, layer_begin, layer_count, num_tiers, score_mode;
  uint32_t budget_bits, rho_bits, decay_bits, pad;
  int32_t q8, q4;    // quantizer variant descriptors of the INT8 and INT4 tiers
  uint32_t e8, e4;   // per-row metadata bytes of an INT8 / INT4 V row
  uint32_t ek8, ek4; // the same for a K row (0 for a per-channel tier)
  uint32_t cb8, cb4; // per-channel entry bytes of one (head, chunk) for the INT8 / INT4 tier
  ReqDesc r[kMaxBatch];
};
static_assert(sizeof(BatchArgs) <= 4000, "kernel arguments");

// One request of a batched score / assign launch.  tok_block_begin: its
// first workgroup in the partial-sum launch (token blocks of 256 / (d / 8)
// tokens); fin_block_begin: its first 256-token block in the finish and
// recency launches.  The assign launches index requests directly (one
// workgroup per request, or one row per request in the split form).
struct ScoreDesc {
  const uint16_t* k;
  const uint16_t* v;
  double* score;
  uint8_t* tier;
  uint64_t* partial;  // KV-norm partial sums: groups x n x 16 bytes
  uint32_t tok_block_begin, fin_block_begin;
  int32_t n, n_sink, n16, n8, n4, pad;
};

constexpr int kMaxScoreBatch = 48;  // requests per launch (descriptors travel as kernel arguments)

struct ScoreBatchArgs {
  int32_t count, pairs, pairs_per_group, groups, parts_per_block, pad;
  ScoreDesc r[kMaxScoreBatch];
};
static_assert(sizeof(ScoreBatchArgs) <= 4000, "kernel arguments");

// Kernel launchers.  Each returns the launch status; none synchronizes.

// Device-to-device copy of `bytes` (a multiple of 16; both pointers 16-byte
// aligned; the ranges do not overlap).
hipError_t launch_link_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream);

hipError_t launch_score_kvnorm(const Geometry& g, const uint16_t* k, const uint16_t* v,
                               const double* w2, uint64_t* partial, double* score,
                               hipStream_t stream);
hipError_t launch_score_recency(const Geometry& g, const double* w1, double* score,
                                hipStream_t stream);
hipError_t launch_score_attn(const Geometry& g, int32_t Hq, int32_t W, const uint16_t* k,
                             const uint16_t* q, const double* w1, void* scratch, double* score,
                             hipStream_t stream);
// Device scratch (bytes) the scoring launches need after the decay table.
uint64_t kvnorm_scratch_bytes(const Geometry& g);
uint64_t attn_scratch_bytes(const Geometry& g, int32_t Hq, int32_t W);

// Tier assignment of one request.  Rows past the resident form's 32768
// non-sink tokens run split over the GPU when scratch (assign_scratch_bytes
// for `rows` rows of n tokens, 256-byte aligned device memory) is given,
// else on one workgroup per row.
uint64_t assign_scratch_bytes(int32_t n, int32_t rows);
hipError_t launch_assign(const Geometry& g, const double* score, uint8_t* tier, void* scratch,
                         hipStream_t stream);

// Batched scoring and assignment (every request shares L, H, d and the
// policy; each has its own n).  kvnorm_batch_shape fills pairs,
// pairs_per_group, groups and parts_per_block of `a` for requests of lengths
// ns[0..count) (one shape for the whole batch, so that every launch chunk of
// it uses the same partial layout).  The launches cover a.count <=
// kMaxScoreBatch requests whose descriptors are complete.
void kvnorm_batch_shape(int32_t L, int32_t H, int32_t d, const int32_t* ns, int32_t count, ScoreBatchArgs* a);
hipError_t launch_score_kvnorm_batch(const ScoreBatchArgs& a, int32_t d, const double* w2, hipStream_t stream);
hipError_t launch_score_recency_batch(const ScoreBatchArgs& a, const double* w1, hipStream_t stream);
// `resident`: every request of the launch fits the resident form
// (n - n_sink <= 32768) and each takes one workgroup.  Otherwise the requests
// run split over the GPU when scratch (assign_scratch_bytes for a.count rows
// of more than 32768 tokens) is given, else on one workgroup each.
hipError_t launch_assign_batch(const ScoreBatchArgs& a, bool resident, void* scratch, hipStream_t stream);
bool assign_fits_resident(int32_t n, int32_t n_sink);

// Batched launches over a.count requests and layers [layer_begin, layer_begin +
// layer_count); `rows` is the total number of row workgroups (sum of
// nchunks * 2 * H * layer_count).  Pack writes the metadata when layer_begin
// is 0; unpack checks the payloads when layer_begin is 0.
hipError_t launch_pack(const BatchArgs& a, uint64_t rows, hipStream_t stream);
// Upgrade payload size; offsets (optional) receives tokens, tiers, scales and
// data offsets, the total and the row bytes.
uint64_t upgrade_bytes(int32_t L, int32_t H, int32_t d, int32_t m, int32_t mode, uint64_t* offsets);
hipError_t launch_pack_upgrade(const Geometry& g, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
                               const int32_t* tokens, int32_t m, int32_t mode, uint8_t* out, uint32_t* status,
                               hipStream_t stream);
hipError_t launch_unpack_upgrade(const Geometry& g, const uint8_t* up, int32_t m, int32_t mode, uint16_t* k_cache,
                                 uint16_t* v_cache, const int32_t* block_table, int32_t num_blocks,
                                 int32_t block_size, uint32_t* status, hipStream_t stream);
hipError_t launch_unpack(const BatchArgs& a, uint64_t rows, uint16_t* k_cache, uint16_t* v_cache,
                         int32_t num_blocks, int32_t block_size, hipStream_t stream);

// Per-layer / per-head tier maps: everything a grouped launch needs.  The
// group table (G x 8 words: sinks, fp16, int8, int4, drop, bits of b_g,
// quantized rows, 0) and the segment table (2LH x {scales offset, rows
// offset}) live in the caller's workspace, written by skv_prepare_groups.
struct GroupLaunch {
  const uint32_t* group_table;
  const uint64_t* segtab;
  int32_t L, H, d, n, gran, G, nchunks, num_tiers, score_mode, num_sink;
  uint32_t budget_bits, rho_bits, decay_bits;
  uint64_t group_off, tiermaps_off, tiermap_stride, chunkidx_off, chunkidx_stride, segtab_off, layers_off, total;
};
hipError_t launch_pack_groups(const GroupLaunch& gl, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
                              uint8_t* payload, uint32_t* status, hipStream_t stream);
hipError_t launch_unpack_groups(const GroupLaunch& gl, const uint8_t* payload, uint16_t* k_cache, uint16_t* v_cache,
                                const int32_t* block_table, int32_t num_blocks, int32_t block_size,
                                uint32_t* status, hipStream_t stream);
hipError_t launch_assign_groups(int32_t G, int32_t n, const uint32_t* group_table, const double* score,
                                uint8_t* tier, void* scratch, hipStream_t stream);
uint64_t kvnorm_scratch_bytes_groups(const Geometry& g, int32_t gran);
hipError_t launch_score_kvnorm_groups(const Geometry& g, int32_t gran, int32_t G, const uint16_t* k,
                                      const uint16_t* v, const double* w2, uint64_t* partial, double* score,
                                      hipStream_t stream);
hipError_t launch_score_recency_groups(const Geometry& g, int32_t G, const double* w1, double* score,
                                       hipStream_t stream);
hipError_t launch_score_attn_groups(const Geometry& g, int32_t gran, int32_t G, int32_t Hq, int32_t W,
                                    const uint16_t* k, const uint16_t* q, const double* w1, void* scratch,
                                    double* score, hipStream_t stream);

}  // namespace skv
