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
  int64_t nchunks;  // ceil(n / 256)
  uint64_t tiermap_off, chunkidx_off, layers_off;
  uint64_t seg_bytes, seg_stride, scales_bytes, layer_stride, total;
};

struct HeaderImage {
  uint32_t w[64];  // the 256-byte payload header, as written by pack
};

skv_status make_geometry(const skv_config* cfg, Geometry* g, skv_plan* plan_out);
void fill_header(const skv_config* cfg, const Geometry& g, HeaderImage* h);

// Kernel launchers.  Each returns the launch status; none synchronizes.
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

hipError_t launch_assign(const Geometry& g, const double* score, uint8_t* tier,
                         hipStream_t stream);

hipError_t launch_pack(const Geometry& g, const HeaderImage& hdr, const uint16_t* k,
                       const uint16_t* v, const uint8_t* tier, uint8_t* payload,
                       uint32_t* dev_status, hipStream_t stream);

hipError_t launch_unpack(const Geometry& g, const HeaderImage& hdr, const uint8_t* payload,
                         uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                         int32_t num_blocks, int32_t block_size, uint32_t* dev_status,
                         hipStream_t stream);

}  // namespace skv
