// Host side of the C ABI declared in include/skv.h: argument checks, the tier
// plan (Sec. 2.1 eq. "budget", Sec. 4.4), payload geometry, the decay table
// and kernel launches.  Nothing here synchronizes with the device except the
// decay-table uploads of skv_prepare and skv_score_static.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "skv_internal.h"

namespace skv {
namespace {

inline uint64_t round_up_256(uint64_t x) { return (x + 255u) / 256u * 256u; }

inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
inline bool dev_ptr_ok(const void* p) { return p != nullptr && aligned(p, 16); }

skv_status check_config(const skv_config* c) {
  if (c == nullptr) return SKV_ERR_INVALID_ARG;
  const int d = c->head_dim;
  if (c->num_layers < 1 || c->num_kv_heads < 1) return SKV_ERR_INVALID_ARG;
  if (static_cast<int64_t>(c->num_layers) * c->num_kv_heads > 65536) return SKV_ERR_INVALID_ARG;
  if (d != 32 && d != 64 && d != 128 && d != 256) return SKV_ERR_INVALID_ARG;
  if (c->num_tokens < 1 || c->num_tokens > kMaxTokens) return SKV_ERR_INVALID_ARG;
  if (!(c->budget > 0.0f) || !(c->budget <= 1.0f)) return SKV_ERR_INVALID_ARG;
  if (!(c->first_ratio >= 0.0f) || !(c->first_ratio <= 1.0f)) return SKV_ERR_INVALID_ARG;
  if (c->num_sink < -1) return SKV_ERR_INVALID_ARG;
  if (!std::isfinite(c->decay) || !(c->decay >= 0.0f)) return SKV_ERR_INVALID_ARG;
  if (2.0 * static_cast<double>(c->decay) * static_cast<double>(c->num_tokens - 1) > 700.0)
    return SKV_ERR_INVALID_ARG;
  if (c->num_tiers != 2 && c->num_tiers != 3) return SKV_ERR_INVALID_ARG;
  for (const int32_t q : {c->quant_int8, c->quant_int4})
    if ((q & ~31) != 0 || (q & 3) == 3) return SKV_ERR_INVALID_ARG;
  switch (c->score_mode) {
    case SKV_SCORE_KVNORM:
    case SKV_SCORE_RECENCY:
      break;
    case SKV_SCORE_ATTN:
      if (c->num_q_heads < 1 || c->num_q_heads % c->num_kv_heads != 0) return SKV_ERR_INVALID_ARG;
      if (c->obs_window < 1) return SKV_ERR_INVALID_ARG;
      if (static_cast<int64_t>(c->num_q_heads / c->num_kv_heads) * c->obs_window > 256)
        return SKV_ERR_INVALID_ARG;
      break;
    default:
      return SKV_ERR_INVALID_ARG;
  }
  return SKV_OK;
}

// Tier counts.  Everything is counted in quarter-units of the fp16 row cost
// (FP16 4, INT8 2, INT4 1, DROP 0), so the budget b becomes B = floor(4 b n)
// units; both products are exact in binary64 (24-bit b times n <= 2^21).
skv_status plan_counts(const skv_config* c, skv_plan* p) {
  const int64_t n = c->num_tokens;
  int64_t sinks;
  if (c->num_sink >= 0) {
    sinks = std::min<int64_t>(c->num_sink, n);
  } else {
    const double want = std::ceil(static_cast<double>(c->first_ratio) * static_cast<double>(n));
    sinks = want >= static_cast<double>(n) ? n : static_cast<int64_t>(want);
  }
  const int64_t units = static_cast<int64_t>(std::floor(4.0 * static_cast<double>(c->budget) * static_cast<double>(n)));
  if (4 * sinks > units) return SKV_ERR_BUDGET;
  const int64_t rest = n - sinks;     // ranked tokens
  const int64_t left = units - 4 * sinks;  // their budget
  int64_t f16 = 0, i8 = 0, i4 = 0, drop = 0;
  if (left >= 2 * rest) {
    // every ranked token affords INT8; the surplus buys FP16 upgrades (+2 units each)
    f16 = (left - 2 * rest) / 2;
    i8 = rest - f16;
  } else if (c->num_tiers == 3) {
    if (left >= rest) {
      // every ranked token affords INT4; the surplus buys INT8 upgrades (+1 unit each)
      i8 = left - rest;
      i4 = rest - i8;
    } else {
      i4 = left;  // INT4 for as many tokens as the budget allows, the rest dropped
      drop = rest - i4;
    }
  } else {
    i8 = left / 2;  // INT4 disabled: INT8 is the lowest tier, the rest dropped
    drop = rest - i8;
  }
  p->n_sink = static_cast<int32_t>(sinks);
  p->n_fp16 = static_cast<int32_t>(f16);
  p->n_int8 = static_cast<int32_t>(i8);
  p->n_int4 = static_cast<int32_t>(i4);
  p->n_drop = static_cast<int32_t>(drop);
  p->budget_units = units;
  p->used_units = 4 * (sinks + f16) + 2 * i8 + i4;
  return SKV_OK;
}

// Bytes of one group's metadata (s, then lo if asymmetric) under descriptor q.
inline uint32_t variant_entry_bytes(int32_t q) {
  return ((q & SKV_QUANT_ASYM) ? 2u : 1u) * ((q & SKV_QUANT_FP16) ? 2u : 4u);
}

// Per-row metadata bytes of one quantized row under variant descriptor q; K
// rows of a per-channel tier carry none (their entries are per chunk).
inline uint32_t variant_meta_bytes(int32_t q, int32_t d, bool k_row = false) {
  if (k_row && (q & SKV_QUANT_CHANNEL)) return 0u;
  int32_t gs = (q & 3) == 0 ? d : (q & 3) == 1 ? 64 : 32;
  gs = std::min(gs, d);
  return static_cast<uint32_t>(d / gs) * variant_entry_bytes(q);
}

// Per-channel entry bytes of one (head, chunk) for a tier under descriptor q.
inline uint32_t channel_block_bytes(int32_t q, int32_t d) {
  return (q & SKV_QUANT_CHANNEL) ? static_cast<uint32_t>(d) * variant_entry_bytes(q) : 0u;
}

inline uint32_t float_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return u;
}

}  // namespace

skv_status make_geometry(const skv_config* cfg, Geometry* g, skv_plan* plan_out) {
  skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  skv_plan p;
  st = plan_counts(cfg, &p);
  if (st != SKV_OK) return st;
  g->L = cfg->num_layers;
  g->H = cfg->num_kv_heads;
  g->d = cfg->head_dim;
  g->n = cfg->num_tokens;
  g->n_sink = p.n_sink;
  g->n16 = p.n_fp16;
  g->n8 = p.n_int8;
  g->n4 = p.n_int4;
  g->nd = p.n_drop;
  g->budget_units = p.budget_units;
  g->used_units = p.used_units;
  g->nq = static_cast<int64_t>(p.n_int8) + p.n_int4;
  g->q8 = cfg->quant_int8;
  g->q4 = cfg->quant_int4;
  g->e8 = variant_meta_bytes(g->q8, cfg->head_dim);
  g->e4 = variant_meta_bytes(g->q4, cfg->head_dim);
  g->ek8 = variant_meta_bytes(g->q8, cfg->head_dim, true);
  g->ek4 = variant_meta_bytes(g->q4, cfg->head_dim, true);
  g->cb8 = channel_block_bytes(g->q8, cfg->head_dim);
  g->cb4 = channel_block_bytes(g->q4, cfg->head_dim);
  g->seg_scale_bytes = static_cast<uint64_t>(p.n_int8) * g->e8 + static_cast<uint64_t>(p.n_int4) * g->e4;
  g->seg_scale_bytes_k = static_cast<uint64_t>(p.n_int8) * g->ek8 + static_cast<uint64_t>(p.n_int4) * g->ek4;
  g->cidx_entry = (g->q8 | g->q4) ? 16u : 8u;
  g->nchunks = (g->n + kChunkTokens - 1) / kChunkTokens;
  const uint64_t d = static_cast<uint64_t>(g->d), H = static_cast<uint64_t>(g->H);
  g->tiermap_off = 256;
  g->chunkidx_off = g->tiermap_off + round_up_256((static_cast<uint64_t>(g->n) + 3) / 4);
  g->layers_off = g->chunkidx_off + round_up_256(g->cidx_entry * static_cast<uint64_t>(g->nchunks));
  g->seg_bytes = static_cast<uint64_t>(p.n_sink + p.n_fp16) * (2 * d) +
                 static_cast<uint64_t>(p.n_int8) * d + static_cast<uint64_t>(p.n_int4) * (d / 2);
  g->seg_stride = round_up_256(g->seg_bytes);
  g->scales_bytes = round_up_256(H * (g->seg_scale_bytes_k + g->seg_scale_bytes));
  g->channel_bytes = round_up_256(H * static_cast<uint64_t>(g->nchunks) * (g->cb8 + g->cb4));
  g->layer_stride = g->scales_bytes + g->channel_bytes + 2 * H * g->seg_stride;
  g->total = g->layers_off + static_cast<uint64_t>(g->L) * g->layer_stride;
  if (plan_out) *plan_out = p;
  return SKV_OK;
}

namespace {

uint64_t decay_table_bytes(const skv_config* c) {
  return round_up_256(8u * static_cast<uint64_t>(c->num_tokens));
}

uint64_t scratch_bytes(const skv_config* c) {
  Geometry g{};
  g.L = c->num_layers;
  g.H = c->num_kv_heads;
  g.d = c->head_dim;
  g.n = c->num_tokens;
  uint64_t score_bytes = 0;
  switch (c->score_mode) {
    case SKV_SCORE_KVNORM: score_bytes = kvnorm_scratch_bytes(g); break;
    case SKV_SCORE_ATTN: score_bytes = attn_scratch_bytes(g, c->num_q_heads, c->obs_window); break;
    default: break;
  }
  // tier assignment reuses the area after scoring (stream order)
  return std::max(score_bytes, assign_scratch_bytes(g.n, 1));
}

inline skv_status launched(hipError_t e) { return e == hipSuccess ? SKV_OK : SKV_ERR_DEVICE; }

// Rate of the decay table: exp(-lambda * Delta) for attention and recency
// scores, exp(-(2 lambda) * Delta) for the squared KV-norm score; the product
// is exact in binary64.
double decay_rate(const skv_config* c) {
  return static_cast<double>(c->decay) * (c->score_mode == SKV_SCORE_KVNORM ? 2.0 : 1.0);
}

// out[i] = exp(-(rate * (begin + i))) for i in [0, count), with the C
// library's binary64 exp (the argument is exact: rate has 25 significant bits
// and the index at most 21).
void fill_decay(double rate, int begin, int count, double* out) {
#pragma clang loop vectorize(disable)
  for (int i = 0; i < count; ++i) out[i] = std::exp(-(rate * static_cast<double>(begin + i)));
}

void fill_common(const skv_config* cfg, int32_t layer_begin, int32_t layer_count, BatchArgs* a) {
  std::memset(a, 0, sizeof(*a));
  a->L = cfg->num_layers;
  a->H = cfg->num_kv_heads;
  a->d = cfg->head_dim;
  a->layer_begin = layer_begin;
  a->layer_count = layer_count;
  a->num_tiers = cfg->num_tiers;
  a->score_mode = cfg->score_mode;
  a->budget_bits = float_bits(cfg->budget);
  a->rho_bits = float_bits(cfg->first_ratio);
  a->decay_bits = float_bits(cfg->decay);
  a->q8 = cfg->quant_int8;
  a->q4 = cfg->quant_int4;
  a->e8 = variant_meta_bytes(cfg->quant_int8, cfg->head_dim);
  a->e4 = variant_meta_bytes(cfg->quant_int4, cfg->head_dim);
  a->ek8 = variant_meta_bytes(cfg->quant_int8, cfg->head_dim, true);
  a->ek4 = variant_meta_bytes(cfg->quant_int4, cfg->head_dim, true);
  a->cb8 = channel_block_bytes(cfg->quant_int8, cfg->head_dim);
  a->cb4 = channel_block_bytes(cfg->quant_int4, cfg->head_dim);
}

void fill_desc(const Geometry& g, const skv_request& q, ReqDesc* r) {
  std::memset(r, 0, sizeof(*r));
  r->k = static_cast<const uint16_t*>(q.k);
  r->v = static_cast<const uint16_t*>(q.v);
  r->tier = q.tier;
  r->payload = static_cast<uint8_t*>(q.payload);
  r->status = q.dev_status;
  r->block_table = q.block_table;
  r->chunkidx_off = g.chunkidx_off;
  r->layers_off = g.layers_off;
  r->seg_bytes = g.seg_bytes;
  r->seg_scale_bytes = g.seg_scale_bytes;
  r->seg_scale_bytes_k = g.seg_scale_bytes_k;
  r->channel_bytes = g.channel_bytes;
  r->seg_stride = g.seg_stride;
  r->scales_bytes = g.scales_bytes;
  r->layer_stride = g.layer_stride;
  r->total = g.total;
  r->nq = g.nq;
  r->budget_units = g.budget_units;
  r->used_units = g.used_units;
  r->n = g.n;
  r->nchunks = static_cast<int32_t>(g.nchunks);
  r->n_sink = g.n_sink;
  r->n16 = g.n16;
  r->n8 = g.n8;
  r->n4 = g.n4;
  r->nd = g.nd;
}

bool layer_range_ok(const skv_config* cfg, int32_t layer_begin, int32_t layer_count) {
  return layer_begin >= 0 && layer_count >= 1 &&
         static_cast<int64_t>(layer_begin) + layer_count <= cfg->num_layers;
}

// Validates every request (pack: unpack == false) and fills their geometry.
skv_status check_requests(const skv_config* cfg, const skv_request* reqs, int32_t count, bool unpack,
                          std::vector<Geometry>* geo) {
  if (cfg == nullptr || reqs == nullptr || count < 1) return SKV_ERR_INVALID_ARG;
  geo->resize(static_cast<size_t>(count));
  for (int32_t i = 0; i < count; ++i) {
    const skv_request& q = reqs[i];
    if (q.reserved != 0) return SKV_ERR_INVALID_ARG;
    skv_config c = *cfg;
    c.num_tokens = q.num_tokens;
    const skv_status st = make_geometry(&c, &(*geo)[i], nullptr);
    if (st != SKV_OK) return st;
    if (!dev_ptr_ok(q.payload)) return SKV_ERR_INVALID_ARG;
    if (!unpack) {
      if (!dev_ptr_ok(q.k) || !dev_ptr_ok(q.v) || !dev_ptr_ok(q.tier)) return SKV_ERR_INVALID_ARG;
      if (q.dev_status != nullptr && !aligned(q.dev_status, 4)) return SKV_ERR_INVALID_ARG;
      if (q.payload_bytes < (*geo)[i].total) return SKV_ERR_CAPACITY;
    } else {
      if (q.block_table == nullptr || !aligned(q.block_table, 4)) return SKV_ERR_INVALID_ARG;
      if (q.dev_status == nullptr || !aligned(q.dev_status, 4)) return SKV_ERR_INVALID_ARG;
      if (q.payload_bytes < (*geo)[i].total) return SKV_ERR_FORMAT;
    }
  }
  return SKV_OK;
}

// Launches the requests kMaxBatch at a time.
template <typename Launch>
skv_status launch_batches(const skv_config* cfg, const skv_request* reqs, int32_t count,
                          const std::vector<Geometry>& geo, int32_t layer_begin, int32_t layer_count,
                          Launch launch) {
  for (int32_t first = 0; first < count; first += kMaxBatch) {
    BatchArgs a;
    fill_common(cfg, layer_begin, layer_count, &a);
    a.count = std::min<int32_t>(kMaxBatch, count - first);
    uint64_t rows = 0;
    for (int32_t i = 0; i < a.count; ++i) {
      const Geometry& g = geo[static_cast<size_t>(first + i)];
      fill_desc(g, reqs[first + i], &a.r[i]);
      a.r[i].block_begin = rows;
      rows += static_cast<uint64_t>(g.nchunks) * 2u * static_cast<uint64_t>(g.H) * static_cast<uint64_t>(layer_count);
    }
    if (launch(a, rows) != hipSuccess) return SKV_ERR_DEVICE;
  }
  return SKV_OK;
}

// ---- per-layer / per-head tier maps ----

int32_t group_count(const skv_config* c, int32_t gran) {
  switch (gran) {
    case SKV_GROUP_TOKEN: return 1;
    case SKV_GROUP_LAYER: return c->num_layers;
    case SKV_GROUP_HEAD: return c->num_layers * c->num_kv_heads;
    default: return -1;
  }
}

struct GroupHost {
  GroupLaunch gl;
  std::vector<skv_plan> plans;
  std::vector<uint32_t> table;   // G x 8 words
  std::vector<uint64_t> segtab;  // 2LH x {scales offset, rows offset}
  uint64_t ws_group_off, ws_segtab_off, ws_scratch_off, ws_total;
};

// Validates cfg and spec, plans every group and lays out the grouped payload
// and the workspace.
skv_status group_host(const skv_config* cfg, const skv_group_spec* spec, GroupHost* out) {
  skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (cfg->quant_int8 != 0 || cfg->quant_int4 != 0) return SKV_ERR_INVALID_ARG;  // descriptor 0 only
  if (spec == nullptr || spec->reserved != 0) return SKV_ERR_INVALID_ARG;
  const int32_t gran = spec->granularity, G = group_count(cfg, gran);
  if (G < 1) return SKV_ERR_INVALID_ARG;
  const int64_t L = cfg->num_layers, H = cfg->num_kv_heads, n = cfg->num_tokens, d = cfg->head_dim;
  if (L * H > 65535) return SKV_ERR_INVALID_ARG;  // a grid dimension holds the (layer, head) pairs
  out->plans.assign(static_cast<size_t>(G), skv_plan{});
  out->table.assign(8u * static_cast<size_t>(G), 0u);
  for (int32_t g = 0; g < G; ++g) {
    skv_config c = *cfg;
    if (spec->budgets != nullptr) {
      const float b = spec->budgets[g];
      if (!(b > 0.0f) || !(b <= 1.0f)) return SKV_ERR_INVALID_ARG;
      c.budget = b;
    }
    skv_plan& p = out->plans[static_cast<size_t>(g)];
    st = plan_counts(&c, &p);
    if (st != SKV_OK) return st;
    uint32_t* e = &out->table[8u * static_cast<size_t>(g)];
    e[0] = static_cast<uint32_t>(p.n_sink);
    e[1] = static_cast<uint32_t>(p.n_fp16);
    e[2] = static_cast<uint32_t>(p.n_int8);
    e[3] = static_cast<uint32_t>(p.n_int4);
    e[4] = static_cast<uint32_t>(p.n_drop);
    e[5] = float_bits(c.budget);
    e[6] = static_cast<uint32_t>(p.n_int8 + p.n_int4);
  }
  GroupLaunch& gl = out->gl;
  std::memset(&gl, 0, sizeof(gl));
  gl.L = cfg->num_layers;
  gl.H = cfg->num_kv_heads;
  gl.d = cfg->head_dim;
  gl.n = cfg->num_tokens;
  gl.gran = gran;
  gl.G = G;
  gl.nchunks = static_cast<int32_t>((n + kChunkTokens - 1) / kChunkTokens);
  gl.num_tiers = cfg->num_tiers;
  gl.score_mode = cfg->score_mode;
  gl.num_sink = cfg->num_sink;
  gl.budget_bits = float_bits(cfg->budget);
  gl.rho_bits = float_bits(cfg->first_ratio);
  gl.decay_bits = float_bits(cfg->decay);
  gl.group_off = 256;
  gl.tiermaps_off = gl.group_off + round_up_256(32u * static_cast<uint64_t>(G));
  gl.tiermap_stride = round_up_256((static_cast<uint64_t>(n) + 3) / 4);
  gl.chunkidx_off = gl.tiermaps_off + static_cast<uint64_t>(G) * gl.tiermap_stride;
  gl.chunkidx_stride = round_up_256(8u * static_cast<uint64_t>(gl.nchunks));
  gl.segtab_off = gl.chunkidx_off + static_cast<uint64_t>(G) * gl.chunkidx_stride;
  gl.layers_off = gl.segtab_off + round_up_256(32u * static_cast<uint64_t>(L * H));
  out->segtab.assign(4u * static_cast<size_t>(L * H), 0u);
  uint64_t off = gl.layers_off;
  for (int64_t l = 0; l < L; ++l) {
    auto group = [&](int64_t h) -> const uint32_t* {
      const int64_t g = gran == SKV_GROUP_TOKEN ? 0 : gran == SKV_GROUP_LAYER ? l : l * H + h;
      return &out->table[8u * static_cast<size_t>(g)];
    };
    uint64_t nscales = 0;
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        out->segtab[2u * static_cast<size_t>((l * 2 + kv) * H + h)] = off + 4u * nscales;
        nscales += group(h)[6];
      }
    uint64_t data = off + round_up_256(4u * nscales);
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        const uint32_t* e = group(h);
        out->segtab[2u * static_cast<size_t>((l * 2 + kv) * H + h) + 1] = data;
        const uint64_t bytes = static_cast<uint64_t>(e[0] + e[1]) * (2u * d) + static_cast<uint64_t>(e[2]) * d +
                               static_cast<uint64_t>(e[3]) * (d / 2);
        data += round_up_256(bytes);
      }
    off = data;
  }
  gl.total = off;
  out->ws_group_off = decay_table_bytes(cfg);
  out->ws_segtab_off = out->ws_group_off + round_up_256(32u * static_cast<uint64_t>(G));
  out->ws_scratch_off = out->ws_segtab_off + round_up_256(32u * static_cast<uint64_t>(L * H));
  Geometry geo{};
  geo.L = gl.L;
  geo.H = gl.H;
  geo.d = gl.d;
  geo.n = gl.n;
  uint64_t scratch = 0;
  if (cfg->score_mode == SKV_SCORE_KVNORM) scratch = kvnorm_scratch_bytes_groups(geo, gran);
  if (cfg->score_mode == SKV_SCORE_ATTN) scratch = attn_scratch_bytes(geo, cfg->num_q_heads, cfg->obs_window);
  // the split tier cut (rows past 32768 tokens) reuses the area after scoring
  scratch = std::max(scratch, assign_scratch_bytes(gl.n, G));
  out->ws_total = out->ws_scratch_off + round_up_256(scratch);
  return SKV_OK;
}

// The launch description with its table pointers inside the workspace ws.
GroupLaunch group_launch(const GroupHost& gh, const void* ws) {
  GroupLaunch gl = gh.gl;
  const uint8_t* base = static_cast<const uint8_t*>(ws);
  gl.group_table = reinterpret_cast<const uint32_t*>(base + gh.ws_group_off);
  gl.segtab = reinterpret_cast<const uint64_t*>(base + gh.ws_segtab_off);
  return gl;
}

// Pointer checks of skv_score's inputs for cfg's score mode.
skv_status check_score_inputs(const skv_config* cfg, const void* k, const void* v, const void* q_obs) {
  switch (cfg->score_mode) {
    case SKV_SCORE_KVNORM: return dev_ptr_ok(k) && dev_ptr_ok(v) ? SKV_OK : SKV_ERR_INVALID_ARG;
    case SKV_SCORE_ATTN: return dev_ptr_ok(k) && dev_ptr_ok(q_obs) ? SKV_OK : SKV_ERR_INVALID_ARG;
    default: return SKV_OK;
  }
}

// The score launches of cfg's mode, with the decay table at `table` and the
// mode's scratch at `scratch` (device memory).
skv_status score_launch(const skv_config* cfg, const void* k, const void* v, const void* q_obs, double* score,
                        const double* table, void* scratch, hipStream_t stream) {
  Geometry g{};
  g.L = cfg->num_layers;
  g.H = cfg->num_kv_heads;
  g.d = cfg->head_dim;
  g.n = cfg->num_tokens;
  switch (cfg->score_mode) {
    case SKV_SCORE_KVNORM:
      return launched(launch_score_kvnorm(g, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                                          table, static_cast<uint64_t*>(scratch), score, stream));
    case SKV_SCORE_ATTN:
      return launched(launch_score_attn(g, cfg->num_q_heads, cfg->obs_window, static_cast<const uint16_t*>(k),
                                        static_cast<const uint16_t*>(q_obs), table, scratch, score, stream));
    default:
      return launched(launch_score_recency(g, table, score, stream));
  }
}

// Host checks of a batched score / assign: cfg, the mode, every request's
// length and pointers; fills each request's plan (cfg at its own n).
skv_status check_score_requests(const skv_config* cfg, const skv_score_request* reqs, int32_t count,
                                bool for_assign, std::vector<skv_plan>* plans) {
  skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (cfg->score_mode == SKV_SCORE_ATTN) return SKV_ERR_INVALID_ARG;
  if (count < 0 || (count > 0 && reqs == nullptr)) return SKV_ERR_INVALID_ARG;
  plans->resize(static_cast<size_t>(count));
  for (int32_t i = 0; i < count; ++i) {
    const skv_score_request& q = reqs[i];
    if (q.reserved != 0 || q.num_tokens < 1 || q.num_tokens > cfg->num_tokens) return SKV_ERR_INVALID_ARG;
    if (!dev_ptr_ok(q.score)) return SKV_ERR_INVALID_ARG;
    if (for_assign && q.tier == nullptr) return SKV_ERR_INVALID_ARG;
    if (!for_assign && cfg->score_mode == SKV_SCORE_KVNORM && (!dev_ptr_ok(q.k) || !dev_ptr_ok(q.v)))
      return SKV_ERR_INVALID_ARG;
    skv_config c = *cfg;
    c.num_tokens = q.num_tokens;
    if (for_assign && (st = plan_counts(&c, &(*plans)[i])) != SKV_OK) return st;
  }
  return SKV_OK;
}

// Partial-sum layout of a batched KV-norm score: the shape shared by the
// batch and each request's byte offset after the decay table.
uint64_t score_batch_layout(const skv_config* cfg, const skv_score_request* reqs, int32_t count, ScoreBatchArgs* shape,
                            std::vector<uint64_t>* offsets) {
  std::vector<int32_t> ns(static_cast<size_t>(count));
  for (int32_t i = 0; i < count; ++i) ns[i] = reqs[i].num_tokens;
  std::memset(shape, 0, sizeof(*shape));
  if (count > 0) kvnorm_batch_shape(cfg->num_layers, cfg->num_kv_heads, cfg->head_dim, ns.data(), count, shape);
  uint64_t off = decay_table_bytes(cfg);
  offsets->resize(static_cast<size_t>(count));
  for (int32_t i = 0; i < count; ++i) {
    (*offsets)[i] = off;
    if (cfg->score_mode == SKV_SCORE_KVNORM)
      off += round_up_256(static_cast<uint64_t>(shape->groups) * static_cast<uint64_t>(ns[i]) * 16u);
  }
  return off;
}

}  // namespace
}  // namespace skv

// Library-owned scoring scratch of skv_score_static: [decay table | score
// scratch], laid out as in a caller's workspace.  Each device holds its own
// copy from the library's load until the process ends.  Host code never uses
// this name as an address (on the host it is only a handle to the symbol):
// the device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) uint8_t scratch[SKV_STATIC_SCRATCH_BYTES];

namespace skv {
namespace {

constexpr int kMaxStaticDevices = 64;

// Per device: the device address of `scratch` (null until first use) and the
// decay table it holds, exp(-table_rate * Delta) for Delta in [0, table_count).
struct StaticScratch {
  uint8_t* base;
  double table_rate;
  int32_t table_count;
};

std::mutex g_static_mutex;
StaticScratch g_static[kMaxStaticDevices];

// Looks up the current device's copy of `scratch` (once per device) and makes
// sure it starts with cfg's decay table: a table of the same rate is reused,
// extended if it is shorter than n; otherwise it is rewritten.  The table is
// computed on the host in pieces held on this thread's stack, each copied in
// stream order and waited for before the piece is overwritten, so nothing is
// allocated.  Since the score scratch follows the table of this call's n,
// only the first n entries are recorded as resident afterwards.
skv_status static_scratch_prepare(const skv_config* cfg, hipStream_t stream, uint8_t** base_out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SKV_ERR_DEVICE;
  if (dev >= kMaxStaticDevices) return SKV_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_static_mutex);
  StaticScratch& ss = g_static[dev];
  if (ss.base == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return SKV_ERR_DEVICE;
    ss.base = static_cast<uint8_t*>(p);
    ss.table_count = 0;
  }
  const int n = cfg->num_tokens;
  const double rate = decay_rate(cfg);
  int have = ss.table_rate == rate ? ss.table_count : 0;
  if (have < n) {
    ss.table_count = 0;  // invalid until every piece has landed
    constexpr int kPiece = 4096;
    double piece[kPiece];
    for (int begin = have; begin < n; begin += kPiece) {
      const int count = std::min(kPiece, n - begin);
      fill_decay(rate, begin, count, piece);
      if (hipMemcpyAsync(ss.base + static_cast<uint64_t>(begin) * sizeof(double), piece, count * sizeof(double),
                         hipMemcpyHostToDevice, stream) != hipSuccess ||
          hipStreamSynchronize(stream) != hipSuccess)
        return SKV_ERR_DEVICE;
    }
    ss.table_rate = rate;
    have = n;
  }
  ss.table_count = std::min(have, n);
  *base_out = ss.base;
  return SKV_OK;
}

}  // namespace
}  // namespace skv

using namespace skv;

extern "C" {

int32_t skv_abi_version(void) { return SKV_ABI_VERSION; }

const char* skv_status_string(int32_t status) {
  switch (status) {
    case SKV_OK: return "ok";
    case SKV_ERR_INVALID_ARG: return "invalid argument";
    case SKV_ERR_BUDGET: return "sink tokens exceed the budget";
    case SKV_ERR_CAPACITY: return "output buffer too small, or request too large for the static scratch";
    case SKV_ERR_FORMAT: return "payload does not match the configuration";
    case SKV_ERR_DEVICE: return "HIP launch or copy failed";
  }
  return "unknown status";
}

skv_status skv_plan_tiers(const skv_config* cfg, skv_plan* out) {
  if (out == nullptr) return SKV_ERR_INVALID_ARG;
  Geometry g;
  return make_geometry(cfg, &g, out);
}

skv_status skv_payload_size(const skv_config* cfg, uint64_t* bytes) {
  if (bytes == nullptr) return SKV_ERR_INVALID_ARG;
  Geometry g;
  const skv_status st = make_geometry(cfg, &g, nullptr);
  if (st == SKV_OK) *bytes = g.total;
  return st;
}

skv_status skv_workspace_size(const skv_config* cfg, uint64_t* bytes) {
  if (bytes == nullptr) return SKV_ERR_INVALID_ARG;
  const skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  *bytes = decay_table_bytes(cfg) + round_up_256(scratch_bytes(cfg));
  return SKV_OK;
}

skv_status skv_prepare(const skv_config* cfg, void* ws, hipStream_t stream) {
  skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  const int n = cfg->num_tokens;
  std::vector<double> table(static_cast<size_t>(n));
  fill_decay(decay_rate(cfg), 0, n, table.data());
  if (hipMemcpyAsync(ws, table.data(), table.size() * sizeof(double), hipMemcpyHostToDevice, stream) != hipSuccess)
    return SKV_ERR_DEVICE;
  return hipStreamSynchronize(stream) == hipSuccess ? SKV_OK : SKV_ERR_DEVICE;
}

skv_status skv_score(const skv_config* cfg, const void* k, const void* v, const void* q_obs,
                     double* score, void* ws, hipStream_t stream) {
  skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(score) || !dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  if (st = check_score_inputs(cfg, k, v, q_obs); st != SKV_OK) return st;
  return score_launch(cfg, k, v, q_obs, score, static_cast<const double*>(ws),
                      static_cast<uint8_t*>(ws) + decay_table_bytes(cfg), stream);
}

skv_status skv_score_static(const skv_config* cfg, const void* k, const void* v, const void* q_obs,
                            double* score, hipStream_t stream) {
  skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(score)) return SKV_ERR_INVALID_ARG;
  if (st = check_score_inputs(cfg, k, v, q_obs); st != SKV_OK) return st;
  const uint64_t table_bytes = decay_table_bytes(cfg);
  if (table_bytes + round_up_256(scratch_bytes(cfg)) > SKV_STATIC_SCRATCH_BYTES) return SKV_ERR_CAPACITY;
  uint8_t* base = nullptr;
  if (st = static_scratch_prepare(cfg, stream, &base); st != SKV_OK) return st;
  return score_launch(cfg, k, v, q_obs, score, reinterpret_cast<const double*>(base), base + table_bytes, stream);
}

skv_status skv_batch_workspace_size(const skv_config* cfg, const skv_score_request* reqs, int32_t count,
                                    uint64_t* bytes) {
  if (bytes == nullptr) return SKV_ERR_INVALID_ARG;
  std::vector<skv_plan> plans;
  const skv_status st = check_score_requests(cfg, reqs, count, false, &plans);
  if (st != SKV_OK) return st;
  ScoreBatchArgs shape;
  std::vector<uint64_t> offsets;
  const uint64_t score_bytes = score_batch_layout(cfg, reqs, count, &shape, &offsets);
  // skv_assign_batch's split tier cut reuses the partial-sum region: one
  // select state per long request of a launch
  int32_t longest = 0, long_rows = 0;
  for (int32_t i = 0; i < count; ++i)
    if (assign_scratch_bytes(reqs[i].num_tokens, 1) != 0) {
      longest = std::max(longest, reqs[i].num_tokens);
      ++long_rows;
    }
  const uint64_t assign_bytes =
      decay_table_bytes(cfg) + assign_scratch_bytes(longest, std::min(long_rows, kMaxScoreBatch));
  *bytes = std::max(score_bytes, assign_bytes);
  return SKV_OK;
}

skv_status skv_score_batch(const skv_config* cfg, const skv_score_request* reqs, int32_t count, void* ws,
                           hipStream_t stream) {
  std::vector<skv_plan> plans;
  const skv_status st = check_score_requests(cfg, reqs, count, false, &plans);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  ScoreBatchArgs a;
  std::vector<uint64_t> offsets;
  score_batch_layout(cfg, reqs, count, &a, &offsets);
  uint8_t* base = static_cast<uint8_t*>(ws);
  const double* table = static_cast<const double*>(ws);
  const int tok = 256 / (cfg->head_dim / 8);  // tokens per partial-sum workgroup
  for (int32_t first = 0; first < count; first += kMaxScoreBatch) {
    a.count = std::min(kMaxScoreBatch, count - first);
    uint32_t tb = 0, fb = 0;
    for (int32_t i = 0; i < a.count; ++i) {
      const skv_score_request& q = reqs[first + i];
      ScoreDesc& d = a.r[i];
      std::memset(&d, 0, sizeof(d));
      d.k = static_cast<const uint16_t*>(q.k);
      d.v = static_cast<const uint16_t*>(q.v);
      d.score = q.score;
      d.partial = reinterpret_cast<uint64_t*>(base + offsets[first + i]);
      d.n = q.num_tokens;
      d.tok_block_begin = tb;
      d.fin_block_begin = fb;
      tb += static_cast<uint32_t>((q.num_tokens + tok - 1) / tok);
      fb += static_cast<uint32_t>((q.num_tokens + 255) / 256);
    }
    const hipError_t e = cfg->score_mode == SKV_SCORE_KVNORM
                             ? launch_score_kvnorm_batch(a, cfg->head_dim, table, stream)
                             : launch_score_recency_batch(a, table, stream);
    if (e != hipSuccess) return SKV_ERR_DEVICE;
  }
  return SKV_OK;
}

skv_status skv_assign_batch(const skv_config* cfg, const skv_score_request* reqs, int32_t count, void* ws,
                            hipStream_t stream) {
  std::vector<skv_plan> plans;
  const skv_status st = check_score_requests(cfg, reqs, count, true, &plans);
  if (st != SKV_OK) return st;
  if (ws != nullptr && !dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  void* scratch = ws == nullptr ? nullptr : static_cast<uint8_t*>(ws) + decay_table_bytes(cfg);
  // requests whose non-sink keys fit the resident form go to resident
  // launches, the rest to split launches (workspace given) or launches of the
  // one-workgroup general form
  for (const bool resident : {true, false}) {
    ScoreBatchArgs a;
    std::memset(&a, 0, sizeof(a));
    for (int32_t i = 0; i <= count; ++i) {
      const bool flush = i == count || a.count == kMaxScoreBatch;
      if (flush && a.count > 0) {
        if (launch_assign_batch(a, resident, scratch, stream) != hipSuccess) return SKV_ERR_DEVICE;
        a.count = 0;
      }
      if (i == count) break;
      const skv_plan& p = plans[i];
      if (assign_fits_resident(reqs[i].num_tokens, p.n_sink) != resident) continue;
      ScoreDesc& d = a.r[a.count++];
      std::memset(&d, 0, sizeof(d));
      d.score = reqs[i].score;
      d.tier = reqs[i].tier;
      d.n = reqs[i].num_tokens;
      d.n_sink = p.n_sink;
      d.n16 = p.n_fp16;
      d.n8 = p.n_int8;
      d.n4 = p.n_int4;
    }
  }
  return SKV_OK;
}

skv_status skv_assign_tiers(const skv_config* cfg, const double* score, uint8_t* tier, void* ws,
                            hipStream_t stream) {
  Geometry g;
  const skv_status st = make_geometry(cfg, &g, nullptr);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(score) || !dev_ptr_ok(tier) || (ws != nullptr && !dev_ptr_ok(ws))) return SKV_ERR_INVALID_ARG;
  void* scratch = ws == nullptr ? nullptr : static_cast<uint8_t*>(ws) + decay_table_bytes(cfg);
  return launched(launch_assign(g, score, tier, scratch, stream));
}

skv_status skv_pack_batch(const skv_config* cfg, const skv_request* reqs, int32_t count,
                          int32_t layer_begin, int32_t layer_count, hipStream_t stream) {
  std::vector<Geometry> geo;
  const skv_status st = check_requests(cfg, reqs, count, false, &geo);
  if (st != SKV_OK) return st;
  if (!layer_range_ok(cfg, layer_begin, layer_count)) return SKV_ERR_INVALID_ARG;
  return launch_batches(cfg, reqs, count, geo, layer_begin, layer_count,
                        [&](const BatchArgs& a, uint64_t rows) { return launch_pack(a, rows, stream); });
}

skv_status skv_unpack_batch(const skv_config* cfg, const skv_request* reqs, int32_t count, void* k_cache,
                            void* v_cache, int32_t num_blocks, int32_t block_size, int32_t layer_begin,
                            int32_t layer_count, hipStream_t stream) {
  std::vector<Geometry> geo;
  const skv_status st = check_requests(cfg, reqs, count, true, &geo);
  if (st != SKV_OK) return st;
  if (!layer_range_ok(cfg, layer_begin, layer_count)) return SKV_ERR_INVALID_ARG;
  if (!dev_ptr_ok(k_cache) || !dev_ptr_ok(v_cache)) return SKV_ERR_INVALID_ARG;
  if (num_blocks < 1 || block_size < 1) return SKV_ERR_INVALID_ARG;
  if (static_cast<uint64_t>(num_blocks) * static_cast<uint64_t>(block_size) > 0xFFFFFFFFull)
    return SKV_ERR_INVALID_ARG;
  return launch_batches(cfg, reqs, count, geo, layer_begin, layer_count, [&](const BatchArgs& a, uint64_t rows) {
    return launch_unpack(a, rows, static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), num_blocks,
                         block_size, stream);
  });
}

skv_status skv_pack(const skv_config* cfg, const void* k, const void* v, const uint8_t* tier,
                    void* payload, uint64_t capacity, uint32_t* dev_status, hipStream_t stream) {
  if (cfg == nullptr) return SKV_ERR_INVALID_ARG;
  skv_request q;
  std::memset(&q, 0, sizeof(q));
  q.num_tokens = cfg->num_tokens;
  q.k = k;
  q.v = v;
  q.tier = tier;
  q.payload = payload;
  q.payload_bytes = capacity;
  q.dev_status = dev_status;
  return skv_pack_batch(cfg, &q, 1, 0, cfg->num_layers, stream);
}

skv_status skv_unpack(const skv_config* cfg, const void* payload, uint64_t payload_bytes,
                      void* k_cache, void* v_cache, const int32_t* block_table, int32_t num_blocks,
                      int32_t block_size, uint32_t* dev_status, hipStream_t stream) {
  if (cfg == nullptr) return SKV_ERR_INVALID_ARG;
  skv_request q;
  std::memset(&q, 0, sizeof(q));
  q.num_tokens = cfg->num_tokens;
  q.payload = const_cast<void*>(payload);
  q.payload_bytes = payload_bytes;
  q.block_table = block_table;
  q.dev_status = dev_status;
  return skv_unpack_batch(cfg, &q, 1, k_cache, v_cache, num_blocks, block_size, 0, cfg->num_layers, stream);
}

skv_status skv_upgrade_size(const skv_config* cfg, int32_t m, int32_t mode, uint64_t* bytes) {
  if (bytes == nullptr) return SKV_ERR_INVALID_ARG;
  const skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (cfg->quant_int8 != 0 || cfg->quant_int4 != 0) return SKV_ERR_INVALID_ARG;  // held rows use descriptor 0
  if (m < 1 || m > cfg->num_tokens || (mode != SKV_UPGRADE_FP16 && mode != SKV_UPGRADE_RESIDUAL8))
    return SKV_ERR_INVALID_ARG;
  *bytes = upgrade_bytes(cfg->num_layers, cfg->num_kv_heads, cfg->head_dim, m, mode, nullptr);
  return SKV_OK;
}

skv_status skv_pack_upgrade(const skv_config* cfg, const void* k, const void* v, const uint8_t* tier,
                            const int32_t* tokens, int32_t m, int32_t mode, void* out, uint64_t capacity,
                            uint32_t* dev_status, hipStream_t stream) {
  uint64_t need = 0;
  const skv_status st = skv_upgrade_size(cfg, m, mode, &need);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(k) || !dev_ptr_ok(v) || !dev_ptr_ok(tier) || !dev_ptr_ok(out)) return SKV_ERR_INVALID_ARG;
  if (tokens == nullptr || !aligned(tokens, 4)) return SKV_ERR_INVALID_ARG;
  if (dev_status != nullptr && !aligned(dev_status, 4)) return SKV_ERR_INVALID_ARG;
  if (capacity < need) return SKV_ERR_CAPACITY;
  Geometry g{};
  g.L = cfg->num_layers;
  g.H = cfg->num_kv_heads;
  g.d = cfg->head_dim;
  g.n = cfg->num_tokens;
  return launched(launch_pack_upgrade(g, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), tier,
                                      tokens, m, mode, static_cast<uint8_t*>(out), dev_status, stream));
}

skv_status skv_unpack_upgrade(const skv_config* cfg, const void* upgrade, uint64_t bytes, int32_t m,
                              int32_t mode, void* k_cache, void* v_cache, const int32_t* block_table,
                              int32_t num_blocks, int32_t block_size, uint32_t* dev_status,
                              hipStream_t stream) {
  uint64_t need = 0;
  const skv_status st = skv_upgrade_size(cfg, m, mode, &need);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(upgrade) || !dev_ptr_ok(k_cache) || !dev_ptr_ok(v_cache)) return SKV_ERR_INVALID_ARG;
  if (block_table == nullptr || !aligned(block_table, 4)) return SKV_ERR_INVALID_ARG;
  if (dev_status == nullptr || !aligned(dev_status, 4)) return SKV_ERR_INVALID_ARG;
  if (num_blocks < 1 || block_size < 1) return SKV_ERR_INVALID_ARG;
  if (static_cast<uint64_t>(num_blocks) * static_cast<uint64_t>(block_size) > 0xFFFFFFFFull)
    return SKV_ERR_INVALID_ARG;
  if (bytes < need) return SKV_ERR_FORMAT;
  Geometry g{};
  g.L = cfg->num_layers;
  g.H = cfg->num_kv_heads;
  g.d = cfg->head_dim;
  g.n = cfg->num_tokens;
  return launched(launch_unpack_upgrade(g, static_cast<const uint8_t*>(upgrade), m, mode,
                                        static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache),
                                        block_table, num_blocks, block_size, dev_status, stream));
}

namespace {

// The host link's second direction runs on a stream of the library's own (one
// per device, default priority, created on first use and kept until the
// process ends), ordered against the caller's stream by two events.
constexpr uint64_t kLinkPiece = 32ull << 20;
constexpr int kMaxLinkDevices = 64;

struct LinkLane {
  hipStream_t up;         // host-to-device copies
  hipEvent_t down_done;   // recorded on the caller's stream after a piece went down
  hipEvent_t up_done;     // recorded on `up` after the last piece went up
};

std::mutex g_link_mutex;
LinkLane g_link[kMaxLinkDevices];

}  // namespace

skv_status skv_link(void* dst, const void* src, uint64_t bytes, void* host_staging,
                    hipStream_t stream) {
  if (bytes == 0) return SKV_OK;
  if (dst == nullptr || src == nullptr) return SKV_ERR_INVALID_ARG;
  if (host_staging == nullptr) {
    if (aligned(dst, 16) && aligned(src, 16) && bytes % 16 == 0)
      return launched(launch_link_copy(dst, src, bytes, stream));
    return launched(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, stream));
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SKV_ERR_DEVICE;
  if (dev >= kMaxLinkDevices) return SKV_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_link_mutex);
  LinkLane& lane = g_link[dev];
  if (lane.up == nullptr) {
    if (hipEventCreateWithFlags(&lane.down_done, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&lane.up_done, hipEventDisableTiming) != hipSuccess ||
        hipStreamCreateWithFlags(&lane.up, hipStreamNonBlocking) != hipSuccess) {
      lane.up = nullptr;
      return SKV_ERR_DEVICE;
    }
  }
  // piece i goes down on the caller's stream, then up on `up` once it is in
  // host memory, so the way up of piece i overlaps the way down of piece i + 1
  // (PCIe carries both directions at once); `up` runs after everything enqueued
  // on the caller's stream before this call, and the caller's stream resumes
  // only after the last piece is up, so the call orders like one copy
  const uint8_t* s8 = static_cast<const uint8_t*>(src);
  uint8_t* d8 = static_cast<uint8_t*>(dst);
  uint8_t* h8 = static_cast<uint8_t*>(host_staging);
  for (uint64_t off = 0; off < bytes; off += kLinkPiece) {
    const uint64_t len = std::min(kLinkPiece, bytes - off);
    if (hipMemcpyAsync(h8 + off, s8 + off, len, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipEventRecord(lane.down_done, stream) != hipSuccess ||
        hipStreamWaitEvent(lane.up, lane.down_done, 0) != hipSuccess ||
        hipMemcpyAsync(d8 + off, h8 + off, len, hipMemcpyHostToDevice, lane.up) != hipSuccess)
      return SKV_ERR_DEVICE;
  }
  if (hipEventRecord(lane.up_done, lane.up) != hipSuccess) return SKV_ERR_DEVICE;
  return launched(hipStreamWaitEvent(stream, lane.up_done, 0));
}

skv_status skv_group_count(const skv_config* cfg, const skv_group_spec* spec, int32_t* count) {
  if (count == nullptr) return SKV_ERR_INVALID_ARG;
  const skv_status st = check_config(cfg);
  if (st != SKV_OK) return st;
  if (spec == nullptr || spec->reserved != 0) return SKV_ERR_INVALID_ARG;
  const int32_t G = group_count(cfg, spec->granularity);
  if (G < 1) return SKV_ERR_INVALID_ARG;
  *count = G;
  return SKV_OK;
}

skv_status skv_plan_groups(const skv_config* cfg, const skv_group_spec* spec, skv_plan* out) {
  if (out == nullptr) return SKV_ERR_INVALID_ARG;
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st != SKV_OK) return st;
  std::copy(gh.plans.begin(), gh.plans.end(), out);
  return SKV_OK;
}

skv_status skv_grouped_payload_size(const skv_config* cfg, const skv_group_spec* spec, uint64_t* bytes) {
  if (bytes == nullptr) return SKV_ERR_INVALID_ARG;
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st == SKV_OK) *bytes = gh.gl.total;
  return st;
}

skv_status skv_group_workspace_size(const skv_config* cfg, const skv_group_spec* spec, uint64_t* bytes) {
  if (bytes == nullptr) return SKV_ERR_INVALID_ARG;
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st == SKV_OK) *bytes = gh.ws_total;
  return st;
}

skv_status skv_prepare_groups(const skv_config* cfg, const skv_group_spec* spec, void* ws, hipStream_t stream) {
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  // decay table (as skv_prepare), group table and segment table in one upload
  std::vector<uint8_t> host(static_cast<size_t>(gh.ws_scratch_off), 0u);
  const int n = cfg->num_tokens;
  const double rate = static_cast<double>(cfg->decay) * (cfg->score_mode == SKV_SCORE_KVNORM ? 2.0 : 1.0);
  double* table = reinterpret_cast<double*>(host.data());
#pragma clang loop vectorize(disable)
  for (int delta = 0; delta < n; ++delta) table[delta] = std::exp(-(rate * static_cast<double>(delta)));
  std::memcpy(host.data() + gh.ws_group_off, gh.table.data(), gh.table.size() * sizeof(uint32_t));
  std::memcpy(host.data() + gh.ws_segtab_off, gh.segtab.data(), gh.segtab.size() * sizeof(uint64_t));
  if (hipMemcpyAsync(ws, host.data(), host.size(), hipMemcpyHostToDevice, stream) != hipSuccess)
    return SKV_ERR_DEVICE;
  return hipStreamSynchronize(stream) == hipSuccess ? SKV_OK : SKV_ERR_DEVICE;
}

skv_status skv_score_groups(const skv_config* cfg, const skv_group_spec* spec, const void* k, const void* v,
                            const void* q_obs, double* score, void* ws, hipStream_t stream) {
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(score) || !dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  Geometry g{};
  g.L = cfg->num_layers;
  g.H = cfg->num_kv_heads;
  g.d = cfg->head_dim;
  g.n = cfg->num_tokens;
  const double* table = static_cast<const double*>(ws);
  void* scratch = static_cast<uint8_t*>(ws) + gh.ws_scratch_off;
  const int32_t gran = spec->granularity, G = gh.gl.G;
  switch (cfg->score_mode) {
    case SKV_SCORE_KVNORM:
      if (!dev_ptr_ok(k) || !dev_ptr_ok(v)) return SKV_ERR_INVALID_ARG;
      return launched(launch_score_kvnorm_groups(g, gran, G, static_cast<const uint16_t*>(k),
                                                 static_cast<const uint16_t*>(v), table,
                                                 static_cast<uint64_t*>(scratch), score, stream));
    case SKV_SCORE_ATTN:
      if (!dev_ptr_ok(k) || !dev_ptr_ok(q_obs)) return SKV_ERR_INVALID_ARG;
      return launched(launch_score_attn_groups(g, gran, G, cfg->num_q_heads, cfg->obs_window,
                                               static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(q_obs),
                                               table, scratch, score, stream));
    default:
      return launched(launch_score_recency_groups(g, G, table, score, stream));
  }
}

skv_status skv_assign_groups(const skv_config* cfg, const skv_group_spec* spec, const double* score,
                             uint8_t* tier, void* ws, hipStream_t stream) {
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(score) || tier == nullptr || !dev_ptr_ok(ws)) return SKV_ERR_INVALID_ARG;
  const GroupLaunch gl = group_launch(gh, ws);
  void* scratch = static_cast<uint8_t*>(ws) + gh.ws_scratch_off;
  return launched(launch_assign_groups(gl.G, gl.n, gl.group_table, score, tier, scratch, stream));
}

skv_status skv_pack_groups(const skv_config* cfg, const skv_group_spec* spec, const void* k, const void* v,
                           const uint8_t* tier, const void* ws, void* payload, uint64_t capacity,
                           uint32_t* dev_status, hipStream_t stream) {
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(k) || !dev_ptr_ok(v) || tier == nullptr || !dev_ptr_ok(ws) || !dev_ptr_ok(payload))
    return SKV_ERR_INVALID_ARG;
  if (dev_status != nullptr && !aligned(dev_status, 4)) return SKV_ERR_INVALID_ARG;
  if (capacity < gh.gl.total) return SKV_ERR_CAPACITY;
  return launched(launch_pack_groups(group_launch(gh, ws), static_cast<const uint16_t*>(k),
                                     static_cast<const uint16_t*>(v), tier, static_cast<uint8_t*>(payload),
                                     dev_status, stream));
}

skv_status skv_unpack_groups(const skv_config* cfg, const skv_group_spec* spec, const void* ws, const void* payload,
                             uint64_t payload_bytes, void* k_cache, void* v_cache, const int32_t* block_table,
                             int32_t num_blocks, int32_t block_size, uint32_t* dev_status, hipStream_t stream) {
  GroupHost gh;
  const skv_status st = group_host(cfg, spec, &gh);
  if (st != SKV_OK) return st;
  if (!dev_ptr_ok(ws) || !dev_ptr_ok(payload) || !dev_ptr_ok(k_cache) || !dev_ptr_ok(v_cache))
    return SKV_ERR_INVALID_ARG;
  if (block_table == nullptr || !aligned(block_table, 4)) return SKV_ERR_INVALID_ARG;
  if (dev_status == nullptr || !aligned(dev_status, 4)) return SKV_ERR_INVALID_ARG;
  if (num_blocks < 1 || block_size < 1) return SKV_ERR_INVALID_ARG;
  if (static_cast<uint64_t>(num_blocks) * static_cast<uint64_t>(block_size) > 0xFFFFFFFFull)
    return SKV_ERR_INVALID_ARG;
  if (payload_bytes < gh.gl.total) return SKV_ERR_FORMAT;
  return launched(launch_unpack_groups(group_launch(gh, ws), static_cast<const uint8_t*>(payload),
                                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), block_table,
                                       num_blocks, block_size, dev_status, stream));
}

}  // extern "C"
