/*
 * skv.h -- C ABI of the SpectrumKV per-token mixed-precision KV transfer codec
 * for AMD Instinct MI355X (gfx950).
 *
 * The codec follows "SpectrumKV: Per-Token Mixed-Precision KV Cache Transfer
 * for Prefill-Decode Disaggregated LLM Serving" (arXiv 2606.08635): on the
 * prefill side it scores every prompt token (Sec. 4.3), pins the sink prefix
 * and assigns each remaining token FP16, INT8 or INT4 (or drops it) by
 * importance under a normalized byte budget (Sec. 2.1, Sec. 4.4, Algorithm 1
 * steps 2-3), then quantizes K and V independently per tier into one
 * compacted payload (Algorithm 1, transfer).  On the decode side it dequantizes
 * the payload into an fp16 paged KV cache (Sec. 4.2, Fig. "sysarch").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named k, v, q_obs, score, tier, payload, k_cache, v_cache,
 *    block_table, ws and dev_status are HIP device pointers (for example
 *    torch tensors' data_ptr()).  They must be 16-byte aligned.  The caller
 *    owns every buffer; the library allocates no device memory and keeps no
 *    global state (except skv_score_static's fixed scratch array), so calls
 *    on different streams with different buffers are independent.  Calls that
 *    share a buffer must be ordered by the caller.
 *  - Device entry points only enqueue work on `stream` and never synchronize
 *    with the host (skv_prepare is the one exception, see there).  A null
 *    stream means the legacy default stream.
 *  - Argument errors are detected on the host before anything is enqueued and
 *    returned as a status.  Data-dependent problems (a payload that does not
 *    match the configuration, out-of-range block-table entries, non-finite
 *    inputs) are reported in device memory, without a host sync.
 *  - K and V layout: binary16, [L][H][n][d] contiguous (layer, KV head, token,
 *    channel).  Observation queries: binary16 [L][Hq][W][d].
 *  - Paged cache layout: binary16 [L][num_blocks][block_size][H][d] for K and
 *    for V; token t of the request lives in physical block block_table[t /
 *    block_size], slot t % block_size.
 *
 * Payload format (version 1, little-endian, every section 256-byte aligned):
 *   [header 256 B]
 *   [tier map: 2 bits per token, token t in bits 2(t%4).. of byte t/4]
 *   [chunk index: per 256-token chunk c, u32 row-width units and u32 quantized
 *    rows before token 256c]
 *   [layer 0][layer 1]...[layer L-1], each layer =
 *     [fp32 scales: for K then V, for each head, one per quantized token in
 *      token order][data: for K then V, for each head, one segment holding the
 *      token rows in token order, FP16 rows 2d bytes, INT8 rows d bytes
 *      (two's complement), INT4 rows d/2 bytes (element 2i in the low nibble
 *      of byte i), DROP rows absent; segments padded to 256 B]
 *   Header fields (byte offset: type): 0 u32 magic 0x31564B53 ("SKV1"),
 *   4 u32 version, 8..20 i32 L, H, d, n, 24 i32 sinks, 28 i32 num_tiers,
 *   32/36/40 f32 bits of budget, first_ratio, decay, 44 i32 score_mode,
 *   48..60 i32 non-sink FP16 / INT8 / INT4 / DROP counts, 64/72 u64 budget and
 *   used quarter-units, 80/88/96 u64 offsets of tier map, chunk index and
 *   layer 0, 104 u64 segment bytes, 112 u64 segment stride, 120 u64 scale
 *   section bytes per layer, 128 u64 layer stride, 136 u64 total bytes,
 *   144 u32 quantized rows holding a non-finite value, 148 u32 pack status,
 *   152 u32 tokens per chunk (256), 156/160 i32 INT8 / INT4 quantizer
 *   descriptors, 168 u64 per-channel area bytes per layer (0 without a
 *   per-channel tier); all other bytes zero.
 */
#ifndef SKV_H_
#define SKV_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SKV_ABI_VERSION 2

typedef enum skv_status {
  SKV_OK = 0,
  SKV_ERR_INVALID_ARG = 1, /* bad shape, range, pointer or alignment           */
  SKV_ERR_BUDGET = 2,      /* the sinks alone exceed the budget (4s > floor(4bn)) */
  SKV_ERR_CAPACITY = 3,    /* output buffer smaller than skv_payload_size, or a
                              request too large for skv_score_static's scratch */
  SKV_ERR_FORMAT = 4,      /* payload_bytes too small for the configuration     */
  SKV_ERR_DEVICE = 5       /* a HIP call or kernel launch failed                */
} skv_status;

/* Tier codes of the precision map (Sec. 2.1: c(16)=1, c(8)=1/2, c(4)=1/4;
 * a dropped token costs 0, the selection view of Sec. 2.1). */
enum { SKV_TIER_FP16 = 0, SKV_TIER_INT8 = 1, SKV_TIER_INT4 = 2, SKV_TIER_DROP = 3 };

/* Importance statistic A_j of I_j = A_j exp(-lambda Delta_j) (Sec. 4.3). */
enum {
  SKV_SCORE_KVNORM = 0,  /* KV-norm fallback: squared Frobenius norm of the token's
                            K and V over every layer and head, times
                            exp(-2 lambda Delta) (the square of I_j, same order)  */
  SKV_SCORE_ATTN = 1,    /* mean softmax mass from an observation window of
                            queries, aggregated over layers and heads (Sec. 3)  */
  SKV_SCORE_RECENCY = 2  /* A_j = 1: the recency factor alone                     */
};

/* Problem statement (Sec. 2.1, Sec. 4.3-4.5).  All fields are read, never
 * written.  Validity: 1 <= L, H; L*H <= 65536; d in {32, 64, 128, 256};
 * 1 <= n <= 2^21; 0 < budget <= 1; 0 <= first_ratio <= 1; num_sink >= -1;
 * decay >= 0 and finite with 2*decay*(n-1) <= 700; num_tiers in {2, 3};
 * attention mode: num_q_heads a multiple of H, obs_window >= 1 and
 * (num_q_heads / H) * obs_window <= 256. */
typedef struct skv_config {
  int32_t num_layers;   /* L                                                      */
  int32_t num_kv_heads; /* H (KV heads)                                           */
  int32_t head_dim;     /* d                                                      */
  int32_t num_tokens;   /* n (prompt length)                                      */
  float budget;         /* b, normalized transfer budget, eq. "budget"            */
  float first_ratio;    /* rho: sinks s = ceil(rho * n) when num_sink == -1       */
  int32_t num_sink;     /* -1: use first_ratio; >= 0: explicit sink count (<= n)  */
  float decay;          /* lambda of exp(-lambda Delta), Delta = n-1-t            */
  int32_t num_tiers;    /* 3: FP16+INT8+INT4; 2: FP16+INT8 (INT4 disabled by the
                           tolerance probe, Sec. 4.5)                             */
  int32_t score_mode;   /* SKV_SCORE_*                                            */
  int32_t num_q_heads;  /* attention mode: query heads Hq (grouped, Hq/H per KV)  */
  int32_t obs_window;   /* attention mode: W observation queries per query head  */
  int32_t quant_int8;   /* quantizer variant of the INT8 tier (SKV_QUANT_*; 0 =
                           row-wise symmetric absmax with an fp32 scale)         */
  int32_t quant_int4;   /* quantizer variant of the INT4 tier                    */
} skv_config;

/* Quantizer variant descriptor bits (the quantizer inside a tier is a free
 * choice: Sec. 6.10, Sec. 8; KIVI-style asymmetric, Sec. 8 and Sec. 10).
 * Bits 0-1: elements per scale group, 0 = the whole row (d), SKV_QUANT_GROUP64,
 * SKV_QUANT_GROUP32 (capped at d); SKV_QUANT_ASYM: asymmetric codes 0..M
 * (M = 255 / 15) with the group minimum lo as zero point, x^ = code s + lo;
 * SKV_QUANT_FP16: s (and lo) stored as binary16.  Per group, symmetric:
 * s = RN32(a/Q), r = RN32(Q/a), a = max |x|; binary16: s = RN16(RN32(a/Q)),
 * r = RN32(1/s); code = clamp(rne(RN32(x r)), -Q, Q).  Asymmetric: lo, hi the
 * minimum and maximum (-0 below +0), range = RN32(hi - lo), s = RN32(range/M),
 * r = RN32(M/range) (binary16: s = RN16(RN32(range/M)), r = RN32(1/s)),
 * code = clamp(rne(RN32(RN32(x - lo) r)), 0, M); decode RN16(RN32(RN32(code s)
 * + lo)), any NaN written as 0x7E00.  A group with an inf/NaN gets NaN
 * metadata and decodes to 0x7E00; a
 * zero a or range, or a binary16 s that underflows, gives zero codes.  With
 * any nonzero descriptor the payload stores per quantized row its groups'
 * metadata (s, then lo if asymmetric; fp32 or binary16) in token order, and
 * chunk-index entries are 16 bytes: {units, quantized rows, metadata bytes
 * before the chunk, 0}; header words 39 and 40 hold the two descriptors.
 * SKV_QUANT_CHANNEL (per-channel key scales, KIVI-style key quantization,
 * Sec. 8 and Sec. 10): the K rows of the tier inside each 256-token chunk form
 * one group per channel (that channel's element of each such row) with the
 * ASYM/FP16 bits above; they carry no per-row metadata.  V rows keep the
 * per-row groups of the other bits.  A chunk without rows of the tier gets
 * zero entries.  With a per-channel tier each layer's per-row metadata holds
 * the H K segments (n8 ek8 + n4 ek4 bytes each, ek = 0 for a per-channel tier)
 * and then the H V segments; a per-channel area follows it (256-aligned,
 * header u64 at byte 168): per (head, chunk) the d INT8 entries (if that tier
 * is per-channel), then the d INT4 entries (if that tier is); the fourth
 * chunk-index word holds the K-side metadata bytes before the chunk.
 * The cold-tier upgrade and the grouped calls require both descriptors 0. */
#define SKV_QUANT_GROUP64 1
#define SKV_QUANT_GROUP32 2
#define SKV_QUANT_ASYM 4
#define SKV_QUANT_FP16 8
#define SKV_QUANT_CHANNEL 16

/* Tier counts of a configuration.  n_fp16/n_int8/n_int4/n_drop count the
 * non-sink tokens; the n_sink sink tokens are FP16 as well.  Budget in
 * quarter-units: budget_units = floor(4 b n), used_units = 4(n_sink + n_fp16)
 * + 2 n_int8 + n_int4 <= budget_units. */
typedef struct skv_plan {
  int32_t n_sink, n_fp16, n_int8, n_int4, n_drop;
  int64_t budget_units, used_units;
} skv_plan;

/* One request of a batched pack or unpack (see skv_pack_batch /
 * skv_unpack_batch).  Every pointer is device memory, 16-byte aligned except
 * block_table and dev_status (4-byte aligned). */
typedef struct skv_request {
  int32_t num_tokens;         /* n of this request (1 .. 2^21)                     */
  int32_t reserved;           /* must be 0                                         */
  const void* k;              /* pack: K, binary16 [L][H][n][d]                    */
  const void* v;              /* pack: V, binary16 [L][H][n][d]                    */
  const uint8_t* tier;        /* pack: tier map uint8[n], on plan                  */
  void* payload;              /* pack: output; unpack: input                       */
  uint64_t payload_bytes;     /* pack: capacity; unpack: bytes available           */
  const int32_t* block_table; /* unpack: int32[ceil(n / block_size)]               */
  uint32_t* dev_status;       /* pack: optional status word; unpack: required      */
} skv_request;

/* ABI version of the loaded library (SKV_ABI_VERSION at build time). */
int32_t skv_abi_version(void);

/* Human-readable name of a status code (any int32 value; values that are not
 * an skv_status give "unknown status"); never NULL. */
const char* skv_status_string(int32_t status);

/* Host only, pure.  Tier counts for cfg: sinks pinned first and charged to the
 * budget (Sec. 4.4), then the budget-to-tier mapping of Sec. 4.4 over the
 * remaining budget: b' >= 1/2 -> FP16 + INT8 (f16 = 2b'-1); 3-tier with
 * 1/4 <= b' < 1/2 -> INT8 + INT4 (f8 = 4b'-1); 3-tier below 1/4 -> INT4 +
 * DROP; 2-tier below 1/2 -> INT8 + DROP (Sec. 7.4.3).  Returns
 * SKV_ERR_INVALID_ARG for an invalid cfg or null out, SKV_ERR_BUDGET when the
 * sinks alone exceed the budget. */
skv_status skv_plan_tiers(const skv_config* cfg, skv_plan* out);

/* Host only.  Exact payload size in bytes for cfg (known before any scoring,
 * because the tier counts depend only on cfg). */
skv_status skv_payload_size(const skv_config* cfg, uint64_t* bytes);

/* Host only.  Device workspace bytes needed by skv_prepare, skv_score and
 * skv_assign_tiers for cfg (the decay table plus scratch; the scratch of the
 * tier cut, for rows past 32768 tokens, shares the area of the score's). */
skv_status skv_workspace_size(const skv_config* cfg, uint64_t* bytes);

/* Fills the decay table exp(-lambda Delta) (attention and recency modes) or
 * exp(-2 lambda Delta) (KV-norm mode), Delta = 0..n-1, at the start of ws.
 * The table is evaluated on the host in binary64 with the C library's exp and
 * copied to ws with a stream-ordered copy; this call waits for that copy
 * before returning.  The table depends only on (decay, n, score_mode), so a
 * workspace prepared once serves any number of skv_score calls with the same
 * three values.  Sec. 4.3, eq. "importance". */
skv_status skv_prepare(const skv_config* cfg, void* ws, hipStream_t stream);

/* Scores every token (Sec. 4.3; Algorithm 1, scoring).  k, v: [L][H][n][d]
 * binary16; q_obs: [L][Hq][W][d] binary16 in attention mode, else ignored;
 * score: double[n], written.  ws must be prepared for cfg by skv_prepare.
 * KV-norm mode: score[t] = RN64(RN64(S_t) * exp(-2 lambda (n-1-t))), S_t the
 * exact sum of squares of token t's finite K and V elements over all layers
 * and heads (non-finite elements contribute 0); the result is bit-exact.
 * Attention mode: score[t] = A_t exp(-lambda (n-1-t)), A_t the mean over
 * (layer, query head, observation query) of softmax over all n keys of
 * q.k/sqrt(d), query head hq reading KV head hq/(Hq/H); fp32 MFMA logits, so
 * within a stated relative tolerance of the binary64 definition.  Non-finite
 * inputs follow IEEE softmax: a NaN or +inf logit in any query row makes that
 * row's normalizer NaN and so every score NaN (assignment ranks NaN as +0); a
 * -inf logit only contributes nothing.  Recency mode: score[t] =
 * exp(-lambda (n-1-t)). */
skv_status skv_score(const skv_config* cfg, const void* k, const void* v, const void* q_obs,
                     double* score, void* ws, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): skv_score
 * without a workspace argument.  Results are those of skv_score (same
 * kernels); the decay table and score scratch live in a library-owned array
 * of SKV_STATIC_SCRATCH_BYTES on each device, which each device holds from
 * the first call until the process ends.  A request fits when
 * skv_workspace_size(cfg) <= SKV_STATIC_SCRATCH_BYTES (the 32-layer x 8-head
 * x 128-dim x 32768-token request fits in every score mode); a larger one
 * returns SKV_ERR_CAPACITY before anything is enqueued.  The call works on
 * the current device and allocates nothing (no hipMalloc, hipFree or
 * allocating library routine).  The decay table is kept between calls: a
 * call whose (score mode's decay rate, n) needs entries the array does not
 * hold computes them on the host and copies them in stream order in pieces
 * from this thread's stack, waiting for each copy (a host synchronization,
 * as in skv_prepare); otherwise nothing is copied and the call only
 * enqueues.  Every call on a device shares that device's array and leaves
 * its contents behind (the kernels write all scratch they read, so nothing
 * needs clearing): calls that overlap on one device -- on different streams,
 * or from different host threads without ordering -- race and give
 * undefined scores.  Argument errors as skv_score. */
#define SKV_STATIC_SCRATCH_BYTES (48u << 20)
skv_status skv_score_static(const skv_config* cfg, const void* k, const void* v, const void* q_obs,
                            double* score, hipStream_t stream);

/* Assigns tiers (Sec. 2.3 Prop. 1; Algorithm 1, scoring and tier assignment).  score: double[n]
 * (any values; NaN and non-positive scores rank as +0); tier: uint8[n],
 * written.  Tokens t < n_sink get FP16.  The other tokens are ranked by
 * descending composite key ((bits(score) >> 20) << 21) | t, i.e. by score cut
 * to 32 fraction bits with ties going to the more recent token, and the first
 * n_fp16 get FP16, the next n_int8 INT8, the next n_int4 INT4, the rest DROP.
 * Radix select over six digits of the key.  Rows of at most 32768 non-sink
 * tokens run on one workgroup and do not use ws.  Longer rows run split over
 * the GPU (one counting launch per digit) when ws is the request's workspace
 * (skv_workspace_size(cfg) bytes; its scratch area after the decay table is
 * overwritten, the decay table is not), or on one workgroup when ws is NULL;
 * both give the same tier map.  Calls that share a workspace (this one,
 * skv_score) must be ordered on one stream. */
skv_status skv_assign_tiers(const skv_config* cfg, const double* score, uint8_t* tier, void* ws,
                            hipStream_t stream);

/* Quantizes K and V per tier and packs the payload (Algorithm 1, transfer;
 * "standard symmetric" quantizer, Sec. 8).  tier: uint8[n] whose counts must
 * equal skv_plan_tiers(cfg) (sinks included in FP16).  payload: capacity bytes,
 * at least skv_payload_size(cfg); exactly that many bytes are written.
 * Per INT8/INT4 row (one row = one layer, K or V, head, token; Q = 127 / 7):
 * a = max |x| (binary16), scale = RN32(a/Q), r = RN32(Q/a),
 * code = clamp(rne(RN32(x r)), -Q, Q); a row with a non-finite element gets a
 * NaN scale and zero codes and is counted in header field 144; an all-zero
 * row gets scale 0.  FP16 rows are copied bit for bit.
 * If the tier map is off plan (a value > 3 or wrong counts) the header status
 * field is set to SKV_ERR_INVALID_ARG and nothing else is written.
 * dev_status (may be NULL): receives the same status (0 on success). */
skv_status skv_pack(const skv_config* cfg, const void* k, const void* v, const uint8_t* tier,
                    void* payload, uint64_t capacity, uint32_t* dev_status, hipStream_t stream);

/* Dequantizes a payload into the paged fp16 cache (Sec. 4.2: dequantize per
 * tier after receipt).  INT8/INT4 elements become RN16(RN32(code * scale))
 * (the product is rounded to binary32 first; a NaN product, possible only
 * for a non-finite scale, is written as 0x7E00);
 * FP16 rows are copied bit for bit; DROP rows are written as +0 (the consumer
 * masks them, Sec. 5 "data hygiene"); elements of a row with a NaN scale are
 * written as 0x7E00.  Cache slots of tokens >= n are not touched.
 * block_table: int32[ceil(n / block_size)], each in [0, num_blocks), the
 * entries distinct (unchecked: with a repeated entry the shared block's
 * contents are unspecified); block_size >= 1.  k_cache, v_cache and payload
 * must not overlap.  dev_status (required): set to 0 on success or to
 * SKV_ERR_FORMAT when the header, tier counts or chunk index disagree with cfg
 * or a block-table entry is out of range; in that case nothing is written.
 * Returns SKV_ERR_FORMAT (host-side) when payload_bytes is below
 * skv_payload_size(cfg). */
skv_status skv_unpack(const skv_config* cfg, const void* payload, uint64_t payload_bytes,
                      void* k_cache, void* v_cache, const int32_t* block_table, int32_t num_blocks,
                      int32_t block_size, uint32_t* dev_status, hipStream_t stream);

/* Batched, variable-length pack: `count` requests that share every field of
 * cfg except num_tokens (ignored; each request carries its own n) are packed
 * by one launch per kernel (up to 16 requests per launch; larger batches are
 * split internally), so many short requests fill the GPU.  Only layers
 * [layer_begin, layer_begin + layer_count) are packed: the payload is
 * layer-major, so a request can be packed layer by layer and each layer
 * block (its scales and segments, contiguous in the payload) sent as soon as
 * it is written.  The call with layer_begin == 0 also validates the tier map
 * and writes the header, tier map and chunk index; calls for later layers
 * must follow it in stream order.  Per request, results and errors are those
 * of skv_pack (status in the header and in dev_status when given).  Every
 * request is checked before anything is enqueued.  Sec. 9 (future work:
 * integration with a PD runtime and batching). */
skv_status skv_pack_batch(const skv_config* cfg, const skv_request* reqs, int32_t count,
                          int32_t layer_begin, int32_t layer_count, hipStream_t stream);

/* Batched, variable-length unpack into one shared paged cache
 * [L][num_blocks][block_size][H][d] (each request has its own block table,
 * the tables must not overlap).  Layer ranges as in skv_pack_batch: the call
 * with layer_begin == 0 checks every payload and writes each request's
 * dev_status; calls for later layers (in stream order after it) write
 * nothing for a request whose status is nonzero.  Per request, results and
 * errors are those of skv_unpack. */
skv_status skv_unpack_batch(const skv_config* cfg, const skv_request* reqs, int32_t count,
                            void* k_cache, void* v_cache, int32_t num_blocks, int32_t block_size,
                            int32_t layer_begin, int32_t layer_count, hipStream_t stream);

/* One request of a batched score / assign (skv_score_batch,
 * skv_assign_batch).  Device pointers, 16-byte aligned (tier: any). */
typedef struct skv_score_request {
  int32_t num_tokens; /* n of this request (1 .. cfg->num_tokens)              */
  int32_t reserved;   /* must be 0                                             */
  const void* k;      /* K, binary16 [L][H][n][d] (KV-norm mode; else unused)  */
  const void* v;      /* V, binary16 [L][H][n][d] (KV-norm mode; else unused)  */
  double* score;      /* double[n]: written by skv_score_batch, read by
                         skv_assign_batch                                      */
  uint8_t* tier;      /* uint8[n]: written by skv_assign_batch                 */
} skv_score_request;

/* Host only.  Workspace bytes of skv_score_batch and skv_assign_batch for
 * these requests: the decay table of cfg (cfg->num_tokens entries, at least
 * every request's n) followed by the larger of each request's partial sums
 * (KV-norm mode) and the split tier cut's select state (49192 bytes for each
 * request longer than 32768 tokens, at most 48 of them).  Errors as
 * skv_score_batch's host checks. */
skv_status skv_batch_workspace_size(const skv_config* cfg, const skv_score_request* reqs, int32_t count,
                                    uint64_t* bytes);

/* Batched scoring (Sec. 4.3; Sec. 9 (i), batching many requests): the
 * `count` requests share every field of cfg except the token count (each
 * carries its own n <= cfg->num_tokens); each request's scores are exactly
 * those of skv_score on that request alone.  KV-norm and recency modes only
 * (attention mode: SKV_ERR_INVALID_ARG).  One launch per kernel covers up to
 * 48 requests (larger batches are split).  ws: at least
 * skv_batch_workspace_size bytes, prepared by skv_prepare(cfg, ...) -- one
 * decay table serves every request, since its entry for Delta does not depend
 * on n.  Every request is checked before anything is enqueued. */
skv_status skv_score_batch(const skv_config* cfg, const skv_score_request* reqs, int32_t count, void* ws,
                           hipStream_t stream);

/* Batched tier assignment (Sec. 2.3 Prop. 1; Sec. 4.4): each request's tier
 * map is exactly skv_assign_tiers' on its scores with the plan of cfg at its
 * own n (SKV_ERR_BUDGET if some request's sinks exceed its budget).  Requests
 * of at most 32768 non-sink tokens take one workgroup each, one launch for up
 * to 48 of them.  Longer requests, up to 48 per launch sequence, run split
 * over the whole GPU (14 launches) when ws is given, else on one workgroup
 * each; both give the same tier maps.  ws: NULL, or a workspace of
 * skv_batch_workspace_size bytes for these requests (device memory, 16-byte
 * aligned; its area after the decay table is overwritten, the decay table is
 * not, and the split form clears what it needs with kernels, so the call can
 * be captured in a HIP graph).  Calls that share ws (this one,
 * skv_score_batch) must be ordered on one stream.  Every request is checked
 * before anything is enqueued. */
skv_status skv_assign_batch(const skv_config* cfg, const skv_score_request* reqs, int32_t count, void* ws,
                            hipStream_t stream);

/* Cold-tier precision upgrade (Sec. 4.2 and its architecture figure: tokens
 * the decoder holds at low precision are upgraded by an on-demand fetch;
 * Sec. 8, cold-tier fetch design).  Upgrade payload, little-endian, sections
 * 256-byte aligned with zero padding:
 *   bytes 0..75    header: u32 magic 0x55564B53, version 1, L, H, d, n, m,
 *                  mode; u64 tokens_off, tiers_off, scales_off, data_off,
 *                  total; u32 status (0); the rest of the 256 bytes zero
 *   tokens_off     int32[m] upgraded tokens, strictly ascending
 *   tiers_off      uint8[m] tier each token was sent at
 *   scales_off     RESIDUAL8 only: binary32[L][2][H][m] residual scales
 *   data_off       rows [L][2 (K,V)][H][m]: FP16 mode d binary16 values
 *                  (2d bytes); RESIDUAL8 mode d int8 codes (d bytes). */
typedef enum skv_upgrade_mode {
  SKV_UPGRADE_FP16 = 0,      /* send the fp16 rows: the cache becomes exact        */
  SKV_UPGRADE_RESIDUAL8 = 1  /* send e = RN32(x - held) as INT8 (absmax, Q = 127) */
} skv_upgrade_mode;

/* Host only.  Bytes of the upgrade payload for m tokens (1 <= m <= n) in
 * `mode`.  SKV_ERR_INVALID_ARG for a bad cfg, m or mode. */
skv_status skv_upgrade_size(const skv_config* cfg, int32_t m, int32_t mode, uint64_t* bytes);

/* Builds an upgrade payload on the prefill side, which still holds K, V
 * ([L][H][n][d] binary16) and the tier map tier (uint8[n]) the original
 * payload was packed with.  tokens: int32[m] device array, strictly
 * ascending, each in [0, n).  out: capacity bytes, at least
 * skv_upgrade_size; exactly that many bytes are written.  RESIDUAL8: for each
 * row, held = the row unpack wrote for its tier (the quantizer of skv_pack
 * followed by its dequantization; +0 for DROP; 0x7E00 for a NaN-scale row),
 * e = RN32(x - held) per element; a row whose e has a non-finite element gets
 * a NaN scale and zero codes, an all-zero e gets scale 0, otherwise
 * a = max |e|, scale = RN32(a/127), r = RN32(127/a),
 * code = clamp(rne(RN32(e r)), -127, 127).  If the token list is not strictly
 * ascending and in range, or a listed tier is > 3, the header status field is
 * set to SKV_ERR_INVALID_ARG and only the header is written.  dev_status (may
 * be NULL) receives the same status.  Host errors: SKV_ERR_INVALID_ARG,
 * SKV_ERR_CAPACITY. */
skv_status skv_pack_upgrade(const skv_config* cfg, const void* k, const void* v, const uint8_t* tier,
                            const int32_t* tokens, int32_t m, int32_t mode, void* out, uint64_t capacity,
                            uint32_t* dev_status, hipStream_t stream);

/* Applies an upgrade payload in place to the paged cache that skv_unpack
 * filled ([L][num_blocks][block_size][H][d], same block table).  FP16 mode
 * overwrites the listed rows; RESIDUAL8 mode sets each element to
 * RN16(RN32(held + RN32(code * scale))) and leaves rows with a NaN scale as
 * they are.  m and mode are the values the payload was built with.
 * dev_status (required) is set to 0, or to SKV_ERR_FORMAT when the header,
 * token list, tiers or a block-table entry disagree with cfg, m and mode; in
 * that case nothing is written.  Returns SKV_ERR_FORMAT (host-side) when
 * bytes is below skv_upgrade_size. */
skv_status skv_unpack_upgrade(const skv_config* cfg, const void* upgrade, uint64_t bytes, int32_t m,
                              int32_t mode, void* k_cache, void* v_cache, const int32_t* block_table,
                              int32_t num_blocks, int32_t block_size, uint32_t* dev_status,
                              hipStream_t stream);

/* Per-layer and per-head tier maps: the extension the paper names as future
 * work -- a per-layer budget allocation that favours layers whose errors are
 * amplified the most (Sec. 2.6, Sec. 6.10) and per-head or per-layer
 * importance scores (Sec. 7.5, Sec. 9 (iii)).  The (layer, KV head) pairs
 * are split into G groups; each group has its own score, its own budget b_g
 * (planned by the Sec. 4.4 mapping with sinks pinned, exactly as
 * skv_plan_tiers does for b) and its own tier map, shared by K and V of its
 * pairs.  Granularity SKV_GROUP_TOKEN (G = 1) is the paper's map;
 * SKV_GROUP_LAYER (G = L, group l); SKV_GROUP_HEAD (G = L*H, group l*H + h;
 * requires L*H <= 65535).
 *
 * Grouped payload, little-endian, sections 256-byte aligned, zero padding:
 *   header 256 B: u32 words 0 magic 0x47564B53 ("SKVG"), 1 version 1, 2-5 L,
 *     H, d, n, 6 granularity, 7 G, 8 num_tiers, 9 score_mode, 10-12 bits of
 *     budget, first_ratio, decay, 13 num_sink as configured, 14 chunk tokens
 *     (256), 15 zero; u64 at words 16, 18, ..., 30: offsets of the group
 *     table, tier maps, tier-map stride, chunk indexes, chunk-index stride,
 *     segment table, layers, and the total size; u32 word 32 the number of
 *     quantized rows holding an inf/NaN, word 33 status; the rest zero
 *   group table: G x 8 u32 [sinks, fp16, int8, int4, drop, bits of b_g,
 *     quantized rows, 0]
 *   G 2-bit tier maps (token t at bits 2(t%4) of byte t/4), each padded to the
 *     tier-map stride; G chunk indexes (u32 row-width units in d/2 bytes and
 *     u32 quantized rows before every 256th token), each padded to its stride
 *   segment table: for (layer, K/V, head) in that order, u64 offsets of the
 *     segment's scales and of its rows
 *   layers: [fp32 scales of the layer's 2H segments back to back, padded]
 *     [its 2H segments, rows in token order at their group's tier widths,
 *     each padded to 256 B] */
typedef enum skv_granularity {
  SKV_GROUP_TOKEN = 0,
  SKV_GROUP_LAYER = 1,
  SKV_GROUP_HEAD = 2
} skv_granularity;

typedef struct skv_group_spec {
  int32_t granularity;   /* skv_granularity                                      */
  int32_t reserved;      /* must be 0                                             */
  const float* budgets;  /* host, G budgets in (0, 1], or NULL: cfg->budget each */
} skv_group_spec;

/* The grouped calls quantize with the default (row, symmetric, fp32)
 * quantizer: cfg->quant_int8 and cfg->quant_int4 must be 0, and every
 * grouped call but skv_group_count returns SKV_ERR_INVALID_ARG otherwise. */

/* Host only.  G for cfg and spec. */
skv_status skv_group_count(const skv_config* cfg, const skv_group_spec* spec, int32_t* count);

/* Host only.  out[g] (G entries): the plan of group g under b_g.  Errors as
 * skv_plan_tiers, for the first group that fails; SKV_ERR_INVALID_ARG for a
 * bad spec or budget. */
skv_status skv_plan_groups(const skv_config* cfg, const skv_group_spec* spec, skv_plan* out);

/* Host only.  Exact size of the grouped payload. */
skv_status skv_grouped_payload_size(const skv_config* cfg, const skv_group_spec* spec, uint64_t* bytes);

/* Host only.  Device workspace bytes for the grouped calls: the decay table,
 * the group table, the segment table and score scratch. */
skv_status skv_group_workspace_size(const skv_config* cfg, const skv_group_spec* spec, uint64_t* bytes);

/* Plans the groups on the host and uploads the decay table (as skv_prepare),
 * the group table and the segment table into ws; waits for the copy.  Every
 * other grouped call takes a workspace prepared with the same cfg and spec. */
skv_status skv_prepare_groups(const skv_config* cfg, const skv_group_spec* spec, void* ws, hipStream_t stream);

/* Scores every token in every group: score is double[G][n].  The statistic of
 * skv_score restricted to the group's pairs: KV-norm, the exact sum of
 * squares over the group's K and V elements (bit-exact); attention, the mean
 * softmax mass over the observation rows of the query heads that read the
 * group's KV heads (same tolerance as skv_score); recency, the same for every
 * group.  With SKV_GROUP_TOKEN the result equals skv_score's. */
skv_status skv_score_groups(const skv_config* cfg, const skv_group_spec* spec, const void* k, const void* v,
                            const void* q_obs, double* score, void* ws, hipStream_t stream);

/* Assigns every group's tiers from its scores (skv_assign_tiers per group, with
 * the group's plan): tier is uint8[G][n].  Rows of at most 32768 tokens: one
 * workgroup per group.  Longer rows run split over the GPU, their scratch in
 * the workspace's area after the tables (overwritten; the decay, group and
 * segment tables are not), so calls sharing a workspace must be ordered on
 * one stream. */
skv_status skv_assign_groups(const skv_config* cfg, const skv_group_spec* spec, const double* score,
                             uint8_t* tier, void* ws, hipStream_t stream);

/* Packs the grouped payload (rows quantized exactly as skv_pack; segment
 * (l, K/V, h) uses its group's map).  tier: uint8[G][n], each map on its
 * group's plan; otherwise the header status and dev_status become
 * SKV_ERR_INVALID_ARG and no row is written.  dev_status may be NULL. */
skv_status skv_pack_groups(const skv_config* cfg, const skv_group_spec* spec, const void* k, const void* v,
                           const uint8_t* tier, const void* ws, void* payload, uint64_t capacity,
                           uint32_t* dev_status, hipStream_t stream);

/* Decodes a grouped payload into the paged cache (as skv_unpack).  Every
 * metadata byte (all but the non-finite count) must be what cfg, spec and the
 * payload's own tier maps imply and every block-table entry in range;
 * otherwise dev_status (required) becomes SKV_ERR_FORMAT and nothing is
 * written.  SKV_ERR_FORMAT (host) when payload_bytes is below the size. */
skv_status skv_unpack_groups(const skv_config* cfg, const skv_group_spec* spec, const void* ws, const void* payload,
                             uint64_t payload_bytes, void* k_cache, void* v_cache, const int32_t* block_table,
                             int32_t num_blocks, int32_t block_size, uint32_t* dev_status, hipStream_t stream);

/* Link emulation for a one-GPU setup (Sec. 4.2: the payload crosses the
 * network between prefill and decode).  Copies `bytes` from src to dst (the
 * two ranges must not overlap), ordered on stream like one copy: device to
 * device when host_staging is NULL (the library's streaming copy kernel when
 * both pointers are 16-byte aligned and bytes is a multiple of 16, else the
 * runtime's copy), otherwise device to pinned host (host_staging, at least `bytes`,
 * allocated with hipHostMalloc) and back to device in 32 MiB pieces, the way
 * up of each piece overlapping the way down of the next on a second stream
 * that the library creates per device on first use (default priority, kept
 * until the process ends).  Host-staged calls on one device are serialized by
 * the library; work enqueued on stream after the call sees dst complete. */
skv_status skv_link(void* dst, const void* src, uint64_t bytes, void* host_staging,
                    hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SKV_H_ */
