// Token scores (Sec. 4.3, eq. "importance"): KV-norm and recency modes.
//
// KV-norm mode ranks token t by I_t^2 = S_t * exp(-2 lambda (n-1-t)), where
// S_t is the sum of squares of every finite K and V element of the token over
// all layers and heads.  S_t is computed exactly, so the score is bit-exact
// whatever the reduction order:
//   * each binary16 x squares exactly in binary32 (22 significant bits), and
//     y = x^2 * 2^8 is split into an integer part fl = floor(y) < 2^40 and a
//     fraction y - fl, a multiple of 2^-40 below 1;
//   * a thread adds at most 2^13 such terms into two binary64 accumulators,
//     which stay exact (integers below 2^53, and multiples of 2^-40 below 2^13);
//   * the accumulators become integers in units of 2^-48 and are combined in
//     128-bit integer arithmetic across lanes and layer groups.
// A non-finite input turns an accumulator into inf/NaN; only then does the
// thread redo its sum with non-finite elements skipped.
#include <algorithm>

#include "device_util.h"
#include "skv_internal.h"

namespace skv {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxPairsPerGroup = 512;  // 2 tensors * 8 elements * 512 = 2^13 terms per thread
#ifndef SKV_KVNORM_PAIR_INFLIGHT
#define SKV_KVNORM_PAIR_INFLIGHT 4  // row slices whose loads are issued together, one-pair parts
#endif
#ifndef SKV_KVNORM_PAIR_ROWS
#define SKV_KVNORM_PAIR_ROWS 8
#endif
constexpr int kPairRows = SKV_KVNORM_PAIR_ROWS;  // row slices per thread, one-pair parts

struct U128 {
  uint64_t lo, hi;
};

__device__ __forceinline__ U128 add128(U128 a, U128 b) {
  U128 r;
  r.lo = a.lo + b.lo;
  r.hi = a.hi + b.hi + (r.lo < a.lo ? 1u : 0u);
  return r;
}

// Correctly rounded (nearest-even) conversion of a 128-bit unsigned integer
// to binary64.
__device__ __forceinline__ double u128_to_double(U128 x) {
  if (x.hi == 0 && x.lo == 0) return 0.0;
  const int lz = x.hi ? __clzll(x.hi) : 64 + __clzll(x.lo);
  uint64_t top, rest;
  if (lz >= 64) {
    top = x.lo << (lz - 64);
    rest = 0;
  } else if (lz == 0) {
    top = x.hi;
    rest = x.lo;
  } else {
    top = (x.hi << lz) | (x.lo >> (64 - lz));
    rest = x.lo << lz;
  }
  uint64_t m = top >> 11;           // 53 significant bits
  const uint64_t rb = top & 0x7FFu;  // the 11 bits below them
  const bool up = rb > 0x400u || (rb == 0x400u && (rest != 0 || (m & 1u)));
  m += up ? 1u : 0u;
  return ldexp(static_cast<double>(m), 75 - lz);
}

__device__ __forceinline__ void acc_word(uint32_t w, double& ah, double& al) {
  const float f0 = half_lo(w), f1 = half_hi(w);
  const double y0 = static_cast<double>(f0 * f0) * 256.0;
  const double y1 = static_cast<double>(f1 * f1) * 256.0;
  const double g0 = floor(y0), g1 = floor(y1);
  ah += g0;
  al += y0 - g0;
  ah += g1;
  al += y1 - g1;
}

__device__ __forceinline__ void acc_word_finite(uint32_t w, double& ah, double& al) {
  if (((w >> 10) & 31u) == 31u) w &= 0xFFFF0000u;
  if (((w >> 26) & 31u) == 31u) w &= 0x0000FFFFu;
  acc_word(w, ah, al);
}

__device__ __forceinline__ void acc16(u32x4 x, double& ah, double& al) {
  acc_word(x.x, ah, al);
  acc_word(x.y, ah, al);
  acc_word(x.z, ah, al);
  acc_word(x.w, ah, al);
}

// One block: TOK tokens x all LPR lanes of their rows, for parts_per_block
// consecutive parts starting at part blockIdx.y * parts_per_block; part j
// covers the (layer, head) pairs [j * pairs_per_group, (j + 1) *
// pairs_per_group).  Writes the 128-bit partial sum of each token and part in
// units of 2^-48 to partial[(part * n + t) * 2 + {0: lo, 1: hi}].
template <int D>
__device__ __forceinline__ void kvnorm_partial_block(const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
                                                     int n, int pairs, int pairs_per_group, int parts_per_block,
                                                     uint64_t* __restrict__ partial, int tok_block, int part_block) {
  constexpr int LPR = D / 8;
  constexpr int TOK = kThreads / LPR;
  __shared__ U128 s_part[kThreads];
  const int lane = threadIdx.x % LPR;
  const int r = threadIdx.x / LPR;
  const int t = tok_block * TOK + r;
  for (int pb = 0; pb < parts_per_block; ++pb) {  // block-uniform
  const int part = part_block * parts_per_block + pb;
  const int p0 = part * pairs_per_group;
  if (p0 >= pairs) break;
  const int p1 = min(pairs, p0 + pairs_per_group);
  const size_t pair_stride = static_cast<size_t>(n) * D;  // elements between (l, h) pairs
  double ah0 = 0.0, al0 = 0.0, ah1 = 0.0, al1 = 0.0;
  if (t < n) {
    const uint16_t* kp = k + static_cast<size_t>(p0) * pair_stride + static_cast<size_t>(t) * D + lane * 8;
    const uint16_t* vp = v + static_cast<size_t>(p0) * pair_stride + static_cast<size_t>(t) * D + lane * 8;
    int p = p0;
    for (; p + 2 <= p1; p += 2) {
      const u32x4 a = ld_nt16(kp), b = ld_nt16(vp);
      const u32x4 c = ld_nt16(kp + pair_stride), e = ld_nt16(vp + pair_stride);
      acc16(a, ah0, al0);
      acc16(b, ah1, al1);
      acc16(c, ah0, al0);
      acc16(e, ah1, al1);
      kp += 2 * pair_stride;
      vp += 2 * pair_stride;
    }
    if (p < p1) {
      acc16(ld_nt16(kp), ah0, al0);
      acc16(ld_nt16(vp), ah1, al1);
    }
    double ah = ah0 + ah1, al = al0 + al1;  // both sums exact (< 2^53 units)
    if (!(__builtin_isfinite(ah) && __builtin_isfinite(al))) {
      // an infinity or NaN was read: redo this thread's sum without them
      ah = 0.0;
      al = 0.0;
      const uint16_t* kq = k + static_cast<size_t>(p0) * pair_stride + static_cast<size_t>(t) * D + lane * 8;
      const uint16_t* vq = v + static_cast<size_t>(p0) * pair_stride + static_cast<size_t>(t) * D + lane * 8;
      for (int q = p0; q < p1; ++q) {
        const u32x4 a = ld_nt16(kq), b = ld_nt16(vq);
        acc_word_finite(a.x, ah, al);
        acc_word_finite(a.y, ah, al);
        acc_word_finite(a.z, ah, al);
        acc_word_finite(a.w, ah, al);
        acc_word_finite(b.x, ah, al);
        acc_word_finite(b.y, ah, al);
        acc_word_finite(b.z, ah, al);
        acc_word_finite(b.w, ah, al);
        kq += pair_stride;
        vq += pair_stride;
      }
    }
    // ah counts units of 2^-8 and al * 2^40 counts units of 2^-48; both are
    // integers below 2^53.
    const uint64_t a = static_cast<uint64_t>(ah);
    const uint64_t b = static_cast<uint64_t>(al * 1099511627776.0);  // * 2^40, exact
    U128 s;
    s.lo = (a << 40) + b;
    s.hi = (a >> 24) + (s.lo < b ? 1u : 0u);
    s_part[threadIdx.x] = s;
  } else {
    s_part[threadIdx.x] = U128{0, 0};
  }
  __syncthreads();
  if (lane == 0 && t < n) {
    U128 s = s_part[threadIdx.x];
#pragma unroll
    for (int i = 1; i < LPR; ++i) s = add128(s, s_part[threadIdx.x + i]);
    uint64_t* out = partial + (static_cast<size_t>(part) * n + t) * 2;
    out[0] = s.lo;
    out[1] = s.hi;
  }
  __syncthreads();  // s_part is reused by the next part
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void kvnorm_partial(const uint16_t* __restrict__ k,
                                                          const uint16_t* __restrict__ v, int n,
                                                          int pairs, int pairs_per_group, int parts_per_block,
                                                          uint64_t* __restrict__ partial) {
  kvnorm_partial_block<D>(k, v, n, pairs, pairs_per_group, parts_per_block, partial, blockIdx.x, blockIdx.y);
}

// Every lane of each aligned group of G lanes (G = 4 .. 32) receives the sum
// of the group's binary64 values: butterfly steps by DPP lane moves inside
// 16-lane rows (each 64-bit value moved as two 32-bit halves), then one
// shuffle across the two rows of a 32-lane group.  The caller's values are
// integers in a common unit below 2^53 with their sum, so every order of
// addition gives the same exact result.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t b = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = dpp_mov<CTRL>(static_cast<uint32_t>(b));
  const uint32_t hi = dpp_mov<CTRL>(static_cast<uint32_t>(b >> 32));
  return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

template <int G>
__device__ __forceinline__ double group_sum_f64(double x) {
  static_assert(G == 4 || G == 8 || G == 16 || G == 32, "group size");
  x += dpp_f64<0xB1>(x);                          // quad_perm [1,0,3,2]
  x += dpp_f64<0x4E>(x);                          // quad_perm [2,3,0,1]
  if constexpr (G >= 8) x += dpp_f64<0x141>(x);   // row_half_mirror
  if constexpr (G >= 16) x += dpp_f64<0x140>(x);  // row_mirror
  if constexpr (G == 32) {  // lanes i and i ^ 16: lower + upper, the same sum in both (addition commutes)
    const uint64_t b = __builtin_bit_cast(uint64_t, x);
    const LanePair lo = lane_pair16(static_cast<uint32_t>(b)), hi = lane_pair16(static_cast<uint32_t>(b >> 32));
    x = __builtin_bit_cast(double, (static_cast<uint64_t>(hi.lo) << 32) | lo.lo) +
        __builtin_bit_cast(double, (static_cast<uint64_t>(hi.hi) << 32) | lo.hi);
  }
  return x;
}

// Partial sums with one (layer, head) pair per part (per-head maps): block
// (x, y) covers pair y and the T * TOK consecutive tokens from x * T * TOK,
// i.e. one contiguous run of each of the pair's K and V planes.  A thread
// takes its T row slices S at a time, all 2 S loads issued before any is
// added (8 slices four at a time: 56 registers, 1 % faster than 4 slices two
// at a time; 4 slices four at a time or 8 eight at a time unroll into 114 or
// 502 registers and run far slower), and the lanes of a row combine their
// sums in binary64 by butterfly lane moves instead of through LDS.  That stays exact: a lane's
// sums hold 16 terms (8 K and 8 V elements), so over the LPR <= 32 lanes of
// a row the integer parts stay below 512 * 2^40 = 2^49 and the fractions,
// multiples of 2^-40, below 2^9; both are exact binary64 integers in their
// units, whatever the order.  A non-finite sum is redone from the registers
// without the non-finite elements.  The 128-bit sum is kvnorm_partial's.
// FINAL (each pair is a whole group): the block writes the group's score,
// RN64(S) * w2[n-1-t], into score[p * n + t], the value kvnorm_finish_groups
// would compute from the partial.
template <int D, int T, bool FINAL>
__global__ __launch_bounds__(kThreads) void kvnorm_partial_pairs(const uint16_t* __restrict__ k,
                                                                const uint16_t* __restrict__ v, int n,
                                                                uint64_t* __restrict__ partial,
                                                                const double* __restrict__ w2,
                                                                double* __restrict__ score) {
  constexpr int LPR = D / 8;
  constexpr int TOK = kThreads / LPR;
  const int lane = threadIdx.x % LPR;
  const int t0 = blockIdx.x * (T * TOK) + threadIdx.x / LPR;
  const int p = blockIdx.y;
  const size_t plane = static_cast<size_t>(p) * n * D;
  constexpr int S = SKV_KVNORM_PAIR_INFLIGHT < T ? SKV_KVNORM_PAIR_INFLIGHT : T;
  static_assert(T % S == 0, "whole groups of row slices");
#pragma unroll 1
  for (int i0 = 0; i0 < T; i0 += S) {  // S row slices (2 S 16-byte loads) in flight
    u32x4 kx[S], vx[S];
#pragma unroll
    for (int u = 0; u < S; ++u) {
      const int t = t0 + (i0 + u) * TOK;
      kx[u] = u32x4{0u, 0u, 0u, 0u};
      vx[u] = u32x4{0u, 0u, 0u, 0u};
      if (t < n) {
        const size_t off = plane + static_cast<size_t>(t) * D + lane * 8;
        kx[u] = ld_nt16(k + off);
        vx[u] = ld_nt16(v + off);
      }
    }
#pragma unroll
    for (int u = 0; u < S; ++u) {
      const int t = t0 + (i0 + u) * TOK;
      double ah = 0.0, al = 0.0;
      acc16(kx[u], ah, al);
      acc16(vx[u], ah, al);
      if (!(__builtin_isfinite(ah) && __builtin_isfinite(al))) {
        ah = 0.0;
        al = 0.0;
        const uint32_t w[8] = {kx[u].x, kx[u].y, kx[u].z, kx[u].w, vx[u].x, vx[u].y, vx[u].z, vx[u].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) acc_word_finite(w[e], ah, al);
      }
      ah = group_sum_f64<LPR>(ah);  // every lane of the row is active
      al = group_sum_f64<LPR>(al);
      if (lane == 0 && t < n) {
        const size_t idx = static_cast<size_t>(p) * n + t;
        if constexpr (FINAL) {
          // S = (ah + al) * 2^-8 exactly, and one binary64 addition of the two
          // exact terms is the correctly rounded sum: RN64(S) without the
          // 128-bit detour (the scaling by 2^-8 is exact: S is 0 or >= 2^-48)
          score[idx] = ((ah + al) * 0x1p-8) * w2[n - 1 - t];
        } else {
          const uint64_t a = static_cast<uint64_t>(ah);
          const uint64_t b = static_cast<uint64_t>(al * 1099511627776.0);  // * 2^40, exact
          const uint64_t lo = (a << 40) + b;
          partial[idx * 2] = lo;
          partial[idx * 2 + 1] = (a >> 24) + (lo < b ? 1u : 0u);
        }
      }
    }
  }
}

// Request of a batched launch that owns flat block `b` (the last whose first
// block is at most b; requests are in block order).
__device__ __forceinline__ int score_request_of(const ScoreBatchArgs& a, uint32_t b, bool finish) {
  int r = 0;
  for (int i = 1; i < a.count; ++i)
    if ((finish ? a.r[i].fin_block_begin : a.r[i].tok_block_begin) <= b) r = i;
  return r;
}

// grid: (sum over requests of their token blocks, part blocks)
template <int D>
__global__ __launch_bounds__(kThreads) void kvnorm_partial_batch(const ScoreBatchArgs a) {
  const ScoreDesc& q = a.r[score_request_of(a, blockIdx.x, false)];
  kvnorm_partial_block<D>(q.k, q.v, q.n, a.pairs, a.pairs_per_group, a.parts_per_block, q.partial,
                          static_cast<int>(blockIdx.x - q.tok_block_begin), blockIdx.y);
}

__device__ __forceinline__ void kvnorm_finish_token(const uint64_t* __restrict__ partial, int groups, int n, int t,
                                                    const double* __restrict__ w2, double* __restrict__ score) {
  U128 s{0, 0};
  for (int g = 0; g < groups; ++g) {
    const uint64_t* p = partial + (static_cast<size_t>(g) * n + t) * 2;
    s = add128(s, U128{p[0], p[1]});
  }
  // RN64(S) then an exact scaling by 2^-48 (the result is 0 or >= 2^-48)
  const double sd = u128_to_double(s) * 0x1p-48;
  score[t] = sd * w2[n - 1 - t];
}

__global__ __launch_bounds__(kThreads) void kvnorm_finish(const uint64_t* __restrict__ partial,
                                                         int groups, int n,
                                                         const double* __restrict__ w2,
                                                         double* __restrict__ score) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (t < n) kvnorm_finish_token(partial, groups, n, t, w2, score);
}

// grid: sum over requests of ceil(n / 256) blocks.  One decay table serves
// every request: entry Delta does not depend on n.
__global__ __launch_bounds__(kThreads) void kvnorm_finish_batch(const ScoreBatchArgs a, const double* __restrict__ w2) {
  const ScoreDesc& q = a.r[score_request_of(a, blockIdx.x, true)];
  const int t = static_cast<int>(blockIdx.x - q.fin_block_begin) * kThreads + threadIdx.x;
  if (t < q.n) kvnorm_finish_token(q.partial, a.groups, q.n, t, w2, q.score);
}

__global__ __launch_bounds__(kThreads) void recency_score_batch(const ScoreBatchArgs a, const double* __restrict__ w1) {
  const ScoreDesc& q = a.r[score_request_of(a, blockIdx.x, true)];
  const int t = static_cast<int>(blockIdx.x - q.fin_block_begin) * kThreads + threadIdx.x;
  if (t < q.n) q.score[t] = w1[q.n - 1 - t];
}

// grid: (token blocks, groups).  Group g's sum is the sum of its
// parts_per_group consecutive partials.
__global__ __launch_bounds__(kThreads) void kvnorm_finish_groups(const uint64_t* __restrict__ partial,
                                                                int parts_per_group, int n,
                                                                const double* __restrict__ w2,
                                                                double* __restrict__ score) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (t >= n) return;
  U128 s{0, 0};
  for (int j = 0; j < parts_per_group; ++j) {
    const uint64_t* p = partial + ((static_cast<size_t>(blockIdx.y) * parts_per_group + j) * n + t) * 2;
    s = add128(s, U128{p[0], p[1]});
  }
  const double sd = u128_to_double(s) * 0x1p-48;
  score[static_cast<size_t>(blockIdx.y) * n + t] = sd * w2[n - 1 - t];
}

// grid: (token blocks, groups)
__global__ __launch_bounds__(kThreads) void recency_score_groups(const double* __restrict__ w1, int n,
                                                                double* __restrict__ score) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (t < n) score[static_cast<size_t>(blockIdx.y) * n + t] = w1[n - 1 - t];
}

__global__ __launch_bounds__(kThreads) void recency_score(const double* __restrict__ w1, int n,
                                                         double* __restrict__ score) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (t < n) score[t] = w1[n - 1 - t];
}

struct KvnormLaunch {
  int pairs, groups, pairs_per_group, blocks_tok;
  int parts_per_block = 1;
};

KvnormLaunch kvnorm_shape(const Geometry& g) {
  KvnormLaunch s;
  s.pairs = g.L * g.H;
  const int tok = kThreads / (g.d / 8);
  s.blocks_tok = (g.n + tok - 1) / tok;
  // enough blocks (about 256 per CU) that many loads are in flight on every
  // CU, and few enough pairs per group that each thread's binary64 sums stay
  // exact
  int groups = (65536 + s.blocks_tok - 1) / s.blocks_tok;
  groups = max(groups, (s.pairs + kMaxPairsPerGroup - 1) / kMaxPairsPerGroup);
  groups = min(min(groups, s.pairs), 32768);  // a grid's y extent stays below 65536
  s.pairs_per_group = (s.pairs + groups - 1) / groups;
  s.groups = (s.pairs + s.pairs_per_group - 1) / s.pairs_per_group;
  return s;
}

// Partials aligned to the groups of a granularity: a group's pairs are
// consecutive (pair p = l * H + h), so parts of pairs_per_part pairs never
// straddle two groups.
KvnormLaunch kvnorm_shape_groups(const Geometry& g, int gran, int* parts_per_group) {
  if (gran == SKV_GROUP_TOKEN) {
    const KvnormLaunch s = kvnorm_shape(g);
    *parts_per_group = s.groups;
    return s;
  }
  KvnormLaunch s;
  s.pairs = g.L * g.H;
  const int tok = kThreads / (g.d / 8);
  s.blocks_tok = (g.n + tok - 1) / tok;
  s.pairs_per_group = (gran == SKV_GROUP_LAYER && g.H <= kMaxPairsPerGroup) ? g.H : 1;
  s.groups = s.pairs / s.pairs_per_group;
  *parts_per_group = gran == SKV_GROUP_LAYER ? g.H / s.pairs_per_group : 1;
  // one part per pair: a block covers several parts (written separately) so
  // that it streams as much as a block of the coarser shapes
  if (s.pairs_per_group == 1) s.parts_per_block = min(8, s.groups);
  return s;
}

}  // namespace

uint64_t kvnorm_scratch_bytes_groups(const Geometry& g, int32_t gran) {
  int ppg;
  const KvnormLaunch s = kvnorm_shape_groups(g, gran, &ppg);
  if (s.pairs_per_group == 1 && ppg == 1) return 0;  // one pair per group: scores written directly
  return static_cast<uint64_t>(s.groups) * g.n * 16u;
}

hipError_t launch_score_kvnorm_groups(const Geometry& g, int32_t gran, int32_t G, const uint16_t* k,
                                      const uint16_t* v, const double* w2, uint64_t* partial, double* score,
                                      hipStream_t stream) {
  int ppg;
  const KvnormLaunch s = kvnorm_shape_groups(g, gran, &ppg);
  const dim3 grid(s.blocks_tok, (s.groups + s.parts_per_block - 1) / s.parts_per_block);
  const int ppb = s.parts_per_block;
  if (s.pairs_per_group == 1) {
    // one pair per part: each block streams a contiguous token run of one
    // pair; a part that is a whole group (per-head maps) writes its scores
    const bool final_scores = ppg == 1;
#define SKV_PAIRS_LAUNCH(D)                                                                                      \
  {                                                                                                             \
    const dim3 pgrid((g.n + kPairRows * (kThreads / (D / 8)) - 1) / (kPairRows * (kThreads / (D / 8))), s.pairs); \
    if (final_scores)                                                                                           \
      kvnorm_partial_pairs<D, kPairRows, true><<<pgrid, kThreads, 0, stream>>>(k, v, g.n, partial, w2, score);  \
    else                                                                                                        \
      kvnorm_partial_pairs<D, kPairRows, false><<<pgrid, kThreads, 0, stream>>>(k, v, g.n, partial, w2, score); \
  }
    switch (g.d) {
      case 32: SKV_PAIRS_LAUNCH(32); break;
      case 64: SKV_PAIRS_LAUNCH(64); break;
      case 128: SKV_PAIRS_LAUNCH(128); break;
      case 256: SKV_PAIRS_LAUNCH(256); break;
      default: return hipErrorInvalidValue;
    }
#undef SKV_PAIRS_LAUNCH
    if (final_scores) return hipGetLastError();
  } else switch (g.d) {
    case 32: kvnorm_partial<32><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    case 64: kvnorm_partial<64><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    case 128: kvnorm_partial<128><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    case 256: kvnorm_partial<256><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 fgrid((g.n + kThreads - 1) / kThreads, G);
  kvnorm_finish_groups<<<fgrid, kThreads, 0, stream>>>(partial, ppg, g.n, w2, score);
  return hipGetLastError();
}

hipError_t launch_score_recency_groups(const Geometry& g, int32_t G, const double* w1, double* score,
                                       hipStream_t stream) {
  const dim3 grid((g.n + kThreads - 1) / kThreads, G);
  recency_score_groups<<<grid, kThreads, 0, stream>>>(w1, g.n, score);
  return hipGetLastError();
}

uint64_t kvnorm_scratch_bytes(const Geometry& g) {
  const KvnormLaunch s = kvnorm_shape(g);
  return static_cast<uint64_t>(s.groups) * g.n * 16u;
}

hipError_t launch_score_kvnorm(const Geometry& g, const uint16_t* k, const uint16_t* v,
                               const double* w2, uint64_t* partial, double* score,
                               hipStream_t stream) {
  const KvnormLaunch s = kvnorm_shape(g);
  const dim3 grid(s.blocks_tok, (s.groups + s.parts_per_block - 1) / s.parts_per_block);
  const int ppb = s.parts_per_block;
  switch (g.d) {
    case 32: kvnorm_partial<32><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    case 64: kvnorm_partial<64><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    case 128: kvnorm_partial<128><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    case 256: kvnorm_partial<256><<<grid, kThreads, 0, stream>>>(k, v, g.n, s.pairs, s.pairs_per_group, ppb, partial); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  kvnorm_finish<<<(g.n + kThreads - 1) / kThreads, kThreads, 0, stream>>>(partial, s.groups, g.n, w2, score);
  return hipGetLastError();
}

void kvnorm_batch_shape(int32_t L, int32_t H, int32_t d, const int32_t* ns, int32_t count, ScoreBatchArgs* a) {
  uint64_t blocks = 0;
  const int tok = kThreads / (d / 8);
  for (int i = 0; i < count; ++i) blocks += (ns[i] + tok - 1) / tok;
  Geometry g{};
  g.L = L;
  g.H = H;
  g.d = d;
  // the single-request shape for a request as long as the whole batch: the
  // same number of workgroups per part, so the launch streams alike
  g.n = static_cast<int32_t>(std::min<uint64_t>(blocks * tok, kMaxTokens));
  const KvnormLaunch s = kvnorm_shape(g);
  a->pairs = s.pairs;
  a->pairs_per_group = s.pairs_per_group;
  a->groups = s.groups;
  a->parts_per_block = s.parts_per_block;
}

hipError_t launch_score_kvnorm_batch(const ScoreBatchArgs& a, int32_t d, const double* w2, hipStream_t stream) {
  const int tok = kThreads / (d / 8);
  uint32_t blocks = 0, fin = 0;
  for (int i = 0; i < a.count; ++i) {
    blocks += (a.r[i].n + tok - 1) / tok;
    fin += (a.r[i].n + kThreads - 1) / kThreads;
  }
  const dim3 grid(blocks, (a.groups + a.parts_per_block - 1) / a.parts_per_block);
  switch (d) {
    case 32: kvnorm_partial_batch<32><<<grid, kThreads, 0, stream>>>(a); break;
    case 64: kvnorm_partial_batch<64><<<grid, kThreads, 0, stream>>>(a); break;
    case 128: kvnorm_partial_batch<128><<<grid, kThreads, 0, stream>>>(a); break;
    case 256: kvnorm_partial_batch<256><<<grid, kThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  kvnorm_finish_batch<<<fin, kThreads, 0, stream>>>(a, w2);
  return hipGetLastError();
}

hipError_t launch_score_recency_batch(const ScoreBatchArgs& a, const double* w1, hipStream_t stream) {
  uint32_t fin = 0;
  for (int i = 0; i < a.count; ++i) fin += (a.r[i].n + kThreads - 1) / kThreads;
  recency_score_batch<<<fin, kThreads, 0, stream>>>(a, w1);
  return hipGetLastError();
}

hipError_t launch_score_recency(const Geometry& g, const double* w1, double* score,
                                hipStream_t stream) {
  recency_score<<<(g.n + kThreads - 1) / kThreads, kThreads, 0, stream>>>(w1, g.n, score);
  return hipGetLastError();
}

}  // namespace skv
