// Attention-mode score (Sec. 3: attention mass aggregated over layers, heads
// and decode observations; Sec. 4.3: I_j = A_j exp(-lambda Delta_j)).
//
// For every (layer l, KV head h) the G = Hq/H query heads of the group give
// M = G*W observation rows q_m (contiguous in q_obs).  With z[m,t] = q_m.k_t/sqrt(d),
//   A_t = (1 / (L*Hq*W)) * sum over (l, h, m) of softmax_t(z[m, :])[t].
// Q.K^T is a dense contraction, so it runs on the matrix cores
// (v_mfma_f32_32x32x16_f16, fp32 accumulation; binary16 products are exact
// in fp32).  A workgroup owns 1024 keys of one (l, h); its four waves take
// one 32-row query tile each (with fewer tiles, the key tiles are split into
// interleaved streams), so the keys are read from HBM once per pass and
// shared by the waves through the caches; the next key tile is loaded while
// the current one is multiplied.
//   attn_stats:   per (l, h, key block) and row, the row maximum and the sum
//                 of exp(z - max) over the block's keys (keys as MFMA rows, so
//                 a lane updates one query's running max and sum: one
//                 exponential per logit; streams merged in order);
//   attn_merge:   per (l, h, row), the blocks merged in key order into
//                 c = max + log(sum);
//   attn_colsum:  recomputes z, p = exp(z - c), and sums p over the rows of
//                 the group for every key (queries as MFMA rows; lane-halves
//                 and waves added in fixed order);
//   attn_finish:  per key, the (l, h) partial sums added in fixed order in
//                 binary64, times 1/(L Hq W) and exp(-lambda Delta).
// Every reduction has a fixed order, so the scores are deterministic; they
// match the binary64 definition to a relative tolerance, not bit for bit.
#include "device_util.h"
#include "skv_internal.h"

namespace skv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kBlockKeys = 1024;              // keys per workgroup
constexpr int kTiles = kBlockKeys / 32;       // 32-key tiles per workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Row of accumulator register r in lane-half hf of a 32x32 MFMA result
// (the column is lane % 32).
__device__ __forceinline__ int acc_row(int r, int hf) { return 8 * (r >> 2) + 4 * hf + (r & 3); }

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Stats of one row, merged: (m, s) stands for s * exp(m); m = -inf means empty.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

// The same in base-2 units scaled by alpha: (m, s) stands for s * 2^(alpha m).
__device__ __forceinline__ void lse_merge2(float& m, float& s, float m2, float s2, float alpha) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;
  s = s * exp2_fast((m - mm) * alpha) + s2 * exp2_fast((m2 - mm) * alpha);
  m = mm;
}

// The 16-byte operand slice of row `row` for MFMA k-step s in lane-half hf:
// elements 16 s + 8 hf .. + 8 (zeros when the row is absent).
template <int D>
__device__ __forceinline__ void load_rows(const uint16_t* base, int row, bool ok, half8 (&out)[D / 16]) {
  const int hf = (threadIdx.x >> 5) & 1;
  const uint16_t* p = base + static_cast<size_t>(ok ? row : 0) * D + 8 * hf;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) out[s] = ok ? __builtin_bit_cast(half8, *reinterpret_cast<const u32x4*>(p + 16 * s)) : half8{};
}

// Work of wave w in round r: query tiles r*4 .. r*4+qg-1 (qg = min(4, MT - 4r))
// are spread over the waves; with fewer than 4 tiles the key tiles of the
// block are split into nstreams interleaved streams so every wave works.
struct WaveRole {
  int qg, nstreams, qtile, stream;
  bool active;
};
__device__ __forceinline__ WaveRole wave_role(int MT, int round, int wave) {
  WaveRole r;
  r.qg = min(4, MT - 4 * round);
  r.nstreams = r.qg == 1 ? 4 : r.qg == 2 ? 2 : 1;
  r.active = wave < r.qg * r.nstreams;
  r.qtile = 4 * round + wave % r.qg;
  r.stream = wave / r.qg;
  return r;
}

template <int N>
__device__ __forceinline__ float tree_max(float (&v)[N]) {
#pragma unroll
  for (int w = N / 2; w >= 1; w /= 2)
#pragma unroll
    for (int i = 0; i < w; ++i) v[i] = fmaxf(v[i], v[i + w]);
  return v[0];
}
template <int N>
__device__ __forceinline__ float tree_sum(float (&v)[N]) {
#pragma unroll
  for (int w = N / 2; w >= 1; w /= 2)
#pragma unroll
    for (int i = 0; i < w; ++i) v[i] = v[i] + v[i + w];
  return v[0];
}

// Online (max, sum) update of one query with the 16 logits of a tile held by
// this lane (y = acc * alpha, base-2 units).  MASK: keys t0 + acc_row >= n
// are excluded.  m is kept in y units.
template <bool MASK>
__device__ __forceinline__ void tile_update(const floatx16& acc, float alpha, int t0, int hf, int n, float& m,
                                            float& sum) {
  float y[16], t[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    y[r] = acc[r] * alpha;
    if (MASK && t0 + acc_row(r, hf) >= n) y[r] = -INFINITY;
    t[r] = y[r];
  }
  const float tmax = tree_max<16>(t);
  if (MASK && tmax == -INFINITY) return;
  const float mn = fmaxf(m, tmax);
#pragma unroll
  for (int r = 0; r < 16; ++r) y[r] = exp2_fast(y[r] - mn);
  sum = sum * exp2_fast(m - mn) + tree_sum<16>(y);
  m = mn;
}

// grid (L*H, key blocks); pstat[(lh * nkb + kb) * Mpad + row] = (max of z, sum of exp(z - max))
// over the block's keys.  The logits are formed transposed (keys as MFMA rows,
// queries as columns), so a lane holds 16 keys of one query and keeps that
// query's running (max, sum) in two registers: one exponential per logit.
template <int D>
__global__ __launch_bounds__(kWaves * 64) void attn_stats(const uint16_t* __restrict__ k,
                                                          const uint16_t* __restrict__ q, int n, int H,
                                                          int Hq, int W, float scale,
                                                          float2* __restrict__ pstat) {
  const int lh = blockIdx.x, kb = blockIdx.y, nkb = gridDim.y;
  const int l = lh / H, h = lh % H, G = Hq / H, M = G * W, MT = (M + 31) / 32, Mpad = MT * 32;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, hf = lane >> 5, j = lane & 31;
  const uint16_t* kbase = k + static_cast<size_t>(lh) * n * D;
  const uint16_t* qbase = q + (static_cast<size_t>(l) * Hq + static_cast<size_t>(h) * G) * W * D;
  const float alpha = scale * kLog2e;
  const int key0 = kb * kBlockKeys;
  __shared__ float2 s_stat[kWaves][32];
  for (int round = 0; 4 * round < MT; ++round) {
    const WaveRole role = wave_role(MT, round, wave);
    if (role.active) {
      half8 qr[D / 16];
      const int qrow = role.qtile * 32 + j;
      load_rows<D>(qbase, qrow, qrow < M, qr);
      float m = -INFINITY, sum = 0.0f;  // m in base-2 units (logit * scale * log2 e)
      // two tiles per step: the second tile's MFMAs run while the first
      // tile's exponentials are computed; the next pair is loaded meanwhile
      const int st = role.nstreams;
      half8 ka[D / 16], kb2[D / 16];
      const int i0 = role.stream;
      load_rows<D>(kbase, key0 + i0 * 32 + j, key0 + i0 * 32 + j < n, ka);
      if (i0 + st < kTiles) load_rows<D>(kbase, key0 + (i0 + st) * 32 + j, key0 + (i0 + st) * 32 + j < n, kb2);
      for (int i = i0; i < kTiles && key0 + i * 32 < n; i += 2 * st) {  // wave-uniform bounds
        const int i1 = i + st;
        const bool has1 = i1 < kTiles && key0 + i1 * 32 < n;
        floatx16 a0{}, a1{};
#pragma unroll
        for (int s = 0; s < D / 16; ++s) a0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(ka[s], qr[s], a0, 0, 0, 0);
        if (has1) {
#pragma unroll
          for (int s = 0; s < D / 16; ++s) a1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(kb2[s], qr[s], a1, 0, 0, 0);
        }
        const int n0 = i + 2 * st, n1 = i + 3 * st;
        if (n0 < kTiles) load_rows<D>(kbase, key0 + n0 * 32 + j, key0 + n0 * 32 + j < n, ka);
        if (n1 < kTiles) load_rows<D>(kbase, key0 + n1 * 32 + j, key0 + n1 * 32 + j < n, kb2);
        const int t0 = key0 + i * 32;
        if (t0 + 32 <= n) tile_update<false>(a0, alpha, t0, hf, n, m, sum);
        else tile_update<true>(a0, alpha, t0, hf, n, m, sum);
        if (has1) {
          const int t1 = key0 + i1 * 32;
          if (t1 + 32 <= n) tile_update<false>(a1, alpha, t1, hf, n, m, sum);
          else tile_update<true>(a1, alpha, t1, hf, n, m, sum);
        }
      }
      // the two lane-halves saw different keys of the same query
      lse_merge2(m, sum, __shfl_xor(m, 32), __shfl_xor(sum, 32), 1.0f);
      if (hf == 0) s_stat[wave][j] = float2{m, sum};
    }
    __syncthreads();
    // merge the streams of each query in stream order; m to z units
    for (int idx = threadIdx.x; idx < role.qg * 32; idx += kWaves * 64) {
      const int qt = idx / 32, jj = idx % 32;
      float mm = -INFINITY, ss = 0.0f;
      for (int st = 0; st < role.nstreams; ++st) {
        const float2 v = s_stat[st * role.qg + qt][jj];
        lse_merge2(mm, ss, v.x, v.y, 1.0f);
      }
      // (max, sum) in logit units: max z = m / log2(e)
      pstat[(static_cast<size_t>(lh) * nkb + kb) * Mpad + (4 * round + qt) * 32 + jj] = float2{mm * kLn2, ss};
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void attn_merge(const float2* __restrict__ pstat, int LH, int nkb, int Mpad,
                                                  int M, float* __restrict__ cstat) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= LH * Mpad) return;
  const int lh = idx / Mpad, row = idx % Mpad;
  float mm = -INFINITY, ss = 0.0f;
  if (row < M)
    for (int kb = 0; kb < nkb; ++kb) {
      const float2 p = pstat[(static_cast<size_t>(lh) * nkb + kb) * Mpad + row];
      lse_merge(mm, ss, p.x, p.y);
    }
  cstat[idx] = row < M ? mm + __logf(ss) : INFINITY;  // padding rows: exp(z - inf) = 0
}

// grid (L*H, key blocks); colsum[lh * n + t] = sum over the group's rows of p[row, t].
// Logits with queries as MFMA rows: a lane holds 16 rows of one key and sums
// their probabilities; the lane-halves and the waves (query tiles and rounds)
// are added in fixed order through shared memory.
template <int D>
__global__ __launch_bounds__(kWaves * 64) void attn_colsum(const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ q, int n, int H,
                                                           int Hq, int W, float scale,
                                                           const float* __restrict__ cstat,
                                                           float* __restrict__ colsum) {
  const int lh = blockIdx.x, kb = blockIdx.y;
  const int l = lh / H, h = lh % H, G = Hq / H, M = G * W, MT = (M + 31) / 32, Mpad = MT * 32;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, hf = lane >> 5, j = lane & 31;
  const uint16_t* kbase = k + static_cast<size_t>(lh) * n * D;
  const uint16_t* qbase = q + (static_cast<size_t>(l) * Hq + static_cast<size_t>(h) * G) * W * D;
  const float alpha = scale * kLog2e;
  const int key0 = kb * kBlockKeys;
  __shared__ float s_col[kWaves][kBlockKeys];
  for (int idx = threadIdx.x; idx < kWaves * kBlockKeys; idx += kWaves * 64) (&s_col[0][0])[idx] = 0.0f;
  __syncthreads();
  for (int round = 0; 4 * round < MT; ++round) {
    const WaveRole role = wave_role(MT, round, wave);
    if (!role.active) continue;
    half8 qr[D / 16];
    const int qrow = role.qtile * 32 + j;
    load_rows<D>(qbase, qrow, qrow < M, qr);
    float beta[16];  // c * log2(e) of the lane's 16 rows; +inf for padding rows
#pragma unroll
    for (int r = 0; r < 16; ++r)
      beta[r] = cstat[static_cast<size_t>(lh) * Mpad + role.qtile * 32 + acc_row(r, hf)] * kLog2e;
    // sum over the lane's 16 rows of p = 2^(acc * alpha - beta), then over both lane-halves
    auto colsum_tile = [&](const floatx16& acc, int i) {
      float e[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) e[r] = exp2_fast(__builtin_fmaf(acc[r], alpha, -beta[r]));
      float p = tree_sum<16>(e);
      p += __shfl_xor(p, 32);  // the other lane-half holds the other 16 rows
      if (hf == 0) s_col[wave][i * 32 + j] += p;
    };
    const int st = role.nstreams;
    half8 ka[D / 16], kb2[D / 16];
    const int i0 = role.stream;
    load_rows<D>(kbase, key0 + i0 * 32 + j, key0 + i0 * 32 + j < n, ka);
    if (i0 + st < kTiles) load_rows<D>(kbase, key0 + (i0 + st) * 32 + j, key0 + (i0 + st) * 32 + j < n, kb2);
    for (int i = i0; i < kTiles && key0 + i * 32 < n; i += 2 * st) {  // wave-uniform bounds
      const int i1 = i + st;
      const bool has1 = i1 < kTiles && key0 + i1 * 32 < n;
      floatx16 a0{}, a1{};
#pragma unroll
      for (int s = 0; s < D / 16; ++s) a0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(qr[s], ka[s], a0, 0, 0, 0);
      if (has1) {
#pragma unroll
        for (int s = 0; s < D / 16; ++s) a1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(qr[s], kb2[s], a1, 0, 0, 0);
      }
      const int n0 = i + 2 * st, n1 = i + 3 * st;
      if (n0 < kTiles) load_rows<D>(kbase, key0 + n0 * 32 + j, key0 + n0 * 32 + j < n, ka);
      if (n1 < kTiles) load_rows<D>(kbase, key0 + n1 * 32 + j, key0 + n1 * 32 + j < n, kb2);
      colsum_tile(a0, i);
      if (has1) colsum_tile(a1, i1);
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < kBlockKeys; idx += kWaves * 64) {
    const int t = key0 + idx;
    if (t < n) colsum[static_cast<size_t>(lh) * n + t] = ((s_col[0][idx] + s_col[1][idx]) + s_col[2][idx]) + s_col[3][idx];
  }
}

__global__ __launch_bounds__(256) void attn_finish(const float* __restrict__ colsum, int LH, int n,
                                                   double inv_rows, const double* __restrict__ w1,
                                                   double* __restrict__ score) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= n) return;
  double a = 0.0;
  int lh = 0;
  for (; lh + 8 <= LH; lh += 8) {  // eight loads in flight, added in (l, h) order
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = colsum[static_cast<size_t>(lh + u) * n + t];
#pragma unroll
    for (int u = 0; u < 8; ++u) a += static_cast<double>(v[u]);
  }
  for (; lh < LH; ++lh) a += static_cast<double>(colsum[static_cast<size_t>(lh) * n + t]);
  score[t] = (a * inv_rows) * w1[n - 1 - t];
}

// grid: (token blocks, groups).  Group g sums the column sums of its
// pairs_per_group consecutive (layer, KV head) pairs.
__global__ __launch_bounds__(256) void attn_finish_groups(const float* __restrict__ colsum, int pairs_per_group,
                                                          int n, double inv_rows, const double* __restrict__ w1,
                                                          double* __restrict__ score) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= n) return;
  double a = 0.0;
  const size_t lh0 = static_cast<size_t>(blockIdx.y) * pairs_per_group;
  for (int j = 0; j < pairs_per_group; ++j) a += static_cast<double>(colsum[(lh0 + j) * n + t]);
  score[static_cast<size_t>(blockIdx.y) * n + t] = (a * inv_rows) * w1[n - 1 - t];
}

inline uint64_t up256(uint64_t x) { return (x + 255u) / 256u * 256u; }

struct AttnShape {
  int LH, M, Mpad, nkb;
  uint64_t pstat_bytes, cstat_bytes, colsum_bytes;
};

AttnShape attn_shape(const Geometry& g, int32_t Hq, int32_t W) {
  AttnShape s;
  s.LH = g.L * g.H;
  s.M = (Hq / g.H) * W;
  s.Mpad = (s.M + 31) / 32 * 32;
  s.nkb = (g.n + kBlockKeys - 1) / kBlockKeys;
  s.pstat_bytes = up256(static_cast<uint64_t>(s.LH) * s.nkb * s.Mpad * sizeof(float2));
  s.cstat_bytes = up256(static_cast<uint64_t>(s.LH) * s.Mpad * sizeof(float));
  s.colsum_bytes = up256(static_cast<uint64_t>(s.LH) * g.n * sizeof(float));
  return s;
}

template <int D>
hipError_t launch_d(const Geometry& g, const AttnShape& s, int Hq, int W, const uint16_t* k, const uint16_t* q,
                    float2* pstat, float* cstat, float* colsum, hipStream_t stream) {
  const float scale = static_cast<float>(1.0 / sqrt(static_cast<double>(D)));
  const dim3 grid(s.LH, s.nkb);
  attn_stats<D><<<grid, kWaves * 64, 0, stream>>>(k, q, g.n, g.H, Hq, W, scale, pstat);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_merge<<<(s.LH * s.Mpad + 255) / 256, 256, 0, stream>>>(pstat, s.LH, s.nkb, s.Mpad, s.M, cstat);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_colsum<D><<<grid, kWaves * 64, 0, stream>>>(k, q, g.n, g.H, Hq, W, scale, cstat, colsum);
  return hipGetLastError();
}

}  // namespace

uint64_t attn_scratch_bytes(const Geometry& g, int32_t Hq, int32_t W) {
  const AttnShape s = attn_shape(g, Hq, W);
  return s.pstat_bytes + s.cstat_bytes + s.colsum_bytes;
}

hipError_t launch_score_attn(const Geometry& g, int32_t Hq, int32_t W, const uint16_t* k, const uint16_t* q,
                             const double* w1, void* scratch, double* score, hipStream_t stream) {
  const AttnShape s = attn_shape(g, Hq, W);
  uint8_t* base = static_cast<uint8_t*>(scratch);
  float2* pstat = reinterpret_cast<float2*>(base);
  float* cstat = reinterpret_cast<float*>(base + s.pstat_bytes);
  float* colsum = reinterpret_cast<float*>(base + s.pstat_bytes + s.cstat_bytes);
  hipError_t e;
  switch (g.d) {
    case 32: e = launch_d<32>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    case 64: e = launch_d<64>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    case 128: e = launch_d<128>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    case 256: e = launch_d<256>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  const double inv_rows = 1.0 / (static_cast<double>(g.L) * Hq * W);
  attn_finish<<<(g.n + 255) / 256, 256, 0, stream>>>(colsum, s.LH, g.n, inv_rows, w1, score);
  return hipGetLastError();
}

hipError_t launch_score_attn_groups(const Geometry& g, int32_t gran, int32_t G, int32_t Hq, int32_t W,
                                    const uint16_t* k, const uint16_t* q, const double* w1, void* scratch,
                                    double* score, hipStream_t stream) {
  const AttnShape s = attn_shape(g, Hq, W);
  uint8_t* base = static_cast<uint8_t*>(scratch);
  float2* pstat = reinterpret_cast<float2*>(base);
  float* cstat = reinterpret_cast<float*>(base + s.pstat_bytes);
  float* colsum = reinterpret_cast<float*>(base + s.pstat_bytes + s.cstat_bytes);
  hipError_t e;
  switch (g.d) {
    case 32: e = launch_d<32>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    case 64: e = launch_d<64>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    case 128: e = launch_d<128>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    case 256: e = launch_d<256>(g, s, Hq, W, k, q, pstat, cstat, colsum, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  const int pairs_per_group = s.LH / G;  // L*H, H or 1
  const double inv_rows = 1.0 / (static_cast<double>(pairs_per_group) * (Hq / g.H) * W);
  const dim3 grid((g.n + 255) / 256, G);
  attn_finish_groups<<<grid, 256, 0, stream>>>(colsum, pairs_per_group, g.n, inv_rows, w1, score);
  return hipGetLastError();
}

}  // namespace skv
