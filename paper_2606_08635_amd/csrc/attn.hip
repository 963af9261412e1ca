// Attention-mode score (Sec. 3: attention mass aggregated over layers, heads
// and decode observations; Sec. 4.3: I_j = A_j exp(-lambda Delta_j)).
//
// For every (layer l, KV head h) the G = Hq/H query heads of the group give
// M = G*W observation rows q_m (contiguous in q_obs).  With z[m,t] = q_m.k_t/sqrt(d),
//   A_t = (1 / (L*Hq*W)) * sum over (l, h, m) of softmax_t(z[m, :])[t].
// Q.K^T is a dense contraction, so it runs on the matrix cores
// (v_mfma_f32_32x32x16_f16: a 32-row block of queries times a 32-key tile,
// fp32 accumulation; binary16 products are exact in fp32).
//   attn_stats:   per (l, h, key block) and row, the row maximum and the sum
//                 of exp(z - max) over the block's keys (lane-local online
//                 update, one lane merge at the end, waves merged in order);
//   attn_merge:   per (l, h, row), the blocks merged in key order into
//                 c = max + log(sum);
//   attn_colsum:  recomputes z, p = exp(z - c), and sums p over the rows of
//                 the group for every key (one write per (l, h, key));
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
constexpr int kTilesPerWave = 4;                        // 32-key tiles per wave
constexpr int kBlockKeys = kWaves * kTilesPerWave * 32;  // 512 keys per workgroup

// Row of accumulator register r in lane-half hf of a 32x32 MFMA result
// (the column is lane % 32).
__device__ __forceinline__ int acc_row(int r, int hf) { return 8 * (r >> 2) + 4 * hf + (r & 3); }

// Stats of one row, merged: (m, s) stands for s * exp(m); m = -inf means empty.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

template <int D>
__device__ __forceinline__ half8 load_row16(const uint16_t* row, int col, bool ok) {
  if (!ok) return half8{};
  return __builtin_bit_cast(half8, ld_nt16(row + col));
}

// Q operand of M-tile `mt`, K-step s: row mt*32 + lane%32, columns 16s + 8hf .. +8.
template <int D, int MTG>
__device__ __forceinline__ void load_q(const uint16_t* q, int M, int mt0, int mt_count, half8 (&qr)[MTG][D / 16]) {
  const int i = threadIdx.x & 31, hf = (threadIdx.x >> 5) & 1;
#pragma unroll
  for (int a = 0; a < MTG; ++a) {
    const int row = (mt0 + a) * 32 + i;
    const bool ok = a < mt_count && row < M;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) qr[a][s] = load_row16<D>(q + static_cast<size_t>(ok ? row : 0) * D, 16 * s + 8 * hf, ok);
  }
}

template <int D, int MTG>
__device__ __forceinline__ void logits(const half8 (&qr)[MTG][D / 16], const half8 (&kr)[D / 16], int mt_count,
                                       floatx16 (&acc)[MTG]) {
#pragma unroll
  for (int a = 0; a < MTG; ++a) {
    acc[a] = floatx16{};
    if (a < mt_count) {
#pragma unroll
      for (int s = 0; s < D / 16; ++s) acc[a] = __builtin_amdgcn_mfma_f32_32x32x16_f16(qr[a][s], kr[s], acc[a], 0, 0, 0);
    }
  }
}

template <int D>
__device__ __forceinline__ void load_k(const uint16_t* kbase, int n, int t, half8 (&kr)[D / 16]) {
  const int hf = (threadIdx.x >> 5) & 1;
  const bool ok = t < n;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) kr[s] = load_row16<D>(kbase + static_cast<size_t>(ok ? t : 0) * D, 16 * s + 8 * hf, ok);
}

// grid (L*H, key blocks); scratch pstat[(lh * nkb + kb) * Mpad + row] = (max, sum)
template <int D, int MTG>
__global__ __launch_bounds__(kWaves * 64) void attn_stats(const uint16_t* __restrict__ k,
                                                          const uint16_t* __restrict__ q, int n, int H,
                                                          int Hq, int W, float scale,
                                                          float2* __restrict__ pstat) {
  const int lh = blockIdx.x, kb = blockIdx.y, nkb = gridDim.y;
  const int l = lh / H, h = lh % H, G = Hq / H, M = G * W, MT = (M + 31) / 32, Mpad = MT * 32;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, hf = lane >> 5;
  const uint16_t* kbase = k + static_cast<size_t>(lh) * n * D;
  const uint16_t* qbase = q + (static_cast<size_t>(l) * Hq + static_cast<size_t>(h) * G) * W * D;
  __shared__ float2 s_stat[kWaves][256];
  for (int mt0 = 0; mt0 < MT; mt0 += MTG) {
    const int mt_count = min(MTG, MT - mt0);
    half8 qr[MTG][D / 16];
    load_q<D, MTG>(qbase, M, mt0, mt_count, qr);
    float m[MTG][16], s[MTG][16];
#pragma unroll
    for (int a = 0; a < MTG; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) { m[a][r] = -INFINITY; s[a][r] = 0.0f; }
    for (int i = 0; i < kTilesPerWave; ++i) {
      const int t0 = (kb * kWaves * kTilesPerWave + wave * kTilesPerWave + i) * 32;
      const int t = t0 + (lane & 31);
      half8 kr[D / 16];
      load_k<D>(kbase, n, t, kr);
      floatx16 acc[MTG];
      logits<D, MTG>(qr, kr, mt_count, acc);
#pragma unroll
      for (int a = 0; a < MTG; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = (mt0 + a) * 32 + acc_row(r, hf);
          if (a < mt_count && row < M && t < n) {
            const float z = acc[a][r] * scale;
            const float e = __expf(-fabsf(z - m[a][r]));  // one exponential per logit
            if (z > m[a][r]) { s[a][r] = s[a][r] * e + 1.0f; m[a][r] = z; }
            else { s[a][r] += e; }
          }
        }
    }
    // merge the 32 lanes that share a lane-half (same rows, different keys)
#pragma unroll
    for (int a = 0; a < MTG; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
#pragma unroll
        for (int o = 1; o < 32; o <<= 1) {
          const float m2 = __shfl_xor(m[a][r], o), s2 = __shfl_xor(s[a][r], o);
          lse_merge(m[a][r], s[a][r], m2, s2);
        }
        if ((lane & 31) == 0 && a < mt_count) s_stat[wave][(mt0 + a) * 32 + acc_row(r, hf) - mt0 * 32] = float2{m[a][r], s[a][r]};
      }
    __syncthreads();
    // the four waves cover consecutive key ranges: merge them in order
    for (int row = threadIdx.x; row < mt_count * 32; row += kWaves * 64) {
      float mm = -INFINITY, ss = 0.0f;
      for (int w = 0; w < kWaves; ++w) lse_merge(mm, ss, s_stat[w][row].x, s_stat[w][row].y);
      pstat[(static_cast<size_t>(lh) * nkb + kb) * Mpad + mt0 * 32 + row] = float2{mm, ss};
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

// grid (L*H, key blocks); colsum[lh * n + t] = sum over the group's rows of p[row, t]
template <int D, int MTG>
__global__ __launch_bounds__(kWaves * 64) void attn_colsum(const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ q, int n, int H,
                                                           int Hq, int W, float scale,
                                                           const float* __restrict__ cstat,
                                                           float* __restrict__ colsum) {
  const int lh = blockIdx.x, kb = blockIdx.y;
  const int l = lh / H, h = lh % H, G = Hq / H, M = G * W, MT = (M + 31) / 32, Mpad = MT * 32;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, hf = lane >> 5;
  const uint16_t* kbase = k + static_cast<size_t>(lh) * n * D;
  const uint16_t* qbase = q + (static_cast<size_t>(l) * Hq + static_cast<size_t>(h) * G) * W * D;
  float col[kTilesPerWave];
#pragma unroll
  for (int i = 0; i < kTilesPerWave; ++i) col[i] = 0.0f;
  for (int mt0 = 0; mt0 < MT; mt0 += MTG) {
    const int mt_count = min(MTG, MT - mt0);
    half8 qr[MTG][D / 16];
    load_q<D, MTG>(qbase, M, mt0, mt_count, qr);
    float c[MTG][16];
#pragma unroll
    for (int a = 0; a < MTG; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = (mt0 + a) * 32 + acc_row(r, hf);
        c[a][r] = (a < mt_count) ? cstat[static_cast<size_t>(lh) * Mpad + row] : INFINITY;
      }
#pragma unroll
    for (int i = 0; i < kTilesPerWave; ++i) {
      const int t0 = (kb * kWaves * kTilesPerWave + wave * kTilesPerWave + i) * 32;
      const int t = t0 + (lane & 31);
      half8 kr[D / 16];
      load_k<D>(kbase, n, t, kr);
      floatx16 acc[MTG];
      logits<D, MTG>(qr, kr, mt_count, acc);
      float sum = 0.0f;
#pragma unroll
      for (int a = 0; a < MTG; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += __expf(acc[a][r] * scale - c[a][r]);
      col[i] += sum;
    }
  }
#pragma unroll
  for (int i = 0; i < kTilesPerWave; ++i) {
    const float total = col[i] + __shfl_xor(col[i], 32);  // the two lane-halves hold different rows
    const int t = (kb * kWaves * kTilesPerWave + wave * kTilesPerWave + i) * 32 + (lane & 31);
    if (lane < 32 && t < n) colsum[static_cast<size_t>(lh) * n + t] = total;
  }
}

__global__ __launch_bounds__(256) void attn_finish(const float* __restrict__ colsum, int LH, int n,
                                                   double inv_rows, const double* __restrict__ w1,
                                                   double* __restrict__ score) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= n) return;
  double a = 0.0;
  for (int lh = 0; lh < LH; ++lh) a += static_cast<double>(colsum[static_cast<size_t>(lh) * n + t]);
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
  constexpr int MTG = 2;  // 32-row query tiles held in registers at a time
  const float scale = static_cast<float>(1.0 / sqrt(static_cast<double>(D)));
  const dim3 grid(s.LH, s.nkb);
  attn_stats<D, MTG><<<grid, kWaves * 64, 0, stream>>>(k, q, g.n, g.H, Hq, W, scale, pstat);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_merge<<<(s.LH * s.Mpad + 255) / 256, 256, 0, stream>>>(pstat, s.LH, s.nkb, s.Mpad, s.M, cstat);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_colsum<D, MTG><<<grid, kWaves * 64, 0, stream>>>(k, q, g.n, g.H, Hq, W, scale, cstat, colsum);
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
