// Tier assignment: sink pinning + importance-sorted cuts (Sec. 2.3 Prop. 1;
// Sec. 4.4; Algorithm 1 steps 2-3).
//
// Non-sink token t carries the 64-bit ranking key
//   c_t = ((bits(score_t) >> 20) << 21) | t     (score <= 0 or NaN ranks as +0),
// all distinct.  With the tier counts fixed by the plan, token t gets FP16 iff
// c_t is among the n16 largest keys, INT8 iff among the next n8, INT4 iff
// among the next n4, DROP otherwise.  The kernel finds the three cut keys
// T1 >= T2 >= T3 (the n16-th, (n16+n8)-th and (n16+n8+n4)-th largest) by one
// radix select per cut over 11-bit digits (6 passes), all three sharing each
// pass over the keys, then classifies every token against them.
//   * One workgroup of 1024 threads.  Keys are recomputed from the scores on
//     every pass (the scores stay in L2), eight loads in flight per thread.
//   * Cuts with the same decided prefix share one LDS histogram.
//   * Consecutive keys of a thread that fall in the same bin are counted
//     before one LDS atomic, so the first pass (where most keys share the
//     binary64 exponent, hence the top digit) does not serialize on one bin.
#include "device_util.h"
#include "skv_internal.h"

namespace skv {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kDigit = 11;
constexpr int kBins = 1 << kDigit;
constexpr int kPasses = 6;   // 5 digits of 11 bits and one of 9
constexpr int kBatch = 8;  // scores loaded per thread before they are counted

__device__ __forceinline__ uint64_t rank_key(double s, int t) {
  uint64_t bits = 0;
  if (s > 0.0) bits = __builtin_bit_cast(uint64_t, s);
  return ((bits >> 20) << 21) | static_cast<uint64_t>(static_cast<uint32_t>(t));
}

// Adds `count` keys to bin `bin` of histogram h unless count is zero.
__device__ __forceinline__ void flush(uint32_t* h, uint32_t bin, uint32_t count) {
  if (count) atomicAdd(&h[bin], count);
}

// One pass: histogram of the digit at `shift` over the keys whose decided
// bits equal the prefix of each active cut group.
struct RunCounter {
  uint32_t bin = 0, count = 0;
  __device__ __forceinline__ void add(uint32_t* h, uint32_t b) {
    if (b != bin) {
      flush(h, bin, count);
      bin = b;
      count = 0;
    }
    ++count;
  }
};

// The whole assignment of one score row by one 1024-thread workgroup.
__device__ __forceinline__ void assign_row(const double* __restrict__ score, uint8_t* __restrict__ tier, int n,
                                           int n_sink, int n16, int n8, int n4) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[3][kBins];
  __shared__ uint64_t s_prefix[3];
  __shared__ uint32_t s_rank[3];  // remaining rank (1-based) inside the current prefix
  __shared__ int s_group[3];      // which histogram a cut reads
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t cut_rank[3] = {static_cast<uint32_t>(n16), static_cast<uint32_t>(n16 + n8),
                                static_cast<uint32_t>(n16 + n8 + n4)};
  if (tid < 3) {
    s_prefix[tid] = 0;
    s_rank[tid] = tid == 0 ? cut_rank[0] : tid == 1 ? cut_rank[1] : cut_rank[2];
  }
  __syncthreads();

  for (int pass = 0; pass < kPasses; ++pass) {
    const int hi_bit = 64 - kDigit * pass;
    const int shift = hi_bit > kDigit ? hi_bit - kDigit : 0;
    const uint32_t mask = (1u << (hi_bit - shift)) - 1u;
    const uint64_t decided = pass == 0 ? 0ull : (~0ull << hi_bit);
    if (tid < 3) {
      int grp = tid;
      for (int j = 0; j < tid; ++j)
        if (s_rank[j] != 0 && s_prefix[j] == s_prefix[tid]) { grp = j; break; }
      s_group[tid] = grp;
    }
    for (int i = tid; i < 3 * kBins; i += kSelThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    const bool act0 = s_rank[0] != 0 && s_group[0] == 0;
    const bool act1 = s_rank[1] != 0 && s_group[1] == 1;
    const bool act2 = s_rank[2] != 0 && s_group[2] == 2;
    const uint64_t pre0 = s_prefix[0], pre1 = s_prefix[1], pre2 = s_prefix[2];
    RunCounter r0, r1, r2;
    for (int base = n_sink + tid; base < n; base += kBatch * kSelThreads) {
      double sc[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int t = base + u * kSelThreads;
        sc[u] = t < n ? score[t] : 0.0;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int t = base + u * kSelThreads;
        if (t >= n) break;
        const uint64_t c = rank_key(sc[u], t);
        const uint32_t bin = static_cast<uint32_t>(c >> shift) & mask;
        const uint64_t hi = c & decided;
        if (act0 && hi == pre0) r0.add(hist[0], bin);
        if (act1 && hi == pre1) r1.add(hist[1], bin);
        if (act2 && hi == pre2) r2.add(hist[2], bin);
      }
    }
    flush(hist[0], r0.bin, r0.count);
    flush(hist[1], r1.bin, r1.count);
    flush(hist[2], r2.bin, r2.count);
    __syncthreads();
    // wave j walks cut j's histogram from the top bin down and picks the bin
    // that holds its remaining rank (32 bins per lane)
    if (wave < 3 && s_rank[wave] != 0) {
      const int j = wave;
      constexpr int kPer = kBins / 64;  // 32 consecutive bins per lane, read 4 at a time
      const u32x4* h4 = reinterpret_cast<const u32x4*>(hist[s_group[j]]);
      const int b0 = kBins - kPer * (lane + 1);  // this lane's lowest bin; lane 0 holds the top
      u32x4 c4[kPer / 4];
      uint32_t sum = 0;
#pragma unroll
      for (int i = 0; i < kPer / 4; ++i) {
        c4[i] = h4[b0 / 4 + i];
        sum += c4[i].x + c4[i].y + c4[i].z + c4[i].w;
      }
      uint32_t inc = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = static_cast<uint32_t>(__shfl_up(static_cast<int>(inc), o));
        if (lane >= o) inc += y;
      }
      uint32_t run = inc - sum;  // keys in the bins above this lane's
      const uint32_t want = s_rank[j];
      if (run < want && want <= run + sum) {
        const uint64_t prefix = s_prefix[j];
#pragma unroll
        for (int i = kPer / 4 - 1; i >= 0; --i) {  // descending bins
          const uint32_t cs[4] = {c4[i].w, c4[i].z, c4[i].y, c4[i].x};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int b = b0 + 4 * i + (3 - e);
            if (run < want && want <= run + cs[e]) {
              s_prefix[j] = prefix | (static_cast<uint64_t>(b) << shift);
              s_rank[j] = want - run;
            }
            run += cs[e];
          }
        }
      }
    }
    __syncthreads();
  }

  // s_prefix[j] is now the cut key itself (keys are distinct); a cut of rank 0
  // admits no key.
  const uint64_t T1 = s_prefix[0], T2 = s_prefix[1], T3 = s_prefix[2];
  const bool has1 = cut_rank[0] != 0, has2 = cut_rank[1] != 0, has3 = cut_rank[2] != 0;
  for (int t = tid; t < n; t += kSelThreads) {
    uint8_t tr = kFP16;  // sinks
    if (t >= n_sink) {
      const uint64_t c = rank_key(score[t], t);
      tr = (has1 && c >= T1) ? kFP16 : (has2 && c >= T2) ? kINT8 : (has3 && c >= T3) ? kINT4 : kDROP;
    }
    tier[t] = tr;
  }
}

__global__ __launch_bounds__(kSelThreads) void assign_tiers(const double* __restrict__ score,
                                                            uint8_t* __restrict__ tier, int n,
                                                            int n_sink, int n16, int n8, int n4) {
  assign_row(score, tier, n, n_sink, n16, n8, n4);
}

// grid: one workgroup per group; plan counts from the group table
// (u32 [sinks, fp16, int8, int4, ...], 32 bytes per group).
__global__ __launch_bounds__(kSelThreads) void assign_tiers_groups(const double* __restrict__ score,
                                                                   uint8_t* __restrict__ tier, int n,
                                                                   const uint32_t* __restrict__ group_table) {
  const uint32_t* e = group_table + 8 * blockIdx.x;
  const size_t row = static_cast<size_t>(blockIdx.x) * n;
  assign_row(score + row, tier + row, n, static_cast<int>(e[0]), static_cast<int>(e[1]), static_cast<int>(e[2]),
             static_cast<int>(e[3]));
}

}  // namespace

hipError_t launch_assign(const Geometry& g, const double* score, uint8_t* tier,
                         hipStream_t stream) {
  assign_tiers<<<1, kSelThreads, 0, stream>>>(score, tier, g.n, g.n_sink, g.n16, g.n8, g.n4);
  return hipGetLastError();
}

hipError_t launch_assign_groups(int32_t G, int32_t n, const uint32_t* group_table, const double* score,
                                uint8_t* tier, hipStream_t stream) {
  assign_tiers_groups<<<G, kSelThreads, 0, stream>>>(score, tier, n, group_table);
  return hipGetLastError();
}

}  // namespace skv
