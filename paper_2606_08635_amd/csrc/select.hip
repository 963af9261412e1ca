// Tier assignment: sink pinning + importance-sorted cuts (Sec. 2.3 Prop. 1;
// Sec. 4.4; Algorithm 1 steps 2-3).
//
// Non-sink token t carries the 64-bit ranking key
//   c_t = ((bits(score_t) >> 20) << 21) | t     (score <= 0 or NaN ranks as +0),
// all distinct.  With the tier counts fixed by the plan, token t gets FP16 iff
// c_t is among the n16 largest keys, INT8 iff among the next n8, INT4 iff
// among the next n4, DROP otherwise.  The kernel finds the three cut keys
// T1 >= T2 >= T3 (the n16-th, (n16+n8)-th and (n16+n8+n4)-th largest) by one
// radix select per cut over 8-bit digits, all three sharing each pass over the
// keys, then classifies every token against them.  One workgroup of 1024
// threads; the keys are recomputed from the scores on every pass, so no
// scratch memory is needed.
#include "device_util.h"
#include "skv_internal.h"

namespace skv {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kBins = 256;

__device__ __forceinline__ uint64_t rank_key(double s, int t) {
  uint64_t bits = 0;
  if (s > 0.0) bits = __builtin_bit_cast(uint64_t, s);
  return ((bits >> 20) << 21) | static_cast<uint64_t>(static_cast<uint32_t>(t));
}

__global__ __launch_bounds__(kSelThreads) void assign_tiers(const double* __restrict__ score,
                                                            uint8_t* __restrict__ tier, int n,
                                                            int n_sink, int n16, int n8, int n4) {
  __shared__ uint32_t hist[3][kBins];
  __shared__ uint64_t s_prefix[3];
  __shared__ uint32_t s_rank[3];  // remaining rank (1-based) inside the current prefix
  __shared__ int s_group[3];      // which histogram a cut reads
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t cut_rank[3] = {static_cast<uint32_t>(n16), static_cast<uint32_t>(n16 + n8),
                                static_cast<uint32_t>(n16 + n8 + n4)};
  if (tid < 3) {
    s_prefix[tid] = 0;
    s_rank[tid] = cut_rank[tid];
  }
  __syncthreads();

  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    const uint64_t decided = pass == 0 ? 0ull : (~0ull << (shift + 8));
    // cuts with the same decided prefix share one histogram
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
    for (int t = n_sink + tid; t < n; t += kSelThreads) {
      const uint64_t c = rank_key(score[t], t);
      const uint32_t bin = static_cast<uint32_t>(c >> shift) & (kBins - 1);
      const uint64_t hi = c & decided;
      if (act0 && hi == pre0) atomicAdd(&hist[0][bin], 1u);
      if (act1 && hi == pre1) atomicAdd(&hist[1][bin], 1u);
      if (act2 && hi == pre2) atomicAdd(&hist[2][bin], 1u);
    }
    __syncthreads();
    // wave j walks cut j's histogram from the top bin down and picks the bin
    // that holds its remaining rank
    if (wave < 3 && s_rank[wave] != 0) {
      const int j = wave;
      const uint32_t* h = hist[s_group[j]];
      uint32_t c[4], sum = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        c[i] = h[kBins - 1 - (lane * 4 + i)];
        sum += c[i];
      }
      uint32_t inc = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = static_cast<uint32_t>(__shfl_up(static_cast<int>(inc), o));
        if (lane >= o) inc += y;
      }
      uint32_t run = inc - sum;  // keys in bins above this lane's four
      const uint32_t want = s_rank[j];
      const uint64_t prefix = s_prefix[j];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (run < want && want <= run + c[i]) {
          s_prefix[j] = prefix | (static_cast<uint64_t>(kBins - 1 - (lane * 4 + i)) << shift);
          s_rank[j] = want - run;
        }
        run += c[i];
      }
    }
    __syncthreads();
  }

  // s_prefix[j] is now the cut key itself (keys are distinct); a cut of rank 0
  // admits no key.
  const uint64_t T1 = s_prefix[0], T2 = s_prefix[1], T3 = s_prefix[2];
  const bool has1 = cut_rank[0] != 0, has2 = cut_rank[1] != 0, has3 = cut_rank[2] != 0;
  for (int t = tid; t < n; t += kSelThreads) {
    uint8_t tr;
    if (t < n_sink) {
      tr = kFP16;
    } else {
      const uint64_t c = rank_key(score[t], t);
      tr = (has1 && c >= T1) ? kFP16 : (has2 && c >= T2) ? kINT8 : (has3 && c >= T3) ? kINT4 : kDROP;
    }
    tier[t] = tr;
  }
}

}  // namespace

hipError_t launch_assign(const Geometry& g, const double* score, uint8_t* tier,
                         hipStream_t stream) {
  assign_tiers<<<1, kSelThreads, 0, stream>>>(score, tier, g.n, g.n_sink, g.n16, g.n8, g.n4);
  return hipGetLastError();
}

}  // namespace skv
