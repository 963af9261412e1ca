// Tier assignment: sink pinning + importance-sorted cuts (Sec. 2.3 Prop. 1;
// Sec. 4.4; Algorithm 1, scoring and tier assignment).
//
// Non-sink token t carries the 64-bit ranking key
//   c_t = ((bits(score_t) >> 20) << 21) | t     (score <= 0 or NaN ranks as +0),
// all distinct.  With the tier counts fixed by the plan, token t gets FP16 iff
// c_t is among the n16 largest keys, INT8 iff among the next n8, INT4 iff
// among the next n4, DROP otherwise.  The kernel finds the three cut keys
// T1 >= T2 >= T3 (the n16-th, (n16+n8)-th and (n16+n8+n4)-th largest) by one
// radix select per cut over six digits (11, 11 and 10 bits of the key's high
// word, then the same of its low word), all three sharing each pass over the
// keys, then classifies every token against them.
//   * One workgroup of 1024 threads, or, for rows past the resident form
//     when the caller gives scratch, the split form below (one launch per
//     pass over the whole GPU; the same cut keys).
//   * Resident form (at most 32 non-sink tokens per thread): the scores are
//     loaded once and the high words of the keys kept in LDS (128 KiB, next
//     to the 24 KiB of histograms).  The three high-word passes and the
//     classification read LDS only; the low-word passes reload a score only
//     for a key whose high word equals a cut's, which after three digits is a
//     handful of tokens.
//   * Longer rows recompute the keys from the scores on every pass (the
//     scores stay in L2), eight loads in flight per thread.
//   * Cuts with the same decided prefix share one LDS histogram.
//   * Neighbouring tokens mostly share the first digit (the binary64
//     exponent; the decay orders exponents by position), so that pass must
//     not serialize on one bin.  In the resident form a wave's lanes that
//     share the first counting lane's bin add to it with one atomic; later
//     passes, and the other form, count consecutive keys of a thread that fall
//     in the same bin before one atomic.
#include "device_util.h"
#include "skv_internal.h"

namespace skv {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kBins = 1 << 11;  // widest digit
constexpr int kPasses = 6;
constexpr int kBatch = 8;       // scores loaded per thread before they are counted
constexpr int kResident = 32;   // keys per thread held by the resident form

// Lowest key bit of digit `pass`: 53, 42, 32 in the high word, 21, 10, 0 in
// the low word.
__device__ __forceinline__ int digit_low_bit(int pass) {
  const int q = pass < 3 ? pass : pass - 3;
  return (pass < 3 ? 32 : 0) + (q == 2 ? 0 : 21 - 11 * q);
}

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

// Adds one to bin `bin` of h for every lane with `pred`: the lanes whose bin
// equals that of the first such lane by one atomic from that lane, the rest
// one atomic each.  Every active lane of the wave must call it.
__device__ __forceinline__ void wave_count(uint32_t* h, bool pred, uint32_t bin, int lane) {
  const uint64_t m = __ballot(pred);
  if (m == 0) return;  // wave-uniform
  const int leader = __ffsll(static_cast<unsigned long long>(m)) - 1;
  const uint32_t lb = static_cast<uint32_t>(__shfl(static_cast<int>(bin), leader));
  const uint64_t same = __ballot(pred && bin == lb);
  if (pred) {
    if (bin != lb)
      atomicAdd(&h[bin], 1u);
    else if (lane == leader)
      atomicAdd(&h[lb], static_cast<uint32_t>(__popcll(same)));
  }
}

// LDS state of one row's selection.
struct SelectState {
  uint32_t hist[3][kBins];
  uint64_t prefix[3];  // decided key bits of each cut
  uint32_t rank[3];    // remaining rank (1-based) inside the current prefix
  int group[3];        // which histogram a cut reads
};

// After a pass's histograms are complete: wave j walks cut j's histogram
// from the top bin down and fixes the digit (at key bit `shift`) of the bin
// that holds its remaining rank (32 bins per lane).
__device__ __forceinline__ void choose_digits(SelectState& st, int shift, int lane, int wave) {
  if (wave >= 3 || st.rank[wave] == 0) return;
  const int j = wave;
  constexpr int kPer = kBins / 64;  // 32 consecutive bins per lane, read 4 at a time
  const u32x4* h4 = reinterpret_cast<const u32x4*>(st.hist[st.group[j]]);
  const int b0 = kBins - kPer * (lane + 1);  // this lane's lowest bin; lane 0 holds the top
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < kPer / 4; ++i) {  // rotated by lane: lanes 128 B apart would share banks
    const u32x4 c = h4[b0 / 4 + ((i + lane) & (kPer / 4 - 1))];
    sum += c.x + c.y + c.z + c.w;
  }
  uint32_t inc = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = static_cast<uint32_t>(__shfl_up(static_cast<int>(inc), o));
    if (lane >= o) inc += y;
  }
  uint32_t run = inc - sum;  // keys in the bins above this lane's
  const uint32_t want = st.rank[j];
  if (run < want && want <= run + sum) {
    const uint64_t prefix = st.prefix[j];
#pragma unroll
    for (int i = kPer / 4 - 1; i >= 0; --i) {  // descending bins
      const u32x4 c = h4[b0 / 4 + i];
      const uint32_t cs[4] = {c.w, c.z, c.y, c.x};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int b = b0 + 4 * i + (3 - e);
        if (run < want && want <= run + cs[e]) {
          st.prefix[j] = prefix | (static_cast<uint64_t>(b) << shift);
          st.rank[j] = want - run;
        }
        run += cs[e];
      }
    }
  }
}

// The whole assignment of one score row by one 1024-thread workgroup.
// RESIDENT requires n - n_sink <= kResident * kSelThreads.
template <bool RESIDENT>
__device__ __forceinline__ void assign_row(const double* __restrict__ score, uint8_t* __restrict__ tier, int n,
                                           int n_sink, int n16, int n8, int n4) {
  __shared__ __attribute__((aligned(16))) SelectState st;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t cut_rank[3] = {static_cast<uint32_t>(n16), static_cast<uint32_t>(n16 + n8),
                                static_cast<uint32_t>(n16 + n8 + n4)};
  // resident form: key u of this thread belongs to token t0 + u * kSelThreads,
  // valid for u < nk.  The loads are clamped to token n - 1 (n >= 1) so that
  // all of them issue together without a branch each.
  const int t0 = n_sink + tid;
  const int nk = t0 < n ? (n - t0 + kSelThreads - 1) / kSelThreads : 0;
  // high word of key u of this thread at hi[u][tid]
  __shared__ uint32_t hi[RESIDENT ? kResident : 1][kSelThreads];
  if constexpr (RESIDENT) {
    double sc[kResident];
#pragma unroll
    for (int u = 0; u < kResident; ++u) sc[u] = score[min(t0 + u * kSelThreads, n - 1)];
#pragma unroll
    for (int u = 0; u < kResident; ++u)
      hi[u][tid] = static_cast<uint32_t>(rank_key(sc[u], t0 + u * kSelThreads) >> 32);
  }
  if (tid < 3) {
    st.prefix[tid] = 0;
    st.rank[tid] = tid == 0 ? cut_rank[0] : tid == 1 ? cut_rank[1] : cut_rank[2];
  }
  __syncthreads();

  int hi_bit = 64;  // digit `pass` is key bits [low, hi_bit)
  for (int pass = 0; pass < kPasses; ++pass) {
    const int low = digit_low_bit(pass);
    const uint32_t mask = (1u << (hi_bit - low)) - 1u;
    if (tid < 3) {
      int grp = tid;
      for (int j = 0; j < tid; ++j)
        if (st.rank[j] != 0 && st.prefix[j] == st.prefix[tid]) { grp = j; break; }
      st.group[tid] = grp;
    }
    for (int i = tid; i < 3 * kBins; i += kSelThreads) (&st.hist[0][0])[i] = 0;
    __syncthreads();
    const bool act0 = st.rank[0] != 0 && st.group[0] == 0;
    const bool act1 = st.rank[1] != 0 && st.group[1] == 1;
    const bool act2 = st.rank[2] != 0 && st.group[2] == 2;
    const uint64_t pre0 = st.prefix[0], pre1 = st.prefix[1], pre2 = st.prefix[2];
    RunCounter r0, r1, r2;
    if constexpr (RESIDENT) {
      const uint32_t h0 = static_cast<uint32_t>(pre0 >> 32), h1 = static_cast<uint32_t>(pre1 >> 32),
                     h2 = static_cast<uint32_t>(pre2 >> 32);
      if (pass < 3) {
        // high word: the decided bits are those at or above hi_bit
        const uint32_t dm = pass == 0 ? 0u : ~0u << (hi_bit - 32);
        if (pass == 0) {
          // every cut's prefix is still empty, so only the first cut of
          // nonzero rank leads a group and every key counts in its histogram
          const int lead = act0 ? 0 : act1 ? 1 : 2;
          const bool any = act0 || act1 || act2;
          for (int u = 0; u < nk; ++u) wave_count(st.hist[lead], any, (hi[u][tid] >> (low - 32)) & mask, lane);
        } else {
#pragma unroll 8
          for (int u = 0; u < nk; ++u) {
            const uint32_t w = hi[u][tid];
            const uint32_t bin = (w >> (low - 32)) & mask, d = w & dm;
            if (act0 && d == h0) r0.add(st.hist[0], bin);
            if (act1 && d == h1) r1.add(st.hist[1], bin);
            if (act2 && d == h2) r2.add(st.hist[2], bin);
          }
        }
      } else {
        // low word: a key takes part only if its whole high word is decided
        const uint32_t dm = pass == 3 ? 0u : ~0u << hi_bit;
        const uint32_t l0 = static_cast<uint32_t>(pre0), l1 = static_cast<uint32_t>(pre1),
                       l2 = static_cast<uint32_t>(pre2);
#pragma unroll 8
        for (int u = 0; u < nk; ++u) {
          const uint32_t w = hi[u][tid];
          const bool m0 = act0 && w == h0, m1 = act1 && w == h1, m2 = act2 && w == h2;
          if (m0 || m1 || m2) {
            const int t = t0 + u * kSelThreads;
            const uint32_t lo = static_cast<uint32_t>(rank_key(score[t], t));
            const uint32_t bin = (lo >> low) & mask, d = lo & dm;
            if (m0 && d == l0) r0.add(st.hist[0], bin);
            if (m1 && d == l1) r1.add(st.hist[1], bin);
            if (m2 && d == l2) r2.add(st.hist[2], bin);
          }
        }
      }
    } else {
      const uint64_t decided = pass == 0 ? 0ull : (~0ull << hi_bit);
      for (int base = t0; base < n; base += kBatch * kSelThreads) {
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
          const uint32_t bin = static_cast<uint32_t>(c >> low) & mask;
          const uint64_t d = c & decided;
          if (act0 && d == pre0) r0.add(st.hist[0], bin);
          if (act1 && d == pre1) r1.add(st.hist[1], bin);
          if (act2 && d == pre2) r2.add(st.hist[2], bin);
        }
      }
    }
    flush(st.hist[0], r0.bin, r0.count);
    flush(st.hist[1], r1.bin, r1.count);
    flush(st.hist[2], r2.bin, r2.count);
    __syncthreads();
    choose_digits(st, low, lane, wave);
    __syncthreads();
    hi_bit = low;
  }

  // st.prefix[j] is now the cut key itself (keys are distinct); a cut of rank
  // 0 admits no key.
  const uint64_t T1 = st.prefix[0], T2 = st.prefix[1], T3 = st.prefix[2];
  const bool has1 = cut_rank[0] != 0, has2 = cut_rank[1] != 0, has3 = cut_rank[2] != 0;
  if constexpr (RESIDENT) {
    // c >= T iff its high word is above T's, or equal with the low word at
    // least T's; the low word is loaded only in the equal case
    const uint32_t H1 = static_cast<uint32_t>(T1 >> 32), H2 = static_cast<uint32_t>(T2 >> 32),
                   H3 = static_cast<uint32_t>(T3 >> 32);
    const uint32_t L1 = static_cast<uint32_t>(T1), L2 = static_cast<uint32_t>(T2), L3 = static_cast<uint32_t>(T3);
    for (int t = tid; t < n_sink && t < n; t += kSelThreads) tier[t] = kFP16;
    for (int u = 0; u < nk; ++u) {
      const int t = t0 + u * kSelThreads;
      const uint32_t w = hi[u][tid];
      uint32_t lo = 0;
      if ((has1 && w == H1) || (has2 && w == H2) || (has3 && w == H3))
        lo = static_cast<uint32_t>(rank_key(score[t], t));
      const bool ge1 = has1 && (w > H1 || (w == H1 && lo >= L1));
      const bool ge2 = has2 && (w > H2 || (w == H2 && lo >= L2));
      const bool ge3 = has3 && (w > H3 || (w == H3 && lo >= L3));
      tier[t] = ge1 ? kFP16 : ge2 ? kINT8 : ge3 ? kINT4 : kDROP;
    }
  } else {
    for (int t = tid; t < n; t += kSelThreads) {
      uint8_t tr = kFP16;  // sinks
      if (t >= n_sink) {
        const uint64_t c = rank_key(score[t], t);
        tr = (has1 && c >= T1) ? kFP16 : (has2 && c >= T2) ? kINT8 : (has3 && c >= T3) ? kINT4 : kDROP;
      }
      tier[t] = tr;
    }
  }
}

bool fits_resident(int n, int n_sink) { return n - n_sink <= kResident * kSelThreads; }

// Split form, for rows past the resident form when the caller gives scratch:
// the same six passes and digit choices, but each pass is one launch over
// the whole GPU.  sel_count gives every workgroup kBatch * 1024 consecutive
// non-sink tokens of one row, counts their digits into shared-memory
// histograms and adds the nonzero bins into the row's histogram in device
// memory (integer atomics, so the totals do not depend on the order);
// sel_choose (one workgroup per row) picks each cut's digit from the totals
// exactly as the one-workgroup form does and clears the histogram of the
// next pass; sel_classify then assigns every token against the three cut
// keys.  The cut keys, and so the tier maps, equal the one-workgroup form's.
// The rows are those of a grouped map (one length; counts from the group
// table, 8 words per row: sinks, fp16, int8, int4, ...), a single request, or
// the requests of a batched launch.
struct SelScratch {
  uint32_t hist[2][3][kBins];  // per pass parity: the cut groups' digit counts
  uint64_t prefix[3];          // decided key bits of each cut
  uint32_t rank[3];            // remaining rank inside the prefix
};

// Rows of one shared length n: row r's scores and tiers sit at r * n, its
// counts come from the group table or, for a single row, the arguments.
struct SelRows {
  const double* score;
  uint8_t* tier;
  int n;
  const uint32_t* table;  // per-row counts, or null: the counts below
  int n_sink, n16, n8, n4;
  __device__ __forceinline__ const double* row_score(int row) const { return score + static_cast<size_t>(row) * n; }
  __device__ __forceinline__ uint8_t* row_tier(int row) const { return tier + static_cast<size_t>(row) * n; }
  __device__ __forceinline__ int row_n(int) const { return n; }
  __device__ __forceinline__ void counts(int row, int& s, int& c16, int& c8, int& c4) const {
    if (table != nullptr) {
      const uint32_t* e = table + 8 * row;
      s = static_cast<int>(e[0]);
      c16 = static_cast<int>(e[1]);
      c8 = static_cast<int>(e[2]);
      c4 = static_cast<int>(e[3]);
    } else {
      s = n_sink;
      c16 = n16;
      c8 = n8;
      c4 = n4;
    }
  }
};

// The requests of one batched launch, each with its own length, buffers and
// counts.
struct BatchRows {
  ScoreBatchArgs a;
  __device__ __forceinline__ const double* row_score(int row) const { return a.r[row].score; }
  __device__ __forceinline__ uint8_t* row_tier(int row) const { return a.r[row].tier; }
  __device__ __forceinline__ int row_n(int row) const { return a.r[row].n; }
  __device__ __forceinline__ void counts(int row, int& s, int& c16, int& c8, int& c4) const {
    const ScoreDesc& q = a.r[row];
    s = q.n_sink;
    c16 = q.n16;
    c8 = q.n8;
    c4 = q.n4;
  }
};
static_assert(sizeof(BatchRows) + sizeof(void*) + sizeof(int) <= 4000, "kernel arguments");

// Cut j reads the histogram of the first cut (in cut order) with a nonzero
// rank and the same decided prefix.
__device__ __forceinline__ int cut_group(const uint64_t (&prefix)[3], const uint32_t (&rank)[3], int j) {
  for (int i = 0; i < j; ++i)
    if (rank[i] != 0 && prefix[i] == prefix[j]) return i;
  return j;
}

// grid: one workgroup (256 threads) per row; the cuts start undecided at
// their ranks
template <typename Rows>
__global__ __launch_bounds__(256) void sel_init(const Rows a, SelScratch* __restrict__ scratch) {
  SelScratch* sc = scratch + blockIdx.x;
  int s, c16, c8, c4;
  a.counts(blockIdx.x, s, c16, c8, c4);
  if (threadIdx.x < 3) {
    sc->prefix[threadIdx.x] = 0;
    sc->rank[threadIdx.x] = static_cast<uint32_t>(threadIdx.x == 0 ? c16 : threadIdx.x == 1 ? c16 + c8 : c16 + c8 + c4);
  }
  for (int i = threadIdx.x; i < 3 * kBins; i += 256) (&sc->hist[0][0][0])[i] = 0;
}

// grid: (ceil(longest row / (kBatch * 1024)), rows); pass `pass`.
// Workgroups past a row's last non-sink token count nothing.
template <typename Rows>
__global__ __launch_bounds__(kSelThreads) void sel_count(const Rows a, SelScratch* __restrict__ scratch, int pass) {
  __shared__ uint32_t hist[3][kBins];
  const int row = blockIdx.y;
  SelScratch* sc = scratch + row;
  int n_sink, c16, c8, c4;
  a.counts(row, n_sink, c16, c8, c4);
  const int n = a.row_n(row);
  if (n_sink + static_cast<int>(blockIdx.x) * kBatch * kSelThreads >= n) return;  // uniform per workgroup
  const double* __restrict__ score = a.row_score(row);
  const int tid = threadIdx.x, lane = tid & 63;
  uint64_t pre[3];
  uint32_t rk[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    pre[j] = sc->prefix[j];
    rk[j] = sc->rank[j];
  }
  const bool act0 = rk[0] != 0, act1 = rk[1] != 0 && cut_group(pre, rk, 1) == 1,
             act2 = rk[2] != 0 && cut_group(pre, rk, 2) == 2;
  const int low = digit_low_bit(pass), hi_bit = pass == 0 ? 64 : digit_low_bit(pass - 1);
  const uint32_t mask = (1u << (hi_bit - low)) - 1u;
  const uint64_t decided = pass == 0 ? 0ull : (~0ull << hi_bit);
  // this workgroup's tokens: base + u * 1024, u < kBatch
  const int base = n_sink + blockIdx.x * kBatch * kSelThreads + tid;
  double v[kBatch];
#pragma unroll
  for (int u = 0; u < kBatch; ++u) {
    const int t = base + u * kSelThreads;
    v[u] = t < n ? score[t] : 0.0;
  }
  for (int i = tid; i < 3 * kBins; i += kSelThreads) (&hist[0][0])[i] = 0;
  __syncthreads();
  if (pass == 0) {
    // every prefix is empty: the first cut of nonzero rank leads the only
    // group, and neighbouring tokens mostly share the exponent digit
    const int lead = act0 ? 0 : act1 ? 1 : 2;
    const bool any = act0 || act1 || act2;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int t = base + u * kSelThreads;
      const uint32_t bin = static_cast<uint32_t>(rank_key(v[u], t) >> low) & mask;
      wave_count(hist[lead], any && t < n, bin, lane);
    }
  } else {
    RunCounter r0, r1, r2;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int t = base + u * kSelThreads;
      if (t >= n) break;
      const uint64_t c = rank_key(v[u], t);
      const uint32_t bin = static_cast<uint32_t>(c >> low) & mask;
      const uint64_t d = c & decided;
      if (act0 && d == pre[0]) r0.add(hist[0], bin);
      if (act1 && d == pre[1]) r1.add(hist[1], bin);
      if (act2 && d == pre[2]) r2.add(hist[2], bin);
    }
    flush(hist[0], r0.bin, r0.count);
    flush(hist[1], r1.bin, r1.count);
    flush(hist[2], r2.bin, r2.count);
  }
  __syncthreads();
  uint32_t* out = &sc->hist[pass & 1][0][0];
  for (int i = tid; i < 3 * kBins; i += kSelThreads) {
    const uint32_t c = (&hist[0][0])[i];
    if (c) atomicAdd(&out[i], c);
  }
}

// grid: one workgroup per row; fixes each cut's digit of pass `pass`
__global__ __launch_bounds__(kSelThreads) void sel_choose(SelScratch* __restrict__ scratch, int pass) {
  __shared__ __attribute__((aligned(16))) SelectState st;
  SelScratch* sc = scratch + blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t* in = &sc->hist[pass & 1][0][0];
  for (int i = tid; i < 3 * kBins; i += kSelThreads) (&st.hist[0][0])[i] = in[i];
  if (tid < 3) {
    uint64_t pre[3];
    uint32_t rk[3];
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      pre[j] = sc->prefix[j];
      rk[j] = sc->rank[j];
    }
    st.prefix[tid] = pre[tid];
    st.rank[tid] = rk[tid];
    st.group[tid] = cut_group(pre, rk, tid);
  }
  __syncthreads();
  choose_digits(st, digit_low_bit(pass), lane, wave);
  __syncthreads();
  if (tid < 3) {
    sc->prefix[tid] = st.prefix[tid];
    sc->rank[tid] = st.rank[tid];
  }
  // the next pass counts into the other histogram
  uint32_t* next = &sc->hist[(pass + 1) & 1][0][0];
  for (int i = tid; i < 3 * kBins; i += kSelThreads) next[i] = 0;
}

// grid: (ceil(longest row / 1024), rows); sc->prefix[j] is now the cut key
// itself (keys are distinct), and a cut of rank 0 admits no key
template <typename Rows>
__global__ __launch_bounds__(kSelThreads) void sel_classify(const Rows a, const SelScratch* __restrict__ scratch) {
  const int row = blockIdx.y, n = a.row_n(row);
  const int t = blockIdx.x * kSelThreads + threadIdx.x;
  if (t >= n) return;
  const SelScratch* sc = scratch + row;
  int n_sink, c16, c8, c4;
  a.counts(row, n_sink, c16, c8, c4);
  const bool has1 = c16 != 0, has2 = c16 + c8 != 0, has3 = c16 + c8 + c4 != 0;
  uint8_t tr = kFP16;  // sinks
  if (t >= n_sink) {
    const uint64_t c = rank_key(a.row_score(row)[t], t);
    tr = (has1 && c >= sc->prefix[0]) ? kFP16 : (has2 && c >= sc->prefix[1]) ? kINT8
         : (has3 && c >= sc->prefix[2])                                       ? kINT4
                                                                               : kDROP;
  }
  a.row_tier(row)[t] = tr;
}

// max_n: the longest row
template <typename Rows>
hipError_t launch_assign_split(const Rows& a, int rows, int max_n, SelScratch* sc, hipStream_t stream) {
  sel_init<<<rows, 256, 0, stream>>>(a, sc);
  hipError_t e = hipGetLastError();
  const int per = kBatch * kSelThreads;
  const dim3 count_grid((max_n + per - 1) / per, rows);
  for (int pass = 0; pass < kPasses && e == hipSuccess; ++pass) {
    sel_count<<<count_grid, kSelThreads, 0, stream>>>(a, sc, pass);
    e = hipGetLastError();
    if (e != hipSuccess) break;
    sel_choose<<<rows, kSelThreads, 0, stream>>>(sc, pass);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  sel_classify<<<dim3((max_n + kSelThreads - 1) / kSelThreads, rows), kSelThreads, 0, stream>>>(a, sc);
  return hipGetLastError();
}

template <bool RESIDENT>
__global__ __launch_bounds__(kSelThreads) void assign_tiers(const double* __restrict__ score,
                                                            uint8_t* __restrict__ tier, int n,
                                                            int n_sink, int n16, int n8, int n4) {
  assign_row<RESIDENT>(score, tier, n, n_sink, n16, n8, n4);
}

// grid: one workgroup per group; plan counts from the group table
// (u32 [sinks, fp16, int8, int4, ...], 32 bytes per group).  Rows of at most
// kResident * kSelThreads tokens (longer rows take the split form).
__global__ __launch_bounds__(kSelThreads) void assign_tiers_groups(const double* __restrict__ score,
                                                                   uint8_t* __restrict__ tier, int n,
                                                                   const uint32_t* __restrict__ group_table) {
  const uint32_t* e = group_table + 8 * blockIdx.x;
  const size_t row = static_cast<size_t>(blockIdx.x) * n;
  assign_row<true>(score + row, tier + row, n, static_cast<int>(e[0]), static_cast<int>(e[1]), static_cast<int>(e[2]),
                   static_cast<int>(e[3]));
}

// grid: one workgroup per request of the launch
template <bool RESIDENT>
__global__ __launch_bounds__(kSelThreads) void assign_tiers_batch(const ScoreBatchArgs a) {
  const ScoreDesc& q = a.r[blockIdx.x];
  assign_row<RESIDENT>(q.score, q.tier, q.n, q.n_sink, q.n16, q.n8, q.n4);
}

}  // namespace

bool assign_fits_resident(int32_t n, int32_t n_sink) { return fits_resident(n, n_sink); }

hipError_t launch_assign_batch(const ScoreBatchArgs& a, bool resident, void* scratch, hipStream_t stream) {
  if (!resident && scratch != nullptr) {
    int max_n = 0;
    for (int i = 0; i < a.count; ++i) max_n = a.r[i].n > max_n ? a.r[i].n : max_n;
    return launch_assign_split(BatchRows{a}, a.count, max_n, static_cast<SelScratch*>(scratch), stream);
  }
  if (resident)
    assign_tiers_batch<true><<<a.count, kSelThreads, 0, stream>>>(a);
  else
    assign_tiers_batch<false><<<a.count, kSelThreads, 0, stream>>>(a);
  return hipGetLastError();
}

uint64_t assign_scratch_bytes(int32_t n, int32_t rows) {
  return fits_resident(n, 0) ? 0 : (static_cast<uint64_t>(rows) * sizeof(SelScratch) + 255) / 256 * 256;
}

hipError_t launch_assign(const Geometry& g, const double* score, uint8_t* tier, void* scratch,
                         hipStream_t stream) {
  if (fits_resident(g.n, g.n_sink))
    assign_tiers<true><<<1, kSelThreads, 0, stream>>>(score, tier, g.n, g.n_sink, g.n16, g.n8, g.n4);
  else if (scratch != nullptr)
    return launch_assign_split(SelRows{score, tier, g.n, nullptr, g.n_sink, g.n16, g.n8, g.n4}, 1, g.n,
                               static_cast<SelScratch*>(scratch), stream);
  else
    assign_tiers<false><<<1, kSelThreads, 0, stream>>>(score, tier, g.n, g.n_sink, g.n16, g.n8, g.n4);
  return hipGetLastError();
}

hipError_t launch_assign_groups(int32_t G, int32_t n, const uint32_t* group_table, const double* score,
                                uint8_t* tier, void* scratch, hipStream_t stream) {
  if (!fits_resident(n, 0)) {
    if (scratch == nullptr) return hipErrorInvalidValue;
    return launch_assign_split(SelRows{score, tier, n, group_table, 0, 0, 0, 0}, G, n,
                               static_cast<SelScratch*>(scratch), stream);
  }
  assign_tiers_groups<<<G, kSelThreads, 0, stream>>>(score, tier, n, group_table);
  return hipGetLastError();
}

}  // namespace skv
