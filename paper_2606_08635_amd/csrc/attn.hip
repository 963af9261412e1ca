// Attention-mode score (Sec. 3: attention mass aggregated over layers, heads
// and decode observations; Sec. 4.3: I_j = A_j exp(-lambda Delta_j)).
//
// For every (layer l, KV head h) the G = Hq/H query heads of the group give
// M = G*W observation rows q_m (contiguous in q_obs).  With z[m,t] = q_m.k_t/sqrt(d),
//   A_t = (1 / (L*Hq*W)) * sum over (l, h, m) of softmax_t(z[m, :])[t].
// Q.K^T is a dense contraction, so it runs on the matrix cores
// (v_mfma_f32_32x32x16_f16, fp32 accumulation; binary16 products are exact
// in fp32).  A workgroup walks a run of two 1024-key blocks of one (l, h)
// (consecutive workgroups take different pairs); its four waves take one
// 32-row query tile each (with fewer tiles, the key tiles are split into
// interleaved streams).  The keys pass through shared memory in stages of
// 8-16 KB (32 KB at d = 256), filled by gfx950's direct global-to-LDS loads:
// each key byte leaves HBM once per pass with contiguous 16-byte reads and
// never occupies registers on the way, and the next stage is in flight while
// the current one is multiplied.  The loads are non-temporal: with the default
// cache policy the same stage stream runs 11 % slower.  The waves take their MFMA operands from the
// stage through an XOR swizzle that keeps the 16-byte operand reads free of
// bank conflicts; the wave role is scalar and the stage and tile loops are
// unrolled, so control flow is scalar and every operand read is one lane
// address plus an immediate.
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

// Tuning (measured on MI355X, alternating forms on one box; the macros
// override them for sweeps): two key stages of two 32-key tiles per
// workgroup (one tile per stage with three or four stages was 1-3 % slower at
// d = 128 and 3-7 % at d = 256), and runs of two blocks per workgroup (one
// block per workgroup was 1.5-2.5 % slower, four blocks lost 13 % at d = 256
// for want of workgroups; 2048-key blocks instead of runs came within 2 %
// of runs of two, with different partial sums), four waves per workgroup
// (eight waves, two query-tile streams each, with two to four 16 KB stage
// buffers: 9-20 % slower although they keep up to 96 KB of keys in flight
// per CU against 64 KB).
#ifndef SKV_ATTN_BUFFERS
#define SKV_ATTN_BUFFERS 2  // key stages resident per workgroup (d <= 128)
#endif
#ifndef SKV_ATTN_BUFFERS_D256
#define SKV_ATTN_BUFFERS_D256 2
#endif
#ifndef SKV_ATTN_TILES_D128
#define SKV_ATTN_TILES_D128 2  // 32-key tiles per stage at d = 128
#endif
#ifndef SKV_ATTN_TILES_D256
#define SKV_ATTN_TILES_D256 2
#endif
#ifndef SKV_ATTN_RUN_BLOCKS
#define SKV_ATTN_RUN_BLOCKS 2
#endif

#ifndef SKV_ATTN_WAVES
#define SKV_ATTN_WAVES 4
#endif
constexpr int kWaves = SKV_ATTN_WAVES;  // waves per workgroup
constexpr int kBlockKeys = 1024;                 // keys per block of partial results
constexpr int kRunBlocks = SKV_ATTN_RUN_BLOCKS;  // key blocks a workgroup walks
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

// The 16-byte operand slice of global row `row` for MFMA k-step s in
// lane-half hf: elements 16 s + 8 hf .. + 8 (zeros when the row is absent).
template <int D>
__device__ __forceinline__ void load_rows(const uint16_t* base, int row, bool ok, half8 (&out)[D / 16]) {
  const int hf = (threadIdx.x >> 5) & 1;
  const uint16_t* p = base + static_cast<size_t>(ok ? row : 0) * D + 8 * hf;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) out[s] = ok ? __builtin_bit_cast(half8, *reinterpret_cast<const u32x4*>(p + 16 * s)) : half8{};
}

// A stage of keys in shared memory: kKeys rows of D binary16 values, filled
// by direct global-to-LDS loads.  Each 16-byte load of a wave lands at LDS
// address base + 16 * lane, so a stage is written as consecutive 16-byte
// pieces; piece p holds row p / kCpr, chunk (p % kCpr) ^ swz(row) of the keys
// (kCpr = D / 8 chunks of 8 elements per row).  The XOR swizzle spreads the
// 16-byte operand reads of 8 consecutive rows (same chunk) over all 32 banks;
// it depends on the row only modulo 32, so a lane's read offsets are the same
// for every tile and every stage.
template <int D>
struct Stage {
  static constexpr int kTiles = D < 128 ? 4 : D == 128 ? SKV_ATTN_TILES_D128 : SKV_ATTN_TILES_D256;  // 32-key tiles per stage
  static constexpr int kKeys = kTiles * 32;
  static constexpr int kCpr = D / 8;                             // 16-byte chunks per row
  static constexpr int kRowsPer128 = kCpr >= 8 ? 1 : 8 / kCpr;   // rows sharing one 128-byte bank line
  static constexpr int kPieces = kKeys * kCpr / (kWaves * 64);   // 16-byte loads per thread per stage
  static constexpr int kTileBytes = 32 * D * 2;
  static constexpr int kBytes = kKeys * D * 2;
  // one stage being multiplied, the others in flight; at d = 256 a stage is 32 KB
  static constexpr int kBuffers = D >= 256 ? SKV_ATTN_BUFFERS_D256 : SKV_ATTN_BUFFERS;
  // register budget: four waves per SIMD up to d = 128 (no spills), two at d = 256
  static constexpr int kWavesPerSimd = D >= 256 ? 2 : 4;
  static_assert(kWaves == 4 || kWaves == 8, "four or eight waves per workgroup");
  static_assert(kPieces * kWaves * 64 == kKeys * kCpr, "a stage is whole 16-byte pieces per thread");
  static_assert(kBlockKeys % kKeys == 0, "a block is whole stages");
  static_assert(kBuffers >= 2 && kBuffers <= 4 && (kBuffers - 2) * kPieces < 64, "outstanding loads fit vmcnt");
  __device__ static __forceinline__ int swz(int row) { return (row / kRowsPer128) % kCpr; }
};

// Waits until at most N of this wave's vector memory loads are outstanding
// (loads complete in issue order, so the older ones have landed).
template <int N>
__device__ __forceinline__ void wait_loads() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  asm volatile("" ::: "memory");
  // s_waitcnt: vmcnt bits 3:0 and 15:14; expcnt (6:4) and lgkmcnt (11:8) at their maxima
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
  asm volatile("" ::: "memory");
}

// Waits until the loads of a stage have landed when `later` stages were
// issued after it (later <= 2).
template <int D>
__device__ __forceinline__ void wait_stage(int later) {
  constexpr int P = Stage<D>::kPieces;
  if (later == 0) wait_loads<0>();
  else if (later == 1) wait_loads<P>();
  else wait_loads<2 * P>();
}

// Workgroup barrier for shared memory only: waits for this wave's LDS
// accesses (lgkmcnt 0) but, unlike __syncthreads, not for the global loads in
// flight; the empty asm statements keep the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One direct global-to-LDS load, non-temporal (the keys are streamed once
// per pass): the 16 bytes at src (per lane) land at LDS byte address
// lds_base + 16 * lane.  Issued from inline assembly so that the
// compiler does not count it among its own loads: the stage loop waits for it
// explicitly (wait_stage), and the compiler's own waits for its loads stay
// correct because they can only wait longer.
__device__ __forceinline__ void load_to_lds(const void* src, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(src), "s"(lds_base) : "memory", "m0");
}

// Issues the direct loads of keys t0 .. t0 + kKeys - 1 into the stage at sk.
// Rows at or beyond n repeat row n - 1 (a valid address); their logits are
// masked or never stored.
template <int D>
__device__ __forceinline__ void stage_issue(const uint16_t* kbase, int t0, int n, uint8_t* sk, int wave) {
  using S = Stage<D>;
  const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)sk));
#pragma unroll
  for (int u = 0; u < S::kPieces; ++u) {
    const int p = u * kWaves * 64 + static_cast<int>(threadIdx.x);
    const int row = p / S::kCpr, chunk = (p % S::kCpr) ^ S::swz(row);
    const uint16_t* src = kbase + static_cast<size_t>(min(t0 + row, n - 1)) * D + 8 * chunk;
    load_to_lds(src, __builtin_amdgcn_readfirstlane(base + static_cast<uint32_t>((u * kWaves * 64 + wave * 64) * 16)));
  }
}

typedef __attribute__((address_space(3))) const half8* lds_half8_ptr;

// LDS byte addresses of this lane's MFMA operand slices in the first tile of
// the stage area at s_k: row j, elements 16 s + 8 hf .. + 8 (chunk 2 s + hf,
// swizzled).  Other tiles and stages add a constant.
template <int D>
__device__ __forceinline__ void lane_addresses(const uint8_t* s_k, uint32_t (&addr)[D / 16]) {
  const int hf = (threadIdx.x >> 5) & 1, j = threadIdx.x & 31;
  const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const uint8_t*)s_k));
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    addr[s] = base + static_cast<uint32_t>(j * D * 2 + 16 * ((2 * s + hf) ^ Stage<D>::swz(j)));
    asm volatile("" : "+v"(addr[s]));  // one register per slice: tile offsets fold into the reads
  }
}

// The MFMA operand of one tile; `offset` is the tile's byte offset in the
// stage area (a constant once the stage and tile loops are unrolled, so it
// becomes the instruction's immediate offset).
template <int D>
__device__ __forceinline__ void stage_rows(const uint32_t (&addr)[D / 16], uint32_t offset, half8 (&out)[D / 16]) {
#pragma unroll
  for (int s = 0; s < D / 16; ++s) out[s] = *reinterpret_cast<lds_half8_ptr>(static_cast<uintptr_t>(addr[s] + offset));
}

// Work of wave w in round r: query tiles r*kWaves .. + qg-1 (qg = min(kWaves, MT - r*kWaves))
// are spread over the waves; with fewer than 4 tiles the key tiles of the
// block are split into nstreams interleaved streams so every wave works.
struct WaveRole {
  int qg, nstreams, qtile, stream;
  bool active;
};
__device__ __forceinline__ WaveRole wave_role(int MT, int round, int wave) {
  WaveRole r;
  r.qg = min(kWaves, MT - kWaves * round);
  r.nstreams = 1;  // the largest power of two with qg * nstreams <= kWaves
  while (2 * r.nstreams * r.qg <= kWaves) r.nstreams *= 2;
  r.active = wave < r.qg * r.nstreams;
  r.qtile = kWaves * round + wave % r.qg;
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

// Online update of one query's (m, sum) with the 16 logits of a tile held by
// this lane; (m, sum) stands for sum * 2^m in base-2 units (logit * alpha).
// The reference m is raised lazily: the tile is first exponentiated against
// the current m (one FMA and one exponential per logit); only when its sum
// leaves [0, 2^32] (m still -inf, a logit 32 binades above m, or a NaN) is
// the tile redone against max(m, tile maximum) and the running sum rescaled.
// m is always the maximum of some earlier tile, so every term that
// underflows is below 2^-126 of a term already in the sum.  MASK: keys
// t0 + acc_row >= n are excluded.
template <bool MASK>
__device__ __forceinline__ void tile_update(const floatx16& acc, float alpha, int t0, int hf, int n, float& m,
                                            float& sum) {
  float x[16], e[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    x[r] = acc[r];
    if (MASK && t0 + acc_row(r, hf) >= n) x[r] = -INFINITY;
    e[r] = exp2_fast(__builtin_fmaf(x[r], alpha, -m));
  }
  const float s = tree_sum<16>(e);
  if (s <= 0x1p32f) {
    sum += s;
    return;
  }
  float y[16], t[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    y[r] = x[r] * alpha;
    t[r] = y[r];
  }
  const float tmax = tree_max<16>(t);
  if (tmax == -INFINITY) return;  // every key masked (and m = -inf)
  const float mn = fmaxf(m, tmax);
#pragma unroll
  for (int r = 0; r < 16; ++r) e[r] = exp2_fast(y[r] - mn);
  sum = sum * exp2_fast(m - mn) + tree_sum<16>(e);
  m = mn;
}

// A workgroup owns a run of consecutive key blocks of one (l, h) pair and
// walks it stage by stage, so the next stages are in flight across block
// boundaries and the pair's query rows are loaded once.  Workgroup w takes
// pair w % LH (consecutive workgroups read different pairs) and run
// w / LH of the pair's R runs.  Every block still gets its own partial
// results, so the arithmetic does not depend on the run length.
template <int D>
struct BlockRun {
  static constexpr int kFull = kBlockKeys / Stage<D>::kKeys;  // stages of a whole block
  int nkb;       // key blocks per pair
  int last;      // stages of a pair's last block
  int lh;        // the pair
  int kb0, kb1;  // its blocks kb0 .. kb1 - 1
  int nst;       // their stages
  __device__ __forceinline__ BlockRun(int n, int LH, int R) {
    nkb = (n + kBlockKeys - 1) / kBlockKeys;
    last = (n - (nkb - 1) * kBlockKeys + Stage<D>::kKeys - 1) / Stage<D>::kKeys;
    lh = static_cast<int>(blockIdx.x % static_cast<uint32_t>(LH));
    const int r = static_cast<int>(blockIdx.x / static_cast<uint32_t>(LH));
    kb0 = r * nkb / R;
    kb1 = (r + 1) * nkb / R;
    nst = (kb1 - kb0) * kFull - (kb1 == nkb ? kFull - last : 0);
  }
  __device__ __forceinline__ int stages(int kb) const { return kb == nkb - 1 ? last : kFull; }
};

// grid: LH * R workgroups (BlockRun); pstat[(lh * nkb + kb) * Mpad + row] =
// (max of z, sum of exp(z - max)) over the keys of block kb of pair lh.  The
// logits are formed transposed (keys as MFMA rows, queries as columns), so a
// lane holds 16 keys of one query and keeps that query's running (max, sum)
// in two registers: one exponential per logit.  The stage loop is unrolled
// over the stage buffers and the tiles of a stage, so every shared-memory
// read is a lane offset plus an immediate.
template <int D>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(Stage<D>::kWavesPerSimd))) void attn_stats(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ q, int n, int H, int Hq, int W, float scale,
    int runs, float2* __restrict__ pstat) {
  using S = Stage<D>;
  const int G = Hq / H, M = G * W, MT = (M + 31) / 32, Mpad = MT * 32;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);  // uniform per wave
  const int lane = threadIdx.x & 63, hf = lane >> 5, j = lane & 31;
  const float alpha = scale * kLog2e;
  const BlockRun<D> run(n, static_cast<int>(gridDim.x) / runs, runs);
  const int lh = run.lh, l = lh / H, h = lh % H, nst = run.nst;
  const uint16_t* kbase = k + static_cast<size_t>(lh) * n * D;
  const uint16_t* qbase = q + (static_cast<size_t>(l) * Hq + static_cast<size_t>(h) * G) * W * D;
  float2* out = pstat + static_cast<size_t>(lh) * run.nkb * Mpad;
  __shared__ __align__(16) uint8_t s_k[S::kBuffers * S::kBytes];
  __shared__ float2 s_stat[2][kWaves][32];  // per block parity, wave and query
  uint32_t raddr[D / 16];
  lane_addresses<D>(s_k, raddr);
  for (int round = 0; kWaves * round < MT; ++round) {
    const WaveRole role = wave_role(MT, round, wave);
    // the next stage to issue: stage ist of block ikb
    int ikb = run.kb0, ist = 0;
    auto issue = [&](uint8_t* buf) {
      stage_issue<D>(kbase, ikb * kBlockKeys + ist * S::kKeys, n, buf, wave);
      if (++ist == run.stages(ikb)) {
        ist = 0;
        ++ikb;
      }
    };
    // merges the streams of each query of block kb (stream order; m to z units)
    auto write_stats = [&](int kb) {
      for (int idx = threadIdx.x; idx < role.qg * 32; idx += kWaves * 64) {
        const int qt = idx / 32, jj = idx % 32;
        float mm = -INFINITY, ss = 0.0f;
        for (int st = 0; st < role.nstreams; ++st) {
          const float2 v = s_stat[kb & 1][st * role.qg + qt][jj];
          lse_merge2(mm, ss, v.x, v.y, 1.0f);
        }
        // (max, sum) in logit units: max z = m / log2(e)
        out[static_cast<size_t>(kb) * Mpad + (kWaves * round + qt) * 32 + jj] = float2{mm * kLn2, ss};
      }
    };
    // up to kBuffers - 1 later stages are in flight while a stage is
    // multiplied; the query rows are waited for once, with stage 0, so that
    // no load of the compiler's own is pending inside the stage loop
    issue(s_k);
    half8 qr[D / 16];
    const int qrow = role.qtile * 32 + j;
    if (role.active) load_rows<D>(qbase, qrow, qrow < M, qr);
    wait_loads<0>();
    for (int g = 1; g < S::kBuffers - 1 && g < nst; ++g) issue(s_k + g * S::kBytes);
    float m = -INFINITY, sum = 0.0f;  // m in base-2 units (logit * scale * log2 e)
    int ckb = run.kb0, cst = 0;       // the stage being multiplied: stage cst of block ckb
    int pending = -1;                 // a block whose per-wave stats wait in s_stat
    for (int g0 = 0; g0 < nst; g0 += S::kBuffers) {
#pragma unroll
      for (int b = 0; b < S::kBuffers; ++b) {
        const int g = g0 + b;  // stage g of the run lives in buffer b
        if (g >= nst) break;
        wait_stage<D>(min(S::kBuffers - 2, nst - 1 - g));  // later stages may still be loading
        // every thread's pieces of stage g have landed, every wave is done
        // with stage g - 1, whose buffer the next issue overwrites, and has
        // written the stats of a block that ended there
        lds_barrier();
        if (g + S::kBuffers - 1 < nst) issue(s_k + ((b + S::kBuffers - 1) % S::kBuffers) * S::kBytes);
        if (pending >= 0) {
          write_stats(pending);
          pending = -1;
        }
        if (role.active) {
          const int ts = ckb * kBlockKeys + cst * S::kKeys;  // first key of the stage
#pragma unroll
          for (int ti = 0; ti < S::kTiles; ++ti) {
            // this wave's tiles: tile index in the block = stream (mod nstreams, a power of two)
            const int t0 = ts + ti * 32;
            if (((cst * S::kTiles + ti) & (role.nstreams - 1)) != role.stream || t0 >= n) continue;
            half8 kr[D / 16];
            stage_rows<D>(raddr, b * S::kBytes + ti * S::kTileBytes, kr);
            floatx16 acc{};
#pragma unroll
            for (int s = 0; s < D / 16; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kr[s], qr[s], acc, 0, 0, 0);
            if (t0 + 32 <= n) tile_update<false>(acc, alpha, t0, hf, n, m, sum);
            else tile_update<true>(acc, alpha, t0, hf, n, m, sum);
          }
        }
        if (++cst == run.stages(ckb)) {  // the end of block ckb
          if (role.active) {
            // the two lane-halves saw different keys of the same query:
            // the lower half's stats merged with the upper half's
            const LanePair mp = lane_pair32(__builtin_bit_cast(uint32_t, m));
            const LanePair sp = lane_pair32(__builtin_bit_cast(uint32_t, sum));
            m = __builtin_bit_cast(float, mp.lo);
            sum = __builtin_bit_cast(float, sp.lo);
            lse_merge2(m, sum, __builtin_bit_cast(float, mp.hi), __builtin_bit_cast(float, sp.hi), 1.0f);
            if (hf == 0) s_stat[ckb & 1][wave][j] = float2{m, sum};
          }
          m = -INFINITY;
          sum = 0.0f;
          pending = ckb;
          cst = 0;
          ++ckb;
        }
      }
    }
    lds_barrier();
    if (pending >= 0) write_stats(pending);
    __syncthreads();  // the next round's first loads overwrite the first stage buffers
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

// grid: LH * R workgroups, as attn_stats; colsum[lh * n + t] = sum over the
// group's rows of p[row, t].  Logits with queries as MFMA rows: a lane holds
// 16 rows of one key and sums their probabilities, the two lane-halves are
// added by a shuffle, and the query tiles of a stage are added in tile order
// from shared memory one stage later (rounds of query tiles add onto the
// stored sums in round order).
template <int D>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(Stage<D>::kWavesPerSimd))) void attn_colsum(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ q, int n, int H, int Hq, int W, float scale,
    int runs, const float* __restrict__ cstat, float* __restrict__ colsum) {
  using S = Stage<D>;
  const int G = Hq / H, M = G * W, MT = (M + 31) / 32, Mpad = MT * 32;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);  // uniform per wave
  const int lane = threadIdx.x & 63, hf = lane >> 5, j = lane & 31;
  const float alpha = scale * kLog2e;
  const BlockRun<D> run(n, static_cast<int>(gridDim.x) / runs, runs);
  const int lh = run.lh, l = lh / H, h = lh % H, nst = run.nst;
  const uint16_t* kbase = k + static_cast<size_t>(lh) * n * D;
  const uint16_t* qbase = q + (static_cast<size_t>(l) * Hq + static_cast<size_t>(h) * G) * W * D;
  float* out = colsum + static_cast<size_t>(lh) * n;
  __shared__ __align__(16) uint8_t s_k[S::kBuffers * S::kBytes];
  __shared__ float s_part[2][kWaves][S::kKeys];  // per stage (double-buffered), per wave, per key
  uint32_t raddr[D / 16];
  lane_addresses<D>(s_k, raddr);
  for (int round = 0; kWaves * round < MT; ++round) {
    const WaveRole role = wave_role(MT, round, wave);
    int ikb = run.kb0, ist = 0;  // the next stage to issue: stage ist of block ikb
    auto issue = [&](uint8_t* buf) {
      stage_issue<D>(kbase, ikb * kBlockKeys + ist * S::kKeys, n, buf, wave);
      if (++ist == run.stages(ikb)) {
        ist = 0;
        ++ikb;
      }
    };
    issue(s_k);
    half8 qr[D / 16];
    float beta[16];  // c * log2(e) of the lane's 16 rows; +inf for padding rows
    // padding rows of a partial query tile: their zero queries can still make
    // a NaN logit against an infinite key element (0 * inf), so their terms
    // are masked out explicitly rather than relying on exp2(z - inf) = 0
    uint32_t valid_rows = 0xFFFFu;
    const bool padded = role.active && role.qtile * 32 + 32 > M;  // uniform per wave
    if (role.active) {
      const int qrow = role.qtile * 32 + j;
      load_rows<D>(qbase, qrow, qrow < M, qr);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        beta[r] = cstat[static_cast<size_t>(lh) * Mpad + role.qtile * 32 + acc_row(r, hf)] * kLog2e;
        if (role.qtile * 32 + acc_row(r, hf) >= M) valid_rows &= ~(1u << r);
      }
    }
    // the stage whose partial sums wait in s_part: its first key, its index
    // in the run and its stage index in its block
    int fl_t0 = 0, fl_g = 0, fl_cst = 0;
    // adds the query tiles' partial sums of that stage (tile order) onto the
    // stored sums (round order); thread i owns key i of the stage
    auto flush = [&]() {
      const int i = threadIdx.x;
      const int t = fl_t0 + i;
      if (i < S::kKeys && t < n) {
        const int stream = (fl_cst * S::kTiles + i / 32) & (role.nstreams - 1);
        float v = s_part[fl_g & 1][stream * role.qg][i];
        for (int qt = 1; qt < role.qg; ++qt) v += s_part[fl_g & 1][stream * role.qg + qt][i];
        out[t] = round == 0 ? v : out[t] + v;
      }
    };
    // the query rows and row constants are waited for once, with stage 0;
    // up to kBuffers - 1 later stages are in flight while a stage is multiplied
    wait_loads<0>();
    for (int g = 1; g < S::kBuffers - 1 && g < nst; ++g) issue(s_k + g * S::kBytes);
    int ckb = run.kb0, cst = 0;  // the stage being multiplied: stage cst of block ckb
    for (int g0 = 0; g0 < nst; g0 += S::kBuffers) {
#pragma unroll
      for (int b = 0; b < S::kBuffers; ++b) {
        const int g = g0 + b;  // stage g of the run lives in buffer b
        if (g >= nst) break;
        wait_stage<D>(min(S::kBuffers - 2, nst - 1 - g));  // later stages may still be loading
        // stage g has landed everywhere; every wave is done with stage g - 1
        // (its buffer is reloaded next) and has written its partial sums
        lds_barrier();
        if (g + S::kBuffers - 1 < nst) issue(s_k + ((b + S::kBuffers - 1) % S::kBuffers) * S::kBytes);
        if (g > 0) flush();
        const int ts = ckb * kBlockKeys + cst * S::kKeys;  // first key of the stage
        if (role.active) {
          float* part = s_part[g & 1][wave];
#pragma unroll
          for (int ti = 0; ti < S::kTiles; ++ti) {
            const int t0 = ts + ti * 32;
            if (((cst * S::kTiles + ti) & (role.nstreams - 1)) != role.stream || t0 >= n) continue;
            half8 kr[D / 16];
            stage_rows<D>(raddr, b * S::kBytes + ti * S::kTileBytes, kr);
            floatx16 acc{};
#pragma unroll
            for (int s = 0; s < D / 16; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(qr[s], kr[s], acc, 0, 0, 0);
            // sum over the lane's 16 rows of p = 2^(acc * alpha - beta), then over both lane-halves
            float e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) e[r] = exp2_fast(__builtin_fmaf(acc[r], alpha, -beta[r]));
            if (padded) {
#pragma unroll
              for (int r = 0; r < 16; ++r) e[r] = (valid_rows >> r) & 1u ? e[r] : 0.0f;
            }
            float p = tree_sum<16>(e);
            // the other lane-half holds the other 16 rows: lower + upper
            const LanePair pp = lane_pair32(__builtin_bit_cast(uint32_t, p));
            p = __builtin_bit_cast(float, pp.lo) + __builtin_bit_cast(float, pp.hi);
            if (hf == 0) part[ti * 32 + j] = p;
          }
        }
        fl_t0 = ts;
        fl_g = g;
        fl_cst = cst;
        if (++cst == run.stages(ckb)) {
          cst = 0;
          ++ckb;
        }
      }
    }
    lds_barrier();
    flush();
    __syncthreads();  // the next round's first loads overwrite the first stage buffers
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
  // a pair's key blocks in runs of about kRunBlocks, each run one workgroup;
  // workgroup w takes pair w % LH, so the workgroups in flight read many pairs
  const int runs = (s.nkb + kRunBlocks - 1) / kRunBlocks;
  if (static_cast<int64_t>(s.LH) * runs > INT32_MAX) return hipErrorInvalidValue;
  const int grid = s.LH * runs;
  attn_stats<D><<<grid, kWaves * 64, 0, stream>>>(k, q, g.n, g.H, Hq, W, scale, runs, pstat);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_merge<<<(s.LH * s.Mpad + 255) / 256, 256, 0, stream>>>(pstat, s.LH, s.nkb, s.Mpad, s.M, cstat);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_colsum<D><<<grid, kWaves * 64, 0, stream>>>(k, q, g.n, g.H, Hq, W, scale, runs, cstat, colsum);
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
