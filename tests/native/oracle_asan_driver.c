/*
 * Test driver: runs every entry point of the CPU oracle on small requests with
 * every buffer allocated at its exact size, so that a build with
 * -fsanitize=address,undefined reports any out-of-bounds access, use of
 * uninitialised heap memory through UB, integer overflow or misaligned access.
 * Exits 0 and prints "ok" when every call returned its expected status.
 * Test infrastructure: it links the oracle and nothing else.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t num_layers, num_kv_heads, head_dim, num_tokens;
  float budget, first_ratio;
  int32_t num_sink;
  float decay;
  int32_t num_tiers, score_mode, num_q_heads, obs_window, quant_int8, quant_int4;
} cfg_t;
typedef struct {
  int32_t n_sink, n_fp16, n_int8, n_int4, n_drop;
  int64_t budget_units, used_units;
} plan_t;

int ora_plan(const cfg_t* c, plan_t* p);
int ora_payload_size(const cfg_t* c, uint64_t* bytes);
int ora_score(const cfg_t* c, const uint16_t* k, const uint16_t* v, const uint16_t* q, double* key);
int ora_assign(const cfg_t* c, const double* key, uint8_t* tier);
int ora_pack(const cfg_t* c, const uint16_t* k, const uint16_t* v, const uint8_t* tier, uint8_t* payload,
             uint64_t capacity);
int ora_unpack(const cfg_t* c, const uint8_t* payload, uint64_t bytes, uint16_t* kc, uint16_t* vc,
               const int32_t* block_table, int32_t num_blocks, int32_t block_size);
int ora_upgrade_size(const cfg_t* c, int32_t m, int32_t mode, uint64_t* bytes);
int ora_pack_upgrade(const cfg_t* c, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
                     const int32_t* tokens, int32_t m, int32_t mode, uint8_t* out, uint64_t capacity);
int ora_unpack_upgrade(const cfg_t* c, const uint8_t* up, uint64_t bytes, uint16_t* kc, uint16_t* vc,
                       const int32_t* block_table, int32_t num_blocks, int32_t block_size);
int32_t ora_group_count(const cfg_t* c, int32_t gran);
int ora_grouped_size(const cfg_t* c, int32_t gran, const float* budgets, uint64_t* bytes);
int ora_score_groups(const cfg_t* c, int32_t gran, const uint16_t* k, const uint16_t* v, const uint16_t* q,
                     double* key);
int ora_assign_groups(const cfg_t* c, int32_t gran, const float* budgets, const double* key, uint8_t* tier);
int ora_pack_groups(const cfg_t* c, int32_t gran, const float* budgets, const uint16_t* k, const uint16_t* v,
                    const uint8_t* tier, uint8_t* payload, uint64_t capacity);
int ora_unpack_groups(const cfg_t* c, int32_t gran, const float* budgets, const uint8_t* payload, uint64_t bytes,
                      uint16_t* kc, uint16_t* vc, const int32_t* block_table, int32_t num_blocks,
                      int32_t block_size);

static int failures = 0;
#define EXPECT(cond)                                                      \
  do {                                                                    \
    if (!(cond)) {                                                        \
      fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                         \
    }                                                                     \
  } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) { /* splitmix64 */
  uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return (uint32_t)((z ^ (z >> 31)) >> 32);
}

/* binary16 values of moderate size, with a few zeros, subnormals and specials */
static uint16_t some_half(void) {
  uint32_t r = next_u32();
  if ((r & 1023) == 0) return 0x7C00;           /* +inf */
  if ((r & 1023) == 1) return 0x7E00;           /* NaN */
  if ((r & 255) == 2) return (uint16_t)(r >> 16) & 0x83FF; /* subnormal or zero */
  uint16_t sign = (uint16_t)((r >> 8) & 0x8000);
  uint16_t exp = (uint16_t)(10 + (r >> 20) % 10); /* 2^-5 .. 2^4 */
  return (uint16_t)(sign | (exp << 10) | ((r >> 4) & 0x3FF));
}

static uint16_t* halves(size_t count) {
  uint16_t* p = (uint16_t*)malloc(count * sizeof(uint16_t) + 1);
  for (size_t i = 0; i < count; ++i) p[i] = some_half();
  return p;
}

static void one_request(int L, int H, int d, int n, float b, int tiers, int mode, int q8, int q4) {
  cfg_t c = {L, H, d, n, b, 0.02f, -1, 0.005f, tiers, mode, mode == 1 ? 2 * H : 0, mode == 1 ? 3 : 0, q8, q4};
  plan_t p;
  if (ora_plan(&c, &p) != 0) return; /* infeasible budget: nothing more to run */
  size_t kv = (size_t)L * H * n * d;
  uint16_t* k = halves(kv);
  uint16_t* v = halves(kv);
  uint16_t* q = mode == 1 ? halves((size_t)L * c.num_q_heads * c.obs_window * d) : NULL;
  double* key = (double*)malloc((size_t)n * sizeof(double));
  uint8_t* tier = (uint8_t*)malloc((size_t)n);
  EXPECT(ora_score(&c, k, v, q, key) == 0);
  EXPECT(ora_assign(&c, key, tier) == 0);
  uint64_t bytes = 0;
  EXPECT(ora_payload_size(&c, &bytes) == 0);
  uint8_t* pay = (uint8_t*)malloc(bytes);
  EXPECT(ora_pack(&c, k, v, tier, pay, bytes) == 0);
  const int bs = 16, nb = (n + bs - 1) / bs + 1;
  int32_t* bt = (int32_t*)malloc((size_t)nb * sizeof(int32_t));
  for (int i = 0; i < nb; ++i) bt[i] = nb - 1 - i;
  size_t cache = (size_t)L * nb * bs * H * d;
  uint16_t* kc = (uint16_t*)malloc(cache * sizeof(uint16_t));
  uint16_t* vc = (uint16_t*)malloc(cache * sizeof(uint16_t));
  memset(kc, 0, cache * 2);
  memset(vc, 0, cache * 2);
  EXPECT(ora_unpack(&c, pay, bytes, kc, vc, bt, nb, bs) == 0);
  /* a short buffer is refused; random single-bit corruptions anywhere either
     decode or are refused (status 0 or format error), never read out of bounds */
  EXPECT(ora_unpack(&c, pay, bytes - 1, kc, vc, bt, nb, bs) != 0);
  for (int trial = 0; trial < 24; ++trial) {
    uint64_t off = (uint64_t)next_u32() % bytes;
    uint8_t bit = (uint8_t)(1u << (next_u32() % 8));
    pay[off] ^= bit;
    int st = ora_unpack(&c, pay, bytes, kc, vc, bt, nb, bs);
    EXPECT(st == 0 || st == 4);
    pay[off] ^= bit;
  }

  if (q8 == 0 && q4 == 0) {
    /* cold-tier upgrade of every non-FP16 token, both modes */
    int32_t m = 0;
    int32_t* tokens = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    for (int t = 0; t < n; ++t)
      if (tier[t] != 0) tokens[m++] = t;
    for (int mode_u = 0; mode_u < 2 && m > 0; ++mode_u) {
      uint64_t ub = 0;
      EXPECT(ora_upgrade_size(&c, m, mode_u, &ub) == 0);
      uint8_t* up = (uint8_t*)malloc(ub);
      EXPECT(ora_pack_upgrade(&c, k, v, tier, tokens, m, mode_u, up, ub) == 0);
      EXPECT(ora_unpack_upgrade(&c, up, ub, kc, vc, bt, nb, bs) == 0);
      free(up);
    }
    free(tokens);
    /* grouped maps at every granularity */
    for (int gran = 0; gran < 3; ++gran) {
      int32_t G = ora_group_count(&c, gran);
      float* budgets = (float*)malloc((size_t)G * sizeof(float));
      for (int g = 0; g < G; ++g) budgets[g] = b;
      uint64_t gb = 0;
      if (ora_grouped_size(&c, gran, budgets, &gb) != 0) { free(budgets); continue; }
      double* gkey = (double*)malloc((size_t)G * n * sizeof(double));
      uint8_t* gtier = (uint8_t*)malloc((size_t)G * n);
      EXPECT(ora_score_groups(&c, gran, k, v, q, gkey) == 0);
      EXPECT(ora_assign_groups(&c, gran, budgets, gkey, gtier) == 0);
      uint8_t* gp = (uint8_t*)malloc(gb);
      EXPECT(ora_pack_groups(&c, gran, budgets, k, v, gtier, gp, gb) == 0);
      EXPECT(ora_unpack_groups(&c, gran, budgets, gp, gb, kc, vc, bt, nb, bs) == 0);
      free(gp);
      free(gtier);
      free(gkey);
      free(budgets);
    }
  }
  free(kc); free(vc); free(bt); free(pay); free(tier); free(key); free(q); free(k); free(v);
}

int main(void) {
  static const int dims[4] = {32, 64, 128, 256};
  static const int tokens[5] = {1, 5, 257, 300, 700};
  static const float budgets[4] = {0.1f, 0.3f, 0.5f, 0.9f};
  static const int quants[6][2] = {{0, 0}, {8, 8}, {2, 14}, {5, 0}, {16, 20}, {28, 26}};
  for (int di = 0; di < 4; ++di)
    for (int ni = 0; ni < 5; ++ni)
      for (int bi = 0; bi < 4; ++bi) {
        int tiers = 2 + ((di + ni + bi) & 1);
        int mode = (di + bi) % 3;
        const int* qq = quants[(di * 5 + ni + bi) % 6];
        one_request(2, 2, dims[di], tokens[ni], budgets[bi], tiers, mode, qq[0], qq[1]);
      }
  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("ok\n");
  return 0;
}
