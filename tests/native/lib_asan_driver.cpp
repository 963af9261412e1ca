// Test driver: runs the host-only entry points of the codec library (sizes,
// plans, grouped plans, upgrade sizes, status strings) and the host-side
// argument checks of the device entry points over many configurations, so
// that a build of the library's host code with address and undefined-behaviour
// sanitizers reports any memory or UB error in them.  No device is touched:
// every device call here is rejected by its argument checks before anything
// is enqueued.  Exits 0 and prints "ok" when every status is as expected.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "skv.h"

static int failures = 0;
#define EXPECT(cond)                                                                   \
  do {                                                                                 \
    if (!(cond)) {                                                                     \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                                      \
    }                                                                                  \
  } while (0)

static skv_config make(int L, int H, int d, int n, float b, int tiers, int q8, int q4) {
  skv_config c;
  std::memset(&c, 0, sizeof(c));
  c.num_layers = L;
  c.num_kv_heads = H;
  c.head_dim = d;
  c.num_tokens = n;
  c.budget = b;
  c.first_ratio = 0.02f;
  c.num_sink = -1;
  c.decay = 0.005f;
  c.num_tiers = tiers;
  c.score_mode = SKV_SCORE_KVNORM;
  c.quant_int8 = q8;
  c.quant_int4 = q4;
  return c;
}

int main() {
  EXPECT(skv_abi_version() == SKV_ABI_VERSION);
  for (int s = -7; s <= 8; ++s) EXPECT(skv_status_string(s) != nullptr);
  EXPECT(skv_status_string(SKV_ERR_FORMAT) != nullptr);

  const int dims[] = {32, 48, 64, 128, 256, 512};
  const int tokens[] = {0, 1, 5, 255, 256, 257, 4099, 1 << 21, (1 << 21) + 1};
  const float budgets[] = {0.0f, 0.01f, 0.25f, 0.3f, 0.5f, 0.75f, 1.0f, 1.5f};
  const int quants[] = {0, 1, 2, 3, 4, 8, 14, 16, 20, 28, 31, 32, -1};
  int ran = 0;
  for (int d : dims)
    for (int n : tokens)
      for (float b : budgets)
        for (int tiers = 1; tiers <= 4; ++tiers)
          for (int qi = 0; qi < 13; qi += 3) {
            const int q8 = quants[qi], q4 = quants[(qi + 5) % 13];
            skv_config c = make(3, 2, d, n, b, tiers, q8, q4);
            skv_plan p;
            uint64_t bytes = 0, ws = 0;
            const skv_status st = skv_plan_tiers(&c, &p);
            EXPECT(skv_payload_size(&c, &bytes) == st);
            const skv_status wst = skv_workspace_size(&c, &ws);
            if (st == SKV_OK) {
              EXPECT(p.n_sink + p.n_fp16 + p.n_int8 + p.n_int4 + p.n_drop == n);
              EXPECT(p.used_units <= p.budget_units);
              EXPECT(bytes >= 256);
              EXPECT(wst == SKV_OK);
              ++ran;
              if (q8 == 0 && q4 == 0) {
                for (int mode = -1; mode <= 2; ++mode)
                  for (int m : {-1, 0, 1, n, n + 1}) {
                    uint64_t ub = 0;
                    skv_upgrade_size(&c, m, mode, &ub);
                  }
                for (int gran = -1; gran <= 3; ++gran) {
                  skv_group_spec spec{gran, 0, nullptr};
                  int32_t G = 0;
                  if (skv_group_count(&c, &spec, &G) != SKV_OK) continue;
                  std::vector<float> bg(static_cast<size_t>(G));
                  for (int g = 0; g < G; ++g) bg[static_cast<size_t>(g)] = g % 2 ? b : 0.9f;
                  spec.budgets = bg.data();
                  std::vector<skv_plan> plans(static_cast<size_t>(G));
                  uint64_t gb = 0, gws = 0;
                  if (skv_plan_groups(&c, &spec, plans.data()) == SKV_OK) {
                    EXPECT(skv_grouped_payload_size(&c, &spec, &gb) == SKV_OK);
                    EXPECT(skv_group_workspace_size(&c, &spec, &gws) == SKV_OK);
                  }
                }
              }
              // device entry points: null and misaligned pointers are refused on the host
              alignas(16) static uint8_t buf[64];
              EXPECT(skv_pack(&c, nullptr, buf, buf, buf, bytes, nullptr, nullptr) == SKV_ERR_INVALID_ARG);
              EXPECT(skv_pack(&c, buf + 1, buf, buf, buf, bytes, nullptr, nullptr) == SKV_ERR_INVALID_ARG);
              EXPECT(skv_pack(&c, buf, buf, buf, buf, bytes - 1, nullptr, nullptr) != SKV_OK);
              EXPECT(skv_unpack(&c, nullptr, bytes, buf, buf, nullptr, 1, 16, nullptr, nullptr) == SKV_ERR_INVALID_ARG);
              EXPECT(skv_score(&c, nullptr, buf, nullptr, reinterpret_cast<double*>(buf), buf, nullptr) ==
                     SKV_ERR_INVALID_ARG);
            }
          }
  // batches: bad counts and null request arrays
  skv_config c = make(2, 2, 64, 300, 0.5f, 3, 0, 0);
  EXPECT(skv_pack_batch(&c, nullptr, 1, 0, 2, nullptr) == SKV_ERR_INVALID_ARG);
  alignas(16) static uint8_t cache[64];
  EXPECT(skv_unpack_batch(&c, nullptr, 1, cache, cache, 1, 16, 0, 2, nullptr) == SKV_ERR_INVALID_ARG);
  if (failures) {
    std::fprintf(stderr, "%d failures (%d configurations ran)\n", failures, ran);
    return 1;
  }
  std::printf("ok %d\n", ran);
  return 0;
}
