// Host-only paths of the library under AddressSanitizer and UBSan: config
// validation and layouts, the recomputation planner, the pipeline schedules,
// the schedule runner's argument checks and graph sharding, on many
// (including invalid) inputs.  Built with g++ against the library's host
// sources and the launch stubs in launch_stubs.cpp (no GPU, no HIP kernel is
// reached); any sanitizer report aborts the program.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <random>
#include <vector>

#include "merak_stage.h"

static int g_checks = 0;
#define EXPECT(c)                                                        \
  do {                                                                   \
    ++g_checks;                                                          \
    if (!(c)) {                                                          \
      fprintf(stderr, "check failed at %s:%d: %s\n", __FILE__, __LINE__, #c); \
      exit(1);                                                           \
    }                                                                    \
  } while (0)

static void configs(std::mt19937& rng) {
  std::uniform_int_distribution<int> pick(0, 9);
  const int hs[] = {0, 64, 256, 384, 512, 1000, 1600, 3072, 6144, 12288};
  const int as[] = {0, 1, 2, 3, 4, 8, 16, 25, 48, 64};
  for (int it = 0; it < 20000; ++it) {
    merak_stage_config c{};
    c.n_blocks = pick(rng) * 8 - 8;
    c.hidden = hs[pick(rng)];
    c.n_heads = as[pick(rng)];
    c.ffn = 4 * hs[pick(rng)];
    c.seq_len = 64 * pick(rng);
    c.micro_batch = pick(rng);
    c.tp_degree = 1 << (pick(rng) % 5);
    c.n_sub_microbatches = 1 + pick(rng) % 4;
    c.recompute_mask = ((uint64_t)rng() << 32) | rng();
    c.dtype = pick(rng) % 3;
    c.ln_eps = pick(rng) ? 1e-5f : 0.0f;
    const int v = merak_stage_validate(&c);
    size_t total = 0, ws = 0, rc = 0;
    std::vector<size_t> offs((size_t)(c.n_blocks > 0 ? c.n_blocks : 1) * MERAK_PARAMS_PER_BLOCK);
    const int a = merak_stage_param_layout(&c, &total, offs.data());
    const int b = merak_stage_workspace_bytes(&c, &ws, &rc);
    EXPECT(a == v && b == v);
    if (v == MERAK_OK) {
      EXPECT(total > 0 && ws > 0);
      for (size_t i = 1; i < offs.size(); ++i) EXPECT(offs[i] > offs[i - 1]);
      EXPECT(offs.back() < total);
    }
    EXPECT(merak_status_str(v) != nullptr);
  }
  EXPECT(merak_stage_validate(nullptr) == MERAK_ERR_INVALID_ARG);
}

static void planner() {
  std::vector<double> alpha(4096);
  std::vector<uint64_t> masks(4096);
  for (int s = 1; s <= 64; ++s)
    for (int k = 0; k <= 20; ++k)
      for (int L : {1, 3, 6, 64}) {
        EXPECT(merak_plan_recompute(s, k / 20.0, L, alpha.data(), masks.data()) == MERAK_OK);
        for (int i = 0; i < s; ++i) EXPECT(alpha[i] >= 0.0 && alpha[i] <= 1.0);
      }
  EXPECT(merak_plan_recompute(0, 0.5, 6, alpha.data(), masks.data()) != MERAK_OK);
  EXPECT(merak_plan_recompute(8, 1.5, 6, alpha.data(), masks.data()) != MERAK_OK);
  EXPECT(merak_plan_recompute(8, 0.5, 65, alpha.data(), masks.data()) != MERAK_OK);
  double a1 = 0.0;
  for (int s = 1; s <= 32; ++s) (void)merak_plan_alpha1(s, 10.0, 2.0, 40.0, 0.01, &a1);
  EXPECT(merak_plan_alpha1(8, 10.0, 2.0, 40.0, 0.0, &a1) == MERAK_ERR_INVALID_ARG);
}

static void schedules() {
  for (int kind = 0; kind <= 2; ++kind)
    for (int s = 1; s <= 12; ++s)
      for (int m = 1; m <= 3 * s + 2; ++m) {
        std::vector<double> busy(s);
        double mk = 0.0;
        EXPECT(merak_schedule_simulate(kind, s, m, 1.0, 1.0, 2.0, &mk, busy.data()) == MERAK_OK);
        for (int i = 0; i < s; ++i) {
          int n = 0, inflight = 0;
          EXPECT(merak_schedule_stage(kind, s, m, i, nullptr, 0, &n) == MERAK_ERR_WORKSPACE);
          std::vector<int32_t> ops(n);
          EXPECT(merak_schedule_stage(kind, s, m, i, ops.data(), n, &n) == MERAK_OK);
          EXPECT(merak_schedule_stage(kind, s, m, i, ops.data(), n - 1, &n) == MERAK_ERR_WORKSPACE);
          EXPECT(merak_schedule_inflight(kind, s, m, i, &inflight) == MERAK_OK);
          EXPECT(inflight >= 1 && inflight <= m);
        }
      }
  EXPECT(merak_schedule_stage(3, 4, 8, 0, nullptr, 0, nullptr) == MERAK_ERR_INVALID_ARG);
  EXPECT(merak_schedule_inflight(2, 4, 8, 4, nullptr) == MERAK_ERR_INVALID_ARG);
  // the runner's argument checks (no handle: nothing is enqueued)
  EXPECT(merak_schedule_run(2, 4, 8, 1, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr,
                            nullptr) == MERAK_ERR_INVALID_ARG);
}

static void graphs(std::mt19937& rng) {
  for (int it = 0; it < 3000; ++it) {
    const int n = 1 + (int)(rng() % 60);
    std::vector<int32_t> kind(n), ptr(n + 1, 0), idx, uses(n, 0), sub(n), io_ptr(2 * n + 1), io(4 * n + 8);
    std::vector<int64_t> params(n);
    for (int i = 0; i < n; ++i) {
      kind[i] = (i < 2 || rng() % 10 == 0) ? MERAK_NODE_INPUT : (rng() % 8 == 0 ? MERAK_NODE_COMMON : 0);
      params[i] = kind[i] == MERAK_NODE_INPUT ? 0 : (int64_t)(rng() % 100);
      if (kind[i] != MERAK_NODE_INPUT && i > 0) {
        const int na = 1 + (int)(rng() % 3);
        for (int q = 0; q < na; ++q) {
          const int a = (int)(rng() % i);
          idx.push_back(a);
          ++uses[a];
        }
      }
      ptr[i + 1] = (int32_t)idx.size();
    }
    for (int i = 0; i < n; ++i)
      if (kind[i] != MERAK_NODE_COMMON) uses[i] = 0;
    int32_t outs[1] = {n - 1}, nsub = 0;
    const int k = 1 + (int)(rng() % 8);
    const int r = merak_graph_shard(n, kind.data(), params.data(), ptr.data(), idx.data(), uses.data(), 1, outs, k,
                                    sub.data(), &nsub, io_ptr.data(), io.data(), (int)io.size());
    EXPECT(r == MERAK_OK || r == MERAK_ERR_WORKSPACE || r == MERAK_ERR_INVALID_ARG);
    if (r == MERAK_OK) EXPECT(nsub >= 0 && nsub <= n);
  }
}

int main() {
  std::mt19937 rng(2206);
  configs(rng);
  planner();
  schedules();
  graphs(rng);
  printf("host checks passed: %d\n", g_checks);
  return 0;
}
