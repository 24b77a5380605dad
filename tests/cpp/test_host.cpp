// Host-only checks of the KV page pool and the tail-batching planner, built
// with g++ and AddressSanitizer/UndefinedBehaviorSanitizer by the CPU tests.
#include <cassert>
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <random>
#include <set>
#include <stdexcept>
#include <vector>

#include "kv_pool.hpp"
#include "tail_batch.hpp"

using rollpack::PagePool;

static int failures = 0;
#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      std::fprintf(stderr, "CHECK failed %s:%d: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                 \
    }                                                             \
  } while (0)

static void test_pool_random() {
  std::mt19937 rng(7);
  PagePool pool(257);
  std::vector<std::vector<int32_t>> owned(20);
  for (int it = 0; it < 20000; ++it) {
    const int o = rng() % 20;
    if (rng() % 2) {
      const int64_t want = rng() % 40;
      const int64_t before = pool.free_pages();
      try {
        pool.take(want, o, owned[o]);
        CHECK(pool.free_pages() == before - want);
      } catch (const std::runtime_error&) {
        CHECK(want > before);
        CHECK(pool.free_pages() == before);  // no side effect on failure
      }
    } else {
      pool.give_back(owned[o], o);
      owned[o].clear();
    }
    // conservation and exclusive ownership
    int64_t held = 0;
    std::set<int32_t> seen;
    for (int k = 0; k < 20; ++k) {
      held += owned[k].size();
      for (int32_t p : owned[k]) {
        CHECK(seen.insert(p).second);
        CHECK(pool.owner_of(p) == k);
      }
    }
    CHECK(held + pool.free_pages() == pool.capacity());
    CHECK(pool.peak_used() >= pool.used_pages());
  }
  for (int k = 0; k < 20; ++k) pool.give_back(owned[k], k);
  CHECK(pool.free_pages() == pool.capacity());
}

static void test_pool_misuse() {
  PagePool pool(4);
  std::vector<int32_t> a, b;
  pool.take(2, 1, a);
  bool threw = false;
  try { pool.give_back(a, 2); } catch (const std::logic_error&) { threw = true; }
  CHECK(threw);
  CHECK(pool.free_pages() == 2);
  threw = false;
  try { pool.take(3, 2, b); } catch (const std::runtime_error&) { threw = true; }
  CHECK(threw && b.empty());
  CHECK(PagePool::pages_for(0, 64) == 0 && PagePool::pages_for(1, 64) == 1 && PagePool::pages_for(64, 64) == 1 &&
        PagePool::pages_for(65, 64) == 2);
}

static void test_plan_invariants() {
  std::mt19937 rng(11);
  for (int it = 0; it < 300; ++it) {
    const int P0 = 1 + rng() % 6, R0 = 1 + rng() % 4, n = rng() % 40;
    const double eta = 1.25;
    const int r_spec = static_cast<int>(std::ceil(eta * R0 - 1e-9));
    std::vector<int32_t> lens(static_cast<size_t>(n) * r_spec);
    for (auto& L : lens) L = 1 + rng() % 500;
    auto plan = rollpack::plan_tail_batching(n, r_spec, lens.data(), P0, R0, eta, eta);
    std::vector<int> accepted(n, 0);
    for (const auto& r : plan.rounds) {
      for (int32_t p : r.accepted) accepted[p]++;
      CHECK(r.run_steps.size() == r.launched.size() * r_spec);
      if (r.kind == 1) CHECK(r.accepted == r.launched);
      else CHECK(static_cast<int>(r.accepted.size()) == std::min<int>(P0, r.launched.size()));
    }
    for (int p = 0; p < n; ++p) {
      CHECK(accepted[p] == 1);
      int kept = 0;
      for (int r = 0; r < r_spec; ++r) kept += plan.kept[static_cast<size_t>(p) * r_spec + r];
      CHECK(kept == R0);
    }
  }
}

int main() {
  test_pool_random();
  test_pool_misuse();
  test_plan_invariants();
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("host tests passed\n");
  return 0;
}
