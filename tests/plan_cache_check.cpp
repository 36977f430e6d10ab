// Host-only check of the bounded plan cache (paper_2502_06155_amd/csrc/plan_cache.h):
// built with g++ and run by tests/test_plan_cache.py. Values are fake plans whose
// "device work" is a flag the test clears, so eviction and retirement can be driven
// without a GPU.
#include <cstdio>
#include <cstdlib>
#include <string>

#include "plan_cache.h"

namespace {

struct FakePlan {
  int id = 0;
  bool* busy = nullptr;  // enqueued work still running
};

struct FakeOps {
  int released = 0;
  int release_while_busy = 0;
  bool idle(FakePlan& p) { return !p.busy || !*p.busy; }
  void release(FakePlan& p) {
    if (p.busy && *p.busy) ++release_while_busy;
    ++released;
  }
};

int failures = 0;
#define CHECK(c)                                                       \
  do {                                                                 \
    if (!(c)) {                                                        \
      std::printf("FAIL line %d: %s\n", __LINE__, #c);                 \
      ++failures;                                                      \
    }                                                                  \
  } while (0)

void many_distinct_masks() {
  const size_t cap = 256;
  ta::PlanCache<FakePlan, FakeOps> cache(cap);
  for (int i = 0; i < 10000; ++i) {
    const std::string key = "mask-" + std::to_string(i);
    CHECK(cache.acquire(key) == nullptr);
    auto h = cache.insert(key, FakePlan{i, nullptr});
    CHECK(h->value.id == i);
    cache.release(h);
    CHECK(cache.size() <= cap);
  }
  CHECK(cache.size() == cap);
  CHECK(cache.retired() == 0);  // nothing was running: every evicted plan was freed
  CHECK(cache.ops().released == 10000 - (int)cap);
  // the most recent ones are the ones kept
  for (int i = 10000 - (int)cap; i < 10000; ++i) {
    auto h = cache.acquire("mask-" + std::to_string(i));
    CHECK(h && h->value.id == i);
    cache.release(h);
  }
  std::printf("many: size %zu retired %zu released %d\n", cache.size(), cache.retired(),
              cache.ops().released);
}

void busy_held_and_pinned_plans_survive() {
  ta::PlanCache<FakePlan, FakeOps> cache(4);
  bool busy0 = true;
  auto h0 = cache.insert("busy", FakePlan{0, &busy0});
  cache.release(h0);  // its kernels are still running (busy0)
  auto h1 = cache.insert("held", FakePlan{1, nullptr});  // a call still enqueuing: held
  auto h2 = cache.insert("pinned", FakePlan{2, nullptr});
  cache.pin(h2);
  cache.release(h2);
  for (int i = 3; i < 40; ++i) cache.release(cache.insert("x" + std::to_string(i), FakePlan{i, nullptr}));
  CHECK(cache.size() <= 4 + 2);  // held and pinned entries may exceed the capacity
  CHECK(cache.acquire("busy") == nullptr);  // evicted from the index ...
  CHECK(cache.retired() == 1);              // ... but kept while its work runs
  CHECK(cache.ops().release_while_busy == 0);
  auto again = cache.acquire("held");
  CHECK(again == h1);  // never evicted while held, same slot
  cache.release(again);
  cache.release(h1);
  auto p = cache.acquire("pinned");
  CHECK(p == h2);
  cache.release(p);
  busy0 = false;  // the kernels finished
  cache.collect();
  CHECK(cache.retired() == 0);
  CHECK(cache.ops().release_while_busy == 0);
  // the held plan is evictable again once released
  for (int i = 40; i < 60; ++i) cache.release(cache.insert("y" + std::to_string(i), FakePlan{i, nullptr}));
  CHECK(cache.acquire("held") == nullptr);
  auto pp = cache.acquire("pinned");
  CHECK(pp == h2);
  cache.release(pp);
  std::printf("busy/held/pinned: size %zu retired %zu released %d\n", cache.size(), cache.retired(),
              cache.ops().released);
}

void hit_refreshes_recency() {
  ta::PlanCache<FakePlan, FakeOps> cache(3);
  for (int i = 0; i < 3; ++i) cache.release(cache.insert("k" + std::to_string(i), FakePlan{i, nullptr}));
  cache.release(cache.acquire("k0"));  // k0 becomes the most recent; k1 is now the oldest
  cache.release(cache.insert("k3", FakePlan{3, nullptr}));
  CHECK(cache.acquire("k1") == nullptr);
  auto h = cache.acquire("k0");
  CHECK(h && h->value.id == 0);
  cache.release(h);
}

}  // namespace

int main() {
  many_distinct_masks();
  busy_held_and_pinned_plans_survive();
  hit_refreshes_recency();
  if (failures) {
    std::printf("%d failures\n", failures);
    return 1;
  }
  std::printf("plan cache ok\n");
  return 0;
}
