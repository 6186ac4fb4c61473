// Host-side stress driver for the waiting queue and the continuous-batching
// engine, built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitize_cpu.py.  It drives the engine the way the runtime
// does (plan, then commit with stand-in tokens) over random workloads --
// every policy, the dynamic switching rule, deferred first tokens, pool
// pressure with preemption, future arrivals -- and checks the invariants
// that must hold whatever the schedule: the pool is never exceeded, a plan
// never decodes a slot twice, every request finishes with its token count,
// and rank() lists pops in the order pop_batch returns them.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <unordered_map>
#include <vector>

#include "../paper_2603_11273_amd/csrc/queue.h"
#include "../paper_2603_11273_amd/csrc/serve.h"

using namespace asr;

#define REQUIRE(c)                                                             \
  do {                                                                         \
    if (!(c)) {                                                                \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
      std::exit(1);                                                            \
    }                                                                          \
  } while (0)

static QEntry entry(int64_t id, int64_t arrival, int64_t n_samples, int32_t max_tokens) {
  return QEntry{id, arrival, n_samples, n_samples * 1000000 / 16000, 16000, max_tokens, 0};
}

static void queue_round(std::mt19937_64& rng, int policy, int kd) {
  WaitQueue q;
  q.set_policy(policy, kd ? 27 : 0, kd);
  std::uniform_int_distribution<int64_t> ns(1, 480000), arr(0, 5000000);
  const int n = 300;
  for (int i = 0; i < n; ++i) q.push(entry(i, arr(rng), ns(rng), 448));
  int64_t now = 0;
  while (q.size() > 0) {
    now += 250000;
    std::vector<int64_t> r = q.rank(now);
    const int k = (int)(rng() % 7);
    std::vector<QEntry> got = q.pop_batch(now, k);
    REQUIRE((int)got.size() == std::min<int>(k, (int)r.size()));
    for (size_t i = 0; i < got.size(); ++i) REQUIRE(got[i].id == r[i]);
    for (const QEntry& e : got) REQUIRE(e.arrival_us <= now && !q.contains(e.id));
  }
  REQUIRE(q.min_arrival() == INT64_MAX && !q.any_eligible(now));
}

static void serve_round(std::mt19937_64& rng, int policy, bool dynamic, bool defer, bool pool) {
  ServeConfig c;
  c.n_slots = 1 + (int)(rng() % 24);
  c.max_admit = 1 + (int)(rng() % 8);
  c.cross_tokens = pool ? 50 : 1500;
  c.kv_capacity = pool ? 50 + 448 + (int64_t)(rng() % 2000) : 0;
  c.defer_first = defer;
  c.dynamic = dynamic;
  c.depth_low = (int)(rng() % 6);
  c.starve_num = 3;
  c.starve_den = 1;
  ServeEngine eng;
  eng.configure(c);
  WaitQueue q;
  q.set_policy(policy, 0, 0);
  std::uniform_int_distribution<int64_t> ns(1, 480000), arr(0, 3000000);
  const int n = 200;
  std::unordered_map<int64_t, int32_t> want;
  for (int i = 0; i < n; ++i) {
    QEntry e = entry(i, arr(rng), ns(rng), 1 + (int)(rng() % 448));
    want[i] = eng.tokens_for(e);
    REQUIRE(!pool || c.cross_tokens + want[i] <= c.kv_capacity);
    q.push(e);
  }
  int64_t now = 0;
  int finished = 0, steps = 0;
  while (finished < n) {
    REQUIRE(++steps < 200000);
    ServePlan p = eng.plan(now, q);
    std::set<int32_t> slots(p.dec_slot.begin(), p.dec_slot.end());
    REQUIRE(slots.size() == p.dec_slot.size());
    REQUIRE((int)p.admitted.size() <= c.max_admit);
    std::vector<int32_t> tok(p.dec_id.size());
    for (size_t i = 0; i < tok.size(); ++i) tok[i] = (int32_t)(rng() % 51866);
    std::vector<int32_t> gen;
    std::vector<int64_t> fin = eng.commit(p, tok.data(), &gen);
    REQUIRE(!pool || eng.kv_used() <= c.kv_capacity);
    for (int64_t id : fin) {
      std::vector<int32_t> t;
      REQUIRE(eng.take_result(id, &t));
      REQUIRE((int32_t)t.size() == want[id]);
      ++finished;
    }
    now += 20000;
  }
  REQUIRE(!eng.busy() && q.size() == 0);
}

int main() {
  std::mt19937_64 rng(20260311);
  for (int rep = 0; rep < 4; ++rep)
    for (int policy = 0; policy < 3; ++policy) {
      queue_round(rng, policy, 0);
      queue_round(rng, policy, 10);
      for (int v = 0; v < 8; ++v) serve_round(rng, policy, v & 1, v & 2, v & 4);
    }
  std::printf("sanitized queue/serve stress: ok\n");
  return 0;
}
