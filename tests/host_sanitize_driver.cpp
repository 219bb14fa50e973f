// Drives every host-only call of libtorpor (include/torpor_plan.h) through valid, malformed
// and random inputs, for a run under AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_host_sanitizers.py builds both this program and the library with them). It
// checks statuses and a few invariants; memory errors and undefined behaviour abort the run.
//
//   host_sanitize_driver <descriptor file>
//
// Descriptor file: per model a line "model arch dtype d0..d7 host_bytes n", then n lines
// "t layer role offset bytes s0 s1 s2 s3".
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <random>
#include <string>
#include <vector>

#include "torpor_plan.h"

namespace {

int failures = 0;
long checks = 0;

void expect(bool ok, const char* what, int line) {
  ++checks;
  if (!ok) {
    std::fprintf(stderr, "check failed (line %d): %s; last error: %s\n", line, what, tp_last_error());
    ++failures;
  }
}
#define EXPECT(c) expect((c), #c, __LINE__)

struct Model {
  tp_model_desc d{};
  std::vector<tp_tensor_desc> t;
  uint64_t host_bytes = 0;
  void fix() {
    d.tensors = t.data();
    d.n_tensors = (uint32_t)t.size();
  }
};

std::vector<Model> read_models(const char* path) {
  std::ifstream f(path);
  std::vector<Model> out;
  std::string tag;
  while (f >> tag) {
    if (tag != "model") break;
    Model m;
    uint32_t n = 0;
    f >> m.d.arch >> m.d.dtype;
    for (int& v : m.d.dims) f >> v;
    f >> m.host_bytes >> n;
    for (uint32_t i = 0; i < n; ++i) {
      tp_tensor_desc t{};
      f >> tag >> t.layer >> t.role >> t.offset >> t.bytes >> t.shape[0] >> t.shape[1] >> t.shape[2] >> t.shape[3];
      m.t.push_back(t);
    }
    m.fix();
    out.push_back(std::move(m));
  }
  return out;
}

void plans(const Model& m) {
  EXPECT(tph_validate(&m.d, m.host_bytes) == TP_OK);
  std::vector<uint64_t> b(4096), e(4096);
  std::vector<uint32_t> fl(4096);
  uint32_t n = 0;
  for (uint64_t g : {0ull, 64ull << 10, 2ull << 20, 16ull << 20, 1ull << 40})
    for (int32_t flags : {0, (int32_t)TP_FLAG_PER_TENSOR}) {
      EXPECT(tph_plan(&m.d, m.host_bytes, g, flags, b.data(), e.data(), fl.data(), (uint32_t)b.size(), &n) == TP_OK);
      EXPECT(n >= 1 && n <= b.size() && b[0] == 0);
      for (uint32_t i = 1; i < n; ++i) EXPECT(b[i] == e[i - 1]);
      // a short output array: only `cap` entries are written, the count is still whole
      uint32_t n2 = 0;
      EXPECT(tph_plan(&m.d, m.host_bytes, g, flags, b.data(), e.data(), fl.data(), 1, &n2) == TP_OK && n2 == n);
    }
  for (int32_t batch : {1, 8, 32}) {
    double est = 0;
    EXPECT(tph_plan_cost_model(&m.d, m.host_bytes, batch, 57.f, 15.f, b.data(), e.data(), fl.data(),
                               (uint32_t)b.size(), &n, &est) == TP_OK);
    EXPECT(n >= 1 && est > 0);
    std::vector<double> us(4096);
    EXPECT(tph_layer_costs(&m.d, m.host_bytes, batch, us.data(), (uint32_t)us.size(), &n) == TP_OK && n >= 1);
    EXPECT(tph_layer_costs(&m.d, m.host_bytes, batch, us.data(), 0, &n) == TP_OK);
  }
  EXPECT(tph_plan_cost_model(&m.d, m.host_bytes, 0, 57.f, 15.f, nullptr, nullptr, nullptr, 0, &n, nullptr) != TP_OK ||
         n >= 1);
}

// every malformation of a valid layout is rejected, never read out of bounds
void malformed(const Model& good) {
  std::mt19937 rng(7);
  for (int k = 0; k < 400; ++k) {
    Model m = good;
    const size_t i = rng() % m.t.size();
    switch (k % 9) {
      case 0: m.t[i].shape[rng() % 4] += 1 + rng() % 3; break;
      case 1: m.t.erase(m.t.begin() + i); break;
      case 2: m.t[i].role = m.t[(i + 1) % m.t.size()].role; break;
      case 3: m.t[i].offset += 2; break;
      case 4: m.t[i].offset = m.t[(i + m.t.size() - 1) % m.t.size()].offset; break;
      case 5: m.t[i].offset = m.host_bytes + 256 * (rng() % 4); break;
      case 6: m.t[i].bytes += 2; break;
      case 7: m.d.dims[rng() % 8] += 1 + rng() % 5; break;
      default: m.t[i].layer += 1000; break;
    }
    m.fix();
    const tp_status s = tph_validate(&m.d, m.host_bytes);
    if (s != TP_OK) EXPECT(s == TP_E_INVAL && tp_last_error()[0] != 0);
    // the planners must reject the same layouts (or plan them, when the change was harmless)
    uint32_t n = 0;
    std::vector<uint64_t> b(4096), e(4096);
    std::vector<uint32_t> fl(4096);
    const tp_status p = tph_plan(&m.d, m.host_bytes, 1 << 20, 0, b.data(), e.data(), fl.data(), 4096, &n);
    EXPECT((p == TP_OK) == (s == TP_OK));
  }
  Model m = good;
  m.d.n_tensors = 0;
  EXPECT(tph_validate(&m.d, m.host_bytes) == TP_E_INVAL);
  m.fix();
  m.d.tensors = nullptr;
  EXPECT(tph_validate(&m.d, m.host_bytes) == TP_E_INVAL);
  EXPECT(tph_validate(nullptr, 1) == TP_E_INVAL);
  m = good;
  m.d.arch = 17;
  EXPECT(tph_validate(&m.d, m.host_bytes) == TP_E_INVAL);
  EXPECT(tph_validate(&good.d, good.host_bytes / 2) == TP_E_INVAL);
}

void cost_units() {
  std::mt19937 rng(11);
  for (int k = 0; k < 300; ++k) {
    const uint32_t n = 1 + rng() % 12;
    std::vector<uint64_t> begin(n);
    std::vector<double> us(n);
    uint64_t at = 0;
    for (uint32_t i = 0; i < n; ++i) {
      begin[i] = at;
      at += 256 * (1 + rng() % 4096);
      us[i] = (rng() % 1000) / 10.0;
    }
    std::vector<uint32_t> first(n);
    uint32_t chunks = 0;
    double est = 0;
    EXPECT(tph_plan_cost(begin.data(), us.data(), n, at, 50e3, 15.0, 5.0, first.data(), n, &chunks, &est) == TP_OK);
    EXPECT(chunks >= 1 && chunks <= n && first[0] == 0 && est > 0);
    EXPECT(tph_plan_cost(begin.data(), us.data(), n, at, 50e3, 15.0, 5.0, first.data(), 0, &chunks, &est) == TP_OK);
  }
  uint64_t b[2] = {0, 10};
  double u[2] = {1, 1};
  uint32_t f[2], c;
  double est;
  EXPECT(tph_plan_cost(b, u, 2, 5, 1.0, 1.0, 1.0, f, 2, &c, &est) == TP_E_INVAL);    // unit past the end
  EXPECT(tph_plan_cost(b, u, 0, 5, 1.0, 1.0, 1.0, f, 2, &c, &est) == TP_E_INVAL);
  EXPECT(tph_plan_cost(nullptr, u, 2, 50, 1.0, 1.0, 1.0, f, 2, &c, &est) == TP_E_INVAL);
  EXPECT(tph_plan_cost(b, u, 2, 50, 0.0, 1.0, 1.0, f, 2, &c, &est) == TP_E_INVAL);
}

// random traces through every placement and eviction policy, with registration churn
void arenas() {
  for (int mode = 0; mode < 6; ++mode) {
    std::mt19937 rng(100 + mode);
    const uint64_t cap = (64ull << 20) + 256 * (rng() % 1000);
    tph_arena* a = nullptr;
    EXPECT(tph_arena_create(cap, 256, &a) == TP_OK);
    if (mode >= 2) EXPECT(tph_arena_set_partitioned(a, (8ull << 20) + 256 * (mode - 2), mode >= 4) == TP_OK);
    EXPECT(tph_arena_set_policy(a, mode % 2 ? TP_EVICT_HEAVINESS : TP_EVICT_LRU) == TP_OK);
    std::vector<int32_t> live;
    int32_t next = 1;
    const uint64_t sizes[] = {1 << 20, 3 << 20, 3 << 20, 7 << 20, 12 << 20, 48 << 20, 5 << 20, 5 << 20};
    std::vector<int32_t> victims(256), ids(512), moved(512);
    std::vector<uint64_t> from(512), to(512);
    for (int step = 0; step < 3000; ++step) {
      const int op = rng() % 20;
      if (live.size() < 3 || op == 0) {
        const uint64_t sz = sizes[rng() % 8] + 256 * (rng() % 3);
        EXPECT(tph_arena_register(a, next, sz) == TP_OK);
        EXPECT(tph_arena_register(a, next, sz) == TP_E_STATE);
        live.push_back(next++);
      } else if (op == 1 && live.size() > 4) {
        const size_t i = rng() % live.size();
        EXPECT(tph_arena_unregister(a, live[i]) == TP_OK);
        live.erase(live.begin() + i);
      } else if (op == 2) {
        EXPECT(tph_arena_evict(a, live[rng() % live.size()]) == TP_OK);
      } else if (op == 3) {
        EXPECT(tph_arena_set_heavy(a, live[rng() % live.size()], rng() % 2) == TP_OK);
      } else {
        int32_t hit = 0;
        uint64_t off = 0;
        uint32_t nv = 0, ns = 0;
        const uint32_t vcap = rng() % 3 ? (uint32_t)victims.size() : 1;     // sometimes a short array
        EXPECT(tph_arena_request(a, live[rng() % live.size()], &hit, &off, victims.data(), vcap, &nv) == TP_OK);
        EXPECT(off % 256 == 0 && off < cap);
        EXPECT(tph_arena_steps(a, ids.data(), moved.data(), from.data(), to.data(), (uint32_t)ids.size(), &ns) ==
               TP_OK);
        EXPECT(ns >= (nv < vcap ? nv : 0));
      }
      tp_arena_stats_t st{};
      EXPECT(tph_arena_stats(a, &st) == TP_OK);
      EXPECT(st.used <= st.capacity && st.largest_free <= st.capacity && st.registered == live.size());
    }
    EXPECT(tph_arena_request(a, 999999, nullptr, nullptr, nullptr, 0, nullptr) != TP_OK);
    EXPECT(tph_arena_evict(a, 999999) == TP_E_NOENT);
    EXPECT(tph_arena_register(a, next, cap + 256) == TP_OK);                 // larger than the arena
    int32_t hit;
    uint64_t off;
    uint32_t nv;
    EXPECT(tph_arena_request(a, next, &hit, &off, victims.data(), 4, &nv) == TP_E_NOSPC);
    EXPECT(tph_arena_set_partitioned(a, 1000, 0) != TP_OK);
    EXPECT(tph_arena_set_policy(a, 99) == TP_E_INVAL);
    EXPECT(tph_arena_destroy(a) == TP_OK);
  }
  EXPECT(tph_arena_create(0, 256, nullptr) == TP_E_INVAL);
}

void scheduling() {
  std::mt19937 rng(5);
  double r = 0;
  EXPECT(tph_rrc(10, 9, 0.98, &r) == TP_OK);
  EXPECT(tph_rrc(10, 9, 1.0, &r) == TP_E_INVAL);
  EXPECT(tph_rrc(10, 11, 0.5, &r) == TP_E_INVAL);
  for (int k = 0; k < 2000; ++k) {
    const uint32_t nf = 1 + rng() % 20, np = rng() % 30;
    std::vector<uint64_t> n(nf), m(nf);
    for (uint32_t f = 0; f < nf; ++f) {
      n[f] = rng() % 50;
      m[f] = n[f] ? rng() % (n[f] + 1) : 0;
    }
    std::vector<int32_t> pend(np);
    for (auto& p : pend) p = (int32_t)(rng() % nf);
    int32_t pick = -2;
    std::vector<uint8_t> high(nf);
    const double alpha = (rng() % 9) / 8.0;
    EXPECT(tph_sched_pick(nf, n.data(), m.data(), 0.98, alpha, np, pend.data(), &pick, high.data()) == TP_OK);
    EXPECT(np ? (pick >= 0 && pick < (int32_t)np) : pick == -1);
    double out = 0;
    EXPECT(tph_alpha_update(alpha > 0 ? alpha : 0.5, (rng() % 100) / 100.0, (rng() % 100) / 100.0, 2.0, 0.04, &out) ==
           TP_OK);
    EXPECT(out > 0 && out <= 1);
  }
  int32_t pick;
  EXPECT(tph_sched_pick(2, nullptr, nullptr, 0.98, 0.5, 0, nullptr, &pick, nullptr) == TP_E_INVAL);
  double out;
  EXPECT(tph_alpha_update(0.5, 0.1, 0.2, 1.0, 0.04, &out) == TP_E_INVAL);
  EXPECT(tph_alpha_update(0.0, 0.1, 0.2, 2.0, 0.04, &out) == TP_E_INVAL);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s <descriptor file>\n", argv[0]);
    return 2;
  }
  const std::vector<Model> models = read_models(argv[1]);
  if (models.empty()) {
    std::fprintf(stderr, "no models in %s\n", argv[1]);
    return 2;
  }
  for (const Model& m : models) {
    plans(m);
    malformed(m);
  }
  cost_units();
  arenas();
  scheduling();
  std::printf("%zu models, %ld checks, %d failed\n", models.size(), checks, failures);
  return failures ? 1 : 0;
}
