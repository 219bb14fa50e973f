// Host-only planning calls (torpor_plan.h) over the arena and model bookkeeping.
#include <new>

#include "arena.hpp"
#include "errors.hpp"
#include "model.hpp"
#include "sched.hpp"
#include "torpor_plan.h"

using namespace tp;

struct tph_arena {
  Arena a;
  std::vector<Arena::Decision::Step> last_steps;
  tph_arena(uint64_t c, uint64_t al) : a(c, al) {}
};

extern "C" {

tp_status tph_validate(const tp_model_desc* desc, uint64_t host_bytes) {
  ModelSpec m;
  std::string err;
  tp_status s = validate_model(desc, host_bytes, &m, &err);
  return s == TP_OK ? ok() : fail(s, err);
}

tp_status tph_touch_span(const tp_model_desc* desc, uint64_t host_bytes, int32_t* applies, uint64_t* lo, uint64_t* hi) {
  ModelSpec m;
  std::string err;
  tp_status s = validate_model(desc, host_bytes, &m, &err);
  if (s != TP_OK) return fail(s, err);
  if (!applies || !lo || !hi) return fail(TP_E_INVAL, "tph_touch_span: NULL output");
  *lo = *hi = 0;
  *applies = touch_span(m, lo, hi) ? 1 : 0;
  return ok();
}

tp_status tph_plan(const tp_model_desc* desc, uint64_t host_bytes, uint64_t chunk_min_bytes, int32_t flags,
                   uint64_t* begin, uint64_t* end, uint32_t* first_layer, uint32_t cap, uint32_t* n) {
  ModelSpec m;
  std::string err;
  tp_status s = validate_model(desc, host_bytes, &m, &err);
  if (s != TP_OK) return fail(s, err);
  if (!n) return fail(TP_E_INVAL, "tph_plan: n is NULL");
  const auto plan = plan_chunks(m, chunk_min_bytes, (flags & TP_FLAG_PER_TENSOR) != 0);
  *n = (uint32_t)plan.size();
  for (uint32_t i = 0; i < plan.size() && i < cap; ++i) {
    if (begin) begin[i] = plan[i].begin;
    if (end) end[i] = plan[i].end;
    if (first_layer) first_layer[i] = plan[i].first_layer;
  }
  return ok();
}

tp_status tph_plan_cost_model(const tp_model_desc* desc, uint64_t host_bytes, int32_t plan_batch, float link_gbs,
                              float chunk_us, uint64_t* begin, uint64_t* end, uint32_t* first_layer, uint32_t cap,
                              uint32_t* n, double* est_us) {
  ModelSpec m;
  std::string err;
  tp_status s = validate_model(desc, host_bytes, &m, &err);
  if (s != TP_OK) return fail(s, err);
  if (!n || plan_batch < 0 || link_gbs < 0 || chunk_us < 0) return fail(TP_E_INVAL, "tph_plan_cost_model: bad argument");
  LinkModel lm;
  if (link_gbs > 0) lm.link_bytes_per_us = link_gbs * 1e3;
  if (chunk_us > 0) lm.chunk_us = chunk_us;
  double est = 0;
  const auto plan = plan_chunks_cost(m, plan_batch > 0 ? plan_batch : 1, lm, &est);
  *n = (uint32_t)plan.size();
  for (uint32_t i = 0; i < plan.size() && i < cap; ++i) {
    if (begin) begin[i] = plan[i].begin;
    if (end) end[i] = plan[i].end;
    if (first_layer) first_layer[i] = plan[i].first_layer;
  }
  if (est_us) *est_us = est;
  return ok();
}

tp_status tph_plan_cost(const uint64_t* unit_begin, const double* unit_us, uint32_t n_units, uint64_t total_bytes,
                        double link_bytes_per_us, double chunk_us, double wait_us, uint32_t* first_unit, uint32_t cap,
                        uint32_t* n_chunks, double* est_us) {
  if (!unit_begin || !unit_us || !n_chunks || n_units == 0 || n_units > 4096)
    return fail(TP_E_INVAL, "tph_plan_cost: NULL argument or unit count outside 1..4096");
  if (!(link_bytes_per_us > 0) || !(chunk_us > 0) || !(wait_us >= 0)) return fail(TP_E_INVAL, "tph_plan_cost: bad link model");
  if (unit_begin[0] != 0) return fail(TP_E_INVAL, "tph_plan_cost: unit_begin[0] must be 0");
  for (uint32_t u = 0; u < n_units; ++u) {
    if (u && unit_begin[u] <= unit_begin[u - 1]) return fail(TP_E_INVAL, "tph_plan_cost: unit offsets must increase");
    if (!(unit_us[u] >= 0)) return fail(TP_E_INVAL, "tph_plan_cost: negative unit time");
  }
  if (total_bytes <= unit_begin[n_units - 1]) return fail(TP_E_INVAL, "tph_plan_cost: total_bytes too small");
  LinkModel lm;
  lm.link_bytes_per_us = link_bytes_per_us;
  lm.chunk_us = chunk_us;
  lm.wait_us = wait_us;
  double est = 0;
  const auto first = plan_cost(std::vector<uint64_t>(unit_begin, unit_begin + n_units), total_bytes,
                               std::vector<double>(unit_us, unit_us + n_units), lm, &est);
  *n_chunks = (uint32_t)first.size();
  for (uint32_t i = 0; first_unit && i < first.size() && i < cap; ++i) first_unit[i] = first[i];
  if (est_us) *est_us = est;
  return ok();
}

tp_status tph_layer_costs(const tp_model_desc* desc, uint64_t host_bytes, int32_t batch, double* us, uint32_t cap,
                          uint32_t* n) {
  ModelSpec m;
  std::string err;
  tp_status s = validate_model(desc, host_bytes, &m, &err);
  if (s != TP_OK) return fail(s, err);
  if (!n || batch < 1) return fail(TP_E_INVAL, "tph_layer_costs: bad argument");
  const auto t = layer_cost_us(m, batch);
  *n = (uint32_t)t.size();
  for (uint32_t i = 0; us && i < t.size() && i < cap; ++i) us[i] = t[i];
  return ok();
}

tp_status tph_rrc(uint64_t n, uint64_t m, double p, double* out) {
  if (!out || !(p > 0 && p < 1) || m > n) return fail(TP_E_INVAL, "tph_rrc: need 0 < p < 1 and m <= n");
  *out = rrc(n, m, p);
  return ok();
}

tp_status tph_sched_pick(uint32_t n_funcs, const uint64_t* n, const uint64_t* m, double p, double alpha,
                         uint32_t n_pending, const int32_t* pending_func, int32_t* pick, uint8_t* high_out) {
  if (!pick || (n_funcs && (!n || !m)) || (n_pending && !pending_func) || !(p > 0 && p < 1) ||
      !(alpha >= 0 && alpha <= 1))
    return fail(TP_E_INVAL, "tph_sched_pick: bad argument");
  std::vector<double> r(n_funcs);
  for (uint32_t f = 0; f < n_funcs; ++f) {
    if (m[f] > n[f]) return fail(TP_E_INVAL, "tph_sched_pick: m > n");
    r[f] = rrc(n[f], m[f], p);
  }
  std::vector<int32_t> pend(pending_func, pending_func + n_pending);
  for (int32_t f : pend)
    if (f < 0 || (uint32_t)f >= n_funcs) return fail(TP_E_INVAL, "tph_sched_pick: function index out of range");
  const std::vector<uint8_t> high = high_group(r, alpha);
  if (high_out) std::copy(high.begin(), high.end(), high_out);
  *pick = sched_pick(r, high, pend);
  return ok();
}

tp_status tph_alpha_update(double alpha, double last_ratio, double new_ratio, double scalar, double threshold,
                           double* out) {
  if (!out || !(scalar > 1) || !(alpha > 0 && alpha <= 1)) return fail(TP_E_INVAL, "tph_alpha_update: bad argument");
  *out = alpha_update(alpha, last_ratio, new_ratio, scalar, threshold);
  return ok();
}

tp_status tph_arena_create(uint64_t capacity, uint64_t align, tph_arena** out) {
  if (!out || align == 0 || (align & (align - 1))) return fail(TP_E_INVAL, "tph_arena_create: bad arguments");
  *out = new (std::nothrow) tph_arena(capacity, align);
  return *out ? ok() : fail(TP_E_NOSPC, "out of host memory");
}

tp_status tph_arena_destroy(tph_arena* a) {
  delete a;
  return ok();
}

tp_status tph_arena_register(tph_arena* a, int32_t id, uint64_t bytes) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  if (a->a.add_model(id, bytes) != TP_OK) return fail(TP_E_STATE, "model id already registered");
  return ok();
}

tp_status tph_arena_unregister(tph_arena* a, int32_t id) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  if (!a->a.known(id)) return fail(TP_E_NOENT, "unknown model id");
  a->a.remove_model(id);
  return ok();
}

tp_status tph_arena_request(tph_arena* a, int32_t id, int32_t* hit, uint64_t* offset, int32_t* victims,
                            uint32_t cap, uint32_t* n_victims) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  a->last_steps.clear();
  if (!a->a.known(id)) return fail(TP_E_NOENT, "unknown model id");
  if (!a->a.fits_at_all(id)) return fail(TP_E_NOSPC, "model larger than the arena");
  Arena::Decision d = a->a.request(id);
  a->last_steps = d.steps;
  if (!d.placed) return fail(TP_E_NOSPC, "model cannot be placed in the arena");
  if (hit) *hit = d.hit;
  if (offset) *offset = d.offset;
  if (n_victims) *n_victims = (uint32_t)d.victims.size();
  for (uint32_t i = 0; victims && i < d.victims.size() && i < cap; ++i) victims[i] = d.victims[i];
  return ok();
}

tp_status tph_arena_evict(tph_arena* a, int32_t id) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  if (!a->a.known(id)) return fail(TP_E_NOENT, "unknown model id");
  a->a.evict(id);
  return ok();
}

tp_status tph_arena_set_policy(tph_arena* a, int32_t policy) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  if (policy != TP_EVICT_LRU && policy != TP_EVICT_HEAVINESS && policy != TP_EVICT_LRU_WINDOW)
    return fail(TP_E_INVAL, "unknown eviction policy");
  a->a.set_policy(policy);
  return ok();
}

tp_status tph_arena_set_heavy(tph_arena* a, int32_t id, int32_t heavy) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  if (!a->a.known(id)) return fail(TP_E_NOENT, "unknown model id");
  a->a.set_heavy(id, heavy != 0);
  return ok();
}

tp_status tph_arena_steps(tph_arena* a, int32_t* model_id, int32_t* moved, uint64_t* from, uint64_t* to, uint32_t cap,
                          uint32_t* n) {
  if (!a || !n) return fail(TP_E_INVAL, "NULL argument");
  *n = (uint32_t)a->last_steps.size();
  for (uint32_t i = 0; i < a->last_steps.size() && i < cap; ++i) {
    const auto& st = a->last_steps[i];
    if (model_id) model_id[i] = st.id;
    if (moved) moved[i] = st.move;
    if (from) from[i] = st.from;
    if (to) to[i] = st.move ? st.to : 0;
  }
  return ok();
}

tp_status tph_arena_set_partitioned(tph_arena* a, uint64_t partition_bytes, int32_t consolidate) {
  if (!a) return fail(TP_E_INVAL, "NULL arena");
  const tp_status s = a->a.set_partitioned(partition_bytes, consolidate != 0);
  if (s == TP_E_STATE) return fail(s, "tph_arena_set_partitioned: models are resident");
  if (s != TP_OK) return fail(s, "tph_arena_set_partitioned: partition size not a multiple of the alignment");
  return ok();
}

tp_status tph_arena_stats(tph_arena* a, tp_arena_stats_t* out) {
  if (!a || !out) return fail(TP_E_INVAL, "NULL argument");
  a->a.stats(out);
  return ok();
}

}  // extern "C"
