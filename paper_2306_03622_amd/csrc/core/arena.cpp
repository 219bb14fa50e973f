#include "arena.hpp"

#include <algorithm>

namespace tp {

tp_status Arena::add_model(int32_t id, uint64_t bytes, bool heavy) {
  if (models_.count(id)) return TP_E_STATE;
  Rec r;
  r.bytes = (bytes + align_ - 1) / align_ * align_;
  r.heavy = heavy;
  models_[id] = r;
  ++class_count_[r.bytes];
  return TP_OK;
}

void Arena::remove_model(int32_t id) {
  evict(id);
  auto it = models_.find(id);
  if (it == models_.end()) return;
  if (--class_count_[it->second.bytes] == 0) class_count_.erase(it->second.bytes);
  models_.erase(it);
}

tp_status Arena::set_partitioned(uint64_t part_bytes, bool consolidate) {
  if (!by_addr_.empty()) return TP_E_STATE;
  if (part_bytes % align_) return TP_E_INVAL;
  consolidate_ = consolidate && part_bytes;
  if (part_bytes == 0)
    parts_.reset();
  else
    parts_.reset(new Partitions(capacity_, part_bytes, align_));
  return TP_OK;
}

bool Arena::place(int32_t id, uint64_t need, uint64_t* off) {
  if (!parts_) return first_fit(need, off);
  return parts_->place(id, need, class_count_.at(need) >= 2, off);
}

uint64_t Arena::used() const {
  uint64_t u = 0;
  for (int32_t id : by_addr_) u += models_.at(id).bytes;
  return u;
}

bool Arena::first_fit(uint64_t need, uint64_t* off) const {
  uint64_t cur = 0;
  for (int32_t id : by_addr_) {
    const Rec& r = models_.at(id);
    if (r.offset >= cur + need) { *off = cur; return true; }
    cur = r.offset + r.bytes;
  }
  if (capacity_ >= cur + need) { *off = cur; return true; }
  return false;
}

std::vector<int32_t> Arena::window_victims(uint64_t need) const {
  // candidate ranges start at 0 or where a resident extent ends; the victims of a range are
  // the extents it overlaps (by_addr_ is sorted by offset, so they follow the range's start)
  struct Key {
    uint64_t newest, bytes, start;
    bool operator<(const Key& o) const {
      return newest != o.newest ? newest < o.newest : bytes != o.bytes ? bytes < o.bytes : start < o.start;
    }
  };
  bool found = false;
  Key best{};
  size_t best_from = 0, best_to = 0;
  for (size_t i = 0; i <= by_addr_.size(); ++i) {
    const uint64_t start = i == 0 ? 0 : models_.at(by_addr_[i - 1]).offset + models_.at(by_addr_[i - 1]).bytes;
    if (start + need > capacity_) continue;
    Key k{0, 0, start};
    size_t j = i;
    for (; j < by_addr_.size(); ++j) {
      const Rec& r = models_.at(by_addr_[j]);
      if (r.offset >= start + need) break;
      k.newest = std::max(k.newest, r.last);
      k.bytes += r.bytes;
    }
    if (!found || k < best) {
      found = true;
      best = k;
      best_from = i;
      best_to = j;
    }
  }
  std::vector<int32_t> v(by_addr_.begin() + (long)best_from, by_addr_.begin() + (long)best_to);
  std::sort(v.begin(), v.end(), [&](int32_t a, int32_t b) { return models_.at(a).last < models_.at(b).last; });
  return v;
}

int32_t Arena::victim() const {
  // least recently used resident model; under the heaviness-aware policy only light models
  // are candidates while any is resident (never the requester: it is not resident)
  int32_t best = -1;
  bool best_light = false;
  uint64_t oldest = UINT64_MAX;
  for (int32_t r : by_addr_) {
    const Rec& rec = models_.at(r);
    const bool light = policy_ == TP_EVICT_HEAVINESS && !rec.heavy;
    if ((light && !best_light) || (light == best_light && rec.last < oldest)) {
      best = r;
      best_light = light;
      oldest = rec.last;
    }
  }
  return best;
}

Arena::Decision Arena::request(int32_t id) {
  Rec& me = models_.at(id);
  me.last = ++clock_;
  Decision d;
  if (me.resident) {
    ++hits_;
    d.hit = true;
    d.offset = me.offset;
    return d;
  }
  ++misses_;
  uint64_t off = 0;
  if (policy_ == TP_EVICT_LRU_WINDOW && !parts_ && !place(id, me.bytes, &off)) {
    for (int32_t victim : window_victims(me.bytes)) {
      if (capacity_ - used() >= me.bytes) ++frag_evictions_;
      d.steps.push_back({false, victim, models_.at(victim).offset, 0});
      evict(victim);
      ++evictions_;
      d.victims.push_back(victim);
    }
  }
  while (!place(id, me.bytes, &off)) {
    if (consolidate_) {
      std::vector<Partitions::Move> mv;
      const bool moved = parts_->evacuate([&](int32_t m) { return models_.at(m).bytes; },
                                          [&](int32_t m) { return class_count_.at(models_.at(m).bytes) >= 2; }, &mv);
      if (moved) {
        for (const auto& x : mv) {
          models_.at(x.id).offset = x.to;
          moved_ += models_.at(x.id).bytes;
          d.moves.push_back(x);
          d.steps.push_back({true, x.id, x.from, x.to});
        }
        std::sort(by_addr_.begin(), by_addr_.end(),
                  [&](int32_t a, int32_t b) { return models_.at(a).offset < models_.at(b).offset; });
        ++evacuations_;
        continue;
      }
    }
    const int32_t victim = this->victim();
    if (victim < 0) {               // nothing left to evict: only if !fits_at_all(id)
      d.placed = false;
      return d;
    }
    if (capacity_ - used() >= me.bytes) ++frag_evictions_;
    d.steps.push_back({false, victim, models_.at(victim).offset, 0});
    evict(victim);
    ++evictions_;
    d.victims.push_back(victim);
  }
  me.resident = true;
  me.offset = off;
  by_addr_.insert(std::upper_bound(by_addr_.begin(), by_addr_.end(), off,
                                   [&](uint64_t o, int32_t r) { return o < models_.at(r).offset; }),
                  id);
  swapped_ += me.bytes;
  d.offset = off;
  return d;
}

void Arena::evict(int32_t id) {
  auto it = models_.find(id);
  if (it == models_.end() || !it->second.resident) return;
  it->second.resident = false;
  by_addr_.erase(std::find(by_addr_.begin(), by_addr_.end(), id));
  if (parts_) parts_->release(id);
}

void Arena::stats(tp_arena_stats_t* s) const {
  s->capacity = capacity_;
  s->used = used();
  uint64_t cur = 0, largest = 0;
  for (int32_t id : by_addr_) {
    const Rec& r = models_.at(id);
    largest = std::max(largest, r.offset - cur);
    cur = r.offset + r.bytes;
  }
  s->largest_free = std::max(largest, capacity_ - cur);
  s->resident = (uint32_t)by_addr_.size();
  s->registered = (uint32_t)models_.size();
  s->hits = hits_;
  s->misses = misses_;
  s->evictions = evictions_;
  s->frag_evictions = frag_evictions_;
  s->bytes_swapped = swapped_;
  s->admit_calls = s->admit_ns_total = s->admit_ns_max = 0;   // timed by the runtime
  s->graph_captures = s->graph_repoints = s->graph_rebases = 0;                   // counted by the runtime
  s->cache_touches = 0;                                                           // counted by the runtime
  s->evacuations = evacuations_;
  s->bytes_moved = moved_;
  s->partitions = parts_ ? parts_->count() : 0;
  s->partitions_free = parts_ ? parts_->free_count() : 0;
}

}  // namespace tp
