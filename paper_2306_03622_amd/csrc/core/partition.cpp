#include "partition.hpp"

#include <algorithm>

namespace tp {

Partitions::Partitions(uint64_t capacity, uint64_t part_bytes, uint64_t align) : part_(part_bytes), align_(align) {
  const uint64_t n = capacity / part_;
  for (uint64_t i = 0; i < n; ++i) {
    Part p;
    p.start = i * part_;
    p.size = part_;
    parts_.push_back(p);
  }
  const uint64_t rest = capacity - n * part_;
  if (rest >= align_) {
    Part p;
    p.start = n * part_;
    p.size = rest;
    parts_.push_back(p);
  }
}

uint32_t Partitions::free_count() const {
  uint32_t n = 0;
  for (const Part& p : parts_) n += p.kind == kFree;
  return n;
}

uint64_t Partitions::block_size(uint64_t part_size, uint64_t need) const {
  if (part_size < need) return 0;
  uint64_t b = part_size;
  while (b % (2 * align_) == 0 && b / 2 >= need) b /= 2;
  return b;
}

int Partitions::fresh(uint64_t need) const {
  for (int i = (int)parts_.size() - 1; i >= 0; --i)
    if (parts_[i].kind == kFree && parts_[i].size >= need) return i;
  return -1;
}

bool Partitions::place_run(int32_t id, uint64_t bytes, uint64_t* off) {
  // lowest-starting run of consecutive free partitions that holds `bytes`
  const uint32_t n = (uint32_t)parts_.size();
  for (uint32_t i = 0; i < n; ++i) {
    if (parts_[i].kind != kFree) continue;
    uint64_t total = 0;
    uint32_t j = i;
    while (j < n && parts_[j].kind == kFree && total < bytes) total += parts_[j++].size;
    if (total < bytes) {
      i = j;          // partitions i..j-1 are free but too few; j is occupied or the end
      continue;
    }
    for (uint32_t k = i; k < j; ++k) parts_[k].kind = kRun;
    where_[id] = {kRun, i, j - 1, 0};
    *off = parts_[i].start;
    return true;
  }
  return false;
}

bool Partitions::place_slab(int32_t id, uint64_t bytes, uint64_t* off, int avoid) {
  int best = -1;
  for (int i = 0; i < (int)parts_.size(); ++i) {
    const Part& p = parts_[i];
    if (i == avoid || p.kind != kSlab || p.cls != bytes || p.slots.size() >= p.size / bytes) continue;
    if (best < 0 || p.slots.size() > parts_[best].slots.size()) best = i;
  }
  if (best < 0) {
    best = avoid >= 0 ? -1 : fresh(bytes);
    if (best < 0) return false;
    parts_[best].kind = kSlab;
    parts_[best].cls = bytes;
  }
  Part& p = parts_[best];
  uint64_t k = 0;                                  // lowest free slot
  for (uint64_t s : p.slots) {
    if (s != k) break;
    ++k;
  }
  p.slots.insert(k);
  where_[id] = {kSlab, (uint32_t)best, (uint32_t)best, k};
  *off = p.start + k * bytes;
  return true;
}

bool Partitions::place_buddy(int32_t id, uint64_t bytes, uint64_t* off, int avoid) {
  int best = -1;
  for (int i = 0; i < (int)parts_.size(); ++i) {
    const Part& p = parts_[i];
    if (i == avoid || p.kind != kBuddy) continue;
    const uint64_t t = block_size(p.size, bytes);
    if (!t || p.free_blk.lower_bound({t, 0}) == p.free_blk.end()) continue;
    if (best < 0 || p.used_bytes > parts_[best].used_bytes) best = i;
  }
  if (best < 0) {
    best = avoid >= 0 ? -1 : fresh(bytes);
    if (best < 0) return false;
    Part& p = parts_[best];
    p.kind = kBuddy;
    p.free_blk.insert({p.size, 0});
  }
  Part& p = parts_[best];
  const uint64_t t = block_size(p.size, bytes);
  auto it = p.free_blk.lower_bound({t, 0});        // smallest large-enough block, lowest offset
  uint64_t sz = it->first, o = it->second;
  p.free_blk.erase(it);
  while (sz > t) {                                  // keep the lower half, free the upper
    sz /= 2;
    p.free_blk.insert({sz, o + sz});
  }
  p.used_blk[o] = sz;
  p.used_bytes += sz;
  where_[id] = {kBuddy, (uint32_t)best, (uint32_t)best, o};
  *off = p.start + o;
  return true;
}

bool Partitions::place(int32_t id, uint64_t bytes, bool common, uint64_t* off, int avoid) {
  if (bytes > part_) return avoid >= 0 ? false : place_run(id, bytes, off);
  return common ? place_slab(id, bytes, off, avoid) : place_buddy(id, bytes, off, avoid);
}

bool Partitions::evacuate(const std::function<uint64_t(int32_t)>& bytes, const std::function<bool(int32_t)>& common,
                          std::vector<Move>* moves) {
  std::vector<std::pair<uint64_t, int>> order;       // (bytes in use, index)
  for (int i = 0; i < (int)parts_.size(); ++i) {
    const Part& p = parts_[i];
    if (p.kind == kSlab) order.push_back({p.slots.size() * p.cls, i});
    if (p.kind == kBuddy) order.push_back({p.used_bytes, i});
  }
  std::sort(order.begin(), order.end());
  for (const auto& cand : order) {
    const int i = cand.second;
    std::vector<std::pair<uint64_t, int32_t>> occ;   // (offset, model) in offset order
    uint64_t need = 0;
    bool irregular = true;                           // every occupant's class irregular now
    for (const auto& w : where_) {
      if (w.second.kind == kRun || (int)w.second.first != i) continue;
      const Part& p = parts_[i];
      occ.push_back({p.start + (w.second.kind == kSlab ? w.second.pos * p.cls : w.second.pos), w.first});
      need += bytes(w.first);
      irregular = irregular && !common(w.first);
    }
    std::sort(occ.begin(), occ.end());
    // cheap rejections that never change the outcome: a slot partition whose class is still
    // common needs as many free slots of its class elsewhere as it has occupants (exact); a
    // buddy partition of irregular occupants needs at least their bytes free in other buddy
    // partitions (occupants whose class has become common go to slots instead)
    const Part& pi = parts_[i];
    if (pi.kind == kSlab && common(occ.front().second)) {
      uint64_t free_slots = 0;
      for (int k = 0; k < (int)parts_.size(); ++k)
        if (k != i && parts_[k].kind == kSlab && parts_[k].cls == pi.cls)
          free_slots += parts_[k].size / pi.cls - parts_[k].slots.size();
      if (free_slots < occ.size()) continue;
    } else if (pi.kind == kBuddy && irregular) {
      uint64_t free_bytes = 0;
      for (int k = 0; k < (int)parts_.size(); ++k)
        if (k != i && parts_[k].kind == kBuddy) free_bytes += parts_[k].size - parts_[k].used_bytes;
      if (free_bytes < need) continue;
    }
    const std::vector<Part> saved_parts = parts_;
    const std::unordered_map<int32_t, Where> saved_where = where_;
    std::vector<Move> mv;
    bool all = true;
    for (const auto& o : occ) {
      release(o.second);
      uint64_t to = 0;
      if (!place(o.second, bytes(o.second), common(o.second), &to, i)) {
        all = false;
        break;
      }
      mv.push_back({o.second, o.first, to});
    }
    if (all) {
      moves->insert(moves->end(), mv.begin(), mv.end());
      return true;
    }
    parts_ = saved_parts;
    where_ = saved_where;
  }
  return false;
}

void Partitions::release(int32_t id) {
  auto w = where_.find(id);
  if (w == where_.end()) return;
  const Where at = w->second;
  where_.erase(w);
  if (at.kind == kRun) {
    for (uint32_t k = at.first; k <= at.last; ++k) parts_[k].reset();
    return;
  }
  Part& p = parts_[at.first];
  if (at.kind == kSlab) {
    p.slots.erase(at.pos);
    if (p.slots.empty()) p.reset();
    return;
  }
  uint64_t o = at.pos, sz = p.used_blk.at(o);
  p.used_blk.erase(o);
  p.used_bytes -= sz;
  while (sz < p.size) {                             // merge with free buddies of equal size
    const uint64_t b = (o / sz) % 2 == 0 ? o + sz : o - sz;
    auto f = p.free_blk.find({sz, b});
    if (f == p.free_blk.end()) break;
    p.free_blk.erase(f);
    o = o < b ? o : b;
    sz *= 2;
  }
  p.free_blk.insert({sz, o});
  if (p.used_blk.empty()) p.reset();
}

}  // namespace tp
