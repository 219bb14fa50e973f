// The HBM weight arena's bookkeeping: one reserved device range, one contiguous extent
// per resident model, placement in the lowest-addressed free gap that fits, and eviction
// (invalidate only) one victim at a time until a gap fits: least recently used, or, under
// the heaviness-aware policy, the least recently used light model while one is resident and
// only then the least recently used heavy one, or, under the contiguous-window policy, all
// victims at once: those of the cheapest contiguous range. Host-only C++; the runtime attaches
// device-side ordering (events) to the decisions made here. With partitioned placement
// (set_partitioned) the offset comes from the two-tier partition scheme instead of first
// fit; a size class is common while at least two registered models have it.
#pragma once
#include <cstdint>
#include <memory>
#include <unordered_map>
#include <vector>

#include "partition.hpp"
#include "torpor.h"

namespace tp {

class Arena {
 public:
  Arena(uint64_t capacity, uint64_t align, int policy = TP_EVICT_LRU)
      : capacity_(capacity), align_(align), policy_(policy) {}

  struct Decision {
    bool hit = false;
    bool placed = true;             // false: the model cannot be placed even in an empty arena
    uint64_t offset = 0;
    std::vector<int32_t> victims;   // evicted by this request, in eviction order
    std::vector<Partitions::Move> moves;   // consolidation moves, in the order made
    // victims and moves interleaved in the order made (a move may fill a victim's range, a
    // victim may be a model moved earlier in the same request): the device replays this
    struct Step {
      bool move;
      int32_t id;
      uint64_t from, to;      // move: old and new offset
    };
    std::vector<Step> steps;
  };

  tp_status add_model(int32_t id, uint64_t bytes, bool heavy = false);
  void set_heavy(int32_t id, bool heavy) { models_.at(id).heavy = heavy; }
  bool heavy(int32_t id) const { return models_.at(id).heavy; }
  void set_policy(int policy) { policy_ = policy; }
  // Switches placement to partitions of part_bytes (a multiple of the alignment; 0 turns
  // partitioning off), with or without consolidation (partition evacuation before each
  // eviction). TP_E_STATE while any model is resident, TP_E_INVAL for a bad size.
  tp_status set_partitioned(uint64_t part_bytes, bool consolidate = false);
  const Partitions* partitions() const { return parts_.get(); }
  void remove_model(int32_t id);               // also drops residency
  bool known(int32_t id) const { return models_.count(id) != 0; }
  bool fits_at_all(int32_t id) const { return models_.at(id).bytes <= capacity_; }

  // One request for model `id`: ticks the clock, counts a hit or miss, and on a miss
  // chooses victims and an offset. Caller checks fits_at_all() first.
  Decision request(int32_t id);

  void evict(int32_t id);                       // explicit invalidation; no counters
  bool resident(int32_t id) const { return models_.at(id).resident; }
  uint64_t offset(int32_t id) const { return models_.at(id).offset; }
  uint64_t bytes(int32_t id) const { return models_.at(id).bytes; }
  uint64_t last_use(int32_t id) const { return models_.at(id).last; }

  void stats(tp_arena_stats_t* s) const;

 private:
  struct Rec {
    uint64_t bytes = 0, offset = 0, last = 0;
    bool resident = false;
    bool heavy = false;
  };
  bool first_fit(uint64_t need, uint64_t* off) const;
  bool place(int32_t id, uint64_t need, uint64_t* off);
  int32_t victim() const;
  // TP_EVICT_LRU_WINDOW: the extents one contiguous range of `need` bytes overlaps, for the
  // range whose most recently used victim is the oldest (then fewest victim bytes, then lowest
  // address); least recently used first
  std::vector<int32_t> window_victims(uint64_t need) const;
  uint64_t used() const;

  uint64_t capacity_, align_;
  int policy_;
  uint64_t clock_ = 0;
  uint64_t hits_ = 0, misses_ = 0, evictions_ = 0, frag_evictions_ = 0, swapped_ = 0;
  uint64_t evacuations_ = 0, moved_ = 0;
  bool consolidate_ = false;
  std::unordered_map<int32_t, Rec> models_;
  std::vector<int32_t> by_addr_;                // resident ids sorted by offset
  std::unique_ptr<Partitions> parts_;           // partitioned placement, else first fit
  std::unordered_map<uint64_t, uint32_t> class_count_;   // registered models per size
};

}  // namespace tp
