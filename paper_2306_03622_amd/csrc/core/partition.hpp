// Two-tier partitioned placement of model extents in the weight arena (the paper's appendix
// "Memory Block Allocation"; Sec. 4.4): the arena is cut into partitions of a fixed size
// (the remainder, if at least one alignment unit, forms a short last partition). A model
// no larger than a partition goes into a slot of a partition dedicated to its size class
// when the class is common (several registered models share it; the caller decides), or
// into a buddy block of a buddy-managed partition when it is irregular; a larger model
// takes a run of consecutive free partitions. A partition returns to the free pool when
// its last occupant leaves. Runs are taken lowest-first and fresh dedicated or buddy
// partitions highest-first. A model's weights are one extent, so they are co-located by
// construction, and evicting a model frees its slot, block or run at once.
//
// Ties: the dedicated partition with the most occupied slots (then the lowest index), its
// lowest free slot; the buddy partition with the most bytes in allocated blocks (then the
// lowest index), in it the smallest large-enough free block (then the lowest offset),
// halved down to the smallest block size that holds the model. Block sizes of a partition
// of S bytes are S / 2^j while the half stays a multiple of the alignment.
//
// Consolidation (evacuate): the slot or buddy partition with the fewest bytes in use (then
// the lowest index) whose occupants can all be placed again, in increasing offset order,
// in other partitions without dedicating a free one, has them moved there and becomes
// free. Host-only C++.
#pragma once
#include <cstdint>
#include <functional>
#include <map>
#include <set>
#include <unordered_map>
#include <vector>

namespace tp {

class Partitions {
 public:
  Partitions(uint64_t capacity, uint64_t part_bytes, uint64_t align);

  // Places an extent of `bytes` (a multiple of the alignment) for model `id`; false (and
  // no change) if no placement exists without evicting. avoid >= 0: that partition is not
  // used and no free partition is dedicated (evacuation).
  bool place(int32_t id, uint64_t bytes, bool common, uint64_t* off, int avoid = -1);
  void release(int32_t id);

  struct Move {
    int32_t id;
    uint64_t from, to;
  };
  // Frees one slot or buddy partition by moving its occupants (appended to *moves in the
  // order made); false, and no change, if no partition can be evacuated. bytes(id) and
  // common(id) give each occupant's extent size and whether its class is common now.
  bool evacuate(const std::function<uint64_t(int32_t)>& bytes, const std::function<bool(int32_t)>& common,
                std::vector<Move>* moves);

  uint32_t count() const { return (uint32_t)parts_.size(); }
  uint32_t free_count() const;
  uint64_t part_bytes() const { return part_; }

 private:
  enum Kind { kFree, kSlab, kBuddy, kRun };
  struct Part {
    uint64_t start = 0, size = 0;
    Kind kind = kFree;
    uint64_t cls = 0;                                  // slab: the size class
    std::set<uint64_t> slots;                          // slab: occupied slot indices
    std::set<std::pair<uint64_t, uint64_t>> free_blk;  // buddy: free (size, offset)
    std::map<uint64_t, uint64_t> used_blk;             // buddy: offset -> size
    uint64_t used_bytes = 0;                           // buddy: bytes in allocated blocks
    void reset() {
      kind = kFree;
      cls = 0;
      slots.clear();
      free_blk.clear();
      used_blk.clear();
      used_bytes = 0;
    }
  };
  struct Where {
    Kind kind;
    uint32_t first, last;   // partition index (run: first..last)
    uint64_t pos;           // slab: slot index; buddy: offset in the partition
  };

  uint64_t block_size(uint64_t part_size, uint64_t need) const;
  int fresh(uint64_t need) const;                       // free partition, highest index first
  bool place_run(int32_t id, uint64_t bytes, uint64_t* off);
  bool place_slab(int32_t id, uint64_t bytes, uint64_t* off, int avoid);
  bool place_buddy(int32_t id, uint64_t bytes, uint64_t* off, int avoid);

  uint64_t part_, align_;
  std::vector<Part> parts_;
  std::unordered_map<int32_t, Where> where_;
};

}  // namespace tp
