// lru_core.h -- bookkeeping of the LRU hot cache of full-resolution history chunks
// (internal to the library; host only, no HIP).  App. B ("Inference and
// Offloading") keeps a few chunks on the GPU and reloads the others from host
// memory when selected; Alg. 1's pointer table is indexed by head and chunk, so
// residency here is per (head, chunk): each head has `slots` chunk slots of its own
// and an LRU order of its own.  offload.hip turns a plan into copies and
// page-table writes.  Not thread-safe; no member throws.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

namespace omnimem {

// One reload: chunk `chunk` of head `head` into the head's slot `slot`, which held
// chunk `evicted` before this request (-1: the slot was free).
struct LruLoad {
  int head, chunk, slot, evicted;
};

class LruCore {
 public:
  // false on sizes < 1 or when the tables cannot be allocated
  bool init(int heads, int slots, int chunks) noexcept;

  int heads() const noexcept { return heads_; }
  int slots() const noexcept { return slots_; }
  int chunks() const noexcept { return chunks_; }

  // Plans one request.  needed[h * n + c] != 0 asks for chunk c of head h, for
  // c < n <= chunks().  Per head, the requested chunks are taken in ascending id:
  // the resident ones are hits and become most recently used in that order; then
  // each other one takes the lowest free slot, or else the slot of the least
  // recently used chunk that this request does not ask for, and becomes most
  // recently used.  Returns -1, changing nothing, if n is out of range or a head
  // asks for more chunks than it has slots; -2, changing nothing, if `loads`
  // cannot grow.  On success returns 0, appends every miss to `loads` (heads in
  // order, chunks ascending) and counts hits; every slot named by a load is
  // already vacated (its old chunk is no longer resident), and the load's chunk
  // becomes resident only through commit().
  int plan(const uint8_t* needed, int n, std::vector<LruLoad>& loads) noexcept;

  // The copy of `l` has been enqueued: its chunk lives in its slot from now on.
  void commit(const LruLoad& l) noexcept;

  // Slot of chunk c of head h, or -1 when it is not resident.
  int slot_of(int h, int c) const noexcept;
  // Chunk held by slot s of head h, or -1 when the slot is free.
  int chunk_in(int h, int s) const noexcept;

  int64_t hits() const noexcept { return hits_; }
  int64_t misses() const noexcept { return misses_; }
  int64_t evictions() const noexcept { return evictions_; }

 private:
  int heads_ = 0, slots_ = 0, chunks_ = 0;
  std::vector<int> slot_chunk_;       // [heads][slots]: chunk held, -1 = free
  std::vector<int> chunk_slot_;       // [heads][chunks]: slot holding it, -1 = not resident
  std::vector<uint64_t> last_use_;    // [heads][slots]: recency stamp
  std::vector<uint64_t> taken_at_;    // [heads][slots]: the request that last claimed the slot
  uint64_t clock_ = 0, requests_ = 0;
  int64_t hits_ = 0, misses_ = 0, evictions_ = 0;
};

}  // namespace omnimem
