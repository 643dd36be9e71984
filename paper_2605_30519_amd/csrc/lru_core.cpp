// lru_core.cpp -- per-(head, chunk) LRU bookkeeping of the hot cache (host only).
#include "lru_core.h"

#include <new>

namespace omnimem {

bool LruCore::init(int heads, int slots, int chunks) noexcept {
  if (heads < 1 || slots < 1 || chunks < 1) return false;
  if (static_cast<int64_t>(heads) * slots > (int64_t{1} << 28) || static_cast<int64_t>(heads) * chunks > (int64_t{1} << 28))
    return false;
  try {
    slot_chunk_.assign(static_cast<size_t>(heads) * slots, -1);
    chunk_slot_.assign(static_cast<size_t>(heads) * chunks, -1);
    last_use_.assign(static_cast<size_t>(heads) * slots, 0);
    taken_at_.assign(static_cast<size_t>(heads) * slots, 0);
  } catch (...) {
    return false;
  }
  heads_ = heads;
  slots_ = slots;
  chunks_ = chunks;
  clock_ = requests_ = 0;
  hits_ = misses_ = evictions_ = 0;
  return true;
}

int LruCore::plan(const uint8_t* needed, int n, std::vector<LruLoad>& loads) noexcept {
  if (heads_ == 0 || n < 0 || n > chunks_ || (n > 0 && needed == nullptr)) return -1;
  // read-only pass: every head's request fits its slots; count the misses
  size_t misses = 0;
  for (int h = 0; h < heads_; ++h) {
    int want = 0;
    for (int c = 0; c < n; ++c) {
      if (!needed[static_cast<size_t>(h) * n + c]) continue;
      ++want;
      if (chunk_slot_[static_cast<size_t>(h) * chunks_ + c] < 0) ++misses;
    }
    if (want > slots_) return -1;
  }
  try {
    loads.reserve(loads.size() + misses);
  } catch (...) {
    return -2;
  }
  const uint64_t req = ++requests_;
  for (int h = 0; h < heads_; ++h) {
    int* slot_chunk = slot_chunk_.data() + static_cast<size_t>(h) * slots_;
    int* chunk_slot = chunk_slot_.data() + static_cast<size_t>(h) * chunks_;
    uint64_t* last_use = last_use_.data() + static_cast<size_t>(h) * slots_;
    uint64_t* taken_at = taken_at_.data() + static_cast<size_t>(h) * slots_;
    const uint8_t* row = needed + static_cast<size_t>(h) * n;
    for (int c = 0; c < n; ++c) {
      const int s = row[c] ? chunk_slot[c] : -1;
      if (s < 0) continue;
      last_use[s] = ++clock_;
      taken_at[s] = req;
      ++hits_;
    }
    for (int c = 0; c < n; ++c) {
      if (!row[c] || chunk_slot[c] >= 0) continue;
      int victim = -1;
      for (int s = 0; s < slots_; ++s) {
        if (taken_at[s] == req) continue;
        if (slot_chunk[s] < 0) {
          victim = s;
          break;
        }
        if (victim < 0 || last_use[s] < last_use[victim]) victim = s;
      }
      // a victim always exists: this head asks for at most slots_ chunks
      const int old = slot_chunk[victim];
      if (old >= 0) {
        chunk_slot[old] = -1;
        ++evictions_;
      }
      slot_chunk[victim] = -1;
      last_use[victim] = ++clock_;
      taken_at[victim] = req;
      loads.push_back(LruLoad{h, c, victim, old});  // capacity reserved above
    }
  }
  return 0;
}

void LruCore::commit(const LruLoad& l) noexcept {
  if (l.head < 0 || l.head >= heads_ || l.slot < 0 || l.slot >= slots_ || l.chunk < 0 || l.chunk >= chunks_) return;
  slot_chunk_[static_cast<size_t>(l.head) * slots_ + l.slot] = l.chunk;
  chunk_slot_[static_cast<size_t>(l.head) * chunks_ + l.chunk] = l.slot;
  ++misses_;
}

int LruCore::slot_of(int h, int c) const noexcept {
  if (h < 0 || h >= heads_ || c < 0 || c >= chunks_) return -1;
  return chunk_slot_[static_cast<size_t>(h) * chunks_ + c];
}

int LruCore::chunk_in(int h, int s) const noexcept {
  if (h < 0 || h >= heads_ || s < 0 || s >= slots_) return -1;
  return slot_chunk_[static_cast<size_t>(h) * slots_ + s];
}

}  // namespace omnimem
