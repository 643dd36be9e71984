// offload.hip -- the GPU hot cache of full-resolution history chunks with LRU
// eviction (App. B "Inference and Offloading"; App. F's LRU-size study; Alg. 1's
// WaitUntilReload).  Host-side runtime: every chunk lives in caller-allocated pinned
// host pools; the GPU page pool holds `slots` chunks.  omnimem_lru_require makes a
// set of chunks resident before the selection attention that reads them: hits
// refresh their recency, misses evict the least recently used chunk outside the set
// (its page-table row becomes -1, "not resident") and are reloaded by asynchronous
// host-to-device copies on the caller's stream, after which their page-table row
// points at the slot.  Everything is enqueued on that stream in order, so the
// attention launched after it on the same stream sees the chunks.
#include <stdint.h>

#include <new>
#include <vector>

#include "../../include/omnimem.h"
#include "device_common.h"

namespace {

// row[o] = first < 0 ? -1 : first + o for o < n: one page-table row, values passed by
// value so the launch needs no staging memory.
__global__ __launch_bounds__(64) void k_set_row(int32_t* __restrict__ row, int n, int32_t first) {
  for (int o = threadIdx.x; o < n; o += 64) row[o] = first < 0 ? -1 : first + o;
}

}  // namespace

struct omnimem_lru {
  int H, D, B, S, Bpc, elem;
  int slots, host_chunks, table_chunks;
  int64_t page_bytes;
  char* k_gpu;
  char* v_gpu;
  const char* k_host;
  const char* v_host;
  int32_t* page_table;
  std::vector<int> slot_chunk;      // chunk held by each slot, -1 = free
  std::vector<int> chunk_slot;      // slot holding each chunk, -1 = on the host only
  std::vector<uint64_t> last_use;   // per slot
  std::vector<uint64_t> pinned_at;  // per slot: the require call that needs it
  uint64_t clock = 0, calls = 0;
  omnimem_lru_stats_t stats{};
};

#define OMNIMEM_API extern "C" __attribute__((visibility("default")))

OMNIMEM_API omnimem_status_t omnimem_lru_create(const omnimem_kv_cache_t* kv, int32_t slots, const void* k_host,
                                                const void* v_host, int32_t host_chunks, void* stream,
                                                omnimem_lru_t** out) {
  if (kv == nullptr || out == nullptr) return OMNIMEM_EINVAL;
  *out = nullptr;
  if (kv->dtype != OMNIMEM_BF16 && kv->dtype != OMNIMEM_F32) return OMNIMEM_EUNSUPPORTED;
  if (kv->num_heads < 1 || kv->chunk_tokens < 1 || kv->num_chunks < 0) return OMNIMEM_EINVAL;
  if (kv->head_dim != 64 && kv->head_dim != 128) return OMNIMEM_EUNSUPPORTED;
  if (kv->block_size != 64 && kv->block_size != 128) return OMNIMEM_EUNSUPPORTED;
  const int Bpc = (kv->chunk_tokens + kv->block_size - 1) / kv->block_size;
  if (slots < 1 || host_chunks < 1 || static_cast<int64_t>(slots) * Bpc > kv->num_pages) return OMNIMEM_EINVAL;
  if (kv->k_pages == nullptr || kv->v_pages == nullptr || kv->page_table == nullptr || k_host == nullptr ||
      v_host == nullptr)
    return OMNIMEM_EINVAL;
  omnimem_lru* L = new (std::nothrow) omnimem_lru;
  if (L == nullptr) return OMNIMEM_EINVAL;
  L->H = kv->num_heads;
  L->D = kv->head_dim;
  L->B = kv->block_size;
  L->S = kv->chunk_tokens;
  L->Bpc = Bpc;
  L->elem = kv->dtype == OMNIMEM_BF16 ? 2 : 4;
  L->slots = slots;
  L->host_chunks = host_chunks;
  L->table_chunks = kv->num_chunks;
  L->page_bytes = static_cast<int64_t>(L->H) * L->B * L->D * L->elem;
  // the descriptor's pointers are const for the compute calls; this runtime is the
  // writer of the pool and the table the caller hands it
  L->k_gpu = static_cast<char*>(const_cast<void*>(kv->k_pages));
  L->v_gpu = static_cast<char*>(const_cast<void*>(kv->v_pages));
  L->k_host = static_cast<const char*>(k_host);
  L->v_host = static_cast<const char*>(v_host);
  L->page_table = const_cast<int32_t*>(kv->page_table);
  try {  // no exception may cross the C boundary
    L->slot_chunk.assign(slots, -1);
    L->chunk_slot.assign(host_chunks, -1);
    L->last_use.assign(slots, 0);
    L->pinned_at.assign(slots, 0);
  } catch (...) {
    delete L;
    return OMNIMEM_EINVAL;
  }
  // nothing resident yet: every row of the page table is -1
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int c = 0; c < L->table_chunks; ++c)
    hipLaunchKernelGGL(k_set_row, dim3(1), dim3(64), 0, s, L->page_table + static_cast<int64_t>(c) * Bpc, Bpc, -1);
  if (hipGetLastError() != hipSuccess) {
    delete L;
    return OMNIMEM_EHIP;
  }
  *out = L;
  return OMNIMEM_OK;
}

OMNIMEM_API void omnimem_lru_destroy(omnimem_lru_t* lru) { delete lru; }

OMNIMEM_API omnimem_status_t omnimem_lru_require(omnimem_lru_t* L, const int32_t* chunks, int32_t count,
                                                 int32_t* reloaded, void* stream) {
  if (L == nullptr || count < 0 || (count > 0 && chunks == nullptr)) return OMNIMEM_EINVAL;
  for (int i = 0; i < count; ++i)
    if (chunks[i] < 0 || chunks[i] >= L->host_chunks || chunks[i] >= L->table_chunks) return OMNIMEM_EINVAL;
  // the distinct chunks of the request must fit in the slots together
  std::vector<int> want;
  try {  // no exception may cross the C boundary
    want.reserve(count);
    std::vector<char> seen(L->host_chunks, 0);
    for (int i = 0; i < count; ++i)
      if (!seen[chunks[i]]) {
        seen[chunks[i]] = 1;
        want.push_back(chunks[i]);
      }
  } catch (...) {
    return OMNIMEM_EINVAL;
  }
  if (static_cast<int>(want.size()) > L->slots) return OMNIMEM_EINVAL;
  const uint64_t call = ++L->calls;
  // hits first: they are pinned for this call so that no miss evicts them
  for (int c : want) {
    const int slot = L->chunk_slot[c];
    if (slot >= 0) {
      L->last_use[slot] = ++L->clock;
      L->pinned_at[slot] = call;
      ++L->stats.hits;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  int loads = 0;
  for (int c : want) {
    if (L->chunk_slot[c] >= 0) continue;
    // victim: a free slot, else the least recently used slot this call does not need
    int victim = -1;
    for (int t = 0; t < L->slots; ++t) {
      if (L->pinned_at[t] == call) continue;
      if (L->slot_chunk[t] < 0) {
        victim = t;
        break;
      }
      if (victim < 0 || L->last_use[t] < L->last_use[victim]) victim = t;
    }
    if (victim < 0) return OMNIMEM_EINVAL;  // cannot happen: want.size() <= slots
    const int old = L->slot_chunk[victim];
    if (old >= 0) {
      hipLaunchKernelGGL(k_set_row, dim3(1), dim3(64), 0, s, L->page_table + static_cast<int64_t>(old) * L->Bpc,
                         L->Bpc, -1);
      L->chunk_slot[old] = -1;
      ++L->stats.evictions;
    }
    const int64_t bytes = L->page_bytes * L->Bpc;
    const int64_t src = static_cast<int64_t>(c) * bytes, dst = static_cast<int64_t>(victim) * bytes;
    if (hipMemcpyAsync(L->k_gpu + dst, L->k_host + src, bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(L->v_gpu + dst, L->v_host + src, bytes, hipMemcpyHostToDevice, s) != hipSuccess)
      return OMNIMEM_EHIP;
    hipLaunchKernelGGL(k_set_row, dim3(1), dim3(64), 0, s, L->page_table + static_cast<int64_t>(c) * L->Bpc, L->Bpc,
                       victim * L->Bpc);
    L->slot_chunk[victim] = c;
    L->chunk_slot[c] = victim;
    L->last_use[victim] = ++L->clock;
    L->pinned_at[victim] = call;
    ++L->stats.misses;
    L->stats.bytes_reloaded += 2 * bytes;
    ++loads;
  }
  if (hipGetLastError() != hipSuccess) return OMNIMEM_EHIP;
  if (reloaded) *reloaded = loads;
  return OMNIMEM_OK;
}

OMNIMEM_API omnimem_status_t omnimem_lru_stats(const omnimem_lru_t* L, omnimem_lru_stats_t* out) {
  if (L == nullptr || out == nullptr) return OMNIMEM_EINVAL;
  *out = L->stats;
  return OMNIMEM_OK;
}

OMNIMEM_API int32_t omnimem_lru_slot_of(const omnimem_lru_t* L, int32_t chunk) {
  if (L == nullptr || chunk < 0 || chunk >= L->host_chunks) return -1;
  return L->chunk_slot[chunk];
}
