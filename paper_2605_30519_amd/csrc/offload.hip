// offload.hip -- the GPU hot cache of full-resolution history chunks with LRU
// eviction (App. B "Inference and Offloading"; App. F's LRU-size study; Alg. 1's
// WaitUntilReload), and the chunk decode of Alg. 1 Step 1.
//
// Residency is per (head, chunk), as Alg. 1's pointer table: the GPU pool's
// per-head page tables map a head's resident chunks to its own slots, and the
// bookkeeping (lru_core.cpp) keeps an LRU per head.  A request names the
// (head, chunk) pairs a selection reads; its reloads run on a copy stream, after
// the work already enqueued on the compute stream (which may still read the slots
// being reused), and an event marks their end; omnimem_lru_wait makes any stream
// wait for it.  Reloading thus overlaps whatever the compute stream runs between
// omnimem_lru_require and omnimem_lru_wait.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <utility>
#include <vector>

#include "../../include/omnimem.h"
#include "device_common.h"
#include "launch.h"
#include "lru_core.h"
#include "numa.h"
#include "validate.h"

#define OMNIMEM_API extern "C" __attribute__((visibility("default")))

namespace {

// Page-table rows written by value (no staging memory): row i of the batch is the
// Bpc entries at table + at[i], set to first[i] + o, or to -1 when first[i] < 0.
constexpr int kRowBatch = 64;
struct RowBatch {
  int64_t at[kRowBatch];
  int32_t first[kRowBatch];
  int32_t count;
  int32_t Bpc;
};

__global__ __launch_bounds__(64) void k_write_rows(int32_t* __restrict__ table, RowBatch rb) {
  const int i = blockIdx.x;
  if (i >= rb.count) return;
  int32_t* row = table + rb.at[i];
  const int32_t first = rb.first[i];
  for (int o = threadIdx.x; o < rb.Bpc; o += 64) row[o] = first < 0 ? -1 : first + o;
}

// Alg. 1 Step 1's decode, per head: needed[h][c] = 1 when some group of head h
// lists a block of chunk c (block b in chunk b div Bpc).  One workgroup per head
// clears its row, then marks it.
__global__ __launch_bounds__(256) void k_selected_chunks(const int32_t* __restrict__ idx,
                                                         const int32_t* __restrict__ cnt, int R, int K, int nb,
                                                         int Bpc, int n, uint8_t* __restrict__ needed) {
  const int h = blockIdx.x;
  uint8_t* row = needed + static_cast<int64_t>(h) * n;
  for (int c = threadIdx.x; c < n; c += 256) row[c] = 0;
  __syncthreads();
  for (int e = threadIdx.x; e < R * K; e += 256) {
    const int r = e / K, t = e % K;
    const int c = cnt[h * R + r];
    if (t >= c) continue;
    const int b = idx[static_cast<int64_t>(h * R + r) * K + t];
    if (b >= 0 && b < nb) row[b / Bpc] = 1;
  }
}

}  // namespace

struct omnimem_lru {
  int H, Bpc, n_table;  // heads, blocks per chunk, chunks each head's table holds
  int64_t slab;         // bytes of one (page, head) slab
  int64_t stride;       // per-head table stride (entries)
  int slots;
  char* k_gpu;
  char* v_gpu;
  const char* k_host;
  const char* v_host;
  int32_t* table;
  omnimem::LruCore core;
  hipEvent_t before;    // end of the compute work enqueued before a request
  hipEvent_t reloaded;  // end of the last request's reloads
  bool pending = false, broken = false;
  int64_t bytes = 0;
};

namespace {

omnimem_status_t write_rows(omnimem_lru* L, const std::vector<std::pair<int64_t, int32_t>>& rows, hipStream_t s) {
  RowBatch rb{};
  rb.Bpc = L->Bpc;
  for (size_t i = 0; i < rows.size(); i += kRowBatch) {
    rb.count = 0;
    for (size_t j = i; j < rows.size() && rb.count < kRowBatch; ++j, ++rb.count) {
      rb.at[rb.count] = rows[j].first;
      rb.first[rb.count] = rows[j].second;
    }
    if (omnimem::launch_kernel(k_write_rows, dim3(rb.count), dim3(64), 0, s, L->table, rb) != hipSuccess)
      return OMNIMEM_EHIP;
  }
  return OMNIMEM_OK;
}

}  // namespace

OMNIMEM_API omnimem_status_t omnimem_selected_chunks(const omnimem_kv_cache_t* kv, const int32_t* idx,
                                                     const int32_t* cnt, int32_t groups, int32_t top_k,
                                                     uint8_t* needed, void* stream) {
  omnimem::CacheGeom g;
  const omnimem_status_t st = omnimem::check_selected_chunks(kv, idx, cnt, groups, top_k, needed, g);
  if (st != OMNIMEM_OK || g.n == 0) return st;
  return omnimem::launch_kernel(k_selected_chunks, dim3(g.H), dim3(256), 0, static_cast<hipStream_t>(stream), idx,
                                cnt, groups, top_k, g.nb, g.Bpc, g.n, needed) == hipSuccess
             ? OMNIMEM_OK
             : OMNIMEM_EHIP;
}

OMNIMEM_API omnimem_status_t omnimem_lru_create(const omnimem_kv_cache_t* kv, int32_t slots, const void* k_host,
                                                const void* v_host, int32_t host_chunks, void* stream,
                                                omnimem_lru_t** out) {
  if (out == nullptr) return OMNIMEM_EINVAL;
  *out = nullptr;
  omnimem::CacheGeom g;
  omnimem_status_t st = omnimem::resolve_cache(kv, g);
  if (st != OMNIMEM_OK) return st;
  if (g.n < 1 || g.pt_stride == 0 || g.page_table == nullptr) return OMNIMEM_EINVAL;  // per-head tables
  if (slots < 1 || host_chunks < g.n || static_cast<int64_t>(slots) * g.Bpc > g.num_pages) return OMNIMEM_EINVAL;
  if (g.k_pages == nullptr || g.v_pages == nullptr || k_host == nullptr || v_host == nullptr) return OMNIMEM_EINVAL;
  omnimem_lru* L = new (std::nothrow) omnimem_lru;
  if (L == nullptr) return OMNIMEM_EINVAL;
  L->H = g.H;
  L->Bpc = g.Bpc;
  L->n_table = g.n;
  L->slab = static_cast<int64_t>(g.B) * g.D * (g.dtype == 0 ? 2 : 4);
  L->stride = g.pt_stride;
  L->slots = slots;
  // the descriptor's pointers are const for the compute calls; this runtime is the
  // writer of the pool and of the tables the caller hands it
  L->k_gpu = static_cast<char*>(const_cast<void*>(g.k_pages));
  L->v_gpu = static_cast<char*>(const_cast<void*>(g.v_pages));
  L->k_host = static_cast<const char*>(k_host);
  L->v_host = static_cast<const char*>(v_host);
  L->table = const_cast<int32_t*>(g.page_table);
  if (!L->core.init(g.H, slots, g.n)) {
    delete L;
    return OMNIMEM_EINVAL;
  }
  if (hipEventCreateWithFlags(&L->before, hipEventDisableTiming) != hipSuccess) {
    delete L;
    return OMNIMEM_EHIP;
  }
  if (hipEventCreateWithFlags(&L->reloaded, hipEventDisableTiming) != hipSuccess) {
    (void)hipEventDestroy(L->before);
    delete L;
    return OMNIMEM_EHIP;
  }
  // nothing resident yet: every row of every head's table is -1
  std::vector<std::pair<int64_t, int32_t>> rows;
  try {
    rows.reserve(static_cast<size_t>(g.H) * g.n);
    for (int h = 0; h < g.H; ++h)
      for (int c = 0; c < g.n; ++c) rows.emplace_back(h * L->stride + static_cast<int64_t>(c) * g.Bpc, -1);
  } catch (...) {
    omnimem_lru_destroy(L);
    return OMNIMEM_EINVAL;
  }
  st = write_rows(L, rows, static_cast<hipStream_t>(stream));
  if (st != OMNIMEM_OK) {
    omnimem_lru_destroy(L);
    return st;
  }
  *out = L;
  return OMNIMEM_OK;
}

OMNIMEM_API void omnimem_lru_destroy(omnimem_lru_t* L) {
  if (L == nullptr) return;
  (void)hipEventDestroy(L->before);
  (void)hipEventDestroy(L->reloaded);
  delete L;
}

OMNIMEM_API omnimem_status_t omnimem_lru_require(omnimem_lru_t* L, const uint8_t* needed, int32_t n,
                                                 void* compute_stream, void* copy_stream, int32_t* reloaded) {
  if (L == nullptr) return OMNIMEM_EINVAL;
  if (L->broken) return OMNIMEM_EHIP;
  if (n < 0 || n > L->n_table || (n > 0 && needed == nullptr)) return OMNIMEM_EINVAL;
  std::vector<omnimem::LruLoad> loads;
  std::vector<std::pair<int64_t, int32_t>> evicted_rows, loaded_rows;
  const int rc = L->core.plan(needed, n, loads);
  if (rc != 0) return OMNIMEM_EINVAL;  // a head asks for more chunks than it has slots
  if (reloaded) *reloaded = static_cast<int32_t>(loads.size());
  if (loads.empty()) return OMNIMEM_OK;
  hipStream_t cs = static_cast<hipStream_t>(compute_stream), xs = static_cast<hipStream_t>(copy_stream);
  // From here on the bookkeeping has moved on: a failure leaves the runtime unusable.
  L->broken = true;
  try {
    evicted_rows.reserve(loads.size());
    loaded_rows.reserve(loads.size());
  } catch (...) {
    return OMNIMEM_EHIP;
  }
  for (const omnimem::LruLoad& l : loads)
    if (l.evicted >= 0) evicted_rows.emplace_back(l.head * L->stride + static_cast<int64_t>(l.evicted) * L->Bpc, -1);
  // the slots are reused only after the compute work that may still read them
  if (hipEventRecord(L->before, cs) != hipSuccess || hipStreamWaitEvent(xs, L->before, 0) != hipSuccess)
    return OMNIMEM_EHIP;
  if (write_rows(L, evicted_rows, xs) != OMNIMEM_OK) return OMNIMEM_EHIP;
  // Copies: the (page, head) slabs of a chunk sit H slabs apart in both pools, so
  // a (head, chunk) load is a strided copy of Bpc slabs; loads of one chunk into
  // one slot for a run of consecutive heads merge into one copy of wider rows.
  std::sort(loads.begin(), loads.end(), [](const omnimem::LruLoad& a, const omnimem::LruLoad& b) {
    if (a.chunk != b.chunk) return a.chunk < b.chunk;
    if (a.slot != b.slot) return a.slot < b.slot;
    return a.head < b.head;
  });
  const size_t pitch = static_cast<size_t>(L->H) * L->slab;
  for (size_t i = 0; i < loads.size();) {
    size_t j = i + 1;
    while (j < loads.size() && loads[j].chunk == loads[i].chunk && loads[j].slot == loads[i].slot &&
           loads[j].head == loads[j - 1].head + 1)
      ++j;
    const omnimem::LruLoad& l = loads[i];
    const size_t width = (j - i) * static_cast<size_t>(L->slab);
    const size_t src = (static_cast<size_t>(l.chunk) * L->Bpc * L->H + l.head) * L->slab;
    const size_t dst = (static_cast<size_t>(l.slot) * L->Bpc * L->H + l.head) * L->slab;
    if (hipMemcpy2DAsync(L->k_gpu + dst, pitch, L->k_host + src, pitch, width, L->Bpc, hipMemcpyHostToDevice,
                         xs) != hipSuccess ||
        hipMemcpy2DAsync(L->v_gpu + dst, pitch, L->v_host + src, pitch, width, L->Bpc, hipMemcpyHostToDevice,
                         xs) != hipSuccess)
      return OMNIMEM_EHIP;
    for (size_t k = i; k < j; ++k) {
      L->core.commit(loads[k]);
      loaded_rows.emplace_back(loads[k].head * L->stride + static_cast<int64_t>(loads[k].chunk) * L->Bpc,
                               loads[k].slot * L->Bpc);
      L->bytes += 2 * L->slab * L->Bpc;
    }
    i = j;
  }
  if (write_rows(L, loaded_rows, xs) != OMNIMEM_OK) return OMNIMEM_EHIP;
  if (hipEventRecord(L->reloaded, xs) != hipSuccess) return OMNIMEM_EHIP;
  L->pending = true;
  L->broken = false;
  return OMNIMEM_OK;
}

OMNIMEM_API omnimem_status_t omnimem_lru_wait(omnimem_lru_t* L, void* stream) {
  if (L == nullptr) return OMNIMEM_EINVAL;
  if (L->broken) return OMNIMEM_EHIP;
  if (!L->pending) return OMNIMEM_OK;
  return hipStreamWaitEvent(static_cast<hipStream_t>(stream), L->reloaded, 0) == hipSuccess ? OMNIMEM_OK
                                                                                            : OMNIMEM_EHIP;
}

OMNIMEM_API omnimem_status_t omnimem_lru_stats(const omnimem_lru_t* L, omnimem_lru_stats_t* out) {
  if (L == nullptr || out == nullptr) return OMNIMEM_EINVAL;
  out->hits = L->core.hits();
  out->misses = L->core.misses();
  out->evictions = L->core.evictions();
  out->bytes_reloaded = L->bytes;
  return OMNIMEM_OK;
}

OMNIMEM_API int32_t omnimem_lru_slot_of(const omnimem_lru_t* L, int32_t head, int32_t chunk) {
  if (L == nullptr) return -1;
  return L->core.slot_of(head, chunk);
}

OMNIMEM_API omnimem_status_t omnimem_numa_bind(int32_t device, int32_t* node) {
  if (node != nullptr) *node = -1;
  char bus[64] = {};
  if (hipDeviceGetPCIBusId(bus, static_cast<int>(sizeof(bus)), device) != hipSuccess) return OMNIMEM_EINVAL;
  const int nd = omnimem::numa_node_of_pci("/sys", bus);
  if (nd < 0) return OMNIMEM_OK;  // the system reports no NUMA node: nothing to bind
  const int rc = omnimem::bind_thread_to_node("/sys", nd);
  if (rc < 0) return OMNIMEM_EINVAL;
  if (node != nullptr && rc == 0) *node = nd;
  return OMNIMEM_OK;
}
