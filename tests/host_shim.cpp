// Host-only build of libomnimem's argument checks and host runtime pieces, for the
// sanitizer test (CPU only; never loaded next to the real library).  Each compute
// entry point below runs the library's own checks from validate.cpp and returns
// their status where the library would launch its kernels; the LRU bookkeeping and
// the NUMA helpers are exposed through small shim_* calls.
#include <stdint.h>

#include <vector>

#include "../include/omnimem.h"
#include "../paper_2605_30519_amd/csrc/lru_core.h"
#include "../paper_2605_30519_amd/csrc/numa.h"
#include "../paper_2605_30519_amd/csrc/validate.h"

using namespace omnimem;

extern "C" {

int32_t omnimem_blocks_per_chunk(int32_t s, int32_t b) { return blocks_per_chunk(s, b); }
int32_t omnimem_awe_active(int32_t n, int32_t e, int32_t t, int32_t k, int32_t bpc) { return awe_active(n, e, t, k, bpc); }
const char* omnimem_status_string(int32_t st) { return status_string(st); }
size_t omnimem_select_workspace_bytes(const omnimem_kv_cache_t* kv, int32_t lq, const omnimem_select_params_t* p) {
  return select_workspace_bytes(kv, lq, p);
}
size_t omnimem_union_workspace_bytes(const omnimem_kv_cache_t* kv) { return union_workspace_bytes(kv); }

omnimem_status_t omnimem_select(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt, float*,
                                int32_t* awe, void* ws, size_t ws_bytes, void*) {
  CacheGeom g;
  SelectPlan plan;
  omnimem_status_t st = check_select(kv, q, lq, p, idx, cnt, g, plan);
  if (st == OMNIMEM_OK) st = check_workspace(plan, lq, ws, ws_bytes);
  if (st == OMNIMEM_OK && awe != nullptr) *awe = plan.awe;
  return st;
}

omnimem_status_t omnimem_select_noalloc(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                        const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt, float*,
                                        int32_t* awe, void*) {
  CacheGeom g;
  SelectPlan plan;
  omnimem_status_t st = check_select(kv, q, lq, p, idx, cnt, g, plan);
  if (st == OMNIMEM_OK && lq > 0 && plan.total > OMNIMEM_NOALLOC_SCRATCH_BYTES) st = OMNIMEM_ESCRATCH;
  if (st == OMNIMEM_OK && awe != nullptr) *awe = plan.awe;
  return st;
}

omnimem_status_t omnimem_sparse_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, const int32_t* idx,
                                     const int32_t* cnt, int32_t top_k, int32_t g_size, float scale, void* out,
                                     float* lse, void*) {
  CacheGeom g;
  AttnLaunch a;
  return check_sparse_attn(kv, q, lq, idx, cnt, top_k, g_size, scale, out, lse, g, a);
}

omnimem_status_t omnimem_dense_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, int32_t c0, int32_t c1,
                                    float scale, void* out, float* lse, void*) {
  CacheGeom g;
  AttnLaunch a;
  return check_dense_attn(kv, q, lq, c0, c1, scale, out, lse, g, a);
}

omnimem_status_t omnimem_union_gather_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                           const int32_t* idx, const int32_t* cnt, int32_t top_k, int32_t g_size,
                                           float scale, void* out, float* lse, int32_t* ub, void* ws,
                                           size_t ws_bytes, void*) {
  CacheGeom g;
  UnionPlan up;
  AttnLaunch a;
  return check_union_gather(kv, q, lq, idx, cnt, top_k, g_size, scale, out, lse, ub, ws, ws_bytes, g, up, a);
}

omnimem_status_t omnimem_compress_chunk(const omnimem_kv_cache_t* kv, int32_t chunk, const omnimem_cmp_cache_t* cc,
                                        void*) {
  CacheGeom g;
  CmpCache c;
  return check_compress_chunk(kv, chunk, cc, g, c);
}

omnimem_status_t omnimem_select_compressed(const omnimem_kv_cache_t* kv, const omnimem_cmp_cache_t* cc,
                                           const void* q, int32_t lq, const omnimem_select_params_t* p,
                                           int32_t* idx, int32_t* cnt, float*, int32_t* awe, void* ws,
                                           size_t ws_bytes, void*) {
  CacheGeom g;
  SelectPlan plan;
  CmpCache c;
  const omnimem_status_t st = check_select_compressed(kv, cc, q, lq, p, idx, cnt, ws, ws_bytes, g, plan, c);
  if (st == OMNIMEM_OK && awe != nullptr) *awe = plan.awe;
  return st;
}

omnimem_status_t omnimem_cmp_attn(const omnimem_cmp_cache_t* cc, int32_t n, const void* q, int32_t lq, float scale,
                                  void* out, float* lse, void*) {
  CacheGeom g;
  AttnLaunch a;
  return check_cmp_attn(cc, n, q, lq, scale, out, lse, g, a);
}

omnimem_status_t omnimem_gated_combine(int32_t dtype, int32_t lq, int32_t h, int32_t d, const void* a,
                                       const void* b, const void* c, const float* gate, void* out, void*) {
  int64_t rows = 0;
  return check_gated_combine(dtype, lq, h, d, a, b, c, gate, out, rows);
}

omnimem_status_t omnimem_selected_chunks(const omnimem_kv_cache_t* kv, const int32_t* idx, const int32_t* cnt,
                                         int32_t groups, int32_t top_k, uint8_t* needed, void*) {
  CacheGeom g;
  return check_selected_chunks(kv, idx, cnt, groups, top_k, needed, g);
}

// ---- LRU bookkeeping
void* shim_lru_new(int heads, int slots, int chunks) {
  LruCore* core = new LruCore;
  if (!core->init(heads, slots, chunks)) {
    delete core;
    return nullptr;
  }
  return core;
}

void shim_lru_free(void* core) { delete static_cast<LruCore*>(core); }

// Plans one request; writes up to `cap` loads as (head, chunk, slot, evicted)
// quadruples and their count.  Returns plan()'s code.
int shim_lru_plan(void* core, const uint8_t* needed, int n, int32_t* loads, int cap, int* count) {
  std::vector<LruLoad> v;
  const int rc = static_cast<LruCore*>(core)->plan(needed, n, v);
  *count = static_cast<int>(v.size());
  for (int i = 0; i < *count && i < cap; ++i) {
    loads[4 * i] = v[i].head;
    loads[4 * i + 1] = v[i].chunk;
    loads[4 * i + 2] = v[i].slot;
    loads[4 * i + 3] = v[i].evicted;
  }
  return rc;
}

void shim_lru_commit(void* core, int head, int chunk, int slot, int evicted) {
  static_cast<LruCore*>(core)->commit(LruLoad{head, chunk, slot, evicted});
}

int shim_lru_slot_of(void* core, int h, int c) { return static_cast<LruCore*>(core)->slot_of(h, c); }
int shim_lru_chunk_in(void* core, int h, int s) { return static_cast<LruCore*>(core)->chunk_in(h, s); }

void shim_lru_counts(void* core, int64_t* out) {
  const LruCore* c = static_cast<LruCore*>(core);
  out[0] = c->hits();
  out[1] = c->misses();
  out[2] = c->evictions();
}

// ---- NUMA helpers
int shim_parse_cpu_list(const char* text, uint64_t* mask, int words) { return parse_cpu_list(text, mask, words); }
int shim_numa_node_of_pci(const char* root, const char* bus) { return numa_node_of_pci(root, bus); }
int shim_bind_thread_to_node(const char* root, int node) { return bind_thread_to_node(root, node); }

}  // extern "C"
