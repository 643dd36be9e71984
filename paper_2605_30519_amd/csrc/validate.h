// validate.h -- the host-side argument checks of every libomnimem entry point
// (internal to the library).  No HIP here: validate.cpp builds with the host
// compiler, so the same checks run inside the library and, on a CPU, under
// AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Each check_* validates one entry point's arguments exactly as that entry point
// does before it enqueues anything, and fills in what its launch needs.  A call
// with lq == 0 passes its checks and has nothing to compute.
#pragma once

#include "../../include/omnimem.h"
#include "plan.h"

namespace omnimem {

int32_t blocks_per_chunk(int32_t chunk_tokens, int32_t block_size);
int32_t awe_active(int32_t n, int32_t E, int32_t T_out, int32_t K, int32_t Bpc);
const char* status_string(int32_t status);

// table_optional: a NULL page table is accepted (selection from pooled keys only).
omnimem_status_t resolve_cache(const omnimem_kv_cache_t* kv, CacheGeom& g, bool table_optional = false);

size_t select_workspace_bytes(const omnimem_kv_cache_t* kv, int32_t lq, const omnimem_select_params_t* p);

// omnimem_select's checks except the workspace (shared with omnimem_select_noalloc).
omnimem_status_t check_select(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                              const omnimem_select_params_t* p, const int32_t* idx, const int32_t* cnt, CacheGeom& g,
                              SelectPlan& plan);
// A caller workspace for `plan`: 256-byte aligned and large enough.
omnimem_status_t check_workspace(const SelectPlan& plan, int32_t lq, const void* workspace, size_t workspace_bytes);

omnimem_status_t check_sparse_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, const int32_t* idx,
                                   const int32_t* cnt, int32_t top_k, int32_t group_size, float scale,
                                   void* out, float* lse, CacheGeom& g, AttnLaunch& a);
omnimem_status_t check_dense_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, int32_t chunk_begin,
                                  int32_t chunk_end, float scale, void* out, float* lse, CacheGeom& g,
                                  AttnLaunch& a);
omnimem_status_t check_compress_chunk(const omnimem_kv_cache_t* kv, int32_t chunk, const omnimem_cmp_cache_t* cc,
                                      CacheGeom& g, CmpCache& c);
omnimem_status_t check_select_compressed(const omnimem_kv_cache_t* kv, const omnimem_cmp_cache_t* cc,
                                         const void* q, int32_t lq, const omnimem_select_params_t* p,
                                         const int32_t* idx, const int32_t* cnt, const void* workspace,
                                         size_t workspace_bytes, CacheGeom& g, SelectPlan& plan, CmpCache& c);
omnimem_status_t check_cmp_attn(const omnimem_cmp_cache_t* cc, int32_t n_chunks, const void* q, int32_t lq,
                                float scale, void* out, float* lse, CacheGeom& g, AttnLaunch& a);
omnimem_status_t check_gated_combine(int32_t dtype, int32_t lq, int32_t num_heads, int32_t head_dim,
                                     const void* o_cmp, const void* o_slc, const void* o_swa,
                                     const float* gate_logits, const void* out, int64_t& rows);
size_t union_workspace_bytes(const omnimem_kv_cache_t* kv);
omnimem_status_t check_union_gather(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, const int32_t* idx,
                                    const int32_t* cnt, int32_t top_k, int32_t group_size, float scale, void* out,
                                    float* lse, const int32_t* union_blocks, const void* workspace,
                                    size_t workspace_bytes, CacheGeom& g, UnionPlan& up, AttnLaunch& a);
// omnimem_selected_chunks: idx/cnt of R groups per head and the [H][n] mask.
omnimem_status_t check_selected_chunks(const omnimem_kv_cache_t* kv, const int32_t* idx, const int32_t* cnt,
                                       int32_t groups, int32_t top_k, const uint8_t* needed, CacheGeom& g);

}  // namespace omnimem
