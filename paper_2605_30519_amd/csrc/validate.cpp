// validate.cpp -- host-side argument checks of the libomnimem entry points.
// Nothing here touches device memory: pointers are checked for presence and
// alignment only, and device-resident contents (page ids, block ids) are
// bounds-checked by the kernels themselves.
#include "validate.h"

#include <math.h>

namespace omnimem {
namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
bool good_scale(float s) { return isfinite(s) && s > 0.f; }

omnimem_status_t check_attn_common(const void* q, int32_t lq, const void* out) {
  if (lq < 0) return OMNIMEM_EINVAL;
  if (lq == 0) return OMNIMEM_OK;
  if (q == nullptr || out == nullptr || !aligned16(q) || !aligned16(out)) return OMNIMEM_EINVAL;
  return OMNIMEM_OK;
}

omnimem_status_t resolve_select(const omnimem_kv_cache_t* kv, int32_t lq, const omnimem_select_params_t* p,
                                CacheGeom& g, SelectPlan& plan, bool table_optional) {
  omnimem_status_t st = resolve_cache(kv, g, table_optional);
  if (st != OMNIMEM_OK) return st;
  if (p == nullptr || lq < 0) return OMNIMEM_EINVAL;
  if (p->top_k < 1 || p->group_size < 1 || p->window_chunks < 0 || p->awe_min_outside_chunks < 0 ||
      !good_scale(p->scale) || (p->score_mode != OMNIMEM_SCORE_LOGIT && p->score_mode != OMNIMEM_SCORE_PROB))
    return OMNIMEM_EINVAL;
  const int awe = awe_active(g.n, p->window_chunks, p->awe_min_outside_chunks, p->top_k, g.Bpc);
  if (lq == 0) {
    plan = SelectPlan{};
    plan.awe = awe;
    return OMNIMEM_OK;
  }
  plan = plan_select(g, lq, p->top_k, p->group_size, p->window_chunks, p->scale, awe, p->score_mode);
  return OMNIMEM_OK;
}

// Validates a compressed cache against the full cache's geometry.
omnimem_status_t resolve_cmp(const omnimem_cmp_cache_t* cc, const CacheGeom& g, CmpCache& c) {
  if (cc == nullptr) return OMNIMEM_EINVAL;
  if ((cc->dtype == OMNIMEM_BF16 ? 0 : cc->dtype == OMNIMEM_F32 ? 1 : -1) != g.dtype) return OMNIMEM_EINVAL;
  if (cc->num_heads != g.H || cc->head_dim != g.D || cc->block_size != g.B || cc->chunk_tokens != g.S)
    return OMNIMEM_EINVAL;
  if (cc->capacity_chunks < 0 || cc->num_pages < 0) return OMNIMEM_EINVAL;
  const int64_t cap = static_cast<int64_t>(cc->capacity_chunks) * g.Bpc;
  if (cap > (int64_t{1} << 30)) return OMNIMEM_EINVAL;
  const int64_t pages = (cap + kCmpPageTokens - 1) / kCmpPageTokens;
  if (cc->num_pages < pages) return OMNIMEM_EINVAL;
  if (cap > 0 && (cc->k_mean == nullptr || cc->k_pages == nullptr || cc->v_pages == nullptr ||
                  cc->page_table == nullptr))
    return OMNIMEM_EINVAL;
  if (!aligned16(cc->k_mean) || !aligned16(cc->k_pages) || !aligned16(cc->v_pages) || !aligned4(cc->page_table))
    return OMNIMEM_EINVAL;
  // the pooled keys' residual piece exists for bf16 caches only
  if (cc->k_lo != nullptr && (g.dtype != 0 || !aligned16(cc->k_lo))) return OMNIMEM_EINVAL;
  c.k_lo = cc->k_lo;
  c.k_mean = cc->k_mean;
  c.k_pages = cc->k_pages;
  c.v_pages = cc->v_pages;
  c.page_table = cc->page_table;
  c.num_pages = cc->num_pages;
  c.cap_blocks = static_cast<int>(cap);
  return OMNIMEM_OK;
}

void fill_lists(AttnLaunch& a, const void* q, int32_t lq, const int32_t* idx, const int32_t* cnt, int32_t top_k,
                int32_t group_size, float scale, void* out, float* lse) {
  a = AttnLaunch{};
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.lq = lq;
  a.group_size = group_size;
  a.R = (lq + group_size - 1) / group_size;
  a.idx = idx;
  a.cnt = cnt;
  a.top_k = top_k;
  a.scale = scale;
}

void fill_dense(AttnLaunch& a, const void* q, int32_t lq, int first_block, int num_blocks, float scale, void* out,
                float* lse) {
  a = AttnLaunch{};
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.lq = lq;
  a.group_size = lq;
  a.R = 1;
  a.top_k = 1;
  a.dense_first_block = first_block;
  a.dense_num_blocks = num_blocks;
  a.scale = scale;
}

}  // namespace

int32_t blocks_per_chunk(int32_t chunk_tokens, int32_t block_size) {
  if (chunk_tokens < 1 || block_size < 1) return -1;
  return (chunk_tokens + block_size - 1) / block_size;
}

int32_t awe_active(int32_t n, int32_t E, int32_t T_out, int32_t K, int32_t Bpc) {
  if (n < 0 || E < 0 || T_out < 0 || K < 1 || Bpc < 1) return -1;
  const int64_t outside = n > E ? static_cast<int64_t>(n) - E : 0;
  return (outside >= T_out && outside * Bpc >= K) ? 1 : 0;
}

const char* status_string(int32_t status) {
  switch (status) {
    case OMNIMEM_OK:
      return "ok";
    case OMNIMEM_EINVAL:
      return "invalid argument";
    case OMNIMEM_EUNSUPPORTED:
      return "unsupported shape or dtype";
    case OMNIMEM_EWORKSPACE:
      return "workspace too small";
    case OMNIMEM_EHIP:
      return "HIP launch error";
    case OMNIMEM_ESCRATCH:
      return "selection needs more scratch than omnimem_select_noalloc's static buffer";
    default:
      return "unknown status";
  }
}

omnimem_status_t resolve_cache(const omnimem_kv_cache_t* kv, CacheGeom& g, bool table_optional) {
  if (kv == nullptr) return OMNIMEM_EINVAL;
  if (kv->dtype != OMNIMEM_BF16 && kv->dtype != OMNIMEM_F32) return OMNIMEM_EUNSUPPORTED;
  if (kv->num_heads < 1 || kv->chunk_tokens < 1 || kv->num_chunks < 0 || kv->num_pages < 0) return OMNIMEM_EINVAL;
  if (kv->head_dim != 64 && kv->head_dim != 128) return OMNIMEM_EUNSUPPORTED;
  if (kv->block_size != 64 && kv->block_size != 128) return OMNIMEM_EUNSUPPORTED;
  g.dtype = kv->dtype == OMNIMEM_BF16 ? 0 : 1;
  g.H = kv->num_heads;
  g.D = kv->head_dim;
  g.B = kv->block_size;
  g.S = kv->chunk_tokens;
  g.n = kv->num_chunks;
  g.Bpc = (g.S + g.B - 1) / g.B;
  const int64_t nb = static_cast<int64_t>(g.n) * g.Bpc;
  if (nb > (int64_t{1} << 30)) return OMNIMEM_EINVAL;
  g.nb = static_cast<int>(nb);
  g.num_pages = kv->num_pages;
  // page pool size in elements must fit comfortably in int64 addressing
  if (g.num_pages > (int64_t{1} << 40) / (static_cast<int64_t>(g.H) * g.B * g.D)) return OMNIMEM_EINVAL;
  g.k_pages = kv->k_pages;
  g.v_pages = kv->v_pages;
  g.page_table = kv->page_table;
  // per-head tables: every head's table holds the n*Bpc blocks, and the last one
  // stays inside int64 index arithmetic
  g.pt_stride = kv->page_table_head_stride;
  if (g.pt_stride < 0 || (g.pt_stride > 0 && g.pt_stride < nb) || g.pt_stride > (int64_t{1} << 40))
    return OMNIMEM_EINVAL;
  if (g.nb > 0) {
    if (g.page_table == nullptr && !table_optional) return OMNIMEM_EINVAL;
    if (g.num_pages > 0 && (g.k_pages == nullptr || g.v_pages == nullptr)) return OMNIMEM_EINVAL;
    if (!aligned16(g.k_pages) || !aligned16(g.v_pages) || !aligned4(g.page_table)) return OMNIMEM_EINVAL;
  }
  return OMNIMEM_OK;
}

size_t select_workspace_bytes(const omnimem_kv_cache_t* kv, int32_t lq, const omnimem_select_params_t* p) {
  CacheGeom g;
  SelectPlan plan;
  // the size does not depend on the page table (NULL for omnimem_select_compressed)
  if (resolve_select(kv, lq, p, g, plan, /*table_optional=*/true) != OMNIMEM_OK) return 0;
  return lq == 0 ? 256 : plan.total;
}

omnimem_status_t check_select(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                              const omnimem_select_params_t* p, const int32_t* idx, const int32_t* cnt, CacheGeom& g,
                              SelectPlan& plan) {
  omnimem_status_t st = resolve_select(kv, lq, p, g, plan, false);
  if (st != OMNIMEM_OK) return st;
  if (p->score_mode != OMNIMEM_SCORE_LOGIT) return OMNIMEM_EINVAL;  // probabilities need the pooled history
  if (lq == 0) return OMNIMEM_OK;
  if (q == nullptr || idx == nullptr || cnt == nullptr || !aligned16(q)) return OMNIMEM_EINVAL;
  return OMNIMEM_OK;
}

omnimem_status_t check_workspace(const SelectPlan& plan, int32_t lq, const void* workspace, size_t workspace_bytes) {
  if (lq == 0) return OMNIMEM_OK;
  if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255u)) return OMNIMEM_EINVAL;
  if (workspace_bytes < plan.total) return OMNIMEM_EWORKSPACE;
  return OMNIMEM_OK;
}

omnimem_status_t check_sparse_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, const int32_t* idx,
                                   const int32_t* cnt, int32_t top_k, int32_t group_size, float scale,
                                   void* out, float* lse, CacheGeom& g, AttnLaunch& a) {
  omnimem_status_t st = resolve_cache(kv, g);
  if (st != OMNIMEM_OK) return st;
  if (top_k < 1 || group_size < 1 || !good_scale(scale)) return OMNIMEM_EINVAL;
  st = check_attn_common(q, lq, out);
  if (st != OMNIMEM_OK) return st;
  if (lq > 0 && (idx == nullptr || cnt == nullptr)) return OMNIMEM_EINVAL;
  fill_lists(a, q, lq, idx, cnt, top_k, group_size, scale, out, lse);
  return OMNIMEM_OK;
}

omnimem_status_t check_dense_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, int32_t chunk_begin,
                                  int32_t chunk_end, float scale, void* out, float* lse, CacheGeom& g,
                                  AttnLaunch& a) {
  omnimem_status_t st = resolve_cache(kv, g);
  if (st != OMNIMEM_OK) return st;
  if (chunk_begin < 0 || chunk_end < chunk_begin || chunk_end > g.n || !good_scale(scale)) return OMNIMEM_EINVAL;
  st = check_attn_common(q, lq, out);
  if (st != OMNIMEM_OK) return st;
  fill_dense(a, q, lq, chunk_begin * g.Bpc, (chunk_end - chunk_begin) * g.Bpc, scale, out, lse);
  return OMNIMEM_OK;
}

omnimem_status_t check_compress_chunk(const omnimem_kv_cache_t* kv, int32_t chunk, const omnimem_cmp_cache_t* cc,
                                      CacheGeom& g, CmpCache& c) {
  omnimem_status_t st = resolve_cache(kv, g);
  if (st != OMNIMEM_OK) return st;
  st = resolve_cmp(cc, g, c);
  if (st != OMNIMEM_OK) return st;
  if (chunk < 0 || chunk >= g.n || chunk >= cc->capacity_chunks) return OMNIMEM_EINVAL;
  return OMNIMEM_OK;
}

omnimem_status_t check_select_compressed(const omnimem_kv_cache_t* kv, const omnimem_cmp_cache_t* cc,
                                         const void* q, int32_t lq, const omnimem_select_params_t* p,
                                         const int32_t* idx, const int32_t* cnt, const void* workspace,
                                         size_t workspace_bytes, CacheGeom& g, SelectPlan& plan, CmpCache& c) {
  omnimem_status_t st = resolve_select(kv, lq, p, g, plan, /*table_optional=*/true);
  if (st != OMNIMEM_OK) return st;
  st = resolve_cmp(cc, g, c);
  if (st != OMNIMEM_OK) return st;
  if (g.n > cc->capacity_chunks) return OMNIMEM_EINVAL;
  if (lq == 0) return OMNIMEM_OK;
  if (q == nullptr || idx == nullptr || cnt == nullptr || !aligned16(q)) return OMNIMEM_EINVAL;
  return check_workspace(plan, lq, workspace, workspace_bytes);
}

omnimem_status_t check_cmp_attn(const omnimem_cmp_cache_t* cc, int32_t n_chunks, const void* q, int32_t lq,
                                float scale, void* out, float* lse, CacheGeom& g, AttnLaunch& a) {
  if (cc == nullptr) return OMNIMEM_EINVAL;
  // the pooled sequence as a one-chunk paged cache of n_chunks * Bpc tokens
  omnimem_kv_cache_t seq{};
  seq.dtype = cc->dtype;
  seq.num_heads = cc->num_heads;
  seq.head_dim = cc->head_dim;
  seq.block_size = cc->block_size;
  seq.chunk_tokens = cc->chunk_tokens;
  CacheGeom full;
  omnimem_status_t st = resolve_cache(&seq, full);
  if (st != OMNIMEM_OK) return st;
  CmpCache c;
  st = resolve_cmp(cc, full, c);
  if (st != OMNIMEM_OK) return st;
  if (n_chunks < 0 || n_chunks > cc->capacity_chunks || !good_scale(scale)) return OMNIMEM_EINVAL;
  const int64_t tokens = static_cast<int64_t>(n_chunks) * full.Bpc;
  g = full;
  g.B = kCmpPageTokens;
  g.S = tokens > 0 ? static_cast<int>(tokens) : 1;
  g.n = tokens > 0 ? 1 : 0;
  g.Bpc = (g.S + g.B - 1) / g.B;
  g.nb = g.n * g.Bpc;
  g.num_pages = c.num_pages;
  g.k_pages = c.k_pages;
  g.v_pages = c.v_pages;
  g.page_table = c.page_table;
  g.pt_stride = 0;
  st = check_attn_common(q, lq, out);
  if (st != OMNIMEM_OK) return st;
  fill_dense(a, q, lq, 0, g.nb, scale, out, lse);
  return OMNIMEM_OK;
}

omnimem_status_t check_gated_combine(int32_t dtype, int32_t lq, int32_t num_heads, int32_t head_dim,
                                     const void* o_cmp, const void* o_slc, const void* o_swa,
                                     const float* gate_logits, const void* out, int64_t& rows) {
  if (dtype != OMNIMEM_BF16 && dtype != OMNIMEM_F32) return OMNIMEM_EUNSUPPORTED;
  if (head_dim != 64 && head_dim != 128) return OMNIMEM_EUNSUPPORTED;
  if (lq < 0 || num_heads < 1) return OMNIMEM_EINVAL;
  rows = static_cast<int64_t>(lq) * num_heads;
  if (lq == 0) return OMNIMEM_OK;
  if (out == nullptr || gate_logits == nullptr || (o_cmp == nullptr && o_slc == nullptr && o_swa == nullptr))
    return OMNIMEM_EINVAL;
  if (!aligned16(out) || !aligned16(o_cmp) || !aligned16(o_slc) || !aligned16(o_swa) || !aligned4(gate_logits))
    return OMNIMEM_EINVAL;
  return OMNIMEM_OK;
}

size_t union_workspace_bytes(const omnimem_kv_cache_t* kv) {
  CacheGeom g;
  if (resolve_cache(kv, g) != OMNIMEM_OK) return 0;
  return plan_union(g).total;
}

omnimem_status_t check_union_gather(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, const int32_t* idx,
                                    const int32_t* cnt, int32_t top_k, int32_t group_size, float scale, void* out,
                                    float* lse, const int32_t* union_blocks, const void* workspace,
                                    size_t workspace_bytes, CacheGeom& g, UnionPlan& up, AttnLaunch& a) {
  omnimem_status_t st = resolve_cache(kv, g);
  if (st != OMNIMEM_OK) return st;
  if (top_k < 1 || group_size < 1 || !good_scale(scale)) return OMNIMEM_EINVAL;
  st = check_attn_common(q, lq, out);
  if (st != OMNIMEM_OK || lq == 0) return st;
  if (idx == nullptr || cnt == nullptr || union_blocks == nullptr || workspace == nullptr) return OMNIMEM_EINVAL;
  if (reinterpret_cast<uintptr_t>(workspace) & 255u) return OMNIMEM_EINVAL;
  if (g.pt_stride != 0) return OMNIMEM_EUNSUPPORTED;  // the comparator reads one shared table
  up = plan_union(g);
  if (workspace_bytes < up.total) return OMNIMEM_EWORKSPACE;
  fill_lists(a, q, lq, idx, cnt, top_k, group_size, scale, out, lse);
  return OMNIMEM_OK;
}

omnimem_status_t check_selected_chunks(const omnimem_kv_cache_t* kv, const int32_t* idx, const int32_t* cnt,
                                       int32_t groups, int32_t top_k, const uint8_t* needed, CacheGeom& g) {
  omnimem_status_t st = resolve_cache(kv, g, /*table_optional=*/true);
  if (st != OMNIMEM_OK) return st;
  if (groups < 0 || top_k < 1) return OMNIMEM_EINVAL;
  if (static_cast<int64_t>(g.H) * groups * top_k > (int64_t{1} << 31) - 1) return OMNIMEM_EINVAL;
  if (g.n > 0 && needed == nullptr) return OMNIMEM_EINVAL;
  if (groups > 0 && (idx == nullptr || cnt == nullptr || !aligned4(idx) || !aligned4(cnt))) return OMNIMEM_EINVAL;
  return OMNIMEM_OK;
}

}  // namespace omnimem
