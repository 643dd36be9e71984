// api.hip -- the extern "C" entry points of libomnimem.so: the host-side checks
// of validate.cpp, then the kernel launches.  Nothing here allocates memory or
// synchronises with the device.
#include <stdint.h>

#include <mutex>

#include "../../include/omnimem.h"
#include "launch.h"
#include "validate.h"

#define OMNIMEM_API extern "C" __attribute__((visibility("default")))

// Device scratch of omnimem_select_noalloc, for callers that cannot allocate.  One
// copy per GPU, alive until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory: only the address resolved per device by
// hipGetSymbolAddress may be passed to kernels.
static __device__ __align__(256) unsigned char scratch[OMNIMEM_NOALLOC_SCRATCH_BYTES];

namespace {

using omnimem::AttnLaunch;
using omnimem::CacheGeom;
using omnimem::CmpCache;
using omnimem::SelectPlan;

omnimem_status_t hip_status(hipError_t e) { return e == hipSuccess ? OMNIMEM_OK : OMNIMEM_EHIP; }

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// Device address of `scratch` on each device, resolved once per device with that
// device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_addr[kMaxDevices];

omnimem_status_t scratch_of_current_device(void** addr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return OMNIMEM_EHIP;
  if (dev >= kMaxDevices) return OMNIMEM_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_addr[dev] == nullptr) {
    void* a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || a == nullptr) return OMNIMEM_EHIP;
    g_scratch_addr[dev] = a;
  }
  *addr = g_scratch_addr[dev];
  return OMNIMEM_OK;
}

}  // namespace

OMNIMEM_API int32_t omnimem_blocks_per_chunk(int32_t chunk_tokens, int32_t block_size) {
  return omnimem::blocks_per_chunk(chunk_tokens, block_size);
}

OMNIMEM_API int32_t omnimem_awe_active(int32_t n, int32_t E, int32_t T_out, int32_t K, int32_t Bpc) {
  return omnimem::awe_active(n, E, T_out, K, Bpc);
}

OMNIMEM_API size_t omnimem_select_workspace_bytes(const omnimem_kv_cache_t* kv, int32_t lq,
                                                  const omnimem_select_params_t* p) {
  return omnimem::select_workspace_bytes(kv, lq, p);
}

OMNIMEM_API omnimem_status_t omnimem_select(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                            const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt,
                                            float* score, int32_t* awe_active, void* workspace,
                                            size_t workspace_bytes, void* stream) {
  CacheGeom g;
  SelectPlan plan;
  omnimem_status_t st = omnimem::check_select(kv, q, lq, p, idx, cnt, g, plan);
  if (st == OMNIMEM_OK) st = omnimem::check_workspace(plan, lq, workspace, workspace_bytes);
  if (st != OMNIMEM_OK) return st;
  if (awe_active) *awe_active = plan.awe;
  if (lq == 0) return OMNIMEM_OK;
  return hip_status(omnimem::launch_select(g, plan, q, idx, cnt, score, workspace, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_select_noalloc(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                                    const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt,
                                                    float* score, int32_t* awe_active, void* stream) {
  CacheGeom g;
  SelectPlan plan;
  omnimem_status_t st = omnimem::check_select(kv, q, lq, p, idx, cnt, g, plan);
  if (st != OMNIMEM_OK) return st;
  if (lq > 0 && plan.total > OMNIMEM_NOALLOC_SCRATCH_BYTES) return OMNIMEM_ESCRATCH;
  void* ws = nullptr;
  if (lq > 0) {
    st = scratch_of_current_device(&ws);
    if (st != OMNIMEM_OK) return st;
  }
  if (awe_active) *awe_active = plan.awe;
  if (lq == 0) return OMNIMEM_OK;
  // the kernels write every scratch word they later read, so the previous call's
  // contents need no clearing
  return hip_status(omnimem::launch_select(g, plan, q, idx, cnt, score, ws, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_sparse_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                                 const int32_t* idx, const int32_t* cnt, int32_t top_k,
                                                 int32_t group_size, float scale, void* out, float* lse,
                                                 void* stream) {
  CacheGeom g;
  AttnLaunch a;
  const omnimem_status_t st = omnimem::check_sparse_attn(kv, q, lq, idx, cnt, top_k, group_size, scale, out, lse, g,
                                                         a);
  if (st != OMNIMEM_OK || lq == 0) return st;
  return hip_status(omnimem::launch_attention(g, a, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_dense_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                                int32_t chunk_begin, int32_t chunk_end, float scale, void* out,
                                                float* lse, void* stream) {
  CacheGeom g;
  AttnLaunch a;
  const omnimem_status_t st = omnimem::check_dense_attn(kv, q, lq, chunk_begin, chunk_end, scale, out, lse, g, a);
  if (st != OMNIMEM_OK || lq == 0) return st;
  return hip_status(omnimem::launch_attention(g, a, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_compress_chunk(const omnimem_kv_cache_t* kv, int32_t chunk,
                                                    const omnimem_cmp_cache_t* cc, void* stream) {
  CacheGeom g;
  CmpCache c;
  const omnimem_status_t st = omnimem::check_compress_chunk(kv, chunk, cc, g, c);
  if (st != OMNIMEM_OK) return st;
  return hip_status(omnimem::launch_compress_chunk(g, c, chunk, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_select_compressed(const omnimem_kv_cache_t* kv, const omnimem_cmp_cache_t* cc,
                                                       const void* q, int32_t lq, const omnimem_select_params_t* p,
                                                       int32_t* idx, int32_t* cnt, float* score, int32_t* awe_active,
                                                       void* workspace, size_t workspace_bytes, void* stream) {
  CacheGeom g;
  SelectPlan plan;
  CmpCache c;
  const omnimem_status_t st = omnimem::check_select_compressed(kv, cc, q, lq, p, idx, cnt, workspace,
                                                               workspace_bytes, g, plan, c);
  if (st != OMNIMEM_OK) return st;
  if (awe_active) *awe_active = plan.awe;
  if (lq == 0) return OMNIMEM_OK;
  return hip_status(omnimem::launch_select_compressed(g, c, plan, q, idx, cnt, score, workspace, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_cmp_attn(const omnimem_cmp_cache_t* cc, int32_t n_chunks, const void* q,
                                              int32_t lq, float scale, void* out, float* lse, void* stream) {
  CacheGeom g;
  AttnLaunch a;
  const omnimem_status_t st = omnimem::check_cmp_attn(cc, n_chunks, q, lq, scale, out, lse, g, a);
  if (st != OMNIMEM_OK || lq == 0) return st;
  return hip_status(omnimem::launch_attention(g, a, as_stream(stream)));
}

OMNIMEM_API omnimem_status_t omnimem_gated_combine(int32_t dtype, int32_t lq, int32_t num_heads, int32_t head_dim,
                                                   const void* o_cmp, const void* o_slc, const void* o_swa,
                                                   const float* gate_logits, void* out, void* stream) {
  int64_t rows = 0;
  const omnimem_status_t st = omnimem::check_gated_combine(dtype, lq, num_heads, head_dim, o_cmp, o_slc, o_swa,
                                                           gate_logits, out, rows);
  if (st != OMNIMEM_OK || lq == 0) return st;
  return hip_status(omnimem::launch_gated_combine(dtype == OMNIMEM_BF16 ? 0 : 1, rows, head_dim, o_cmp, o_slc, o_swa,
                                                  gate_logits, out, as_stream(stream)));
}

OMNIMEM_API size_t omnimem_union_workspace_bytes(const omnimem_kv_cache_t* kv) {
  return omnimem::union_workspace_bytes(kv);
}

OMNIMEM_API omnimem_status_t omnimem_union_gather_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                                       const int32_t* idx, const int32_t* cnt, int32_t top_k,
                                                       int32_t group_size, float scale, void* out, float* lse,
                                                       int32_t* union_blocks, void* workspace,
                                                       size_t workspace_bytes, void* stream) {
  CacheGeom g;
  omnimem::UnionPlan up;
  AttnLaunch a;
  const omnimem_status_t st = omnimem::check_union_gather(kv, q, lq, idx, cnt, top_k, group_size, scale, out, lse,
                                                          union_blocks, workspace, workspace_bytes, g, up, a);
  if (st != OMNIMEM_OK || lq == 0) return st;
  return hip_status(omnimem::launch_union_gather(g, up, a, union_blocks, workspace, as_stream(stream)));
}

OMNIMEM_API const char* omnimem_status_string(int32_t status) { return omnimem::status_string(status); }
