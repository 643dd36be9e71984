/*
 * omnimem.h -- C ABI of libomnimem.so: OmniMem's memory-retrieval attention step
 * (arXiv 2605.30519) on AMD Instinct MI355X (gfx950).
 *
 * One autoregressive step of a chunk-based video DiT: the Lq queries of the chunk
 * being generated attend to a growing history of n cached chunks (App. A).  The
 * step has two stages:
 *   1. omnimem_select: query-shared top-K block selection over the whole history
 *      with Adaptive Window Exclusion (Sec. 3.2 Eq. 2; Sec. 3.3 Eq. 3);
 *   2. omnimem_sparse_attn: per-head scattered block-sparse attention that reads
 *      each head's own selected blocks straight from the paged cache (Sec. 3.3
 *      Eq. 5; App. C, Alg. 1 Step 2).
 * omnimem_dense_attn is dense attention over a contiguous chunk range: the whole
 * history (the full-attention reference of Sec. 4.3) or the sliding window (App. C).
 * omnimem_union_gather_attn is the naive comparator of Sec. 3.3 that materialises
 * the cross-head union of selected blocks in a head-aligned buffer first.
 *
 * Conventions shared by every entry point
 *  - Every buffer pointer is a DEVICE pointer unless marked (host).  The caller
 *    allocates and owns every buffer, including workspaces; the library allocates
 *    no memory and keeps no mutable global state, so calls on different streams
 *    may run concurrently on disjoint outputs.
 *  - All work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *    is asynchronous: no entry point synchronises with the host.
 *  - Arguments are validated on the host before anything is enqueued; on failure
 *    a negative status is returned and nothing is launched.  Device-resident
 *    contents (page-table entries, block ids) are not readable by the host: the
 *    kernels treat an out-of-range page id or block id like a non-resident block
 *    or a padding entry and skip it, so a bad table never causes an
 *    out-of-bounds access.  A failed launch returns OMNIMEM_EHIP.
 *  - Outputs are deterministic: identical inputs give bitwise identical outputs.
 *  - Device pointers to tensors read or written with vector accesses (Q, the
 *    page pools, O) must be 16-byte aligned.
 */
#ifndef OMNIMEM_H
#define OMNIMEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of Q, K, V and O. */
typedef enum { OMNIMEM_BF16 = 0, OMNIMEM_F32 = 1 } omnimem_dtype_t;

typedef enum {
  OMNIMEM_OK = 0,
  OMNIMEM_EINVAL = -1,      /* a null, misaligned or out-of-range argument */
  OMNIMEM_EUNSUPPORTED = -2,/* a shape or dtype this build has no kernel for */
  OMNIMEM_EWORKSPACE = -3,  /* the workspace is smaller than the size query returns */
  OMNIMEM_EHIP = -4         /* the HIP runtime reported an error at launch */
} omnimem_status_t;

/*
 * Paged full-resolution KV cache of one attention layer (App. C: the chunk-level
 * cache shared by the selection and sliding-window branches, with its pointer
 * table re-expressed as a page table).
 *
 * Geometry: H = num_heads, d = head_dim, B = block_size tokens per KV block,
 * S = chunk_tokens, Bpc = ceil(S/B) blocks per chunk, n = num_chunks cached
 * history chunks (the chunk being generated is NOT in the cache).  Blocks are
 * chunk-aligned: block b covers tokens [o*B, min((o+1)*B, S)) of chunk c, with
 * c = b div Bpc and o = b mod Bpc (Alg. 1, Step 1); N_b = n*Bpc.
 *
 * k_pages, v_pages: [num_pages][H][B][d] elements of `dtype`.  A page holds one
 *     block of every head; the (page, head) slab of B*d elements is contiguous.
 *     Slots past the last token of a chunk's final block are never read into a
 *     result (their contents do not matter, NaN included).
 * page_table: [n][Bpc] int32 page ids.  A negative id marks a block that is not
 *     resident on the GPU: it is never selected and never attended (the pointer
 *     table's 0 entry of App. C).  Ids >= num_pages are treated the same way.
 */
typedef struct {
  int32_t dtype;        /* omnimem_dtype_t */
  int32_t num_heads;    /* H >= 1 */
  int32_t head_dim;     /* d in {64, 128} */
  int32_t block_size;   /* B in {64, 128} */
  int32_t chunk_tokens; /* S >= 1 */
  int32_t num_chunks;   /* n >= 0 */
  int64_t num_pages;    /* capacity of k_pages / v_pages, in pages */
  const void* k_pages;
  const void* v_pages;
  const int32_t* page_table;
} omnimem_kv_cache_t;

/*
 * Selection parameters (Sec. 3.2-3.3; App. B "Memory Module").
 *  top_k                  K >= 1: blocks selected per (head, query group).
 *  group_size             G_q >= 1: adjacent queries sharing one selection;
 *                         R = ceil(Lq/G_q) groups, group r = rows [r*G_q, min((r+1)*G_q, Lq)).
 *  window_chunks          E >= 0: the most recent E chunks form the excluded window W.
 *  awe_min_outside_chunks T_out >= 0: exclusion is applied only once at least
 *                         T_out whole chunks lie outside the window, and (Eq. 2's
 *                         guard) at least K blocks do.
 *  scale                  score scale sigma > 0 (1/sqrt(d) in the workloads).
 */
typedef struct {
  int32_t top_k;
  int32_t group_size;
  int32_t window_chunks;
  int32_t awe_min_outside_chunks;
  float scale;
} omnimem_select_params_t;

/* Blocks per chunk, ceil(S/B); -1 if S < 1 or B < 1.  Host only, pure. */
int32_t omnimem_blocks_per_chunk(int32_t chunk_tokens, int32_t block_size);

/*
 * Adaptive Window Exclusion state for a history of n chunks (Eq. 2 with the
 * activation rule of App. B): 1 when (n - E >= T_out) and ((n - E) * Bpc >= K),
 * else 0; -1 on invalid arguments (n < 0, E < 0, T_out < 0, K < 1, Bpc < 1).
 * Host only, pure integer logic.
 */
int32_t omnimem_awe_active(int32_t num_chunks, int32_t window_chunks, int32_t awe_min_outside_chunks, int32_t top_k,
                           int32_t blocks_per_chunk);

/* Bytes of device workspace omnimem_select needs (0 on invalid arguments). */
size_t omnimem_select_workspace_bytes(const omnimem_kv_cache_t* kv, int32_t lq, const omnimem_select_params_t* p);

/*
 * Query-shared block selection with Adaptive Window Exclusion (Eq. 2, Eq. 3).
 *
 * For every head h and query group r:
 *   kbar[h][b]  = mean over the tokens of block b of K          (compression pooling, App. B)
 *   qbar[h][r]  = mean over the rows of group r of Q            (proxy query; Eq. 3 by linearity)
 *   s[h][r][b]  = scale * <qbar[h][r], kbar[h][b]>
 *   Omega       = resident blocks, minus the window blocks of the last E chunks when exclusion is active
 *   I[h][r]     = the min(K, |Omega|) blocks of Omega with the highest s; equal scores rank the lower id first
 *
 * q:     [lq][H][d] of kv->dtype, lq >= 0 (lq = 0 does nothing).
 * idx:   [H][R][K] int32 (out): I[h][r] in ascending block-id order, padded with -1.
 * cnt:   [H][R] int32 (out): |I[h][r]|.
 * score: [H][R][K] float (out, may be NULL): s of each listed block; -inf at padding.
 * awe_active: (host, out, may be NULL) the exclusion state used.
 * workspace: device scratch of at least omnimem_select_workspace_bytes(), 256-byte aligned.
 * Accumulation is fp32 on exact inputs; ranking is on fp32 scores.
 */
omnimem_status_t omnimem_select(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt, float* score,
                                int32_t* awe_active, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Per-head scattered block-sparse attention (Sec. 3.3 Eq. 5; Alg. 1 Step 2).
 *
 * Query row i (group r = i div group_size) of head h attends to the tokens of the
 * blocks idx[h][r][0 : cnt[h][r]], read in place from the paged cache, in list
 * order (a block listed twice is attended twice).  Entries < 0 or >= N_b, and
 * blocks whose page is not resident, are skipped.
 *   O[i][h]   = sum_j softmax_j(scale * <q_i, k_j>) v_j
 *   lse[h][i] = ln sum_j exp(scale * <q_i, k_j>)
 * An empty key set gives O = 0 and lse = -inf.
 *
 * q:   [lq][H][d]; idx: [H][R][top_k] int32; cnt: [H][R] int32 with R = ceil(lq/group_size).
 * out: [lq][H][d] of kv->dtype (out).  lse: [H][lq] float (out, may be NULL).
 * bf16: QK^T and PV on bf16 MFMA with fp32 accumulation and an fp32 online
 * softmax; P is rounded to bf16 before PV.  f32: fp32 arithmetic throughout.
 */
omnimem_status_t omnimem_sparse_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, const int32_t* idx,
                                     const int32_t* cnt, int32_t top_k, int32_t group_size, float scale, void* out,
                                     float* lse, void* stream);

/*
 * Dense attention of every query over all resident tokens of history chunks
 * [chunk_begin, chunk_end), 0 <= chunk_begin <= chunk_end <= n: [0, n) is
 * full-history attention (the baseline of Sec. 4.3), [n-W, n) the
 * sliding-window branch (App. C).  Same outputs and arithmetic as
 * omnimem_sparse_attn.
 */
omnimem_status_t omnimem_dense_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq, int32_t chunk_begin,
                                    int32_t chunk_end, float scale, void* out, float* lse, void* stream);

/* Bytes of device workspace omnimem_union_gather_attn needs (0 on invalid arguments). */
size_t omnimem_union_workspace_bytes(const omnimem_kv_cache_t* kv);

/*
 * Comparator: union-gather-then-attend (the head-aligned selected-KV buffer of
 * Sec. 3.3, footprint proportional to H * |U|, U = union over h and r of I[h][r]).
 * Marks U, gathers every block of U for every head into a compact buffer inside
 * the workspace, and runs the attention of omnimem_sparse_attn on that buffer.
 * Results equal omnimem_sparse_attn's bit for bit.
 * union_blocks: device int32 scalar (out): |U|.
 */
omnimem_status_t omnimem_union_gather_attn(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                           const int32_t* idx, const int32_t* cnt, int32_t top_k, int32_t group_size,
                                           float scale, void* out, float* lse, int32_t* union_blocks,
                                           void* workspace, size_t workspace_bytes, void* stream);

/* Static, human-readable text for a status code. */
const char* omnimem_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* OMNIMEM_H */
