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
 * The compressed history (App. C's first cache level) pools each chunk once, when
 * it is appended (omnimem_compress_chunk); omnimem_select_compressed then scores
 * from the pooled keys instead of streaming all of K, and omnimem_cmp_attn is the
 * compression branch of Eq. 1 over the pooled keys and values.
 *
 * Conventions shared by every entry point
 *  - Every buffer pointer is a DEVICE pointer unless marked (host).  The caller
 *    allocates and owns every buffer, including workspaces; the library allocates
 *    no memory (except omnimem_lru_create's host bookkeeping object, released by
 *    omnimem_lru_destroy) and keeps no mutable global state, so calls on
 *    different streams may run concurrently on disjoint outputs.  The one
 *    exception is omnimem_select_noalloc, whose static per-GPU scratch is shared
 *    by all of its calls.
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
  OMNIMEM_EUNSUPPORTED = -2,/* a shape or dtype the library has no kernel for */
  OMNIMEM_EWORKSPACE = -3,  /* the workspace is smaller than the size query returns */
  OMNIMEM_EHIP = -4,        /* the HIP runtime reported an error at launch */
  OMNIMEM_ESCRATCH = -5     /* the problem needs more than omnimem_select_noalloc's static scratch */
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
 * page_table_head_stride: 0 = one table shared by every head.  Otherwise every
 *     head has a table of its own (App. C's pointer table is indexed by head and
 *     chunk): head h reads the [n][Bpc] table at page_table + h * stride, and the
 *     (page, h) slab holds its block, so a page may hold blocks of different
 *     chunks for different heads.  stride >= n*Bpc.  omnimem_union_gather_attn
 *     accepts shared tables only (OMNIMEM_EUNSUPPORTED otherwise).
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
  int64_t page_table_head_stride; /* 0 = shared by every head; else >= n*Bpc (per-head tables) */
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
 *  score_mode             what s[h][r][b] is (Sec. 3.1: the compression-attention
 *                         score, averaged over the group by Eq. 3):
 *                         OMNIMEM_SCORE_LOGIT (0, the default of a zeroed struct): the
 *                           group-mean logit, scale * <qbar[h][r], kbar[h][b]>;
 *                         OMNIMEM_SCORE_PROB (1): the group mean of each query's
 *                           softmax probability of block b over every pooled key
 *                           of the history (the compression branch's attention
 *                           weights).  omnimem_select_compressed only.
 */
enum { OMNIMEM_SCORE_LOGIT = 0, OMNIMEM_SCORE_PROB = 1 };

typedef struct {
  int32_t top_k;
  int32_t group_size;
  int32_t window_chunks;
  int32_t awe_min_outside_chunks;
  float scale;
  int32_t score_mode;
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

/* Bytes of device workspace omnimem_select (and omnimem_select_compressed) needs
   (0 on invalid arguments); kv->page_table may be NULL here. */
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
 * p->score_mode must be OMNIMEM_SCORE_LOGIT here (OMNIMEM_EINVAL otherwise).
 */
omnimem_status_t omnimem_select(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt, float* score,
                                int32_t* awe_active, void* workspace, size_t workspace_bytes, void* stream);

/*
 * omnimem_select without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same contract, outputs and bits as omnimem_select; the
 * scratch is a static device array of OMNIMEM_NOALLOC_SCRATCH_BYTES inside the
 * library, one per GPU, held until the process ends.  The call allocates nothing
 * and calls no allocating routine; the caller still passes q and the outputs.
 *  - Runs on the current device (hipSetDevice); `stream` must belong to it.
 *  - Returns OMNIMEM_ESCRATCH, launching nothing, when
 *    omnimem_select_workspace_bytes(kv, lq, p) exceeds the static size.
 *  - Every call on one GPU shares that GPU's array: calls that can overlap on one
 *    GPU (other streams, other host threads) race and must be serialised by the
 *    caller.  The array keeps the last call's contents; nothing read depends on them.
 */
#define OMNIMEM_NOALLOC_SCRATCH_BYTES (8u << 20)

omnimem_status_t omnimem_select_noalloc(const omnimem_kv_cache_t* kv, const void* q, int32_t lq,
                                        const omnimem_select_params_t* p, int32_t* idx, int32_t* cnt, float* score,
                                        int32_t* awe_active, void* stream);

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

/*
 * Compressed history of one layer (App. C: the compact first cache level; Sec. 3.1:
 * the compression branch pools with a plain mean, App. B).  Each block of each
 * appended chunk is pooled once into one pooled key and one pooled value, the
 * means over the block's valid tokens.  Pooled token t is history block t
 * (t = c*Bpc + o, Alg. 1's block numbering), so n chunks hold pooled tokens
 * [0, n*Bpc) in append order.
 *
 *   k_mean      [H][capacity_chunks*Bpc][d] float: the pooled keys in fp32, read by
 *               omnimem_select_compressed (the scores then equal omnimem_select's).
 *   k_pages,    [num_pages][H][64][d] of dtype: the pooled keys and values rounded
 *   v_pages     to dtype (bf16: to nearest even), 64 pooled tokens per page, page p
 *               holding tokens [64p, 64p + 64); read by omnimem_cmp_attn.
 *               num_pages >= ceil(capacity_chunks*Bpc / 64).
 *   page_table  [num_pages] int32: entry p = p, written by omnimem_compress_chunk
 *               for every page its chunk touches.
 *   k_lo        optional (NULL: absent), bf16 caches only: [num_pages][H][64][d] bf16,
 *               the rounding residual of the pooled keys, bf16(k_mean - k_pages), in
 *               k_pages' layout; written by omnimem_compress_chunk when present.  With
 *               it, the probability-averaged scores of omnimem_select_compressed read
 *               the fp32 pooled keys as the two bf16 pieces k_pages + k_lo instead of
 *               splitting k_mean on every call (the results are the same bit for bit).
 *               Every chunk must then have been pooled with k_lo present.
 * The caller allocates and owns every buffer (16-byte aligned; page_table 4-byte).
 * Geometry (dtype, H, d, B, S) must equal the full cache's.
 */
typedef struct {
  omnimem_dtype_t dtype;        /* of k_pages and v_pages: the full cache's dtype */
  int32_t num_heads, head_dim;  /* H, d */
  int32_t block_size;           /* B of the full cache: one pooled token per block */
  int32_t chunk_tokens;         /* S of the full cache: Bpc = ceil(S/B) pooled tokens per chunk */
  int32_t capacity_chunks;      /* chunks the buffers hold */
  float* k_mean;
  void* k_pages;
  void* v_pages;
  int32_t* page_table;
  int64_t num_pages;            /* pages of k_pages / v_pages (and k_lo) */
  void* k_lo;                   /* optional residual of the pooled keys (bf16 caches) */
} omnimem_cmp_cache_t;

/*
 * Pools history chunk `chunk` (0 <= chunk < kv->num_chunks, < capacity_chunks) of
 * the full cache into the compressed cache (App. C: each generated chunk's KV is
 * pooled once and appended).  For each block b = chunk*Bpc + o and head h:
 *   k_mean[h][b] = (1/|b|) sum over the block's valid tokens of K   (fp32)
 *   pooled token b of k_pages / v_pages = the means of K / V rounded to dtype.
 * A block whose page is not resident (page id < 0 or >= kv->num_pages) pools to 0.
 * Re-pooling a chunk overwrites it with the same values.
 */
omnimem_status_t omnimem_compress_chunk(const omnimem_kv_cache_t* kv, int32_t chunk, const omnimem_cmp_cache_t* cc,
                                        void* stream);

/*
 * omnimem_select over the compressed history: the same contract, arguments and
 * outputs, with the pooled keys read from cc->k_mean (chunks [0, kv->num_chunks)
 * must have been pooled; kv->num_chunks <= capacity_chunks) instead of pooled from
 * the full cache's pages.  kv still supplies the geometry, the history length and
 * residency (a block whose page is not resident is not a candidate); with
 * kv->page_table == NULL every block is a candidate, residency being handled by
 * the caller (omnimem_lru_require before the selection attention).  The workspace
 * is sized by omnimem_select_workspace_bytes(kv, lq, p).
 *
 * With p->score_mode == OMNIMEM_SCORE_PROB the scores are
 *   u[h][i][b]  = scale * <q_i, kbar[h][b]>                 for all n*Bpc pooled keys
 *   s[h][r][b]  = (1/|G_r|) sum over rows i of group r of exp(u[h][i][b] - LSE[h][i]),
 *                 LSE[h][i] = ln sum over all b of exp(u[h][i][b])
 * (the softmax includes the window and non-resident blocks; Omega restricts only
 * the top-K), and `score` returns these group-mean probabilities.  The products
 * run on bf16 MFMA with fp32 accumulation, kbar split into two bf16 pieces (and
 * fp32 queries too), which keeps the logits to about 2^-16 relative of fp32.
 */
omnimem_status_t omnimem_select_compressed(const omnimem_kv_cache_t* kv, const omnimem_cmp_cache_t* cc,
                                           const void* q, int32_t lq, const omnimem_select_params_t* p,
                                           int32_t* idx, int32_t* cnt, float* score, int32_t* awe_active,
                                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * Compression attention, the CMP branch of Eq. 1 (Sec. 3.1, App. C): every query
 * attends to the n_chunks*Bpc pooled tokens of the compressed history,
 *   O[i][h]   = sum_t softmax_t(scale * <q_i, kc_t>) vc_t
 *   lse[h][i] = ln sum_t exp(scale * <q_i, kc_t>)
 * with kc, vc the pooled keys and values as stored in k_pages / v_pages.
 * 0 <= n_chunks <= capacity_chunks; n_chunks = 0 gives O = 0 and lse = -inf.
 * q, out, lse and the arithmetic are as in omnimem_dense_attn.
 */
omnimem_status_t omnimem_cmp_attn(const omnimem_cmp_cache_t* cc, int32_t n_chunks, const void* q, int32_t lq,
                                  float scale, void* out, float* lse, void* stream);

/*
 * Eq. 1's fusion of the three branches (Sec. 3.1): for every query row i and head h
 *   out[i][h] = sum over c in (CMP, SLC, SWA) of g^c[i][h] * o_c[i][h],
 *   g^c[i][h] = 1 / (1 + exp(-gate_logits[i][h][c]))  in [0, 1]
 * (App. B: learned per-branch sigmoid gates; the logits are the caller's).
 * o_cmp, o_slc, o_swa: [lq][num_heads][head_dim] of dtype (omnimem_cmp_attn,
 * omnimem_sparse_attn and omnimem_dense_attn over the window give them); a NULL
 * branch is absent and contributes nothing (at least one must be given).
 * gate_logits: [lq][num_heads][3] float, branch order CMP, SLC, SWA.
 * out: [lq][num_heads][head_dim] of dtype; it may be one of the branch buffers.
 * Arithmetic in fp32, the result rounded to dtype (bf16: nearest even).
 */
omnimem_status_t omnimem_gated_combine(int32_t dtype, int32_t lq, int32_t num_heads, int32_t head_dim,
                                       const void* o_cmp, const void* o_slc, const void* o_swa,
                                       const float* gate_logits, void* out, void* stream);

/*
 * Alg. 1 Step 1's chunk decode, on the device: for every head h and history
 * chunk c < n,
 *   needed[h][c] = 1 if some group r < groups lists, among its first cnt[h][r]
 *                  entries of idx[h][r][0 : top_k], a block b in [0, N_b) with
 *                  b div Bpc = c; else 0.
 * idx [H][groups][top_k] and cnt [H][groups] int32 as omnimem_select writes them;
 * needed [H][n] uint8 (out).  H, n and Bpc come from kv; its pages and page
 * table are not read (the table may be NULL).  The result is the request of
 * omnimem_lru_require once copied to the host.
 */
omnimem_status_t omnimem_selected_chunks(const omnimem_kv_cache_t* kv, const int32_t* idx, const int32_t* cnt,
                                         int32_t groups, int32_t top_k, uint8_t* needed, void* stream);

/*
 * GPU hot cache of full-resolution history chunks with LRU eviction (App. B,
 * "Inference and Offloading": the GPU keeps a few chunks, the rest sit in pinned
 * host memory and are reloaded over PCIe when selected; App. F studies the cache's
 * size; Alg. 1 waits for a selected chunk's reload before reading it).  Host-side
 * runtime state for one layer.
 *
 * Residency is per (head, chunk), like Alg. 1's pointer table: every head has
 * `slots` chunk slots and its own least-recently-used order.  The caller
 * allocates and owns every buffer:
 *   kv->k_pages, v_pages   the GPU pool, kv->num_pages >= slots*Bpc: slot s of
 *                          head h is the head-h slabs of pages [s*Bpc, (s+1)*Bpc);
 *   kv->page_table         per-head tables (kv->page_table_head_stride >= n*Bpc,
 *                          n = kv->num_chunks >= 1), written by this runtime only:
 *                          head h's row of chunk c holds the slot's pages while the
 *                          pair is resident and -1 (not resident) otherwise;
 *   k_host, v_host         pinned host pools (hipHostMalloc) of host_chunks >= n
 *                          chunks: chunk c in pages [c*Bpc, (c+1)*Bpc), the page
 *                          layout of kv ([page][H][B][d]).
 * The object keeps host bookkeeping and two HIP events (no device or pinned memory
 * of its own); it is not thread-safe.  Selection over the compressed history
 * (omnimem_select_compressed with kv->page_table == NULL) needs nothing resident.
 */
typedef struct omnimem_lru omnimem_lru_t;

typedef struct {
  int64_t hits, misses, evictions; /* (head, chunk) pairs found resident / reloaded / evicted */
  int64_t bytes_reloaded;          /* host-to-device bytes (K and V) */
} omnimem_lru_stats_t;

/* Creates the state (*out, released by omnimem_lru_destroy) and enqueues on
   `stream` the write of -1 to every row of every head's table.  slots >= 1. */
omnimem_status_t omnimem_lru_create(const omnimem_kv_cache_t* kv, int32_t slots, const void* k_host,
                                    const void* v_host, int32_t host_chunks, void* stream, omnimem_lru_t** out);
void omnimem_lru_destroy(omnimem_lru_t* lru);

/*
 * Makes resident every (head, chunk) pair with needed[h*n + c] != 0 (host array
 * [H][n], n <= kv->num_chunks; omnimem_selected_chunks computes it).  Per head, in
 * ascending chunk order: resident pairs are hits and become most recently used;
 * every other pair takes the head's lowest free slot, else the slot of its least
 * recently used chunk that the request does not name, and becomes most recently
 * used; the evicted pair's row becomes -1.
 * Reloads and row writes are enqueued on copy_stream, after all work already
 * enqueued on compute_stream (which may still read the slots being reused); the
 * two may be the same stream.  Nothing on another stream may read the rows of the
 * evicted chunks meanwhile.  omnimem_lru_wait orders later work after the reloads.
 * A head that names more chunks than it has slots: OMNIMEM_EINVAL, nothing changed.
 * *reloaded (host, may be NULL): the number of pairs reloaded.
 * OMNIMEM_EHIP leaves the runtime unusable (every later call returns it).
 */
omnimem_status_t omnimem_lru_require(omnimem_lru_t* lru, const uint8_t* needed, int32_t n, void* compute_stream,
                                     void* copy_stream, int32_t* reloaded);

/* Makes `stream` wait until the reloads of the last omnimem_lru_require have
   landed (Alg. 1's WaitUntilReload); no-op if nothing was ever reloaded. */
omnimem_status_t omnimem_lru_wait(omnimem_lru_t* lru, void* stream);

/* Counters since creation (host). */
omnimem_status_t omnimem_lru_stats(const omnimem_lru_t* lru, omnimem_lru_stats_t* out);

/* The slot holding chunk `chunk` of head `head`, or -1 when not resident (host). */
int32_t omnimem_lru_slot_of(const omnimem_lru_t* lru, int32_t head, int32_t chunk);

/*
 * Binds the calling thread to the NUMA node of GPU `device`'s PCI function (App. B
 * binds generation to the node that owns the GPU's PCIe root): its CPU affinity
 * becomes that node's CPUs among those it may already use, and its memory policy
 * prefers the node, so pinned host pools it allocates afterwards sit next to the
 * GPU.  Threads it starts later inherit both.  *node (host, may be NULL): the node
 * bound, or -1 when the system reports none or the node shares no CPU with the
 * thread's affinity (nothing is changed then).  OMNIMEM_EINVAL on an unknown
 * device or a failed system call.
 */
omnimem_status_t omnimem_numa_bind(int32_t device, int32_t* node);

#ifdef __cplusplus
}
#endif

#endif /* OMNIMEM_H */
