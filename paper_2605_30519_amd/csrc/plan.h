// plan.h -- host-side geometry and work plans of the libomnimem entry points
// (internal to the library).  No HIP here: this header and plan.cpp /
// validate.cpp build with the host compiler alone, so the argument checks and
// the workspace arithmetic can also be run on a CPU under sanitizers.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace omnimem {

// Geometry of one paged layer cache, resolved and validated on the host.
struct CacheGeom {
  int dtype;          // 0 = bf16, 1 = f32
  int H, D, B, S;     // heads, head dim, tokens per block, tokens per chunk
  int n;              // cached history chunks
  int Bpc;            // blocks per chunk = ceil(S/B)
  int nb;             // history blocks = n * Bpc
  int64_t num_pages;
  const void* k_pages;
  const void* v_pages;
  const int32_t* page_table;
  int64_t pt_stride;  // 0: one table shared by every head; else head h's table starts at h * pt_stride
};

// ---------------------------------------------------------------- selection
struct SelectPlan {
  int lq, G, R, K;
  int awe;              // exclusion active
  int first_excluded;   // blocks >= this id are outside Omega (nb when exclusion is off)
  float scale;
  int qsplit;           // row splits per group in the proxy-query reduction
  bool inline_scores;   // scores computed inside the pooling kernel (small R)
  // probability-averaged scores (score_mode 1): query slices of at most 128 rows,
  // either whole groups (multi: gps groups per slice) or parts of one group (spg
  // slices per group); for parts, one partial row of nb sums per (head, slice);
  // the pooled keys split into bf16 pieces, 64-key tiles
  int score_mode;
  bool prob_multi;
  int prob_gps, prob_spg, prob_slices, prob_nseg;
  // workspace carve-up (byte offsets)
  size_t off_qpart, off_kbar, off_keys, off_part, off_ksplit, total;
};

constexpr int kQRowsPerSplit = 512;
constexpr int kProbSliceRows = 128;  // query rows per workgroup of the probability scores
constexpr int kInlineGroups = 4;

SelectPlan plan_select(const CacheGeom& g, int lq, int K, int G, int E, float scale, int awe, int score_mode = 0);

// ---------------------------------------------------------------- compressed history
// One pooled key/value per history block, in block order (token t = block t).
struct CmpCache {
  float* k_mean;         // [H][cap_blocks][D] fp32 pooled keys
  void* k_pages;         // [num_pages][H][64][D] pooled keys in the cache dtype
  void* v_pages;         // same, pooled values
  int32_t* page_table;   // [num_pages], entry p = p
  int64_t num_pages;
  int cap_blocks;        // capacity in pooled tokens
  void* k_lo;            // optional [num_pages][H][64][D] bf16 residual of the pooled keys
};
constexpr int kCmpPageTokens = 64;

// ---------------------------------------------------------------- attention
struct AttnLaunch {
  const void* q;
  void* out;
  float* lse;
  int lq;
  int group_size, R;
  // sparse mode: per-(h, r) lists; dense mode: idx == nullptr, contiguous block range
  const int32_t* idx;
  const int32_t* cnt;
  int top_k;
  int dense_first_block, dense_num_blocks;
  float scale;
};

// ---------------------------------------------------------------- union gather
struct UnionPlan {
  size_t off_flags, off_table, off_kbuf, off_vbuf, total;
  int64_t slab_bytes;  // one (page, head) slab
};

UnionPlan plan_union(const CacheGeom& g);

inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace omnimem
