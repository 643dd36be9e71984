// plan.cpp -- workspace plans of the selection and the union-gather comparator
// (host only).
#include "plan.h"

namespace omnimem {

SelectPlan plan_select(const CacheGeom& g, int lq, int K, int G, int E, float scale, int awe, int score_mode) {
  SelectPlan p{};
  p.score_mode = score_mode;
  p.lq = lq;
  p.G = G;
  p.R = (lq + G - 1) / G;
  p.K = K;
  p.awe = awe;
  p.first_excluded = awe ? (g.n - E) * g.Bpc : g.nb;
  p.scale = scale;
  const int rows = G < lq ? G : lq;
  p.qsplit = (rows + kQRowsPerSplit - 1) / kQRowsPerSplit;
  p.inline_scores = p.R <= kInlineGroups;
  size_t off = 0;
  p.off_qpart = off;
  off = align256(off + static_cast<size_t>(g.H) * p.R * p.qsplit * g.D * sizeof(float));
  p.off_kbar = off;
  if (!p.inline_scores) off = align256(off + static_cast<size_t>(g.H) * g.nb * g.D * sizeof(float));
  p.off_keys = off;
  off = align256(off + static_cast<size_t>(g.H) * p.R * ((g.nb + 3) / 4 * 4 + (g.nb == 0)) * sizeof(uint32_t));
  p.off_part = off;
  if (score_mode == 1) {
    constexpr int kSliceRows = kProbSliceRows;
    p.prob_multi = G <= kSliceRows / 2;
    if (p.prob_multi) {
      p.prob_gps = kSliceRows / G;
      p.prob_spg = 1;
      p.prob_slices = (p.R + p.prob_gps - 1) / p.prob_gps;
      p.prob_nseg = p.R;
    } else {
      p.prob_gps = 1;
      p.prob_spg = (rows + kSliceRows - 1) / kSliceRows;
      p.prob_slices = p.R * p.prob_spg;
      p.prob_nseg = p.prob_slices;
    }
    if (!p.prob_multi) off = align256(off + static_cast<size_t>(g.H) * p.prob_nseg * g.nb * sizeof(float));
    p.off_ksplit = off;
    off = align256(off + static_cast<size_t>(g.H) * ((g.nb + 63) / 64) * 2 * 64 * g.D * sizeof(uint16_t));
  }
  p.total = off;
  return p;
}

UnionPlan plan_union(const CacheGeom& g) {
  UnionPlan u{};
  const size_t eb = g.dtype == 0 ? 2 : 4;
  u.slab_bytes = static_cast<int64_t>(g.B) * g.D * eb;
  const size_t nb = g.nb > 0 ? g.nb : 1;
  size_t off = 0;
  u.off_flags = off;
  off = align256(off + nb * sizeof(int32_t));
  u.off_table = off;
  off = align256(off + nb * sizeof(int32_t));
  u.off_kbuf = off;
  off = align256(off + nb * g.H * static_cast<size_t>(u.slab_bytes));
  u.off_vbuf = off;
  off = align256(off + nb * g.H * static_cast<size_t>(u.slab_bytes));
  u.total = off;
  return u;
}

}  // namespace omnimem
