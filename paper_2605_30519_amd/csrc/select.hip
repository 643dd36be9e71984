// select.hip -- query-shared block selection with Adaptive Window Exclusion
// (Sec. 3.2 Eq. 2, Sec. 3.3 Eq. 3) for gfx950.
//
// Pipeline (one stream, no host round trip):
//   k_qmean_partial  Q rows -> fp32 partial column sums per (head, group, row split)
//   k_qmean_final    partial sums -> proxy queries qbar[h][r][:] (group means)
//   k_pool_score     streams every candidate K block once: block mean over its valid
//                    tokens, then s[h][r][b] = scale * <qbar[h][r], kbar[h][b]>
//                    (for many groups it writes kbar and k_score does the products)
//   k_topk           per (head, group): exact top-K over Omega by an MSB-first
//                    radix select on order-preserving 32-bit score keys in LDS,
//                    ties to the lower block id, ids written in ascending order.
// The dominant cost is the K stream in k_pool_score, which is HBM-bound: each wave
// owns whole (page, head) slabs (B*d contiguous elements) and reads them with
// 16-byte loads, all lanes of a wave in flight on one slab at a time.
#include <float.h>
#include <math.h>

#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

constexpr int kThreads = 256;

// -------------------------------------------------------------- proxy queries
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void k_qmean_partial(const T* __restrict__ q, int lq, int H, int G, int R,
                                                            int nsplit, float* __restrict__ partial) {
  using V = Vec16<T>;
  constexpr int VEC = V::N;
  constexpr int CPR = D / VEC;            // 16-byte chunks per row
  constexpr int PHASES = kThreads / CPR;  // rows summed side by side
  __shared__ float red[PHASES][D];

  const int s = blockIdx.x, r = blockIdx.y, h = blockIdx.z;
  const int g0 = r * G, g1 = min(g0 + G, lq);
  const int r0 = g0 + s * kQRowsPerSplit, r1 = min(r0 + kQRowsPerSplit, g1);
  const int c = threadIdx.x % CPR, ph = threadIdx.x / CPR;

  float acc[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
  for (int row = r0 + ph; row < r1; row += PHASES) {
    float x[VEC];
    V::load(q + (static_cast<int64_t>(row) * H + h) * D + c * VEC, x);
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] += x[j];
  }
#pragma unroll
  for (int j = 0; j < VEC; ++j) red[ph][c * VEC + j] = acc[j];
  __syncthreads();
  for (int col = threadIdx.x; col < D; col += kThreads) {
    float sum = 0.f;
    for (int p = 0; p < PHASES; ++p) sum += red[p][col];
    partial[((static_cast<int64_t>(h) * R + r) * nsplit + s) * D + col] = sum;
  }
}

template <int D>
__global__ __launch_bounds__(D) void k_qmean_final(const float* __restrict__ partial, int lq, int G, int R, int nsplit,
                                                   float* __restrict__ qbar) {
  const int r = blockIdx.x, h = blockIdx.y, col = threadIdx.x;
  const int g0 = r * G, rows = min(g0 + G, lq) - g0;
  const int used = (rows + kQRowsPerSplit - 1) / kQRowsPerSplit;
  const float* p = partial + (static_cast<int64_t>(h) * R + r) * nsplit * D + col;
  float sum = 0.f;
  for (int s = 0; s < used; ++s) sum += p[static_cast<int64_t>(s) * D];
  qbar[(static_cast<int64_t>(h) * R + r) * D + col] = sum / static_cast<float>(rows);
}

// -------------------------------------------------------------- pooling + scores
// One wave per (page, head) slab.  Lane layout inside a slab: lane = ph * CPR + c,
// c = 16-byte column chunk, ph = row phase; the wave covers 64/CPR rows per pass.
template <typename T, int D, int B>
struct SlabShape {
  static constexpr int VEC = Vec16<T>::N;
  static constexpr int CPR = D / VEC;
  static constexpr int ROWS_PER_PASS = kWave / CPR;
  static constexpr int PASSES = B / ROWS_PER_PASS;
};

template <typename T, int D, int B>
__device__ __forceinline__ void pool_slab(const T* __restrict__ slab, int nvalid, int lane,
                                          float (&colsum)[Vec16<T>::N]) {
  using Sh = SlabShape<T, D, B>;
  const int c = lane % Sh::CPR, ph = lane / Sh::CPR;
  // issue every 16-byte load of the slab first (raw words, no widening yet)
  uint4 raw[Sh::PASSES];
#pragma unroll
  for (int i = 0; i < Sh::PASSES; ++i) {
    const int row = ph + i * Sh::ROWS_PER_PASS;
    raw[i] = row < nvalid ? *reinterpret_cast<const uint4*>(slab + row * D + c * Sh::VEC) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int j = 0; j < Sh::VEC; ++j) colsum[j] = 0.f;
#pragma unroll
  for (int i = 0; i < Sh::PASSES; ++i) {
    float x[Sh::VEC];
    Vec16<T>::widen(raw[i], x);
#pragma unroll
    for (int j = 0; j < Sh::VEC; ++j) colsum[j] += x[j];
  }
  // sum the row phases: lanes c, c+CPR, c+2*CPR, ...
#pragma unroll
  for (int m = Sh::CPR; m < kWave; m <<= 1)
#pragma unroll
    for (int j = 0; j < Sh::VEC; ++j) colsum[j] += __shfl_xor(colsum[j], m);
}

struct PoolArgs {
  const void* k_pages;
  const int32_t* page_table;
  int64_t num_pages;
  int H, S, Bpc, nb, first_excluded;
  const float* qbar;  // [H][R][D]
  int R;
  float scale;
  float* scores;  // [H][R][nb] (inline mode)
  float* kbar;    // [H][nb][D] (kbar mode)
  int blocks_per_wave;
};

__device__ __forceinline__ bool block_page(const PoolArgs& a, int b, int64_t& page) {
  if (b >= a.first_excluded) return false;
  const int32_t p = a.page_table[b];
  if (p < 0 || p >= a.num_pages) return false;
  page = p;
  return true;
}

template <typename T, int D, int B, bool INLINE>
__global__ __launch_bounds__(kThreads) void k_pool_score(PoolArgs a) {
  using Sh = SlabShape<T, D, B>;
  constexpr int VEC = Sh::VEC;
  const int h = blockIdx.y;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int c = lane % Sh::CPR;
  const int first = (blockIdx.x * (kThreads / kWave) + wave) * a.blocks_per_wave;
  const int last = min(first + a.blocks_per_wave, a.nb);
  const T* pages = static_cast<const T*>(a.k_pages);

  float q[INLINE ? kInlineGroups : 1][VEC];
  if (INLINE) {
#pragma unroll
    for (int r = 0; r < kInlineGroups; ++r)
#pragma unroll
      for (int j = 0; j < VEC; ++j)
        q[r][j] = r < a.R ? a.qbar[(static_cast<int64_t>(h) * a.R + r) * D + c * VEC + j] : 0.f;
  }

  for (int b = first; b < last; ++b) {
    int64_t page;
    const bool live = block_page(a, b, page);
    if (!live) {
      if (INLINE) {
        if (lane < a.R) a.scores[(static_cast<int64_t>(h) * a.R + lane) * a.nb + b] = -INFINITY;
      }
      continue;
    }
    const int o = b % a.Bpc;
    const int nvalid = o == a.Bpc - 1 ? a.S - o * B : B;
    const T* slab = pages + (page * a.H + h) * static_cast<int64_t>(B) * D;
    float colsum[VEC];
    pool_slab<T, D, B>(slab, nvalid, lane, colsum);
    const float inv = 1.0f / static_cast<float>(nvalid);
    if (INLINE) {
#pragma unroll
      for (int r = 0; r < kInlineGroups; ++r) {
        if (r >= a.R) break;
        float dot = 0.f;
#pragma unroll
        for (int j = 0; j < VEC; ++j) dot += q[r][j] * (colsum[j] * inv);
#pragma unroll
        for (int m = 1; m < Sh::CPR; m <<= 1) dot += __shfl_xor(dot, m);
        if (lane == 0) a.scores[(static_cast<int64_t>(h) * a.R + r) * a.nb + b] = a.scale * dot;
      }
    } else {
      if (lane < Sh::CPR) {
        float* dst = a.kbar + (static_cast<int64_t>(h) * a.nb + b) * D + c * VEC;
#pragma unroll
        for (int j = 0; j < VEC; ++j) dst[j] = colsum[j] * inv;
      }
    }
  }
}

// scores for many groups: tile of 64 blocks x 16 groups per workgroup
template <int D>
__global__ __launch_bounds__(kThreads) void k_score(const float* __restrict__ kbar, const float* __restrict__ qbar,
                                                    const int32_t* __restrict__ page_table, int64_t num_pages,
                                                    int nb, int first_excluded, int R, float scale,
                                                    float* __restrict__ scores) {
  constexpr int TB = 64, TR = 16;
  __shared__ float ks[TB][D + 1];
  __shared__ float qs[TR][D + 1];
  const int b0 = blockIdx.x * TB, r0 = blockIdx.y * TR, h = blockIdx.z;
  for (int i = threadIdx.x; i < TB * D; i += kThreads) {
    const int bb = i / D, j = i % D;
    ks[bb][j] = b0 + bb < nb ? kbar[(static_cast<int64_t>(h) * nb + b0 + bb) * D + j] : 0.f;
  }
  for (int i = threadIdx.x; i < TR * D; i += kThreads) {
    const int rr = i / D, j = i % D;
    qs[rr][j] = r0 + rr < R ? qbar[(static_cast<int64_t>(h) * R + r0 + rr) * D + j] : 0.f;
  }
  __syncthreads();
  for (int t = threadIdx.x; t < TB * TR; t += kThreads) {
    const int bb = t % TB, rr = t / TB;
    const int b = b0 + bb, r = r0 + rr;
    if (b >= nb || r >= R) continue;
    float dot = 0.f;
    for (int j = 0; j < D; ++j) dot += qs[rr][j] * ks[bb][j];
    const int32_t p = page_table[b];
    const bool live = b < first_excluded && p >= 0 && p < num_pages;
    scores[(static_cast<int64_t>(h) * R + r) * nb + b] = live ? scale * dot : -INFINITY;
  }
}

// -------------------------------------------------------------- top-K
// Order-preserving map of an fp32 score to uint32 (larger score -> larger key).
// -0 is folded onto +0 first so that equal scores compare equal.  Candidate keys
// are forced >= 1 so that 0 can mark "not a candidate".
__device__ __forceinline__ uint32_t score_key(float s) {
  s = s + 0.0f;
  const uint32_t u = __float_as_uint(s);
  const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return k == 0u ? 1u : k;
}

constexpr int kTopkLdsMax = 12288;  // candidates staged in LDS (48 KB) up to this many blocks

template <bool IN_LDS>
__global__ __launch_bounds__(kThreads) void k_topk(const float* __restrict__ scores,
                                                   const int32_t* __restrict__ page_table, int64_t num_pages, int nb,
                                                   int first_excluded, int R, int K, int32_t* __restrict__ idx,
                                                   int32_t* __restrict__ cnt, float* __restrict__ score_out) {
  extern __shared__ uint32_t keys[];  // [nb] when IN_LDS
  __shared__ int hist[256];
  __shared__ int scan_tmp[kThreads / kWave];
  __shared__ int pick[2];

  const int r = blockIdx.x, h = blockIdx.y;
  const int64_t row = static_cast<int64_t>(h) * R + r;
  const float* s = scores + row * nb;

  auto key_of = [&](int b) -> uint32_t {
    const int32_t p = page_table[b];
    const bool cand = b < first_excluded && p >= 0 && p < num_pages;
    return cand ? score_key(s[b]) : 0u;
  };
  auto key_at = [&](int b) -> uint32_t { return IN_LDS ? keys[b] : key_of(b); };

  int mine = 0;
  for (int b = threadIdx.x; b < nb; b += kThreads) {
    const uint32_t k = key_of(b);
    if (IN_LDS) keys[b] = k;
    mine += k != 0u;
  }
  int ncand;
  block_exclusive_scan<kThreads>(mine, scan_tmp, ncand);  // also a barrier for `keys`

  // Radix select of the K-th largest key: after the four 8-bit passes `prefix`
  // is that key and `need` the number of keys equal to it that are taken.
  uint32_t prefix = 0u, mask = 0u;
  int need = K;
  const bool all = ncand <= K;
  if (!all) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[threadIdx.x] = 0;
      __syncthreads();
      for (int b = threadIdx.x; b < nb; b += kThreads) {
        const uint32_t k = key_at(b);
        if (k != 0u && (k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
      }
      __syncthreads();
      if (threadIdx.x < kWave) {
        // lane l owns digits 255-4l .. 252-4l (descending)
        const int lane = threadIdx.x;
        int hcount[4], lane_sum = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          hcount[j] = hist[255 - 4 * lane - j];
          lane_sum += hcount[j];
        }
        const int incl = wave_inclusive_scan(lane_sum);
        const int excl = incl - lane_sum;
        if (excl < need && need <= incl) {
          int run = excl;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (run + hcount[j] >= need) {
              pick[0] = 255 - 4 * lane - j;
              pick[1] = run;
              break;
            }
            run += hcount[j];
          }
        }
      }
      __syncthreads();
      need -= pick[1];
      prefix |= static_cast<uint32_t>(pick[0]) << shift;
      mask |= 255u << shift;
      __syncthreads();
    }
  }

  // Emit in ascending id order: thread t owns ids [t*per, (t+1)*per).
  const int per = (nb + kThreads - 1) / kThreads;
  const int lo = min(threadIdx.x * per, nb), hi = min(lo + per, nb);
  int n_eq = 0;
  if (!all)
    for (int b = lo; b < hi; ++b) n_eq += key_at(b) == prefix;
  int tot_eq;
  int eq_rank = block_exclusive_scan<kThreads>(n_eq, scan_tmp, tot_eq);
  int n_sel = 0;
  {
    int er = eq_rank;
    for (int b = lo; b < hi; ++b) {
      const uint32_t k = key_at(b);
      bool take;
      if (all) {
        take = k != 0u;
      } else if (k == prefix) {
        take = er < need;
        ++er;
      } else {
        take = k > prefix;
      }
      n_sel += take;
    }
  }
  int total;
  int pos = block_exclusive_scan<kThreads>(n_sel, scan_tmp, total);
  int32_t* out_idx = idx + row * K;
  float* out_score = score_out ? score_out + row * K : nullptr;
  {
    int er = eq_rank;
    for (int b = lo; b < hi; ++b) {
      const uint32_t k = key_at(b);
      bool take;
      if (all) {
        take = k != 0u;
      } else if (k == prefix) {
        take = er < need;
        ++er;
      } else {
        take = k > prefix;
      }
      if (take) {
        if (pos < K) {  // holds by construction; the guard keeps a bad input from writing past the row
          out_idx[pos] = b;
          if (out_score) out_score[pos] = s[b];
        }
        ++pos;
      }
    }
  }
  for (int t = total + threadIdx.x; t < K; t += kThreads) {
    out_idx[t] = -1;
    if (out_score) out_score[t] = -INFINITY;
  }
  if (threadIdx.x == 0) cnt[row] = total < K ? total : K;
}

inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

template <typename T, int D>
hipError_t launch_select_typed(const CacheGeom& g, const SelectPlan& p, const void* q, int32_t* idx, int32_t* cnt,
                               float* score, void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  float* qpart = reinterpret_cast<float*>(ws + p.off_qpart);
  float* qbar = reinterpret_cast<float*>(ws + p.off_qbar);
  float* kbar = reinterpret_cast<float*>(ws + p.off_kbar);
  float* scores = reinterpret_cast<float*>(ws + p.off_scores);

  hipLaunchKernelGGL((k_qmean_partial<T, D>), dim3(p.qsplit, p.R, g.H), dim3(kThreads), 0, stream,
                     static_cast<const T*>(q), p.lq, g.H, p.G, p.R, p.qsplit, qpart);
  hipLaunchKernelGGL((k_qmean_final<D>), dim3(p.R, g.H), dim3(D), 0, stream, qpart, p.lq, p.G, p.R, p.qsplit, qbar);

  if (g.nb > 0) {
    PoolArgs a;
    a.k_pages = g.k_pages;
    a.page_table = g.page_table;
    a.num_pages = g.num_pages;
    a.H = g.H;
    a.S = g.S;
    a.Bpc = g.Bpc;
    a.nb = g.nb;
    a.first_excluded = p.first_excluded;
    a.qbar = qbar;
    a.R = p.R;
    a.scale = p.scale;
    a.scores = scores;
    a.kbar = kbar;
    a.blocks_per_wave = 2;
    const int waves = (g.nb + a.blocks_per_wave - 1) / a.blocks_per_wave;
    const dim3 grid((waves + kThreads / kWave - 1) / (kThreads / kWave), g.H);
    if (g.B == 64) {
      if (p.inline_scores)
        hipLaunchKernelGGL((k_pool_score<T, D, 64, true>), grid, dim3(kThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((k_pool_score<T, D, 64, false>), grid, dim3(kThreads), 0, stream, a);
    } else {
      if (p.inline_scores)
        hipLaunchKernelGGL((k_pool_score<T, D, 128, true>), grid, dim3(kThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((k_pool_score<T, D, 128, false>), grid, dim3(kThreads), 0, stream, a);
    }
    if (!p.inline_scores) {
      const dim3 sgrid((g.nb + 63) / 64, (p.R + 15) / 16, g.H);
      hipLaunchKernelGGL((k_score<D>), sgrid, dim3(kThreads), 0, stream, kbar, qbar, g.page_table, g.num_pages, g.nb,
                         p.first_excluded, p.R, p.scale, scores);
    }
  }
  const dim3 tgrid(p.R, g.H);
  if (g.nb <= kTopkLdsMax) {
    hipLaunchKernelGGL((k_topk<true>), tgrid, dim3(kThreads), static_cast<size_t>(g.nb) * 4 + 16, stream, scores,
                       g.page_table, g.num_pages, g.nb, p.first_excluded, p.R, p.K, idx, cnt, score);
  } else {
    hipLaunchKernelGGL((k_topk<false>), tgrid, dim3(kThreads), 0, stream, scores, g.page_table, g.num_pages, g.nb,
                       p.first_excluded, p.R, p.K, idx, cnt, score);
  }
  return hipGetLastError();
}

}  // namespace

SelectPlan plan_select(const CacheGeom& g, int lq, int K, int G, int E, int T_out, float scale, int awe) {
  (void)T_out;
  SelectPlan p{};
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
  p.off_qbar = off;
  off = align256(off + static_cast<size_t>(g.H) * p.R * g.D * sizeof(float));
  p.off_kbar = off;
  if (!p.inline_scores) off = align256(off + static_cast<size_t>(g.H) * g.nb * g.D * sizeof(float));
  p.off_scores = off;
  off = align256(off + static_cast<size_t>(g.H) * p.R * (g.nb > 0 ? g.nb : 1) * sizeof(float));
  p.total = off;
  return p;
}

hipError_t launch_select(const CacheGeom& g, const SelectPlan& p, const void* q, int32_t* idx, int32_t* cnt,
                         float* score, void* workspace, hipStream_t stream) {
  if (g.dtype == 0) {
    if (g.D == 128) return launch_select_typed<uint16_t, 128>(g, p, q, idx, cnt, score, workspace, stream);
    return launch_select_typed<uint16_t, 64>(g, p, q, idx, cnt, score, workspace, stream);
  }
  if (g.D == 128) return launch_select_typed<float, 128>(g, p, q, idx, cnt, score, workspace, stream);
  return launch_select_typed<float, 64>(g, p, q, idx, cnt, score, workspace, stream);
}

}  // namespace omnimem
