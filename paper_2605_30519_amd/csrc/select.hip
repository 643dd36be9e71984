// select.hip -- query-shared block selection with Adaptive Window Exclusion
// (Sec. 3.2 Eq. 2, Sec. 3.3 Eq. 3) for gfx950.
//
// Pipeline (one stream, no host round trip):
//   k_qmean_partial  Q rows -> fp32 partial column sums per (head, group, 512-row split)
//   k_pool_score     streams every candidate K block once: block mean over its valid
//                    tokens, then s[h][r][b] = scale * <qbar[h][r], kbar[h][b]>, stored
//                    as an order-preserving 32-bit key (0 outside Omega), the
//                    proxy query qbar (group mean) being summed from the partials in
//                    each wave's prologue (for many groups it writes kbar and k_score
//                    does the products)
//   k_topk           one workgroup per (head, group): exact top-K over Omega by
//                    histogram refinement of the key interval holding the K-th key,
//                    keys held in registers, ties to the lower block id, ids written
//                    in ascending order (for K <= 16, k_topk_small: one wave per row,
//                    per-lane sorted lists merged by wave-wide maxima).
// The dominant cost is the K stream in k_pool_score, which is HBM-bound: each wave
// owns whole (page, head) slabs (B*d contiguous elements) and reads them with
// 16-byte loads, all lanes of a wave in flight on one slab at a time.
#include <float.h>
#include <math.h>

#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

constexpr int kThreads = 256;

// -------------------------------------------------------------- proxy queries
constexpr int kQThreads = 512;
constexpr int kQColSplits = 2;       // the big variant: each workgroup sums half of d (one 128-byte line per row)
constexpr int kQSmallThreads = 64;   // groups of at most kQSmallRows rows: one wave per split
constexpr int kQSmallRows = 64;

// NT threads per (split, column range of D/DS); UNROLL rows per thread in flight
// (the big variant covers a 512-row split in one round, the one-wave variant small
// groups).  blockIdx.x = split * DS + column range.
template <typename T, int D, int NT, int DS>
__global__ __launch_bounds__(NT) void k_qmean_partial(const T* __restrict__ q, int lq, int H, int G, int R,
                                                      int nsplit, float* __restrict__ partial) {
  using V = Vec16<T>;
  constexpr int VEC = V::N;
  constexpr int DC = D / DS;          // columns of this workgroup
  constexpr int CPR = DC / VEC;       // 16-byte chunks per row
  constexpr int PHASES = NT / CPR;    // rows summed side by side
  constexpr int SPLIT_ROWS = NT == kQSmallThreads ? kQSmallRows : kQRowsPerSplit;
  constexpr int UNROLL = (SPLIT_ROWS + PHASES - 1) / PHASES;
  constexpr int kWaves = NT / kWave, PH_PER_WAVE = kWave / CPR;
  __shared__ float red[kWaves][DC];

  const int s = blockIdx.x / DS, cs = blockIdx.x % DS, r = blockIdx.y, h = blockIdx.z;
  const int g0 = r * G, g1 = min(g0 + G, lq);
  const int r0 = g0 + s * kQRowsPerSplit, r1 = min(r0 + kQRowsPerSplit, g1);
  const int c = threadIdx.x % CPR, ph = threadIdx.x / CPR;

  float acc[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
  for (int row = r0 + ph; row < r1; row += UNROLL * PHASES) {
    uint4 raw[UNROLL];  // UNROLL independent loads in flight before the adds
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int rr = row + u * PHASES;
      raw[u] = rr < r1 ? load_once(q + (static_cast<int64_t>(rr) * H + h) * D + cs * DC + c * VEC)
                       : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      float x[VEC];
      V::widen(raw[u], x);
#pragma unroll
      for (int j = 0; j < VEC; ++j) acc[j] += x[j];
    }
  }
  // the row phases of a wave (lanes c, c + CPR, ...) by shuffles, then the waves through LDS
#pragma unroll
  for (int m = CPR; m < kWave; m <<= 1)
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] += __shfl_xor(acc[j], m);
  const int wave = threadIdx.x / kWave;
  if (threadIdx.x % kWave < CPR) {
#pragma unroll
    for (int j = 0; j < VEC; ++j) red[wave][c * VEC + j] = acc[j];
  }
  __syncthreads();
  static_assert(PH_PER_WAVE >= 1, "a wave spans whole rows");
  for (int col = threadIdx.x; col < DC; col += NT) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) sum += red[w][col];
    partial[((static_cast<int64_t>(h) * R + r) * nsplit + s) * D + cs * DC + col] = sum;
  }
}

// Proxy query columns [col, col + N) of group r: the partial sums added in split
// order (the same order everywhere, so every reader gets identical values), divided
// by the group's row count.  The partials are fetched kBatch at a time, every load
// of a batch in flight before its adds.
template <int N>
__device__ __forceinline__ void proxy_cols(const float* __restrict__ partial, int h, int r, int R, int nsplit, int D,
                                           int col, int lq, int G, float (&out)[N]) {
  constexpr int kBatch = 16;
  const int g0 = r * G, rows = min(g0 + G, lq) - g0;
  const int used = (rows + kQRowsPerSplit - 1) / kQRowsPerSplit;
  const float* p = partial + (static_cast<int64_t>(h) * R + r) * nsplit * D + col;
#pragma unroll
  for (int j = 0; j < N; ++j) out[j] = 0.f;
  for (int s0 = 0; s0 < used; s0 += kBatch) {
    float v[kBatch][N];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
#pragma unroll
      for (int j = 0; j < N; ++j) v[u][j] = s0 + u < used ? p[static_cast<int64_t>(s0 + u) * D + j] : 0.f;
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
#pragma unroll
      for (int j = 0; j < N; ++j)
        if (s0 + u < used) out[j] += v[u][j];
  }
  const float inv_rows = 1.0f / static_cast<float>(rows);
#pragma unroll
  for (int j = 0; j < N; ++j) out[j] = out[j] * inv_rows;
}

// -------------------------------------------------------------- score keys
// Inverse of score_key on candidate keys (returns the score with -0 as +0).
__device__ __forceinline__ float key_score(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
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

// Issues every 16-byte load of a slab (rows past nvalid read as zero).
template <typename T, int D, int B>
__device__ __forceinline__ void load_slab(const T* __restrict__ slab, int nvalid, int lane,
                                          uint4 (&raw)[SlabShape<T, D, B>::PASSES]) {
  using Sh = SlabShape<T, D, B>;
  const int c = lane % Sh::CPR, ph = lane / Sh::CPR;
#pragma unroll
  for (int i = 0; i < Sh::PASSES; ++i) {
    const int row = ph + i * Sh::ROWS_PER_PASS;
    raw[i] = row < nvalid ? load_once(slab + row * D + c * Sh::VEC) : make_uint4(0, 0, 0, 0);
  }
}

// Column sums of a loaded slab; every lane ends with the sums of its column chunk.
template <typename T, int D, int B>
__device__ __forceinline__ void sum_slab(const uint4 (&raw)[SlabShape<T, D, B>::PASSES],
                                         float (&colsum)[Vec16<T>::N]) {
  using Sh = SlabShape<T, D, B>;
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

// Column sums of a slab read CHUNK loads per lane at a time (for slabs whose loads
// would not all fit in registers at once); the same per-lane order of adds as
// load_slab + sum_slab, so the same sums bit for bit.
template <typename T, int D, int B, int CHUNK>
__device__ __forceinline__ void load_sum_slab(const T* __restrict__ slab, int nvalid, int lane,
                                              float (&colsum)[Vec16<T>::N]) {
  using Sh = SlabShape<T, D, B>;
  static_assert(Sh::PASSES % CHUNK == 0, "whole chunks of loads");
  const int c = lane % Sh::CPR, ph = lane / Sh::CPR;
#pragma unroll
  for (int j = 0; j < Sh::VEC; ++j) colsum[j] = 0.f;
#pragma unroll 1
  for (int i0 = 0; i0 < Sh::PASSES; i0 += CHUNK) {  // one chunk's loads live at a time
    uint4 raw[CHUNK];
#pragma unroll
    for (int i = 0; i < CHUNK; ++i) {
      const int row = ph + (i0 + i) * Sh::ROWS_PER_PASS;
      raw[i] = row < nvalid ? load_once(slab + row * D + c * Sh::VEC) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < CHUNK; ++i) {
      float x[Sh::VEC];
      Vec16<T>::widen(raw[i], x);
#pragma unroll
      for (int j = 0; j < Sh::VEC; ++j) colsum[j] += x[j];
    }
  }
#pragma unroll
  for (int m = Sh::CPR; m < kWave; m <<= 1)
#pragma unroll
    for (int j = 0; j < Sh::VEC; ++j) colsum[j] += __shfl_xor(colsum[j], m);
}

struct PoolArgs {
  const void* k_pages;
  const int32_t* page_table;
  int64_t pt_stride;  // per-head tables: head h's row of block b at h * pt_stride + b
  int64_t num_pages;
  int H, S, Bpc, nb, first_excluded;
  const float* qpart;  // [H][R][nsplit][D] partial row sums of Q
  int nsplit, lq, G;
  int R;
  float scale;
  uint32_t* keys;  // [H][R][nbp] score keys, 0 outside Omega (inline mode)
  int nbp;         // key row stride: nb rounded up to a multiple of 4
  float* kbar;    // [H][nb][D] (kbar mode)
  int blocks_per_wave;
};

// NR > 0: scores of up to NR groups computed in place; NR == 0: kbar written for k_score.
template <typename T, int D, int B, int NR>
__global__ __launch_bounds__(kThreads) void k_pool_score(PoolArgs a) {
  using Sh = SlabShape<T, D, B>;
  constexpr int VEC = Sh::VEC;
  constexpr int kMaxBlocksPerWave = 8;
  const int h = blockIdx.y;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int c = lane % Sh::CPR;
  const int first = (blockIdx.x * (kThreads / kWave) + wave) * a.blocks_per_wave;
  const int last = min(first + a.blocks_per_wave, a.nb);
  const T* pages = static_cast<const T*>(a.k_pages);

  int32_t page_ids[kMaxBlocksPerWave];  // the wave's page ids, loaded together before any slab
  const int32_t* table = a.page_table + static_cast<int64_t>(h) * a.pt_stride;
#pragma unroll
  for (int i = 0; i < kMaxBlocksPerWave; ++i) page_ids[i] = first + i < last ? table[first + i] : -1;
  auto live = [&](int i) {
    const int64_t page = page_ids[i];
    return first + i < last && first + i < a.first_excluded && page >= 0 && page < a.num_pages;
  };
  auto valid_rows = [&](int b) {
    const int o = b % a.Bpc;
    return o == a.Bpc - 1 ? a.S - o * B : B;
  };
  auto slab_of = [&](int i) { return pages + (static_cast<int64_t>(page_ids[i]) * a.H + h) * static_cast<int64_t>(B) * D; };

  // the first slab's loads go out before the proxy-query prologue, so that its
  // latency overlaps theirs
  uint4 raw[Sh::PASSES];
  if (live(0)) load_slab<T, D, B>(slab_of(0), valid_rows(first), lane, raw);

  float q[NR > 0 ? NR : 1][VEC];
  if (NR > 0) {
    // the workgroup's proxy queries, summed from the partials once and shared in LDS
    __shared__ float qs[NR > 0 ? NR : 1][D];
    for (int i = threadIdx.x; i < a.R * D; i += kThreads) {
      float v[1];
      proxy_cols<1>(a.qpart, h, i / D, a.R, a.nsplit, D, i % D, a.lq, a.G, v);
      qs[i / D][i % D] = v[0];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
      for (int j = 0; j < VEC; ++j) q[r][j] = r < a.R ? qs[r][c * VEC + j] : 0.f;
  }

#pragma unroll
  for (int i = 0; i < kMaxBlocksPerWave; ++i) {
    const int b = first + i;
    if (b >= last) break;
    if (!live(i)) {
      if (NR > 0) {
        if (lane < a.R) a.keys[(static_cast<int64_t>(h) * a.R + lane) * a.nbp + b] = 0u;
      }
      continue;
    }
    const int nvalid = valid_rows(b);
    if (i > 0) load_slab<T, D, B>(slab_of(i), nvalid, lane, raw);
    float colsum[VEC];
    sum_slab<T, D, B>(raw, colsum);
    const float inv = 1.0f / static_cast<float>(nvalid);
    if (NR > 0) {
#pragma unroll
      for (int r = 0; r < (NR > 0 ? NR : 1); ++r) {
        if (r >= a.R) break;
        float dot = 0.f;
#pragma unroll
        for (int j = 0; j < VEC; ++j) dot += q[r][j] * (colsum[j] * inv);
#pragma unroll
        for (int m = 1; m < Sh::CPR; m <<= 1) dot += __shfl_xor(dot, m);
        if (lane == 0) a.keys[(static_cast<int64_t>(h) * a.R + r) * a.nbp + b] = score_key(a.scale * dot);
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

// score keys for many groups: tile of 64 blocks x 16 groups per workgroup
template <int D>
__global__ __launch_bounds__(kThreads) void k_score(const float* __restrict__ kbar, int64_t kbar_stride,
                                                    const float* __restrict__ qpart,
                                                    int nsplit, int lq, int G, const int32_t* __restrict__ page_table,
                                                    int64_t pt_stride, int64_t num_pages, int nb, int nbp,
                                                    int first_excluded, int R, float scale,
                                                    uint32_t* __restrict__ keys) {
  constexpr int TB = 64, TR = 16;
  __shared__ float ks[TB][D + 1];
  __shared__ float qs[TR][D + 1];
  const int b0 = blockIdx.x * TB, r0 = blockIdx.y * TR, h = blockIdx.z;
  for (int i = threadIdx.x; i < TB * D; i += kThreads) {
    const int bb = i / D, j = i % D;
    ks[bb][j] = b0 + bb < nb ? kbar[(static_cast<int64_t>(h) * kbar_stride + b0 + bb) * D + j] : 0.f;
  }
  for (int i = threadIdx.x; i < TR * D; i += kThreads) {
    const int rr = i / D, j = i % D;
    float v[1] = {0.f};
    if (r0 + rr < R) proxy_cols<1>(qpart, h, r0 + rr, R, nsplit, D, j, lq, G, v);
    qs[rr][j] = v[0];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < TB * TR; t += kThreads) {
    const int bb = t % TB, rr = t / TB;
    const int b = b0 + bb, r = r0 + rr;
    if (b >= nb || r >= R) continue;
    float dot = 0.f;
    for (int j = 0; j < D; ++j) dot += qs[rr][j] * ks[bb][j];
    // no page table: every block is a candidate (residency is managed elsewhere)
    const int32_t p = page_table != nullptr ? page_table[static_cast<int64_t>(h) * pt_stride + b] : 0;
    const bool live = b < first_excluded && p >= 0 && (page_table == nullptr || p < num_pages);
    keys[(static_cast<int64_t>(h) * R + r) * nbp + b] = live ? score_key(scale * dot) : 0u;
  }
}

// Score keys for few groups (R <= kInlineGroups) from stored pooled keys: one wave
// per run of kScoreRowsPerWave blocks of a head; lane l holds dimensions
// [D/64 * l, D/64 * (l + 1)) of every proxy query in registers and of each pooled key
// row as it is read (one coalesced row read per block), then the dot products are
// reduced across the wave by shuffles.
constexpr int kScoreRowsPerWave = 8;

template <int D, int NR>
__global__ __launch_bounds__(kThreads) void k_score_rows(const float* __restrict__ kbar, int64_t kbar_stride,
                                                         const float* __restrict__ qpart, int nsplit, int lq, int G,
                                                         const int32_t* __restrict__ page_table, int64_t pt_stride,
                                                         int64_t num_pages, int nb, int nbp, int first_excluded, int R,
                                                         float scale, uint32_t* __restrict__ keys) {
  constexpr int PL = D / kWave;  // dimensions per lane: 2 (d = 128) or 1 (d = 64)
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave, h = blockIdx.y;
  const int first = (blockIdx.x * (kThreads / kWave) + wave) * kScoreRowsPerWave;
  float q[NR][PL];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    float v[PL];
#pragma unroll
    for (int j = 0; j < PL; ++j) v[j] = 0.f;
    if (r < R) proxy_cols<PL>(qpart, h, r, R, nsplit, D, PL * lane, lq, G, v);
#pragma unroll
    for (int j = 0; j < PL; ++j) q[r][j] = v[j];
  }
  float k[kScoreRowsPerWave][PL];  // every row's loads in flight before the products
#pragma unroll
  for (int i = 0; i < kScoreRowsPerWave; ++i) {
    const int b = first + i;
#pragma unroll
    for (int j = 0; j < PL; ++j)
      k[i][j] = b < nb ? kbar[(static_cast<int64_t>(h) * kbar_stride + b) * D + PL * lane + j] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < kScoreRowsPerWave; ++i) {
    const int b = first + i;
    if (b >= nb) break;
    const int32_t p = page_table != nullptr ? page_table[static_cast<int64_t>(h) * pt_stride + b] : 0;
    const bool live = b < first_excluded && p >= 0 && (page_table == nullptr || p < num_pages);
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      if (r >= R) break;
      float dot = 0.f;
#pragma unroll
      for (int j = 0; j < PL; ++j) dot = fmaf(q[r][j], k[i][j], dot);
#pragma unroll
      for (int m = 1; m < kWave; m <<= 1) dot += __shfl_xor(dot, m);
      if (lane == 0) keys[(static_cast<int64_t>(h) * R + r) * nbp + b] = live ? score_key(scale * dot) : 0u;
    }
  }
}

// Score keys for many groups (R >= kScoreTiledMinGroups): the products q_r . k_b form
// a dense R x N_b contraction per head, run on fp32 MFMA (v_mfma_f32_32x32x2_f32,
// fp32 products and accumulation).  A workgroup takes 64 groups x 64 blocks, each of
// its four waves a 32 x 32 quarter; proxy queries and pooled keys pass through LDS
// 32 dimensions at a time, stored dimension-major with a row stride of 96 floats so
// that the two half-waves of an operand read (dimensions 2s and 2s + 1) fall on
// disjoint banks.
constexpr int kScoreTiledMinGroups = 32;

template <int D>
__global__ __launch_bounds__(kThreads) void k_score_tiled(const float* __restrict__ kbar, int64_t kbar_stride,
                                                          const float* __restrict__ qpart, int nsplit, int lq, int G,
                                                          const int32_t* __restrict__ page_table, int64_t pt_stride,
                                                          int64_t num_pages, int nb, int nbp, int first_excluded,
                                                          int R, float scale, uint32_t* __restrict__ keys) {
  constexpr int TB = 64, TR = 64, KC = 32, STRIDE = 96;
  __shared__ __align__(16) float ks[KC][STRIDE];  // [dimension][block]
  __shared__ __align__(16) float qs[KC][STRIDE];  // [dimension][group]
  const int b0 = blockIdx.x * TB, r0 = blockIdx.y * TR, h = blockIdx.z;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int wr = 32 * (wave / 2), wb = 32 * (wave % 2);  // this wave's quarter
  f32x16 acc = {};
  // one row per lane, four dimensions per load (the LDS stores of a wave are then
  // conflict-free); the next chunk's loads are in flight during this chunk's MFMAs
  constexpr int PER = TB * (KC / 4) / kThreads;  // loads per thread per chunk
  float4 kv[PER], qv[PER];
  // groups of one split (the usual case here: small groups) hold their sum in one
  // partial: one load, scaled by the group's reciprocal row count
  float inv_rows[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int r = r0 + (threadIdx.x + u * kThreads) % TB;
    inv_rows[u] = r < R ? 1.0f / static_cast<float>(min(r * G + G, lq) - r * G) : 0.f;
  }
  auto fetch = [&](int j0) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = threadIdx.x + u * kThreads, row = i % TB, jq = i / TB;
      kv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (b0 + row < nb)
        kv[u] = *reinterpret_cast<const float4*>(kbar + (static_cast<int64_t>(h) * kbar_stride + b0 + row) * D + j0 +
                                                 4 * jq);
      qv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (r0 + row < R) {
        if (nsplit == 1) {
          const float4 sum = *reinterpret_cast<const float4*>(
              qpart + (static_cast<int64_t>(h) * R + r0 + row) * D + j0 + 4 * jq);
          qv[u] = make_float4(sum.x * inv_rows[u], sum.y * inv_rows[u], sum.z * inv_rows[u], sum.w * inv_rows[u]);
        } else {
          float q4[4];
          proxy_cols<4>(qpart, h, r0 + row, R, nsplit, D, j0 + 4 * jq, lq, G, q4);
          qv[u] = make_float4(q4[0], q4[1], q4[2], q4[3]);
        }
      }
    }
  };
  fetch(0);
  for (int j0 = 0; j0 < D; j0 += KC) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = threadIdx.x + u * kThreads, row = i % TB, jq = i / TB;
      ks[4 * jq + 0][row] = kv[u].x;
      ks[4 * jq + 1][row] = kv[u].y;
      ks[4 * jq + 2][row] = kv[u].z;
      ks[4 * jq + 3][row] = kv[u].w;
      qs[4 * jq + 0][row] = qv[u].x;
      qs[4 * jq + 1][row] = qv[u].y;
      qs[4 * jq + 2][row] = qv[u].z;
      qs[4 * jq + 3][row] = qv[u].w;
    }
    __syncthreads();
    if (j0 + KC < D) fetch(j0 + KC);
#pragma unroll
    for (int st = 0; st < KC / 2; ++st) {
      const int j = 2 * st + lane / 32;
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qs[j][wr + lane % 32], ks[j][wb + lane % 32], acc, 0, 0, 0);
    }
    __syncthreads();
  }
  // accumulator element i of lane l: group wr + 8 (i / 4) + 4 (l / 32) + i % 4, block wb + l % 32
  const int b = b0 + wb + lane % 32;
  if (b >= nb) return;
  const int32_t p = page_table != nullptr ? page_table[static_cast<int64_t>(h) * pt_stride + b] : 0;
  const bool live = b < first_excluded && p >= 0 && (page_table == nullptr || p < num_pages);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = r0 + wr + 8 * (i / 4) + 4 * (lane / 32) + i % 4;
    if (r < R) keys[(static_cast<int64_t>(h) * R + r) * nbp + b] = live ? score_key(scale * acc[i]) : 0u;
  }
}

// -------------------------------------------------------------- compressed history
// Pools one history chunk into the compressed cache: one wave per (block, head)
// slab; the block's K and V column means go to k_mean (fp32) and, rounded to the
// cache dtype, to pooled token b of the paged pooled sequence.
struct CompressArgs {
  const void* k_pages;
  const void* v_pages;
  const int32_t* page_table;
  int64_t pt_stride;
  int64_t num_pages;
  int H, S, Bpc, chunk;
  float* k_mean;
  void* ck_pages;
  void* cv_pages;
  void* ck_lo;  // optional: bf16 residual of the pooled keys (bf16 caches)
  int32_t* c_page_table;
  int cap_blocks;
};

template <typename T>
__device__ __forceinline__ void store_rounded(T* dst, const float (&x)[Vec16<T>::N]);

template <>
__device__ __forceinline__ void store_rounded<uint16_t>(uint16_t* dst, const float (&x)[8]) {
  uint4 w;
  w.x = f32_to_bf16_rne(x[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[1])) << 16);
  w.y = f32_to_bf16_rne(x[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[3])) << 16);
  w.z = f32_to_bf16_rne(x[4]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[5])) << 16);
  w.w = f32_to_bf16_rne(x[6]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[7])) << 16);
  *reinterpret_cast<uint4*>(dst) = w;
}

template <>
__device__ __forceinline__ void store_rounded<float>(float* dst, const float (&x)[4]) {
  *reinterpret_cast<float4*>(dst) = make_float4(x[0], x[1], x[2], x[3]);
}

// The residual of 8 fp32 values after their rounding to bf16, itself rounded to bf16
// (both to nearest even): x ~= hi + lo to about 2^-17 relative.
__device__ __forceinline__ void store_residual_bf16(uint16_t* dst, const float (&x)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 8; j += 2) {
    const float r0 = x[j] - __uint_as_float(static_cast<uint32_t>(f32_to_bf16_rne(x[j])) << 16);
    const float r1 = x[j + 1] - __uint_as_float(static_cast<uint32_t>(f32_to_bf16_rne(x[j + 1])) << 16);
    w[j / 2] = f32_to_bf16_rne(r0) | (static_cast<uint32_t>(f32_to_bf16_rne(r1)) << 16);
  }
  *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
}

template <typename T, int D, int B>
__global__ __launch_bounds__(kThreads) void k_compress_chunk(CompressArgs a) {
  using Sh = SlabShape<T, D, B>;
  constexpr int VEC = Sh::VEC;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int o = blockIdx.x * (kThreads / kWave) + wave, h = blockIdx.y;
  if (o >= a.Bpc) return;
  const int b = a.chunk * a.Bpc + o;
  const int c = lane % Sh::CPR;
  const int64_t page = a.page_table[static_cast<int64_t>(h) * a.pt_stride + b];
  const bool live = page >= 0 && page < a.num_pages;
  const int nvalid = o == a.Bpc - 1 ? a.S - o * B : B;
  float ks[VEC], vs[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) ks[j] = vs[j] = 0.f;
  if (live) {
    const int64_t off = (page * a.H + h) * static_cast<int64_t>(B) * D;
    if constexpr (Sh::PASSES <= 32) {
      uint4 kraw[Sh::PASSES], vraw[Sh::PASSES];  // both slabs' loads in flight before the sums
      load_slab<T, D, B>(static_cast<const T*>(a.k_pages) + off, nvalid, lane, kraw);
      load_slab<T, D, B>(static_cast<const T*>(a.v_pages) + off, nvalid, lane, vraw);
      sum_slab<T, D, B>(kraw, ks);
      sum_slab<T, D, B>(vraw, vs);
    } else {
      // fp32 slabs of 128 tokens (64 loads per lane each): K, then V, 32 loads in flight
      load_sum_slab<T, D, B, 32>(static_cast<const T*>(a.k_pages) + off, nvalid, lane, ks);
      load_sum_slab<T, D, B, 32>(static_cast<const T*>(a.v_pages) + off, nvalid, lane, vs);
    }
    const float inv = 1.0f / static_cast<float>(nvalid);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      ks[j] *= inv;
      vs[j] *= inv;
    }
  }
  if (lane < Sh::CPR) {
    float* km = a.k_mean + (static_cast<int64_t>(h) * a.cap_blocks + b) * D + c * VEC;
#pragma unroll
    for (int j = 0; j < VEC; j += 4) *reinterpret_cast<float4*>(km + j) = make_float4(ks[j], ks[j + 1], ks[j + 2], ks[j + 3]);
    const int64_t cp = b / kCmpPageTokens, slot = b % kCmpPageTokens;
    const int64_t at = ((cp * a.H + h) * kCmpPageTokens + slot) * D + c * VEC;
    store_rounded<T>(static_cast<T*>(a.ck_pages) + at, ks);
    store_rounded<T>(static_cast<T*>(a.cv_pages) + at, vs);
    if constexpr (std::is_same_v<T, uint16_t>)
      if (a.ck_lo != nullptr) store_residual_bf16(static_cast<uint16_t*>(a.ck_lo) + at, ks);
    if (lane == 0 && h == 0 && (slot == 0 || o == 0)) a.c_page_table[cp] = static_cast<int32_t>(cp);
  }
}

// -------------------------------------------------------------- top-K
__device__ __forceinline__ int lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0));
}

// Exact top-K of one (head, group) key row, one workgroup of NT threads.
//
// Every key stays in a register: wave w holds the contiguous ids
// [w C, (w + 1) C), C = 256 J, lane l the four ids w C + 256 j + 4 l + e (j < J, e < 4).
// The K-th largest key is found by refinement over key intervals [lo, hi] for which
// #{key >= lo} >= K and #{key > hi} < K: the interval is cut into 2048 equal bins
// (a shift of key - lo), an LDS histogram and a suffix scan name the bin holding
// the K-th key, and that bin's keys become the next interval.  Once a bin holds at
// most kTopkList keys, their exact ranks (pairwise comparison in LDS) give the key;
// a bin spans at most 2^-10 of its interval, so a few levels suffice for any input.
// Emission walks the waves' ranges in id order: keys above the K-th are taken, ties
// at it go to the lowest ids, positions come from ballot ranks.
constexpr int kTopkMaxThreads = 1024;
constexpr int kTopkVecPerLane = 8;                                        // J <= 8: 32 keys per lane
constexpr int kTopkRegMax = kTopkMaxThreads * 4 * kTopkVecPerLane;        // larger rows take k_topk_wide
constexpr int kTopkBinBits = 11;
constexpr int kTopkBins = 1 << kTopkBinBits;
constexpr int kTopkList = 256;
constexpr int kTopkManyRows = 1024;  // (head, group) rows from which k_topk<256> is used
constexpr int kPoolBlocksPerWave = 2;  // at most the pooling kernel's page-id batch (kMaxBlocksPerWave)

// Called by all NT threads of a workgroup; out_score may be null.
template <int NT>
__device__ __forceinline__ void topk_row(const uint32_t* __restrict__ kp, int nb, int K, int32_t* __restrict__ out_idx,
                         float* __restrict__ out_score, int32_t* __restrict__ out_cnt) {
  constexpr int kWaves = NT / kWave, kBinsPerThread = kTopkBins / NT;
  __shared__ int hist[kTopkBins];
  __shared__ __align__(16) uint32_t list[kTopkList];
  __shared__ int wave_a[kWaves], wave_b[kWaves];
  __shared__ uint32_t wave_lo[kWaves], wave_hi[kWaves];
  __shared__ int s_bin, s_above, s_m;
  __shared__ uint32_t s_kth;
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int J = min(kTopkVecPerLane, (nb + 4 * NT - 1) / (4 * NT));
  const int base = wave * J * 4 * kWave;

  uint32_t kr[4 * kTopkVecPerLane];
#pragma unroll
  for (int j = 0; j < kTopkVecPerLane; ++j) {
    const int i = base + (j * kWave + lane) * 4;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (j < J && i < nb) v = *reinterpret_cast<const uint4*>(kp + i);  // i + 3 < nbp
    kr[4 * j + 0] = v.x;
    kr[4 * j + 1] = i + 1 < nb ? v.y : 0u;
    kr[4 * j + 2] = i + 2 < nb ? v.z : 0u;
    kr[4 * j + 3] = i + 3 < nb ? v.w : 0u;
  }
#pragma unroll
  for (int u = 0; u < kBinsPerThread; ++u) hist[tid * kBinsPerThread + u] = 0;
  {
    int n = 0;
    uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
    for (int j = 0; j < 4 * kTopkVecPerLane; ++j) {
      if (j >= 4 * J) break;
      n += kr[j] != 0u;
      kmin = min(kmin, kr[j] != 0u ? kr[j] : 0xffffffffu);
      kmax = max(kmax, kr[j]);
    }
    n = __reduce_add_sync(~0ull, n);
    kmin = __reduce_min_sync(~0ull, kmin);
    kmax = __reduce_max_sync(~0ull, kmax);
    if (lane == 0) {
      wave_a[wave] = n;
      wave_lo[wave] = kmin;
      wave_hi[wave] = kmax;
    }
  }
  __syncthreads();
  int ncand = 0;
  uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    ncand += wave_a[w];
    lo = min(lo, wave_lo[w]);
    hi = max(hi, wave_hi[w]);
  }
  const bool all = ncand <= K;
  uint32_t kth = 0u;  // with `all`, every key > 0 is taken
  if (!all) {
    int above = 0;  // #{key > hi}
    while (true) {
      if (lo == hi) {
        kth = lo;
        break;
      }
      const int width = 32 - __clz(hi - lo);
      const int shift = width > kTopkBinBits ? width - kTopkBinBits : 0;
#pragma unroll
      for (int j = 0; j < 4 * kTopkVecPerLane; ++j) {
        if (j >= 4 * J) break;
        if (kr[j] - lo <= hi - lo) atomicAdd(&hist[(kr[j] - lo) >> shift], 1);
      }
      __syncthreads();
      // suffix scan from the top bin: thread t owns the kBinsPerThread bins that
      // start kBinsPerThread * t bins below the top, in descending order
      int c[kBinsPerThread], csum = 0;
#pragma unroll
      for (int u = 0; u < kBinsPerThread; ++u) {
        c[u] = hist[kTopkBins - 1 - (tid * kBinsPerThread + u)];
        csum += c[u];
      }
      const int incl = wave_inclusive_scan(csum);
      if (lane == kWave - 1) wave_b[wave] = incl;
      if (tid == 0) s_m = 0;
      for (int i = tid; i < kTopkList; i += NT) list[i] = 0u;  // zero padding for the rank step
      __syncthreads();
      int before = above + incl - csum;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) before += w < wave ? wave_b[w] : 0;
#pragma unroll
      for (int u = 0; u < kBinsPerThread; ++u) {
        if (before < K && before + c[u] >= K) {
          s_bin = kTopkBins - 1 - (tid * kBinsPerThread + u);
          s_above = before;
        }
        before += c[u];
      }
      __syncthreads();
      const int bstar = s_bin;
      above = s_above;
#pragma unroll
      for (int u = 0; u < kBinsPerThread; ++u) hist[tid * kBinsPerThread + u] = 0;  // ready for a further level
      // gather the keys of bin b* into the list: one LDS atomic per wave reserves
      // the wave's slots, ballot ranks place the keys
      const uint32_t bin_lo = lo + (static_cast<uint32_t>(bstar) << shift);
      const uint32_t bin_span = static_cast<uint32_t>(
          min(static_cast<uint64_t>(hi - bin_lo), (1ull << shift) - 1u));  // bin = [bin_lo, bin_lo + bin_span]
      auto member = [&](uint32_t k) { return k - bin_lo <= bin_span; };
      int wave_members = 0;
#pragma unroll
      for (int j = 0; j < 4 * kTopkVecPerLane; ++j) {
        if (j >= 4 * J) break;
        wave_members += __popcll(__ballot(member(kr[j])));
      }
      if (wave_members > 0) {
        int at = 0;
        if (lane == 0) at = atomicAdd(&s_m, wave_members);
        at = __shfl(at, 0);
#pragma unroll
        for (int j = 0; j < 4 * kTopkVecPerLane; ++j) {
          if (j >= 4 * J) break;
          const bool mem = member(kr[j]);
          const uint64_t mask = __ballot(mem);
          const int pos = at + lane_rank(mask);
          if (mem && pos < kTopkList) list[pos] = kr[j];
          at += __popcll(mask);
        }
      }
      __syncthreads();
      const int m = s_m;
      if (m <= kTopkList) {
        // exact ranks inside the bin: the K-th key x has g(x) < need <= g(x) + e(x)
        const int need = K - above;
        if (tid < m) {
          // entries past m are 0, below every candidate key
          const uint32_t x = list[tid];
          const uint4* l4 = reinterpret_cast<const uint4*>(list);
          int g = 0, e = 0;
          for (int i = 0; i < m; i += 16) {
            uint4 y[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) y[u] = l4[i / 4 + u];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              g += (y[u].x > x) + (y[u].y > x) + (y[u].z > x) + (y[u].w > x);
              e += (y[u].x == x) + (y[u].y == x) + (y[u].z == x) + (y[u].w == x);
            }
          }
          if (g < need && need <= g + e) s_kth = x;
        }
        __syncthreads();
        kth = s_kth;
        break;
      }
      // more than kTopkList keys in b*: refine inside the bin's key range, which
      // keeps #{key >= lo} >= K and #{key > hi} < K
      lo = bin_lo;
      hi = bin_lo + bin_span;
    }
  }

  // per-wave counts above and at the K-th key, then emission in id order
  {
    int gt = 0, eq = 0;
#pragma unroll
    for (int j = 0; j < 4 * kTopkVecPerLane; ++j) {
      if (j >= 4 * J) break;
      gt += kr[j] > kth;
      eq += kr[j] == kth;
    }
    gt = __reduce_add_sync(~0ull, gt);
    eq = __reduce_add_sync(~0ull, eq);
    __syncthreads();  // wave_a / wave_b are reused
    if (lane == 0) {
      wave_a[wave] = gt;
      wave_b[wave] = eq;
    }
  }
  __syncthreads();
  int gt_all = 0, gt_before = 0, eq_before = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    gt_all += wave_a[w];
    if (w < wave) {
      gt_before += wave_a[w];
      eq_before += wave_b[w];
    }
  }
  const int total = all ? ncand : K;
  const int need = all ? 0 : K - gt_all;  // ties at the K-th key still to take
  int pos = gt_before + min(eq_before, need);
  int eq_run = eq_before;
#pragma unroll
  for (int j = 0; j < kTopkVecPerLane; ++j) {
    if (j >= J) break;
    bool tie[4], take[4];
    uint64_t tie_mask[4], take_mask[4];
    int tie_below = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tie[e] = !all && kr[4 * j + e] == kth;
      tie_mask[e] = __ballot(tie[e]);
      tie_below += lane_rank(tie_mask[e]);
    }
    int mine = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      take[e] = kr[4 * j + e] > kth || (tie[e] && eq_run + tie_below + mine < need);
      mine += tie[e];
    }
    int take_below = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      take_mask[e] = __ballot(take[e]);
      take_below += lane_rank(take_mask[e]);
    }
    int at = pos + take_below;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (take[e]) {
        if (at < K) {  // holds by construction; keeps a bad input inside the row
          out_idx[at] = base + (j * kWave + lane) * 4 + e;
          if (out_score) out_score[at] = key_score(kr[4 * j + e]);
        }
        ++at;
      }
      pos += __popcll(take_mask[e]);
      eq_run += __popcll(tie_mask[e]);
    }
  }
  for (int i = total + tid; i < K; i += NT) {
    out_idx[i] = -1;
    if (out_score) out_score[i] = -INFINITY;
  }
  if (tid == 0) *out_cnt = total < K ? total : K;
}

template <int NT>
__global__ __launch_bounds__(NT) void k_topk(const uint32_t* __restrict__ keys, int nb, int nbp, int K,
                                             int32_t* __restrict__ idx, int32_t* __restrict__ cnt,
                                             float* __restrict__ score_out) {
  const int64_t row = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  topk_row<NT>(keys + row * nbp, nb, K, idx + row * K, score_out ? score_out + row * K : nullptr, cnt + row);
}

// Top-K for small K (at most kTopkSmallK; the small-group setting selects K = 4):
// one wave per (head, group) row.  Lane l reads the ids 4 l + 256 j + e in increasing
// order and keeps the KM best (key, id) pairs it has seen in a sorted register list
// (an equal key arriving later has a higher id, so it ranks below); K rounds of a
// wave-wide maximum over the lanes' list heads, keyed by (key, lower id), then name
// the winners, which are written in ascending id order.
constexpr int kTopkSmallK = 16;
constexpr int kTopkSmallWaves = 4;  // rows per workgroup

template <int KM>
__global__ __launch_bounds__(kTopkSmallWaves* kWave) void k_topk_small(const uint32_t* __restrict__ keys, int rows,
                                                                         int nb, int nbp, int K,
                                                                         int32_t* __restrict__ idx,
                                                                         int32_t* __restrict__ cnt,
                                                                         float* __restrict__ score_out) {
  constexpr int kBatch = 8;  // 16-byte loads in flight per lane
  const int lane = threadIdx.x % kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kTopkSmallWaves + threadIdx.x / kWave;
  if (row >= rows) return;  // wave-uniform
  const uint32_t* kp = keys + row * nbp;

  uint32_t lk[KM];
  int li[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    lk[j] = 0u;
    li[j] = 0;
  }
  auto insert = [&](uint32_t k, int id) {
    if (k <= lk[KM - 1]) return;  // also drops non-candidates (key 0)
    bool placed = false;
#pragma unroll
    for (int j = KM - 1; j > 0; --j) {
      if (!placed) {
        if (k > lk[j - 1]) {
          lk[j] = lk[j - 1];
          li[j] = li[j - 1];
        } else {
          lk[j] = k;
          li[j] = id;
          placed = true;
        }
      }
    }
    if (!placed) {
      lk[0] = k;
      li[0] = id;
    }
  };
  for (int b0 = 0; b0 < nb; b0 += kBatch * 4 * kWave) {
    uint4 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = b0 + (u * kWave + lane) * 4;
      v[u] = i < nb ? *reinterpret_cast<const uint4*>(kp + i) : make_uint4(0u, 0u, 0u, 0u);  // i + 3 < nbp
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = b0 + (u * kWave + lane) * 4;
      insert(v[u].x, i);
      insert(i + 1 < nb ? v[u].y : 0u, i + 1);
      insert(i + 2 < nb ? v[u].z : 0u, i + 2);
      insert(i + 3 < nb ? v[u].w : 0u, i + 3);
    }
  }

  // K rounds: the largest (key, lower id) among the lanes' heads wins and leaves its list
  uint32_t wkey = 0u;
  int wid = 0, taken = 0;
  for (int r = 0; r < KM; ++r) {
    if (r >= K) break;
    const uint64_t mine =
        lk[0] == 0u ? 0ull : (static_cast<uint64_t>(lk[0]) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(li[0]));
    uint64_t best = mine;
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) {
      const uint64_t o = __shfl_xor(best, off);
      best = o > best ? o : best;
    }
    if (best == 0ull) break;  // fewer than K candidates
    if (mine == best) {
#pragma unroll
      for (int j = 0; j + 1 < KM; ++j) {
        lk[j] = lk[j + 1];
        li[j] = li[j + 1];
      }
      lk[KM - 1] = 0u;
    }
    if (lane == r) {
      wkey = static_cast<uint32_t>(best >> 32);
      wid = static_cast<int>(~static_cast<uint32_t>(best));
    }
    ++taken;
  }
  // ascending ids: lane r < taken writes winner r at its rank among the winners' ids
  int rank = 0;
  for (int s = 0; s < taken; ++s) rank += __shfl(wid, s) < wid;
  int32_t* out_idx = idx + row * K;
  float* out_score = score_out ? score_out + row * K : nullptr;
  if (lane < taken) {
    out_idx[rank] = wid;
    if (out_score) out_score[rank] = key_score(wkey);
  } else if (lane < K) {
    out_idx[lane] = -1;
    if (out_score) out_score[lane] = -INFINITY;
  }
  if (lane == 0) cnt[row] = taken;
}

// Scores and top-K in one kernel, for many query groups and small K (the small-group
// setting: groups of G_q rows, K blocks each): no score row is stored.  A workgroup
// takes 16 groups of one head; its NW waves split the head's blocks, each streaming
// its share 16 blocks at a time, two tiles ahead.  A tile's 16 x 16 scores come from
// fp32 MFMA (16x16x4): at step (u, e) lane group j = l / 16 supplies dimension
// 16 u + 4 j + e of its lane's group (A operand) and block (B operand), so the proxy
// queries stay in registers and the four lane groups of a block read 64 contiguous
// bytes of its row per load.  Lane l ends a tile with block b0 + l % 16 scored
// against groups 4 j .. 4 j + 3 and keeps, per group, the KM best (key, id) pairs it
// has seen (ids arrive in increasing order).  The lists meet in LDS, where half a
// wave per group merges them; ranking and ties are those of k_topk (key, then lower
// id).
constexpr int kStkGroups = 16;

template <int D, int KM, int NW>
__global__ __launch_bounds__(NW* kWave) void k_score_topk(
    const float* __restrict__ kbar, int64_t kbar_stride, const float* __restrict__ qpart, int nsplit, int lq, int G,
    const int32_t* __restrict__ page_table, int64_t pt_stride, int64_t num_pages, int nb, int first_excluded, int R,
    float scale, int K, int32_t* __restrict__ idx, int32_t* __restrict__ cnt, float* __restrict__ score_out) {
  constexpr int DS = D / 4;    // dimensions per lane group
  constexpr int NV = DS / 4;   // 16-byte loads per lane per tile: load u covers dimensions [16 u, 16 u + 16)
  __shared__ uint64_t cand[kStkGroups][NW * 16 * KM];
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = lane % 16, j = lane / 16;
  // workgroups of one head on one XCD, whose L2 then holds that head's pooled keys
  const int wg = xcd_contiguous_id(blockIdx.x, gridDim.x), tiles = (R + kStkGroups - 1) / kStkGroups;
  const int h = wg / tiles, g0 = (wg % tiles) * kStkGroups;

  // the proxy query of group g0 + col, dimensions 16 u + 4 j + e: its partial sums
  // added in split order, divided by the group's row count
  float qa[DS];
  {
    const int g = g0 + col;
    float4 sum[NV];
#pragma unroll
    for (int u = 0; u < NV; ++u) sum[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    float inv_rows = 0.f;
    if (g < R) {
      const int rows = min(g * G + G, lq) - g * G;
      const int used = (rows + kQRowsPerSplit - 1) / kQRowsPerSplit;
      const float* src = qpart + (static_cast<int64_t>(h) * R + g) * nsplit * D + 4 * j;
      for (int sp = 0; sp < used; ++sp) {
        float4 v[NV];
#pragma unroll
        for (int u = 0; u < NV; ++u) v[u] = *reinterpret_cast<const float4*>(src + static_cast<int64_t>(sp) * D + 16 * u);
#pragma unroll
        for (int u = 0; u < NV; ++u) {
          sum[u].x += v[u].x;
          sum[u].y += v[u].y;
          sum[u].z += v[u].z;
          sum[u].w += v[u].w;
        }
      }
      inv_rows = 1.0f / static_cast<float>(rows);
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      qa[4 * u + 0] = sum[u].x * inv_rows;
      qa[4 * u + 1] = sum[u].y * inv_rows;
      qa[4 * u + 2] = sum[u].z * inv_rows;
      qa[4 * u + 3] = sum[u].w * inv_rows;
    }
  }

  // this wave's blocks [bw0, bw1): share (wave + group tile) mod NW, so that the
  // workgroups of one head read different rows of its pooled keys at a time
  const int per = ((nb + NW - 1) / NW + 15) / 16 * 16;
  const int share = (wave + wg % tiles) % NW;
  const int bw0 = share * per, bw1 = min(bw0 + per, nb);
  const int32_t* table = page_table ? page_table + static_cast<int64_t>(h) * pt_stride : nullptr;
  const float* kh = kbar + static_cast<int64_t>(h) * kbar_stride * D;

  uint32_t lk[4][KM];
  int li[4][KM];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < KM; ++t) {
      lk[i][t] = 0u;
      li[i][t] = 0;
    }
  // insertion into a descending list without branches (k > lk[t] holds for a prefix
  // of t), skipped as a whole when no lane of the wave has a key to insert
  auto insert = [&](uint32_t (&lkk)[KM], int (&lii)[KM], uint32_t k, int id) {
    if (!__any(k > lkk[KM - 1])) return;
    bool gt[KM];
#pragma unroll
    for (int t = 0; t < KM; ++t) gt[t] = k > lkk[t];
#pragma unroll
    for (int t = KM - 1; t > 0; --t) {
      lkk[t] = gt[t - 1] ? lkk[t - 1] : (gt[t] ? k : lkk[t]);
      lii[t] = gt[t - 1] ? lii[t - 1] : (gt[t] ? id : lii[t]);
    }
    lkk[0] = gt[0] ? k : lkk[0];
    lii[0] = gt[0] ? id : lii[0];
  };

  // three tile buffers: tile t is scored while tiles t + 1 and t + 2 are in flight.
  // A tile's page ids are loaded with it and looked at only when it is scored, so
  // that no wait for its loads is placed at the fetch.
  float4 kb0[NV], kb1[NV], kb2[NV];
  int pg0 = -1, pg1 = -1, pg2 = -1;
  // Loads are unconditional (rows past the wave's share read a valid row, whose
  // scores are then not candidates): no branch around them, so the compiler's
  // waits count the loads still in flight instead of draining them all.
  auto fetch = [&](int b0, float4 (&dst)[NV], int& page) {
    const int b = min(b0 + col, nb - 1);
#pragma unroll
    for (int u = 0; u < NV; ++u)
      dst[u] = *reinterpret_cast<const float4*>(kh + static_cast<int64_t>(b) * D + 16 * u + 4 * j);
    page = table ? table[b] : 0;
  };
  // scores of the tile in kv (block b0 + col), four independent MFMA chains
  auto score_tile = [&](int b0, const float4 (&kv)[NV], int page) {
    const int b = b0 + col;
    const bool live = b < bw1 && b < first_excluded && page >= 0 && (table == nullptr || page < num_pages);
    f32x4 acc[4] = {};
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[4 * u + 0], kv[u].x, acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[4 * u + 1], kv[u].y, acc[1], 0, 0, 0);
      acc[2] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[4 * u + 2], kv[u].z, acc[2], 0, 0, 0);
      acc[3] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[4 * u + 3], kv[u].w, acc[3], 0, 0, 0);
    }
    // acc: block b0 + col against groups g0 + 4 j + i
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float dot = (acc[0][i] + acc[1][i]) + (acc[2][i] + acc[3][i]);
      insert(lk[i], li[i], live ? score_key(scale * dot) : 0u, b0 + col);
    }
  };
  fetch(bw0, kb0, pg0);
  fetch(bw0 + 16, kb1, pg1);
  for (int b0 = bw0; b0 < bw1; b0 += 48) {
    fetch(b0 + 32, kb2, pg2);
    score_tile(b0, kb0, pg0);
    if (b0 + 16 >= bw1) break;
    fetch(b0 + 48, kb0, pg0);
    score_tile(b0 + 16, kb1, pg1);
    if (b0 + 32 >= bw1) break;
    fetch(b0 + 64, kb1, pg1);
    score_tile(b0 + 32, kb2, pg2);
  }

  // every lane's lists to LDS, per group: candidate (wave, col, t) of group 4 j + i
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < KM; ++t)
      cand[4 * j + i][(wave * 16 + col) * KM + t] =
          lk[i][t] == 0u ? 0ull
                         : (static_cast<uint64_t>(lk[i][t]) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(li[i][t]));
  __syncthreads();

  // half-wave (32 lanes) per group: each lane keeps the KM best of its share of the
  // group's NW * 16 * KM candidates, then K rounds of a 32-lane maximum name the
  // winners (the largest (key, lower id) composite), written in ascending id order
  constexpr int kPerLane = NW * 16 * KM / 32;
  const int half = lane / 32, l32 = lane % 32;
  for (int m = 2 * wave + half; m < kStkGroups; m += 2 * NW) {
    uint64_t top[KM];
#pragma unroll
    for (int t = 0; t < KM; ++t) top[t] = 0ull;
#pragma unroll
    for (int c = 0; c < kPerLane; ++c) {
      uint64_t v = cand[m][l32 + 32 * c];
      if (v > top[KM - 1]) {
#pragma unroll
        for (int t = 0; t < KM; ++t) {  // insertion into the descending list
          const uint64_t hi = top[t] > v ? top[t] : v, lo = top[t] > v ? v : top[t];
          top[t] = hi;
          v = lo;
        }
      }
    }
    uint64_t win = 0ull;
    int taken = 0;
    for (int r = 0; r < K; ++r) {
      uint64_t best = top[0];
#pragma unroll
      for (int off = 16; off >= 1; off >>= 1) {
        const uint64_t o = __shfl_xor(best, off);
        best = o > best ? o : best;
      }
      if (best == 0ull) break;  // fewer than K candidates (uniform within the half)
      if (top[0] == best) {
#pragma unroll
        for (int t = 0; t + 1 < KM; ++t) top[t] = top[t + 1];
        top[KM - 1] = 0ull;
      }
      if (l32 == r) win = best;
      ++taken;
    }
    const int g = g0 + m;
    if (g < R) {
      const int id = static_cast<int>(~static_cast<uint32_t>(win));
      int rank = 0;
      for (int s2 = 0; s2 < taken; ++s2) rank += __shfl(id, half * 32 + s2) < id;
      const int64_t row = static_cast<int64_t>(h) * R + g;
      if (l32 < taken) {
        idx[row * K + rank] = id;
        if (score_out) score_out[row * K + rank] = key_score(static_cast<uint32_t>(win >> 32));
      } else if (l32 < K) {
        idx[row * K + l32] = -1;
        if (score_out) score_out[row * K + l32] = -INFINITY;
      }
      if (l32 == 0) cnt[row] = taken;
    }
  }
}

// Top-K for rows longer than the register-resident kernel holds: one wavefront,
// keys re-read at every step of a plain bisection.
__global__ __launch_bounds__(kWave) void k_topk_wide(const uint32_t* __restrict__ keys, int nb, int nbp, int K,
                                                     int32_t* __restrict__ idx, int32_t* __restrict__ cnt,
                                                     float* __restrict__ score_out) {
  const int lane = threadIdx.x;
  const int64_t row = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  const uint32_t* kp = keys + row * nbp;
  int ncand = 0;
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  for (int b = lane; b < nb; b += kWave) {
    const uint32_t k = kp[b];
    if (k != 0u) {
      ++ncand;
      kmin = min(kmin, k);
      kmax = max(kmax, k);
    }
  }
  ncand = __reduce_add_sync(~0ull, ncand);
  kmin = __reduce_min_sync(~0ull, kmin);
  kmax = __reduce_max_sync(~0ull, kmax);
  auto count_ge = [&](uint32_t th, bool strict) -> int {
    int c = 0;
    for (int b = lane; b < nb; b += kWave) c += strict ? kp[b] > th : kp[b] >= th;
    return __reduce_add_sync(~0ull, c);
  };
  const bool all = ncand <= K;
  uint32_t kth = 0u;
  int need = 0;
  if (!all) {
    uint32_t lo = kmin, hi = kmax;
    while (lo < hi) {
      const uint32_t mid = lo + (hi - lo) / 2 + 1;
      if (count_ge(mid, false) >= K) lo = mid; else hi = mid - 1;
    }
    kth = lo;
    need = K - count_ge(kth, true);
  }
  int32_t* out_idx = idx + row * K;
  float* out_score = score_out ? score_out + row * K : nullptr;
  int pos = 0, eq_run = 0;
  for (int b0 = 0; b0 < nb; b0 += kWave) {
    const int b = b0 + lane;
    const uint32_t k = b < nb ? kp[b] : 0u;
    const bool tie = !all && k == kth;
    const uint64_t tie_mask = __ballot(tie);
    const bool take = k > kth || (tie && eq_run + lane_rank(tie_mask) < need);
    const uint64_t take_mask = __ballot(take);
    const int at = pos + lane_rank(take_mask);
    if (take && at < K) {
      out_idx[at] = b;
      if (out_score) out_score[at] = key_score(k);
    }
    pos += __popcll(take_mask);
    eq_run += __popcll(tie_mask);
  }
  const int total = all ? ncand : K;
  for (int i = total + lane; i < K; i += kWave) {
    out_idx[i] = -1;
    if (out_score) out_score[i] = -INFINITY;
  }
  if (lane == 0) cnt[row] = total < K ? total : K;
}

template <int D>
hipError_t launch_score(const CacheGeom& g, const SelectPlan& p, const float* kbar, int64_t kbar_stride,
                        const float* qpart, int nbp, uint32_t* keys, hipStream_t stream) {
  if (p.R <= kInlineGroups) {
    const int waves = (g.nb + kScoreRowsPerWave - 1) / kScoreRowsPerWave;
    const dim3 grid((waves + kThreads / kWave - 1) / (kThreads / kWave), g.H);
    if (p.R == 1)
      return launch_kernel(k_score_rows<D, 1>, grid, dim3(kThreads), 0, stream, kbar, kbar_stride, qpart, p.qsplit,
                           p.lq, p.G, g.page_table, g.pt_stride, g.num_pages, g.nb, nbp, p.first_excluded, p.R, p.scale, keys);
    return launch_kernel(k_score_rows<D, kInlineGroups>, grid, dim3(kThreads), 0, stream, kbar, kbar_stride, qpart,
                         p.qsplit, p.lq, p.G, g.page_table, g.pt_stride, g.num_pages, g.nb, nbp, p.first_excluded, p.R, p.scale,
                         keys);
  }
  if (p.R >= kScoreTiledMinGroups) {
    const dim3 grid((g.nb + 63) / 64, (p.R + 63) / 64, g.H);
    return launch_kernel(k_score_tiled<D>, grid, dim3(kThreads), 0, stream, kbar, kbar_stride, qpart, p.qsplit, p.lq,
                         p.G, g.page_table, g.pt_stride, g.num_pages, g.nb, nbp, p.first_excluded, p.R, p.scale, keys);
  }
  const dim3 grid((g.nb + 63) / 64, (p.R + 15) / 16, g.H);
  return launch_kernel(k_score<D>, grid, dim3(kThreads), 0, stream, kbar, kbar_stride, qpart, p.qsplit, p.lq, p.G,
                       g.page_table, g.pt_stride, g.num_pages, g.nb, nbp, p.first_excluded, p.R, p.scale, keys);
}

// Proxy-query partial sums: two 512-thread workgroups per 512-row split (one per
// half of d), or one wave per group when groups hold at most kQSmallRows rows (one
// split each).
template <typename T, int D>
hipError_t launch_qmean(const SelectPlan& p, const CacheGeom& g, const T* q, float* qpart, hipStream_t stream) {
  if (p.G <= kQSmallRows)
    return launch_kernel(k_qmean_partial<T, D, kQSmallThreads, 1>, dim3(p.qsplit, p.R, g.H), dim3(kQSmallThreads), 0,
                         stream, q, p.lq, g.H, p.G, p.R, p.qsplit, qpart);
  return launch_kernel(k_qmean_partial<T, D, kQThreads, kQColSplits>, dim3(p.qsplit * kQColSplits, p.R, g.H),
                       dim3(kQThreads), 0, stream, q, p.lq, g.H, p.G, p.R, p.qsplit, qpart);
}

hipError_t launch_topk(const CacheGeom& g, const SelectPlan& p, const uint32_t* keys, int nbp, int32_t* idx,
                       int32_t* cnt, float* score, hipStream_t stream) {
  const dim3 tgrid(p.R, g.H);
  // small K: one wave per row
  const int rows = p.R * g.H;
  const dim3 sgrid((rows + kTopkSmallWaves - 1) / kTopkSmallWaves);
  if (p.K <= 4)
    return launch_kernel(k_topk_small<4>, sgrid, dim3(kTopkSmallWaves * kWave), 0, stream, keys, rows, g.nb, nbp, p.K,
                         idx, cnt, score);
  if (p.K <= kTopkSmallK)
    return launch_kernel(k_topk_small<kTopkSmallK>, sgrid, dim3(kTopkSmallWaves * kWave), 0, stream, keys, rows, g.nb,
                         nbp, p.K, idx, cnt, score);
  // 512 threads hold rows of up to 16384 keys in registers (32 per lane), 1024 twice
  // that; with many rows (small query groups) 256-thread workgroups pack more rows
  // per CU
  if (p.R * g.H >= kTopkManyRows && g.nb <= 256 * 4 * kTopkVecPerLane)
    return launch_kernel(k_topk<256>, tgrid, dim3(256), 0, stream, keys, g.nb, nbp, p.K, idx, cnt, score);
  if (g.nb <= 512 * 4 * kTopkVecPerLane)
    return launch_kernel(k_topk<512>, tgrid, dim3(512), 0, stream, keys, g.nb, nbp, p.K, idx, cnt, score);
  if (g.nb <= kTopkRegMax)
    return launch_kernel(k_topk<1024>, tgrid, dim3(1024), 0, stream, keys, g.nb, nbp, p.K, idx, cnt, score);
  return launch_kernel(k_topk_wide, tgrid, dim3(kWave), 0, stream, keys, g.nb, nbp, p.K, idx, cnt, score);
}

// Many groups and small K: the scores and their top-K in one kernel.
bool fused_score_topk(const SelectPlan& p) { return p.K <= kTopkSmallK && p.R >= kScoreTiledMinGroups; }

template <int D>
hipError_t launch_score_topk(const CacheGeom& g, const SelectPlan& p, const float* kbar, int64_t kbar_stride,
                             const float* qpart, int32_t* idx, int32_t* cnt, float* score, hipStream_t stream) {
  // eight waves (two per SIMD) for K <= 4; the longer lists of K <= 16 take four
  const dim3 grid((p.R + kStkGroups - 1) / kStkGroups * g.H);
  if (p.K <= 4)
    return launch_kernel(k_score_topk<D, 4, 8>, grid, dim3(8 * kWave), 0, stream, kbar, kbar_stride, qpart, p.qsplit,
                         p.lq, p.G, g.page_table, g.pt_stride, g.num_pages, g.nb, p.first_excluded, p.R, p.scale, p.K,
                         idx, cnt, score);
  return launch_kernel(k_score_topk<D, kTopkSmallK, 4>, grid, dim3(4 * kWave), 0, stream, kbar, kbar_stride, qpart,
                       p.qsplit, p.lq, p.G, g.page_table, g.pt_stride, g.num_pages, g.nb, p.first_excluded, p.R,
                       p.scale, p.K, idx, cnt, score);
}

template <typename T, int D>
hipError_t launch_select_typed(const CacheGeom& g, const SelectPlan& p, const void* q, int32_t* idx, int32_t* cnt,
                               float* score, void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  float* qpart = reinterpret_cast<float*>(ws + p.off_qpart);
  float* kbar = reinterpret_cast<float*>(ws + p.off_kbar);
  uint32_t* keys = reinterpret_cast<uint32_t*>(ws + p.off_keys);
  const int nbp = (g.nb + 3) / 4 * 4;

  LaunchStatus st;
  st.add(launch_qmean<T, D>(p, g, static_cast<const T*>(q), qpart, stream));
  if (g.nb > 0) {
    PoolArgs a;
    a.k_pages = g.k_pages;
    a.page_table = g.page_table;
    a.pt_stride = g.pt_stride;
    a.num_pages = g.num_pages;
    a.H = g.H;
    a.S = g.S;
    a.Bpc = g.Bpc;
    a.nb = g.nb;
    a.first_excluded = p.first_excluded;
    a.qpart = qpart;
    a.nsplit = p.qsplit;
    a.lq = p.lq;
    a.G = p.G;
    a.R = p.R;
    a.scale = p.scale;
    a.keys = keys;
    a.nbp = nbp;
    a.kbar = kbar;
    a.blocks_per_wave = kPoolBlocksPerWave;
    const int waves = (g.nb + a.blocks_per_wave - 1) / a.blocks_per_wave;
    const dim3 grid((waves + kThreads / kWave - 1) / (kThreads / kWave), g.H);
    auto pool = [&](auto kernel) { st(kernel, grid, dim3(kThreads), 0, stream, a); };
    if (g.B == 64) {
      if (!p.inline_scores) pool(k_pool_score<T, D, 64, 0>);
      else if (p.R == 1) pool(k_pool_score<T, D, 64, 1>);
      else pool(k_pool_score<T, D, 64, kInlineGroups>);
    } else {
      if (!p.inline_scores) pool(k_pool_score<T, D, 128, 0>);
      else if (p.R == 1) pool(k_pool_score<T, D, 128, 1>);
      else pool(k_pool_score<T, D, 128, kInlineGroups>);
    }
    if (!p.inline_scores && st.err == hipSuccess) {
      if (fused_score_topk(p))
        return launch_score_topk<D>(g, p, kbar, static_cast<int64_t>(g.nb), qpart, idx, cnt, score, stream);
      st.add(launch_score<D>(g, p, kbar, static_cast<int64_t>(g.nb), qpart, nbp, keys, stream));
    }
  }
  if (st.err != hipSuccess) return st.err;
  return launch_topk(g, p, keys, nbp, idx, cnt, score, stream);
}

}  // namespace

template <typename T, int D>
hipError_t launch_compress_typed(const CacheGeom& g, const CmpCache& cc, int chunk, hipStream_t stream) {
  CompressArgs a;
  a.k_pages = g.k_pages;
  a.v_pages = g.v_pages;
  a.page_table = g.page_table;
  a.pt_stride = g.pt_stride;
  a.num_pages = g.num_pages;
  a.H = g.H;
  a.S = g.S;
  a.Bpc = g.Bpc;
  a.chunk = chunk;
  a.k_mean = cc.k_mean;
  a.ck_pages = cc.k_pages;
  a.cv_pages = cc.v_pages;
  a.ck_lo = cc.k_lo;
  a.c_page_table = cc.page_table;
  a.cap_blocks = cc.cap_blocks;
  const dim3 grid((g.Bpc + kThreads / kWave - 1) / (kThreads / kWave), g.H);
  if (g.B == 64) return launch_kernel(k_compress_chunk<T, D, 64>, grid, dim3(kThreads), 0, stream, a);
  return launch_kernel(k_compress_chunk<T, D, 128>, grid, dim3(kThreads), 0, stream, a);
}

template <typename T, int D>
hipError_t launch_select_compressed_typed(const CacheGeom& g, const CmpCache& cc, const SelectPlan& p, const void* q,
                                          int32_t* idx, int32_t* cnt, float* score, void* workspace,
                                          hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  float* qpart = reinterpret_cast<float*>(ws + p.off_qpart);
  uint32_t* keys = reinterpret_cast<uint32_t*>(ws + p.off_keys);
  const int nbp = (g.nb + 3) / 4 * 4;
  if (p.score_mode == 1) {
    if (g.nb > 0) {
      float* part = reinterpret_cast<float*>(ws + p.off_part);
      const hipError_t e = launch_prob_keys(g, p, q, cc.k_mean, static_cast<int64_t>(cc.cap_blocks), part,
                                            ws + p.off_ksplit, cc.k_lo != nullptr ? cc.k_pages : nullptr, cc.k_lo,
                                            keys, nbp, stream);
      if (e != hipSuccess) return e;
    }
    return launch_topk(g, p, keys, nbp, idx, cnt, score, stream);
  }
  hipError_t e = launch_qmean<T, D>(p, g, static_cast<const T*>(q), qpart, stream);
  if (e == hipSuccess && g.nb > 0 && fused_score_topk(p))
    return launch_score_topk<D>(g, p, cc.k_mean, static_cast<int64_t>(cc.cap_blocks), qpart, idx, cnt, score, stream);
  if (e == hipSuccess && g.nb > 0)
    e = launch_score<D>(g, p, cc.k_mean, static_cast<int64_t>(cc.cap_blocks), qpart, nbp, keys, stream);
  if (e != hipSuccess) return e;
  return launch_topk(g, p, keys, nbp, idx, cnt, score, stream);
}

hipError_t launch_compress_chunk(const CacheGeom& g, const CmpCache& cc, int chunk, hipStream_t stream) {
  if (g.dtype == 0) {
    if (g.D == 128) return launch_compress_typed<uint16_t, 128>(g, cc, chunk, stream);
    return launch_compress_typed<uint16_t, 64>(g, cc, chunk, stream);
  }
  if (g.D == 128) return launch_compress_typed<float, 128>(g, cc, chunk, stream);
  return launch_compress_typed<float, 64>(g, cc, chunk, stream);
}

hipError_t launch_select_compressed(const CacheGeom& g, const CmpCache& cc, const SelectPlan& p, const void* q,
                                    int32_t* idx, int32_t* cnt, float* score, void* workspace, hipStream_t stream) {
  if (g.dtype == 0) {
    if (g.D == 128) return launch_select_compressed_typed<uint16_t, 128>(g, cc, p, q, idx, cnt, score, workspace, stream);
    return launch_select_compressed_typed<uint16_t, 64>(g, cc, p, q, idx, cnt, score, workspace, stream);
  }
  if (g.D == 128) return launch_select_compressed_typed<float, 128>(g, cc, p, q, idx, cnt, score, workspace, stream);
  return launch_select_compressed_typed<float, 64>(g, cc, p, q, idx, cnt, score, workspace, stream);
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
