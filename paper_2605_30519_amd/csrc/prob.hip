// prob.hip -- the probability-averaged compression score (Sec. 3.1, Eq. 3; App. C)
// for gfx950.  For every head h and query group r:
//   u[i][b]    = scale * <q_i, kbar[h][b]>                       every pooled key b
//   sbar[r][b] = (1/|G_r|) sum over rows i of group r of exp(u[i][b] - LSE_i)
// with LSE_i the log-sum-exp of row i over all pooled keys, so that sbar is the
// group mean of the compression branch's attention weights.
//
// The fp32 pooled keys enter the MFMAs as two bf16 pieces (kbar ~= hi + lo, exact to
// about 2^-17 relative, both rounded to nearest even).  With a bf16 compressed cache
// that keeps the residual, the pieces are its pooled-key pages and residual pages,
// written once per chunk when the chunk is pooled; otherwise k_split_keys splits the
// fp32 pooled keys once per call, tile by tile (64 keys, hi then lo).  Either way a
// workgroup stages a tile with plain coalesced 16-byte loads.
// k_prob_partial: one workgroup per (head, slice of at most 128 query rows), the
// slices of one head contiguous on one XCD so that its L2 holds that head's keys.
// Each wave owns 64 rows (two 32-row MFMA tiles that share every key fragment) and
// 32 keys of each tile; a slice that is part of one group double-buffers the key
// tiles in LDS (one barrier per tile), a slice of whole groups stages each tile
// between two barriers, its LDS holding the probability tile that it reduces per
// group.  The workgroup walks the tiles twice: first for each row's LSE
// (online, exp2 domain, the hardware exp2: probabilities below 2^-126 count as 0),
// then for exp(u - LSE) summed over the rows of each group segment of the slice.  The products are bf16 MFMA (32x32x16) with fp32
// accumulation: hi*q + lo*q for bf16 queries (exact), plus hi*q_lo for fp32 queries
// split the same way.  The first pass forms S^T = K Q^T (a lane owns one query
// row: its max and sum stay in the lane), the second S = Q K^T (a lane owns one
// key: the sum over a group's rows is a sum over the lane's accumulator rows).
// The group means become the order-preserving keys that k_topk ranks (0 outside
// Omega): written by k_prob_partial when its slice holds whole groups, else by
// k_prob_merge, which sums a group's slices in a fixed order.
#include <math.h>

#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

constexpr int kPThreads = 256;
constexpr int kPRows = kProbSliceRows;  // query rows per slice: 64 per wave, two waves deep
static_assert(kPRows == 128, "the wave layout assumes 128-row slices");
constexpr int kPKeys = 64;    // pooled keys per tile: 32 per wave, two waves wide
static_assert(kPKeys == kCmpPageTokens, "a key tile is one page of the compressed cache");
constexpr int kPRedStride = kPKeys + 1;
constexpr float kLog2eP = 1.4426950408889634f;

template <typename T>
struct QueryPieces;  // bf16 pieces per query element
template <>
struct QueryPieces<uint16_t> {
  static constexpr int N = 1;
};
template <>
struct QueryPieces<float> {
  static constexpr int N = 2;
};

struct ProbArgs {
  const void* q;
  int lq, H, G, R;
  // bf16 pieces of the pooled keys, 64-key tiles of [64][D]: piece p of tile t of
  // head h starts at piece[p] + t * tile_stride + h * head_stride (16-byte units)
  const uint4* piece[2];
  int64_t tile_stride, head_stride;
  int ntiles, nb;
  float scale;
  int multi;            // 1: a slice holds gps whole groups; 0: a slice is part of one group
  int gps, spg, slices, nseg;
  float* part;          // [H][nseg][nb] (parts of groups)
  // whole-group slices write the ranking keys themselves
  uint32_t* keys;       // [H][R][nbp]
  int nbp, first_excluded;
  const int32_t* page_table;
  int64_t pt_stride;
  int64_t num_pages;
};

// Merges two (max, sum) states of a log-sum-exp; maxima in raw units, sums of
// exp2(c2 * (x - max)).
__device__ __forceinline__ void lse_merge(float& m, float& l, float m2, float l2, float c2) {
  const float mx = fmaxf(m, m2);
  if (mx == -INFINITY) {
    m = mx;
    l = 0.f;
    return;
  }
  l = l * exp2f(c2 * (m - mx)) + l2 * exp2f(c2 * (m2 - mx));
  m = mx;
}

// 8 fp32 values -> bf16 hi and lo pieces (x ~= hi + lo), packed as MFMA operands;
// both roundings to nearest even (the hardware conversion).
__device__ __forceinline__ void split8(const float (&x)[8], uint4& hi, uint4& lo) {
  bf16x8 h, l;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    h[e] = static_cast<__bf16>(x[e]);
    l[e] = static_cast<__bf16>(x[e] - static_cast<float>(h[e]));
  }
  hi = __builtin_bit_cast(uint4, h);
  lo = __builtin_bit_cast(uint4, l);
}

// One workgroup per (tile of 64 keys, head); keys past nb are zero.  Every load of
// a thread is in flight before the first split.
template <int D>
__global__ __launch_bounds__(kPThreads) void k_split_keys(const float* __restrict__ kbar, int64_t kbar_stride, int nb,
                                                          int ntiles, uint4* __restrict__ ksplit) {
  constexpr int CH = D / 8;
  constexpr int PER = kPKeys * CH / kPThreads;  // 8-element chunks per thread
  static_assert(PER * kPThreads == kPKeys * CH, "whole chunks per thread");
  const int t = blockIdx.x, h = blockIdx.y;
  uint4* dst = ksplit + (static_cast<int64_t>(h) * ntiles + t) * (2 * kPKeys * CH);
  float4 x0[PER], x1[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + u * kPThreads, row = e / CH, c = e % CH, b = t * kPKeys + row;
    x0[u] = x1[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (b < nb) {
      const float* src = kbar + (static_cast<int64_t>(h) * kbar_stride + b) * D + 8 * c;
      x0[u] = *reinterpret_cast<const float4*>(src);
      x1[u] = *reinterpret_cast<const float4*>(src + 4);
    }
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + u * kPThreads;
    const float x[8] = {x0[u].x, x0[u].y, x0[u].z, x0[u].w, x1[u].x, x1[u].y, x1[u].z, x1[u].w};
    uint4 hi, lo;
    split8(x, hi, lo);
    dst[e] = hi;
    dst[kPKeys * CH + e] = lo;
  }
}

// Split-key tiles: 16-byte chunk e of tile t (piece e / (64 CH), key row, chunk c)
// is fetched by thread e mod 256 and goes to chunk c ^ (row mod CH) of its LDS
// row, so that the fragment reads of 8 consecutive rows hit 8 different chunk
// columns.
template <int D>
__device__ __forceinline__ void fetch_tile(const ProbArgs& a, int h, int t, u32x4 (&kv)[2 * kPKeys * D / 8 / kPThreads]) {
  constexpr int PIECE_CHUNKS = kPKeys * D / 8;
  static_assert(PIECE_CHUNKS % kPThreads == 0, "a thread's chunks of a tile lie in one piece each");
  const int64_t off = t * a.tile_stride + h * a.head_stride;
#pragma unroll
  for (int u = 0; u < 2 * PIECE_CHUNKS / kPThreads; ++u) {
    const int e = threadIdx.x + u * kPThreads, piece = e / PIECE_CHUNKS;  // piece: compile-time per u
    kv[u] = reinterpret_cast<const u32x4*>(a.piece[piece])[off + e % PIECE_CHUNKS];
  }
}

template <int D>
__device__ __forceinline__ void stage_tile(const u32x4 (&kv)[2 * kPKeys * D / 8 / kPThreads], uint16_t* ktile) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int u = 0; u < 2 * kPKeys * CH / kPThreads; ++u) {
    const int e = threadIdx.x + u * kPThreads, piece = e / (kPKeys * CH), rem = e % (kPKeys * CH);
    const int row = rem / CH, c = rem % CH;
    *reinterpret_cast<u32x4*>(ktile + piece * kPKeys * D + row * D + 8 * (c ^ (row % CH))) = kv[u];
  }
}

// The 8 bf16 of key row krow, d = 16 kk + 8 half + 0..7, of one piece (0 hi, 1 lo).
template <int D>
__device__ __forceinline__ bf16x8 key_frag(const uint16_t* ktile, int piece, int kk, int krow, int half) {
  constexpr int CH = D / 8;
  const int pc = (2 * kk + half) ^ (krow % CH);
  return *reinterpret_cast<const bf16x8*>(ktile + piece * kPKeys * D + krow * D + 8 * pc);
}

// MULTI: the slice holds whole groups, and a 128 x 64 probability tile is reduced
// through LDS; the key tile then has one LDS buffer, staged between two barriers.
// Otherwise the slice is part of one group: two key-tile buffers, tile t + 1
// staged right after tile t's MFMAs, one barrier per tile.
template <typename T, int D, bool MULTI>
__global__ __launch_bounds__(kPThreads, 2) void k_prob_partial(ProbArgs a) {
  constexpr int KK = D / 16;                      // MFMA steps over d
  constexpr int CH = D / 8;                       // 16-byte chunks per key row
  constexpr int LPT = 2 * kPKeys * CH / kPThreads;  // 16-byte loads per thread per tile
  constexpr int QP = QueryPieces<T>::N;
  constexpr int NBUF = MULTI ? 1 : 2;
  constexpr int TILE = 2 * kPKeys * D;            // bf16 elements of one split tile
  __shared__ __align__(16) uint16_t ktile[NBUF * TILE];
  // MULTI: the probability tile; else two buffers of the two row halves' key sums
  __shared__ float red[MULTI ? kPRows * kPRedStride : 2 * 2 * kPKeys];
  __shared__ float mrg_m[2][kPRows], mrg_l[2][kPRows];
  __shared__ float lse2[kPRows];

  const int id = xcd_contiguous_id(blockIdx.x, gridDim.x);
  const int h = id / a.slices, slice = id % a.slices;
  int row0, rows, seg0;
  if constexpr (MULTI) {
    seg0 = slice * a.gps;
    row0 = seg0 * a.G;
    rows = min(a.gps * a.G, a.lq - row0);
  } else {
    const int r = slice / a.spg, k = slice % a.spg;
    seg0 = slice;
    row0 = r * a.G + k * kPRows;
    rows = min(kPRows, min(r * a.G + a.G, a.lq) - row0);
  }
  if (rows <= 0) return;  // workgroup-uniform, before any barrier

  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave, half = lane / 32;
  const int rh = wave & 1, kq = wave >> 1;  // rows [64 rh, +64) of the slice, keys [32 kq, +32) of a tile
  const int krow = 32 * kq + lane % 32;     // tile-local key this lane supplies

  // query operands of the wave's two 32-row tiles: row 64 rh + 32 s + lane%32,
  // d = 16 kk + 8 half + 0..7 (zero past the slice)
  bf16x8 qh[2][KK], ql[2][KK];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int qrow = 64 * rh + 32 * s + lane % 32;
    const bool live = qrow < rows;
    const int64_t base = (static_cast<int64_t>(row0 + qrow) * a.H + h) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      uint4 hi = make_uint4(0, 0, 0, 0), lo = make_uint4(0, 0, 0, 0);
      if constexpr (QP == 1) {
        if (live) hi = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.q) + base + 16 * kk + 8 * half);
      } else {
        if (live) {
          const float* src = static_cast<const float*>(a.q) + base + 16 * kk + 8 * half;
          const float4 x0 = *reinterpret_cast<const float4*>(src), x1 = *reinterpret_cast<const float4*>(src + 4);
          const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
          split8(x, hi, lo);
        }
      }
      qh[s][kk] = __builtin_bit_cast(bf16x8, hi);
      ql[s][kk] = __builtin_bit_cast(bf16x8, lo);
    }
  }

  u32x4 kv[LPT];
  const float c2 = a.scale * kLog2eP;

  // ---- pass 1: LSE of every row over all pooled keys (S^T = K Q^T, lane = row)
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
  fetch_tile<D>(a, h, 0, kv);
  if constexpr (NBUF == 2) {
    stage_tile<D>(kv, ktile);
    __syncthreads();
    if (a.ntiles > 1) fetch_tile<D>(a, h, 1, kv);
  }
  for (int t = 0; t < a.ntiles; ++t) {
    const uint16_t* kt = ktile + (NBUF == 2 ? (t & 1) * TILE : 0);
    if constexpr (NBUF == 1) {
      __syncthreads();
      stage_tile<D>(kv, ktile);
      __syncthreads();
      if (t + 1 < a.ntiles) fetch_tile<D>(a, h, t + 1, kv);
    }
    f32x16 acc[2] = {};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8 kh = key_frag<D>(kt, 0, kk, krow, half), kl = key_frag<D>(kt, 1, kk, krow, half);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, qh[s][kk], acc[s], 0, 0, 0);
        acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kl, qh[s][kk], acc[s], 0, 0, 0);
        if constexpr (QP == 2) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, ql[s][kk], acc[s], 0, 0, 0);
      }
    }
    // acc[s][i]: key t*64 + 32 kq + 8 (i/4) + 4 half + i%4 against row 64 rh + 32 s + lane%32;
    // the running max is kept in raw (unscaled) units, scale > 0
    if (t * kPKeys + kPKeys > a.nb) {  // workgroup-uniform: only the last tile is partial
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int b = t * kPKeys + 32 * kq + 8 * (i / 4) + 4 * half + i % 4;
        if (b >= a.nb) acc[0][i] = acc[1][i] = -INFINITY;
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float mx = acc[s][0];
#pragma unroll
      for (int i = 1; i < 16; ++i) mx = fmaxf(mx, acc[s][i]);
      if (mx > -INFINITY) {
        const float mnew = fmaxf(m_run[s], mx), off = -c2 * mnew;
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) sum += __builtin_amdgcn_exp2f(fmaf(acc[s][i], c2, off));
        l_run[s] = l_run[s] * __builtin_amdgcn_exp2f(c2 * (m_run[s] - mnew)) + sum;
        m_run[s] = mnew;
      }
    }
    if constexpr (NBUF == 2) {
      if (t + 1 < a.ntiles) stage_tile<D>(kv, ktile + ((t + 1) & 1) * TILE);
      __syncthreads();
      if (t + 2 < a.ntiles) fetch_tile<D>(a, h, t + 2, kv);
    }
  }
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    lse_merge(m_run[s], l_run[s], __shfl_xor(m_run[s], 32), __shfl_xor(l_run[s], 32), c2);
    if (half == 0) {
      mrg_m[kq][64 * rh + 32 * s + lane % 32] = m_run[s];
      mrg_l[kq][64 * rh + 32 * s + lane % 32] = l_run[s];
    }
  }
  __syncthreads();
  if (tid < kPRows) {
    float m = mrg_m[0][tid], l = mrg_l[0][tid];
    lse_merge(m, l, mrg_m[1][tid], mrg_l[1][tid], c2);
    lse2[tid] = tid < rows ? c2 * m + log2f(l) : INFINITY;  // log2 domain; rows past the slice weigh 0
  }
  __syncthreads();

  // ---- pass 2: exp(u - LSE) summed over each segment's rows (S = Q K^T, lane = key)
  float lr[2][16];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int i = 0; i < 16; ++i) lr[s][i] = lse2[64 * rh + 32 * s + 8 * (i / 4) + 4 * half + i % 4];
  const int ngroups = MULTI ? min(a.gps, a.R - seg0) : 1;
  float* const part_row = a.part + (static_cast<int64_t>(h) * a.nseg + seg0) * a.nb;
  fetch_tile<D>(a, h, 0, kv);
  if constexpr (NBUF == 2) {
    stage_tile<D>(kv, ktile);
    __syncthreads();
    if (a.ntiles > 1) fetch_tile<D>(a, h, 1, kv);
  }
  for (int t = 0; t < a.ntiles; ++t) {
    const uint16_t* kt = ktile + (NBUF == 2 ? (t & 1) * TILE : 0);
    if constexpr (NBUF == 1) {
      __syncthreads();
      stage_tile<D>(kv, ktile);
      __syncthreads();
      if (t + 1 < a.ntiles) fetch_tile<D>(a, h, t + 1, kv);
    }
    f32x16 acc[2] = {};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8 kh = key_frag<D>(kt, 0, kk, krow, half), kl = key_frag<D>(kt, 1, kk, krow, half);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qh[s][kk], kh, acc[s], 0, 0, 0);
        acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qh[s][kk], kl, acc[s], 0, 0, 0);
        if constexpr (QP == 2) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ql[s][kk], kh, acc[s], 0, 0, 0);
      }
    }
    // acc[s][i]: row 64 rh + 32 s + 8 (i/4) + 4 half + i%4 against key t*64 + krow
    const int b0 = t * kPKeys;
    if constexpr (!MULTI) {
      // the key sums of tile t go to buffer t & 1; those of tile t - 1, written
      // before the last barrier, are added and stored now
      float v = 0.f;
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i) v += __builtin_amdgcn_exp2f(fmaf(acc[s][i], c2, -lr[s][i]));
      v += __shfl_xor(v, 32);
      if (half == 0) red[(t & 1) * 2 * kPKeys + rh * kPKeys + krow] = v;
      if (t > 0 && tid < kPKeys && b0 - kPKeys + tid < a.nb) {
        const float* r = red + ((t - 1) & 1) * 2 * kPKeys;
        part_row[b0 - kPKeys + tid] = r[tid] + r[kPKeys + tid];
      }
    } else {
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          red[(64 * rh + 32 * s + 8 * (i / 4) + 4 * half + i % 4) * kPRedStride + krow] =
              __builtin_amdgcn_exp2f(fmaf(acc[s][i], c2, -lr[s][i]));
      __syncthreads();
      for (int e = tid; e < ngroups * kPKeys; e += kPThreads) {
        const int j = e / kPKeys, col = e % kPKeys;
        const int r_end = min(j * a.G + a.G, rows);
        float sum = 0.f;
        for (int r = j * a.G; r < r_end; ++r) sum += red[r * kPRedStride + col];
        const int b = b0 + col;
        if (b < a.nb) {
          const int32_t pg = a.page_table != nullptr ? a.page_table[static_cast<int64_t>(h) * a.pt_stride + b] : 0;
          const bool live = b < a.first_excluded && pg >= 0 && (a.page_table == nullptr || pg < a.num_pages);
          a.keys[(static_cast<int64_t>(h) * a.R + seg0 + j) * a.nbp + b] =
              live ? score_key(sum / static_cast<float>(r_end - j * a.G)) : 0u;
        }
      }
    }
    if constexpr (NBUF == 2) {
      if (t + 1 < a.ntiles) stage_tile<D>(kv, ktile + ((t + 1) & 1) * TILE);
      __syncthreads();
      if (t + 2 < a.ntiles) fetch_tile<D>(a, h, t + 2, kv);
    }
  }
  if constexpr (!MULTI) {  // the last tile's key sums, written before the loop's last barrier
    const int t = a.ntiles - 1, b = t * kPKeys + tid;
    if (tid < kPKeys && b < a.nb) {
      const float* r = red + (t & 1) * 2 * kPKeys;
      part_row[b] = r[tid] + r[kPKeys + tid];
    }
  }
}

// Slices that are parts of one group: the group's parts summed, four lanes per
// pooled key.  Lane j of a key adds parts j, j + 4, j + 8, ... in order, with every
// load in flight before its adds, and the four sums meet as (s0 + s1) + (s2 + s3):
// a fixed order, so the result does not depend on timing.
constexpr int kMergeLanes = 4;
__global__ __launch_bounds__(kPThreads) void k_prob_merge(const float* __restrict__ part, int nseg, int nb, int nbp,
                                                          int lq, int G, int R, int spg,
                                                          const int32_t* __restrict__ page_table, int64_t pt_stride,
                                                          int64_t num_pages,
                                                          int first_excluded, uint32_t* __restrict__ keys) {
  const int b = blockIdx.x * (kPThreads / kMergeLanes) + static_cast<int>(threadIdx.x) / kMergeLanes;
  const int j = static_cast<int>(threadIdx.x) % kMergeLanes, r = blockIdx.y, h = blockIdx.z;
  const int rows = min(r * G + G, lq) - r * G;
  const int parts = (rows + kPRows - 1) / kPRows;
  float s = 0.f;
  if (b < nb) {  // no return before the shuffles: every lane takes part in them
    constexpr int kBatch = 16;
    const float* src = part + (static_cast<int64_t>(h) * nseg + r * spg) * nb + b;
    for (int k0 = j; k0 < parts; k0 += kBatch * kMergeLanes) {
      float v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int k = k0 + kMergeLanes * u;
        v[u] = k < parts ? src[static_cast<int64_t>(k) * nb] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (k0 + kMergeLanes * u < parts) s += v[u];
    }
  }
  s += __shfl_xor(s, 1);
  s += __shfl_xor(s, 2);
  if (b >= nb || j != 0) return;
  s = s / static_cast<float>(rows);
  const int32_t p = page_table != nullptr ? page_table[static_cast<int64_t>(h) * pt_stride + b] : 0;
  const bool live = b < first_excluded && p >= 0 && (page_table == nullptr || p < num_pages);
  keys[(static_cast<int64_t>(h) * R + r) * nbp + b] = live ? score_key(s) : 0u;
}

template <typename T, int D>
hipError_t launch_prob_typed(const CacheGeom& g, const SelectPlan& p, const void* q, const float* kbar,
                             int64_t kbar_stride, float* part, uint4* ksplit, const uint4* hi_pages,
                             const uint4* lo_pages, uint32_t* keys, int nbp, hipStream_t stream) {
  const int ntiles = (g.nb + kPKeys - 1) / kPKeys;
  constexpr int64_t PIECE_CHUNKS = kPKeys * D / 8;
  LaunchStatus st;
  ProbArgs a;
  if (hi_pages != nullptr && lo_pages != nullptr) {
    // the compressed cache's pages: tile t of head h is page t's slab of head h
    a.piece[0] = hi_pages;
    a.piece[1] = lo_pages;
    a.tile_stride = static_cast<int64_t>(g.H) * PIECE_CHUNKS;
    a.head_stride = PIECE_CHUNKS;
  } else {
    st(k_split_keys<D>, dim3(ntiles, g.H), dim3(kPThreads), 0, stream, kbar, kbar_stride, g.nb, ntiles, ksplit);
    a.piece[0] = ksplit;
    a.piece[1] = ksplit + PIECE_CHUNKS;
    a.tile_stride = 2 * PIECE_CHUNKS;
    a.head_stride = ntiles * 2 * PIECE_CHUNKS;
  }
  a.q = q;
  a.lq = p.lq;
  a.H = g.H;
  a.G = p.G;
  a.R = p.R;
  a.ntiles = ntiles;
  a.nb = g.nb;
  a.scale = p.scale;
  a.multi = p.prob_multi ? 1 : 0;
  a.gps = p.prob_gps;
  a.spg = p.prob_spg;
  a.slices = p.prob_slices;
  a.nseg = p.prob_nseg;
  a.part = part;
  a.keys = keys;
  a.nbp = nbp;
  a.first_excluded = p.first_excluded;
  a.page_table = g.page_table;
  a.pt_stride = g.pt_stride;
  a.num_pages = g.num_pages;
  if (a.multi)
    st(k_prob_partial<T, D, true>, dim3(p.prob_slices * g.H), dim3(kPThreads), 0, stream, a);
  else
    st(k_prob_partial<T, D, false>, dim3(p.prob_slices * g.H), dim3(kPThreads), 0, stream, a);
  if (!a.multi) {
    constexpr int kMergeKeys = kPThreads / kMergeLanes;
    const dim3 mgrid((g.nb + kMergeKeys - 1) / kMergeKeys, p.R, g.H);
    st(k_prob_merge, mgrid, dim3(kPThreads), 0, stream, part, p.prob_nseg, g.nb, nbp, p.lq, p.G, p.R, p.prob_spg,
       g.page_table, g.pt_stride, g.num_pages, p.first_excluded, keys);
  }
  return st.err;
}

}  // namespace

hipError_t launch_prob_keys(const CacheGeom& g, const SelectPlan& p, const void* q, const float* kbar,
                            int64_t kbar_stride, float* part, void* ksplit, const void* hi_pages,
                            const void* lo_pages, uint32_t* keys, int nbp, hipStream_t stream) {
  uint4* ks = static_cast<uint4*>(ksplit);
  const uint4* hi = static_cast<const uint4*>(hi_pages);
  const uint4* lo = static_cast<const uint4*>(lo_pages);
  if (g.dtype == 0) {
    if (g.D == 128)
      return launch_prob_typed<uint16_t, 128>(g, p, q, kbar, kbar_stride, part, ks, hi, lo, keys, nbp, stream);
    return launch_prob_typed<uint16_t, 64>(g, p, q, kbar, kbar_stride, part, ks, hi, lo, keys, nbp, stream);
  }
  // fp32 caches: the pooled keys in k_pages are fp32, so the pieces are always split
  if (g.D == 128)
    return launch_prob_typed<float, 128>(g, p, q, kbar, kbar_stride, part, ks, nullptr, nullptr, keys, nbp, stream);
  return launch_prob_typed<float, 64>(g, p, q, kbar, kbar_stride, part, ks, nullptr, nullptr, keys, nbp, stream);
}

}  // namespace omnimem
