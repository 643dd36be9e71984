// prob.hip -- the probability-averaged compression score (Sec. 3.1, Eq. 3; App. C)
// for gfx950.  For every head h and query group r:
//   u[i][b]    = scale * <q_i, kbar[h][b]>                       every pooled key b
//   sbar[r][b] = (1/|G_r|) sum over rows i of group r of exp(u[i][b] - LSE_i)
// with LSE_i the log-sum-exp of row i over all pooled keys, so that sbar is the
// group mean of the compression branch's attention weights.
//
// k_prob_partial: one workgroup per (head, slice of at most 64 query rows).  It walks
// the pooled keys in tiles of 64 twice: first for each row's LSE (online, exp2
// domain), then for exp(u - LSE) summed over the rows of each group segment in the
// slice.  The products are bf16 MFMA (32x32x16) with fp32 accumulation; each fp32
// pooled key is split into two bf16 pieces (hi + lo, exact to about 2^-17), bf16
// queries are exact, fp32 queries are split the same way (hi*hi + lo*hi + hi*lo).
// The first pass forms S^T = K Q^T (a lane owns one query row: the row's max and sum
// stay in the lane), the second S = Q K^T (a lane owns one pooled key: the sum over
// a group's rows is a sum over the lane's accumulator rows).
// k_prob_merge: sums a group's slices in order, divides by the group's row count and
// writes the order-preserving keys that k_topk ranks (0 outside Omega).
#include <math.h>

#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

constexpr int kPThreads = 256;
constexpr int kPRows = 64;    // query rows per slice (two 32-row MFMA tiles)
constexpr int kPKeys = 64;    // pooled keys per tile (two 32-key MFMA tiles)
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
  const float* kbar;
  int64_t kbar_stride;  // pooled keys per head in kbar
  int nb;
  float scale;
  int multi;            // 1: a slice holds gps whole groups; 0: a slice is part of one group
  int gps, spg, nseg;
  float* part;          // [H][nseg][nb]
};

__device__ __forceinline__ void lse_merge(float& m, float& l, float m2, float l2) {
  const float mx = fmaxf(m, m2);
  if (mx == -INFINITY) {
    m = mx;
    l = 0.f;
    return;
  }
  l = l * exp2f(m - mx) + l2 * exp2f(m2 - mx);
  m = mx;
}

// 8 fp32 values -> bf16 hi and lo pieces (x ~= hi + lo), packed as MFMA operands.
__device__ __forceinline__ void split8(const float (&x)[8], uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint16_t h0 = f32_to_bf16_rne(x[2 * e]), h1 = f32_to_bf16_rne(x[2 * e + 1]);
    const uint16_t l0 = f32_to_bf16_rne(x[2 * e] - bf16_to_f32(h0));
    const uint16_t l1 = f32_to_bf16_rne(x[2 * e + 1] - bf16_to_f32(h1));
    h[e] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
    l[e] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

template <typename T, int D>
__global__ __launch_bounds__(kPThreads) void k_prob_partial(ProbArgs a) {
  constexpr int KK = D / 16;            // MFMA steps over d
  constexpr int CH = D / 8;             // 16-byte bf16 chunks per pooled key
  constexpr int CPT = CH / 4;           // chunks staged per thread (4 threads per key)
  constexpr int QP = QueryPieces<T>::N;
  __shared__ __align__(16) uint16_t khi[kPKeys * D];
  __shared__ __align__(16) uint16_t klo[kPKeys * D];
  __shared__ float red[kPRows * kPRedStride];
  __shared__ float mrg_m[2][kPRows], mrg_l[2][kPRows];
  __shared__ float lse2[kPRows];

  const int h = blockIdx.y, slice = blockIdx.x;
  int row0, rows, seg0;
  if (a.multi) {
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
  const int rq = wave & 1, kq = wave >> 1;  // this wave's 32 query rows and 32 pooled keys of a tile
  const int qrow = 32 * rq + lane % 32;     // slice-local query row this lane supplies
  const int krow = 32 * kq + lane % 32;     // tile-local pooled key this lane supplies

  // query operand: row qrow, d = 16 kk + 8 half + 0..7 (zero past the slice)
  bf16x8 qh[KK], ql[KK];
  {
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
      qh[kk] = __builtin_bit_cast(bf16x8, hi);
      ql[kk] = __builtin_bit_cast(bf16x8, lo);
    }
  }

  // pooled-key tile: thread tid stages key tid/4, dimensions [(tid%4) D/4, +D/4)
  float4 kv[2 * CPT];
  auto fetch = [&](int b0) {
    const int b = b0 + tid / 4;
    const float* src = a.kbar + (static_cast<int64_t>(h) * a.kbar_stride + b) * D + (tid % 4) * (D / 4);
#pragma unroll
    for (int u = 0; u < 2 * CPT; ++u)
      kv[u] = b < a.nb ? *reinterpret_cast<const float4*>(src + 4 * u) : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  // chunk c of key row r sits at chunk c ^ (r mod CH): the fragment reads of 8
  // consecutive rows hit 8 different chunk columns
  auto stage = [&]() {
    const int r = tid / 4;
#pragma unroll
    for (int cc = 0; cc < CPT; ++cc) {
      const float x[8] = {kv[2 * cc].x,     kv[2 * cc].y,     kv[2 * cc].z,     kv[2 * cc].w,
                          kv[2 * cc + 1].x, kv[2 * cc + 1].y, kv[2 * cc + 1].z, kv[2 * cc + 1].w};
      uint4 hi, lo;
      split8(x, hi, lo);
      const int c = (tid % 4) * CPT + cc, pc = c ^ (r % CH);
      *reinterpret_cast<uint4*>(khi + r * D + 8 * pc) = hi;
      *reinterpret_cast<uint4*>(klo + r * D + 8 * pc) = lo;
    }
  };
  auto frag = [&](const uint16_t* base, int kk) {
    const int pc = (2 * kk + half) ^ (krow % CH);
    return *reinterpret_cast<const bf16x8*>(base + krow * D + 8 * pc);
  };

  const float c2 = a.scale * kLog2eP;
  const int ntiles = (a.nb + kPKeys - 1) / kPKeys;

  // ---- pass 1: LSE of every row over all pooled keys (S^T = K Q^T, lane = row)
  float m_run = -INFINITY, l_run = 0.f;
  fetch(0);
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    stage();
    __syncthreads();
    if (t + 1 < ntiles) fetch((t + 1) * kPKeys);
    f32x16 acc = {};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8 kh = frag(khi, kk), kl = frag(klo, kk);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, qh[kk], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kl, qh[kk], acc, 0, 0, 0);
      if constexpr (QP == 2) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, ql[kk], acc, 0, 0, 0);
    }
    // acc[i]: pooled key t*64 + 32 kq + 8 (i/4) + 4 half + i%4 against row qrow
    float x[16], mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int b = t * kPKeys + 32 * kq + 8 * (i / 4) + 4 * half + i % 4;
      x[i] = b < a.nb ? c2 * acc[i] : -INFINITY;
      mx = fmaxf(mx, x[i]);
    }
    if (mx > -INFINITY) {
      const float mnew = fmaxf(m_run, mx);
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) s += exp2f(x[i] - mnew);
      l_run = l_run * exp2f(m_run - mnew) + s;
      m_run = mnew;
    }
  }
  lse_merge(m_run, l_run, __shfl_xor(m_run, 32), __shfl_xor(l_run, 32));
  if (half == 0) {
    mrg_m[kq][qrow] = m_run;
    mrg_l[kq][qrow] = l_run;
  }
  __syncthreads();
  if (tid < kPRows) {
    float m = mrg_m[0][tid], l = mrg_l[0][tid];
    lse_merge(m, l, mrg_m[1][tid], mrg_l[1][tid]);
    lse2[tid] = tid < rows ? m + log2f(l) : INFINITY;  // rows past the slice weigh 0
  }
  __syncthreads();

  // ---- pass 2: exp(u - LSE) summed over each segment's rows (S = Q K^T, lane = key)
  float lr[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) lr[i] = lse2[32 * rq + 8 * (i / 4) + 4 * half + i % 4];
  const int ngroups = a.multi ? min(a.gps, a.R - seg0) : 1;
  fetch(0);
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    stage();
    __syncthreads();
    if (t + 1 < ntiles) fetch((t + 1) * kPKeys);
    f32x16 acc = {};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8 kh = frag(khi, kk), kl = frag(klo, kk);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qh[kk], kh, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qh[kk], kl, acc, 0, 0, 0);
      if constexpr (QP == 2) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ql[kk], kh, acc, 0, 0, 0);
    }
    // acc[i]: row 32 rq + 8 (i/4) + 4 half + i%4 against pooled key t*64 + krow
    const int b0 = t * kPKeys;
    if (!a.multi) {
      float v = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) v += exp2f(c2 * acc[i] - lr[i]);
      v += __shfl_xor(v, 32);
      if (half == 0) red[rq * kPKeys + krow] = v;
      __syncthreads();
      if (tid < kPKeys && b0 + tid < a.nb)
        a.part[(static_cast<int64_t>(h) * a.nseg + seg0) * a.nb + b0 + tid] = red[tid] + red[kPKeys + tid];
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        red[(32 * rq + 8 * (i / 4) + 4 * half + i % 4) * kPRedStride + krow] = exp2f(c2 * acc[i] - lr[i]);
      __syncthreads();
      for (int e = tid; e < ngroups * kPKeys; e += kPThreads) {
        const int j = e / kPKeys, col = e % kPKeys;
        const int r_end = min(j * a.G + a.G, rows);
        float s = 0.f;
        for (int r = j * a.G; r < r_end; ++r) s += red[r * kPRedStride + col];
        if (b0 + col < a.nb) a.part[(static_cast<int64_t>(h) * a.nseg + seg0 + j) * a.nb + b0 + col] = s;
      }
    }
  }
}

__global__ __launch_bounds__(kPThreads) void k_prob_merge(const float* __restrict__ part, int nseg, int nb, int nbp,
                                                          int lq, int G, int R, int multi, int spg,
                                                          const int32_t* __restrict__ page_table, int64_t num_pages,
                                                          int first_excluded, uint32_t* __restrict__ keys) {
  const int b = blockIdx.x * kPThreads + threadIdx.x, r = blockIdx.y, h = blockIdx.z;
  if (b >= nb) return;
  const int rows = min(r * G + G, lq) - r * G;
  float s;
  if (multi) {
    s = part[(static_cast<int64_t>(h) * nseg + r) * nb + b];
  } else {
    s = 0.f;
    const int parts = (rows + kPRows - 1) / kPRows;
    for (int k = 0; k < parts; ++k) s += part[(static_cast<int64_t>(h) * nseg + r * spg + k) * nb + b];
  }
  s = s / static_cast<float>(rows);
  const int32_t p = page_table != nullptr ? page_table[b] : 0;
  const bool live = b < first_excluded && p >= 0 && (page_table == nullptr || p < num_pages);
  keys[(static_cast<int64_t>(h) * R + r) * nbp + b] = live ? score_key(s) : 0u;
}

template <typename T, int D>
hipError_t launch_prob_typed(const CacheGeom& g, const SelectPlan& p, const void* q, const float* kbar,
                             int64_t kbar_stride, float* part, uint32_t* keys, int nbp, hipStream_t stream) {
  ProbArgs a;
  a.q = q;
  a.lq = p.lq;
  a.H = g.H;
  a.G = p.G;
  a.R = p.R;
  a.kbar = kbar;
  a.kbar_stride = kbar_stride;
  a.nb = g.nb;
  a.scale = p.scale;
  a.multi = p.prob_multi ? 1 : 0;
  a.gps = p.prob_gps;
  a.spg = p.prob_spg;
  a.nseg = p.prob_nseg;
  a.part = part;
  hipLaunchKernelGGL((k_prob_partial<T, D>), dim3(p.prob_slices, g.H), dim3(kPThreads), 0, stream, a);
  const dim3 mgrid((g.nb + kPThreads - 1) / kPThreads, p.R, g.H);
  hipLaunchKernelGGL(k_prob_merge, mgrid, dim3(kPThreads), 0, stream, part, p.prob_nseg, g.nb, nbp, p.lq, p.G, p.R,
                     a.multi, p.prob_spg, g.page_table, g.num_pages, p.first_excluded, keys);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prob_keys(const CacheGeom& g, const SelectPlan& p, const void* q, const float* kbar,
                            int64_t kbar_stride, float* part, uint32_t* keys, int nbp, hipStream_t stream) {
  if (g.dtype == 0) {
    if (g.D == 128) return launch_prob_typed<uint16_t, 128>(g, p, q, kbar, kbar_stride, part, keys, nbp, stream);
    return launch_prob_typed<uint16_t, 64>(g, p, q, kbar, kbar_stride, part, keys, nbp, stream);
  }
  if (g.D == 128) return launch_prob_typed<float, 128>(g, p, q, kbar, kbar_stride, part, keys, nbp, stream);
  return launch_prob_typed<float, 64>(g, p, q, kbar, kbar_stride, part, keys, nbp, stream);
}

}  // namespace omnimem
