// attention.hip -- attention over per-(head, group) block lists read in place from
// the paged KV cache (Sec. 3.3 Eq. 5, Per-Head Scattered KV Access; App. C Alg. 1
// Step 2), and over contiguous chunk ranges (dense / sliding-window attention).
//
// bf16 kernel (k_attn_bf16): flash-style, one workgroup = 4 waves = a tile of
// query rows of one (head, query group); the group's block list is walked 64 keys
// at a time.  Each 64-key tile of K and V (one (page, head) slab, or half of one at
// B = 128) is staged in LDS with 16-byte coalesced loads, prefetched into registers
// one tile ahead.  Every wave keeps 32 query rows of Q in registers and computes
//   S^T = K Q^T        on v_mfma_f32_32x32x16_bf16 (K rows as the A operand),
//   O^T += V^T P^T     on the same instruction, V^T read with ds_read_b64_tr_b16,
// so that each lane owns one query column of both S^T and O^T: the online softmax
// (fp32, exp2 domain with the scale folded in) and the rescaling of O need one
// cross-lane exchange (lane l <-> l^32) per tile and no transposes.  The A-operand
// rows of K are fed in an order (bits 2 and 3 of the row swapped) that makes the
// S^T accumulator registers line up with the B-operand layout of P^T, so P goes from
// accumulator to MFMA operand with a bf16 pack and nothing else.
//
// The same arithmetic runs in three data-movement shapes: k_attn_bf16_r64 (d = 128,
// groups of more than 32 rows: 64 rows per wave, tiles by buffer-to-LDS DMA),
// k_attn_bf16 (d = 64, more than 32 rows) and k_attn_bf16_groups (groups of at most
// 32 rows: one wave per group, every wave streaming its own groups' tiles).
//
// f32 kernel (k_attn_f32): one lane per query row, fp32 dot products and exact
// expf-based online softmax, for fp32 inputs.
#include <limits.h>
#include <math.h>
#include <atomic>
#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kTileKeys = 64;  // keys per attention tile (one B = 64 block, half of a B = 128 block)

struct AttnArgs {
  const void* q;
  const void* k_pages;
  const void* v_pages;
  const int32_t* page_table;
  int64_t pt_stride;  // 0: one table for every head; else head h's table at h * pt_stride
  int64_t num_pages;
  int H, S, B, Bpc, nb;
  int lq, G, R;
  const int32_t* idx;
  const int32_t* cnt;
  int top_k;
  int dense_first, dense_count;
  float scale;
  void* out;
  float* lse;
  int tiles_per_group;
};

// Walks the (block, sub-tile) sequence of a block list, skipping padding,
// out-of-range ids and non-resident pages.  Everything here is workgroup-uniform.
template <int TK>
struct TileWalk {
  const AttnArgs& a;
  const int32_t* table;  // the head's page table
  const int32_t* list;
  int count;
  int t = 0, sub = 0;
  int64_t page = 0;
  int nvalid = 0;

  __device__ TileWalk(const AttnArgs& args, const int32_t* pt, const int32_t* l, int c)
      : a(args), table(pt), list(l), count(c) {}

  // position on the next non-empty tile at or after (t, sub); false at the end
  __device__ bool seek() {
    while (t < count) {
      const int id = list ? list[t] : a.dense_first + t;
      if (id >= 0 && id < a.nb) {
        const int32_t p = table[id];
        if (p >= 0 && p < a.num_pages) {
          const int o = id % a.Bpc;
          const int in_block = (o == a.Bpc - 1 ? a.S - o * a.B : a.B) - sub * TK;
          if (in_block > 0) {
            page = p;
            nvalid = in_block < TK ? in_block : TK;
            return true;
          }
        }
      }
      ++t;
      sub = 0;
    }
    return false;
  }
  __device__ void advance() {
    if (++sub * TK >= a.B) {
      ++t;
      sub = 0;
    }
  }
  __device__ int64_t slab_offset(int h, int D) const {
    return (page * a.H + h) * static_cast<int64_t>(a.B) * D + static_cast<int64_t>(sub) * TK * D;
  }
};

__device__ __forceinline__ void resolve_tile(const AttnArgs& a, int rows_per_wg, int& h, int& hr, int& row0,
                                             int& row_end) {
  const int id = xcd_contiguous_id(blockIdx.x, gridDim.x);
  const int tile = id % a.tiles_per_group;
  hr = id / a.tiles_per_group;
  const int r = hr % a.R;
  h = hr / a.R;
  const int g_begin = r * a.G;
  const int g_end = min(g_begin + a.G, a.lq);
  row0 = g_begin + tile * rows_per_wg;
  row_end = min(row0 + rows_per_wg, g_end);
}

// The page table head h reads.
__device__ __forceinline__ const int32_t* head_table(const AttnArgs& a, int h) {
  return a.page_table + static_cast<int64_t>(h) * a.pt_stride;
}

__device__ __forceinline__ void resolve_list(const AttnArgs& a, int hr, const int32_t*& list, int& count) {
  if (a.idx) {
    list = a.idx + static_cast<int64_t>(hr) * a.top_k;
    const int c = a.cnt[hr];
    count = c < 0 ? 0 : (c > a.top_k ? a.top_k : c);
  } else {
    list = nullptr;
    count = a.dense_count;
  }
}

// Decodes list entries [first, first + NT) into a compact table of 64-key tiles in
// LDS: entry i = (page, (sub-tile << 8) | valid keys).  Padding, out-of-range ids and
// non-resident pages produce no tile; a B = 128 block produces up to two.  One list
// entry per thread, compacted with a block-wide prefix sum; returns the tile count.
// Contains barriers: every thread of the workgroup must call it.  pre_id, unless
// INT_MIN, is this thread's list entry, already read by the caller.
template <int NT>
__device__ int decode_tiles(const AttnArgs& a, const int32_t* pt, const int32_t* list, int count, int first,
                            int2* table, int* scan_tmp, int pre_id = INT_MIN) {
  const int e = first + static_cast<int>(threadIdx.x);
  int ntiles = 0, page = 0, nvb = 0;
  if (e < count) {
    const int id = pre_id != INT_MIN ? pre_id : list ? list[e] : a.dense_first + e;
    if (id >= 0 && id < a.nb) {
      const int32_t p = pt[id];
      if (p >= 0 && p < a.num_pages) {
        const int o = id % a.Bpc;
        nvb = o == a.Bpc - 1 ? a.S - o * a.B : a.B;
        page = p;
        ntiles = (nvb + kTileKeys - 1) / kTileKeys;
      }
    }
  }
  int total;
  const int pos = block_exclusive_scan<NT>(ntiles, scan_tmp, total);
  for (int s = 0; s < ntiles; ++s) {
    const int nv = nvb - s * kTileKeys;
    table[pos + s] = make_int2(page, (s << 8) | (nv < kTileKeys ? nv : kTileKeys));
  }
  __syncthreads();
  return total;
}

// ------------------------------------------------------------------ bf16 / MFMA
constexpr int kWaves = 8;  // 256 query rows per workgroup, two waves per SIMD

// A-operand row order for S^T = K Q^T: swapping bits 2 and 3 of the row makes the
// accumulator element i of lane l hold key 8*(l/32)+i (i < 8) or 16+8*(l/32)+(i-8).
__device__ __forceinline__ int s_row_perm(int x) { return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1); }

// LDS row strides (bf16 elements), chosen for gfx950's 64 four-byte banks:
//  K rows are read 16 B per lane, 16 lanes (16 rows) per pass: a stride of 4 (mod 64)
//    dwords puts the 16 rows on disjoint bank quads;
//  V rows are read by ds_read_b64_tr_b16, 4 rows x 32 B per 16-lane group and two
//    groups per pass: a stride of 16 or 48 (mod 64) dwords makes the 8 row segments of a
//    pass disjoint.
template <int D>
struct AttnLds {
  static constexpr int K_STRIDE = D == 128 ? 136 : 72;
  static constexpr int V_STRIDE = D == 128 ? 160 : 96;
  static constexpr int K_ELEMS = kTileKeys * K_STRIDE;
  static constexpr int V_ELEMS = kTileKeys * V_STRIDE;
  static constexpr int K_STAGES = 2;
  static constexpr int V_STAGES = 3;  // the phase-shifted waves still read the previous tile's V
  static constexpr int TOTAL_ELEMS = K_STAGES * K_ELEMS + V_STAGES * V_ELEMS;
};

// NW waves of 32 query rows, the upper half of the waves running half a tile behind
// the lower half (see below); for d = 64 and groups of more than 32 rows.
template <int D, int NW>
__global__ __launch_bounds__(NW* kWave) void k_attn_bf16(AttnArgs a) {
  using L = AttnLds<D>;
  constexpr int NT = NW * kWave;
  constexpr int ROWS = NW * 32;
  constexpr int CHUNKS_PER_ROW = D / 8;                        // 16-byte chunks per key row
  constexpr int CPT = kTileKeys * CHUNKS_PER_ROW / NT;         // chunks per thread per tile (K and V each)
  constexpr int DT = D / 32;                                   // 32-wide output tiles along d
  constexpr int KK = D / 16;                                   // k-steps of QK^T
  static_assert(CPT >= 1, "tile too small for the workgroup");
  __shared__ __attribute__((aligned(16))) uint16_t lds[L::TOTAL_ELEMS];
  __shared__ int2 table[2 * NT];  // decoded tiles of up to NT list entries
  __shared__ int scan_tmp[NW];
  uint16_t* const k_ring = lds;
  uint16_t* const v_ring = lds + L::K_STAGES * L::K_ELEMS;

  int h, hr, row0, row_end;
  resolve_tile(a, ROWS, h, hr, row0, row_end);
  if (row0 >= row_end) return;  // workgroup-uniform: no barrier has been reached
  const int32_t* list;
  int count;
  resolve_list(a, hr, list, count);

  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int half = lane / 32;
  const uint16_t* qp = static_cast<const uint16_t*>(a.q);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k_pages);
  const uint16_t* vp = static_cast<const uint16_t*>(a.v_pages);

  // Q^T as the B operand: lane holds query (lane % 32), d = 16*kk + 8*half + 0..7
  const int my_row = row0 + wave * 32 + lane % 32;
  const bool wave_live = row0 + wave * 32 < row_end;  // wave-uniform
  bf16x8 qreg[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (my_row < row_end)
      raw = *reinterpret_cast<const uint4*>(qp + (static_cast<int64_t>(my_row) * a.H + h) * D + 16 * kk + 8 * half);
    qreg[kk] = __builtin_bit_cast(bf16x8, raw);
  }

  f32x16 o_acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) o_acc[dt][i] = 0.f;
  // running max (raw score units) and this lane's share of the denominator
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.scale * kLog2e;

  uint4 kreg[CPT], vreg[CPT];
  // loads one tile (page, sub-tile, valid keys) into the staging registers
  auto prefetch = [&](int page, int meta) {
    const int sub = meta >> 8, nv = meta & 255;
    const int64_t slab = (static_cast<int64_t>(page) * a.H + h) * a.B * D + static_cast<int64_t>(sub) * kTileKeys * D;
    const uint16_t* ks = kp + slab;
    const uint16_t* vs = vp + slab;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int cid = tid + i * NT;
      const int row = cid / CHUNKS_PER_ROW, c8 = cid % CHUNKS_PER_ROW;
      if (row < nv) {
        kreg[i] = *reinterpret_cast<const uint4*>(ks + row * D + c8 * 8);
        vreg[i] = *reinterpret_cast<const uint4*>(vs + row * D + c8 * 8);
      } else {
        kreg[i] = make_uint4(0, 0, 0, 0);
        vreg[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto stage = [&](int kst, int vst) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int cid = tid + i * NT;
      const int row = cid / CHUNKS_PER_ROW, c8 = cid % CHUNKS_PER_ROW;
      *reinterpret_cast<uint4*>(k_ring + kst * L::K_ELEMS + row * L::K_STRIDE + c8 * 8) = kreg[i];
      *reinterpret_cast<uint4*>(v_ring + vst * L::V_ELEMS + row * L::V_STRIDE + c8 * 8) = vreg[i];
    }
  };

  // The two waves that share a SIMD (w and w + 4) run the same tile half a step
  // apart: waves 0-3 do QK(t), softmax(t), PV(t); waves 4-7 do PV(t-1), QK(t),
  // softmax(t).  While one of them is in its softmax (VALU) the other issues MFMAs.
  const bool late = wave >= NW / 2;
  bf16x8 pb[4];
  auto pv = [&](const uint16_t* v_lds) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key0 = 16 * j + 8 * half + (lane % 16) / 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int col = 32 * dt + 16 * ((lane / 16) % 2) + 4 * (lane % 4);
        typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(v_lds + key0 * L::V_STRIDE + col));
        const i16x4 hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(v_lds + (key0 + 4) * L::V_STRIDE + col));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        o_acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[j], o_acc[dt], 0, 0, 0);
      }
    }
  };

  // tile table: decode list entries NT at a time; `ti` indexes the current table
  int next_entry = 0, ntab = 0, ti = 0;
  while (ntab == 0 && next_entry < count) {
    ntab = decode_tiles<NT>(a, head_table(a, h), list, count, next_entry, table, scan_tmp);
    next_entry += NT;
  }
  bool have = ntab > 0;
  int2 cur_tile = have ? table[0] : make_int2(0, 0);
  cur_tile.x = __builtin_amdgcn_readfirstlane(cur_tile.x);
  cur_tile.y = __builtin_amdgcn_readfirstlane(cur_tile.y);
  if (have) {
    prefetch(cur_tile.x, cur_tile.y);
    stage(0, 0);
  }
  __syncthreads();
  const int krow = s_row_perm(lane % 32);
  int t = 0;
  while (have) {
    const int cur_nvalid = cur_tile.y & 255;
    if (++ti == ntab) {  // table exhausted: decode the next list entries (dense lists only)
      ntab = 0;
      ti = 0;
      while (ntab == 0 && next_entry < count) {
        ntab = decode_tiles<NT>(a, head_table(a, h), list, count, next_entry, table, scan_tmp);
        next_entry += NT;
      }
    }
    have = ti < ntab;
    if (have) {
      cur_tile = table[ti];
      cur_tile.x = __builtin_amdgcn_readfirstlane(cur_tile.x);
      cur_tile.y = __builtin_amdgcn_readfirstlane(cur_tile.y);
      prefetch(cur_tile.x, cur_tile.y);  // next tile: global loads in flight during this tile's math
    }
    const uint16_t* k_lds = k_ring + (t % 2) * L::K_ELEMS;
    const uint16_t* v_lds = v_ring + (t % L::V_STAGES) * L::V_ELEMS;

    if (wave_live) {
      if (late && t > 0) pv(v_ring + ((t + L::V_STAGES - 1) % L::V_STAGES) * L::V_ELEMS);  // PV of the previous tile
      // ---- S^T = K Q^T for keys [0, 64): two 32-key accumulators
      f32x16 s_acc[2];
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
#pragma unroll
        for (int i = 0; i < 16; ++i) s_acc[t2][i] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          const bf16x8 kf =
              *reinterpret_cast<const bf16x8*>(k_lds + (32 * t2 + krow) * L::K_STRIDE + 16 * kk + 8 * half);
          s_acc[t2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qreg[kk], s_acc[t2], 0, 0, 0);
        }
      }
      // ---- online softmax for this lane's query (exp2 domain, scale folded into one FMA)
      if (cur_nvalid < kTileKeys) {  // partial tile: mask the keys past the block's end
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = 32 * t2 + (i < 8 ? 8 * half + i : 16 + 8 * half + (i - 8));
            if (key >= cur_nvalid) s_acc[t2][i] = -INFINITY;
          }
      }
      float mloc = s_acc[0][0];
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i) mloc = fmaxf(mloc, s_acc[t2][i]);
      const float m_tile = fmaxf(mloc, __shfl_xor(mloc, 32));
      // rescale only when some lane's running max grows (exact: alpha == 1 otherwise)
      if (__any(m_tile > m_run)) {
        const float m_new = fmaxf(m_run, m_tile);
        const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_run - m_new) * c);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int i = 0; i < 16; ++i) o_acc[dt][i] *= alpha;
        m_run = m_new;
      }
      const float mc = m_run == -INFINITY ? 0.f : m_run * c;
      float psum = 0.f;
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s_acc[t2][i], c, -mc));
          psum += p;
          pb[2 * t2 + i / 8][i % 8] = static_cast<__bf16>(p);
        }
      l_run += psum;
      if (!late) pv(v_lds);
    }
    if (have) stage((t + 1) % 2, (t + 1) % L::V_STAGES);  // stages not read in this step
    __syncthreads();
    ++t;
  }
  if (late && wave_live && t > 0) pv(v_ring + ((t + L::V_STAGES - 1) % L::V_STAGES) * L::V_ELEMS);  // the last tile's PV
  __syncthreads();  // the rings are reused below for the output

  // ---- epilogue: normalise, stage O through LDS, store rows with 16-byte writes
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  constexpr int SSTRIDE = D + 8;
  static_assert(NW * 32 * SSTRIDE <= L::TOTAL_ELEMS, "output staging does not fit");
  uint16_t* stage_o = lds + wave * 32 * SSTRIDE;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i4 = 0; i4 < 4; ++i4) {
      const int d0 = 32 * dt + 8 * i4 + 4 * half;
      bf16x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(o_acc[dt][4 * i4 + e] * inv);
      *reinterpret_cast<bf16x4*>(stage_o + (lane % 32) * SSTRIDE + d0) = w;
    }
  __syncthreads();
  uint16_t* op = static_cast<uint16_t*>(a.out);
  constexpr int OCHUNKS = 32 * CHUNKS_PER_ROW;
#pragma unroll
  for (int i = 0; i < OCHUNKS / kWave; ++i) {
    const int cid = lane + i * kWave;
    const int row = cid / CHUNKS_PER_ROW, c8 = cid % CHUNKS_PER_ROW;
    const int qrow = row0 + wave * 32 + row;
    if (qrow < row_end)
      *reinterpret_cast<uint4*>(op + (static_cast<int64_t>(qrow) * a.H + h) * D + c8 * 8) =
          *reinterpret_cast<const uint4*>(stage_o + row * SSTRIDE + c8 * 8);
  }
  if (a.lse && lane < 32 && my_row < row_end)
    a.lse[static_cast<int64_t>(h) * a.lq + my_row] =
        l_tot > 0.f ? (m_run * c + __log2f(l_tot)) * kLn2 : -INFINITY;
}

// ------------------------------------------------------------------ bf16 / MFMA, one wave per query group
// Query groups of at most 32 rows (the small-group setting of App. B, where every
// group of G_q rows keeps its own top-K blocks, and short dense calls): a group is
// one 32-row MFMA tile, so its attention is a gather with little arithmetic per
// byte.  Every wave runs on its own, with no barrier: it walks a sequence of
// (head, group) pairs (pair first + k * stride, the grid resident at once), and
// the tiles of consecutive groups form one stream, the next tile's K and V always
// in flight while the current one is computed, across group boundaries too.  K
// goes from memory straight into registers in the MFMA A-operand layout; V passes
// through the wave's own LDS tile for the transposing reads.  The next group's list
// entries are fetched when the walk enters a group, its Q rows with its first tile.
// The arithmetic is that of the 32-row kernel: the same operand layouts, the same
// online softmax, the same rounding.
constexpr int kGrpWaves = 4;

template <int D>
__global__ __launch_bounds__(kGrpWaves* kWave, 1) void k_attn_bf16_groups(AttnArgs a) {
  using L = AttnLds<D>;
  constexpr int KK = D / 16;                       // k-steps of QK^T
  constexpr int DT = D / 32;                       // 32-wide output tiles along d
  constexpr int CPR = D / 8;                       // 16-byte chunks per key row
  constexpr int VROWS = kWave / CPR;               // V rows per load instruction
  constexpr int VLOADS = kTileKeys / VROWS;        // V load instructions per tile
  __shared__ __attribute__((aligned(16))) uint16_t v_all[kGrpWaves * L::V_ELEMS];

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave, half = lane / 32;
  uint16_t* const v_lds = v_all + wave * L::V_ELEMS;
  const int total = a.H * a.R;
  const int stride = gridDim.x * kGrpWaves;
  const int first = xcd_contiguous_id(blockIdx.x, gridDim.x) * kGrpWaves + wave;
  if (first >= total) return;  // wave-uniform; no barrier anywhere below
  const uint16_t* qp = static_cast<const uint16_t*>(a.q);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k_pages);
  const uint16_t* vp = static_cast<const uint16_t*>(a.v_pages);
  uint16_t* op = static_cast<uint16_t*>(a.out);
  const float c = a.scale * kLog2e;
  const int krow = s_row_perm(lane % 32);

  // ---- the walk over groups and tiles (wave-uniform state; w_* and nx_id per lane)
  int p_hr = first, p_count = 0, p_base = 0, p_e = 0, p_sub = 0, p_emitted = 0;
  const int32_t* p_list = nullptr;
  int w_page = -1, w_nvb = 0;  // entry p_base + lane: page (-1: no tile) and valid tokens
  int nx_id = -1, nx_count = 0;
  const int32_t* nx_list = nullptr;

  auto group_list = [&](int hr, const int32_t*& list) -> int {
    int count;
    resolve_list(a, hr, list, count);
    return count;
  };
  auto entry_id = [&](const int32_t* list, int count, int e) -> int {
    if (e >= count) return -1;
    return list ? list[e] : a.dense_first + e;
  };
  // this lane's entry of the window: its page and valid tokens, or no tile
  auto resolve_window = [&](int id) {
    w_page = -1;
    w_nvb = 0;
    if (id >= 0 && id < a.nb) {
      const int32_t p = head_table(a, p_hr / a.R)[id];
      const int o = id % a.Bpc;
      const int nvb = o == a.Bpc - 1 ? a.S - o * a.B : a.B;
      if (p >= 0 && p < a.num_pages && nvb > 0) {
        w_page = p;
        w_nvb = nvb;
      }
    }
  };
  auto prefetch_next_ids = [&]() {
    const int nhr = p_hr + stride;
    nx_count = 0;
    nx_id = -1;
    if (nhr < total) {
      nx_count = group_list(nhr, nx_list);
      nx_id = entry_id(nx_list, nx_count, lane);
    }
  };
  // output of a group without a single tile: O = 0, lse = -inf
  auto write_empty = [&](int hr) {
    const int h = hr / a.R, g0 = (hr % a.R) * a.G, rows = min(g0 + a.G, a.lq) - g0;
    for (int i = lane; i < rows * CPR; i += kWave)
      *reinterpret_cast<uint4*>(op + (static_cast<int64_t>(g0 + i / CPR) * a.H + h) * D + (i % CPR) * 8) =
          make_uint4(0, 0, 0, 0);
    if (a.lse && lane < rows) a.lse[static_cast<int64_t>(h) * a.lq + g0 + lane] = -INFINITY;
  };
  // first group: its ids now, then the next group's
  p_count = group_list(p_hr, p_list);
  resolve_window(entry_id(p_list, p_count, lane));
  prefetch_next_ids();

  // the next tile of the walk: page, (sub-tile << 8) | valid keys, its group, and
  // whether it opens the group; false at the end
  auto next_tile = [&](int& page, int& meta, int& hr, bool& opens) -> bool {
    for (;;) {
      while (p_e < p_count) {
        if (p_e >= p_base + kWave) {  // lists longer than a wave: the next window
          p_base += kWave;
          resolve_window(entry_id(p_list, p_count, p_base + lane));
          continue;
        }
        const uint64_t live = __ballot(w_page >= 0) & (~0ull << (p_e - p_base));
        if (live == 0) {
          p_e = p_base + kWave;
          p_sub = 0;
          continue;
        }
        const int l = __builtin_ctzll(live);
        if (p_base + l != p_e) {
          p_e = p_base + l;
          p_sub = 0;
        }
        const int nvb = __builtin_amdgcn_readlane(w_nvb, l);
        page = __builtin_amdgcn_readlane(w_page, l);
        const int left = nvb - p_sub * kTileKeys;
        meta = (p_sub << 8) | (left < kTileKeys ? left : kTileKeys);
        hr = p_hr;
        opens = p_emitted == 0;
        ++p_emitted;
        if (++p_sub * kTileKeys >= nvb) {
          ++p_e;
          p_sub = 0;
        }
        return true;
      }
      if (p_emitted == 0) write_empty(p_hr);
      p_hr += stride;
      if (p_hr >= total) return false;
      p_list = nx_list;
      p_count = nx_count;
      p_base = p_e = p_sub = p_emitted = 0;
      resolve_window(nx_id);
      prefetch_next_ids();
    }
  };

  // ---- registers of the stream: K of two tiles (current, next), V of the next, Q
  bf16x8 ka[2][KK], kb[2][KK], q[KK], qn[KK];
  uint4 vn[VLOADS];
  auto load_tile = [&](int page, int meta, int hr, bf16x8 (&kf)[2][KK]) {
    const int sub = meta >> 8, nv = meta & 255;
    const int64_t slab = (static_cast<int64_t>(page) * a.H + hr / a.R) * a.B * D + static_cast<int64_t>(sub) * kTileKeys * D;
    const uint16_t* ks = kp + slab;
    const uint16_t* vs = vp + slab;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const int row = 32 * t2 + krow;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        uint4 raw = make_uint4(0, 0, 0, 0);
        if (row < nv) raw = *reinterpret_cast<const uint4*>(ks + row * D + 16 * kk + 8 * half);
        kf[t2][kk] = __builtin_bit_cast(bf16x8, raw);
      }
    }
#pragma unroll
    for (int i = 0; i < VLOADS; ++i) {
      const int row = i * VROWS + lane / CPR;
      vn[i] = row < nv ? *reinterpret_cast<const uint4*>(vs + row * D + (lane % CPR) * 8) : make_uint4(0, 0, 0, 0);
    }
  };
  auto load_q = [&](int hr) {
    const int h = hr / a.R, g0 = (hr % a.R) * a.G, g1 = min(g0 + a.G, a.lq);
    const int row = g0 + lane % 32;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      uint4 raw = make_uint4(0, 0, 0, 0);
      if (row < g1) raw = *reinterpret_cast<const uint4*>(qp + (static_cast<int64_t>(row) * a.H + h) * D + 16 * kk + 8 * half);
      qn[kk] = __builtin_bit_cast(bf16x8, raw);
    }
  };

  // ---- per-group softmax state
  f32x16 o_acc[DT];
  float m_run = -INFINITY, l_run = 0.f;
  int cur_hr = -1;
  auto finish = [&](int hr) {
    const int h = hr / a.R, g0 = (hr % a.R) * a.G, g1 = min(g0 + a.G, a.lq);
    const int row = g0 + lane % 32;
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    if (row < g1) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          bf16x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(o_acc[dt][4 * i4 + e] * inv);
          *reinterpret_cast<bf16x4*>(op + (static_cast<int64_t>(row) * a.H + h) * D + 32 * dt + 8 * i4 + 4 * half) = w;
        }
      if (a.lse && lane < 32)
        a.lse[static_cast<int64_t>(h) * a.lq + row] = l_tot > 0.f ? (m_run * c + __log2f(l_tot)) * kLn2 : -INFINITY;
    }
  };
  auto open_group = [&](int hr) {
    if (cur_hr >= 0) finish(cur_hr);
    cur_hr = hr;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) q[kk] = qn[kk];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) o_acc[dt][i] = 0.f;
    m_run = -INFINITY;
    l_run = 0.f;
  };

  bf16x8 pb[4];
  auto pv = [&]() {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key0 = 16 * j + 8 * half + (lane % 16) / 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int col = 32 * dt + 16 * ((lane / 16) % 2) + 4 * (lane % 4);
        typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(v_lds + key0 * L::V_STRIDE + col));
        const i16x4 hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(v_lds + (key0 + 4) * L::V_STRIDE + col));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        o_acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[j], o_acc[dt], 0, 0, 0);
      }
    }
  };
  // QK^T, online softmax and PV of one tile whose K is in kf and V in the LDS tile
  auto compute = [&](const bf16x8 (&kf)[2][KK], int nvalid) {
    f32x16 s_acc[2];
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
#pragma unroll
      for (int i = 0; i < 16; ++i) s_acc[t2][i] = 0.f;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) s_acc[t2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[t2][kk], q[kk], s_acc[t2], 0, 0, 0);
    }
    if (nvalid < kTileKeys) {  // partial tile: mask the keys past the block's end
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = 32 * t2 + (i < 8 ? 8 * half + i : 16 + 8 * half + (i - 8));
          if (key >= nvalid) s_acc[t2][i] = -INFINITY;
        }
    }
    float mloc = s_acc[0][0];
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) mloc = fmaxf(mloc, s_acc[t2][i]);
    const float m_tile = fmaxf(mloc, __shfl_xor(mloc, 32));
    if (__any(m_tile > m_run)) {  // rescale only when some lane's running max grows
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_run - m_new) * c);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) o_acc[dt][i] *= alpha;
      m_run = m_new;
    }
    const float mc = m_run == -INFINITY ? 0.f : m_run * c;
    float psum = 0.f;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s_acc[t2][i], c, -mc));
        psum += p;
        pb[2 * t2 + i / 8][i % 8] = static_cast<__bf16>(p);
      }
    l_run += psum;
    pv();
  };

  int page = 0, meta = 0, hr = 0;
  bool opens = false;
  bool have = next_tile(page, meta, hr, opens);
  if (have) {
    load_tile(page, meta, hr, ka);
    if (opens) load_q(hr);
  }
  // one tile: its K in kc, its V in vn; the next tile's loads go to kn and vn
  auto step = [&](bf16x8 (&kc)[2][KK], bf16x8 (&kn)[2][KK]) {
    const int nvalid = meta & 255;
    if (opens) open_group(hr);
#pragma unroll
    for (int i = 0; i < VLOADS; ++i)
      *reinterpret_cast<uint4*>(v_lds + (i * VROWS + lane / CPR) * L::V_STRIDE + (lane % CPR) * 8) = vn[i];
    have = next_tile(page, meta, hr, opens);
    if (have) {
      load_tile(page, meta, hr, kn);
      if (opens) load_q(hr);
    }
    compute(kc, nvalid);
  };
  while (have) {
    step(ka, kb);
    if (!have) break;
    step(kb, ka);
  }
  if (cur_hr >= 0) finish(cur_hr);
}

// ------------------------------------------------------------------ bf16 / MFMA, 64 rows per wave
// Four waves (one per SIMD) x 64 query rows, as two 32-row halves that share every
// K and V operand read from LDS: each 1 KB operand fragment feeds two MFMAs, half the
// LDS bytes per flop of the 32-row kernel, whose operand traffic equals the LDS
// bandwidth at the MFMA peak.  With one wave per SIMD the matrix core is kept busy
// from inside the wave: the instruction stream alternates MFMAs of one half with
// the softmax VALU work of the other (QK of half 1 with the exponentials of half
// 0, PV of half 0 with the exponentials of half 1), and MFMAs run asynchronously.
// The running max starts as the first tile's own max and may then lag the true one:
// O and l are rescaled only when exponentials against the stale max could exceed 2^8,
// well inside fp32 and bf16 range, and the final normalisation cancels the stale max
// exactly.
constexpr int kR64Waves = 4;
constexpr float kSlackSum = 256.0f;  // 2^8: how far exponentials may exceed 1 before O is rescaled
constexpr float kNoMax = -1.0e30f;   // running max before the first tile: finite, below any score

// max / sum of a value over the lane pair (l, l ^ 32)
__device__ __forceinline__ float pair_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Pins values at this point of the instruction stream: the exponentials of one half
// are computed between the other half's MFMAs, not moved down past the check that
// follows them to their first use.
__device__ __forceinline__ void keep_here(const bf16x8 (&pb)[4], float l) {
  asm volatile("" ::"v"(pb[0]), "v"(pb[1]), "v"(pb[2]), "v"(pb[3]), "v"(l));
}

// Workgroup barrier for LDS traffic only.  __syncthreads() also orders global memory,
// which makes every wave drain its outstanding loads, including the DMA of tiles
// meant to stay in flight across the barrier; LDS written by DMA is covered by the
// explicit vmcnt wait before it, and the asm statements keep the compiler from
// moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// LDS tiles of the 64-row kernel: 64 rows of 256 bytes (d = 128 bf16), unpadded, with
// the 16-byte chunks of each row permuted so that both the K fragment reads and the
// transposing V reads touch every bank once per pass:
//   K: chunk c of row r sits at chunk position c ^ (r mod 16)
//   V: chunk c of row r sits at chunk position c ^ 4 (r mod 4)
// Tiles arrive by buffer-to-LDS DMA: one instruction moves 64 lanes x 16 bytes into a
// contiguous 1 KB (rows 4m .. 4m + 3), lane l filling chunk position l mod 16 of row
// 4m + l / 16, so each lane fetches the global chunk that belongs at its position.
constexpr int kR64TileBytes = kTileKeys * 128 * 2;
__device__ __forceinline__ int k_pos(int r, int c) { return r * 256 + ((c ^ (r & 15)) << 4); }
__device__ __forceinline__ int v_pos(int r, int c) { return r * 256 + ((c ^ (4 * (r & 3))) << 4); }

// s_waitcnt operand that waits for at most n outstanding vector-memory operations
// and for nothing else (gfx9 encoding: vmcnt in bits 3:0 and 15:14)
constexpr int vmcnt_only(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// Buffer resource (raw, stride 0) over `bytes` bytes at p, in scalar registers; the
// caller guarantees p and bytes are the same in every lane.  Offsets at or past the
// end read as zero.
__device__ __forceinline__ u32x4 buffer_rsrc(const void* p, int bytes) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  u32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
  r[1] = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32) & 0xffffu);
  r[2] = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bytes));
  r[3] = 0x00020000u;
  return r;
}

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)p));
}
// P V product with its accumulator in AccVGPRs.  Selected by the compiler, every
// MFMA accumulator sits in the VGPRs that the softmax VALU work also uses, and an
// MFMA writing its result there slows that work down; the asm keeps O in AccVGPRs.
// The asm also hides the MFMA from the compiler's hazard checks, so the wait states
// are explicit: two before the MFMA (any operand may have been written by VALU code
// just before it: a rematerialised constant, a copy out of a spill), the callers
// keep the A and B operands unchanged until the MFMA has read them (it reads them
// over its passes), and VALU code touches the accumulators only after
// acc_settled().
__device__ __forceinline__ void pv_mfma(f32x16& acc, const bf16x8& v, const bf16x8& p) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(v), "v"(p));
}
// Sixteen wait states (more than an 8-pass MFMA result needs) before VALU code reads
// or writes the accumulators; they pass through the asm so that no access moves
// ahead of it.
__device__ __forceinline__ void acc_settled(f32x16 (&o)[4]) {
  asm volatile("s_nop 7\n\ts_nop 7" : "+a"(o[0]), "+a"(o[1]), "+a"(o[2]), "+a"(o[3]));
}


// One buffer-to-LDS DMA instruction: lane l's 16 bytes at rsrc + voffset land at LDS
// byte lds + 16 l.  It is written as inline asm so that the compiler does not track
// it as an LDS store (it would make every later LDS read wait for all DMA in flight);
// the kernel orders it itself, with explicit vmcnt waits before the barriers that
// publish a stage.
__device__ __forceinline__ void dma_16x64(u32x4 rsrc, int voffset, uint32_t lds) {
  // M0 (the LDS destination) is set by the compiler; the s_nop is the wait state an
  // LDS DMA needs after an M0 write
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voffset), "s"(rsrc), "{m0}"(lds) : "memory");
}

template <int D>
__global__ __launch_bounds__(kR64Waves* kWave, 1) void k_attn_bf16_r64(AttnArgs a) {
  static_assert(D == 128, "the 64-row kernel is laid out for d = 128");
  constexpr int NT = kR64Waves * kWave;
  constexpr int ROWS = kR64Waves * 64;
  constexpr int DT = D / 32;
  constexpr int KK = D / 16;
  constexpr int DMA_PER_WAVE = kR64TileBytes / 1024 / kR64Waves;  // 1 KB DMA instructions per wave, K and V each
  // Four stages of K and V, tile t in stage t mod 4: iteration t reads the K of tile t
  // and the V of tile t - 1 while tile t + 1 has landed and tile t + 2 arrives in the
  // stage of tile t - 2.
  constexpr int kStages = 4;
  __shared__ __attribute__((aligned(1024))) uint8_t k_ring[kStages * kR64TileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_ring[kStages * kR64TileBytes];
  __shared__ int2 table[2 * NT];
  __shared__ int scan_tmp[kR64Waves];

  int h, hr, row0, row_end;
  resolve_tile(a, ROWS, h, hr, row0, row_end);
  if (row0 >= row_end) return;  // workgroup-uniform: no barrier has been reached
  const int32_t* list;
  int count;
  resolve_list(a, hr, list, count);

  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  // this thread's entry of the first decoded stretch, read without waiting for the
  // count (the list holds top_k entries)
  const int id0 = list != nullptr && tid < a.top_k ? list[tid] : INT_MIN;
  const int half = lane / 32;
  const uint16_t* qp = static_cast<const uint16_t*>(a.q);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k_pages);
  const uint16_t* vp = static_cast<const uint16_t*>(a.v_pages);

  // Q^T B operands of the two halves: lane holds query wrow + 32 g + lane % 32
  const float c = a.scale * kLog2e;  // scores to the softmax's log2 units, applied in fp32
  const int wrow = row0 + wave * 64;
  const bool wave_live = wrow < row_end;  // wave-uniform
  // the Q rows are loaded here and moved to AccVGPRs once the first tiles' DMA is
  // issued, so that their latency overlaps the block-list decode
  uint4 qx0[KK], qx1[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const int r0 = wrow + lane % 32, r1 = r0 + 32;
    qx0[kk] = qx1[kk] = make_uint4(0, 0, 0, 0);
    if (r0 < row_end)
      qx0[kk] = *reinterpret_cast<const uint4*>(qp + (static_cast<int64_t>(r0) * a.H + h) * D + 16 * kk + 8 * half);
    if (r1 < row_end)
      qx1[kk] = *reinterpret_cast<const uint4*>(qp + (static_cast<int64_t>(r1) * a.H + h) * D + 16 * kk + 8 * half);
  }
  bf16x8 q0[KK], q1[KK];

  f32x16 o0[DT], o1[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      o0[dt][i] = 0.f;
      o1[dt][i] = 0.f;
    }
  // running max in scaled log2 units (max * scale * log2 e) and this lane's share of l
  float ms0 = kNoMax, ms1 = kNoMax, l0 = 0.f, l1 = 0.f;

  // ---- tile sequence: (page, sub-tile << 8 | valid keys), from the decoded table
  int next_entry = 0, ntab = 0, ti = 0;
  // The next table entry as read from LDS (the same in every lane; made scalar where
  // used, so that the read's latency is not waited for here).  Called by every thread
  // together: it refills the table (with barriers) when it runs out.
  auto next_tile_raw = [&]() -> int2 {
    if (ti == ntab) {
      ntab = 0;
      ti = 0;
      while (ntab == 0 && next_entry < count) {
        ntab = decode_tiles<NT>(a, head_table(a, h), list, count, next_entry, table, scan_tmp,
                                next_entry == 0 ? id0 : INT_MIN);
        next_entry += NT;
      }
      if (ntab == 0) return make_int2(0, 0);  // past the end: an empty tile
    }
    return table[ti++];
  };
  auto scalar_tile = [](int2 m) {
    return make_int2(__builtin_amdgcn_readfirstlane(m.x), __builtin_amdgcn_readfirstlane(m.y));
  };
  // this lane's source offsets for its DMA instructions (row 4 m + lane / 16, m = wave + 4 i)
  int k_src[DMA_PER_WAVE], v_src[DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < DMA_PER_WAVE; ++i) {
    const int r = 4 * (wave + kR64Waves * i) + lane / 16, p = lane % 16;
    k_src[i] = r * 256 + ((p ^ (r & 15)) << 4);
    v_src[i] = r * 256 + ((p ^ (4 * (r & 3))) << 4);
  }
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);  // scalar copy: LDS destinations go to M0
  // Scalar bases: this head's slab of page 0, the page stride, and the wave's first
  // LDS destination.  Everything about a tile's DMA is then a few scalar ops.
  const int64_t h_elems = static_cast<int64_t>(__builtin_amdgcn_readfirstlane(h)) * a.B * D;
  const uint16_t* const kp_h = kp + h_elems;
  const uint16_t* const vp_h = vp + h_elems;
  const int64_t page_elems = static_cast<int64_t>(a.H) * a.B * D;
  const uint32_t m0_k = lds_offset(k_ring) + wave_s * 1024, m0_v = lds_offset(v_ring) + wave_s * 1024;
  // the DMA of tile m into stage st, instruction i of K and of V (empty tiles load
  // nothing and write zeros); m is workgroup-uniform.  The LDS bases pass through an
  // empty asm so that each destination is formed where it is used: hoisted out of
  // the loop, the 32 stage/instruction combinations would each hold a scalar register.
  auto issue_part = [&](int2 m, int st, int i) {
    const int sub = m.y >> 8, nv = m.y & 255;
    const int64_t slab = static_cast<int64_t>(m.x) * page_elems + static_cast<int64_t>(sub) * kTileKeys * D;
    const u32x4 kr = buffer_rsrc(kp_h + slab, nv * D * 2), vr = buffer_rsrc(vp_h + slab, nv * D * 2);
    uint32_t mk = m0_k, mv = m0_v;
    asm volatile("" : "+s"(mk), "+s"(mv));
    const uint32_t off = st * kR64TileBytes + kR64Waves * i * 1024;
    dma_16x64(kr, k_src[i], mk + off);
    dma_16x64(vr, v_src[i], mv + off);
  };
  auto issue = [&](int2 m, int st) {
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) issue_part(m, st, i);
  };

  // keys past the block's end of a partial tile get -inf scores (the key base goes
  // through an empty asm so that none of this is computed ahead of the rare branch)
  auto mask_tail = [&](f32x16 (&s)[2], int nvalid) {
    int kb = 8 * half;
    asm volatile("" : "+v"(kb));
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = 32 * t2 + (i < 8 ? kb + i : 16 + kb + (i - 8));
        if (key >= nvalid) s[t2][i] = -INFINITY;
      }
  };
  // A half's softmax as a stream over its 32 S elements per lane (element E is
  // s[E / 16][E % 16]; it lands in P^T fragment E / 8 at position E % 8).  Slot g
  // forms the exponent c s - max of element g (one fma: the scale is applied in
  // fp32), takes the exponential of element g - 1, adds element g - 2 to the row sum
  // and, on odd slots, packs elements g - 3 and g - 2 into P (late enough for the PV
  // run that carries the early slots to have read the previous tile's P fragment 0).
  // No op of a slot reads a result of the same slot, so a slot placed next to one
  // MFMA issues without waiting on VALU latency; slots 32 and 33 finish the stream.
  // Each result goes through an empty asm so that the IR passes keep it in its slot
  // (they would otherwise sink every op next to its first use).  The row sum is taken
  // over the fp32 values.
  auto soft_slot = [&](const f32x16 (&s)[2], float ms, float& acc, bf16x8 (&pb)[4], float (&tq)[32],
                       float (&uq)[32], int g) {
    if (g < 32) {
      tq[g] = fmaf(s[g / 16][g % 16], c, -ms);
      asm volatile("" : "+v"(tq[g]));
    }
    if (g >= 1 && g <= 32) {
      uq[g - 1] = __builtin_amdgcn_exp2f(tq[g - 1]);
      asm volatile("" : "+v"(uq[g - 1]));
    }
    if (g >= 2 && g <= 33) {
      acc += uq[g - 2];
      asm volatile("" : "+v"(acc));
    }
    if (g % 2 == 1 && g >= 3 && g <= 33) {
      const int e = g - 3;
      bf16x2 pk = {static_cast<__bf16>(uq[e]), static_cast<__bf16>(uq[e + 1])};
      asm volatile("" : "+v"(pk));
      pb[e / 8][e % 8] = pk[0];
      pb[e / 8][e % 8 + 1] = pk[1];
    }
  };
  const int krow = s_row_perm(lane % 32);
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  // Operand fragments, read from LDS ahead of the MFMAs that use them: K fragments four
  // ahead, V fragments three (four would take the PV run past 256 VGPRs).
  // The lane's part of each address is fixed for the whole loop (8 K and 4 V byte
  // offsets, the chunk permutations depending only on the lane); the stage, the key
  // group and the ring base are compile-time constants that fold into the reads'
  // offset fields.
  // (masked to the 18 bits of the LDS address space, which lets the compiler see that
  // base + constant cannot wrap)
  uint32_t k_lane[KK], v_lane[DT];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) k_lane[kk] = (lds_offset(k_ring) + k_pos(krow, 2 * kk + half)) & 0x3ffffu;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    const int key0 = 8 * half + (lane % 16) / 4;
    const int ch = 4 * dt + 2 * ((lane / 16) % 2) + (lane % 4) / 2;
    v_lane[dt] = (lds_offset(v_ring) + v_pos(key0, ch) + 8 * (lane % 2)) & 0x3ffffu;
  }
  typedef __attribute__((address_space(3))) const uint8_t lds_u8;
  auto k_frag = [&](int st, int f) {  // f = 8 t2 + kk: keys 32 t2 .., k-step kk
    lds_u8* p = reinterpret_cast<lds_u8*>(static_cast<uintptr_t>(k_lane[f % KK])) + (st * kR64TileBytes + (f / KK) * 32 * 256);
    return *reinterpret_cast<__attribute__((address_space(3))) const bf16x8*>(p);
  };
  auto v_frag = [&](int st, int f) {  // f = 4 j + dt: keys 16 j .., d 32 dt ..; two transposing reads (keys +4)
    lds_u8* p = reinterpret_cast<lds_u8*>(static_cast<uintptr_t>(v_lane[f % DT])) + (st * kR64TileBytes + (f / DT) * 16 * 256);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * 256));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // The exponentials of a half are computed against its running max before the
  // tile's own max is known (the first tile's against its own max, taken once).  They
  // stand (every p <= 2^8) unless some lane's sum of them exceeds 2^8 or overflowed,
  // which takes a rise of the max by more than 3 log2 units; only then is the tile's S
  // formed again from the K still in LDS (stage kst, nvalid keys), its max taken, O
  // and l moved to the new max and the exponentials redone.  The next tile's
  // exponentials are formed after this point, against the new max.  The rare path is
  // laid out away from the loop, which then runs straight through.
  auto settle = [&](float& ms, float& l, float acc, f32x16 (&o)[DT], bf16x8 (&pb)[4], const bf16x8 (&q)[KK], int kst,
                    int nvalid) {
    if (__builtin_expect(__any(acc > kSlackSum), 0)) {
      f32x16 s[2];
#pragma unroll
      for (int f = 0; f < 2 * KK; ++f) {
        s[f / KK] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_frag(kst, f), q[f % KK], f % KK ? s[f / KK] : f32x16{}, 0,
                                                           0, 0);
        __builtin_amdgcn_sched_barrier(0);  // one fragment at a time: this path must not raise register use
      }
      if (nvalid < kTileKeys) mask_tail(s, nvalid);
      float m0 = fmaxf(s[0][0], s[1][0]), m1 = fmaxf(s[0][1], s[1][1]);
#pragma unroll
      for (int i = 2; i < 16; i += 2) {
        m0 = fmaxf(m0, fmaxf(s[0][i], s[1][i]));
        m1 = fmaxf(m1, fmaxf(s[0][i + 1], s[1][i + 1]));
      }
      const float m_new = fmaxf(ms, pair_max(fmaxf(m0, m1)) * c);
      const float alpha = __builtin_amdgcn_exp2f(ms - m_new);
      l *= alpha;
      acc_settled(o);
      // one 16-register block at a time through VGPRs (O stays in AccVGPRs)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        f32x16 t = o[dt];
        asm volatile("" : "+v"(t));
#pragma unroll
        for (int i = 0; i < 16; ++i) t[i] *= alpha;
        o[dt] = t;
        asm volatile("" : "+a"(o[dt]));
      }
      ms = m_new;
      acc = 0.f;
#pragma unroll
      for (int e = 0; e < 32; e += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[e / 16][e % 16], c, -m_new));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[e / 16][e % 16 + 1], c, -m_new));
        acc += p0 + p1;
        pb[e / 8][e % 8] = static_cast<__bf16>(p0);
        pb[e / 8][e % 8 + 1] = static_cast<__bf16>(p1);
      }
    }
    l += acc;
  };

  // ---- Software pipeline over tiles.  Iteration t runs two runs of 32 MFMAs, each
  // MFMA carrying one softmax stream slot (one exponential, a half-rate VALU op, and
  // two or three other VALU ops fill the MFMA shadow only when spread this thin):
  //   QK run  S of tile t, both halves (each K fragment feeds the two halves' MFMAs
  //           back to back); slots 15-33 of tile t-1's two streams; DMA of tile t+2
  //   PV run  O += P V of tile t-1, both halves (each V^T fragment feeds two MFMAs);
  //           slots 0-14 of tile t's two streams
  // with both halves' softmax checks of tile t-1 between the runs.  Operand fragments
  // are read just in time, so the registers hold S of two tiles and P of one.  One
  // barrier per iteration, at its end: tile t+1 has landed and every wave is past its
  // reads of the stages that the next iteration's DMA refills.  "Tile -1" is an
  // all-masked dummy (S = -inf, P = 0, its V stage DMA'd from an empty tile: zeros),
  // and the sequence ends with one empty tile whose iteration finishes the last one.
  static_assert(2 * KK == 16 && 4 * DT == 16 && DMA_PER_WAVE == 4, "the MFMA runs are laid out for d = 128");
  f32x16 sa0[2], sa1[2], sb0[2], sb1[2];
  bf16x8 pb0[4], pb1[4];
  // the first tile's max of a half's S in scaled log2 units, from both lanes of each
  // row (masked keys are -inf: with no valid key at all it stays kNoMax)
  bool first_tile = true;
  auto tile_max = [&](const f32x16 (&s)[2]) {
    float m0 = fmaxf(s[0][0], s[1][0]), m1 = fmaxf(s[0][1], s[1][1]);
#pragma unroll
    for (int i = 2; i < 16; i += 2) {
      m0 = fmaxf(m0, fmaxf(s[0][i], s[1][i]));
      m1 = fmaxf(m1, fmaxf(s[0][i + 1], s[1][i + 1]));
    }
    return fmaxf(kNoMax, pair_max(fmaxf(m0, m1)) * c);
  };
  float acc0 = 0.f, acc1 = 0.f;
  // the two halves' softmax streams (only a few elements of each are live at a time)
  float tq0[32], uq0[32], tq1[32], uq1[32];
#pragma unroll
  for (int t2i = 0; t2i < 2; ++t2i)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      sa0[t2i][i] = -INFINITY;
      sa1[t2i][i] = -INFINITY;
    }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    pb0[j] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
    pb1[j] = pb0[j];
  }
  tq0[14] = tq1[14] = -INFINITY;  // the dummy tile's streams enter the loop at slot 15
  uq0[12] = uq0[13] = uq1[12] = uq1[13] = 0.f;
  int prev_nvalid = 0;

  int2 cur = scalar_tile(next_tile_raw());
  int2 t1 = scalar_tile(next_tile_raw());
  issue(make_int2(0, 0), kStages - 1);  // V of tile -1
  issue(cur, 0);
  issue(t1, 1);
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    q0[kk] = __builtin_bit_cast(bf16x8, qx0[kk]);
    q1[kk] = __builtin_bit_cast(bf16x8, qx1[kk]);
    // Q lives in AccVGPRs next to O; the VGPRs hold S, P and the operand fragments
    asm volatile("" : "+a"(q0[kk]), "+a"(q1[kk]));
  }
  // The Q loads and the block-list reads have landed (the compiler waited for them
  // before the decode and the scaling, so it knows of no load of its own pending in
  // the loop, where any wait it inserted would also drain the DMA in flight, which it
  // does not see); of the DMA, the dummy stage and tile 0 must land before the loop,
  // tile 1 may still be in flight.
  __builtin_amdgcn_s_waitcnt(vmcnt_only(2 * DMA_PER_WAVE));
  lds_barrier();

  // Iteration t (t mod 4 = T, a compile-time constant, as are the stages) with tile
  // t-1's S in (so0, so1) and tile t's formed in (sn0, sn1); consecutive iterations
  // swap the two, so that no S is ever copied.  Returns false after the iteration of
  // the empty tile that ends the sequence.
  auto iteration = [&](f32x16 (&so0)[2], f32x16 (&so1)[2], f32x16 (&sn0)[2], f32x16 (&sn1)[2], auto tmod) {
    constexpr int T = decltype(tmod)::value;
    constexpr int kst = T, vst = (T + kStages - 1) % kStages, st2 = (T + 2) % kStages;
    bf16x8 kf[2 * KK], vf[4 * DT];
    if (wave_live) {
      kf[0] = k_frag(kst, 0);
      kf[1] = k_frag(kst, 1);
      kf[2] = k_frag(kst, 2);
      kf[3] = k_frag(kst, 3);
    }
    const int2 t2 = scalar_tile(next_tile_raw());  // every thread; refills the table at its end
    const int cur_nvalid = cur.y & 255;
    if (wave_live) {
      // ---- QK run
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const int f = i / 2;
        if (i % 2 == 0) {
          sn0[f / KK] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[f], q0[f % KK], f % KK ? sn0[f / KK] : f32x16{}, 0, 0, 0);
          soft_slot(so0, ms0, acc0, pb0, tq0, uq0, 15 + f);
          if (f + 4 < 2 * KK) kf[f + 4] = k_frag(kst, f + 4);
        } else {
          sn1[f / KK] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[f], q1[f % KK], f % KK ? sn1[f / KK] : f32x16{}, 0, 0, 0);
          soft_slot(so1, ms1, acc1, pb1, tq1, uq1, 15 + f);
        }
        if (i % 8 == 5) issue_part(t2, st2, i / 8);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int g = 31; g < 34; ++g) {
        soft_slot(so0, ms0, acc0, pb0, tq0, uq0, g);
        soft_slot(so1, ms1, acc1, pb1, tq1, uq1, g);
      }
      keep_here(pb0, acc0);
      keep_here(pb1, acc1);
      vf[0] = v_frag(vst, 0);
      vf[1] = v_frag(vst, 1);
      vf[2] = v_frag(vst, 2);
      settle(ms0, l0, acc0, o0, pb0, q0, vst, prev_nvalid);
      settle(ms1, l1, acc1, o1, pb1, q1, vst, prev_nvalid);
      acc0 = 0.f;
      acc1 = 0.f;
      if (__builtin_expect(cur_nvalid < kTileKeys, 0)) {
        mask_tail(sn0, cur_nvalid);
        mask_tail(sn1, cur_nvalid);
      }
      if (T == 0 && first_tile) {  // the first tile's exponentials use its own max
        first_tile = false;
        ms0 = tile_max(sn0);
        ms1 = tile_max(sn1);
      }
      // ---- PV run.  Stream slot (g, half) of tile t rides on MFMA 2 g + half + 2,
      // past the last MFMA that reads the previous tile's P fragment it overwrites.
      // An MFMA reads its A and B registers over its passes, so each MFMA's operands
      // are held (an empty asm use) until the end of the next slot, when it has
      // finished: the compiler, which does not see these MFMAs, would otherwise give
      // the registers to the next value as soon as the MFMA is issued.
      bf16x8 hold_a = vf[0], hold_b = pb0[0];
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const int f = i / 2;
        const bf16x8 op_a = vf[f], op_b = i % 2 ? pb1[f / DT] : pb0[f / DT];
        if (i % 2 == 0) {
          pv_mfma(o0[f % DT], op_a, op_b);
          if (f + 3 < 4 * DT) vf[f + 3] = v_frag(vst, f + 3);
        } else {
          pv_mfma(o1[f % DT], op_a, op_b);
        }
        if (i >= 2) {
          if (i % 2 == 0) soft_slot(sn0, ms0, acc0, pb0, tq0, uq0, (i - 2) / 2);
          else soft_slot(sn1, ms1, acc1, pb1, tq1, uq1, (i - 2) / 2);
        }
        if (i > 0) asm volatile("" ::"v"(hold_a), "v"(hold_b));
        hold_a = op_a;
        hold_b = op_b;
        __builtin_amdgcn_sched_barrier(0);
      }
      asm volatile("s_nop 7\n\ts_nop 3" ::"v"(hold_a), "v"(hold_b));  // the last MFMA's operands
    } else {
      issue(t2, st2);
    }
    // ---- tile t+1 has landed (the DMA of tile t+2 may still be in flight) and every
    // wave is past its reads of the stages refilled next
    __builtin_amdgcn_s_waitcnt(vmcnt_only(2 * DMA_PER_WAVE));
    lds_barrier();
    cur = t1;
    t1 = t2;
    prev_nvalid = cur_nvalid;
    return cur_nvalid != 0;
  };
  for (;;) {
    if (!iteration(sa0, sa1, sb0, sb1, std::integral_constant<int, 0>{})) break;
    if (!iteration(sb0, sb1, sa0, sa1, std::integral_constant<int, 1>{})) break;
    if (!iteration(sa0, sa1, sb0, sb1, std::integral_constant<int, 2>{})) break;
    if (!iteration(sb0, sb1, sa0, sa1, std::integral_constant<int, 3>{})) break;
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_only(0));  // no DMA may land in the stages reused below
  __syncthreads();

  // ---- epilogue: normalise, stage O through LDS (one 16 KB stage per wave, chunks
  // permuted like K), store rows with 16-byte nontemporal writes (each row is written
  // once, and the L2 then holds no dirty lines of O for the end of the kernel to
  // write back)
  uint8_t* const stage_o = k_ring + wave * kR64TileBytes;  // 64 rows x 256 B per wave
  auto finish = [&](f32x16 (&o)[DT], float ms, float l, int g) {
    const float l_tot = pair_sum(l);
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    const int r = 32 * g + lane % 32;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        bf16x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(o[dt][4 * i4 + e] * inv);
        // d = 32 dt + 8 i4 + 4 half: chunk 4 dt + i4, byte 8 half within it
        *reinterpret_cast<bf16x4*>(stage_o + k_pos(r, 4 * dt + i4) + 8 * half) = w;
      }
    const int qr = wrow + r;
    if (a.lse && lane < 32 && qr < row_end)
      a.lse[static_cast<int64_t>(h) * a.lq + qr] = l_tot > 0.f ? (ms + __log2f(l_tot)) * kLn2 : -INFINITY;
  };
  if (wave_live) {
    acc_settled(o0);
    acc_settled(o1);
    finish(o0, ms0, l0, 0);
    finish(o1, ms1, l1, 1);
  }
  __syncthreads();
  uint16_t* op = static_cast<uint16_t*>(a.out);
  if (wave_live) {
#pragma unroll
    for (int i = 0; i < 64 * 16 / kWave; ++i) {
      const int cid = lane + i * kWave;
      const int r = cid / 16, ch = cid % 16;
      const int qrow = wrow + r;
      if (qrow < row_end)
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(stage_o + k_pos(r, ch)),
                                    reinterpret_cast<u32x4*>(op + (static_cast<int64_t>(qrow) * a.H + h) * D + ch * 8));
    }
  }
}

// ------------------------------------------------------------------ fp32 / SIMT
constexpr int kF32Keys = 32;

template <int D>
__global__ __launch_bounds__(kWave) void k_attn_f32(AttnArgs a) {
  __shared__ float k_lds[kF32Keys][D];
  __shared__ float v_lds[kF32Keys][D];
  int h, hr, row0, row_end;
  resolve_tile(a, kWave, h, hr, row0, row_end);
  if (row0 >= row_end) return;
  const int32_t* list;
  int count;
  resolve_list(a, hr, list, count);
  const int lane = threadIdx.x;
  const int my_row = row0 + lane;
  const bool active = my_row < row_end;
  const float* qp = static_cast<const float*>(a.q);
  const float* kp = static_cast<const float*>(a.k_pages);
  const float* vp = static_cast<const float*>(a.v_pages);

  float qv[D], o[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    qv[j] = active ? qp[(static_cast<int64_t>(my_row) * a.H + h) * D + j] : 0.f;
    o[j] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  TileWalk<kF32Keys> walk(a, head_table(a, h), list, count);
  while (walk.seek()) {
    const float* ks = kp + walk.slab_offset(h, D);
    const float* vs = vp + walk.slab_offset(h, D);
    const int nvalid = walk.nvalid;
    for (int i = lane; i < kF32Keys * D / 4; i += kWave) {
      const int row = i / (D / 4), c4 = i % (D / 4);
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
      if (row < nvalid) {
        kv = *reinterpret_cast<const float4*>(ks + row * D + 4 * c4);
        vv = *reinterpret_cast<const float4*>(vs + row * D + 4 * c4);
      }
      *reinterpret_cast<float4*>(&k_lds[row][4 * c4]) = kv;
      *reinterpret_cast<float4*>(&v_lds[row][4 * c4]) = vv;
    }
    __syncthreads();
    for (int key = 0; key < nvalid; ++key) {
      float dot = 0.f;
#pragma unroll
      for (int j = 0; j < D; ++j) dot = fmaf(qv[j], k_lds[key][j], dot);
      const float s = a.scale * dot;
      const float m_new = fmaxf(m, s);
      const float alpha = expf(m - m_new);
      const float p = expf(s - m_new);
      l = l * alpha + p;
#pragma unroll
      for (int j = 0; j < D; ++j) o[j] = fmaf(p, v_lds[key][j], o[j] * alpha);
      m = m_new;
    }
    __syncthreads();
    walk.advance();
  }
  if (!active) return;
  float* op = static_cast<float*>(a.out) + (static_cast<int64_t>(my_row) * a.H + h) * D;
  const float inv = l > 0.f ? 1.0f / l : 0.f;
#pragma unroll
  for (int j = 0; j < D; ++j) op[j] = o[j] * inv;
  if (a.lse) a.lse[static_cast<int64_t>(h) * a.lq + my_row] = l > 0.f ? m + logf(l) : -INFINITY;
}

// Workgroups of the one-wave-per-group kernel: one wave per group, at most as many
// workgroups as the device holds at once (its CU count times the kernel's
// occupancy, looked up once per device).
template <int D>
int group_workgroups(int64_t groups) {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> resident[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev >= kMaxDevices) dev = -1;
  int n = dev >= 0 ? resident[dev].load(std::memory_order_relaxed) : 0;
  if (n <= 0) {
    int cus = 0, per_cu = 0;
    if (dev < 0 || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_attn_bf16_groups<D>, kGrpWaves * kWave, 0) !=
            hipSuccess ||
        per_cu <= 0)
      per_cu = 1;
    n = cus * per_cu;
    if (dev >= 0) resident[dev].store(n, std::memory_order_relaxed);
  }
  const int64_t need = (groups + kGrpWaves - 1) / kGrpWaves;
  return static_cast<int>(need < n ? need : n);
}

}  // namespace

hipError_t launch_attention(const CacheGeom& g, const AttnLaunch& L, hipStream_t stream) {
  AttnArgs a;
  a.q = L.q;
  a.k_pages = g.k_pages;
  a.v_pages = g.v_pages;
  a.page_table = g.page_table;
  a.pt_stride = g.pt_stride;
  a.num_pages = g.num_pages;
  a.H = g.H;
  a.S = g.S;
  a.B = g.B;
  a.Bpc = g.Bpc;
  a.nb = g.nb;
  a.lq = L.lq;
  a.G = L.group_size;
  a.R = L.R;
  a.idx = L.idx;
  a.cnt = L.cnt;
  a.top_k = L.top_k;
  a.dense_first = L.dense_first_block;
  a.dense_count = L.dense_num_blocks;
  a.scale = L.scale;
  a.out = L.out;
  a.lse = L.lse;
  const int rows = L.group_size < L.lq ? L.group_size : L.lq;
  // bf16, d = 128 and groups of more than 32 rows: 64 rows per wave; else 32
  const bool r64 = g.dtype == 0 && g.D == 128 && rows > 32;
  const bool small = rows <= 32;  // one 32-row tile per group: a wave per group
  const int rows_per_wg = g.dtype != 0 ? kWave : r64 ? kR64Waves * 64 : small ? 32 : kWaves * 32;
  a.tiles_per_group = (rows + rows_per_wg - 1) / rows_per_wg;
  const int64_t nwg = static_cast<int64_t>(g.H) * L.R * a.tiles_per_group;
  if (nwg <= 0) return hipSuccess;
  if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<unsigned>(nwg));
  // bf16 with d = 128 and more than 32 rows per group always takes the 64-row kernel
  if (r64) return launch_kernel(k_attn_bf16_r64<128>, grid, dim3(kR64Waves * kWave), 0, stream, a);
  if (g.dtype == 0) {
    if (!small) return launch_kernel(k_attn_bf16<64, kWaves>, grid, dim3(kWaves * kWave), 0, stream, a);
    if (g.D == 128)
      return launch_kernel(k_attn_bf16_groups<128>, dim3(group_workgroups<128>(nwg)), dim3(kGrpWaves * kWave), 0,
                           stream, a);
    return launch_kernel(k_attn_bf16_groups<64>, dim3(group_workgroups<64>(nwg)), dim3(kGrpWaves * kWave), 0, stream,
                         a);
  }
  if (g.D == 128) return launch_kernel(k_attn_f32<128>, grid, dim3(kWave), 0, stream, a);
  return launch_kernel(k_attn_f32<64>, grid, dim3(kWave), 0, stream, a);
}

}  // namespace omnimem
