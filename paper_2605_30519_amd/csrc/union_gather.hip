// union_gather.hip -- the naive comparator of Sec. 3.3: materialise the cross-head
// union U of all selected blocks in a head-aligned buffer (footprint proportional
// to H * |U|), then attend over that buffer.  The buffer is laid out exactly like
// the page pool ([slot][H][B][d]) and described by its own page table, so the
// attention kernel that runs on it is the one of omnimem_sparse_attn, reading the
// same values in the same order: the outputs match bit for bit.
#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

__global__ void k_fill_i32(int32_t* __restrict__ p, int n, int32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// flags[b] = 1 for every resident block that appears in any (h, r) list
__global__ void k_union_mark(const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, int rows, int K,
                             int nb, const int32_t* __restrict__ page_table, int64_t num_pages,
                             int32_t* __restrict__ flags) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(rows) * K) return;
  const int row = static_cast<int>(e / K), t = static_cast<int>(e % K);
  const int c = cnt[row];
  if (t >= c) return;
  const int b = idx[e];
  if (b < 0 || b >= nb) return;
  const int32_t p = page_table[b];
  if (p < 0 || p >= num_pages) return;
  flags[b] = 1;
}

// table[b] = slot of b in the compact buffer (ascending id order) or -1; |U| out
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void k_union_scan(const int32_t* __restrict__ flags, int nb,
                                                             int32_t* __restrict__ table,
                                                             int32_t* __restrict__ union_blocks) {
  __shared__ int tmp[kScanThreads / kWave];
  const int per = (nb + kScanThreads - 1) / kScanThreads;
  const int lo = min(static_cast<int>(threadIdx.x) * per, nb), hi = min(lo + per, nb);
  int mine = 0;
  for (int b = lo; b < hi; ++b) mine += flags[b] != 0;
  int total;
  int pos = block_exclusive_scan<kScanThreads>(mine, tmp, total);
  for (int b = lo; b < hi; ++b) table[b] = flags[b] ? pos++ : -1;
  if (threadIdx.x == 0) *union_blocks = total;
}

// copy the (page, head) slabs of every union block into its slot, for K and V; the
// sources are read once (nontemporal loads), four rounds of loads in flight before
// their stores
__global__ __launch_bounds__(256) void k_union_gather(const uint4* __restrict__ k_pages,
                                                      const uint4* __restrict__ v_pages,
                                                      const int32_t* __restrict__ page_table,
                                                      const int32_t* __restrict__ table, int H,
                                                      int64_t slab_vec, uint4* __restrict__ kbuf,
                                                      uint4* __restrict__ vbuf) {
  constexpr int kRounds = 4;
  const int b = blockIdx.x, h = blockIdx.y;
  const int slot = table[b];
  if (slot < 0) return;
  const int64_t src = (static_cast<int64_t>(page_table[b]) * H + h) * slab_vec;
  const int64_t dst = (static_cast<int64_t>(slot) * H + h) * slab_vec;
  for (int64_t i0 = threadIdx.x; i0 < slab_vec; i0 += kRounds * blockDim.x) {
    uint4 kv[kRounds], vv[kRounds];
#pragma unroll
    for (int u = 0; u < kRounds; ++u) {
      const int64_t i = i0 + static_cast<int64_t>(u) * blockDim.x;
      if (i < slab_vec) {
        kv[u] = load_once(k_pages + src + i);
        vv[u] = load_once(v_pages + src + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kRounds; ++u) {
      const int64_t i = i0 + static_cast<int64_t>(u) * blockDim.x;
      if (i < slab_vec) {
        kbuf[dst + i] = kv[u];
        vbuf[dst + i] = vv[u];
      }
    }
  }
}

}  // namespace

hipError_t launch_union_gather(const CacheGeom& g, const UnionPlan& up, const AttnLaunch& a, int32_t* union_blocks,
                               void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  int32_t* flags = reinterpret_cast<int32_t*>(ws + up.off_flags);
  int32_t* table = reinterpret_cast<int32_t*>(ws + up.off_table);
  void* kbuf = ws + up.off_kbuf;
  void* vbuf = ws + up.off_vbuf;
  const int nb = g.nb;
  LaunchStatus st;
  if (nb == 0) {
    st(k_fill_i32, dim3(1), dim3(64), 0, stream, union_blocks, 1, 0);
  } else {
    st(k_fill_i32, dim3((nb + 255) / 256), dim3(256), 0, stream, flags, nb, 0);
    const int rows = g.H * a.R;
    const int64_t entries = static_cast<int64_t>(rows) * a.top_k;
    st(k_union_mark, dim3(static_cast<unsigned>((entries + 255) / 256)), dim3(256), 0, stream, a.idx, a.cnt, rows,
       a.top_k, nb, g.page_table, g.num_pages, flags);
    st(k_union_scan, dim3(1), dim3(kScanThreads), 0, stream, flags, nb, table, union_blocks);
    st(k_union_gather, dim3(nb, g.H), dim3(256), 0, stream, static_cast<const uint4*>(g.k_pages),
       static_cast<const uint4*>(g.v_pages), g.page_table, table, g.H, up.slab_bytes / 16, static_cast<uint4*>(kbuf),
       static_cast<uint4*>(vbuf));
  }
  if (st.err != hipSuccess) return st.err;
  CacheGeom gu = g;
  gu.k_pages = kbuf;
  gu.v_pages = vbuf;
  gu.page_table = table;
  gu.pt_stride = 0;
  gu.num_pages = nb;
  return launch_attention(gu, a, stream);
}

}  // namespace omnimem
