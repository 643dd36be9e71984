// launch.h -- host-side launchers of the libomnimem kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>
#include <type_traits>
#include <utility>

#include "plan.h"

namespace omnimem {

// Launches one kernel and returns that launch's own status.  The runtime's
// per-thread "last error" is neither read nor cleared, so an error left there by
// the caller's own HIP work is not reported as the library's, and is not lost.
template <typename... KArgs, typename... Args>
inline hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t stream,
                                Args&&... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
  std::tuple<std::decay_t<KArgs>...> vals(static_cast<std::decay_t<KArgs>>(std::forward<Args>(args))...);
  void* ptrs[sizeof...(KArgs) > 0 ? sizeof...(KArgs) : 1] = {};
  std::apply([&ptrs](auto&... v) {
    size_t i = 0;
    ((ptrs[i++] = static_cast<void*>(&v)), ...);
  }, vals);
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, shmem, stream);
}

// The status of a sequence of launches: the first failure is kept and the launches
// after it are not issued.
struct LaunchStatus {
  hipError_t err = hipSuccess;
  template <typename Kernel, typename... Args>
  void operator()(Kernel kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t stream, Args&&... args) {
    if (err == hipSuccess) err = launch_kernel(kernel, grid, block, shmem, stream, std::forward<Args>(args)...);
  }
  void add(hipError_t e) {
    if (err == hipSuccess) err = e;
  }
};

// Probability-averaged score keys (score_mode 1) from pooled keys kbar
// [H][kbar_stride][D] fp32: order-preserving keys [H][R][nbp], 0 outside Omega.
// hi_pages / lo_pages: the compressed cache's bf16 pooled keys and their residual
// ([pages][H][64][D] each), or both null: the pieces are then split from kbar into
// ksplit first.
hipError_t launch_prob_keys(const CacheGeom& g, const SelectPlan& p, const void* q, const float* kbar,
                            int64_t kbar_stride, float* part, void* ksplit, const void* hi_pages,
                            const void* lo_pages, uint32_t* keys, int nbp, hipStream_t stream);

hipError_t launch_select(const CacheGeom& g, const SelectPlan& p, const void* q, int32_t* idx, int32_t* cnt,
                         float* score, void* workspace, hipStream_t stream);

// ---------------------------------------------------------------- compressed history
hipError_t launch_compress_chunk(const CacheGeom& g, const CmpCache& cc, int chunk, hipStream_t stream);

// Selection with the pooled keys read from cc.k_mean (plan from plan_select).
hipError_t launch_select_compressed(const CacheGeom& g, const CmpCache& cc, const SelectPlan& p, const void* q,
                                    int32_t* idx, int32_t* cnt, float* score, void* workspace, hipStream_t stream);

// ---------------------------------------------------------------- attention
hipError_t launch_attention(const CacheGeom& g, const AttnLaunch& a, hipStream_t stream);

// ---------------------------------------------------------------- gated fusion (Eq. 1)
// out = sum_c sigmoid(gate[row][c]) * o_c over the present branches (null = absent);
// rows = lq * H rows of D elements, dtype 0 = bf16, 1 = f32.
hipError_t launch_gated_combine(int dtype, int64_t rows, int D, const void* o_cmp, const void* o_slc,
                                const void* o_swa, const float* gate, void* out, hipStream_t stream);

// ---------------------------------------------------------------- union gather
hipError_t launch_union_gather(const CacheGeom& g, const UnionPlan& up, const AttnLaunch& a, int32_t* union_blocks,
                               void* workspace, hipStream_t stream);

}  // namespace omnimem
