// fuse.hip -- Eq. 1's gated fusion of the three attention branches for gfx950:
//   out[i][h] = sum over c in (CMP, SLC, SWA) of sigmoid(gate[i][h][c]) * o_c[i][h].
// HBM-bound and elementwise: one thread per 16-byte chunk of an output row reads the
// row's three gate logits and the matching chunk of each present branch, combines
// in fp32 and stores the chunk rounded to the output dtype.
#include <math.h>

#include "device_common.h"
#include "launch.h"

namespace omnimem {
namespace {

constexpr int kFuseThreads = 256;

template <typename T>
struct Chunk;

template <>
struct Chunk<uint16_t> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void store(uint16_t* p, const float (&x)[8]) {
    uint4 w;
    w.x = f32_to_bf16_rne(x[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[1])) << 16);
    w.y = f32_to_bf16_rne(x[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[3])) << 16);
    w.z = f32_to_bf16_rne(x[4]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[5])) << 16);
    w.w = f32_to_bf16_rne(x[6]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[7])) << 16);
    *reinterpret_cast<uint4*>(p) = w;
  }
};

template <>
struct Chunk<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void store(float* p, const float (&x)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
};

template <typename T>
__global__ __launch_bounds__(kFuseThreads) void k_gated_combine(const T* __restrict__ o_cmp, const T* __restrict__ o_slc,
                                                                const T* __restrict__ o_swa,
                                                                const float* __restrict__ gate, int64_t rows, int cpr,
                                                                T* out) {
  constexpr int N = Chunk<T>::N;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * kFuseThreads + threadIdx.x;
  if (t >= rows * cpr) return;
  const int64_t row = t / cpr;
  const int64_t at = t * N;  // element offset: rows are cpr chunks of N elements
  const T* src[3] = {o_cmp, o_slc, o_swa};
  float acc[N];
#pragma unroll
  for (int j = 0; j < N; ++j) acc[j] = 0.f;
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    if (src[c] == nullptr) continue;
    const float g = 1.0f / (1.0f + expf(-gate[row * 3 + c]));  // the branch's sigmoid gate, in [0, 1]
    float x[N];
    Vec16<T>::widen(*reinterpret_cast<const uint4*>(src[c] + at), x);
#pragma unroll
    for (int j = 0; j < N; ++j) acc[j] = fmaf(g, x[j], acc[j]);
  }
  Chunk<T>::store(out + at, acc);
}

}  // namespace

hipError_t launch_gated_combine(int dtype, int64_t rows, int D, const void* o_cmp, const void* o_slc,
                                const void* o_swa, const float* gate, void* out, hipStream_t stream) {
  const int vec = dtype == 0 ? 8 : 4;
  const int cpr = D / vec;
  const int64_t threads = rows * cpr;
  if (threads <= 0) return hipSuccess;
  const int64_t blocks = (threads + kFuseThreads - 1) / kFuseThreads;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<unsigned>(blocks));
  if (dtype == 0)
    return launch_kernel(k_gated_combine<uint16_t>, grid, dim3(kFuseThreads), 0, stream,
                         static_cast<const uint16_t*>(o_cmp), static_cast<const uint16_t*>(o_slc),
                         static_cast<const uint16_t*>(o_swa), gate, rows, cpr, static_cast<uint16_t*>(out));
  return launch_kernel(k_gated_combine<float>, grid, dim3(kFuseThreads), 0, stream,
                       static_cast<const float*>(o_cmp), static_cast<const float*>(o_slc),
                       static_cast<const float*>(o_swa), gate, rows, cpr, static_cast<float*>(out));
}

}  // namespace omnimem
