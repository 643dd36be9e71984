// probe.hip -- roofline probes for gfx950 (libomnimem_probe.so): an MFMA issue
// loop and streaming HBM copy / read kernels, so that the fractions of the published
// peaks can be set beside what the chip sustains at its working clock.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/omnimem_probe.h"
#include "launch.h"

#define PROBE_API extern "C" __attribute__((visibility("default")))

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// A counter-based hash (the 32-bit finaliser of MurmurHash3), for operand values.
__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x85ebca6bu;
  x ^= x >> 13;
  x *= 0xc2b2ae35u;
  x ^= x >> 16;
  return x;
}

// RANDOM = 0: one smooth per-lane operand pair shared by the four chains (few bits
// toggle from one MFMA to the next).  RANDOM = 1: four pairs of random operands, one
// per chain, roughly normal with unit-order values, so that consecutive MFMAs see
// unrelated data, as attention's K, Q, P and V fragments do.  The MFMA power, and with
// it the clock the chip holds, depends on how many operand bits toggle.
template <int RANDOM>
__global__ __launch_bounds__(512) void k_mfma_loop(int64_t iters, float* __restrict__ sink) {
  bf16x8 a[4], b[4];
  const uint32_t t = threadIdx.x + 512u * blockIdx.x;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float va, vb;
      if (RANDOM) {
        // sums of two 16-bit uniforms, centred: triangular on (-1, 1)
        const uint32_t h = mix32(t * 64u + s * 8u + i), g = mix32(h ^ 0x9e3779b9u);
        va = static_cast<float>((h & 0xffffu) + (h >> 16)) * (1.0f / 65536.f) - 1.0f;
        vb = static_cast<float>((g & 0xffffu) + (g >> 16)) * (1.0f / 65536.f) - 1.0f;
      } else {
        // depends on the lane so that nothing folds
        const float x = 1.0f + 1e-3f * static_cast<float>(threadIdx.x % 64);
        va = x * static_cast<float>(i + 1) * 1e-3f;
        vb = x * static_cast<float>(8 - i) * 1e-3f;
      }
      a[s][i] = static_cast<__bf16>(va);
      b[s][i] = static_cast<__bf16>(vb);
    }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int64_t it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[1], c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[2], b[2], c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[3], b[3], c3, 0, 0, 0);
  }
  float s = 0.f;
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  if (s == -1.2345e30f) sink[0] = s;
}

// The attention kernel's MFMA slot in isolation: each v_mfma_f32_32x32x16_bf16 (four
// independent chains, random operands) is followed by the softmax VALU work of one
// score per lane: an fma (c s - max), an exponential, a row-sum add, and on every
// other slot a bf16 pack; no op reads a result of its own slot.  LDS = 1: the MFMAs
// of each slot pair take their A operand from a 1 KB LDS fragment read two pairs
// ahead, like the attention kernel's K fragments.  One wave per SIMD.
template <int LDS>
__global__ __launch_bounds__(256) void k_slot_loop(int64_t iters, float* __restrict__ sink) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;
  __shared__ __attribute__((aligned(1024))) uint4 frags[LDS ? 64 * 64 : 1];
  const uint32_t t = threadIdx.x + 256u * blockIdx.x;
  auto rnd = [](uint32_t h) {  // triangular on (-1, 1)
    return static_cast<float>((h & 0xffffu) + (h >> 16)) * (1.0f / 65536.f) - 1.0f;
  };
  bf16x8 a[4], b[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t h = mix32(t * 64u + q * 8u + i), g = mix32(h ^ 0x9e3779b9u);
      a[q][i] = static_cast<__bf16>(rnd(h));
      b[q][i] = static_cast<__bf16>(rnd(g));
    }
  if constexpr (LDS) {
    for (int i = threadIdx.x; i < 64 * 64; i += 256) {
      bf16x8 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = static_cast<__bf16>(rnd(mix32(i * 8u + e)));
      frags[i] = __builtin_bit_cast(uint4, v);
    }
    __syncthreads();
  }
  const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(frags)) + (threadIdx.x % 64) * 16;
  auto frag = [&](int64_t f) {  // fragment f mod 64: 64 lanes x 16 bytes
    return *reinterpret_cast<lds_bf16x8*>(static_cast<uintptr_t>(base + static_cast<uint32_t>(f % 64) * 1024));
  };
  f32x16 c[4] = {};
  float x[8], y[8], acc = 0.f;
  const float cs = 0.125f, ms = 0.5f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    x[i] = rnd(mix32(t ^ (i * 0x3c6ef372u)));
    y[i] = 0.f;
  }
  bf16x2 pk = {};
  bf16x8 kf[4];
  if constexpr (LDS) {
    kf[0] = frag(0);
    kf[1] = frag(1);
  }
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int sl = 0; sl < 8; ++sl) {
      const int pr = sl / 2;
      if constexpr (LDS) {
        c[sl % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[pr], b[sl % 4], c[sl % 4], 0, 0, 0);
        if (sl % 2 == 0) kf[(pr + 2) % 4] = frag(4 * it + pr + 2);
      } else {
        c[sl % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[sl % 4], b[sl % 4], c[sl % 4], 0, 0, 0);
      }
      x[sl] = fmaf(x[sl], cs, -ms);
      asm volatile("" : "+v"(x[sl]));
      y[sl] = __builtin_amdgcn_exp2f(x[(sl + 7) % 8]);
      asm volatile("" : "+v"(y[sl]));
      acc += y[(sl + 6) % 8];
      asm volatile("" : "+v"(acc));
      if (sl % 2 == 1) {
        pk = bf16x2{static_cast<__bf16>(y[(sl + 5) % 8]), static_cast<__bf16>(y[(sl + 4) % 8])};
        asm volatile("" : "+v"(pk));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  float s = acc + static_cast<float>(pk[0]);
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += c[q][i];
#pragma unroll
  for (int i = 0; i < 8; ++i) s += x[i] + y[i];
  if (s == -1.2345e30f) sink[0] = s;
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// fp32 MFMA issue loop: SHAPE 0 = v_mfma_f32_16x16x4_f32 (2048 flops), 1 =
// v_mfma_f32_32x32x2_f32 (4096 flops); 4 independent chains per wave.
template <int SHAPE>
__global__ __launch_bounds__(512) void k_mfma_f32_loop(int64_t iters, float* __restrict__ sink) {
  const float a = 1.0f + 1e-3f * static_cast<float>(threadIdx.x % 64), b = 1.0f - 1e-3f * static_cast<float>(threadIdx.x % 64);
  float s = 0.f;
  if constexpr (SHAPE == 0) {
    f32x4 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int64_t it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c3, 0, 0, 0);
    }
    for (int i = 0; i < 4; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  } else {
    f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int64_t it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c3, 0, 0, 0);
    }
    for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  }
  if (s == -1.2345e30f) sink[0] = s;
}

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// 16-byte load with the nontemporal hint (streamed data: on gfx950 it raises a
// streaming read from ~5.6 to ~6.3 TB/s)
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_once(const uint4* p) {
  const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__global__ __launch_bounds__(kThreads) void k_copy(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                   int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = load_once(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) dst[i + u * stride] = v[u];
  }
  for (; i < n; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(kThreads) void k_read(const uint4* __restrict__ src, int64_t n,
                                                   float* __restrict__ sink) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = load_once(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n; i += stride) acc ^= src[i].x ^ src[i].y ^ src[i].z ^ src[i].w;
  if (acc == 0x9e3779b9u && threadIdx.x == 0) sink[0] = static_cast<float>(acc);
}

int32_t status(hipError_t e) { return e == hipSuccess ? 0 : -4; }

using omnimem::launch_kernel;

}  // namespace

PROBE_API int32_t omnimem_probe_mfma_f32(int32_t shape, int64_t iters, int32_t workgroups, int32_t waves_per_simd,
                                         float* sink, void* stream) {
  if (shape < 0 || shape > 1 || iters < 1 || workgroups < 1 || waves_per_simd < 1 || waves_per_simd > 2 ||
      sink == nullptr)
    return -1;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (shape == 0)
    return status(launch_kernel(k_mfma_f32_loop<0>, dim3(workgroups), dim3(256 * waves_per_simd), 0, st, iters, sink));
  return status(launch_kernel(k_mfma_f32_loop<1>, dim3(workgroups), dim3(256 * waves_per_simd), 0, st, iters, sink));
}

PROBE_API int32_t omnimem_probe_mfma_bf16(int32_t operands, int64_t iters, int32_t workgroups, int32_t waves_per_simd,
                                          float* sink, void* stream) {
  if (operands < 0 || operands > 1 || iters < 1 || workgroups < 1 || waves_per_simd < 1 || waves_per_simd > 2 ||
      sink == nullptr)
    return -1;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (operands == 0)
    return status(launch_kernel(k_mfma_loop<0>, dim3(workgroups), dim3(256 * waves_per_simd), 0, st, iters, sink));
  return status(launch_kernel(k_mfma_loop<1>, dim3(workgroups), dim3(256 * waves_per_simd), 0, st, iters, sink));
}

PROBE_API int32_t omnimem_probe_softmax_slot(int32_t lds_operands, int64_t iters, int32_t workgroups, float* sink,
                                             void* stream) {
  if (lds_operands < 0 || lds_operands > 1 || iters < 1 || workgroups < 1 || sink == nullptr) return -1;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (lds_operands == 0)
    return status(launch_kernel(k_slot_loop<0>, dim3(workgroups), dim3(256), 0, st, iters, sink));
  return status(launch_kernel(k_slot_loop<1>, dim3(workgroups), dim3(256), 0, st, iters, sink));
}

PROBE_API int32_t omnimem_probe_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream) {
  if (src == nullptr || dst == nullptr || bytes < 16 || bytes % 16 || workgroups < 1 ||
      (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u)
    return -1;
  return status(launch_kernel(k_copy, dim3(workgroups), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                              static_cast<const uint4*>(src), static_cast<uint4*>(dst), bytes / 16));
}

PROBE_API int32_t omnimem_probe_read(const void* src, int64_t bytes, int32_t workgroups, float* sink, void* stream) {
  if (src == nullptr || sink == nullptr || bytes < 16 || bytes % 16 || workgroups < 1 ||
      (reinterpret_cast<uintptr_t>(src) & 15u))
    return -1;
  return status(launch_kernel(k_read, dim3(workgroups), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                              static_cast<const uint4*>(src), bytes / 16, sink));
}
