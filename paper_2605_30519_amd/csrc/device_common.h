// device_common.h -- small device helpers shared by the libomnimem kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace omnimem {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies, workgroups dispatched round-robin

// The hardware dispatches workgroup i to XCD (i mod 8).  Remap so that the
// workgroups that land on one XCD get a contiguous range of logical ids; work that
// shares data (all query tiles of one head) then shares that XCD's L2.
__device__ __forceinline__ int xcd_contiguous_id(int bid, int nblocks) {
  const int per = nblocks / kNumXcd, rem = nblocks % kNumXcd;
  const int xcd = bid % kNumXcd, local = bid / kNumXcd;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// 16-byte load with the nontemporal hint, for data read once (the K stream of the
// selection, Q): it is not kept in the caches, and on gfx950 a stream of such loads
// sustains ~6.3 TB/s against ~5.6 TB/s for plain loads.
__device__ __forceinline__ uint4 load_once(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// fp32 -> bf16 bit pattern, rounded to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Order-preserving map of an fp32 score to uint32 (larger score -> larger key).
// -0 is folded onto +0 first so that equal scores compare equal.  Candidate keys
// are forced >= 1 so that 0 can mark "not a candidate".
__device__ __forceinline__ uint32_t score_key(float s) {
  s = s + 0.0f;
  const uint32_t u = __float_as_uint(s);
  const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return k == 0u ? 1u : k;
}

// 16-byte vector load widened to fp32: 8 bf16 or 4 fp32 values.
template <typename T>
struct Vec16;

template <>
struct Vec16<uint16_t> {  // bf16 storage
  static constexpr int N = 8;
  __device__ __forceinline__ static void load(const uint16_t* p, float (&out)[8]) {
    widen(*reinterpret_cast<const uint4*>(p), out);
  }
  __device__ __forceinline__ static void widen(const uint4 raw, float (&out)[8]) {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = __uint_as_float(w[i] << 16);
      out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};

template <>
struct Vec16<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void load(const float* p, float (&out)[4]) {
    widen(*reinterpret_cast<const uint4*>(p), out);
  }
  __device__ __forceinline__ static void widen(const uint4 raw, float (&out)[4]) {
    out[0] = __uint_as_float(raw.x);
    out[1] = __uint_as_float(raw.y);
    out[2] = __uint_as_float(raw.z);
    out[3] = __uint_as_float(raw.w);
  }
};

__device__ __forceinline__ float wave_xor_sum(float v, int lane_mask_lo, int lane_mask_hi) {
  for (int m = lane_mask_lo; m <= lane_mask_hi; m <<= 1) v += __shfl_xor(v, m);
  return v;
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x % kWave;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(v, off);
    if (lane >= off) v += t;
  }
  return v;
}

// Exclusive prefix sum over a workgroup of NT threads; `total` gets the sum.
// `tmp` must hold NT/64 ints of LDS.  Contains barriers: call from all threads.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int* tmp, int& total) {
  constexpr int kWaves = NT / kWave;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int incl = wave_inclusive_scan(v);
  if (lane == kWave - 1) tmp[wave] = incl;
  __syncthreads();
  int before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int t = tmp[w];
    if (w < wave) before += t;
    sum += t;
  }
  __syncthreads();
  total = sum;
  return before + incl - v;
}

}  // namespace omnimem
