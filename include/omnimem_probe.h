/*
 * omnimem_probe.h -- C ABI of libomnimem_probe.so: roofline probes that measure
 * what one MI355X (gfx950) sustains, next to the published peaks that the
 * benchmark's roofline fractions use.  Measurement only; the attention path does
 * not use this library.
 *
 * Every pointer is a DEVICE pointer; every call is asynchronous on `stream` (a
 * hipStream_t, NULL = null stream) and returns 0 on success, -1 on an invalid
 * argument (nothing launched), -4 when the launch failed.
 */
#ifndef OMNIMEM_PROBE_H
#define OMNIMEM_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* MFMA issue loop: `workgroups` workgroups of 4*waves_per_simd waves, each wave
   issuing `iters` rounds of 4 independent v_mfma_f32_32x32x16_bf16 (4 x 32768
   flops per round).  operands: 0 = one smooth per-lane operand pair for all four
   chains (few operand bits toggle), 1 = four pairs of random unit-order operands,
   one per chain (consecutive MFMAs see unrelated data; the chip's power limit then
   sets a lower clock).  sink: >= 1 float, written only if the sums take an
   impossible value (it keeps the loop from being optimised away). */
int32_t omnimem_probe_mfma_bf16(int32_t operands, int64_t iters, int32_t workgroups, int32_t waves_per_simd,
                                float* sink, void* stream);

/* fp32 MFMA issue loop, as above with 4 independent chains of
   v_mfma_f32_16x16x4_f32 (shape 0, 2048 flops each) or v_mfma_f32_32x32x2_f32
   (shape 1, 4096 flops each) per round. */
int32_t omnimem_probe_mfma_f32(int32_t shape, int64_t iters, int32_t workgroups, int32_t waves_per_simd, float* sink,
                               void* stream);

/* The attention kernel's MFMA slot in isolation: `workgroups` workgroups of 4 waves
   (one per SIMD), each wave issuing `iters` rounds of 8 slots; a slot is one
   v_mfma_f32_32x32x16_bf16 (32768 flops, four independent chains, random operands)
   followed by the softmax VALU work of one score per lane (fma, exponential, add,
   and a bf16 pack every other slot).  lds_operands: 0 = MFMA operands in registers,
   1 = the A operand of each slot pair read from LDS two pairs ahead (1 KB per
   fragment).  sink as above. */
int32_t omnimem_probe_softmax_slot(int32_t lds_operands, int64_t iters, int32_t workgroups, float* sink,
                                   void* stream);

/* Streaming copy of `bytes` (a multiple of 16, 16-byte aligned buffers) from src
   to dst with 16-byte loads (nontemporal) and stores, grid-stride over `workgroups`
   workgroups of 256 threads. */
int32_t omnimem_probe_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream);

/* Streaming read of `bytes` (a multiple of 16, 16-byte aligned) with nontemporal
   16-byte loads; sink as above. */
int32_t omnimem_probe_read(const void* src, int64_t bytes, int32_t workgroups, float* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OMNIMEM_PROBE_H */
