/*
 * ardit_micro.h -- measurement kernels of libardit.
 *
 * Not part of the block's computation: these give the measured denominators
 * that the block kernels' roofline fractions are also reported against, next
 * to the published MI355X peaks (bf16 2.5 PFLOP/s and fp8 5.0 PFLOP/s dense,
 * HBM 8 TB/s), and the fill that flushes the caches before a cold timing.
 * Same conventions as ardit.h (status codes, asynchrony, device pointers).
 */
#ifndef ARDIT_MICRO_H
#define ARDIT_MICRO_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* MFMA throughput: `workgroups` workgroups of 4 waves (two waves per SIMD when
 * the grid covers the GPU), each wave running `iters` iterations of
 * independent accumulator chains on register operands (dtype 0: 8 chains of
 * v_mfma_f32_16x16x32_bf16; dtype 1: 4 chains of the fp8 (E4M3)
 * v_mfma_scale_f32_32x32x64_f8f6f4), then writing one float per thread to
 * sink (device, workgroups * 256 floats) so nothing is elided.  *flops (host)
 * receives the launch's floating-point operations. */
int ardit_micro_mfma(hipStream_t stream, int32_t dtype, int32_t workgroups, int32_t iters,
                     float* sink, double* flops);

/* Device copy: dst = src, `bytes` read and `bytes` written with 16-byte
 * streaming (nontemporal) accesses (16-byte aligned, non-overlapping,
 * bytes % 16 == 0). */
int ardit_micro_copy(hipStream_t stream, const void* src, void* dst, size_t bytes);

/* Device read of `bytes` of src (16-byte aligned, bytes % 16 == 0) with
 * 16-byte loads, four in flight per thread, folded into one 32-bit word per
 * workgroup written to sink (device, 4-byte aligned, sink_bytes at least 4
 * per workgroup: 32 KiB covers any size; ARDIT_EINVAL otherwise). */
int ardit_micro_read(hipStream_t stream, const void* src, size_t bytes, void* sink,
                     size_t sink_bytes);

/* Device fill of `bytes` with a 32-bit value. */
int ardit_micro_fill(hipStream_t stream, void* dst, size_t bytes, uint32_t value);

#ifdef __cplusplus
}
#endif

#endif /* ARDIT_MICRO_H */
