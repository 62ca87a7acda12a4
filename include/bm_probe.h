/*
 * bm_probe.h -- roofline probes of libbatchmax.so (measurement only).
 *
 * The roofline fractions of the attention kernels are taken against the
 * published MI355X peaks (8 TB/s HBM, 2.5 PFLOP/s dense bf16 MFMA).  These two
 * kernels measure what one device actually sustains on the same two
 * resources, as context for those fractions: a plain streaming read of device
 * memory, and a loop of independent bf16 MFMAs with no memory traffic.  Both
 * enqueue one kernel on `stream` and return at once; time them with events on
 * that stream.  They compute nothing of the method (Sec. 3 of the paper has no
 * counterpart); no device memory is allocated.
 */
#ifndef BM_PROBE_H
#define BM_PROBE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` bytes at `src` (device memory, 16-byte aligned, bytes a
 * multiple of 16) once, 16 bytes per lane, `blocks` workgroups of 256 threads
 * striding over the buffer; each workgroup writes one 32-bit word of the XOR of
 * what it read to sink[blockIdx] (`sink`: `blocks` words of device memory), so
 * the loads cannot be dropped.  nontemporal = 1 marks the loads as streaming
 * (not kept in the caches).  BM_ERR_INVALID_ARG for a null pointer, a
 * misaligned address or size, or blocks < 1. */
int bm_probe_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t blocks,
                         int32_t nontemporal, hipStream_t stream);

/* `blocks` workgroups of 256 threads; every wave issues `iters` rounds of four
 * independent v_mfma_f32_32x32x16_bf16 (4 accumulators, operands in
 * registers, no memory traffic in the loop) and writes one float per wave to
 * sink (blocks * 4 floats).  Work: blocks * 4 waves * iters * 4 * 32768
 * flops.  BM_ERR_INVALID_ARG for a null sink, blocks < 1 or iters < 1. */
int bm_probe_mfma(int32_t iters, float* sink, int32_t blocks, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* BM_PROBE_H */
