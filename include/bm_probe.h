/*
 * bm_probe.h -- roofline probes and the prefill timeline of libbatchmax.so
 * (measurement only).
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
 * striding over the buffer, eight loads per lane in flight; each workgroup writes one 32-bit word of the XOR of
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

/* Prefill timeline (measurement only).  In a library built with
 * BM_PREFILL_TIMELINE defined (`python -m paper_2412_05693_amd.build
 * --timeline` writes libbatchmax_timeline.so), thread 0 of every prefill
 * attention workgroup records the device's constant-rate real-time counter
 * (s_memrealtime, 100 MHz) at fixed points of its run, plus the time it
 * spent at three kinds of waits, into a device array of
 * BM_TIMELINE_MAX_RECORDS records of BM_TIMELINE_FIELDS 64-bit words (record
 * i = workgroup i of the launch; workgroups past the array record nothing);
 * every prefill launch overwrites the records of the one before.  The
 * ordinary library records nothing.  Field meanings, by index: */
#define BM_TIMELINE_FIELDS 16
#define BM_TIMELINE_MAX_RECORDS 65536
enum {
  BM_TL_ENTRY = 0,          /* first instruction of the workgroup */
  BM_TL_QUERY_ISSUED = 1,   /* its query loads issued */
  BM_TL_COPIES_ISSUED = 2,  /* its first tile copies issued */
  BM_TL_FIRST_TILE = 3,     /* first tiles in LDS, block rows appended, barrier passed */
  BM_TL_SWEEP1_END = 4,     /* online-softmax sweep done */
  BM_TL_OUTPUT_STORED = 5,  /* output rows stored */
  BM_TL_SWEEP2_START = 6,   /* column-sum sweep's first logits computed */
  BM_TL_END = 7,            /* last partial sums written */
  BM_TL_S1_COPY_ISSUE = 8,  /* ticks spent issuing tile copies in sweep 1 */
  BM_TL_S1_WAIT = 9,        /* ticks waiting for copies at sweep-1 tile ends */
  BM_TL_S1_BARRIER = 10,    /* ticks in sweep-1 barriers */
  BM_TL_S2_WAIT = 11,       /* the same two for sweep 2 */
  BM_TL_S2_BARRIER = 12,
  BM_TL_HW_ID = 13,         /* HW_ID register (compute unit, shader array and engine) in
                               the low 32 bits, XCC_ID (the XCD) in the high 32 bits */
  BM_TL_ITEM = 14,          /* (unit << 32) | position tile of the workgroup */
  BM_TL_TILES = 15          /* key tiles of the workgroup */
};

/* Copy the first n_records records of the last prefill launch to host
 * memory dst (n_records * BM_TIMELINE_FIELDS words); synchronises the device.
 * BM_ERR_UNSUPPORTED from a library built without BM_PREFILL_TIMELINE,
 * BM_ERR_INVALID_ARG for a null dst or n_records outside
 * [1, BM_TIMELINE_MAX_RECORDS]. */
int bm_prefill_timeline(uint64_t* dst, int32_t n_records);

#ifdef __cplusplus
}
#endif

#endif /* BM_PROBE_H */
