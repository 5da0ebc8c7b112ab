/*
 * mg3m_measure.h -- measurement kernels shipped with the convolution library.
 *
 * Not part of the convolution: they give the benchmark the machine's own
 * ceilings to set the convolution's numbers against (the hardware-efficiency
 * metric of Sec. 5, runtime performance over theoretical peak, needs both the
 * nominal peak and what the chip sustains):
 *   - an empty kernel, whose launch-to-launch time is the floor under any
 *     layer that runs for a few microseconds (launch-latency-bound layers);
 *   - an fp32-MFMA-only kernel (no memory traffic in its loop), the sustained
 *     fp32 matrix-core rate under a full chip of waves;
 *   - a copy and a fill kernel (16-byte accesses, four in flight per
 *     thread, one 16 KB block per work-group), the HBM bandwidth a streaming
 *     kernel reaches (read + write, write only).
 *
 * Pointers are DEVICE pointers on the current HIP device; stream is a
 * hipStream_t (NULL = the default stream); every call only queues work.
 * Return values are mg3m_status codes (mg3m.h); HIP launch errors return
 * MG3M_ERR_HIP with the text in mg3m_last_error().
 */
#ifndef MG3M_MEASURE_H
#define MG3M_MEASURE_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One work-group of 64 threads that does nothing. */
int mg3m_launch_empty(void *stream);

/* blocks work-groups of four waves; each wave issues iters rounds of eight
 * independent v_mfma_f32_32x32x2_f32 on register operands and finally writes
 * one float per thread to sink[blocks * 256] (caller-owned, that many floats,
 * so the results stay live).  *flops: host out-parameter, the fp32 flops the
 * launch performs (blocks * 4 * iters * 8 * 4096).  blocks 1..2^20, iters
 * 1..2^24, else MG3M_ERR_ARG; sink and flops non-NULL, else MG3M_ERR_NULL. */
int mg3m_probe_mfma_f32(float *sink, int blocks, int iters, void *stream, double *flops);

/* dst[i] = src[i] over `bytes` bytes: 16-byte loads and stores.
 * bytes a positive multiple of 16, src and dst 16-byte aligned and not
 * overlapping, else MG3M_ERR_ARG / MG3M_ERR_ALIGN / MG3M_ERR_ALIAS. */
int mg3m_probe_copy(const void *src, void *dst, size_t bytes, void *stream);

/* dst[i] = 0 over `bytes` bytes: 16-byte stores.  bytes a
 * positive multiple of 16 and dst 16-byte aligned, else MG3M_ERR_ARG /
 * MG3M_ERR_ALIGN. */
int mg3m_probe_fill(void *dst, size_t bytes, void *stream);

/* Timing events: hipEvent_t handles that record timestamps without the
 * system-scope memory fence a default HIP event performs when it is reached.
 * That fence writes back and invalidates the GPU's caches at every event, a
 * cost the timed work would otherwise pay between kernels; these events only
 * time, they do not order host reads of device memory.  Create (into *event,
 * on the current device), record on a stream (NULL = the default stream),
 * read the milliseconds between two recorded events once both have
 * completed (after a synchronisation), destroy.  The handles also serve
 * mg3m_time_next_kernel.  NULL handles or outputs: MG3M_ERR_NULL; HIP
 * failures: MG3M_ERR_HIP with the text in mg3m_last_error(). */
int mg3m_timing_event_create(void **event);
int mg3m_timing_event_record(void *event, void *stream);
int mg3m_timing_event_elapsed_ms(void *start, void *stop, float *ms);
int mg3m_timing_event_destroy(void *event);

#ifdef __cplusplus
}
#endif

#endif /* MG3M_MEASURE_H */
