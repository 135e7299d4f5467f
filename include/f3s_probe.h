/*
 * f3s_probe.h -- memory-system probes of libf3s.so (measurement aids, not
 * part of the operator).
 *
 * The fused operator is bound by memory bandwidth (its arithmetic intensity
 * is about 1 flop per byte, far below the GPU's ridge point), so its speed
 * is judged against what the memory system delivers.  These calls measure
 * that in the caller's process, with kernels of the same build:
 *   f3s_probe_read / _copy / _write   what HBM delivers to plain streaming
 *       kernels (16-byte accesses, coalesced, one pass); over a buffer much
 *       larger than the 256 MB Infinity Cache this is the achievable DRAM
 *       bandwidth of the device.
 *   f3s_probe_gather                  the fused kernel's memory accesses on
 *       a plan (Q rows, column ids, bitmaps, the K and V rows of every block,
 *       16 x d fp32 results per work item), in the same order and
 *       granularity, with no arithmetic and more waves in flight: the
 *       ceiling of that access pattern, from the caches and HBM together.
 * All calls are asynchronous on `stream`, allocate nothing and return
 * F3S_ERR_INVALID_VALUE for a null or misaligned (16-byte) pointer or a
 * size that is not a multiple of 16 bytes.
 */
#ifndef F3S_PROBE_H
#define F3S_PROBE_H

#include "f3s.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` of device memory at src once; `sink` is device memory of
 * 256 uint32 that the kernel may write (it practically never does; the
 * dependency keeps the loads). */
f3s_status_t f3s_probe_read(const void *src, size_t bytes, uint32_t *sink,
                            hipStream_t stream);

/* Copies `bytes` from src to dst (device memory, not overlapping). */
f3s_status_t f3s_probe_copy(const void *src, void *dst, size_t bytes, hipStream_t stream);

/* Writes `bytes` at dst (a pattern derived from value). */
f3s_status_t f3s_probe_write(void *dst, size_t bytes, uint32_t value, hipStream_t stream);

/* The access pattern of f3s_run(plan, Q, K, V, O, d, ...) for fp16 Q, K, V
 * [N, d] and fp32 O [N, d] without its arithmetic; d in {32, 64, 128, 256}
 * (else F3S_ERR_UNSUPPORTED).  O (and the plan's partial buffers, for split
 * windows) receive meaningless values. */
f3s_status_t f3s_probe_gather(f3s_plan_t plan, const void *Q, const void *K, const void *V,
                              float *O, int32_t d, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* F3S_PROBE_H */
