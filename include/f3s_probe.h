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
 *   f3s_probe_gather_lds              the same accesses with the K and V
 *       rows loaded straight into LDS and never waited for: the pattern's
 *       rate with as many rows in flight as the hardware allows.
 *   f3s_probe_rows                    uniformly random whole-row gathers from
 *       a table: the hardware's rate for gather-bound work whose working set
 *       is the table, independent of the operator's own access pattern.
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

/* f3s_probe_gather with the K and V chunks loaded into LDS (16 bytes per
 * lane, global-to-LDS loads) instead of registers: each wave issues the
 * loads of its block pairs one pair after another without waiting for any,
 * all into one LDS area that is read once at the end, so nothing but the
 * hardware's count of outstanding loads bounds the rows in flight.  An upper
 * bound for a kernel that gathers into LDS, which must keep each pair there
 * until it is used.  d in {32, 64, 128} and Q, K, V below 4 GiB, else
 * F3S_ERR_UNSUPPORTED.  O receives meaningless values. */
f3s_status_t f3s_probe_gather_lds(f3s_plan_t plan, const void *Q, const void *K,
                                  const void *V, float *O, int32_t d, hipStream_t stream);

/*
 * Random row gathers: `rows` rows of `row_bytes` bytes (16, 32, 64, 128, 256,
 * 512 or 1024) at table, read in 16-byte pieces by row_bytes / 16
 * consecutive lanes each.  The launch has `workgroups` workgroups of 256
 * threads; every group of lanes reads in_flight * rounds rows, each chosen
 * uniformly from the table by a fixed integer hash of the group and the
 * step, in_flight (1, 2, 4, 8 or 16) of them in flight at a time.  Every
 * call reads exactly workgroups * rounds * in_flight * 4096 bytes (16 bytes
 * per thread and row).  sink: device memory of 256 uint32 that the kernel
 * may write (it practically never does).  rows >= 1 and < 2^32, workgroups
 * in [1, 2^31 - 1], rounds >= 1; a row size or in_flight outside the lists
 * gives F3S_ERR_UNSUPPORTED.
 */
f3s_status_t f3s_probe_rows(const void *table, int64_t rows, int32_t row_bytes,
                            int32_t in_flight, int32_t workgroups, int32_t rounds,
                            uint32_t *sink, hipStream_t stream);

/*
 * f3s_run(plan, Q, K, V, O, d, scale, stream) with a record of where and when
 * each workgroup ran: the load-balance view of the paper's per-SM active
 * time (Section 4.3, row-window reordering), for one head, fp16 in, fp32 out.
 * O receives exactly f3s_run's result.  trace: device memory of at least
 * 32 * n_items bytes (f3s_plan_info), 16-byte aligned; record k (workgroup
 * k = work item k of the launch order) holds eight uint32:
 *   [0], [1]  start time, low and high word   (constant clock; see
 *   [2], [3]  end time, low and high word      f3s_wall_clock_khz)
 *   [4]       the HW_ID register: CU id bits 8-11, shader array bit 12,
 *             shader engine bits 13-15
 *   [5]       the XCC_ID register (bits 0-3: which accelerator die)
 *   [6]       workgroup index, [7] 0
 * Patterns whose Q, K, V exceed 4 GiB give F3S_ERR_UNSUPPORTED; a short or
 * misaligned trace buffer F3S_ERR_INVALID_VALUE.  Otherwise as f3s_run.
 */
f3s_status_t f3s_run_trace(f3s_plan_t plan, const void *Q, const void *K, const void *V,
                           float *O, int32_t d, float scale, uint32_t *trace,
                           size_t trace_bytes, hipStream_t stream);

/* Frequency of the constant clock of the trace records on `device`, in kHz
 * (0 if the query fails). */
int32_t f3s_wall_clock_khz(int32_t device);

#ifdef __cplusplus
}
#endif

#endif /* F3S_PROBE_H */
