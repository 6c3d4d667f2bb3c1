/*
 * delta_probe.h — measurement helpers shipped with the DELTA attention library (not part of the
 * method): a streaming read of a device buffer and a gather of 4 KB chunks from it, used to
 * measure the HBM read bandwidth that MI355X delivers to these two access patterns, the
 * ceilings the attention kernels' achieved bandwidth is compared with.
 */
#ifndef DELTA_PROBE_H
#define DELTA_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` bytes (rounded down to 16) of device buffer `buf` (16-byte aligned) with
 * `n_workgroups` workgroups of 256 threads, each streaming its own contiguous share with
 * non-temporal loads, each thread keeping `unroll` (1, 2, 4 or 8) 16-byte loads in flight, and
 * writes one word per workgroup to device array sink[n_workgroups].  Enqueued on `stream` (hipStream_t as void*); no synchronisation.
 * Returns 0, -1 for a bad argument (nothing enqueued), -4 if the launch failed. */
int delta_hbm_read_probe(const void* buf, size_t bytes, uint32_t* sink, int32_t n_workgroups,
                         int32_t unroll, void* stream);

/* Gathers n_chunks 4 KB chunks of device buffer `buf` (`bytes` long, 16-byte aligned): chunk i
 * is bytes [4096 * chunks[i], 4096 * chunks[i] + 4096) (chunks: device int64 array, every entry
 * in [0, bytes / 4096)).  The chunks are split evenly over `n_workgroups` workgroups of 256
 * threads (at most 4096 chunks each); a workgroup reads its chunks in list order, one 16-byte
 * non-temporal load per thread and chunk, each thread keeping the loads of its next two chunks in
 * flight (the access pattern of the attention kernels' page tiles), and writes one word per
 * thread to device array sink[n_workgroups * 256].  Enqueued on `stream`; no synchronisation.
 * Returns 0, -1 for a bad argument (nothing enqueued; the entries of `chunks` are not checked),
 * -4 if the launch failed. */
int delta_hbm_gather_probe(const void* buf, size_t bytes, const int64_t* chunks, int32_t n_chunks,
                           uint32_t* sink, int32_t n_workgroups, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DELTA_PROBE_H */
