/*
 * delta_probe.h — measurement helper shipped with the DELTA attention library (not part of the
 * method): a streaming read of a device buffer, used to measure the HBM read bandwidth that
 * MI355X delivers, the ceiling the attention kernels' achieved bandwidth is compared with.
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

#ifdef __cplusplus
}
#endif

#endif /* DELTA_PROBE_H */
