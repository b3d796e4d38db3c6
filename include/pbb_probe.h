/*
 * pbb_probe.h -- C ABI of libpbbprobe, a measurement helper beside libpbb (not part of the
 * decode method).  It measures the practical HBM read rate of the decode's access pattern on
 * MI355X: every (sequence, KV head) unit streams its first rows[u] rows of a K region and of
 * a V region (256-byte rows, head_dim 128 in bf16) from HBM into LDS with LDS DMA
 * (global_load_lds_dwordx4), 32 rows of each per wave step, two steps in flight per wave, one
 * workgroup of `waves` waves per unit -- the streaming skeleton of the bf16 decode kernel with
 * no arithmetic.  The rate it reaches is the ceiling the decode's ring reads are compared with
 * (the paper profiles its kernels' memory requests the same way, Appendix F.3).
 *
 * Layout: unit u's K rows start at k + u * unit_stride, its V rows at v + u * unit_stride.
 * rows: int32 [units] in device memory; each entry is clamped to [0, max_rows].  Reads never
 * leave [k, k + units * unit_stride) and the same range of v.  The kernel writes `sink[0]` only
 * if the data it read sums to one particular float (so the loads cannot be optimised away).
 *
 * Returns 0 on success, or a nonzero hipError_t code (1 = invalid argument, checked on the host
 * before anything is enqueued: NULL or unaligned pointers, units < 1, waves not 2 or 4,
 * max_rows < 1 or max_rows * 256 > unit_stride).  Asynchronous on `stream` (a hipStream_t).
 */
#ifndef PBB_PROBE_H_
#define PBB_PROBE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int pbb_probe_stream(const void *k, const void *v, size_t unit_stride, const int32_t *rows,
                     int32_t units, int32_t max_rows, int32_t waves, int32_t nontemporal,
                     float *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PBB_PROBE_H_ */
