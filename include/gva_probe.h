/*
 * gva_probe.h -- measurement helper exported by libgva.so: the achievable
 * HBM streaming-read bandwidth of the device, the ceiling the decode
 * kernels' bandwidth is compared with beside the published HBM3E peak.
 * It is not part of the decode path.
 */
#ifndef GVA_PROBE_H_
#define GVA_PROBE_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * gva_probe_read -- enqueue one read of the first floor(bytes/16)*16 bytes
 * of the device buffer `buf` by `workgroups` workgroups of 256 threads,
 * each lane with four 16-byte non-temporal loads in flight.  `sink` is a
 * device unsigned the kernel may write (it never does for realistic data;
 * the write only keeps the loads alive).  Time it with events on `stream`.
 * buf 16-byte aligned, sink 4-byte aligned.  The caller owns both.
 * Returns 0 (ok), -1 (invalid argument) or -3 (HIP launch error), the
 * gva_status values of gva.h.
 */
int gva_probe_read(const void* buf, int64_t bytes, int32_t workgroups, unsigned* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GVA_PROBE_H_ */
