/*
 * cq_measure.h -- measurement aids exported by libcq.so beside the C ABI of
 * cq.h.  They are not part of the CubicQuant method: a benchmark uses them to
 * state the hardware ceilings its kernels are compared with.
 */
#ifndef CQ_MEASURE_H
#define CQ_MEASURE_H

#include "cq.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * cq_probe_read -- read `bytes` of device memory at
 * `buf` once, as a plain streaming kernel, so that a benchmark can state the
 * HBM read ceiling its weight-streaming kernels are compared with.  buf is
 * 16-byte aligned and bytes a multiple of 16 (else CQ_ERR_ALIGN / CQ_ERR_ARG);
 * sink is a caller-owned device word the kernel writes only in a case that
 * does not arise for real data (it keeps the loads from being removed).
 */
cq_status cq_probe_read(const void *buf, int64_t bytes, uint32_t *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* CQ_MEASURE_H */
