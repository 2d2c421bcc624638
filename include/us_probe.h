/*
 * us_probe.h - measurement kernels that ship with the UnionSparse library.
 *
 * They are not part of the paper's method. They give the benchmark its
 * reference points on the same GPU: the streaming-read rate of HBM at the
 * byte count of an encoded matrix (the ceiling a bandwidth-bound SpMM can
 * approach), a plain copy whose byte count calibrates hardware traffic
 * counters, and a bounded busy-wait that lets a host queue many launches
 * before the GPU reaches them, so that launch cost on the host does not
 * appear in GPU-side timings.
 *
 * Same conventions as us.h: device pointers, hipStream_t as void *,
 * asynchronous, no allocation, checked arguments.
 */
#ifndef UNIONSPARSE_US_PROBE_H
#define UNIONSPARSE_US_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include "us.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` (a multiple of 16) from `src` (16-byte aligned) once, with
 * 16-byte loads, and fold them into one uint32 per workgroup at sink[0..]
 * (sink holds us_probe_read_sink_words(bytes) words). */
us_status us_probe_read(const void *src, size_t bytes, uint32_t *sink, void *stream);
size_t us_probe_read_sink_words(size_t bytes);

/* dst[0 .. bytes) = src[0 .. bytes); both 16-byte aligned, bytes % 16 == 0. */
us_status us_probe_copy(const void *src, void *dst, size_t bytes, void *stream);

/* One wavefront spins until `ns` nanoseconds of the GPU's constant-rate clock
 * have passed (at most one second), then exits. */
us_status us_probe_spin(uint64_t ns, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* UNIONSPARSE_US_PROBE_H */
