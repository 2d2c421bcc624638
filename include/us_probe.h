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

/* Launch shapes of us_probe_read: 0 = 256 threads per workgroup, 4 loads
 * issued together, 8 workgroups per compute unit; 1 = 512, 4, 1; 2 = 1024,
 * 4, 8; 3 = 256, 8, 1. No one shape is fastest at every size, so the read
 * ceiling at a byte count is the fastest of them. */
#define US_PROBE_READ_SHAPES 4

/* Read `bytes` (a multiple of 16) from `src` (16-byte aligned) once, with
 * non-temporal 16-byte loads in launch shape `shape` (0 ..
 * US_PROBE_READ_SHAPES - 1), and fold them by XOR into one uint32 per
 * wavefront at sink[wavefront index]. sink holds
 * us_probe_read_sink_words(bytes) words, enough for every shape; on a
 * zeroed sink the XOR of all its words is the XOR of the data. US_ERR_ARG
 * for a null pointer, bad size or alignment, or an unknown shape. */
us_status us_probe_read(const void *src, size_t bytes, uint32_t *sink, int32_t shape, void *stream);
size_t us_probe_read_sink_words(size_t bytes);

/* dst[0 .. bytes) = src[0 .. bytes); both 16-byte aligned, bytes % 16 == 0. */
us_status us_probe_copy(const void *src, void *dst, size_t bytes, void *stream);

/* The same copy, reading `src` with the loads the SpMM kernels stage their
 * payload with (non-temporal 16-byte buffer loads straight into LDS), then
 * storing from LDS; bytes at most 2 GiB. It calibrates HBM read counters for
 * that kind of load. US_ERR_ARG as us_probe_copy, or for a larger size. */
us_status us_probe_copy_lds(const void *src, void *dst, size_t bytes, void *stream);

/* One wavefront spins until `ns` nanoseconds of the GPU's constant-rate clock
 * have passed (at most one second), then exits. */
us_status us_probe_spin(uint64_t ns, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* UNIONSPARSE_US_PROBE_H */
