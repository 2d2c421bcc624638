// Payload bytes a wavefront stages for a run of LTs, from the run's first and
// end offsets (Section V-A: LT t's values are [o_t, o_{t+1}) of the
// compressed-values array, counted in values). Used by the SpMM kernels on
// the device and by a host test; the including file provides __host__ and
// __device__ (the HIP runtime, or empty definitions in a host build).
//
// The arithmetic saturates: offsets that decrease, or that point past the
// payload, give a range that starts at most at the end of the payload and
// ends inside it, so the buffer descriptor built from it never addresses
// memory outside the payload allocation. Such offsets are not a valid
// encoding and their Y is unspecified; only the memory safety is guaranteed.
#ifndef UNIONSPARSE_US_RANGE_H
#define UNIONSPARSE_US_RANGE_H

#include <stdint.h>

namespace us_range {

// First staged byte: the byte holding value `ob`, rounded down to 16 bytes,
// and never past `pay_bytes` (a multiple of 16, the staged payload size).
template <int BITS>
__host__ __device__ inline uint32_t first_byte(uint32_t ob, uint32_t pay_bytes) {
    constexpr int kValShift = BITS == 4 ? 1 : 2;          // log2(values per byte)
    const uint32_t a0 = (ob >> kValShift) & ~15u;
    return a0 < pay_bytes ? a0 : pay_bytes;
}

// Bytes from `a0` that a run ending at value `oe` needs: its values plus the
// 8-byte overhang of its last 32-bit window, in whole 16-byte pieces, at most
// `max_pieces` of them and never past `pay_bytes`. Zero when `oe` lies before
// the first staged value or `a0` is at the end of the payload.
template <int BITS>
__host__ __device__ inline uint32_t range_bytes(uint32_t oe, uint32_t a0, uint32_t pay_bytes, uint32_t max_pieces) {
    constexpr int kValShift = BITS == 4 ? 1 : 2;
    const uint64_t first = (uint64_t)a0 << kValShift;     // value index of the first staged byte
    if (a0 >= pay_bytes || (uint64_t)oe < first) return 0u;
    const uint64_t span = (((((uint64_t)oe - first) * (uint64_t)BITS) >> 5) << 2) + 8u;
    uint64_t nq = (span + 15u) >> 4;
    if (nq > max_pieces) nq = max_pieces;
    const uint64_t room = (uint64_t)(pay_bytes - a0);
    return (uint32_t)(16u * nq < room ? 16u * nq : room);
}

}  // namespace us_range

#endif  // UNIONSPARSE_US_RANGE_H
