// Host check of the SpMM kernels' payload-range helper (us_range.h): the
// same inline functions the kernels use, compiled for the host. Run by
// tests/test_range_host.py; prints "ok" or the first failing case.
#define __host__
#define __device__
#include <cstdio>
#include <cstdint>
#include "us_range.h"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint64_t next() {                      // xorshift64*
    state ^= state >> 12;
    state ^= state << 25;
    state ^= state >> 27;
    return state * 0x2545F4914F6CDD1Dull;
}

template <int BITS>
static bool check(uint32_t ob, uint32_t oe, uint32_t pay_bytes, uint32_t max_pieces, bool valid) {
    const uint32_t a0 = us_range::first_byte<BITS>(ob, pay_bytes);
    const uint32_t n = us_range::range_bytes<BITS>(oe, a0, pay_bytes, max_pieces);
    // Memory safety, for any offsets: the staged range lies inside the payload.
    bool ok = a0 <= pay_bytes && a0 % 16 == 0 && (uint64_t)a0 + n <= pay_bytes && n % 16 == 0 &&
              n <= 16ull * max_pieces;
    // Coverage, for offsets of a valid encoding: every value of [ob, oe) and
    // the 8 bytes after the dword holding the last value's start are staged
    // (as far as the payload reaches), and the first staged byte is at or
    // before the first value.
    if (valid && ok) {
        const uint64_t first_byte = ((uint64_t)ob * BITS) / 8;
        const uint64_t need = 4 * (((uint64_t)oe * BITS) / 32) + 8;
        const uint64_t have = (uint64_t)a0 + n;
        ok = a0 <= first_byte && have >= (need < pay_bytes ? need : pay_bytes);
    }
    if (!ok)
        std::printf("FAIL bits=%d ob=%u oe=%u pay_bytes=%u max_pieces=%u valid=%d -> a0=%u n=%u\n", BITS, ob, oe,
                    pay_bytes, max_pieces, (int)valid, a0, n);
    return ok;
}

template <int BITS>
static bool run() {
    const uint32_t vpb = 8 / BITS;                         // values per byte
    // Offsets that decrease, and offsets past the end of the payload.
    if (!check<BITS>(4000, 100, 2048, 354, false)) return false;
    if (!check<BITS>(100, 0, 2048, 354, false)) return false;
    if (!check<BITS>(4096 * vpb, 4096 * vpb + 960, 2048, 354, false)) return false;
    if (!check<BITS>(0xFFFFFFF0u, 0xFFFFFFFFu, 2048, 354, false)) return false;
    if (!check<BITS>(0, 0xFFFFFFFFu, 2048, 354, false)) return false;
    if (!check<BITS>(2000 * vpb, 2100 * vpb, 2048, 354, false)) return false;
    if (!check<BITS>(0, 0, 0, 354, true)) return false;   // an empty payload
    for (int it = 0; it < 2000000; ++it) {
        const uint32_t pay = 16 * (uint32_t)(next() % 100000);
        const uint32_t pieces = 1 + (uint32_t)(next() % 1100);
        if (it % 2) {                                      // arbitrary words
            if (!check<BITS>((uint32_t)next(), (uint32_t)next(), pay, pieces, false)) return false;
        } else {                                           // a valid run of LTs within the payload
            const uint64_t nvals = (uint64_t)(pay > 16 ? pay - 16 : 0) * vpb;   // values the payload holds
            const uint32_t ob = nvals ? (uint32_t)(next() % (nvals + 1)) : 0;
            const uint32_t len = (uint32_t)(next() % 1025) * 4;                 // up to one LT, whole groups
            const uint32_t oe = (uint32_t)(ob + len <= nvals ? ob + len : nvals);
            // Enough pieces for the run, as the kernels size their stages.
            const uint32_t need_pieces = (uint32_t)((((uint64_t)(oe - (ob / (16 * vpb)) * 16 * vpb) * BITS / 8) + 8 + 15 + 15) / 16);
            if (!check<BITS>(ob, oe, pay, pieces > need_pieces ? pieces : need_pieces, true)) return false;
        }
    }
    return true;
}

int main() {
    if (!run<4>() || !run<2>()) return 1;
    std::printf("ok\n");
    return 0;
}
