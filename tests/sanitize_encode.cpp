// Host-side entry points of the library (encoders, byte accounting, free) built
// with AddressSanitizer and UBSan by test_encoder_sanitized.py: every encoder
// mode over edge sparsities and padded leading dimensions, then the error
// paths. Exits non-zero on a failed expectation; the sanitizers abort on a
// memory or undefined-behaviour error.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include "us.h"
static int fails = 0;
#define EXPECT(c) do { if (!(c)) { printf("FAIL %s line %d\n", #c, __LINE__); ++fails; } } while (0)
static std::vector<int8_t> mat(int M, int K, int64_t ld, double s, int lo, int hi, unsigned seed) {
    std::mt19937 r(seed); std::uniform_real_distribution<double> u(0, 1); std::uniform_int_distribution<int> v(lo, hi);
    std::vector<int8_t> w((size_t)M * ld, 77);   // padding columns hold an out-of-range value: must be ignored
    for (int m = 0; m < M; ++m) for (int k = 0; k < K; ++k) { int x = 0; if (u(r) >= s) { do x = v(r); while (x == 0); } w[(size_t)m * ld + k] = (int8_t)x; }
    return w;
}
static void run(int M, int K, int64_t ld, double s, int bits, bool reorder, unsigned seed) {
    auto w = mat(M, K, ld, s, bits == 2 ? -2 : -8, bits == 2 ? 1 : 7, seed);
    us_iebme e{};
    us_status st = bits == 2 ? us_encode_w2(w.data(), M, K, ld, &e) : reorder ? us_encode_reordered(w.data(), M, K, ld, &e) : us_encode(w.data(), M, K, ld, &e);
    EXPECT(st == US_OK);
    if (st != US_OK) return;
    // touch every array end to end
    uint64_t acc = 0;
    for (int64_t i = 0; i < e.n_lt * 4; ++i) acc ^= e.bitmaps[i];
    for (int64_t i = 0; i <= e.n_lt; ++i) acc ^= e.offsets[i];
    for (int64_t i = 0; i < e.payload_bytes; ++i) acc ^= e.payload[i];
    if (e.perm) for (int64_t i = 0; i < e.n_lt; ++i) acc ^= e.perm[i];
    us_pmr_report pr; EXPECT(us_pmr(&e, 8, &pr) == US_OK); EXPECT(us_pmr(&e, 0, &pr) == US_OK);
    us_format_report fr[US_NUM_FORMATS];
    for (int vb : {16, 8, 4, 2}) EXPECT(us_pmr_formats(&e, vb, 8, fr) == US_OK);
    us_iebme_free(&e);
    us_iebme_free(&e);          // freeing twice is allowed (the struct was zeroed)
    if (acc == 0x123456789ull) printf(".");
}
int main() {
    const double sp[] = {0.0, 0.3, 0.5, 0.7, 0.95, 1.0};
    unsigned seed = 1;
    for (auto [M, K] : std::vector<std::pair<int, int>>{{16, 64}, {32, 128}, {48, 640}, {16, 8128}, {80, 2560}, {128, 1536}})
        for (double s : sp)
            for (int64_t pad : {0, 13})
                for (int mode = 0; mode < 3; ++mode)
                    run(M, K, K + pad, s, mode == 2 ? 2 : 4, mode == 1, seed++);
    // error paths
    std::vector<int8_t> w(64 * 64, 0);
    us_iebme e{};
    EXPECT(us_encode(nullptr, 16, 64, 64, &e) != US_OK);
    EXPECT(us_encode(w.data(), 16, 64, 64, nullptr) != US_OK);
    EXPECT(us_encode(w.data(), 15, 64, 64, &e) == US_ERR_SHAPE);
    EXPECT(us_encode(w.data(), 16, 63, 64, &e) == US_ERR_SHAPE);
    EXPECT(us_encode(w.data(), 16, 64, 32, &e) != US_OK);
    w[5] = 8; EXPECT(us_encode(w.data(), 16, 64, 64, &e) == US_ERR_RANGE);
    w[5] = 2; EXPECT(us_encode_w2(w.data(), 16, 64, 64, &e) == US_ERR_RANGE);
    w[5] = -9; EXPECT(us_encode_reordered(w.data(), 16, 64, 64, &e) == US_ERR_RANGE);
    EXPECT(us_pmr(nullptr, 8, nullptr) != US_OK);
    for (int s = -7; s <= 0; ++s) EXPECT(us_status_string((us_status)s) != nullptr);
    printf("done, %d failures\n", fails);
    return fails != 0;
}
