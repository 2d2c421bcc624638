// Host side of the IE-BME format: encoder (Section V-A), bitmap-aware row
// reordering (Section V-B) and byte accounting (Eq. 1, Eq. 2). Runs offline
// on the CPU, as the paper's format conversion does; its cost is not part of
// the SpMM latency.
#include <algorithm>
#include <atomic>
#include <climits>
#include <cstdlib>
#include <cstring>
#include <thread>
#include <vector>

#include "us.h"

namespace {

constexpr int kAreaH = US_LT_H / US_RA;   // 8 union-mask rows
constexpr int kAreaW = US_LT_W / US_CA;   // 32 union-mask columns

// Run body(lo, hi) over [0, n) on up to hardware_concurrency threads.
template <typename F>
void parallel_ranges(int64_t n, F body) {
    unsigned hw = std::thread::hardware_concurrency();
    int64_t nt = std::max<int64_t>(1, std::min<int64_t>(hw ? hw : 1, (n + 1023) / 1024));
    if (nt == 1) {
        body(int64_t(0), n);
        return;
    }
    std::vector<std::thread> th;
    th.reserve(nt);
    for (int64_t t = 0; t < nt; ++t)
        th.emplace_back([=] { body(n * t / nt, n * (t + 1) / nt); });
    for (auto &x : th) x.join();
}

inline int popcount64(uint64_t v) { return __builtin_popcountll(v); }

// Value of area q at union-mask position (i, j) of an LT whose (possibly
// reordered) rows are `rows`: area q = a * C_A + c covers rows [8a, 8a+8)
// and columns [32c, 32c+32).
inline int8_t area_value(const int8_t *const *rows, int q, int i, int j) {
    const int a = q / US_CA, c = q % US_CA;
    return rows[a * kAreaH + i][c * kAreaW + j];
}

// Bitmap-aware row reordering of one LT (Section V-B) for R_A = C_A = 2.
//
// With two area columns, row r activates grouped column j (Eq. 3) when it is
// nonzero at column j or j + 32: `fold[r]` holds those 32 bits. A pair of
// rows then costs popcount(fold[r] | fold[s]) union-mask entries (Eq. 4),
// and Eq. 5 pairs up all 16 rows at minimum total cost. The DP state is the
// set of rows still unpaired; each step pairs its lowest row with one other
// row, so only row sets reachable that way are visited (1596 of 2^16).
class RowPairing {
public:
    // Canonical permutation: pi[g] and pi[8 + g] are the rows of pair g,
    // pairs sorted by their first row. Returns the minimum cost.
    int solve(const uint32_t fold[US_LT_H], uint8_t pi[US_LT_H]) {
        for (int r = 0; r < US_LT_H; ++r)
            for (int s = 0; s < US_LT_H; ++s) cost_[r][s] = (uint8_t)__builtin_popcount(fold[r] | fold[s]);
        if (++gen_ == 0) {                       // stamps wrapped: forget everything
            std::fill(stamp_.begin(), stamp_.end(), 0u);
            gen_ = 1;
        }
        const uint32_t all = (1u << US_LT_H) - 1u;
        const int total = best(all);
        // The lowest unpaired row grows from step to step, so the pairs come
        // out sorted and each pair's first row is its smaller one.
        uint32_t left = all;
        for (int g = 0; g < US_LT_H / 2; ++g) {
            const int r = __builtin_ctz(left);
            const int s = partner_[left];
            pi[g] = (uint8_t)r;
            pi[US_LT_H / 2 + g] = (uint8_t)s;
            left &= ~((1u << r) | (1u << s));
        }
        return total;
    }

private:
    // F(left): minimum cost of pairing the rows in `left`. Partners are
    // tried in increasing row order and only a strictly lower cost replaces
    // the current choice.
    int best(uint32_t left) {
        if (left == 0) return 0;
        if (stamp_[left] == gen_) return value_[left];
        const int r = __builtin_ctz(left);
        const uint32_t others = left & (left - 1u);
        int min_cost = INT_MAX, arg = -1;
        for (uint32_t x = others; x; x &= x - 1u) {
            const int s = __builtin_ctz(x);
            const int v = cost_[r][s] + best(others & ~(1u << s));
            if (v < min_cost) {
                min_cost = v;
                arg = s;
            }
        }
        stamp_[left] = gen_;
        value_[left] = (uint16_t)min_cost;
        partner_[left] = (uint8_t)arg;
        return min_cost;
    }

    uint8_t cost_[US_LT_H][US_LT_H];
    std::vector<uint32_t> stamp_ = std::vector<uint32_t>(1u << US_LT_H, 0u);
    std::vector<uint16_t> value_ = std::vector<uint16_t>(1u << US_LT_H);
    std::vector<uint8_t> partner_ = std::vector<uint8_t>(1u << US_LT_H);
    uint32_t gen_ = 0;
};

us_status encode_impl(const int8_t *w, int32_t M, int32_t K, int64_t ldw, bool reorder, int bits, us_iebme *out);

}  // namespace

extern "C" const char *us_status_string(us_status s) {
    switch (s) {
        case US_OK: return "ok";
        case US_ERR_ARG: return "invalid argument";
        case US_ERR_SHAPE: return "unsupported shape";
        case US_ERR_RANGE: return "weight outside INT4 range";
        case US_ERR_NOMEM: return "out of host memory";
        case US_ERR_DEVICE: return "HIP launch error";
        case US_ERR_FORMAT: return "inconsistent IE-BME arrays";
    }
    return "unknown status";
}

extern "C" us_status us_encode(const int8_t *w, int32_t M, int32_t K, int64_t ldw, us_iebme *out) {
    return encode_impl(w, M, K, ldw, false, 4, out);
}

extern "C" us_status us_encode_w2(const int8_t *w, int32_t M, int32_t K, int64_t ldw, us_iebme *out) {
    return encode_impl(w, M, K, ldw, false, 2, out);
}

extern "C" us_status us_encode_reordered(const int8_t *w, int32_t M, int32_t K, int64_t ldw, us_iebme *out) {
    return encode_impl(w, M, K, ldw, true, 4, out);
}

namespace {

us_status encode_impl(const int8_t *w, int32_t M, int32_t K, int64_t ldw, bool reorder, int bits, us_iebme *out) {
    if (!w || !out) return US_ERR_ARG;
    if (M <= 0 || K <= 0 || M % US_LT_H || K % US_LT_W) return US_ERR_SHAPE;
    if (ldw < K) return US_ERR_ARG;
    if ((uint64_t)M * (uint64_t)K >= (1ull << 32)) return US_ERR_SHAPE;

    // Every weight must be a signed `bits`-bit value.
    const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
    std::atomic<bool> bad{false};
    parallel_ranges(M, [&](int64_t r0, int64_t r1) {
        for (int64_t r = r0; r < r1 && !bad.load(std::memory_order_relaxed); ++r) {
            const int8_t *row = w + r * ldw;
            for (int32_t k = 0; k < K; ++k)
                if (row[k] < lo || row[k] > hi) { bad = true; break; }
        }
    });
    if (bad) return US_ERR_RANGE;

    const int64_t nkb = K / US_LT_W;
    const int64_t n_lt = (int64_t)(M / US_LT_H) * nkb;
    uint64_t *bitmaps = (uint64_t *)std::calloc((size_t)n_lt * US_WORDS_PER_LT, sizeof(uint64_t));
    uint32_t *offsets = (uint32_t *)std::calloc((size_t)n_lt + 1, sizeof(uint32_t));
    uint64_t *perm = reorder ? (uint64_t *)std::calloc((size_t)n_lt, sizeof(uint64_t)) : nullptr;
    std::vector<uint32_t> P;
    try {
        P.resize((size_t)n_lt);
    } catch (...) {
        std::free(bitmaps);
        std::free(offsets);
        std::free(perm);
        return US_ERR_NOMEM;
    }
    if (!bitmaps || !offsets || (reorder && !perm)) {
        std::free(bitmaps);
        std::free(offsets);
        std::free(perm);
        return US_ERR_NOMEM;
    }

    // Rows of LT t in encoding order: the identity, or pi_t from perm[t].
    auto lt_rows = [&](int64_t t, const int8_t *rows[US_LT_H]) {
        const int8_t *base = w + (t / nkb) * US_LT_H * ldw + (t % nkb) * US_LT_W;
        for (int p = 0; p < US_LT_H; ++p) {
            const int r = perm ? (int)((perm[t] >> (4 * p)) & 0xF) : p;
            rows[p] = base + (int64_t)r * ldw;
        }
    };

    // Pass 1: row reordering (optional), then the shared union mask B_t and
    // P_t = ||B_t||_0 per LT; count nonzeros.
    std::atomic<int64_t> nnz{0};
    std::atomic<bool> oom{false};
    parallel_ranges(n_lt, [&](int64_t t0, int64_t t1) {
        RowPairing *dp = nullptr;
        if (reorder) {
            try {
                dp = new RowPairing();
            } catch (...) {
                oom = true;
                return;
            }
        }
        int64_t local_nnz = 0;
        for (int64_t t = t0; t < t1; ++t) {
            if (dp) {
                const int8_t *base = w + (t / nkb) * US_LT_H * ldw + (t % nkb) * US_LT_W;
                uint32_t fold[US_LT_H];
                for (int r = 0; r < US_LT_H; ++r) {
                    const int8_t *row = base + (int64_t)r * ldw;
                    uint32_t f = 0;
                    for (int j = 0; j < kAreaW; ++j)
                        if (row[j] != 0 || row[kAreaW + j] != 0) f |= 1u << j;
                    fold[r] = f;
                }
                uint8_t pi[US_LT_H];
                dp->solve(fold, pi);
                uint64_t word = 0;
                for (int p = 0; p < US_LT_H; ++p) word |= (uint64_t)pi[p] << (4 * p);
                perm[t] = word;
            }
            const int8_t *rows[US_LT_H];
            lt_rows(t, rows);
            uint64_t *bm = bitmaps + t * US_WORDS_PER_LT;
            uint32_t p = 0;
            for (int i = 0; i < kAreaH; ++i) {
                for (int j = 0; j < kAreaW; ++j) {
                    bool any = false;
                    for (int q = 0; q < US_RA * US_CA; ++q) {
                        const bool nz = area_value(rows, q, i, j) != 0;
                        local_nnz += nz;
                        any |= nz;
                    }
                    if (any) {
                        const int L = i * kAreaW + j;   // row-major, leftmost = LSB
                        bm[L >> 6] |= 1ull << (L & 63);
                        ++p;
                    }
                }
            }
            P[(size_t)t] = p;
        }
        delete dp;
        nnz += local_nnz;
    });
    if (oom) {
        std::free(bitmaps);
        std::free(offsets);
        std::free(perm);
        return US_ERR_NOMEM;
    }

    // Union Value Offsets: o_t = sum over earlier LTs of Q * P_tau.
    uint64_t run = 0;
    for (int64_t t = 0; t < n_lt; ++t) {
        offsets[t] = (uint32_t)run;
        run += (uint64_t)(US_RA * US_CA) * P[(size_t)t];
    }
    offsets[n_lt] = (uint32_t)run;   // run <= M * K < 2^32

    const int per_byte = 8 / bits;                        // values per payload byte
    const int64_t payload_bytes = (int64_t)((run + per_byte - 1) / per_byte) + US_PAYLOAD_PAD;
    uint8_t *payload = (uint8_t *)std::calloc((size_t)payload_bytes, 1);
    if (!payload) {
        std::free(bitmaps);
        std::free(offsets);
        std::free(perm);
        return US_ERR_NOMEM;
    }

    // Pass 2: Compressed Values: area q = a C_A + c's value at (i, j), zeros
    // of active groups included, for every active (i, j) of rank rho. The
    // areas of one area row alternate by rank (value o_t + a C_A P_t +
    // C_A rho + c), so the C_A values a rank selects in an area row sit
    // together; the paper lists each area's values in turn (o_t + q P_t +
    // rho), which holds the same values per LT. Value n takes bits
    // (n mod per_byte) * bits of byte n / per_byte. Each LT starts on a
    // multiple of four values, so LTs never share a byte.
    parallel_ranges(n_lt, [&](int64_t t0, int64_t t1) {
        for (int64_t t = t0; t < t1; ++t) {
            const int8_t *rows[US_LT_H];
            lt_rows(t, rows);
            const uint64_t *bm = bitmaps + t * US_WORDS_PER_LT;
            const uint64_t o = offsets[t];
            const uint64_t Pt = P[(size_t)t];
            uint64_t rho = 0;
            for (int L = 0; L < kAreaH * kAreaW; ++L) {
                if (!((bm[L >> 6] >> (L & 63)) & 1)) continue;
                const int i = L / kAreaW, j = L % kAreaW;
                for (int q = 0; q < US_RA * US_CA; ++q) {
                    const uint64_t n = o + (uint64_t)(q / US_CA) * US_CA * Pt + (uint64_t)US_CA * rho + (q % US_CA);
                    const uint8_t v = (uint8_t)area_value(rows, q, i, j) & (uint8_t)((1 << bits) - 1);
                    payload[n / per_byte] |= (uint8_t)(v << ((n % per_byte) * bits));
                }
                ++rho;
            }
        }
    });

    out->M = M;
    out->K = K;
    out->lt_h = US_LT_H;
    out->lt_w = US_LT_W;
    out->ra = US_RA;
    out->ca = US_CA;
    out->n_lt = n_lt;
    out->nnz = nnz.load();
    out->n_payload = (int64_t)run;
    out->payload_bytes = payload_bytes;
    out->bitmaps = bitmaps;
    out->offsets = offsets;
    out->payload = payload;
    out->perm = perm;
    out->bits = bits;
    return US_OK;
}

}  // namespace

extern "C" void us_iebme_free(us_iebme *m) {
    if (!m) return;
    std::free(m->bitmaps);
    std::free(m->offsets);
    std::free(m->payload);
    std::free(m->perm);
    std::memset(m, 0, sizeof(*m));
}

extern "C" us_status us_pmr(const us_iebme *m, int32_t N, us_pmr_report *out) {
    if (!m || !out || !m->bitmaps || !m->offsets) return US_ERR_ARG;
    if (N < 0) return US_ERR_ARG;
    if (m->M <= 0 || m->K <= 0 || m->M % US_LT_H || m->K % US_LT_W) return US_ERR_SHAPE;
    if (m->lt_h != US_LT_H || m->lt_w != US_LT_W || m->ra != US_RA || m->ca != US_CA)
        return US_ERR_FORMAT;
    const int64_t n_lt = (int64_t)(m->M / US_LT_H) * (m->K / US_LT_W);
    if (m->n_lt != n_lt) return US_ERR_FORMAT;

    // offsets[t + 1] - offsets[t] must be Q times the LT's union-mask popcount.
    if (m->offsets[0] != 0) return US_ERR_FORMAT;
    for (int64_t t = 0; t < n_lt; ++t) {
        int p = 0;
        for (int k = 0; k < US_WORDS_PER_LT; ++k) p += popcount64(m->bitmaps[t * US_WORDS_PER_LT + k]);
        if ((uint64_t)m->offsets[t + 1] != (uint64_t)m->offsets[t] + (uint64_t)(US_RA * US_CA) * p)
            return US_ERR_FORMAT;
    }
    if ((int64_t)m->offsets[n_lt] != m->n_payload) return US_ERR_FORMAT;
    if (m->nnz < 0 || m->nnz > m->n_payload) return US_ERR_FORMAT;

    const int bits = m->bits == 0 ? 4 : m->bits;
    if (bits != 4 && bits != 2) return US_ERR_FORMAT;
    const double bw = bits / 8.0;   // bytes per weight (B_w)
    us_pmr_report r;
    std::memset(&r, 0, sizeof(r));
    r.nnz = m->nnz;
    r.stored_values = m->n_payload;
    r.n_lt = n_lt;
    r.payload_stored_bytes = (m->n_payload * bits + 7) / 8;
    r.bitmap_bytes = 8 * US_WORDS_PER_LT * n_lt;
    r.offset_bytes = 4 * n_lt;
    r.meta_bytes = r.bitmap_bytes + r.offset_bytes;
    r.payload_useful_bytes = bw * (double)m->nnz;
    r.pmr = r.payload_useful_bytes / (double)r.meta_bytes;
    r.pmr_stored = bw * (double)m->n_payload / (double)r.meta_bytes;
    r.perm_bytes = m->perm ? 8 * n_lt : 0;
    if (N > 0 && m->nnz > 0) {
        // Eq. 2 as printed: 2 M N (1-s) / (B_w M (1-s)(1 + 1/PMR) + B_w N).
        const double keep = (double)m->nnz / ((double)m->M * (double)m->K);
        const double Md = m->M, Nd = N;
        r.ci_eff = 2.0 * Md * Nd * keep / (bw * Md * keep * (1.0 + 1.0 / r.pmr) + bw * Nd);
    }
    *out = r;
    return US_OK;
}

extern "C" us_status us_pmr_formats(const us_iebme *m, int32_t value_bits, int32_t N,
                                    us_format_report out[US_NUM_FORMATS]) {
    if (!out || N < 1) return US_ERR_ARG;
    if (value_bits != 16 && value_bits != 8 && value_bits != 4 && value_bits != 2) return US_ERR_ARG;
    us_pmr_report base;
    const us_status st = us_pmr(m, 0, &base);          // validates the arrays
    if (st != US_OK) return st;

    const double bw = value_bits / 8.0;                // B_w
    const double M = m->M, K = m->K, Nd = N;
    const double nnz = (double)m->nnz;
    const double keep = nnz / (M * K);                 // 1 - s
    // Eq. 2 as printed: 2 M N (1-s) / (B_w M (1-s) (1 + 1/PMR) + B_w N);
    // with no metadata the 1/PMR term is absent.
    auto ci = [&](double keep_, double pmr) {
        const double inflation = pmr > 0.0 ? 1.0 + 1.0 / pmr : 1.0;
        const double den = bw * M * keep_ * inflation + bw * Nd;
        return den > 0.0 ? 2.0 * M * Nd * keep_ / den : 0.0;
    };
    const int64_t n_lt = base.n_lt;
    for (int f = 0; f < US_NUM_FORMATS; ++f) {
        us_format_report r;
        std::memset(&r, 0, sizeof(r));
        r.format = f;
        r.value_bits = value_bits;
        switch (f) {
            case US_FMT_DENSE:
                r.meta_bytes = 0;
                r.payload_useful_bytes = bw * M * K;
                r.payload_stored_bytes = bw * M * K;
                r.pmr = 0.0;
                r.ci_eff = ci(1.0, 0.0);
                break;
            case US_FMT_CSR:
                r.meta_bytes = 4 * m->nnz + 4 * ((int64_t)m->M + 1);
                r.payload_useful_bytes = bw * nnz;
                r.payload_stored_bytes = bw * nnz;
                break;
            case US_FMT_AREA_BITMAP:
                r.meta_bytes = (int64_t)(US_RA * US_CA) * (32 + 4) * n_lt;
                r.payload_useful_bytes = bw * nnz;
                r.payload_stored_bytes = bw * nnz;
                break;
            default:
                r.meta_bytes = base.meta_bytes;
                r.payload_useful_bytes = bw * nnz;
                r.payload_stored_bytes = bw * (double)m->n_payload;
                break;
        }
        if (f != US_FMT_DENSE) {
            r.pmr = r.meta_bytes > 0 ? r.payload_useful_bytes / (double)r.meta_bytes : 0.0;
            r.ci_eff = keep > 0.0 ? ci(keep, r.pmr) : 0.0;
        }
        r.total_bytes = (double)r.meta_bytes + r.payload_stored_bytes;
        const double macs = f == US_FMT_DENSE ? M * K : nnz;
        r.ci_stored = 2.0 * macs * Nd / (r.total_bytes + bw * Nd * K);
        out[f] = r;
    }
    return US_OK;
}
