// Host side of the IE-BME SpMM (Section VI, "UnionSparse Kernel"
// algorithm): argument checks, the choice of split and chunk configuration,
// and the launch. The kernel is in us_spmm_kernel.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>

#include "us.h"
#include "us_spmm_kernel.h"

namespace {

using namespace us_spmm_detail;

bool aligned(const void *ptr, uintptr_t n) { return ((uintptr_t)ptr % n) == 0; }

bool chunk_option_ok(int ch) { return ch == 0 || ch == 4 || ch == 8 || ch == 11 || ch == 16; }

// Wavefronts per workgroup (= K slices per row block) and chunk
// configuration, by a cost model of the kernel's time per CU, summed over
// the generations of resident workgroups that a CU runs one after another:
//   generation cost = 40 + chunks per slice * (20 + LTs per chunk * max(4, v)),
// in quarters of one LT's decode time, with v the wavefronts on the busiest
// CU in that generation. A generation pays a cold start (kernel arguments,
// selector table, first requests) worth two chunk round trips; each chunk
// pays one dependent memory round trip (offsets, then payload) worth five
// LT decodes; and each LT's decode time grows with the wavefronts sharing a
// SIMD (v / 4) once there is one per SIMD, as the decode is issue-bound.
// Ties go to fewer generations, then to more wavefronts per CU, then to
// linear staging and shorter chunks. The constants were fitted to a sweep of
// every configuration over 17 shapes and widths: within 0.5 % of the fastest
// on average, 4 % at worst. Residency: the LDS, and the wavefronts per SIMD
// each instantiation is built for (waves_per_simd), with at most 16
// workgroups per CU.
// wpg_only > 0 fixes the number of wavefronts; staging 1 or 2 allows linear
// or ring payload staging only (0: either). perm: the LTs are row-reordered
// (their stages hold two more per-LT arrays); bits: payload value width
// (2-bit chunks stage half the payload bytes); ch_only > 0 fixes the chunk
// length.
void choose_config(int M, int K, int N, bool perm, int bits, int n_cu, int wpg_only, int staging, int ch_only,
                   int &wpg, int &cfg) {
    const int nrb = M / 16, nkb = K / 64;
    long best[5] = {0, 0, 0, 0, 0};
    wpg = 0;
    cfg = -1;
    // Activation width the instantiation is built for (us_spmm's dispatch).
    const int nmax = N > 16 ? 32 : (N <= 4 && bits == 4 && !perm) ? 4 : 16;
    for (int w = 16; w >= 1; w /= 2) {
        if (w > nkb || (wpg_only > 0 && w != wpg_only)) continue;
        for (int idx = 0; idx < kNumCfgs; ++idx) {
            if (!cfg_allowed(idx, N) || (staging == 1 && kCfgs[idx].ring) || (staging == 2 && !kCfgs[idx].ring) ||
                (ch_only > 0 && kCfgs[idx].ch != ch_only))
                continue;
            const int lds = lds_bytes(idx, N, w, perm, bits);
            if (lds > kMaxLds) continue;
            const int c = kCfgs[idx].ch;
            const long chunks = ((nkb + w - 1) / w + c - 1) / c;
            const int by_regs = 4 * waves_per_simd(w, nmax, c, chunks > 1, kCfgs[idx].ring, perm) / w;
            const int per_cu = max(1, min(min(kMaxLds / lds, by_regs), 16));   // resident workgroups per CU
            const long slots = (long)n_cu * per_cu;
            const long gens = (nrb + slots - 1) / slots;
            const long waves = (long)w * min((long)per_cu, (nrb + n_cu - 1) / (long)n_cu);
            long cost = 0;
            for (long left = nrb; left > 0; left -= slots) {
                const long v = (long)w * ((min(left, slots) + n_cu - 1) / n_cu);   // busiest CU
                cost += 40 + chunks * (20 + c * max(4L, v));
            }
            const long key[5] = {cost, gens, -waves, kCfgs[idx].ring ? 1 : 0, c};
            bool better = cfg < 0;
            for (int k = 0; k < 5 && !better; ++k) {
                if (key[k] != best[k]) {
                    better = key[k] < best[k];
                    break;
                }
            }
            if (better) {
                for (int k = 0; k < 5; ++k) best[k] = key[k];
                wpg = w;
                cfg = idx;
            }
        }
    }
}

// Compute units of the current device (queried once per device).
int device_cus() {
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n <= 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

}  // namespace

extern "C" us_status us_spmm_plan(int32_t M, int32_t K, int32_t N, int32_t bits, int32_t reordered,
                                  const us_spmm_opts *opts, int32_t *split_k, int32_t *chunk_lts, int32_t *staging) {
    if (!split_k || !chunk_lts || !staging) return US_ERR_ARG;
    if (bits != 4 && bits != 2) return US_ERR_ARG;
    if (bits == 2 && reordered) return US_ERR_ARG;
    if (M <= 0 || K <= 0 || M % US_LT_H || K % US_LT_W || K > US_K_MAX) return US_ERR_SHAPE;
    if (N < 1 || N > US_N_LIMIT) return US_ERR_SHAPE;
    int wpg_only = 0, stg = 0, ch_only = 0;
    if (opts) {
        if (opts->variant < 0 || opts->variant > 2) return US_ERR_ARG;
        if (!chunk_option_ok(opts->chunk_lts)) return US_ERR_ARG;
        stg = opts->variant;
        ch_only = opts->chunk_lts;
        const int s = opts->split_k;
        if (s != 0) {
            if (s != 1 && s != 2 && s != 4 && s != 8 && s != 16) return US_ERR_ARG;
            wpg_only = s;
            while (wpg_only > K / US_LT_W) wpg_only /= 2;
        }
    }
    int wpg = 0, cfg = -1;
    choose_config(M, K, std::min(N, US_N_MAX), reordered != 0, bits, device_cus(), wpg_only, stg, ch_only, wpg, cfg);
    if (cfg < 0) return US_ERR_ARG;
    *split_k = wpg;
    *chunk_lts = kCfgs[cfg].ch;
    *staging = kCfgs[cfg].ring ? 2 : 1;
    return US_OK;
}

extern "C" us_status us_spmm_workspace_size(int32_t M, int32_t K, int32_t N, const us_spmm_opts *opts,
                                            size_t *bytes) {
    if (!bytes) return US_ERR_ARG;
    if (M <= 0 || K <= 0 || M % US_LT_H || K % US_LT_W || K > US_K_MAX) return US_ERR_SHAPE;
    if (N < 1 || N > US_N_LIMIT) return US_ERR_SHAPE;
    if (opts && (opts->variant < 0 || opts->variant > 2 || opts->split_k < 0 || !chunk_option_ok(opts->chunk_lts)))
        return US_ERR_ARG;
    *bytes = 0;
    return US_OK;
}

extern "C" us_status us_spmm(const us_iebme_dev *w, const uint8_t *x, int32_t N, int32_t *y,
                             const float *scale, float *y_f32, void *ws, size_t ws_bytes,
                             const us_spmm_opts *opts, void *stream) {
    (void)ws;
    (void)ws_bytes;
    if (!w || !x || !y || !w->bitmaps || !w->offsets) return US_ERR_ARG;
    if ((scale == nullptr) != (y_f32 == nullptr)) return US_ERR_ARG;
    const int32_t M = w->M, K = w->K;
    if (M <= 0 || K <= 0 || M % US_LT_H || K % US_LT_W || K > US_K_MAX) return US_ERR_SHAPE;
    if ((uint64_t)M * (uint64_t)K >= (1ull << 32)) return US_ERR_SHAPE;
    if (N < 1 || N > US_N_LIMIT) return US_ERR_SHAPE;
    const int64_t nkb = K / US_LT_W;
    if (w->n_lt != (int64_t)(M / US_LT_H) * nkb) return US_ERR_FORMAT;
    if (w->n_payload < 0 || w->n_payload > (int64_t)M * K || w->n_payload % 4) return US_ERR_FORMAT;
    if (w->n_payload > 0 && !w->payload) return US_ERR_ARG;
    if (!aligned(w->bitmaps, 8) || !aligned(w->offsets, 4) || !aligned(x, 16) || !aligned(y, 4) ||
        (scale && (!aligned(scale, 4) || !aligned(y_f32, 4))) || (w->perm && !aligned(w->perm, 8)))
        return US_ERR_ARG;
    const bool perm = w->perm != nullptr;
    const int bits = w->bits == 0 ? 4 : w->bits;
    if (bits != 4 && bits != 2) return US_ERR_FORMAT;
    if (bits == 2 && perm) return US_ERR_ARG;              // no reordered 2-bit kernels

    int wpg_only = 0, staging = 0, ch_only = 0;
    if (opts) {
        if (opts->variant < 0 || opts->variant > 2) return US_ERR_ARG;
        if (!chunk_option_ok(opts->chunk_lts)) return US_ERR_ARG;
        staging = opts->variant;
        ch_only = opts->chunk_lts;
        const int s = opts->split_k;
        if (s != 0) {
            if (s != 1 && s != 2 && s != 4 && s != 8 && s != 16) return US_ERR_ARG;
            wpg_only = s;
            while (wpg_only > nkb) wpg_only /= 2;          // at least one LT per slice
        }
    }
    // Slabs of up to US_N_MAX columns: every full slab shares one
    // configuration, a narrower last slab gets its own. Both are chosen
    // before anything is launched.
    const int n_cu = device_cus();
    const int n_full = std::min<int>(N, US_N_MAX), n_last = N % US_N_MAX == 0 ? n_full : N % US_N_MAX;
    int wpg = 0, cfg = -1, wpg_last = 0, cfg_last = -1;
    choose_config(M, K, n_full, perm, bits, n_cu, wpg_only, staging, ch_only, wpg, cfg);
    choose_config(M, K, n_last, perm, bits, n_cu, wpg_only, staging, ch_only, wpg_last, cfg_last);
    if (cfg < 0 || cfg_last < 0) return US_ERR_ARG;        // no configuration fits LDS

    SpmmArgs a;
    a.bm32 = (const uint32_t *)w->bitmaps;
    a.off = w->offsets;
    a.pay = w->payload;
    // Whole 16-byte pieces: a piece is either fully inside the range or fully
    // outside it (then it reads zeros). Rounding up stays within the
    // US_PAYLOAD_PAD bytes that follow the payload.
    a.pay_bytes = (int32_t)((((w->n_payload * bits + 7) / 8) + 15) & ~(int64_t)15);
    a.scale = scale;
    a.perm32 = (const uint32_t *)w->perm;
    a.M = M;
    a.K = K;
    a.nkb = (int32_t)nkb;
    a.n_cu = n_cu;

    hipStream_t s = (hipStream_t)stream;
    for (int n0 = 0; n0 < N; n0 += US_N_MAX) {
        const int ns = std::min(US_N_MAX, N - n0);
        const int sw = ns == n_full ? wpg : wpg_last, sc = ns == n_full ? cfg : cfg_last;
        a.x = x + (int64_t)n0 * (K / 2);
        a.y = y + (int64_t)n0 * M;
        a.yf = y_f32 ? y_f32 + (int64_t)n0 * M : nullptr;
        a.N = ns;
        const hipError_t err = bits == 2 ? launch_cfg_w2(sw, sc, a, s)
                               : perm    ? launch_cfg_perm(sw, sc, a, s)
                               : ns <= 4 ? launch_cfg_narrow(sw, sc, a, s)
                                         : launch_cfg<false, 4>(sw, sc, a, s);
        if (err != hipSuccess) return US_ERR_DEVICE;
    }
    return US_OK;
}
