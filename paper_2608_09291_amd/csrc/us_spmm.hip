// Host side of the IE-BME SpMM (Section VI, "UnionSparse Kernel"
// algorithm): argument checks, the choice of kernel family, split and chunk
// configuration, and the launch. The kernels are in us_spmm_kernel.h
// (chunked) and us_spmm_burst.h (single pass).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>

#include "us.h"
#include "us_spmm_burst.h"
#include "us_spmm_kernel.h"

namespace {

using namespace us_spmm_detail;

bool aligned(const void *ptr, uintptr_t n) { return ((uintptr_t)ptr % n) == 0; }

bool chunk_option_ok(int ch) { return ch == 0 || ch == 4 || ch == 8 || ch == 11 || ch == 16; }

bool burst_ch_ok(int ch) {
    for (int c : kBurstChs)
        if (c == ch) return true;
    return false;
}

// Staging variants of us_spmm_opts.variant.
constexpr int kVariantWhole = 1, kVariantRing = 2, kVariantBurst = 3;

// A single-pass (burst) launch: wavefronts per workgroup, LTs per slice
// (instantiation), K blocks across workgroups.
struct BurstPlan {
    int wpg = 0, ch = 0, kblocks = 1;
};

// Whether a burst plan can run this shape: every wavefront gets 1..ch LTs,
// at most 16 activation columns, and the stage fits the LDS.
bool burst_fits(const BurstPlan &b, int nkb, int N, bool perm, int bits) {
    if (b.wpg < 1 || b.kblocks < 1 || N > 16 || !burst_ch_ok(b.ch)) return false;
    const int rmin = nkb / b.kblocks, rmax = (nkb + b.kblocks - 1) / b.kblocks;
    if (rmin < b.wpg) return false;
    if ((rmax + b.wpg - 1) / b.wpg > b.ch) return false;
    return burst_lds_bytes(b.ch, N, b.wpg, perm, bits) <= kMaxLds;
}

// Workspace bytes of a plan with `kblocks` K blocks for M rows and up to
// `ncols` columns per pass: int32 accumulators, then one ticket per 16-row
// block (zero between calls).
size_t burst_ws_bytes(int kblocks, int M, int ncols) {
    if (kblocks <= 1) return 0;
    return (size_t)4 * (size_t)M * (size_t)ncols + (size_t)4 * (size_t)(M / 16);
}

// Burst plan from explicit options (variant 3): split_k wavefronts per
// workgroup (required), chunk_lts LTs per slice (0: the shortest that fits),
// k_blocks K blocks (0 or 1: none).
bool burst_from_opts(const us_spmm_opts &o, int nkb, int N, bool perm, int bits, BurstPlan &b) {
    b.wpg = o.split_k;
    b.kblocks = o.k_blocks > 0 ? o.k_blocks : 1;
    if (b.wpg != 1 && b.wpg != 2 && b.wpg != 4 && b.wpg != 8 && b.wpg != 16) return false;
    if (o.chunk_lts > 0) {
        b.ch = o.chunk_lts;
        return burst_fits(b, nkb, N, perm, bits);
    }
    for (int c : kBurstChs) {
        b.ch = c;
        if (burst_fits(b, nkb, N, perm, bits)) return true;
    }
    return false;
}

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
// linear staging and shorter chunks. The kernels of up to 4 columns on rows
// in stored order differ in two ways, both measured: they take a ring stage
// only when no linear one fits (linear staging was the faster on every
// shape swept at N <= 4, by up to 7 %), and, with at least one row block
// per CU, a tie goes to fewer wavefronts as long as 8 or more stay on the
// CU (their per-wavefront start outweighs the added parallelism there:
// 12288x4096 at N = 1-4 runs 5-7 % faster as 4 x 16 than as 8 x 8, while
// one wavefront per slice of 28672x7168, fewer row blocks than CUs
// (1024x4096) or reordered rows (28672x8192 at N = 1) run 3-23 % slower). The constants were
// fitted to a sweep of every configuration over 17 shapes and widths; a
// later sweep of 27 shapes and widths puts the choice within 0.7 % of the
// fastest on average, 7 % at worst. Residency: the LDS, and the wavefronts per SIMD
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
    long best[6] = {0, 0, 0, 0, 0, 0};
    wpg = 0;
    cfg = -1;
    // Activation width the instantiation is built for (us_spmm's dispatch).
    const int nmax = N > 16 ? 32 : (N <= 4 && bits == 4) ? 4 : 16;
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
            const bool narrow = nmax == 4 && !perm;               // see the rules above
            const long ring_last = narrow && kCfgs[idx].ring ? 1 : 0;
            const long tie = narrow && nrb >= n_cu ? (waves >= 8 ? waves : 1000000 - waves) : -waves;
            const long key[6] = {ring_last, cost, gens, tie, kCfgs[idx].ring ? 1 : 0, c};
            bool better = cfg < 0;
            for (int k = 0; k < 6 && !better; ++k) {
                if (key[k] != best[k]) {
                    better = key[k] < best[k];
                    break;
                }
            }
            if (better) {
                for (int k = 0; k < 6; ++k) best[k] = key[k];
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

// The launch of one slab of up to US_N_MAX columns: a chunked configuration
// (us_spmm_kernel.h) or a single-pass one (us_spmm_burst.h).
struct Plan {
    bool burst = false;
    int wpg = 0, cfg = -1;     // chunked: wavefronts per workgroup, kCfgs index
    BurstPlan b;               // burst
};

// Options checked once for every entry point.
us_status check_opts(const us_spmm_opts *o) {
    if (!o) return US_OK;
    if (o->variant < 0 || o->variant > kVariantBurst) return US_ERR_ARG;
    if (o->split_k != 0 && o->split_k != 1 && o->split_k != 2 && o->split_k != 4 && o->split_k != 8 &&
        o->split_k != 16)
        return US_ERR_ARG;
    if (o->k_blocks < 0 || o->k_blocks > US_K_BLOCKS_MAX) return US_ERR_ARG;
    if (o->variant == kVariantBurst) {
        if (o->split_k == 0 || (o->chunk_lts != 0 && !burst_ch_ok(o->chunk_lts))) return US_ERR_ARG;
    } else {
        if (!chunk_option_ok(o->chunk_lts) || o->k_blocks > 1) return US_ERR_ARG;
    }
    return US_OK;
}

// Plan for one slab of N <= US_N_MAX columns. ws_ok: a workspace was given
// (a split across workgroups is possible; its size is checked by the caller).
us_status make_plan(int M, int K, int N, bool perm, int bits, const us_spmm_opts *opts, int n_cu, bool ws_ok,
                    Plan &pl) {
    const int nkb = K / US_LT_W;
    pl = Plan();
    if (opts && opts->variant == kVariantBurst) {
        if (!burst_from_opts(*opts, nkb, N, perm, bits, pl.b)) return US_ERR_ARG;
        if (pl.b.kblocks > 1 && !ws_ok) return US_ERR_ARG;
        pl.burst = true;
        return US_OK;
    }
    int wpg_only = 0, staging = 0, ch_only = 0;
    if (opts) {
        staging = opts->variant;
        ch_only = opts->chunk_lts;
        if (opts->split_k != 0) {
            wpg_only = opts->split_k;
            while (wpg_only > nkb) wpg_only /= 2;          // at least one LT per slice
        }
    }
    choose_config(M, K, N, perm, bits, n_cu, wpg_only, staging, ch_only, pl.wpg, pl.cfg);
    return pl.cfg < 0 ? US_ERR_ARG : US_OK;               // no configuration fits LDS
}

us_status check_shape(int32_t M, int32_t K, int32_t N) {
    if (M <= 0 || K <= 0 || M % US_LT_H || K % US_LT_W || K > US_K_MAX) return US_ERR_SHAPE;
    if ((uint64_t)M * (uint64_t)K >= (1ull << 32)) return US_ERR_SHAPE;
    if (N < 1 || N > US_N_LIMIT) return US_ERR_SHAPE;
    return US_OK;
}

}  // namespace

extern "C" us_status us_spmm_plan(int32_t M, int32_t K, int32_t N, int32_t bits, int32_t reordered,
                                  const us_spmm_opts *opts, int32_t *split_k, int32_t *chunk_lts, int32_t *staging,
                                  int32_t *k_blocks) {
    if (!split_k || !chunk_lts || !staging) return US_ERR_ARG;
    if (bits != 4 && bits != 2) return US_ERR_ARG;
    if (bits == 2 && reordered) return US_ERR_ARG;
    us_status st = check_shape(M, K, N);
    if (st != US_OK) return st;
    if ((st = check_opts(opts)) != US_OK) return st;
    Plan pl;
    st = make_plan(M, K, std::min(N, US_N_MAX), reordered != 0, bits, opts, device_cus(), true, pl);
    if (st != US_OK) return st;
    if (pl.burst) {
        *split_k = pl.b.wpg;
        *chunk_lts = pl.b.ch;
        *staging = kVariantBurst;
    } else {
        *split_k = pl.wpg;
        *chunk_lts = kCfgs[pl.cfg].ch;
        *staging = kCfgs[pl.cfg].ring ? kVariantRing : kVariantWhole;
    }
    if (k_blocks) *k_blocks = pl.burst ? pl.b.kblocks : 1;
    return US_OK;
}

extern "C" us_status us_spmm_workspace_size(int32_t M, int32_t K, int32_t N, const us_spmm_opts *opts,
                                            size_t *bytes) {
    if (!bytes) return US_ERR_ARG;
    us_status st = check_shape(M, K, N);
    if (st != US_OK) return st;
    if ((st = check_opts(opts)) != US_OK) return st;
    const int kb = (opts && opts->variant == kVariantBurst) ? std::max(1, (int)opts->k_blocks) : 1;
    *bytes = burst_ws_bytes(kb, M, std::min(N, 16));
    return US_OK;
}

extern "C" us_status us_spmm(const us_iebme_dev *w, const uint8_t *x, int32_t N, int32_t *y,
                             const float *scale, float *y_f32, void *ws, size_t ws_bytes,
                             const us_spmm_opts *opts, void *stream) {
    if (!w || !x || !y || !w->bitmaps || !w->offsets) return US_ERR_ARG;
    if ((scale == nullptr) != (y_f32 == nullptr)) return US_ERR_ARG;
    const int32_t M = w->M, K = w->K;
    us_status st = check_shape(M, K, N);
    if (st != US_OK) return st;
    const int64_t nkb = K / US_LT_W;
    if (w->n_lt != (int64_t)(M / US_LT_H) * nkb) return US_ERR_FORMAT;
    if (w->n_payload < 0 || w->n_payload > (int64_t)M * K || w->n_payload % 4) return US_ERR_FORMAT;
    if (w->n_payload > 0 && !w->payload) return US_ERR_ARG;
    if (!aligned(w->bitmaps, 8) || !aligned(w->offsets, 4) || !aligned(x, 16) || !aligned(y, 4) ||
        (scale && (!aligned(scale, 4) || !aligned(y_f32, 4))) || (w->perm && !aligned(w->perm, 8)) ||
        !aligned(ws, 4))
        return US_ERR_ARG;
    const bool perm = w->perm != nullptr;
    const int bits = w->bits == 0 ? 4 : w->bits;
    if (bits != 4 && bits != 2) return US_ERR_FORMAT;
    if (bits == 2 && perm) return US_ERR_ARG;              // no reordered 2-bit kernels
    if ((st = check_opts(opts)) != US_OK) return st;

    // Slabs of up to US_N_MAX columns: every full slab shares one plan, a
    // narrower last slab gets its own. Both are made before anything is
    // launched. A split across workgroups needs the workspace for the
    // slab's columns.
    const int n_cu = device_cus();
    const int n_full = std::min<int>(N, US_N_MAX), n_last = N % US_N_MAX == 0 ? n_full : N % US_N_MAX;
    Plan p_full, p_last;
    if ((st = make_plan(M, K, n_full, perm, bits, opts, n_cu, ws != nullptr, p_full)) != US_OK) return st;
    if ((st = make_plan(M, K, n_last, perm, bits, opts, n_cu, ws != nullptr, p_last)) != US_OK) return st;
    for (const Plan *pl : {&p_full, &p_last}) {
        if (pl->burst && pl->b.kblocks > 1 &&
            (ws == nullptr || ws_bytes < burst_ws_bytes(pl->b.kblocks, M, pl == &p_full ? n_full : n_last)))
            return US_ERR_ARG;
    }

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
        const Plan &pl = ns == n_full ? p_full : p_last;
        a.x = x + (int64_t)n0 * (K / 2);
        a.y = y + (int64_t)n0 * M;
        a.yf = y_f32 ? y_f32 + (int64_t)n0 * M : nullptr;
        a.N = ns;
        hipError_t err;
        if (pl.burst) {
            BurstArgs b;
            b.a = a;
            b.kblocks = pl.b.kblocks;
            b.ws_acc = (int32_t *)ws;
            b.ws_tick = ws ? (uint32_t *)((char *)ws + (size_t)4 * M * ns) : nullptr;
            err = bits == 2 ? launch_burst_w2(pl.b.wpg, pl.b.ch, b, s)
                  : perm    ? launch_burst_perm(pl.b.wpg, pl.b.ch, b, s)
                  : ns <= 4 ? launch_burst_narrow(pl.b.wpg, pl.b.ch, b, s)
                            : launch_burst_plain(pl.b.wpg, pl.b.ch, b, s);
        } else {
            err = bits == 2 ? launch_cfg_w2(pl.wpg, pl.cfg, a, s)
                  : perm    ? launch_cfg_perm(pl.wpg, pl.cfg, a, s)
                  : ns <= 4 ? launch_cfg_narrow(pl.wpg, pl.cfg, a, s)
                            : launch_cfg<false, 4>(pl.wpg, pl.cfg, a, s);
        }
        if (err != hipSuccess) return US_ERR_DEVICE;
    }
    return US_OK;
}

// The reduction workspace of us_spmm_noalloc: one array per device that the
// library's code object is loaded on, zero when it is loaded. Host code never
// uses the array's name as an address: the per-device address comes from
// hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[US_NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on the current device, looked up once per
// device (with that device current); nullptr if the lookup fails.
void *scratch_address() {
    static std::atomic<void *> addr[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    void *p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        void *q = nullptr;
        if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return nullptr;
        addr[dev].store(q, std::memory_order_release);
        p = q;
    }
    return p;
}

}  // namespace

extern "C" us_status us_spmm_noalloc(const us_iebme_dev *w, const uint8_t *x, int32_t N, int32_t *y,
                                     const float *scale, float *y_f32, const us_spmm_opts *opts, void *stream) {
    // The arguments are checked by us_spmm; only the workspace is ours: it
    // must fit the array (us_spmm refuses a plan whose workspace exceeds
    // the bytes it is given, before launching anything).
    if (!w) return US_ERR_ARG;
    const us_status st = check_shape(w->M, w->K, N);
    if (st != US_OK) return st;
    size_t need = 0;
    if (check_opts(opts) == US_OK && opts && opts->variant == kVariantBurst && opts->k_blocks > 1 &&
        (need = burst_ws_bytes(opts->k_blocks, w->M, std::min<int>(N, 16))) > US_NOALLOC_SCRATCH_BYTES)
        return US_ERR_SHAPE;
    void *ws = scratch_address();
    if (!ws) return US_ERR_DEVICE;
    return us_spmm(w, x, N, y, scale, y_f32, ws, US_NOALLOC_SCRATCH_BYTES, opts, stream);
}
