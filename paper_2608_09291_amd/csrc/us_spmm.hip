// IE-BME x INT4 -> INT32 sparse product on gfx950 (CDNA4).
//
// The operation is the UnionSparse kernel of Section VI: Y = W X with W in
// IE-BME (Section V-A), X dense INT4, INT32 accumulation. What is kept from
// the paper and what is re-designed for CDNA4:
//
//  * Work split. One workgroup per 16-row block of W; its wavefronts split the
//    block's K range into contiguous slices (the paper's split-K with its
//    InitSchedule and Reduction steps). Because every wavefront of a slice set
//    lives in one workgroup, the split-K sums are combined in LDS at the end:
//    no workspace, no second launch. In row-block-major LT order a slice is a
//    contiguous run of LTs, so its bitmaps and payload are contiguous bytes.
//
//  * Staging (the paper's double-buffered producer/consumer pipeline). Each
//    wavefront streams its slice in batches of 8 LTs: the payload bytes of
//    batch b+1 are fetched with 16-byte buffer loads into registers while
//    batch b is decoded from the wavefront's own LDS stage. No workgroup
//    barrier is needed inside the loop: a wavefront's LDS accesses are
//    executed in order.
//
//  * Decode (the paper's LSPD, Section VI-B). One LT (16 x 64) is decoded by
//    one wavefront straight into the A operand of v_mfma_i32_16x16x64_i8.
//    Lane l owns MFMA row l % 16 = 2 i + a (union-mask row i, area row a) and
//    k-group g = l / 16, which is the G = 8 bit segment g of mask row i. The
//    lane's idx_base (earlier rows' popcounts plus the popcount of its row
//    before bit 8 g) comes from a DPP row scan; the same index then reads
//    area stream q = 2a (columns 8g..8g+7) and stream q = 2a + 1 (columns
//    32+8g..32+8g+7), which is the paper's "one rank reused across all area
//    streams". Active nibbles are placed into their byte slots with two
//    v_perm_b32 per 8 positions, selectors taken from a 256-entry LDS table
//    indexed by the 8-bit segment; inactive slots get selector 0x0C (zero).
//
//  * INT4 -> INT8. CDNA4 has no INT4 matrix instruction. Weights and
//    activations are expanded to bytes that hold the value in the high
//    nibble (16 v, exact in int8), so the MFMA sums are 256 Y; the epilogue
//    shifts right by 8. |256 Y| <= 256 * 64 * K < 2^31 for K <= US_K_MAX.
//    Both operands put the even and the odd positions of each 8-group in
//    separate dwords, the same slot order on both sides of the product.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "us.h"

namespace {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr int kBatch = 8;                           // LTs per staged batch
// Payload bytes of one batch stage. A batch holds at most 8 LTs x 512 bytes;
// the stage starts at the 16-byte boundary at or below the first LT's first
// byte (up to 15 bytes early), a segment window may read 8 bytes past the
// last value, and the end is rounded up to 16: at most 4135 -> 259 pieces.
constexpr int kStagePayload = 4160;
constexpr int kStagePieces = kStagePayload / 16;    // 260
constexpr int kLoadsPerLane = 5;                    // 5 * 64 >= 260
constexpr int kStageBitmap = kBatch * 32;
constexpr int kStageWords = (kStagePayload + kStageBitmap) / 4;
constexpr uint32_t kHiNib = 0xF0F0F0F0u;
constexpr int kBufferDword3 = 0x00020000;           // raw buffer, 32-bit data (gfx9 family)

static_assert(kLoadsPerLane * 64 >= kStagePieces, "stage loads");
static_assert(kStagePayload % 16 == 0, "stage alignment");

struct SpmmArgs {
    const uint32_t *bm32;   // union bitmaps as dwords: LT t owns [8t, 8t + 8)
    const uint32_t *off;    // union value offsets, n_lt + 1
    const uint8_t *pay;     // compressed values
    int32_t pay_bytes;      // buffer range: payload bytes rounded up to 16 (inside the pad)
    const uint32_t *x32;    // activations, N rows of K/8 dwords
    int32_t *y;
    const float *scale;
    float *yf;
    int32_t M, K, N, nkb;
};

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_row(uint32_t v) {
    // Out-of-row source lanes read zero (bound_ctrl).
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}

// s_waitcnt vmcnt(0): every vector-memory load of this wavefront has returned.
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ uint32_t lane_value(uint32_t v, int lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// Selector pair for one 8-bit union-mask segment m. Slot s of the output
// (dword 0: s = 0..3, dword 1: s = 4..7) holds segment position 2s (s < 4) or
// 2(s-4)+1 (s >= 4). An active position of rank r takes the r-th packed
// value: even r sits in byte r/2 of the "low" source, odd r in byte r/2 of the
// "high" source (bytes 4..7 of v_perm_b32's 8-byte input).
__device__ uint2 perm_selectors(uint32_t m) {
    uint32_t sel[2] = {0u, 0u};
    for (int s = 0; s < 8; ++s) {
        const int pos = s < 4 ? 2 * s : 2 * (s - 4) + 1;
        uint32_t b = 0x0Cu;                                   // v_perm: constant zero
        if ((m >> pos) & 1u) {
            const uint32_t r = __popc(m & ((1u << pos) - 1u));
            b = (r & 1u) ? 4u + (r >> 1) : (r >> 1);
        }
        sel[s >> 2] |= b << (8 * (s & 3));
    }
    return make_uint2(sel[0], sel[1]);
}

// 32 bits of the staged payload starting at bit `bn` (nibble index * 4).
__device__ __forceinline__ uint32_t stage_window(const uint32_t *st, uint32_t bn) {
    const uint32_t d = bn >> 5;
    return __builtin_amdgcn_alignbit(st[d + 1], st[d], bn);
}

// Eight packed INT4 values -> the two slot dwords of one segment
// (even positions, odd positions).
__device__ __forceinline__ int2 place(uint32_t w, uint2 sel) {
    const uint32_t hi = w & kHiNib;            // odd ranks, already in the high nibble
    const uint32_t lo = (w << 4) & kHiNib;     // even ranks moved up
    return make_int2((int32_t)__builtin_amdgcn_perm(hi, lo, sel.x),
                     (int32_t)__builtin_amdgcn_perm(hi, lo, sel.y));
}

template <int WPG, int NB>
__global__ __launch_bounds__(64 * WPG) void us_spmm_kernel(SpmmArgs p) {
    __shared__ __attribute__((aligned(16))) uint32_t stage_all[WPG][kStageWords];
    __shared__ uint2 lut[256];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int mb = blockIdx.x;

    for (int e = threadIdx.x; e < 256; e += 64 * WPG) lut[e] = perm_selectors((uint32_t)e);
    __syncthreads();

    // This wavefront's K slice: LTs t0 .. t0 + nlt - 1 of row block mb.
    const int nkb = p.nkb;
    const int kb0 = wave * nkb / WPG;
    const int nlt = (wave + 1) * nkb / WPG - kb0;       // <= 127, checked by the host
    const int64_t t0 = (int64_t)mb * nkb + kb0;

    // Offsets o_{t0} .. o_{t0 + nlt} spread over two registers.
    const uint32_t offA = lane <= nlt ? p.off[t0 + lane] : 0u;
    const uint32_t offB = 64 + lane <= nlt ? p.off[t0 + 64 + lane] : 0u;
    auto o_at = [&](int j) -> uint32_t {                  // j wave-uniform
        return j < 64 ? lane_value(offA, j) : lane_value(offB, j - 64);
    };

    // Lane roles.
    const int rr = lane & 15;
    const uint32_t a = rr & 1;                            // area row partition
    const int i = rr >> 1;                                // union-mask row
    const int g = lane >> 4;                              // segment / MFMA k-group
    const uint32_t himask = ~((1u << (8 * g)) - 1u);      // mask bits from the segment on

    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void *)p.pay, (short)0, p.pay_bytes, kBufferDword3);

    const uint32_t *xrow[NB];
    bool xok[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int n = nb * 16 + rr;
        xok[nb] = n < p.N;
        xrow[nb] = p.x32 + (int64_t)(xok[nb] ? n : 0) * (p.K / 8);
    }

    uint32_t *st = stage_all[wave];
    uint32_t *st_bm = st + kStagePayload / 4;

    i32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (i32x4){0, 0, 0, 0};

    // Registers holding the next batch.
    i32x4 pf[kLoadsPerLane];
    uint32_t pfbm = 0;
    uint32_t pfx[kBatch][NB][2];

    auto geometry = [&](int b, int &cnt, uint32_t &A0, uint32_t &nq) {
        const int tb = b * kBatch;
        cnt = min(kBatch, nlt - tb);
        const uint32_t ob = o_at(tb), oe = o_at(tb + cnt);
        A0 = (ob >> 1) & ~15u;
        const uint32_t span = (((oe - 2u * A0) >> 3) << 2) + 8u;
        nq = min((span + 15u) >> 4, (uint32_t)kStagePieces);
    };

    auto issue = [&](int b) {
        int cnt;
        uint32_t A0, nq;
        geometry(b, cnt, A0, nq);
        const int tb = b * kBatch;
#pragma unroll
        for (int u = 0; u < kLoadsPerLane; ++u) {
            const uint32_t piece = (uint32_t)(lane + 64 * u);
            // The whole offset goes in the vector operand: that is the part
            // the buffer range check sees, so a piece past the end reads 0.
            if (piece < nq) pf[u] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, A0 + 16u * piece, 0, 0);
        }
        if (lane < 8 * cnt) pfbm = p.bm32[8 * (t0 + tb) + lane];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int kb = kb0 + tb + j;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const bool ok = (j < cnt) && xok[nb];
                pfx[j][nb][0] = ok ? xrow[nb][8 * kb + g] : 0u;
                pfx[j][nb][1] = ok ? xrow[nb][8 * kb + g + 4] : 0u;
            }
        }
    };

    const int nbatch = (nlt + kBatch - 1) / kBatch;
    wait_vm_all();                       // the offset registers
    if (nbatch > 0) issue(0);

    for (int b = 0; b < nbatch; ++b) {
        int cnt;
        uint32_t A0, nq;
        geometry(b, cnt, A0, nq);
        const int tb = b * kBatch;
        uint32_t o[kBatch + 1];          // o_t of this batch's LTs (wave-uniform)
#pragma unroll
        for (int j = 0; j <= kBatch; ++j) o[j] = o_at(tb + min(j, cnt));

        // Batch b has landed. Waiting here, before batch b+1 is issued, keeps
        // every later use free of waits on the prefetch in flight.
        wait_vm_all();

        // Commit batch b to the LDS stage.
#pragma unroll
        for (int u = 0; u < kLoadsPerLane; ++u) {
            const uint32_t piece = (uint32_t)(lane + 64 * u);
            if (piece < nq) *(i32x4 *)(st + 4 * piece) = pf[u];
        }
        if (lane < 8 * cnt) st_bm[lane] = pfbm;
        uint32_t cx[kBatch][NB][2];
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                cx[j][nb][0] = pfx[j][nb][0];
                cx[j][nb][1] = pfx[j][nb][1];
            }
        __asm__ volatile("" ::: "memory");

        if (b + 1 < nbatch) issue(b + 1);

#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            if (j >= cnt) break;
            const uint32_t P = (o[j + 1] - o[j]) >> 2;          // P_t
            const uint32_t orel = o[j] - 2u * A0;               // o_t within the stage

            // idx_base(i, g): popcount of rows < i plus row i's bits below 8g.
            const uint32_t mrow = st_bm[8 * j + i];
            const uint32_t rp = __popc(mrow);
            uint32_t incl = rp + dpp_row<0x112>(rp);           // row_shr:2 = previous mask row
            incl += dpp_row<0x114>(incl);
            incl += dpp_row<0x118>(incl);
            const uint32_t idx = incl - __popc(mrow & himask);

            const uint2 sel = lut[(mrow >> (8 * g)) & 0xFFu];
            const uint32_t bn0 = (orel + (a ? 2u * P : 0u) + idx) << 2;   // stream q = 2a
            const uint32_t bn1 = bn0 + 4u * P;                            // stream q = 2a + 1

            const int2 c0 = place(stage_window(st, bn0), sel);
            const int2 c1 = place(stage_window(st, bn1), sel);
            const i32x4 A = {c0.x, c0.y, c1.x, c1.y};

#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const uint32_t x0 = cx[j][nb][0], x1 = cx[j][nb][1];
                const i32x4 B = {(int32_t)((x0 << 4) & kHiNib), (int32_t)(x0 & kHiNib),
                                 (int32_t)((x1 << 4) & kHiNib), (int32_t)(x1 & kHiNib)};
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, B, acc[nb], 0, 0, 0);
            }
        }
        __asm__ volatile("" ::: "memory");
    }

    // Split-K combine: each wavefront leaves its 16 x (16 NB) partial in its
    // own stage; after the barrier all threads sum the WPG partials.
    // MFMA result layout: lane l, element v is row 4 (l / 16) + v, column l % 16.
    int32_t *red = (int32_t *)st;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int rho = 4 * g + v;
            const int r = 8 * (rho & 1) + (rho >> 1);         // MFMA row 2i + a -> W row 8a + i
            red[r * (16 * NB) + nb * 16 + rr] = acc[nb][v];
        }
    __syncthreads();

    const int64_t M = p.M;
    for (int e = threadIdx.x; e < 16 * p.N; e += 64 * WPG) {
        const int r = e & 15, n = e >> 4;
        int32_t s = 0;
#pragma unroll
        for (int w = 0; w < WPG; ++w) s += ((const int32_t *)stage_all[w])[r * (16 * NB) + n];
        const int32_t yv = s >> 8;                            // exact: s = 256 Y
        const int64_t m = (int64_t)mb * 16 + r;
        p.y[n * M + m] = yv;
        if (p.scale) p.yf[n * M + m] = (float)yv * p.scale[m];
    }
}

template <int WPG, int NB>
hipError_t launch_spmm(const SpmmArgs &a, hipStream_t s) {
    hipLaunchKernelGGL((us_spmm_kernel<WPG, NB>), dim3(a.M / 16), dim3(64 * WPG), 0, s, a);
    return hipGetLastError();
}

template <int NB>
hipError_t launch_spmm_wpg(int wpg, const SpmmArgs &a, hipStream_t s) {
    switch (wpg) {
        case 1: return launch_spmm<1, NB>(a, s);
        case 2: return launch_spmm<2, NB>(a, s);
        case 4: return launch_spmm<4, NB>(a, s);
        case 8: return launch_spmm<8, NB>(a, s);
        default: return launch_spmm<16, NB>(a, s);
    }
}

bool aligned(const void *ptr, uintptr_t n) { return ((uintptr_t)ptr % n) == 0; }

constexpr int kMaxLtPerWave = 127;

// Wavefronts per workgroup (= K slices per row block) for a shape: aim at
// about 16 wavefronts per CU over 256 CUs, keep at least one LT per slice and
// at most 127.
int auto_split(int M, int K) {
    const int nrb = M / 16, nkb = K / 64;
    int w = 1;
    while (w < 16 && nrb * w * 2 <= 256 * 16) w *= 2;
    while (w > 1 && w > nkb) w /= 2;
    while (w < 16 && (nkb + w - 1) / w > kMaxLtPerWave) w *= 2;
    return w;
}

}  // namespace

extern "C" us_status us_spmm_workspace_size(int32_t M, int32_t K, int32_t N, const us_spmm_opts *opts,
                                            size_t *bytes) {
    if (!bytes) return US_ERR_ARG;
    if (M <= 0 || K <= 0 || M % US_LT_H || K % US_LT_W || K > US_K_MAX) return US_ERR_SHAPE;
    if (N < 1 || N > US_N_MAX) return US_ERR_SHAPE;
    if (opts && (opts->variant != 0 || opts->split_k < 0)) return US_ERR_ARG;
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
    if (N < 1 || N > US_N_MAX) return US_ERR_SHAPE;
    const int64_t nkb = K / US_LT_W;
    if (w->n_lt != (int64_t)(M / US_LT_H) * nkb) return US_ERR_FORMAT;
    if (w->n_payload < 0 || w->n_payload > (int64_t)M * K || w->n_payload % 4) return US_ERR_FORMAT;
    if (w->n_payload > 0 && !w->payload) return US_ERR_ARG;
    if (!aligned(w->bitmaps, 8) || !aligned(w->offsets, 4) || !aligned(x, 4) || !aligned(y, 4) ||
        (scale && (!aligned(scale, 4) || !aligned(y_f32, 4))))
        return US_ERR_ARG;

    int wpg = auto_split(M, K);
    if (opts) {
        if (opts->variant != 0) return US_ERR_ARG;
        const int s = opts->split_k;
        if (s != 0) {
            if (s != 1 && s != 2 && s != 4 && s != 8 && s != 16) return US_ERR_ARG;
            if ((nkb + s - 1) / s > kMaxLtPerWave) return US_ERR_ARG;
            wpg = s;
        }
    }

    SpmmArgs a;
    a.bm32 = (const uint32_t *)w->bitmaps;
    a.off = w->offsets;
    a.pay = w->payload;
    // Whole 16-byte pieces: a piece is either fully inside the range or fully
    // outside it (then it reads zeros). Rounding up stays within the
    // US_PAYLOAD_PAD bytes that follow the payload.
    a.pay_bytes = (int32_t)((((w->n_payload + 1) / 2) + 15) & ~(int64_t)15);
    a.x32 = (const uint32_t *)x;
    a.y = y;
    a.scale = scale;
    a.yf = y_f32;
    a.M = M;
    a.K = K;
    a.N = N;
    a.nkb = (int32_t)nkb;

    hipStream_t s = (hipStream_t)stream;
    const hipError_t err = N > 16 ? launch_spmm_wpg<2>(wpg, a, s) : launch_spmm_wpg<1>(wpg, a, s);
    return err == hipSuccess ? US_OK : US_ERR_DEVICE;
}
