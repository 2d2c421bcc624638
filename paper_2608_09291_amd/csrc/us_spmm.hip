// IE-BME x INT4 -> INT32 sparse product on gfx950 (CDNA4).
//
// The operation is the UnionSparse kernel of Section VI: Y = W X with W in
// IE-BME (Section V-A), X dense INT4, INT32 accumulation. What is kept from
// the paper and what is re-designed for CDNA4:
//
//  * Work split. One workgroup per 16-row block of W; its wavefronts split the
//    block's K range into contiguous slices (the paper's split-K with its
//    InitSchedule and Reduction steps). Because every slice of a row block
//    lives in one workgroup, the split-K sums are combined in LDS at the end:
//    no workspace, no second launch. In row-block-major LT order a slice is a
//    contiguous run of LTs, so its bitmaps and payload are contiguous bytes.
//
//  * Staging (the paper's producer/consumer pipeline, re-cut for CDNA4). A
//    wavefront's slice is processed in chunks of up to CH LTs, normally one.
//    For a chunk the wavefront first reads the chunk's offsets, then requests
//    all of its payload (16-byte buffer loads), bitmaps and activations at
//    once: one memory round trip per chunk, with the whole machine's requests
//    in flight together. The data is then copied into the wavefront's own LDS
//    stage and decoded. A wavefront's LDS accesses execute in order, so no
//    workgroup barrier is needed between staging and decoding.
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
//    LTs are decoded in pairs so that two independent chains interleave.
//
//  * INT4 -> INT8. CDNA4 has no INT4 matrix instruction. Weights and
//    activations are expanded to bytes that hold the value in the high
//    nibble (16 v, exact in int8), so the MFMA sums are 256 Y; the epilogue
//    shifts right by 8. |256 Y| <= 256 * 64 * K < 2^31 for K <= US_K_MAX.
//    Both operands put the even and the odd positions of each 8-group in
//    separate dwords, the same slot order on both sides of the product.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "us.h"

#ifndef US_SPMM_WINDOW
#define US_SPMM_WINDOW 3
#endif

namespace {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kHiNib = 0xF0F0F0F0u;
constexpr int kWindow = US_SPMM_WINDOW;                // payload loads in flight per wavefront
constexpr int kNonTemporal = 2;                        // buffer cache policy: nt
constexpr int kBufferDword3 = 0x00020000;           // raw buffer, 32-bit data (gfx9 family)

// LDS stage of one chunk of CH LTs (per wavefront):
//   payload : at most 512 CH bytes; the stage starts at the 16-byte boundary
//             at or below the chunk's first byte (up to 15 bytes early) and a
//             segment window may read 8 bytes past the last value, so at most
//             32 CH + 2 pieces of 16 bytes are staged;
//   bitmaps : 32 bytes per LT;
//   X       : the chunk's activation slice, N rows of 32 bytes per LT, packed;
//             rows are kXRowPad bytes apart so that the 16 rows read by one
//             instruction fall in different LDS banks.
template <int CH>
struct Chunk {
    static constexpr int kPayBytes = 512 * CH + 64;
    static constexpr int kPieces = kPayBytes / 16;
    static constexpr int kLoads = (32 * CH + 2 + 63) / 64;   // 16-byte payload loads per lane
    static constexpr int kBmWords = 8 * CH;                   // union-bitmap dwords
    static constexpr int kBmLoads = (kBmWords + 63) / 64;
    static constexpr int kBmOffset = kPayBytes;               // bytes into the stage
    static constexpr int kXOffset = kPayBytes + 4 * kBmWords;
    static_assert(kLoads * 64 >= 32 * CH + 2 && kPieces >= 32 * CH + 2, "stage size");
    // Stage bytes for N activation columns.
    static constexpr int kXRowWords = 8 * CH + 4;             // row stride, dwords (+16 bytes)
    static constexpr int bytes(int N) { return kXOffset + 4 * kXRowWords * N; }
};

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

// s_waitcnt vmcnt(n): at most n of this wavefront's vector-memory loads are
// still outstanding (they complete in issue order for this counter).
template <int n>
__device__ __forceinline__ void wait_vm() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void wait_vm_all() { wait_vm<0>(); }

// f(std::integral_constant<int, U>) for U = B .. E-1, as straight-line code.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

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

// Decode one LT of the stage into the MFMA A operand of this lane.
//   mrow   : union-mask row i of the LT (zero for a padding LT)
//   s4orel : bit index, within the stage, of the LT's first payload value
//   sd     : o_{t+1} - o_t = 4 P_t values; one area stream is P_t values = sd bits
//   inj    : 2 P_t on lanes of area row a = 1, else 0 (their streams start 2 P_t later)
__device__ __forceinline__ i32x4 decode_tile(const uint32_t *st, const uint2 *lut, uint32_t mrow,
                                             uint32_t s4orel, uint32_t sd, uint32_t inj, int g,
                                             uint32_t lomask) {
    // idx_base(i, g) plus the area-row stream offset: an inclusive scan over the
    // previous mask rows (lanes 2 i + a of a 16-lane DPP row hold rows
    // i = 0..7; row 0 starts from inj), plus row i's bits below 8 g.
    const uint32_t rp = __popc(mrow);
    uint32_t ex = (uint32_t)__builtin_amdgcn_update_dpp((int)inj, (int)rp, 0x112, 0xF, 0xF, false);
    ex += dpp_row<0x112>(ex);
    ex += dpp_row<0x114>(ex);
    ex += dpp_row<0x118>(ex);
    const uint32_t idx = __popc(mrow & lomask) + ex;

    const uint2 sel = lut[(mrow >> (8 * g)) & 0xFFu];
    const uint32_t bn0 = s4orel + 4u * idx;             // stream q = 2a
    const uint32_t bn1 = bn0 + sd;                      // stream q = 2a + 1
    const int2 c0 = place(stage_window(st, bn0), sel);
    const int2 c1 = place(stage_window(st, bn1), sel);
    return (i32x4){c0.x, c0.y, c1.x, c1.y};
}

__device__ __forceinline__ i32x4 unpack_x(uint32_t x0, uint32_t x1) {
    return (i32x4){(int32_t)((x0 << 4) & kHiNib), (int32_t)(x0 & kHiNib),
                   (int32_t)((x1 << 4) & kHiNib), (int32_t)(x1 & kHiNib)};
}

template <int WPG, int NB, int CH>
__global__ __launch_bounds__(64 * WPG) void us_spmm_kernel(SpmmArgs p, int stage_bytes) {
    using C = Chunk<CH>;
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    uint2 *lut = (uint2 *)lds;                               // 256 selector pairs

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int mb = blockIdx.x;
    const int N = p.N;

    // This wavefront's K slice: LTs t0 .. t0 + nlt - 1 of row block mb.
    const int nkb = p.nkb;
    const int kb0 = wave * nkb / WPG;
    const int nlt = (wave + 1) * nkb / WPG - kb0;
    const int64_t t0 = (int64_t)mb * nkb + kb0;

    // Offsets of the first chunk; the selector table is built while they load.
    uint32_t offv = p.off[t0 + min(lane, min(nlt, CH))];   // nlt = 0 reads o_{t0} only
    for (int e = threadIdx.x; e < 256; e += 64 * WPG) lut[e] = perm_selectors((uint32_t)e);
    __syncthreads();

    // Lane roles.
    const int rr = lane & 15;
    const uint32_t amask = (rr & 1) ? ~0u : 0u;            // area row partition a = 1
    const int i = rr >> 1;                                 // union-mask row
    const int g = lane >> 4;                               // segment / MFMA k-group
    const uint32_t lomask = (1u << (8 * g)) - 1u;          // mask bits before the segment

    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void *)p.pay, (short)0, p.pay_bytes, kBufferDword3);

    uint32_t *st = lds + (2048 + wave * stage_bytes) / 4;
    uint32_t *st_bm = st + C::kBmOffset / 4;
    uint32_t *st_x = st + C::kXOffset / 4;
    // X stage: row n holds 8 dwords per LT; lane (n, g) reads dwords g and g + 4.
    // Rows >= N would only feed output columns that are never stored: clamp.
    const uint32_t *xq[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) xq[nb] = st_x + min(nb * 16 + rr, N - 1) * C::kXRowWords + g;
    const int64_t xrow_bytes = p.K / 2;
    const uint8_t *x8 = (const uint8_t *)p.x32;

    i32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (i32x4){0, 0, 0, 0};

    // X staging: a row of the chunk's activation slice is 2 CH pieces of 16
    // bytes; one load instruction covers kXRowsPerLoad rows, lane = row slot *
    // kXLaneSpan + piece (powers of two, so no division).
    constexpr int kXLaneSpan = (2 * CH <= 8) ? 8 : (2 * CH <= 16) ? 16 : 32;
    constexpr int kXRowsPerLoad = 64 / kXLaneSpan;
    constexpr int kXLoads = (16 * NB + kXRowsPerLoad - 1) / kXRowsPerLoad;
    const int x_row_slot = lane / kXLaneSpan, x_piece = lane % kXLaneSpan;
    const int x_loads = (N + kXRowsPerLoad - 1) / kXRowsPerLoad;   // wave-uniform
    // Requests for a chunk's bitmaps and activations; they do not depend on
    // the offsets. Addresses are clamped into the matrix.
    auto request_side = [&](int c0, uint32_t (&pbm)[C::kBmLoads], i32x4 (&px)[kXLoads]) {
        const int cnt = max(1, min(CH, nlt - c0));         // clamped: a slice may be empty
        const int kbs = kb0 + c0;
#pragma unroll
        for (int v = 0; v < C::kBmLoads; ++v)
            pbm[v] = p.bm32[8 * (t0 + c0) + min(lane + 64 * v, 8 * cnt - 1)];
        const int kb = min(kbs + (min(x_piece, 2 * CH - 1) >> 1), nkb - 1);
#pragma unroll
        for (int u = 0; u < kXLoads; ++u) {
            if (u < x_loads) {                             // wave-uniform
                const int n = min(u * kXRowsPerLoad + x_row_slot, N - 1);
                px[u] = *(const i32x4 *)(x8 + n * xrow_bytes + 32 * kb + 16 * (x_piece & 1));
            }
        }
    };

    uint32_t pbm[C::kBmLoads];
    i32x4 px[kXLoads];
    request_side(0, pbm, px);

    auto process_chunk = [&](int c0) {
        const int cnt = min(CH, nlt - c0);
        wait_vm_all();                                     // offsets, bitmaps, activations

        const uint32_t ob = lane_value(offv, 0), oe = lane_value(offv, cnt);
        const uint32_t A0 = (ob >> 1) & ~15u;              // first staged byte
        const uint32_t span = (((oe - 2u * A0) >> 3) << 2) + 8u;
        const uint32_t nq = min((span + 15u) >> 4, (uint32_t)C::kPieces);
        // Payload: 16-byte pieces; load u brings stage bytes [1024 u, 1024 u + 1024).
        // At most kWindow loads are in flight per wavefront, so early pieces are
        // not queued behind the whole machine's requests and decoding starts
        // while the rest streams. Non-temporal: the stream does not displace
        // the activations, which every workgroup re-reads, from L2.
        i32x4 pf[C::kLoads];
        auto load_piece = [&](int u) {
            // The whole offset goes in the vector operand: that is the part
            // the buffer range check sees, so a piece past the end reads 0.
            const uint32_t piece = min((uint32_t)(lane + 64 * u), nq - 1u);
            pf[u] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, A0 + 16u * piece, 0, kNonTemporal);
        };
        static_for<0, kWindow>([&](auto uc) {
            if constexpr (decltype(uc)::value < C::kLoads) load_piece(decltype(uc)::value);
        });

        // Bitmaps and activations landed first (issued earlier); stage them
        // while the payload is in flight. Bitmap words past the chunk are zero:
        // padding LTs decode to zero and read inside the stage.
#pragma unroll
        for (int v = 0; v < C::kBmLoads; ++v)
            if (lane + 64 * v < C::kBmWords) st_bm[lane + 64 * v] = lane + 64 * v < 8 * cnt ? pbm[v] : 0u;
#pragma unroll
        for (int u = 0; u < kXLoads; ++u) {
            const int n = u * kXRowsPerLoad + x_row_slot;
            if (u < x_loads && n < N && x_piece < 2 * CH) *(i32x4 *)(st_x + n * C::kXRowWords + 4 * x_piece) = px[u];
        }

        // Bit address, within the stage, of payload value 0 of the whole matrix.
        const uint32_t s4base = 4u * (0u - 2u * A0);
        auto o_at = [&](int j) { return lane_value(offv, j); };
        auto decode_one = [&](int j) {
            const uint32_t oj = o_at(j), sd = o_at(j + 1) - oj;
            const i32x4 A = decode_tile(st, lut, st_bm[8 * j + i], s4base + 4u * oj, sd, amask & (sd >> 1),
                                        g, lomask);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const uint32_t *xl = xq[nb] + 8 * j;
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, unpack_x(xl[0], xl[4]), acc[nb], 0, 0, 0);
            }
        };
        auto decode_two = [&](int j) {
            const uint32_t o0 = o_at(j), o1 = o_at(j + 1), o2 = o_at(j + 2);
            const uint32_t sd0 = o1 - o0, sd1 = o2 - o1;
            const i32x4 A0v = decode_tile(st, lut, st_bm[8 * j + i], s4base + 4u * o0, sd0,
                                          amask & (sd0 >> 1), g, lomask);
            const i32x4 A1v = decode_tile(st, lut, st_bm[8 * (j + 1) + i], s4base + 4u * o1, sd1,
                                          amask & (sd1 >> 1), g, lomask);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const uint32_t *xl = xq[nb] + 8 * j;
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A0v, unpack_x(xl[0], xl[4]), acc[nb], 0, 0, 0);
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A1v, unpack_x(xl[8], xl[12]), acc[nb], 0, 0, 0);
            }
        };

        // The payload lands in issue order: after load u, stage bytes
        // [0, 1024 (u + 1)) are present, so every LT whose windows end there
        // (o_{t+1} - 2 A0 + 16 <= 2048 (u + 1) values) can be decoded.
        int j = 0;
        static_for<0, C::kLoads>([&](auto uc) {
            constexpr int u = decltype(uc)::value;
            constexpr int later = (kWindow - 1 < C::kLoads - 1 - u) ? kWindow - 1 : C::kLoads - 1 - u;
            wait_vm<later>();                              // piece u has landed
            if constexpr (u + kWindow < C::kLoads) load_piece(u + kWindow);
            const uint32_t piece = (uint32_t)(lane + 64 * u);
            if (piece < nq) *(i32x4 *)(st + 4 * piece) = pf[u];
            __asm__ volatile("" ::: "memory");
            if constexpr (u + 1 < C::kLoads) {
                const uint32_t lim = 2u * A0 + 2048u * (u + 1) - 16u;   // wraps only when ready is unprovable
                while (j + 1 < cnt && o_at(j + 2) <= lim) {
                    decode_two(j);
                    j += 2;
                }
            } else {
                for (; j + 1 < cnt; j += 2) decode_two(j);
                if (j < cnt) decode_one(j);
            }
        });
        __asm__ volatile("" ::: "memory");

        // Next chunk (long slices only): offsets, then its side data.
        const int nnext = nlt - c0 - CH;
        if (nnext > 0) {
            offv = p.off[t0 + c0 + CH + min(lane, min(nnext, CH))];
            request_side(c0 + CH, pbm, px);
        }
    };
    // The first chunk is straight-line code after the prologue, so every
    // wait above counts loads exactly; later chunks only occur for long slices.
    if (nlt > 0) process_chunk(0);
    for (int c0 = CH; c0 < nlt; c0 += CH) process_chunk(c0);

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
    for (int e = threadIdx.x; e < 16 * N; e += 64 * WPG) {
        const int r = e & 15, n = e >> 4;
        int32_t s = 0;
#pragma unroll
        for (int w = 0; w < WPG; ++w) s += ((const int32_t *)(lds + (2048 + w * stage_bytes) / 4))[r * (16 * NB) + n];
        const int32_t yv = s >> 8;                            // exact: s = 256 Y
        const int64_t m = (int64_t)mb * 16 + r;
        p.y[n * M + m] = yv;
        if (p.scale) p.yf[n * M + m] = (float)yv * p.scale[m];
    }
}

constexpr int kLutBytes = 2048;
constexpr int kMaxLds = 160 * 1024;

template <int CH>
int stage_bytes(int N) { return (Chunk<CH>::bytes(N) + 15) & ~15; }

int lds_bytes(int ch, int N, int wpg) {
    const int st = ch == 16 ? stage_bytes<16>(N)
                 : ch == 12 ? stage_bytes<12>(N)
                 : ch == 8  ? stage_bytes<8>(N)
                            : stage_bytes<4>(N);
    return kLutBytes + wpg * st;
}

template <int WPG, int NB, int CH>
hipError_t launch_spmm(const SpmmArgs &a, hipStream_t s) {
    auto kern = us_spmm_kernel<WPG, NB, CH>;
    // Allow more than 64 KB of dynamic LDS (set once per instantiation).
    static const hipError_t attr =
        hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds);
    (void)attr;
    const int st = stage_bytes<CH>(a.N);
    hipLaunchKernelGGL(kern, dim3(a.M / 16), dim3(64 * WPG), kLutBytes + WPG * st, s, a, st);
    return hipGetLastError();
}

template <int NB, int CH>
hipError_t launch_spmm_wpg(int wpg, const SpmmArgs &a, hipStream_t s) {
    switch (wpg) {
        case 1: return launch_spmm<1, NB, CH>(a, s);
        case 2: return launch_spmm<2, NB, CH>(a, s);
        case 4: return launch_spmm<4, NB, CH>(a, s);
        case 8: return launch_spmm<8, NB, CH>(a, s);
        default: return launch_spmm<16, NB, CH>(a, s);
    }
}

hipError_t launch_cfg(int wpg, int ch, const SpmmArgs &a, hipStream_t s) {
    if (a.N > 16) return ch == 8 ? launch_spmm_wpg<2, 8>(wpg, a, s) : launch_spmm_wpg<2, 4>(wpg, a, s);
    switch (ch) {
        case 16: return launch_spmm_wpg<1, 16>(wpg, a, s);
        case 12: return launch_spmm_wpg<1, 12>(wpg, a, s);
        case 8: return launch_spmm_wpg<1, 8>(wpg, a, s);
        default: return launch_spmm_wpg<1, 4>(wpg, a, s);
    }
}

bool aligned(const void *ptr, uintptr_t n) { return ((uintptr_t)ptr % n) == 0; }

// Chunk length for wpg slices: the smallest of 4, 8, 12, 16 LTs (4 or 8 with
// two MFMA column blocks) that holds a whole slice and fits LDS; else the
// largest that fits (the slice then takes several chunks). 4 always fits.
int pick_chunk(int nkb, int N, int wpg) {
    const int slice = (nkb + wpg - 1) / wpg;
    const int cands[4] = {4, 8, 12, 16};
    const int nc = N > 16 ? 2 : 4;
    int best = 0;
    for (int c = 0; c < nc; ++c) {
        if (lds_bytes(cands[c], N, wpg) > kMaxLds) break;
        best = cands[c];
        if (cands[c] >= slice) return best;
    }
    return best;
}

// Wavefronts per workgroup (= K slices per row block): at least 16 wavefronts
// per CU over 256 CUs, one chunk per slice where 16 slices allow it, at least
// one LT per slice, and an LDS footprint that fits.
void auto_config(int M, int K, int N, int &wpg, int &ch) {
    const int nrb = M / 16, nkb = K / 64;
    int w = 1;
    while (w < 16 && nrb * w < 256 * 16) w *= 2;
    while (w > 1 && w > nkb) w /= 2;
    wpg = w;
    ch = pick_chunk(nkb, N, w);
    // Widen while a slice still needs several chunks and a wider split fits.
    while (w < 16 && 2 * w <= nkb && ch < (nkb + w - 1) / w) {
        w *= 2;
        const int c = pick_chunk(nkb, N, w);
        if (lds_bytes(c, N, w) > kMaxLds) break;
        wpg = w;
        ch = c;
    }
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
    if (!aligned(w->bitmaps, 8) || !aligned(w->offsets, 4) || !aligned(x, 16) || !aligned(y, 4) ||
        (scale && (!aligned(scale, 4) || !aligned(y_f32, 4))))
        return US_ERR_ARG;

    int wpg = 0, ch = 0;
    auto_config(M, K, N, wpg, ch);
    if (opts) {
        if (opts->variant != 0) return US_ERR_ARG;
        const int s = opts->split_k;
        if (s != 0) {
            if (s != 1 && s != 2 && s != 4 && s != 8 && s != 16) return US_ERR_ARG;
            wpg = s;
            ch = pick_chunk((int)nkb, N, wpg);
        }
    }
    if (ch == 0) return US_ERR_ARG;                        // no chunk fits LDS

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
    const hipError_t err = launch_cfg(wpg, ch, a, s);
    return err == hipSuccess ? US_OK : US_ERR_DEVICE;
}
