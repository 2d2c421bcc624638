// IE-BME x INT4 -> INT32 sparse product on gfx950: the single-pass kernel
// family. Same operation and decode as the chunked kernel of us_spmm_kernel.h
// (Section VI: the UnionSparse kernel, its LSPD decode and split-K), with
// three differences:
//
//  * Split-K across workgroups (Section VI-C, the "UnionSparse Kernel"
//    algorithm: a grid of split-K batches by row tiles, each batch storing
//    its partial tile to a reduction workspace, then a reduction). With
//    kblocks > 1 the grid is (row blocks) x (K blocks). Each workgroup's WPG
//    wavefronts split its K block and combine their partial tiles in LDS;
//    the workgroup then adds its tile into a workspace accumulator with
//    relaxed device-scope integer atomics (exact in any order) and takes a
//    ticket. The workgroup that arrives last reads and clears the
//    accumulator with an atomic exchange, writes Y (and the dequantised Y)
//    and resets the ticket. Every access to the shared words is an atomic
//    performed at the device's coherence point, so no cache maintenance is
//    needed and the workspace is left zeroed for the next call. This lets a
//    matrix with fewer 16-row blocks than the GPU has compute units use all
//    of them.
//
//  * One pass per wavefront, static decode order. A wavefront's K slice (at
//    most CH LTs of one 16-row block) is staged whole; its inputs (offsets,
//    bitmaps, permutations, activations) go straight into LDS with
//    direct-to-LDS loads, and its payload is streamed with a window of WIN
//    loads. LTs are decoded in pairs in a fixed order, every LDS address a
//    loop-invariant register plus an immediate offset; before a pair the
//    wavefront waits for the load that holds the pair's bytes in the worst
//    case, so the schedule needs no data-dependent scalar bookkeeping.
//
//  * Row reordering (Section V-B): with PERM each LT's row base and mask row
//    are stored together per MFMA lane row ([base, mask row], 8 bytes), routed
//    to the lane row of the original row in the row-base pass, and the decode
//    reads both with one LDS instruction.
#ifndef UNIONSPARSE_US_SPMM_BURST_H
#define UNIONSPARSE_US_SPMM_BURST_H

#include "us_spmm_kernel.h"

namespace us_spmm_detail {

// LDS stage of one wavefront's slice of at most CH LTs, in bytes from the
// stage start:
//   payload : the slice's compressed values from the 16-byte boundary at or
//             below its first byte; 8 BITS CH + 2 pieces of 16 bytes cover
//             the largest slice (an LT holds at most 1024 values) with the
//             12-byte overhang of its last window;
//   bitmaps : union-mask rows, 8 dwords per LT;
//   records : without PERM the row base (a slot address, see the chunked
//             kernel) of each lane row (16 dwords per LT); with PERM
//             [row base, mask row] per lane row (32 dwords per LT);
//   offsets : o_t of the slice's LTs and the end offset;
//   perm    : (PERM) the row permutation word of each LT;
//   X       : the slice's activations, one row of 32 bytes per LT for each
//             column, rows padded by 16 bytes so that the 16 rows read by one
//             instruction fall in different banks.
// Per-LT arrays have room for whole 4-LT passes of the row-base step.
template <int CH, bool PERM, int BITS>
struct Burst {
    static constexpr int kPayPieces = 8 * BITS * CH + 2;
    static constexpr int kLoads = (kPayPieces + 63) / 64;     // payload loads of 1 KB per wavefront
    static constexpr int kPasses = (CH + 3) / 4;
    static constexpr int kLtPad = 4 * kPasses;
    static constexpr int kRec = PERM ? 128 : 64;              // record bytes per LT
    static constexpr int kBmOffset = 16 * kPayPieces;
    static constexpr int kRecOffset = kBmOffset + 32 * kLtPad;
    static constexpr int kOffOffset = kRecOffset + kRec * kLtPad;
    static constexpr int kPermOffset = (kOffOffset + 4 * (kLtPad + 1) + 7) & ~7;
    static constexpr int kXOffset = (kPermOffset + (PERM ? 8 * kLtPad : 0) + 15) & ~15;
    static constexpr int kXRowWords = 8 * CH + 4;
    static constexpr int kXPieces = 2 * CH;                   // 16-byte pieces of one activation row
    static constexpr int kXRowsPerLoad = kXPieces <= 32 ? 2 : 1;  // activation rows per 64-lane load
    static_assert(kLoads <= 32, "vmcnt range");
    static_assert(kXPieces <= 64, "one activation row per load");
    static constexpr int bytes(int N) { return kXOffset + 4 * kXRowWords * N; }
};

// A raw buffer descriptor over `bytes` bytes from `base` (32-bit data, no
// swizzle); loads past the range read zero without a memory access.
__device__ __forceinline__ u32x4 raw_desc(const void *base, uint32_t bytes) {
    const uint64_t a = (uint64_t)(size_t)base;
    return (u32x4){(uint32_t)a, (uint32_t)(a >> 32) & 0xFFFFu, bytes, (uint32_t)kBufferDword3};
}

// Direct-to-LDS loads for the inputs (see dma16, which the payload uses):
// dma4 moves 4 bytes per lane to LDS [lds + 4 lane, lds + 4 lane + 4)
// (non-temporal: read once); dma16_keep moves 16 bytes per lane like dma16
// but with the default cache policy (the activations are read by every
// workgroup).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma4(u32x4 desc, uint32_t lds, uint32_t voff, uint32_t soff) {
    __asm__ volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen nt lds"
                     :
                     : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(desc),
                       "s"(__builtin_amdgcn_readfirstlane(soff))
                     : "memory", "m0");
}
__device__ __forceinline__ void dma16_keep(u32x4 desc, uint32_t lds, uint32_t voff, uint32_t soff) {
    __asm__ volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                     :
                     : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(desc),
                       "s"(__builtin_amdgcn_readfirstlane(soff))
                     : "memory", "m0");
}
#pragma clang diagnostic pop

// Eight INT4 activations of each of two dwords -> the four B-operand dwords,
// values in the high nibble (16 x), slot order of unpack_x.
__device__ __forceinline__ i32x4 unpack_x2(uint2 x) {
    const uint64_t v = ((uint64_t)x.y << 32) | x.x;
    const uint64_t s = v << 4;
    return (i32x4){(int32_t)((uint32_t)s & kHiNib), (int32_t)(x.x & kHiNib), (int32_t)((uint32_t)(s >> 32) & kHiNib),
                   (int32_t)(x.y & kHiNib)};
}

// Resident wavefronts per SIMD a burst instantiation is built for (its
// launch bound, and the host's residency model).
constexpr int burst_waves_per_simd(int wpg, int nmax) { return nmax > 4 ? (wpg >= 4 ? 6 : 5) : (wpg >= 4 ? 7 : 6); }

struct BurstArgs {
    SpmmArgs a;
    int32_t kblocks;        // K blocks (grid.y); > 1 uses the workspace
    int32_t *ws_acc;        // N x M int32 accumulators (kblocks > 1), zero between calls
    uint32_t *ws_tick;      // M / 16 arrival tickets (kblocks > 1), zero between calls
};

template <int WPG, int NMAX, int CH, bool PERM, int BITS, int WIN>
__global__ __launch_bounds__(64 * WPG, burst_waves_per_simd(WPG, NMAX)) void us_spmm_burst_kernel(BurstArgs ba,
                                                                                                  int stage_bytes) {
    const SpmmArgs &p = ba.a;
    using C = Burst<CH, PERM, BITS>;
    static_assert(BITS == 4 || BITS == 2, "payload values are 4 or 2 bits");
    static_assert(NMAX <= 16, "one MFMA column block");
    static_assert(WIN >= 1 && WIN <= C::kLoads, "payload window");
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    __shared__ u32x2 lut[256];
    __shared__ int last_arrival;
    const uint32_t lds0 = (uint32_t)(size_t)(lds_u32 *)lds;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int mb = blockIdx.x;
    const int N = p.N;

    // K range of this workgroup (K block blockIdx.y of ba.kblocks), then this
    // wavefront's slice of it; the first (range mod WPG) wavefronts take one
    // LT more. The host guarantees 1 <= nlt <= CH.
    const int nkb = p.nkb;
    const int kbk = blockIdx.y;
    const int r0 = (int)(((int64_t)nkb * kbk) / ba.kblocks), r1 = (int)(((int64_t)nkb * (kbk + 1)) / ba.kblocks);
    const int rn = r1 - r0;
    const int kb0 = __builtin_amdgcn_readfirstlane(r0 + wave * (rn / WPG) + min(wave, rn % WPG));
    const int nlt = __builtin_amdgcn_readfirstlane(rn / WPG + (wave < rn % WPG ? 1 : 0));
    const int64_t t0 = (int64_t)mb * nkb + kb0;

    const int rr = lane & 15;
    const int i = rr >> 1;
    const int g = lane >> 4;
    const uint32_t amask = (rr & 1) ? ~0u : 0u;
    const uint32_t lomask = (1u << (8 * g)) - 1u;
    const uint32_t rot = (uint32_t)(8 * g + 29) & 31u;

    const uint32_t st = lds0 + (uint32_t)(wave * stage_bytes);
    const uint32_t st_bm = st + C::kBmOffset, st_rec = st + C::kRecOffset;
    const uint32_t st_off = st + C::kOffOffset;
    const uint32_t st_pm = st + C::kPermOffset, st_x = st + C::kXOffset;

    // Inputs, straight into the stage with direct-to-LDS loads, each lane
    // reading only bytes of this slice: offsets (lane j <= nlt: o_{t0 + j}),
    // bitmaps (one 16-byte piece per half LT), permutation words (one dword
    // per half word), and the activation slice, one load per activation row
    // (piece q < 2 nlt of the row). No input passes through registers.
    {
        const u32x4 odesc = raw_desc(p.off, 0xFFFFFFFFu);
        if (lane <= nlt) dma4(odesc, st_off, (uint32_t)(4 * (t0 + lane)), 0u);
        const u32x4 bdesc = raw_desc(p.bm32, 0xFFFFFFFFu);
        if (lane < 2 * nlt) dma16(bdesc, st_bm, (uint32_t)(32 * t0 + 16 * lane), 0u);
        if constexpr (PERM) {
            const u32x4 pdesc = raw_desc(p.perm32, 0xFFFFFFFFu);
            if (lane < 2 * nlt) dma4(pdesc, st_pm, (uint32_t)(8 * t0 + 4 * lane), 0u);
        }
        const u32x4 xdesc = raw_desc(p.x, (uint32_t)(N * (p.K / 2)));
        const uint32_t xoff = (uint32_t)(32 * kb0 + 16 * lane);
        if (lane < 2 * nlt) {
            for (int n = 0; n < N; ++n)
                dma16_keep(xdesc, st_x + 4u * (uint32_t)(n * C::kXRowWords), xoff, (uint32_t)(n * (p.K / 2)));
        }
    }
    // The dequant scale of the output row this thread stores in the
    // epilogue (a zero-sized range without a scale array).
    const __amdgpu_buffer_rsrc_t ssrc =
        __builtin_amdgcn_make_buffer_rsrc((void *)p.scale, (short)0, p.scale ? 4 * p.M : 0, kBufferDword3);
    const float row_scale = __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(ssrc, (uint32_t)(4 * (mb * 16 + (int)(threadIdx.x & 15))), 0, 0));

    // Selector table, computed while the requests fly.
    for (int e = threadIdx.x; e < 256; e += 64 * WPG) lut[e] = perm_selectors<BITS>((uint32_t)e);
    // The youngest wavefronts of a CU, which its SIMDs' arbiters serve last,
    // start at a higher issue priority: the workgroup's dispatch round
    // (blockIdx / CUs) plus the wavefront's place among the workgroup's
    // wavefronts on its SIMD (wave / 4), at most 3; every wavefront returns
    // to 0 once half of its slice is decoded.
    {
        const int rank = min(3, (int)((blockIdx.x + blockIdx.y * gridDim.x) / max(p.n_cu, 1)) + (wave >> 2));
        if (rank == 1) __builtin_amdgcn_s_setprio(1);
        else if (rank == 2) __builtin_amdgcn_s_setprio(2);
        else if (rank >= 3) __builtin_amdgcn_s_setprio(3);
    }
    __syncthreads();                                       // selector table complete
    // The payload is requested once the inputs have landed: requested
    // earlier, it queues ahead of the other wavefronts' inputs, and no
    // wavefront can decode before its inputs are in.
    wait_vm_all();
    __asm__ volatile("" ::: "memory");

    // The slice's payload span. A0 is the first staged byte (16-byte
    // aligned, never past the end of the payload); pieces beyond the span or
    // the payload read zero and cost no traffic.
    const uint32_t ob = __builtin_amdgcn_readfirstlane(lds_load(st_off));
    const uint32_t oe = __builtin_amdgcn_readfirstlane(lds_load(st_off + 4 * nlt));
    const uint32_t pay_bytes = (uint32_t)p.pay_bytes;
    const uint32_t A0 = us_range::first_byte<BITS>(ob, pay_bytes);
    const uint32_t prange = us_range::range_bytes<BITS>(oe, A0, pay_bytes, (uint32_t)C::kPayPieces);

    // Payload: 16-byte pieces from A0; load u brings stage bytes
    // [1024 u, 1024 u + 1024). At most WIN loads are in flight: the first WIN
    // go out now, and load u + WIN once load u has landed. The schedule is
    // static: before LT pair p the wavefront waits for the load that holds
    // the pair's last window in the worst case (every LT of the slice at its
    // largest, 128 BITS bytes), so no scalar bookkeeping depends on the
    // data. Loads past the slice's last piece read zero and cost no traffic;
    // the last one writes only the pieces the stage holds.
    const uint64_t pa = (uint64_t)(size_t)(p.pay + A0);
    const u32x4 pdesc = (u32x4){(uint32_t)pa, (uint32_t)(pa >> 32) & 0xFFFFu, prange, (uint32_t)kBufferDword3};
    auto issue = [&](auto uc) {
        constexpr int u = decltype(uc)::value;
        if constexpr (u < C::kLoads) {
            if (u + 1 < C::kLoads || C::kPayPieces % 64 == 0 || lane + 64 * u < C::kPayPieces)
                dma16(pdesc, st + 1024u * u, (uint32_t)(16 * lane), 1024u * u);
        }
    };
    static_for<0, WIN>([&](auto uc) { issue(uc); });

    // Row bases (the LSPD prefix scan, once per LT and lane row): lanes
    // 16 jj + rr handle LT 4 pass + jj, mask row i, area row a; see the
    // chunked kernel for the scan. With PERM the record of reordered row
    // 8a + i goes to the lane row of original row pi[8a + i].
    {
        const uint32_t jj = (uint32_t)lane >> 4;
#pragma unroll
        for (int ps = 0; ps < C::kPasses; ++ps) {
            const uint32_t j = 4 * ps + jj;
            const uint32_t mrow = lds_load(st_bm + 32 * j + 4 * i);
            const uint2 o = lds_load2(st_off + 4 * min(j, (uint32_t)CH - 1));
            [[maybe_unused]] uint32_t pm = 0;
            if constexpr (PERM) pm = lds_load(st_pm + 8 * j + 4 * (rr & 1));
            const uint32_t inj = amask & ((o.y - o.x) >> 2);      // P_t
            uint32_t ex = (uint32_t)__builtin_amdgcn_update_dpp((int)inj, (int)__popc(mrow), 0x112, 0xF, 0xF, false);
            ex += dpp_row<0x112>(ex);
            ex += dpp_row<0x114>(ex);
            ex += dpp_row<0x118>(ex);
            constexpr uint32_t kSlotsPerByte = 4 / BITS;
            const uint32_t bval = kSlotsPerByte * st + ((o.x >> 1) + ex - kSlotsPerByte * A0);
            if constexpr (PERM) {
                const uint32_t rec = st_rec + C::kRec * j;
                lds_store2(rec + 8 * rr, (u32x2){bval, mrow});
                const uint32_t r = (pm >> (4 * i)) & 15u;
                lds_store2(rec + 8u * (((r & 7u) << 1) | (r >> 3)), (u32x2){bval, mrow});
            } else {
                lds_store(st_rec + C::kRec * j + 4 * rr, bval);
            }
        }
    }

    // Decode, pair by pair, in a fixed order.
    const uint32_t a_bm = st_bm + 4 * i;
    const uint32_t a_rec = st_rec + (PERM ? 8 : 4) * rr;
    uint32_t a_x = st_x + 4u * (uint32_t)(min(rr, N - 1) * C::kXRowWords + g);
    __asm__("" : "+v"(a_x));                               // one base register, immediate offsets per LT
    i32x4 acc = (i32x4){0, 0, 0, 0};

    // Row base and mask row of LT j for this lane.
    auto row_of = [&](auto jc, uint32_t &mrow, uint32_t &base) {
        constexpr int j = decltype(jc)::value;
        if constexpr (PERM) {
            const u32x2 rb = *(const lds_u2 *)(size_t)(a_rec + C::kRec * j);
            base = rb.x;
            mrow = rb.y;
        } else {
            mrow = lds_load(a_bm + 32 * j);
            base = lds_load(a_rec + C::kRec * j);
        }
    };
    auto x_of = [&](auto jc) {
        constexpr int j = decltype(jc)::value;
        return make_uint2(lds_load(a_x + 32 * j), lds_load(a_x + 32 * j + 16));
    };
    auto decode_one = [&](auto jc) {
        uint32_t mrow, base;
        row_of(jc, mrow, base);
        const i32x4 A = decode_tile<BITS>(lut, mrow, base, lomask, rot);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, unpack_x2(x_of(jc)), acc, 0, 0, 0);
    };
    // Two LTs with every LDS request of both issued before either waits:
    // addresses of both, then the windows, selectors and activations of both,
    // then the placement of both.
    auto decode_two = [&](auto jc) {
        constexpr int j = decltype(jc)::value;
        uint32_t m0, b0, m1, b1;
        row_of(std::integral_constant<int, j>(), m0, b0);
        row_of(std::integral_constant<int, j + 1>(), m1, b1);
        const uint32_t p0 = b0 + (uint32_t)__popc(m0 & lomask);
        const uint32_t p1 = b1 + (uint32_t)__popc(m1 & lomask);
        const uint2 w0 = slot_window<BITS>(p0), w1 = slot_window<BITS>(p1);
        const uint2 e0 = selectors(lut, m0, rot), e1 = selectors(lut, m1, rot);
        const uint2 x0 = x_of(std::integral_constant<int, j>()), x1 = x_of(std::integral_constant<int, j + 1>());
        const i32x4 A0v = place_slots<BITS>(w0, e0);
        const i32x4 A1v = place_slots<BITS>(w1, e1);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(A0v, unpack_x2(x0), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(A1v, unpack_x2(x1), acc, 0, 0, 0);
    };
    // A pair whose second LT exists takes a straight-line path of its own.
    // Pair p covers LTs 2p and 2p + 1: at most 128 BITS (2p + 2) + 15 bytes
    // from A0 with the alignment, plus the window overhang (12 bytes for
    // 4-bit slots, 8 for 2-bit), so it needs loads up to
    // U(p) = min(kLoads - 1, (256 BITS (p + 1) + 15 + overhang) / 1024).
    constexpr int kSpan = BITS == 4 ? 27 : 23;
    static_for<0, (CH + 1) / 2>([&](auto pc) {
        constexpr int pr = decltype(pc)::value;
        constexpr int kNeed = (256 * BITS * (pr + 1) + kSpan) / 1024 < C::kLoads - 1
                                  ? (256 * BITS * (pr + 1) + kSpan) / 1024
                                  : C::kLoads - 1;
        constexpr int kPrev = pr == 0 ? -1
                              : ((256 * BITS * pr + kSpan) / 1024 < C::kLoads - 1 ? (256 * BITS * pr + kSpan) / 1024
                                                                                  : C::kLoads - 1);
        if (2 * pr < nlt) {
            // Loads issued so far: those up to kPrev + WIN (or the first WIN).
            constexpr int kIssued = (kPrev + 1 + WIN) < C::kLoads ? kPrev + 1 + WIN : C::kLoads;
            constexpr int kAllowed = kIssued - 1 - kNeed;      // loads that may stay in flight
            wait_vm<kAllowed < 0 ? 0 : kAllowed>();
            static_for<kIssued, (kNeed + 1 + WIN < C::kLoads ? kNeed + 1 + WIN : C::kLoads)>([&](auto uc) { issue(uc); });
            if constexpr (4 * pr + 4 >= CH) __builtin_amdgcn_s_setprio(0);
            __asm__ volatile("" ::: "memory");
            if constexpr (2 * pr + 1 < CH) {
                if (2 * pr + 1 < nlt) {
                    decode_two(std::integral_constant<int, 2 * pr>());
                } else {
                    decode_one(std::integral_constant<int, 2 * pr>());
                }
            } else {
                decode_one(std::integral_constant<int, 2 * pr>());
            }
        }
    });
    wait_vm_all();                                         // no payload write may still target the stage
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_setprio(0);

    // Split-K combine: each wavefront leaves its 16 x 16 partial in its stage
    // (MFMA result layout: lane l, element v -> row 4 (l / 16) + v, column
    // l % 16); after the barrier, threads e, e + 64 WPG, ... sum the WPG
    // partials of outputs e < 16 N (row e mod 16, column e / 16), all of them
    // in the row of the dequant scale the thread loaded.
    lds_store4(st + 16 * lane, (u32x4)acc);
    __syncthreads();
    const int64_t M = p.M;
    constexpr int kShift = BITS == 4 ? 8 : 10;
    auto partial_sum = [&](int e) {
        const int r = e & 15, n = e >> 4;
        const int R = 2 * (r & 7) + (r >> 3);              // W row 8a + i is MFMA row 2i + a
        const uint32_t idx = 4u * (uint32_t)(4 * (16 * (R >> 2) + n) + (R & 3));
        int32_t s = 0;
#pragma unroll
        for (int w = 0; w < WPG; ++w) s += (int32_t)lds_load(lds0 + (uint32_t)(w * stage_bytes) + idx);
        return s;
    };
    auto store = [&](int e, int32_t total) {
        const int64_t m = (int64_t)mb * 16 + (e & 15), n = e >> 4;
        const int32_t yv = total >> kShift;                    // exact: total = 256 Y (1024 Y)
        p.y[n * M + m] = yv;
        if (p.scale) p.yf[n * M + m] = (float)yv * row_scale;
    };
    if (ba.kblocks == 1) {
        for (int e = threadIdx.x; e < 16 * N; e += 64 * WPG) store(e, partial_sum(e));
        return;
    }
    // Across workgroups: accumulate, take a ticket, the last one finishes.
    for (int e = threadIdx.x; e < 16 * N; e += 64 * WPG) {
        const int64_t m = (int64_t)mb * 16 + (e & 15), n = e >> 4;
        __hip_atomic_fetch_add(ba.ws_acc + n * M + m, partial_sum(e), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    wait_vm_all();                                         // the adds are performed before the ticket
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t old = __hip_atomic_fetch_add(ba.ws_tick + mb, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last_arrival = old == (uint32_t)(ba.kblocks - 1);
    }
    __syncthreads();
    if (!last_arrival) return;
    for (int e = threadIdx.x; e < 16 * N; e += 64 * WPG) {
        const int64_t m = (int64_t)mb * 16 + (e & 15), n = e >> 4;
        store(e, __hip_atomic_exchange(ba.ws_acc + n * M + m, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    }
    if (threadIdx.x == 0) __hip_atomic_store(ba.ws_tick + mb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// LTs per wavefront slice of the burst instantiations.
constexpr int kBurstChs[] = {4, 8, 11, 16, 22, 32};
constexpr int kNumBurstChs = sizeof(kBurstChs) / sizeof(kBurstChs[0]);

template <int CH, bool PERM, int BITS>
int burst_stage_bytes(int N) { return (Burst<CH, PERM, BITS>::bytes(N) + 15) & ~15; }

template <bool PERM, int BITS>
int burst_lds_bytes_t(int ch, int N, int wpg) {
    int st = 0;
    switch (ch) {
        case 4: st = burst_stage_bytes<4, PERM, BITS>(N); break;
        case 8: st = burst_stage_bytes<8, PERM, BITS>(N); break;
        case 11: st = burst_stage_bytes<11, PERM, BITS>(N); break;
        case 16: st = burst_stage_bytes<16, PERM, BITS>(N); break;
        case 22: st = burst_stage_bytes<22, PERM, BITS>(N); break;
        default: st = burst_stage_bytes<32, PERM, BITS>(N); break;
    }
    return kLutBytes + 16 + wpg * st;
}

inline int burst_lds_bytes(int ch, int N, int wpg, bool perm, int bits) {
    if (bits == 2) return perm ? burst_lds_bytes_t<true, 2>(ch, N, wpg) : burst_lds_bytes_t<false, 2>(ch, N, wpg);
    return perm ? burst_lds_bytes_t<true, 4>(ch, N, wpg) : burst_lds_bytes_t<false, 4>(ch, N, wpg);
}

#ifndef US_BURST_WINDOW
#define US_BURST_WINDOW 2
#endif
constexpr int kBurstWindow = US_BURST_WINDOW;              // payload loads in flight per wavefront

template <int WPG, int NMAX, int CH, bool PERM, int BITS>
hipError_t launch_burst(const BurstArgs &b, hipStream_t s) {
    constexpr int kWin = kBurstWindow < Burst<CH, PERM, BITS>::kLoads ? kBurstWindow : Burst<CH, PERM, BITS>::kLoads;
    auto kern = us_spmm_burst_kernel<WPG, NMAX, CH, PERM, BITS, kWin>;
    static std::atomic<unsigned long long> attr_set{0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    const unsigned long long bit = 1ull << (dev & 63);
    if (!(attr_set.load(std::memory_order_acquire) & bit)) {
        const hipError_t e =
            hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds - kLutBytes - 16);
        if (e != hipSuccess) return e;
        attr_set.fetch_or(bit, std::memory_order_release);
    }
    const int st = burst_stage_bytes<CH, PERM, BITS>(b.a.N);
    hipLaunchKernelGGL(kern, dim3(b.a.M / 16, b.kblocks), dim3(64 * WPG), WPG * st, s, b, st);
    return hipGetLastError();
}

template <int NMAX, int CH, bool PERM, int BITS>
hipError_t launch_burst_wpg(int wpg, const BurstArgs &b, hipStream_t s) {
    switch (wpg) {
        case 1: return launch_burst<1, NMAX, CH, PERM, BITS>(b, s);
        case 2: return launch_burst<2, NMAX, CH, PERM, BITS>(b, s);
        case 4: return launch_burst<4, NMAX, CH, PERM, BITS>(b, s);
        case 8: return launch_burst<8, NMAX, CH, PERM, BITS>(b, s);
        default: return launch_burst<16, NMAX, CH, PERM, BITS>(b, s);
    }
}

template <bool PERM, int BITS, int NMAX>
hipError_t launch_burst_cfg(int wpg, int ch, const BurstArgs &b, hipStream_t s) {
    switch (ch) {
        case 4: return launch_burst_wpg<NMAX, 4, PERM, BITS>(wpg, b, s);
        case 8: return launch_burst_wpg<NMAX, 8, PERM, BITS>(wpg, b, s);
        case 11: return launch_burst_wpg<NMAX, 11, PERM, BITS>(wpg, b, s);
        case 16: return launch_burst_wpg<NMAX, 16, PERM, BITS>(wpg, b, s);
        case 22: return launch_burst_wpg<NMAX, 22, PERM, BITS>(wpg, b, s);
        default: return launch_burst_wpg<NMAX, 32, PERM, BITS>(wpg, b, s);
    }
}

// Instantiation families, one translation unit each.
hipError_t launch_burst_plain(int wpg, int ch, const BurstArgs &b, hipStream_t s);    // 4-bit, N <= 16
hipError_t launch_burst_narrow(int wpg, int ch, const BurstArgs &b, hipStream_t s);   // 4-bit, N <= 4
hipError_t launch_burst_perm(int wpg, int ch, const BurstArgs &b, hipStream_t s);     // reordered, N <= 16
hipError_t launch_burst_w2(int wpg, int ch, const BurstArgs &b, hipStream_t s);       // 2-bit, N <= 16

}  // namespace us_spmm_detail

#endif  // UNIONSPARSE_US_SPMM_BURST_H
