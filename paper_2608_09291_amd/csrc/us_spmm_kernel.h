// IE-BME x INT4 -> INT32 sparse product on gfx950 (CDNA4): the chunked
// kernel and its launch templates, instantiated by us_spmm.hip (4-bit
// weights, rows in stored order), us_spmm_narrow.hip (the same for N <= 4),
// us_spmm_perm.hip (row-reordered LTs) and us_spmm_w2.hip (2-bit weights);
// the single-pass family (us_spmm_burst.h) shares its decode helpers.
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
//    For a chunk the wavefront first reads the chunk's offsets, then streams
//    its payload with 16-byte buffer loads (a few in flight, the rest issued
//    as earlier ones land) while the bitmaps and the activation slice, which
//    were requested together with the offsets, are copied into the
//    wavefront's own LDS stage. The payload is staged whole (loaded straight
//    into LDS up to 16 activation columns, via registers above) or through
//    a 4 KB ring via registers (see Chunk). A slice of several chunks
//    requests the next chunk's inputs ahead of the current payload; above
//    16 activation columns it also requests the next chunk's first payload
//    pieces during the current chunk's last steps, so that its payload
//    streams on across chunk boundaries (kPipe). Only the wavefront itself
//    reads its stage: its vmcnt waits and its in-order LDS accesses order
//    staging before decoding, with no workgroup barrier. The host picks the
//    split, the chunk length and the staging per shape (choose_config).
//
//  * Decode (the paper's LSPD, Section VI-B). One LT (16 x 64) is decoded by
//    one wavefront straight into the A operand of v_mfma_i32_16x16x64_i8.
//    Lane l owns MFMA row l % 16 = 2 i + a (union-mask row i, area row a) and
//    k-group g = l / 16, which is the G = 8 bit segment g of mask row i.
//    idx_base is split in two: the popcount of the rows before row i is the
//    same for all four segments of a row, so it is computed once per LT and
//    chunk by a DPP scan over 16 lanes and kept in LDS as a stage slot
//    address; each lane adds the popcount of its row below bit 8 g. As in
//    the paper, one rank serves every area stream; here the payload stores
//    the two areas of an area row interleaved by rank, so that rank is one
//    slot holding both values (area q = 2a, columns 8g..8g+7, and q = 2a + 1,
//    columns 32+8g..32+8g+7), and one window of eight slots serves both
//    areas. Active values are placed into their byte slots with four
//    v_perm_b32 per window, selectors taken from a 256-entry table indexed by
//    the 8-bit segment; inactive slots get selector 0x0C (zero). LTs are
//    decoded in pairs so that two independent chains interleave.
//
//  * Row reordering (Section V-B). A reordered LT stores row pi[p] of the
//    original LT as its row p, so union-mask row i pairs rows pi[i] and
//    pi[8 + i]. The MFMA rows keep the original row order (the accumulator
//    is shared by all LTs of a row block), so PERM kernels route each
//    reordered row's row base and mask row to the lane row of its original
//    row while computing the row bases. The routed values overwrite the
//    LT's own bitmap and row-base areas of the stage (16-bit row bases in
//    the bitmap area, two LTs to a dword, the routed mask row in the
//    row-base area, where the permutation word was staged), so a reordered
//    stage is exactly as large as a plain one and takes the same
//    configurations.
//
//  * INT4 -> INT8. CDNA4 has no INT4 matrix instruction. Weights and
//    activations are expanded to bytes that hold the value in the high
//    nibble (16 v, exact in int8), so the MFMA sums are 256 Y; the epilogue
//    shifts right by 8. |256 Y| <= 256 * 64 * K < 2^31 for K <= US_K_MAX.
//    2-bit weights (BITS = 2, the W2A4 setting of Section VII) go to the top
//    two bits of a byte (64 v): the sums are 1024 Y, |1024 Y| <= 1024 * 16 K
//    < 2^31, and the epilogue shifts by 10.
//    Both operands put the even and the odd positions of each 8-group in
//    separate dwords, the same slot order on both sides of the product.
#ifndef UNIONSPARSE_US_SPMM_KERNEL_H
#define UNIONSPARSE_US_SPMM_KERNEL_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "us.h"
#include "us_range.h"

#ifndef US_SPMM_WINDOW
#define US_SPMM_WINDOW 2
#endif

namespace us_spmm_detail {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) u32x2 lds_u2;
typedef __attribute__((address_space(3))) u32x4 lds_u4;

constexpr uint32_t kHiNib = 0xF0F0F0F0u;
constexpr int kWindow = US_SPMM_WINDOW;                // payload loads in flight per wavefront
constexpr int kNonTemporal = 2;                        // buffer cache policy: nt
constexpr int kBufferDword3 = 0x00020000;              // raw buffer, 32-bit data (gfx9 family)
constexpr int kLutBytes = 2048;                        // 256 selector pairs (static LDS)
constexpr int kMaxLds = 160 * 1024;

// Selector pair for one 8-bit union-mask segment m. Byte s of the output
// (dword 0: s = 0..3, dword 1: s = 4..7) holds segment position 2s (s < 4) or
// 2(s-4)+1 (s >= 4). An active position of rank r takes the r-th slot of
// the window, which v_perm_b32 reads from the 8 bytes it is given: with
// 4-bit values byte r of the window (slots 0..3 in the "low" source, 4..7
// in the "high" one); with 2-bit values the window w and w >> 4 hold slot r
// in the low nibble of byte r / 2 of w (r even) or of w >> 4 (r odd, the
// "high" source).
template <int BITS>
__device__ inline u32x2 perm_selectors(uint32_t m) {
    uint32_t sel[2] = {0u, 0u};
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        const int pos = s < 4 ? 2 * s : 2 * (s - 4) + 1;
        uint32_t b = 0x0Cu;                                   // v_perm: constant zero
        if ((m >> pos) & 1u) {
            const uint32_t r = __popc(m & ((1u << pos) - 1u));
            b = BITS == 4 ? r : (r & 1u) * 4u + (r >> 1);
        }
        sel[s >> 2] |= b << (8 * (s & 3));
    }
    return (u32x2){sel[0], sel[1]};
}

// LDS stage of one chunk of CH LTs (per wavefront), in bytes from the stage start:
//   payload : the chunk's compressed values, streamed from the 16-byte
//             boundary at or below the chunk's first byte (up to 15 bytes
//             early); a segment window may read 12 bytes past the last value,
//             so a chunk needs at most 8 BITS CH + 2 pieces of 16 bytes (an
//             LT holds at most 1024 values).
//             Linear staging (RING = false) keeps the whole chunk. RING =
//             true keeps a ring of four 1 KB slots (stream byte b in slot
//             (b / 1024) mod 4), so the stage does not grow with CH: an LT
//             spans at most 128 BITS + 16 bytes with its window overhang, so
//             the four slots hold every LT that is ready for decoding. The
//             160 bytes after the ring repeat its first 160 bytes, so windows
//             that start past the end of the ring (by at most one mask row's
//             slots plus a window) read on into it;
//   bitmaps : union-mask rows, 8 dwords per LT;
//             (this and the next three arrays have room for a whole number
//             of 4-LT passes; entries past the chunk are never decoded)
//   bases   : per LT and lane row rr = 2i + a, the slot address of the
//             first rank of mask row i in area row a (folded into the ring
//             with RING; 16 dwords per LT);
//   offsets : o_t of the chunk's LTs and the end offset (CH + 1 dwords);
//   (PERM: the bases area of LT j first holds its permutation word; after
//   the row-base step the bitmap area holds per LT pair and lane row the two
//   16-bit row bases, stage-relative byte addresses, LT 2m in the low and
//   LT 2m + 1 in the high half of the pair's dword, and the bases area the
//   union-mask row that lane row decodes)
//   X       : the chunk's activation slice, one row of 32 bytes per LT for
//             each activation column; rows are 16 bytes longer than the
//             slice so that the 16 rows read by one instruction fall in
//             different LDS banks.
template <int CH, bool RING, bool PERM, int BITS>
struct Chunk {
    static constexpr int kPayPieces = 8 * BITS * CH + 2;
    static constexpr int kLoads = (kPayPieces + 63) / 64;     // payload loads per lane
    static constexpr int kRing = 4096;                        // ring: four 1 KB slots
    static constexpr int kGuard = 160;                        // copy of the ring's first bytes
    static constexpr int kPasses = (CH + 3) / 4;              // base passes, 4 LTs each
    static constexpr int kLtPad = 4 * kPasses;                // per-LT arrays padded to whole passes
    static constexpr int kBmOffset = RING ? kRing + kGuard : 16 * kPayPieces;
    static constexpr int kBaseOffset = kBmOffset + 32 * kLtPad;
    static constexpr int kOffOffset = kBaseOffset + 64 * kLtPad;
    static constexpr int kXOffset = (kOffOffset + 4 * (kLtPad + 1) + 15) & ~15;
    static_assert(!PERM || (RING ? kRing + kGuard : 16 * kPayPieces) <= 65536,
                  "16-bit row bases address the payload stage");
    static constexpr int kXRowWords = 8 * CH + 4;
    static constexpr int kXPieces = 2 * CH;                   // 16-byte pieces of one activation row
    static_assert(2 * CH <= 64, "bitmap rows: one 16-byte load per half LT");
    static constexpr int bytes(int N) { return kXOffset + 4 * kXRowWords * N; }
};

struct SpmmArgs {
    const uint32_t *bm32;   // union bitmaps as dwords: LT t owns [8t, 8t + 8)
    const uint32_t *off;    // union value offsets, n_lt + 1
    const uint8_t *pay;     // compressed values
    int32_t pay_bytes;      // payload bytes rounded up to 16 (inside the pad)
    const uint8_t *x;       // activations, N rows of K/2 bytes
    int32_t *y;
    const float *scale;
    float *yf;
    const uint32_t *perm32; // row permutation words as dword pairs (PERM kernels)
    int32_t M, K, N, nkb;
    int32_t n_cu;           // compute units of the device (wavefront priorities)
};

// Resident wavefronts per SIMD an instantiation is built for: its launch
// bound, and the host's residency model. The figures sit at or above what
// the kernels need: single-chunk slices keep only one chunk's state (at most
// 64 VGPRs with four or more wavefronts per workgroup, 72 above 16
// activation columns, 80 with fewer wavefronts);
// multi-chunk slices also hold the next chunk's inputs, more of them for
// longer chunks and wider activation tiles (and, for reordered LTs, their
// permutation words), and ring staging, like every kernel above 16
// activation columns and the pipelined 16-column kernels of 11- and 16-LT
// chunks, holds the payload pieces in flight in registers.
constexpr int waves_per_simd(int wpg, int nmax, int ch, bool multi, bool ring, bool perm) {
    return nmax > 16   ? (multi ? 4 : wpg >= 4 ? 7 : 6)
           : !multi    ? (wpg >= 4 ? 8 : 6)
           : ring      ? (nmax <= 4 ? 5 : 4)
           : nmax <= 4 ? (perm && ch > 11 ? 6 : 7)
                       : (ch <= 4 ? 7 : ch <= 8 || (perm && ch <= 11) ? 5 : 4);
}

// The launch bound itself: waves_per_simd, except for the kernels above 16
// activation columns on rows in stored order, which are left to the
// compiler. Their natural use (at most 128 VGPRs, four wavefronts per
// SIMD) is what waves_per_simd assumes, and a bound makes their code slower.
constexpr int launch_waves(int wpg, int nmax, int ch, bool multi, bool ring, bool perm) {
    return nmax > 16 && !perm ? 1 : waves_per_simd(wpg, nmax, ch, multi, ring, perm);
}

__device__ __forceinline__ uint32_t lds_load(uint32_t addr) { return *(const lds_u32 *)(size_t)addr; }
// Two consecutive dwords at a 4-byte aligned address.
__device__ __forceinline__ uint2 lds_load2(uint32_t addr) { return make_uint2(lds_load(addr), lds_load(addr + 4)); }
__device__ __forceinline__ void lds_store(uint32_t addr, uint32_t v) { *(lds_u32 *)(size_t)addr = v; }
typedef __attribute__((address_space(3))) uint16_t lds_u16;
__device__ __forceinline__ void lds_store16(uint32_t addr, uint16_t v) { *(lds_u16 *)(size_t)addr = v; }
__device__ __forceinline__ void lds_store2(uint32_t addr, u32x2 v) { *(lds_u2 *)(size_t)addr = v; }
__device__ __forceinline__ void lds_store4(uint32_t addr, u32x4 v) { *(lds_u4 *)(size_t)addr = v; }

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

// 16 bytes per lane from a raw buffer (descriptor `desc`, byte offset voff +
// soff) straight into LDS: lane l writes LDS bytes [lds + 16 l, lds + 16 l +
// 16) (buffer_load_dwordx4 with the LDS bit; M0 holds the LDS base, and one
// wait state separates its write from the load). The load is counted by
// vmcnt like any other, and the callers order their LDS reads after it with
// their own vmcnt waits. It is issued from assembly because the compiler,
// unable to tell which later LDS reads it may alias, would otherwise wait
// for it before every one of them. M0 is listed as clobbered for the
// reader; the compiler reserves M0 and, in these kernels, generates no use
// of it (a host test checks that every M0 write in the built kernels is
// this one), so nothing of its own lives across the statement.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// The LDS base and the scalar offset must be wave-uniform; they are passed
// through readfirstlane so that they always reach the instruction in scalar
// registers (a no-op for values the compiler already keeps there).
__device__ __forceinline__ void dma16(u32x4 desc, uint32_t lds, uint32_t voff, uint32_t soff) {
    __asm__ volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen nt lds"
                     :
                     : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(desc),
                       "s"(__builtin_amdgcn_readfirstlane(soff))
                     : "memory", "m0");
}
#pragma clang diagnostic pop

// (q MAGIC) >> SHIFT equals q / P for every 0 <= q < qend.
constexpr bool row_by_multiply(int P, uint32_t magic, int shift, int qend) {
    for (int q = 0; q < qend; ++q)
        if ((((uint32_t)q * magic) >> shift) != (uint32_t)(q / P)) return false;
    return true;
}

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

// Rank slots. The payload stores the two areas of an area row interleaved by
// rank (area (a, c) at value o_t + 4 a P_t + 2 rho + c), so rank rho of an
// area row is one slot holding both of its values: a byte with 4-bit values
// (area column 0 in the low nibble), a nibble with 2-bit values (area column
// 0 in its low two bits). A slot address is an LDS byte address (4-bit) or
// twice an LDS byte address plus the nibble (2-bit).
//
// The eight slots from slot address s, as two dwords (slots 0..3, 4..7):
// 4-bit slots are the 8 bytes at s, aligned from the three dwords that hold
// them (an unaligned 8-byte LDS read gives the same bytes but takes far
// longer); 2-bit slots are the 32 bits at nibble s, taken from the two
// dwords that hold them, and returned with the same bits shifted down by
// one nibble (see perm_selectors).
template <int BITS>
__device__ __forceinline__ uint2 slot_window(uint32_t s) {
    if constexpr (BITS == 4) {
        const uint32_t a = s & ~3u;
        const uint2 d = lds_load2(a);
        const uint32_t d2 = lds_load(a + 8);
        return make_uint2(__builtin_amdgcn_alignbyte(d.y, d.x, s), __builtin_amdgcn_alignbyte(d2, d.y, s));
    } else {
        const uint2 d = lds_load2((s >> 1) & ~3u);
        const uint32_t w = __builtin_amdgcn_alignbit(d.y, d.x, s << 2);
        return make_uint2(w, w >> 4);
    }
}

// Eight slots -> the MFMA A operand of one segment: the selector pair picks
// the byte holding each position's slot (0x0C = zero), and each area
// column's value is moved to the high nibble (16 v) or the top two bits
// (64 v) of its byte.
template <int BITS>
__device__ __forceinline__ i32x4 place_slots(uint2 w, uint2 sel) {
    const uint32_t p0 = __builtin_amdgcn_perm(w.y, w.x, sel.x);
    const uint32_t p1 = __builtin_amdgcn_perm(w.y, w.x, sel.y);
    if constexpr (BITS == 4) {
        return (i32x4){(int32_t)((p0 << 4) & kHiNib), (int32_t)((p1 << 4) & kHiNib), (int32_t)(p0 & kHiNib),
                       (int32_t)(p1 & kHiNib)};
    } else {
        constexpr uint32_t kTop2 = 0xC0C0C0C0u;
        return (i32x4){(int32_t)((p0 << 6) & kTop2), (int32_t)((p1 << 6) & kTop2), (int32_t)((p0 << 4) & kTop2),
                       (int32_t)((p1 << 4) & kTop2)};
    }
}

// The selector pair of this lane's segment of mask row mrow; rot = (8 g - 3)
// mod 32 puts segment g at bits 3..10, the table's byte offset.
__device__ __forceinline__ uint2 selectors(const u32x2 *lut, uint32_t mrow, uint32_t rot) {
    const u32x2 sv = *(const u32x2 *)((const char *)lut + (__builtin_amdgcn_alignbit(mrow, mrow, rot) & 0x7F8u));
    return make_uint2(sv.x, sv.y);
}

// Decode one LT into the MFMA A operand of this lane.
//   mrow : union-mask row i of the LT
//   s    : slot address of the first rank of the lane's segment of row i
//          in area row a
template <int BITS>
__device__ __forceinline__ i32x4 decode_at(const u32x2 *lut, uint32_t mrow, uint32_t s, uint32_t rot) {
    return place_slots<BITS>(slot_window<BITS>(s), selectors(lut, mrow, rot));
}

// The same from the row's base slot: the segment starts one slot per active
// position of the row before it further on.
template <int BITS>
__device__ __forceinline__ i32x4 decode_tile(const u32x2 *lut, uint32_t mrow, uint32_t base, uint32_t lomask,
                                             uint32_t rot) {
    return decode_at<BITS>(lut, mrow, base + (uint32_t)__popc(mrow & lomask), rot);
}

// The same for a 4-bit row base given as a stage-relative byte address q and
// the stage's byte address st.
__device__ __forceinline__ i32x4 decode_tile_q(const u32x2 *lut, uint32_t mrow, uint32_t q, uint32_t st,
                                               uint32_t lomask, uint32_t rot) {
    return decode_at<4>(lut, mrow, st + (q + (uint32_t)__popc(mrow & lomask)), rot);
}

// Dwords g and g + 4 of an activation row's 8 dwords for one LT.
__device__ __forceinline__ uint2 x_pair(uint32_t addr) { return make_uint2(lds_load(addr), lds_load(addr + 16)); }

__device__ __forceinline__ i32x4 unpack_x(uint2 x) {
    return (i32x4){(int32_t)((x.x << 4) & kHiNib), (int32_t)(x.x & kHiNib),
                   (int32_t)((x.y << 4) & kHiNib), (int32_t)(x.y & kHiNib)};
}

// MULTI: some slices take several chunks (their inputs are then requested
// one chunk ahead); otherwise every slice is a single chunk. RING: the
// payload is staged in a 4 KB ring instead of whole (see Chunk). PERM: the
// LTs were row-reordered and p.perm32 holds their permutations. BITS: bits
// per payload value (4, or 2 for W2A4). NMAX: the widest activation matrix
// the instantiation stages (4, 16 or 32; NB = 2 column blocks above 16): the
// activation-staging registers are sized for it, so the N <= 4 kernels of
// the decode regime keep about 30 fewer VGPRs live. Every instantiation fits
// waves_per_simd() resident wavefronts per SIMD (at most 512 / that many
// VGPRs; held there by its launch bound, see launch_waves), which is also
// what the host's residency model assumes.
//
// The arguments are SpmmArgs field by field, in the order the kernel's first
// loads need them: the library is built with kernel-argument preloading
// (the dispatch places the leading argument dwords in scalar registers
// before the wavefront starts, which gfx950 supports for scalar arguments,
// not for a structure passed by value). The first loads then wait for no
// argument fetch; 14 dwords are preloaded, through `scale`.
template <int WPG, int NMAX, int CH, bool MULTI, bool RING, bool PERM, int BITS>
__global__ __launch_bounds__(64 * WPG, launch_waves(WPG, NMAX, CH, MULTI, RING, PERM)) void us_spmm_kernel(
    const uint32_t *off, const uint32_t *bm32, const uint8_t *x, int32_t nkb_, int32_t n_, int32_t k_,
    int32_t pay_bytes, const uint8_t *pay, const float *scale, int32_t n_cu, int stage_bytes, int32_t *y, float *yf,
    const uint32_t *perm32, int32_t m_) {
    SpmmArgs p;
    p.off = off;
    p.bm32 = bm32;
    p.x = x;
    p.nkb = nkb_;
    p.N = n_;
    p.K = k_;
    p.pay_bytes = pay_bytes;
    p.pay = pay;
    p.scale = scale;
    p.n_cu = n_cu;
    p.y = y;
    p.yf = yf;
    p.perm32 = perm32;
    p.M = m_;
    constexpr int NB = NMAX > 16 ? 2 : 1;                 // MFMA column blocks
    using C = Chunk<CH, RING, PERM, BITS>;
    // Pipelined chunks: slices of several chunks in linear staging request
    // the first pieces of their next chunk while the current chunk's last
    // pieces are decoded, so that a slice's payload streams without a round
    // trip at every chunk boundary. Their payload passes through registers
    // (the next chunk's early pieces wait there until its stage is free), and
    // their loads are all visible to the compiler, whose own waits then order
    // every use exactly. This holds above 16 activation columns, and at 16
    // for chunks of 11 or 16 LTs, whose stage already leaves one workgroup
    // per CU; not for reordered chunks longer than 4 LTs, whose registers
    // would not fit the early pieces.
    constexpr bool kPipe = MULTI && !RING && (NMAX > 16 || (NMAX == 16 && CH >= 11)) && !(PERM && CH > 4);
    static_assert(!kPipe || C::kLoads >= kWindow, "a pipelined chunk takes at least one window of pieces");
    static_assert(BITS == 4 || BITS == 2, "payload values are 4 or 2 bits");
    static_assert(!PERM || BITS == 4, "16-bit row bases hold stage-relative byte slots (4-bit values)");
    constexpr int kValShift = BITS == 4 ? 1 : 2;          // log2(values per byte)
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    __shared__ u32x2 lut[256];                               // selector table
    const uint32_t lds0 = (uint32_t)(size_t)(lds_u32 *)lds;  // LDS address of the dynamic block

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int mb = blockIdx.x;
    const int N = p.N;

    // This wavefront's K slice: LTs t0 .. t0 + nlt - 1 of row block mb
    // (nlt >= 1 because WPG <= K / 64). When the LTs do not divide evenly,
    // the first K/64 mod WPG wavefronts take one more; the last ones, which
    // the SIMDs serve last, are the short slices. (Unsigned arithmetic: the
    // scalar instructions before the first loads are few, as every
    // wavefront of a CU issues them at once.)
    const int nkb = p.nkb;
    const uint32_t unkb = (uint32_t)nkb;
    const int kb0 = (int)((uint32_t)wave * (unkb / WPG) + min((uint32_t)wave, unkb % WPG));
    const int nlt = (int)(unkb / WPG + ((uint32_t)wave < unkb % WPG ? 1u : 0u));
    const uint64_t t0 = (uint64_t)(uint32_t)mb * unkb + (uint32_t)kb0;
    [[maybe_unused]] const uint32_t *const off_s = p.off + t0;   // the slice's offsets and bitmaps
    [[maybe_unused]] const uint32_t *const bm_s = p.bm32 + 8 * t0;

    // Lane roles in the decode.
    const int rr = lane & 15;
    const int i = rr >> 1;                                 // union-mask row
    const int g = lane >> 4;                               // segment / MFMA k-group
    const uint32_t amask = (rr & 1) ? ~0u : 0u;            // area row partition a = 1
    const uint32_t lomask = (1u << (8 * g)) - 1u;          // mask bits before the segment
    const uint32_t rot = (uint32_t)(8 * g + 29) & 31u;

    const uint32_t st = lds0 + (uint32_t)(wave * stage_bytes);   // stage, LDS bytes
    const uint32_t st_bm = st + C::kBmOffset, st_base = st + C::kBaseOffset;
    const uint32_t st_off = st + C::kOffOffset;
    const uint32_t st_x = st + C::kXOffset;

    // Activation reads in the decode: lane (column rr, k-group g) reads dwords
    // g and g + 4 of its row's 8 dwords for the LT. Columns >= N only feed
    // outputs that are never stored: clamp them to a staged row.
    uint32_t xq[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) xq[nb] = st_x + 4u * (uint32_t)(min(nb * 16 + rr, N - 1) * C::kXRowWords + g);

    // Activation loads: whole rows of K/2 bytes; rows >= N read zero.
    const int xrow_bytes = (int)((uint32_t)p.K >> 1);
    const __amdgpu_buffer_rsrc_t xsrc =
        __builtin_amdgcn_make_buffer_rsrc((void *)p.x, (short)0, N * xrow_bytes, kBufferDword3);
    // Activation staging: the chunk's N x 2 CH pieces of 16 bytes, piece
    // q = lane + 64 u in load u. Only the loads that carry pieces are issued (all of them in pipelined slices, whose
    // wait counts must not depend on N: the others read zero, with no
    // memory traffic): the texture path, not HBM, limits how fast a CU takes
    // them in at the start of the kernel.
    constexpr int kXLoads = (NMAX * C::kXPieces + 63) / 64;
    const int x_loads = (int)(((uint32_t)N * C::kXPieces + 63u) >> 6);        // wave-uniform
    // Piece q is row n = q / (2 CH), piece q - 2 CH n of it; rows >= N read
    // zero. With 2 CH a power of two that is a shift. Otherwise (11-LT
    // chunks) n comes from a multiply and a shift (exact for every q the
    // loads reach), and the piece's offsets follow from n and q without a
    // division: in the slice n K/2 + 16 (q - 2 CH n) bytes, in LDS st_x +
    // 16 (q + n), as a staged row holds 16 bytes more than its 2 CH pieces.
    // This address arithmetic runs before the loads can be issued, on every
    // wavefront of the CU at once.
    constexpr bool kXPow2 = (C::kXPieces & (C::kXPieces - 1)) == 0;
    constexpr int kXShift = 20;
    constexpr uint32_t kXMagic = ((1u << kXShift) + C::kXPieces - 1) / C::kXPieces;
    static_assert(row_by_multiply(C::kXPieces, kXMagic, kXShift, 64 * kXLoads), "inexact activation row");
    auto x_piece = [&](int u) { return (uint32_t)(lane + 64 * u); };
    auto x_row = [&](int u) { return (x_piece(u) * kXMagic) >> kXShift; };
    const int x_step = xrow_bytes - 16 * C::kXPieces;      // |x_step| < 2^23
    // Global byte offsets, and LDS addresses (0: a row >= N) where kept: in
    // every multi-chunk slice and with a power-of-two row; single-chunk
    // slices of 11-LT chunks compute them when the pieces are stored.
    uint32_t xv[kXLoads];
    [[maybe_unused]] uint32_t xs[kXLoads];
#pragma unroll
    for (int u = 0; u < kXLoads; ++u) {
        if constexpr (kXPow2) {
            const int q = lane + 64 * u, n = q / C::kXPieces, pj = q % C::kXPieces;
            xv[u] = (uint32_t)(n * xrow_bytes + 16 * pj);
            xs[u] = n < N ? st_x + 4u * (uint32_t)(n * C::kXRowWords) + 16u * (uint32_t)pj : 0u;
        } else {
            xv[u] = 16u * x_piece(u) + (uint32_t)__mul24((int)x_row(u), x_step);
        }
    }

    i32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (i32x4){0, 0, 0, 0};

    // A chunk's offsets, bitmaps, permutations and activations; they are
    // requested together (none depends on another). Addresses are clamped
    // into the matrix.
    uint32_t offv;
    u32x4 pbm;
    [[maybe_unused]] u32x2 pperm;                        // (PERM) lane j: word of the chunk's LT j
    i32x4 px[kXLoads];
    auto request = [&](int c0) {
        const int cnt = min(CH, nlt - c0);                 // >= 1
        if constexpr (!PERM) {
            offv = off_s[(uint32_t)(c0 + min(lane, cnt))];
            pbm = *(const u32x4 *)(bm_s + (uint32_t)(8 * c0 + 4 * min(lane, 2 * cnt - 1)));
        } else {
            // (64-bit lane addresses: scalar bases would leave the reordered
            // multi-chunk kernels above 16 columns short of registers)
            offv = p.off[t0 + c0 + min(lane, cnt)];
            pbm = *(const u32x4 *)(p.bm32 + 8 * (t0 + c0) + 4 * min(lane, 2 * cnt - 1));
            pperm = *(const u32x2 *)(p.perm32 + 2 * (t0 + c0 + min(lane, cnt - 1)));
        }
        const uint32_t xk = (uint32_t)(32 * (kb0 + c0));
#pragma unroll
        for (int u = 0; u < kXLoads; ++u)
            if (kPipe || u < x_loads) px[u] = __builtin_amdgcn_raw_buffer_load_b128(xsrc, xv[u] + xk, 0, 0);
    };

    request(0);
    if constexpr (MULTI && !kXPow2) {
#pragma unroll
        for (int u = 0; u < kXLoads; ++u) {
            const uint32_t n = x_row(u);
            xs[u] = n < (uint32_t)N ? st_x + 16u * (x_piece(u) + n) : 0u;
        }
    }
    // The dequant scale of the output row this thread stores in the epilogue
    // (outputs e = threadIdx.x + 64 WPG k all have row e mod 16), requested
    // now so that the epilogue does not wait for it.
    float row_scale = 0.0f;
    if (p.scale && (int)threadIdx.x < 16 * N) row_scale = p.scale[(int64_t)mb * 16 + (threadIdx.x & 15)];
    // Selector table, computed while the first requests fly.
    for (int e = threadIdx.x; e < 256; e += 64 * WPG) lut[e] = perm_selectors<BITS>((uint32_t)e);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);                     // nothing that waits on the inputs moves above

    // Chunk state shared by the staging and the decoding half.
    int cnt = 0;
    uint32_t A0 = 0;
    __amdgpu_buffer_rsrc_t psrc;                          // payload, through registers
    u32x4 pdesc;                                          // the same range as a plain descriptor
    i32x4 pf[C::kLoads];
    // Payload piece u (16 bytes per lane from the chunk's first staged byte
    // on, stage bytes [1024 u, 1024 u + 1024)). Ring staging goes through
    // registers, as its slots are refilled. Whole staging up to 16
    // activation columns loads straight into the stage, which keeps the
    // pieces out of the registers (measured slower above 16 columns); its
    // last load writes only the pieces the payload area holds.
    auto load_piece = [&](int u) {
        pf[u] = __builtin_amdgcn_raw_buffer_load_b128(psrc, (uint32_t)(16 * lane + 1024 * u), 0, kNonTemporal);
    };
    [[maybe_unused]] uint32_t A0n = 0;                     // (kPipe) the next chunk's first staged byte
    [[maybe_unused]] __amdgpu_buffer_rsrc_t psrcn;         // (kPipe) and its payload range
    constexpr bool kDirect = !RING && NMAX <= 16 && !kPipe;  // payload straight into LDS
    auto dma_piece = [&](auto uc) {
        constexpr int u = decltype(uc)::value;
        if (u + 1 < C::kLoads || C::kPayPieces % 64 == 0 || lane + 64 * u < C::kPayPieces)
            dma16(pdesc, st + 1024u * u, (uint32_t)(16 * lane), 1024u * u);
    };

    // Bitmaps (zero past the chunk), offsets and activations into the stage.
    auto commit_inputs = [&]() {
        if (lane < 2 * CH) lds_store4(st_bm + 16 * lane, lane < 2 * cnt ? pbm : (u32x4){0u, 0u, 0u, 0u});
        if (lane <= CH) lds_store(st_off + 4 * lane, offv);
        if constexpr (PERM) {
            // The lane row of original row r is 2 (r mod 8) + r / 8,
            // r's 4 bits rotated left by one: done here for every
            // nibble at once.
            auto lane_rows = [](uint32_t w) { return ((w << 1) & 0xEEEEEEEEu) | ((w >> 3) & 0x11111111u); };
            if (lane < CH) lds_store2(st_base + 64 * lane, (u32x2){lane_rows(pperm.x), lane_rows(pperm.y)});
        }
        // Loads past x_loads were not issued. The reordered and 2-bit
        // single-chunk kernels for up to 16 columns branch past their
        // stores on that wave-uniform count (4-5 % faster on 4096x11008 at
        // N = 8, 2 % on 12288x4096); the plain 4-bit, the multi-chunk and
        // the 4-column kernels measured 1-2 % slower with the branch and
        // mask the stores lane by lane instead.
        constexpr bool kXBranch = (PERM || BITS == 2) && !MULTI && NMAX == 16;
#pragma unroll
        for (int u = 0; u < kXLoads; ++u) {
            if (kXBranch && u >= x_loads) break;
            if constexpr (MULTI || kXPow2) {
                if ((kXBranch || u < x_loads) && xs[u] != 0u) lds_store4(xs[u], (u32x4)px[u]);
            } else {
                const uint32_t n = x_row(u);
                if ((kXBranch || u < x_loads) && n < (uint32_t)N) lds_store4(st_x + 16u * (x_piece(u) + n), (u32x4)px[u]);
            }
        }
    };
    // (kPipe) Stage a chunk of a pipelined slice; NX: another chunk follows.
    // The first chunk requests its first pieces here; a later chunk's were
    // requested during the previous chunk's decode. Either way the next
    // chunk's inputs are requested after this chunk's first pieces.
    auto stage_pipe = [&](int c0, auto nx, auto first) {
        cnt = min(CH, nlt - c0);
        if constexpr (decltype(first)::value) {
            wait_vm_all();                                 // offsets, bitmaps, activations
            const uint32_t ob = lane_value(offv, 0), oe = lane_value(offv, cnt);
            A0 = us_range::first_byte<BITS>(ob, (uint32_t)p.pay_bytes);
            const uint32_t prange =
                us_range::range_bytes<BITS>(oe, A0, (uint32_t)p.pay_bytes, (uint32_t)C::kPayPieces);
            psrc = __builtin_amdgcn_make_buffer_rsrc((void *)(p.pay + A0), (short)0, (int)prange, kBufferDword3);
            static_for<0, kWindow>([&](auto uc) { load_piece(decltype(uc)::value); });
        } else {
            A0 = A0n;
            psrc = psrcn;
        }
        commit_inputs();
        if constexpr (decltype(nx)::value) request(c0 + CH);
    };
    auto stage_chunk = [&](int c0) {
        cnt = min(CH, nlt - c0);
        wait_vm_all();                                     // offsets, bitmaps, activations

        const uint32_t ob = lane_value(offv, 0), oe = lane_value(offv, cnt);
        // Payload: 16-byte pieces from A0, the first staged byte; load u
        // brings stage bytes [1024 u, 1024 u + 1024). Pieces past the chunk
        // read zero (range check) and cost no memory traffic. The range
        // saturates, so offsets that are not a valid encoding never move the
        // descriptor outside the payload. kWindow loads are in flight per
        // wavefront, so early pieces are not queued behind the whole
        // machine's requests and decoding starts while the rest streams.
        // Non-temporal: the stream does not displace the activations, which
        // every workgroup re-reads, from L2.
        A0 = us_range::first_byte<BITS>(ob, (uint32_t)p.pay_bytes);
        const uint32_t prange = us_range::range_bytes<BITS>(oe, A0, (uint32_t)p.pay_bytes, (uint32_t)C::kPayPieces);
        if constexpr (!kDirect) {
            psrc = __builtin_amdgcn_make_buffer_rsrc((void *)(p.pay + A0), (short)0, (int)prange, kBufferDword3);
        } else {
            const uint64_t pa = (uint64_t)(size_t)(p.pay + A0);
            pdesc = (u32x4){(uint32_t)pa, (uint32_t)(pa >> 32) & 0xFFFFu, prange, (uint32_t)kBufferDword3};
        }
        auto issue_window = [&]() {
            static_for<0, kWindow>([&](auto uc) {
                if constexpr (decltype(uc)::value < C::kLoads) {
                    if constexpr (!kDirect) load_piece(decltype(uc)::value);
                    else dma_piece(uc);
                }
            });
        };
        if (MULTI && nlt - c0 > CH) {
            // A later chunk follows: once this chunk's inputs are in LDS their
            // registers take the next chunk's inputs, requested ahead of this
            // chunk's payload so that the payload waits below cover them.
            commit_inputs();
            request(c0 + CH);
            issue_window();
        } else {
            issue_window();
            commit_inputs();
        }
    };

    // NX: (kPipe) another chunk of the slice follows this one.
    auto decode_chunk = [&](int c0, auto nx) {
        constexpr bool NX = decltype(nx)::value;

        // Row bases: lanes 16 jj + rr handle LT j = 4 pass + jj, mask row i,
        // area row a. The scan over the 16 lanes of a DPP row adds the
        // popcounts of the rows before i. With PERM the row base and the
        // mask row of (i, a), i.e. of reordered row 8a + i, go to the lane
        // row of original row r = pi[8a + i]: 2 (r mod 8) + r / 8; the row
        // base (as a 16-bit slot address relative to the stage) into the LT
        // pair's bitmap area, the mask row into the LT's bases area. Every
        // bitmap and permutation word of the chunk is read before the first
        // of them is overwritten.
        // Area row a's slots start P_t slots (2 P_t values) after area row
        // 0's, and rank rho is slot rho of its area row: the scan injects P_t
        // on area-row a = 1 lanes. Slot rho of LT t's area row 0 is slot
        // o_t / 2 of the matrix; the chunk's stage starts at its byte A0
        // (slot A0 * kSlotsPerByte), at stage slot address kSlotsPerByte st,
        // taken mod the ring's slots with the ring.
        constexpr uint32_t kSlotsPerByte = 4 / BITS;
        const uint32_t smask = RING ? (uint32_t)C::kRing * kSlotsPerByte - 1u : ~0u;
        {
            const uint32_t jj = (uint32_t)lane >> 4;
            const uint32_t p_bm = st_bm + 32 * jj + 4 * i, p_off = st_off + 4 * jj;
            const uint32_t q_base = st_base + 64 * jj, p_base = q_base + 4 * rr;
            const uint32_t q_b16 = st_bm + 64 * (jj >> 1) + 2 * (jj & 1), p_b16 = q_b16 + 4 * rr;
            const uint32_t p_pm = q_base + 4 * (rr & 1);
            uint32_t mrow[C::kPasses];
            uint2 o[C::kPasses];
            [[maybe_unused]] uint32_t pm[C::kPasses];
#pragma unroll
            for (int ps = 0; ps < C::kPasses; ++ps) {
                mrow[ps] = lds_load(p_bm + 128 * ps);
                o[ps] = lds_load2(p_off + 16 * ps);
                if constexpr (PERM) pm[ps] = lds_load(p_pm + 256 * ps);   // lane rows of pi[8a .. 8a + 7], LT 4 ps + jj
            }
#pragma unroll
            for (int ps = 0; ps < C::kPasses; ++ps) {
                const uint32_t inj = amask & ((o[ps].y - o[ps].x) >> 2);    // P_t
                uint32_t ex = (uint32_t)__builtin_amdgcn_update_dpp((int)inj, (int)__popc(mrow[ps]), 0x112, 0xF,
                                                                    0xF, false);
                ex += dpp_row<0x112>(ex);
                ex += dpp_row<0x114>(ex);
                ex += dpp_row<0x118>(ex);
                const uint32_t rel = ((o[ps].x >> 1) + ex - kSlotsPerByte * A0) & smask;   // stage slot
                if constexpr (PERM) {
                    // The base is first written under this lane's own lane
                    // row, so that a word that is not a permutation still
                    // leaves every lane row with a base inside the stage.
                    // (16 bits hold rel: a byte address below the payload
                    // area's 64 KB.)
                    const uint32_t lr = (pm[ps] >> (4 * i)) & 15u;
                    const uint16_t b16 = (uint16_t)rel;
                    lds_store16(p_b16 + 128 * ps, b16);
                    lds_store(q_base + 4 * lr + 256 * ps, mrow[ps]);
                    lds_store16(q_b16 + 4 * lr + 128 * ps, b16);
                } else {
                    lds_store(p_base + 256 * ps, kSlotsPerByte * st + rel);
                }
            }
        }
        // LT k can be decoded once the pieces holding its windows have landed:
        // a window reads up to 12 (4-bit) or 8 (2-bit) bytes from a slot at
        // most one past the LT's last, so BITS o_{k+1} - 8 A0 + 96 (64) <=
        // 8192 (u + 1) stream bits, i.e. after load u = need_k.
        constexpr uint32_t kOverhangBits = BITS == 4 ? 95u : 63u;
        const uint32_t need =
            ((uint32_t)BITS * lds_load(st_off + 4 * min(lane + 1, CH)) - 8u * A0 + kOverhangBits) >> 13;

        // LDS addresses of the next LT's mask row, row base and activations
        // for this lane; they advance as LTs are decoded. PERM reads the mask
        // row routed to this lane row from the bases area and the 16-bit row
        // bases of an LT pair from one dword of the bitmap area (pairs start
        // at even LTs; a lone LT is the chunk's last, at an even position, in
        // the low half).
        uint32_t a_bm = st_bm + (PERM ? 4 * rr : 4 * i), a_base = st_base + 4 * rr;
        auto row_at = [&](int k) { return PERM ? a_base + 64 * k : a_bm + 32 * k; };
        uint32_t a_x[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) a_x[nb] = xq[nb];
        auto decode_one = [&]() {
            const uint32_t mrow = lds_load(row_at(0));
            i32x4 A;
            if constexpr (PERM) A = decode_tile_q(lut, mrow, lds_load(a_bm) & 0xFFFFu, st, lomask, rot);
            else A = decode_tile<BITS>(lut, mrow, lds_load(a_base), lomask, rot);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, unpack_x(x_pair(a_x[nb])), acc[nb], 0, 0, 0);
                a_x[nb] += 32;
            }
            a_bm += 32;
            a_base += 64;
        };
        auto decode_two = [&]() {
            const uint32_t m0 = lds_load(row_at(0)), m1 = lds_load(row_at(1));
            i32x4 A0v, A1v;
            if constexpr (PERM) {
                const uint32_t w = lds_load(a_bm);
                A0v = decode_tile_q(lut, m0, w & 0xFFFFu, st, lomask, rot);
                A1v = decode_tile_q(lut, m1, w >> 16, st, lomask, rot);
            } else {
                A0v = decode_tile<BITS>(lut, m0, lds_load(a_base), lomask, rot);
                A1v = decode_tile<BITS>(lut, m1, lds_load(a_base + 64), lomask, rot);
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A0v, unpack_x(x_pair(a_x[nb])), acc[nb], 0, 0, 0);
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A1v, unpack_x(x_pair(a_x[nb] + 32)), acc[nb], 0, 0, 0);
                a_x[nb] += 64;
            }
            a_bm += 64;
            a_base += 128;
        };

        // The payload lands in issue order: after load u, stream bytes
        // [0, 1024 (u + 1)) have arrived (and, with the ring, bytes from
        // 1024 (u - 3) on are still held), so LTs with need <= u can be
        // decoded. LTs go in pairs; one that waits for its partner waits one
        // step at most (the partner spans at most 528 more bytes). With the
        // ring the chunk's last LT goes alone as soon as it is ready, as
        // later steps may refill its slots.
        //
        // (kPipe, NX) Once all of this chunk's pieces are requested, each
        // step requests one of the next chunk's first kWindow pieces instead,
        // into the registers of pieces already staged; the next chunk's
        // payload range comes from its offsets, requested with this chunk's
        // inputs.
        int j = 0;
        if constexpr (kPipe && NX) {
            const int cn = min(CH, nlt - c0 - CH);
            const uint32_t obn = lane_value(offv, 0), oen = lane_value(offv, cn);
            A0n = us_range::first_byte<BITS>(obn, (uint32_t)p.pay_bytes);
            const uint32_t prn = us_range::range_bytes<BITS>(oen, A0n, (uint32_t)p.pay_bytes, (uint32_t)C::kPayPieces);
            psrcn = __builtin_amdgcn_make_buffer_rsrc((void *)(p.pay + A0n), (short)0, (int)prn, kBufferDword3);
        }
        static_for<0, C::kLoads>([&](auto uc) {
            constexpr int u = decltype(uc)::value;
            [[maybe_unused]] constexpr int later = (kWindow - 1 < C::kLoads - 1 - u) ? kWindow - 1 : C::kLoads - 1 - u;
            if constexpr (kPipe) {
                // Piece u into the stage, then the next request (which may
                // reuse piece u's registers).
                if (u + 1 < C::kLoads || lane + 64 * u < C::kPayPieces)
                    lds_store4(st + 1024 * u + 16 * lane, (u32x4)pf[u]);
                if constexpr (u + kWindow < C::kLoads) {
                    load_piece(u + kWindow);
                } else if constexpr (NX) {
                    constexpr int v = u + kWindow - C::kLoads;   // the next chunk's piece v
                    pf[v] = __builtin_amdgcn_raw_buffer_load_b128(psrcn, (uint32_t)(16 * lane + 1024 * v), 0,
                                                                  kNonTemporal);
                }
            } else if constexpr (kDirect) {
                wait_vm<later>();                          // piece u has landed
                if constexpr (u + kWindow < C::kLoads) dma_piece(std::integral_constant<int, u + kWindow>());
            } else {
                wait_vm<later>();
                if constexpr (u + kWindow < C::kLoads) load_piece(u + kWindow);
                if constexpr (RING) {
                    lds_store4(st + 1024 * (u & 3) + 16 * lane, (u32x4)pf[u]);
                    if ((u & 3) == 0 && lane < C::kGuard / 16) lds_store4(st + C::kRing + 16 * lane, (u32x4)pf[u]);
                } else if (u + 1 < C::kLoads || lane + 64 * u < C::kPayPieces) {
                    lds_store4(st + 1024 * u + 16 * lane, (u32x4)pf[u]);
                }
            }
            __asm__ volatile("" ::: "memory");
            if constexpr (!MULTI) {
                if (2 * j >= cnt) __builtin_amdgcn_s_setprio(0);   // second half: back to age order
            }
            if constexpr (u + 1 < C::kLoads) {
                const int ready = __builtin_popcountll(__builtin_amdgcn_ballot_w64(lane < cnt && need <= (uint32_t)u));
                for (; j + 1 < ready; j += 2) decode_two();
                if (RING && j < ready && ready == cnt) {
                    decode_one();
                    ++j;
                }
            } else {
                for (; j + 1 < cnt; j += 2) decode_two();
                if (j < cnt) decode_one();
            }
        });
        __asm__ volatile("" ::: "memory");
    };
    // The first chunk is straight-line code after the prologue, so every
    // wait above counts loads exactly; later chunks only occur for long slices.
    // Every slice holds at least one LT (the host never splits K into more
    // slices than LTs), so the first chunk needs no branch.
    // Multi-chunk slices lower their issue priority as they progress: 3 for
    // the first quarter of the slice, one step less per quarter after it.
    // A SIMD's arbiter otherwise favours its oldest wavefronts, and with equal
    // work per slice the youngest workgroups of a CU then finish well after
    // the oldest, with few wavefronts left to hide latency at the end.
    //
    // Single-chunk slices instead start at a priority that grows with their
    // expected age rank on the CU: the workgroup's dispatch round (blockIdx /
    // CUs) plus the wavefront's place among the workgroup's wavefronts on its
    // SIMD (wave / 4), at most 3. Every wavefront returns to 0 once half of
    // its slice is decoded. The youngest wavefronts, which the arbiter
    // would serve last, get ahead early and the oldest catch up later, so
    // that fewer wavefronts are left running alone at the end.
    if constexpr (MULTI) {
        __builtin_amdgcn_s_setprio(3);
    } else {
        const int rank = min(3, (int)blockIdx.x / max(p.n_cu, 1) + (wave >> 2));   // wave-uniform
        if (rank == 1) __builtin_amdgcn_s_setprio(1);
        else if (rank == 2) __builtin_amdgcn_s_setprio(2);
        else if (rank >= 3) __builtin_amdgcn_s_setprio(3);
    }
    auto chunk_prio = [&](int c0) {
        const int quarter = 4 * c0 / nlt;                  // wave-uniform
        if (quarter == 1) __builtin_amdgcn_s_setprio(2);
        else if (quarter == 2) __builtin_amdgcn_s_setprio(1);
        else if (quarter >= 3) __builtin_amdgcn_s_setprio(0);
    };
    using Yes = std::integral_constant<bool, true>;
    using No = std::integral_constant<bool, false>;
    if constexpr (kPipe) {
        // Whether another chunk follows is known to every chunk's code, so
        // that the requests, and the waits the compiler puts before their
        // uses, form one straight sequence per chunk.
        if (nlt > CH) {
            stage_pipe(0, Yes(), Yes());
            decode_chunk(0, Yes());
            int c0 = CH;
            for (; nlt - c0 > CH; c0 += CH) {
                chunk_prio(c0);
                stage_pipe(c0, Yes(), No());
                decode_chunk(c0, Yes());
            }
            chunk_prio(c0);
            stage_pipe(c0, No(), No());
            decode_chunk(c0, No());
        } else {
            stage_pipe(0, No(), Yes());
            decode_chunk(0, No());
        }
    } else {
        stage_chunk(0);
        decode_chunk(0, No());
        if constexpr (MULTI) {
            for (int c0 = CH; c0 < nlt; c0 += CH) {
                chunk_prio(c0);
                stage_chunk(c0);
                decode_chunk(c0, No());
            }
        }
    }

    // Split-K combine: each wavefront leaves its 16 x (16 NB) partial in its
    // own stage, in MFMA result layout (lane l, element v: row 4 (l / 16) + v,
    // column l % 16); after the barrier the first 16 N threads sum the WPG
    // partials of one output each.
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) lds_store4(st + 16 * (64 * nb + lane), (u32x4)acc[nb]);
    __syncthreads();

    for (int e = threadIdx.x; e < 16 * N; e += 64 * WPG) {
        const int r = e & 15, n = e >> 4;
        const int R = 2 * (r & 7) + (r >> 3);                 // W row 8a + i is MFMA row 2i + a
        const uint32_t idx = 4u * (uint32_t)(4 * (64 * (n >> 4) + 16 * (R >> 2) + (n & 15)) + (R & 3));
        int32_t s = 0;
#pragma unroll
        for (int w = 0; w < WPG; ++w) s += (int32_t)lds_load(lds0 + (uint32_t)(w * stage_bytes) + idx);
        const int32_t yv = s >> (BITS == 4 ? 8 : 10);         // exact: s = 256 Y (1024 Y)
        const int64_t m = (int64_t)mb * 16 + r;
        const int64_t M = p.M;
        p.y[n * M + m] = yv;
        if (p.scale) p.yf[n * M + m] = (float)yv * row_scale;
    }
}

// Chunk configurations: chunk length and payload staging (see Chunk).
// Two MFMA column blocks (N > 16) use the short linear ones only.
struct ChunkCfg {
    int ch;
    bool ring;
};
constexpr ChunkCfg kCfgs[] = {{4, false}, {8, false}, {11, false}, {16, false}, {16, true}, {11, true}};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

inline bool cfg_allowed(int idx, int N) { return N <= 16 || (kCfgs[idx].ch <= 8 && !kCfgs[idx].ring); }

template <int CH, bool RING, bool PERM, int BITS>
int stage_bytes(int N) { return (Chunk<CH, RING, PERM, BITS>::bytes(N) + 15) & ~15; }

template <bool PERM, int BITS>
int lds_bytes_t(int idx, int N, int wpg) {
    int st = 0;
    switch (idx) {
        case 0: st = stage_bytes<4, false, PERM, BITS>(N); break;
        case 1: st = stage_bytes<8, false, PERM, BITS>(N); break;
        case 2: st = stage_bytes<11, false, PERM, BITS>(N); break;
        case 3: st = stage_bytes<16, false, PERM, BITS>(N); break;
        case 4: st = stage_bytes<16, true, PERM, BITS>(N); break;
        default: st = stage_bytes<11, true, PERM, BITS>(N); break;
    }
    return kLutBytes + wpg * st;
}

inline int lds_bytes(int idx, int N, int wpg, bool perm, int bits) {
    if (bits == 2) return perm ? lds_bytes_t<true, 2>(idx, N, wpg) : lds_bytes_t<false, 2>(idx, N, wpg);
    return perm ? lds_bytes_t<true, 4>(idx, N, wpg) : lds_bytes_t<false, 4>(idx, N, wpg);
}

template <int WPG, int NMAX, int CH, bool RING, bool PERM, int BITS>
hipError_t launch_spmm(const SpmmArgs &a, hipStream_t s) {
    const bool multi = (a.nkb + WPG - 1) / WPG > CH;
    auto kern = multi ? us_spmm_kernel<WPG, NMAX, CH, true, RING, PERM, BITS>
                      : us_spmm_kernel<WPG, NMAX, CH, false, RING, PERM, BITS>;
    // Allow more than 64 KB of dynamic LDS: once per instantiation and device
    // (concurrent first calls may both set it, which is harmless).
    static std::atomic<unsigned long long> attr_set{0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    const unsigned long long bit = 1ull << (dev & 63);
    if (!(attr_set.load(std::memory_order_acquire) & bit)) {
        for (const void *f : {(const void *)us_spmm_kernel<WPG, NMAX, CH, true, RING, PERM, BITS>,
                              (const void *)us_spmm_kernel<WPG, NMAX, CH, false, RING, PERM, BITS>}) {
            const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds - kLutBytes);
            if (e != hipSuccess) return e;
        }
        attr_set.fetch_or(bit, std::memory_order_release);
    }
    const int st = stage_bytes<CH, RING, PERM, BITS>(a.N);
    hipLaunchKernelGGL(kern, dim3(a.M / 16), dim3(64 * WPG), WPG * st, s, a.off, a.bm32, a.x, a.nkb, a.N, a.K,
                       a.pay_bytes, a.pay, a.scale, a.n_cu, st, a.y, a.yf, a.perm32, a.M);
    return hipGetLastError();
}

template <int NMAX, int CH, bool RING, bool PERM, int BITS>
hipError_t launch_spmm_wpg(int wpg, const SpmmArgs &a, hipStream_t s) {
    switch (wpg) {
        case 1: return launch_spmm<1, NMAX, CH, RING, PERM, BITS>(a, s);
        case 2: return launch_spmm<2, NMAX, CH, RING, PERM, BITS>(a, s);
        case 4: return launch_spmm<4, NMAX, CH, RING, PERM, BITS>(a, s);
        case 8: return launch_spmm<8, NMAX, CH, RING, PERM, BITS>(a, s);
        default: return launch_spmm<16, NMAX, CH, RING, PERM, BITS>(a, s);
    }
}

// Launch configuration idx of kCfgs with wpg wavefronts per workgroup, for
// N <= 16 (NMAX = 4 or 16) or N <= 32.
// The instantiations above 16 activation columns (NMAX = 32) of every weight
// form live in translation units of their own: us_spmm_wide.hip (4-LT
// chunks) and us_spmm_wide8.hip (8-LT chunks), the latter built with the
// compiler's default scheduling strategy, as the one the other units use
// leaves some of its kernels above the registers of four wavefronts per SIMD.
template <bool PERM, int BITS>
hipError_t launch_cfg_wide(int wpg, int idx, const SpmmArgs &a, hipStream_t s);
template <bool PERM, int BITS>
hipError_t launch_cfg_wide8(int wpg, const SpmmArgs &a, hipStream_t s);

template <bool PERM, int BITS, int NMAX = 16>
hipError_t launch_cfg(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    if constexpr (NMAX > 4) {
        if (a.N > 16) return launch_cfg_wide<PERM, BITS>(wpg, idx, a, s);
    }
    switch (idx) {
        case 5: return launch_spmm_wpg<NMAX, 11, true, PERM, BITS>(wpg, a, s);
        case 4: return launch_spmm_wpg<NMAX, 16, true, PERM, BITS>(wpg, a, s);
        case 3: return launch_spmm_wpg<NMAX, 16, false, PERM, BITS>(wpg, a, s);
        case 2: return launch_spmm_wpg<NMAX, 11, false, PERM, BITS>(wpg, a, s);
        case 1: return launch_spmm_wpg<NMAX, 8, false, PERM, BITS>(wpg, a, s);
        default: return launch_spmm_wpg<NMAX, 4, false, PERM, BITS>(wpg, a, s);
    }
}

// The row-reordered (4-bit), the 2-bit and the narrow (N <= 4, 4-bit, rows
// in stored order) instantiations live in their own translation units.
hipError_t launch_cfg_perm(int wpg, int idx, const SpmmArgs &a, hipStream_t s);
hipError_t launch_cfg_w2(int wpg, int idx, const SpmmArgs &a, hipStream_t s);
hipError_t launch_cfg_narrow(int wpg, int idx, const SpmmArgs &a, hipStream_t s);

}  // namespace us_spmm_detail

#endif  // UNIONSPARSE_US_SPMM_KERNEL_H

