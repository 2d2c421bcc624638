// Dense INT8 GEMM on the int8 matrix cores (the in-library dense comparison
// point), and the measurement probes of us_probe.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "us.h"
#include "us_probe.h"

namespace {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Y = W X, W int8 M x K, X int8 N x K (row n = column n of X), Y int32 N x M.
// One workgroup per 16-row block, WPG wavefronts split K and combine in LDS,
// as in the sparse kernel. Lane l reads 16 consecutive k of W row l % 16 and
// of X row l % 16 (k-group l / 16); both operands use the same slot order.
template <int WPG, int NB>
__global__ __launch_bounds__(64 * WPG) void us_gemm_i8_kernel(const int8_t *__restrict__ w,
                                                              const int8_t *__restrict__ x,
                                                              int32_t *__restrict__ y, int M, int K,
                                                              int N) {
    __shared__ int32_t red[WPG][16 * 16 * NB];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int mb = blockIdx.x;
    const int nkb = K / 64;
    const int kb0 = wave * nkb / WPG, kb1 = (wave + 1) * nkb / WPG;
    const int rr = lane & 15, g = lane >> 4;

    const i32x4 *wrow = (const i32x4 *)(w + ((int64_t)mb * 16 + rr) * K) + g;
    const i32x4 *xrow[NB];
    bool xok[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int n = nb * 16 + rr;
        xok[nb] = n < N;
        xrow[nb] = (const i32x4 *)(x + (int64_t)(xok[nb] ? n : 0) * K) + g;
    }
    i32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (i32x4){0, 0, 0, 0};

    const i32x4 zero = {0, 0, 0, 0};
    int kb = kb0;
    for (; kb + 4 <= kb1; kb += 4) {
        i32x4 A[4], B[4][NB];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            A[u] = __builtin_nontemporal_load(wrow + 4 * (kb + u));
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) B[u][nb] = xok[nb] ? xrow[nb][4 * (kb + u)] : zero;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[u], B[u][nb], acc[nb], 0, 0, 0);
    }
    for (; kb < kb1; ++kb) {
        const i32x4 A = __builtin_nontemporal_load(wrow + 4 * kb);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const i32x4 B = xok[nb] ? xrow[nb][4 * kb] : zero;
            acc[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, B, acc[nb], 0, 0, 0);
        }
    }

#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[wave][(4 * g + v) * (16 * NB) + nb * 16 + rr] = acc[nb][v];
    __syncthreads();
    for (int e = threadIdx.x; e < 16 * N; e += 64 * WPG) {
        const int r = e & 15, n = e >> 4;
        int32_t s = 0;
#pragma unroll
        for (int wv = 0; wv < WPG; ++wv) s += red[wv][r * (16 * NB) + n];
        y[(int64_t)n * M + (int64_t)mb * 16 + r] = s;
    }
}

template <int WPG, int NB>
hipError_t launch_gemm(const int8_t *w, const int8_t *x, int32_t *y, int M, int K, int N, hipStream_t s) {
    hipLaunchKernelGGL((us_gemm_i8_kernel<WPG, NB>), dim3(M / 16), dim3(64 * WPG), 0, s, w, x, y, M, K, N);
    return hipGetLastError();
}

template <int NB>
hipError_t launch_gemm_wpg(int wpg, const int8_t *w, const int8_t *x, int32_t *y, int M, int K, int N,
                           hipStream_t s) {
    switch (wpg) {
        case 1: return launch_gemm<1, NB>(w, x, y, M, K, N, s);
        case 2: return launch_gemm<2, NB>(w, x, y, M, K, N, s);
        case 4: return launch_gemm<4, NB>(w, x, y, M, K, N, s);
        case 8: return launch_gemm<8, NB>(w, x, y, M, K, N, s);
        default: return launch_gemm<16, NB>(w, x, y, M, K, N, s);
    }
}

// ---------------------------------------------------------------------------
// Probes
// ---------------------------------------------------------------------------

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 4;
constexpr size_t kProbeMaxBlocks = 4096;

// Workgroups of the copy probe: one pass of kProbeUnroll pieces per thread,
// at most kProbeMaxBlocks.
size_t probe_blocks(size_t n16) {
    size_t b = (n16 + kProbeThreads * kProbeUnroll - 1) / (kProbeThreads * kProbeUnroll);
    if (b < 1) b = 1;
    return b < kProbeMaxBlocks ? b : kProbeMaxBlocks;
}

// Read probe shapes: threads per workgroup, 16-byte loads issued together
// per thread, workgroups per compute unit. No one shape reads fastest at
// every size on this GPU: many workgroups with few loads each win at tens of
// MB, few large workgroups at hundreds of MB. A caller that wants the
// ceiling times every shape and keeps the fastest.
struct ProbeShape {
    int threads, unroll, per_cu;
};
constexpr ProbeShape kReadShapes[US_PROBE_READ_SHAPES] = {{256, 4, 8}, {512, 4, 1}, {1024, 4, 8}, {256, 8, 1}};
constexpr int kReadMaxWavesPerCu = 128;                 // 8 x 1024 / 64

// Each thread reads pieces idx, idx + stride, ... (stride = all threads of
// the grid), U at a time, and folds them into one word by XOR. The
// wavefront folds its 64 words with lane shuffles, and lane 0 stores the
// result at sink[wavefront index in the grid]: no barrier, and the XOR of
// the words stored equals the XOR of the data read.
template <int T, int U>
__global__ __launch_bounds__(T) void probe_read_kernel(const i32x4 *__restrict__ src, size_t n16,
                                                       uint32_t *__restrict__ sink) {
    uint32_t acc = 0;
    const size_t stride = (size_t)gridDim.x * T;
    size_t idx = (size_t)blockIdx.x * T + threadIdx.x;
    for (; idx + (U - 1) * stride < n16; idx += U * stride) {
        i32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + idx + u * stride);
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= (uint32_t)(v[u].x ^ v[u].y ^ v[u].z ^ v[u].w);
    }
    for (; idx < n16; idx += stride) {
        const i32x4 v = __builtin_nontemporal_load(src + idx);
        acc ^= (uint32_t)(v.x ^ v.y ^ v.z ^ v.w);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
    if ((threadIdx.x & 63) == 0) sink[(size_t)blockIdx.x * (T / 64) + threadIdx.x / 64] = acc;
}

int probe_cus() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    return n;
}

__global__ __launch_bounds__(kProbeThreads) void probe_copy_kernel(const i32x4 *__restrict__ src,
                                                                   i32x4 *__restrict__ dst, size_t n16) {
    const size_t stride = (size_t)gridDim.x * kProbeThreads;
    for (size_t idx = (size_t)blockIdx.x * kProbeThreads + threadIdx.x; idx < n16; idx += stride)
        dst[idx] = src[idx];
}

// The same copy with the loads the SpMM kernels stage their payload with:
// non-temporal buffer_load_dwordx4 straight into LDS, 1 KB per wavefront
// and step (lane l's 16 bytes at LDS base + 16 l, the base in M0); each lane
// then reads its 16 bytes back from LDS and stores them to dst. Bytes past
// the buffer's range read as zero and are not stored. The LDS read of one
// step is complete (its value feeds the store) before the next step's load
// overwrites the buffer.
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) i32x4 lds_i32x4;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void probe_dma16_nt(u32x4 desc, uint32_t lds, uint32_t voff) {
    __asm__ volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds\n\ts_waitcnt vmcnt(0)"
                     :
                     : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(desc)
                     : "memory", "m0");
}
#pragma clang diagnostic pop

__global__ __launch_bounds__(kProbeThreads) void probe_copy_lds_kernel(const uint8_t *__restrict__ src,
                                                                       i32x4 *__restrict__ dst, uint32_t n16) {
    __shared__ __attribute__((aligned(16))) uint32_t buf[kProbeThreads * 4];
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t lds = (uint32_t)(size_t)(lds_u32 *)buf + 1024u * wave;
    const uint64_t sa = (uint64_t)(size_t)src;
    const u32x4 desc = (u32x4){(uint32_t)sa, (uint32_t)(sa >> 32) & 0xFFFFu, 16u * n16, 0x00020000u};
    const uint32_t waves = gridDim.x * (kProbeThreads / 64);
    for (uint32_t piece = blockIdx.x * (kProbeThreads / 64) + wave; 64ull * piece < n16; piece += waves) {
        probe_dma16_nt(desc, lds, 1024u * piece + 16u * lane);
        const i32x4 v = *(const lds_i32x4 *)(size_t)(lds + 16u * lane);
        if (64u * piece + lane < n16) dst[64u * piece + lane] = v;
    }
}

__global__ void probe_spin_kernel(uint64_t ticks) {
    const uint64_t t0 = wall_clock64();
    while (wall_clock64() - t0 < ticks) __builtin_amdgcn_s_sleep(8);
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

extern "C" us_status us_gemm_i8(const int8_t *w, const int8_t *x, int32_t M, int32_t K, int32_t N,
                                int32_t *y, void *stream) {
    if (!w || !x || !y) return US_ERR_ARG;
    if (M <= 0 || K <= 0 || M % 16 || K % 64 || K > US_K_MAX) return US_ERR_SHAPE;
    if (N < 1 || N > US_N_LIMIT) return US_ERR_SHAPE;
    if (!aligned16(w) || !aligned16(x) || ((uintptr_t)y & 3)) return US_ERR_ARG;
    const int nrb = M / 16, nkb = K / 64;
    int wpg = 1;
    while (wpg < 16 && nrb * wpg * 2 <= 256 * 16) wpg *= 2;
    while (wpg > 1 && wpg > nkb) wpg /= 2;
    hipStream_t s = (hipStream_t)stream;
    // Slabs of up to US_N_MAX columns, as in us_spmm.
    for (int n0 = 0; n0 < N; n0 += US_N_MAX) {
        const int ns = N - n0 < US_N_MAX ? N - n0 : US_N_MAX;
        const int8_t *xs = x + (int64_t)n0 * K;
        int32_t *ys = y + (int64_t)n0 * M;
        const hipError_t err = ns > 16 ? launch_gemm_wpg<2>(wpg, w, xs, ys, M, K, ns, s)
                                       : launch_gemm_wpg<1>(wpg, w, xs, ys, M, K, ns, s);
        if (err != hipSuccess) return US_ERR_DEVICE;
    }
    return US_OK;
}

extern "C" size_t us_probe_read_sink_words(size_t bytes) {
    (void)bytes;
    return (size_t)kReadMaxWavesPerCu * (size_t)probe_cus();
}

extern "C" us_status us_probe_read(const void *src, size_t bytes, uint32_t *sink, int32_t shape, void *stream) {
    if (!src || !sink || bytes == 0 || bytes % 16 || !aligned16(src)) return US_ERR_ARG;
    if (shape < 0 || shape >= US_PROBE_READ_SHAPES) return US_ERR_ARG;
    const size_t n16 = bytes / 16;
    const ProbeShape sh = kReadShapes[shape];
    const dim3 grid((unsigned)(sh.per_cu * probe_cus()));
    const hipStream_t st = (hipStream_t)stream;
    const i32x4 *s16 = (const i32x4 *)src;
    switch (shape) {
        case 0: hipLaunchKernelGGL((probe_read_kernel<256, 4>), grid, dim3(256), 0, st, s16, n16, sink); break;
        case 1: hipLaunchKernelGGL((probe_read_kernel<512, 4>), grid, dim3(512), 0, st, s16, n16, sink); break;
        case 2: hipLaunchKernelGGL((probe_read_kernel<1024, 4>), grid, dim3(1024), 0, st, s16, n16, sink); break;
        default: hipLaunchKernelGGL((probe_read_kernel<256, 8>), grid, dim3(256), 0, st, s16, n16, sink); break;
    }
    return hipGetLastError() == hipSuccess ? US_OK : US_ERR_DEVICE;
}

extern "C" us_status us_probe_copy(const void *src, void *dst, size_t bytes, void *stream) {
    if (!src || !dst || bytes == 0 || bytes % 16 || !aligned16(src) || !aligned16(dst)) return US_ERR_ARG;
    const size_t n16 = bytes / 16;
    hipLaunchKernelGGL(probe_copy_kernel, dim3((unsigned)probe_blocks(n16)), dim3(kProbeThreads), 0,
                       (hipStream_t)stream, (const i32x4 *)src, (i32x4 *)dst, n16);
    return hipGetLastError() == hipSuccess ? US_OK : US_ERR_DEVICE;
}

extern "C" us_status us_probe_copy_lds(const void *src, void *dst, size_t bytes, void *stream) {
    if (!src || !dst || bytes == 0 || bytes % 16 || !aligned16(src) || !aligned16(dst)) return US_ERR_ARG;
    if (bytes > ((size_t)1 << 31)) return US_ERR_ARG;
    const size_t n16 = bytes / 16;
    hipLaunchKernelGGL(probe_copy_lds_kernel, dim3((unsigned)probe_blocks(n16)), dim3(kProbeThreads), 0,
                       (hipStream_t)stream, (const uint8_t *)src, (i32x4 *)dst, (uint32_t)n16);
    return hipGetLastError() == hipSuccess ? US_OK : US_ERR_DEVICE;
}

extern "C" us_status us_probe_spin(uint64_t ns, void *stream) {
    if (ns > 1000000000ull) return US_ERR_ARG;
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess) return US_ERR_DEVICE;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0)
        return US_ERR_DEVICE;
    const uint64_t ticks = ns * (uint64_t)khz / 1000000ull;
    hipLaunchKernelGGL(probe_spin_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, ticks);
    return hipGetLastError() == hipSuccess ? US_OK : US_ERR_DEVICE;
}
