// Instantiations of the SpMM kernel above 16 activation columns (NMAX = 32,
// two MFMA column blocks) for every weight form: 4-bit rows in stored
// order, row-reordered 4-bit, and 2-bit. A translation unit of its own, as
// the library builds it with the compiler's default scheduling strategy
// (the plain and 2-bit units use the iterative ILP strategy, which leaves
// some of these kernels above the registers of four wavefronts per SIMD).
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

template <bool PERM, int BITS>
hipError_t launch_cfg_wide(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    return idx == 1 ? launch_spmm_wpg<32, 8, false, PERM, BITS>(wpg, a, s)
                    : launch_spmm_wpg<32, 4, false, PERM, BITS>(wpg, a, s);
}

template hipError_t launch_cfg_wide<false, 4>(int, int, const SpmmArgs &, hipStream_t);
template hipError_t launch_cfg_wide<true, 4>(int, int, const SpmmArgs &, hipStream_t);
template hipError_t launch_cfg_wide<false, 2>(int, int, const SpmmArgs &, hipStream_t);

}  // namespace us_spmm_detail
