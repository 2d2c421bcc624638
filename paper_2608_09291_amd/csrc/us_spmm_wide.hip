// Instantiations of the SpMM kernel above 16 activation columns (NMAX = 32,
// two MFMA column blocks) with 4-LT chunks, for every weight form: 4-bit
// rows in stored order, row-reordered 4-bit, and 2-bit. The 8-LT chunks sit
// in us_spmm_wide8.hip, which the library builds with the compiler's default
// scheduling strategy (under the iterative ILP strategy this unit uses,
// some of them exceed the registers of four wavefronts per SIMD).
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

template <bool PERM, int BITS>
hipError_t launch_cfg_wide(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    return idx == 1 ? launch_cfg_wide8<PERM, BITS>(wpg, a, s) : launch_spmm_wpg<32, 4, false, PERM, BITS>(wpg, a, s);
}

template hipError_t launch_cfg_wide<false, 4>(int, int, const SpmmArgs &, hipStream_t);
template hipError_t launch_cfg_wide<true, 4>(int, int, const SpmmArgs &, hipStream_t);
template hipError_t launch_cfg_wide<false, 2>(int, int, const SpmmArgs &, hipStream_t);

}  // namespace us_spmm_detail
