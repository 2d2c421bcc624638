// Instantiations of the SpMM kernel above 16 activation columns (NMAX = 32)
// with 8-LT chunks, for every weight form, in a translation unit that the
// library builds with the compiler's default scheduling strategy: under the
// iterative ILP strategy of the other units some of them exceed the
// registers of four wavefronts per SIMD.
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

template <bool PERM, int BITS>
hipError_t launch_cfg_wide8(int wpg, const SpmmArgs &a, hipStream_t s) {
    return launch_spmm_wpg<32, 8, false, PERM, BITS>(wpg, a, s);
}

template hipError_t launch_cfg_wide8<false, 4>(int, const SpmmArgs &, hipStream_t);
template hipError_t launch_cfg_wide8<true, 4>(int, const SpmmArgs &, hipStream_t);
template hipError_t launch_cfg_wide8<false, 2>(int, const SpmmArgs &, hipStream_t);

}  // namespace us_spmm_detail
