// Instantiations of the SpMM kernel for row-reordered LTs (Section V-B), the
// narrow N <= 4 ones included, in a translation unit of their own so that the
// kernel families compile in parallel.
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

hipError_t launch_cfg_perm(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    return a.N <= 4 ? launch_cfg<true, 4, 4>(wpg, idx, a, s) : launch_cfg<true, 4>(wpg, idx, a, s);
}

}  // namespace us_spmm_detail
