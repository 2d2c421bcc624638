// Instantiations of the SpMM kernel for row-reordered LTs (Section V-B), in a
// translation unit of their own so that the two kernel families compile in
// parallel.
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

hipError_t launch_cfg_perm(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    return launch_cfg<true, 4>(wpg, idx, a, s);
}

}  // namespace us_spmm_detail
