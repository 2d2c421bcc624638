// Instantiations of the SpMM kernel for 2-bit weights (the W2A4 setting of
// Section VII), in a translation unit of their own so that the kernel
// families compile in parallel.
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

hipError_t launch_cfg_w2(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    return launch_cfg<false, 2>(wpg, idx, a, s);
}

}  // namespace us_spmm_detail
