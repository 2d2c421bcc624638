// Instantiations of the SpMM kernel for the decode regime's narrow activation
// matrices (N <= 4, 4-bit weights, rows in stored order): their activation
// staging needs a quarter of the registers. A translation unit of its own so
// that the kernel families compile in parallel.
#include "us_spmm_kernel.h"

namespace us_spmm_detail {

hipError_t launch_cfg_narrow(int wpg, int idx, const SpmmArgs &a, hipStream_t s) {
    return launch_cfg<false, 4, 4>(wpg, idx, a, s);
}

}  // namespace us_spmm_detail
