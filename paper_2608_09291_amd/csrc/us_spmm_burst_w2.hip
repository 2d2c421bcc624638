// Single-pass SpMM instantiations: 2-bit weights (the W2A4 setting of
// Section VII), up to 16 activation columns.
// A translation unit of its own so that the kernel families compile in
// parallel.
#include "us_spmm_burst.h"

namespace us_spmm_detail {

hipError_t launch_burst_w2(int wpg, int ch, const BurstArgs &b, hipStream_t s) {
    return launch_burst_cfg<false, 2, 16>(wpg, ch, b, s);
}

}  // namespace us_spmm_detail
