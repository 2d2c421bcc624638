// Single-pass SpMM instantiations: 4-bit weights in stored row order, up to
// 16 activation columns.
// A translation unit of its own so that the kernel families compile in
// parallel.
#include "us_spmm_burst.h"

namespace us_spmm_detail {

hipError_t launch_burst_plain(int wpg, int ch, const BurstArgs &b, hipStream_t s) {
    return launch_burst_cfg<false, 4, 16>(wpg, ch, b, s);
}

}  // namespace us_spmm_detail
