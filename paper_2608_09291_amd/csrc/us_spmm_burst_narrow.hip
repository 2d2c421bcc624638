// Single-pass SpMM instantiations: 4-bit weights in stored row order, up to
// 4 activation columns (the decode regime's narrow batches; a quarter of the
// activation staging registers).
// A translation unit of its own so that the kernel families compile in
// parallel.
#include "us_spmm_burst.h"

namespace us_spmm_detail {

hipError_t launch_burst_narrow(int wpg, int ch, const BurstArgs &b, hipStream_t s) {
    return launch_burst_cfg<false, 4, 4>(wpg, ch, b, s);
}

}  // namespace us_spmm_detail
