// Backward instantiations of the fused WTConv kernel for k = 9 (see
// wtconv_fused.h), in a translation unit of their own: these kernels hold the
// most kernel-gradient sums per lane and take the longest to compile.
#include "wtconv_fused.h"

namespace wtc {

hipError_t launch_backward_k9(wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
    return launch_dt<9, true>(dt, a, grid, s);
}

}  // namespace wtc
