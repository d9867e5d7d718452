// Backward instantiations of the fused WTConv kernel (see wtconv_fused.h).
#include "wtconv_fused.h"

namespace wtc {

hipError_t launch_backward(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
    return dispatch<true>(k, dt, a, grid, s);
}

}  // namespace wtc
