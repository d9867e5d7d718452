// Forward instantiations of the fused WTConv kernel (see wtconv_fused.h).
#include "wtconv_fused.h"

namespace wtc {

hipError_t launch_forward(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
    return dispatch<false>(k, dt, a, grid, s);
}

}  // namespace wtc
