// Forward instantiations of the fused WTConv kernel (see wtconv_fused.h).
#include "wtconv_fused.h"

namespace wtc {

hipError_t launch_forward(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
    if (a.mx_rounds > 0) return launch_forward_mixed(k, dt, a, grid, s);
    return dispatch<false>(k, dt, a, grid, s);
}

namespace {

template <int K, typename ST, bool ONE>
int wgs_variant(int fallback)
{
    static std::atomic<int> cache{0};
    return wgs_by_regs(reinterpret_cast<const void*>(&fused_kernel<K, ST, false, ONE, false>), cache, fallback);
}

template <int K, typename ST>
int wgs_dt(bool one, int fallback)
{
    return one ? wgs_variant<K, ST, true>(fallback) : wgs_variant<K, ST, false>(fallback);
}

template <int K>
int wgs_k(wtconv_dtype dt, bool one, int fallback)
{
    switch (dt) {
        case WTCONV_F32: return wgs_dt<K, float>(one, fallback);
        case WTCONV_BF16: return wgs_dt<K, uint16_t>(one, fallback);
        case WTCONV_F16: return wgs_dt<K, _Float16>(one, fallback);
    }
    return fallback;
}

}  // namespace

int forward_wgs_by_regs(int k, wtconv_dtype dt, bool one, int fallback)
{
    switch (k) {
        case 1: return wgs_k<1>(dt, one, fallback);
        case 3: return wgs_k<3>(dt, one, fallback);
        case 5: return wgs_k<5>(dt, one, fallback);
        case 7: return wgs_k<7>(dt, one, fallback);
        case 9: return wgs_k<9>(dt, one, fallback);
    }
    return fallback;
}

}  // namespace wtc
