// Auxiliary kernels of libwtconv for gfx950: the level-m raw LL carrier of the
// split and region executions, and the fixed-order reduction of the
// per-workgroup kernel-gradient partials with the eq. (foldgrad) unfold.
#include "wtconv_fused.h"

namespace wtc {
namespace {

// One wavefront per (channel, kernel row).
__global__ void __launch_bounds__(64) reduce_kernel(const ReduceArgs a)
{
    reduce_task(a, blockIdx.x, blockIdx.y, threadIdx.x);
}

// Raw LL carrier of level M (1 <= M <= 6): M levels of the orthonormal
// butterfly's LL compose to 2^-M times the sum of each 2^M x 2^M pixel block
// (zero outside the plane), written in the input's storage type. One thread
// per output site. A workgroup covers
// 256 consecutive sites: the (plane, row, column) of its first site is
// computed once (uniformly), and each thread steps from there with fp32
// reciprocals of small offsets (exact below 2^20). The block's loads are all
// independent (fully unrolled), vectorised along rows when the plane allows.
template <typename T, int M>
__global__ void __launch_bounds__(256) carrier_kernel(const CarrierArgs a)
{
    constexpr int E = 1 << M;
    const long n = a.planes * a.H1 * a.W1;
    const T* in = reinterpret_cast<const T*>(a.in);
    const bool vec = a.vec_ok != 0;
    const float r_w1 = 1.0f / (float)a.W1, r_h1 = 1.0f / (float)a.H1;
    for (long e0 = (long)blockIdx.x * 256; e0 < n; e0 += (long)gridDim.x * 256) {
        const long pj0 = e0 / a.W1;  // uniform
        const int i0 = (int)(e0 - pj0 * a.W1);
        const long p0 = pj0 / a.H1;
        const int j0 = (int)(pj0 - p0 * a.H1);
        const long e = e0 + threadIdx.x;
        if (e >= n) continue;
        const int qi = fdiv(i0 + (int)threadIdx.x, r_w1);  // rows advanced
        const int i = i0 + (int)threadIdx.x - qi * a.W1;
        const int qj = fdiv(j0 + qi, r_h1);                 // planes advanced
        const int j = j0 + qi - qj * a.H1;
        const long p = p0 + qj;
        const int y0 = j << M, x0 = i << M;
        const T* base = in + (p * a.H + y0) * a.W + x0;
        const bool full = vec && x0 + E <= a.W;
        float s = 0.f;
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const T* row = base + (long)r * a.W;
            float rs = 0.f;
            if (y0 + r >= a.H) {
                // rows below the plane are zero
            } else if (full && M == 1) {
                float v[2];
                load2(row, v);
                rs = v[0] + v[1];
            } else if (full) {
#pragma unroll
                for (int c = 0; c < E; c += 4) {
                    float v[4];
                    load4(row + c, v);
                    rs += (v[0] + v[1]) + (v[2] + v[3]);
                }
            } else {
#pragma unroll
                for (int c = 0; c < E; ++c)
                    if (x0 + c < a.W) rs += to_f32(row[c]);
            }
            s += rs;
        }
        reinterpret_cast<T*>(a.out)[e] = from_f32<T>(__builtin_ldexpf(s, -M));
    }
}

template <typename T>
hipError_t launch_carrier_t(const CarrierArgs& a, int grid, hipStream_t s)
{
    switch (a.m) {
        case 1: hipLaunchKernelGGL((carrier_kernel<T, 1>), dim3(grid), dim3(256), 0, s, a); break;
        case 2: hipLaunchKernelGGL((carrier_kernel<T, 2>), dim3(grid), dim3(256), 0, s, a); break;
        case 3: hipLaunchKernelGGL((carrier_kernel<T, 3>), dim3(grid), dim3(256), 0, s, a); break;
        case 4: hipLaunchKernelGGL((carrier_kernel<T, 4>), dim3(grid), dim3(256), 0, s, a); break;
        case 5: hipLaunchKernelGGL((carrier_kernel<T, 5>), dim3(grid), dim3(256), 0, s, a); break;
        case 6: hipLaunchKernelGGL((carrier_kernel<T, 6>), dim3(grid), dim3(256), 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_carrier(wtconv_dtype dt, const CarrierArgs& a, hipStream_t s)
{
    if (a.m < 1 || a.m > 6) return hipErrorInvalidValue;
    const long n = a.planes * a.H1 * a.W1;
    const long blocks = (n + 255) / 256;
    const int grid = (int)(blocks < 16384 ? blocks : 16384);
    switch (dt) {
        case WTCONV_F32: return launch_carrier_t<float>(a, grid, s);
        case WTCONV_BF16: return launch_carrier_t<uint16_t>(a, grid, s);
        case WTCONV_F16: return launch_carrier_t<_Float16>(a, grid, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s)
{
    const dim3 grid(a.C, 1 + 4 * a.L);
    hipLaunchKernelGGL(reduce_kernel, grid, dim3(64), 0, s, a);
    return hipGetLastError();
}

}  // namespace wtc
