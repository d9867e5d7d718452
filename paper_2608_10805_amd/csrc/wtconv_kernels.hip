// Auxiliary kernels of libwtconv for gfx950: the level-m raw LL carrier of the
// split and region executions, and the fixed-order reduction of the
// per-workgroup kernel-gradient partials with the eq. (foldgrad) unfold.
#include "wtconv_fused.h"

namespace wtc {
namespace {

// Sum the per-workgroup partials over chunks in increasing order, then unfold
// eq. (foldgrad): dW = s * G and ds = <G, W>, where G is the gradient of the
// folded kernel s*W (the level partials carry an extra 4^l from the
// unnormalised pyramids, removed here exactly); for the base row also the bias
// terms d b0 = s0 * sum(dy) and b0 * sum(dy) in d s0. One wavefront per
// (channel, band row); lane t owns tap t (lane k*k the sum of dy); the
// d(scale) dot product is a fixed-order wavefront reduction.
__global__ void __launch_bounds__(64) reduce_kernel(const ReduceArgs a)
{
    const int KK = a.k * a.k;
    const int NP = partial_floats_per_channel(a.k, a.L);
    const int c = blockIdx.x;
    const int band = blockIdx.y;  // 0 = base, else 1 + (l-1)*4 + q
    const int t = threadIdx.x;
    if (band == 0 && a.skip_base) return;
    float scale, norm;
    const float* w;
    float* dw;
    float* ds;
    if (band == 0) {
        scale = a.p.s0[c];
        norm = 1.f;
        w = a.p.w0 + (long)c * KK;
        dw = a.dw0 + (long)c * KK;
        ds = a.ds0 + c;
    } else {
        const int l = (band - 1) / 4 + 1, q = (band - 1) % 4;
        const int ch = 4 * c + q;
        scale = a.p.ls[l - 1][ch];
        norm = __builtin_ldexpf(1.f, -2 * l);
        w = a.p.lw[l - 1] + (long)ch * KK;
        dw = a.dlw[l - 1] + (long)ch * KK;
        ds = a.dls[l - 1] + ch;
    }
    float prod = 0.f;
    if (t < KK) {
        const float* src = a.partial + (long)c * NP + band * KK + t;
        const long step = (long)a.C * NP;
        // chunk order is kept; the loads of a group of 8 chunks are issued
        // together so that their latencies overlap
        float G = 0.f;
        int ch = 0;
        for (; ch + 8 <= a.nchunks; ch += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = src[(long)(ch + u) * step];
#pragma unroll
            for (int u = 0; u < 8; ++u) G += v[u];
        }
        for (; ch < a.nchunks; ++ch) G += src[(long)ch * step];
        G *= norm;
        dw[t] = scale * G;
        prod = G * w[t];
    } else if (band == 0 && t == KK) {
        // folded base bias b~ = s0 * b0: its gradient is the sum of dy, so
        // d b0 = s0 * sum(dy) and d s0 gains b0 * sum(dy) (eq. foldgrad)
        const float* src = a.partial + (long)c * NP + (NP - 1);
        const long step = (long)a.C * NP;
        float Gb = 0.f;
        for (int ch = 0; ch < a.nchunks; ++ch) Gb += src[(long)ch * step];
        if (a.db0) a.db0[c] = scale * Gb;
        if (a.p.b0) prod = a.p.b0[c] * Gb;
    }
    prod = wave_sum(prod);
    if (t == 0) *ds = prod;
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
