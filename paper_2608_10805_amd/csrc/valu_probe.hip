// Sustained fp32 FMA throughput probe (measurement helper of the benchmark,
// not part of the operator). Every lane runs kChains independent FMA chains
// for `iters` steps, so the VALU issues back to back without dependency
// stalls; the result is stored so that nothing is optimised away. The
// benchmark divides the FMA count by the measured time to get the chip's
// sustained non-packed fp32 rate (and, through the lane count, its clock).
#include <hip/hip_runtime.h>

namespace {

constexpr int kChains = 8;

__global__ void __launch_bounds__(256) fma_probe_kernel(float* out, int iters, float a, float b)
{
    float acc[kChains];
#pragma unroll
    for (int i = 0; i < kChains; ++i) acc[i] = (float)(threadIdx.x + i) * 1e-3f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
#pragma unroll
            for (int i = 0; i < kChains; ++i) acc[i] = __builtin_fmaf(acc[i], a, b);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kChains; ++i) s += acc[i];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

extern "C" {

// FMAs one launch performs: blocks * 256 lanes * iters * 16 * kChains.
long long valu_probe_fmas(int blocks, int iters) { return (long long)blocks * 256 * iters * 16 * kChains; }

// Enqueue the probe on `stream`; `out` holds blocks * 256 floats.
int valu_probe_launch(float* out, int blocks, int iters, hipStream_t stream)
{
    if (!out || blocks < 1 || iters < 1) return 1;
    hipLaunchKernelGGL(fma_probe_kernel, dim3(blocks), dim3(256), 0, stream, out, iters, 0.999f, 1e-3f);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
