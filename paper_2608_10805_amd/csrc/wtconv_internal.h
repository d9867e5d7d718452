// Internal interface between the host dispatcher (wtconv_api.cpp) and the
// gfx950 kernels (wtconv_kernels.hip). Not part of the public ABI.
#pragma once

#include <algorithm>
#include <atomic>

#include <hip/hip_runtime.h>

#include "wtconv.h"

namespace wtc {

constexpr int kLdsBytesMax = 160 * 1024;  // one compute unit's LDS

// Lets kernel `fn` launch with up to a whole compute unit's LDS, on the
// current device. The attribute persists for the process, so it is set once
// per (kernel, device): `done` is the calling kernel's own set of devices
// (bit d for device d < 64; larger ids set it on every launch). Two threads
// racing both set it, which is harmless.
inline hipError_t allow_full_lds(const void* fn, std::atomic<unsigned long long>& done)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const unsigned long long bit = (dev >= 0 && dev < 64) ? 1ull << dev : 0ull;
    if (bit && (done.load(std::memory_order_relaxed) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytesMax);
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_relaxed);
    return e;
}

// Workgroups per compute unit that a 256-thread kernel's registers allow, from
// its compiled VGPR count (512 per SIMD lane, allocated in blocks of 8, at
// most 8 wavefronts per SIMD), or `fallback` if the HIP runtime cannot report
// it (no device). The answer is cached in `cache` (0: not asked yet, -1: the
// runtime could not tell).
inline int wgs_by_regs(const void* fn, std::atomic<int>& cache, int fallback)
{
    int v = cache.load(std::memory_order_relaxed);
    if (v > 0) return v;
    if (v < 0) return fallback;
    hipFuncAttributes attr;
    if (hipFuncGetAttributes(&attr, fn) != hipSuccess || attr.numRegs <= 0) {
        (void)hipGetLastError();  // clear the error state left by a failed query
        cache.store(-1, std::memory_order_relaxed);
        return fallback;
    }
    const int regs = (attr.numRegs + 7) / 8 * 8;
    v = std::max(1, std::min(8, 512 / regs));
    cache.store(v, std::memory_order_relaxed);
    return v;
}

constexpr int kMaxLevels = WTCONV_MAX_LEVELS;
constexpr int kThreads = 256;  // 4 wavefronts of 64 lanes per workgroup
constexpr int kWaves = kThreads / 64;

// Caps on how many tiles of one subband a lane may hold in registers while a
// level is filtered in place (the filtered coefficients overwrite the
// unfiltered ones only after every read of the level is done).
constexpr int kMaxRounds4 = 4;   // 4x4-site tiles
constexpr int kMaxRounds2 = 8;   // 2x2-site tiles
constexpr int kMaxRounds1 = 16;  // single sites
// Task rounds per lane of the mixed forward kernel (its results stay in
// registers until every window has been read).
constexpr int kMixedMaxRounds = 4;
constexpr int kMixedMaxSegs = 4 * kMaxLevels + 4;

// On-chip layout of one level of the Haar pyramid of one plane: four
// band-planar arrays, each with a zero halo of R sites on every side.
// Site (j, i) of band q lives at off + q * band + (j + R) * pitch + (i + R).
struct LevelGeom {
    int h, w;    // grid size ceil(H / 2^l) x ceil(W / 2^l)
    int T;       // edge of the site tiles used to filter this level (1, 2, 4)
    int eh, ew;  // tile-aligned extents (multiples of T)
    int pitch;   // floats per row, multiple of 4
    int band;    // floats per band, multiple of 4
    int off;     // float offset of band 0 within the plane's region
    // fp32 reciprocals of the divisors used to decompose flat indices
    float r_w;     // 1 / w
    float r_hw;    // 1 / (h * w)
    float r_tx;    // 1 / (ew / T), tiles per row
    float r_tper;  // 1 / ((ew / T) * (eh / T)), tiles per plane
};

// On-chip layout of one plane: the zero-haloed input plane (pixel (y, x) at
// (y + R) * xpitch + (x + R)) followed by the L levels.
struct PlaneGeom {
    int H, W, L;
    int xpitch, xrows;
    int tiles_x, tiles_y;  // 4x4-pixel output tiles per row / column
    LevelGeom lv[kMaxLevels + 1];  // entries 1..L are used
    int plane_floats;              // size of one plane's region (multiple of 4)
    float r_W;                     // 1 / W
    float r_tiles_x;               // 1 / tiles_x
    float r_tiles;                 // 1 / (tiles_x * tiles_y)
    // Lanes per row of output tiles in the forward's block loads and output
    // tiles (>= tiles_x; the lanes past tiles_x idle). A multiple of 8 keeps
    // each group of 8 lanes of a 16-byte LDS access inside one tile row.
    int tiles_xl;
    float r_tiles_xl;              // 1 / tiles_xl
    float r_tiles_l;               // 1 / (tiles_xl * tiles_y)
};

struct ParamPtrs {
    const float* w0;  // [C][k][k]
    const float* s0;  // [C]
    const float* b0;  // [C] base bias, or null (zero)
    const float* lw[kMaxLevels];  // [4C][k][k] per level
    const float* ls[kMaxLevels];  // [4C] per level
    // 1: the forward kernels fold every kernel rotated by 180 degrees. The
    // forward pass on dy with rotated kernels is dx (the adjoint of a "same"
    // correlation is the correlation with the rotated kernel, and synthesis
    // and analysis are each other's transposes).
    int rot;
};

// Finalize of the kernel gradients: the fixed-order sum of [nchunks][C][NP]
// partials and the unfold of eq. (foldgrad), one wavefront per (channel,
// kernel row).
struct ReduceArgs {
    const float* partial;
    int nchunks, C, k, L;
    int skip_base;  // do not write the base gradients
    ParamPtrs p;
    float* dw0;
    float* ds0;
    float* db0;  // nullable
    float* dlw[kMaxLevels];
    float* dls[kMaxLevels];
};

struct FusedArgs {
    const void* in;      // forward: x; backward: dy
    const void* aux;     // backward: x (correlation partner of dy); forward: unused
    void* out;           // forward: y; backward: dx (may be null)
    float* partial;      // backward: [nchunks][C][NP] kernel-gradient partials
    ParamPtrs p;
    int B, C;
    int nb;              // planes of one channel handled by one workgroup
    int PP;              // planes resident on chip at once
    int vec_ok;          // 1 if plane bases allow 16-byte (f32) / 8-byte (16-bit) vector access
    int lds_floats;      // dynamic LDS of the workgroup, in floats
    int one_round;       // 1 if every level is filtered in a single register-tile round
    int merge_deep;      // forward: levels 1 and >= 3 share one round of 4x4 site tiles
    int skip_base;       // 1: no base path and no base-kernel gradient (coarse sub-problem)
    // Region mode (planes too large for LDS): each workgroup processes an
    // rg_T x rg_T output tile of a real_H x real_W plane through a region with
    // a halo of rg_h pixels on every side; g describes the region. `carry`
    // (nullable, any mode) is the contribution of the levels above
    // carry_level, on the level-carry_level grid ([B][C][carry_H][carry_W]).
    int rg_ntx, rg_nty;  // tiles per plane row / column
    int rg_T, rg_h;
    int real_H, real_W;
    float rg_r_itx;      // 1 / (rg_T / 4): inner output tiles per tile row
    float rg_r_itiles;   // 1 / (rg_T / 4)^2
    const void* carry;  // storage type of the pass
    int carry_H, carry_W, carry_level;
    // Mixed task rounds (forward, resident planes, every level in 4x4 site
    // tiles; wtconv_mixed.hip): mx_rounds > 0 selects it. Round r runs the
    // segments mx_seg[mx_seg0[r] .. mx_seg0[r + 1]), each a run of tasks:
    // every 4x4 tile (over the PP planes) of one band of one level, or the
    // next `count` output tiles. Packed: kind (1 output, 2 band) | level << 2 |
    // band << 6 | count << 8. Band segments sit in rounds <= mx_first_out,
    // output segments in rounds >= mx_first_out. mx_ntask[r]: tasks of round r;
    // mx_out0[r]: output tiles in the rounds before r.
    int mx_rounds, mx_first_out;
    int mx_seg0[kMixedMaxRounds + 1];
    int mx_ntask[kMixedMaxRounds], mx_out0[kMixedMaxRounds];
    int mx_seg[kMixedMaxSegs];
    // Forward kernels only: when fin_blocks > 0 the first fin_blocks
    // workgroups of the grid run the finalize `fin` (four (channel, kernel
    // row) tasks each, one per wavefront) and the plane work starts at
    // workgroup fin_blocks; the partials come from an earlier launch on the
    // stream.
    int fin_blocks;
    ReduceArgs fin;
    PlaneGeom g;
};

// Level-m raw LL carrier of every plane: 2^-m times the sum of each 2^m x 2^m
// block of the zero-extended input, a [planes][H1][W1] array in the input's
// storage type (H1, W1 = ceil(H / 2^m), ceil(W / 2^m)), summed in fp32 and
// rounded once.
struct CarrierArgs {
    const void* in;
    void* out;
    long planes;
    int H, W, H1, W1;
    int m;
    int vec_ok;  // 1 if the rows allow vector loads: 2-element loads for m = 1 (W even),
                 // 4-element ones beyond (W % 4 == 0); the input base is 16-byte aligned
};

// Planes of at most 8 x 8 pixels (wtconv_tiny.hip): one workgroup per four
// channels and 64 batch entries, one lane per batch entry.
struct TinyArgs {
    const void* in;   // forward: x; backward: dy
    const void* aux;  // backward: x
    void* out;        // forward: y; backward: dx (may be null)
    float* partial;   // backward: [ceil(B / 64)][C][NP] kernel-gradient partials
    ParamPtrs p;
    int B, C, H, W, L;
    int skip_base;    // 1: no base path and no base-kernel gradient (coarse sub-problem)
};
constexpr int kTinyMaxEdge = 8;

// Kernel-gradient pass (wtconv_grad.hip): one workgroup owns channel c and a
// run of nb batch planes of it, PP resident at once, at most one 4x4 pixel
// block per thread per batch. The x side is held in LDS with zero halos (the
// layout `g` of the fused kernels: the correlation windows are read there);
// the dy side is the correlation centre: its pixels and levels 1-2 stay in the
// registers of the thread that loaded them, and its level pyramid is stored
// compact (no halo): level l band q site (j, i) at
// dy_off[l] + q * dy_band[l] + j * dy_pitch[l] + i within a plane's region.
// Level 1 of the dy side is written over the x plane (dy_off[1] == 0) once
// the base correlation no longer needs it, when it fits there.
struct GradArgs {
    const void* x;
    const void* dy;
    float* partial;  // [nchunks][C][NP] kernel-gradient partials, resident layout
    int B, C;
    int nb, PP;
    int rounds;      // 4x4 block rounds per plane: 1, or more with one resident plane
    int vec_ok;      // 1 if both plane bases allow 16-byte (f32) / 8-byte (16-bit) loads
    int lds_floats;
    int skip_base;   // 1: no base-kernel gradient (coarse sub-problem)
    int stride;      // floats per plane region (x side + dy side)
    float r_ring;    // 1 / (xpitch - 4 * tiles_x): ring columns of a middle row of the x plane
    // [tail0, tail1): floats of the x plane past dy level 1 that hold deeper
    // dy levels (when dy level 1 is stored over the x plane); cleared every
    // batch before those levels are built, so that their sites past the grid
    // read as zero; tail0 == tail1 when unused
    int tail0, tail1;
    int dy_off[kMaxLevels + 1], dy_pitch[kMaxLevels + 1], dy_band[kMaxLevels + 1];
    // Optional (one block round only, rounds == 1): the raw LL carriers of x
    // and dy at level cm (1 or 2) for a coarse sub-problem, [B][C][cH][cW] in
    // the storage type, as the carrier kernel writes them (same sums in the
    // same order); null when not wanted.
    void* cx;
    void* cdy;
    int cm, cH, cW;
    // Region mode (rg_ntx > 0; one block round, one resident region, L = 1):
    // workgroup (chunk, tile) covers the rg_T x rg_T output tile whose
    // top-left pixel is (ty * rg_T, tx * rg_T) of the real_H x real_W plane
    // through a region with a halo of rg_h pixels on every side; g describes
    // the region. Only the tile's own pixels and level-1 sites are counted,
    // and carriers are written for the tile's own sites; partials are
    // [nchunks * tiles][C][NP], tile-minor, as the fused region backward's.
    int rg_ntx, rg_nty, rg_T, rg_h, real_H, real_W;
    PlaneGeom g;
};

// Gradient pass: levels 1..grad_reg_levels(L >= 4) keep their kernel-gradient
// sums in registers across a workgroup's planes (levels 3-5 only in the
// variant for pyramids of 4 or more levels); deeper levels use LDS slots.
__host__ __device__ constexpr int grad_reg_levels(bool deep) { return deep ? 5 : 2; }

// Number of kernel-gradient floats per (chunk, channel): base k*k, then
// levels 1..L x bands 0..3 x k*k, then the sum of dy over the channel's pixels
// (the gradient of the folded base bias).
__host__ __device__ inline int partial_floats_per_channel(int k, int L) { return k * k * (1 + 4 * L) + 1; }

// Sites per chunk of the row-wise kernel-gradient correlation of a w-site-wide
// level: 4 up to 4 sites, else 8 or 16, whichever pads the row less (16 on
// ties: fewer chunks).
__host__ __device__ inline int row_chunk(int w)
{
    return w <= 4 ? 4 : (((w + 7) / 8 * 8 < (w + 15) / 16 * 16) ? 8 : 16);
}

// Lanes per row group of the row-wise kernel-gradient correlation: one lane
// per tap row, rounded up to a power of two (the groups are summed with an xor
// tree over the wavefront).
__host__ __device__ constexpr int row_group_lanes(int k)
{
    return k <= 1 ? 1 : (k <= 2 ? 2 : (k <= 4 ? 4 : (k <= 8 ? 8 : 16)));
}

hipError_t launch_forward(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s);
// Workgroups per CU that the registers of the forward kernel for (k, dt,
// single-round variant) allow; `fallback` if the runtime cannot tell.
int forward_wgs_by_regs(int k, wtconv_dtype dt, bool one, int fallback);
// The forward with mixed task rounds (a.mx_rounds in 1..kMixedMaxRounds).
hipError_t launch_forward_mixed(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s);
// Workgroups per CU that the registers of the mixed forward kernel for (k, dt,
// rounds) allow; `fallback` if the runtime cannot tell.
int mixed_wgs_by_regs(int k, wtconv_dtype dt, int rounds, int fallback);
hipError_t launch_backward(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s);
// The fused backward kernels for k = 9 (wtconv_bwd9.hip).
hipError_t launch_backward_k9(wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s);
hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s);
hipError_t launch_grad(int k, wtconv_dtype dt, const GradArgs& a, int grid, hipStream_t s);
hipError_t launch_carrier(wtconv_dtype dt, const CarrierArgs& a, hipStream_t s);
hipError_t launch_tiny(int k, wtconv_dtype dt, bool bwd, const TinyArgs& a, hipStream_t s);
// LDS of one workgroup of the tiny kernel (wtconv_tiny.hip): a staging area
// of 64 rows of 65 floats per wavefront (also the gradient scratch), the
// folded kernels of its four channels, 4 x 64 flush offsets and, in the
// backward pass, four more staging areas for the dx accumulation.
constexpr int kTinyStageFloats = 64 * 65;
inline size_t tiny_lds_bytes(int k, int L, bool bwd)
{
    return (size_t)((bwd ? 8 : 4) * kTinyStageFloats + 4 * (1 + 4 * L) * k * k + 4 * 64) * sizeof(float);
}

}  // namespace wtc
