// Kernel-gradient pass of the WTConv backward for gfx950 (MI355X).
//
// eq. (foldgrad): the gradient of a folded kernel is the correlation of the
// upstream gradient at its convolution output with that convolution's input.
// For the base path that is
//   G0[p][t] = sum over pixels of dy(y, x) * x(y + p - R, x + t - R),
// and for level l, band q, the same correlation between the level-l band-q
// coefficients of dy and of x on the ceil(H / 2^l) x ceil(W / 2^l) grid, zero
// outside it (backward through the synthesis of Algorithm 1 is the analysis,
// Section 2.2, so the upstream gradient of Z_l is the Haar pyramid of dy).
// dx is not formed here: it is the forward pass on dy with rotated kernels.
//
// One workgroup owns channel c and a run of batch planes. Per batch of PP
// resident planes:
//   1. each thread loads one 4x4 pixel block of x and of dy. x goes to LDS
//      with its Haar levels 1-2 (the zero-haloed layout of the fused kernels);
//      dy stays in registers with its level-1 (2x2 sites x 4 bands) and
//      level-2 (one site) butterflies;
//   2. base correlation of the thread's dy block with the x window around it;
//      the deeper x levels by the butterfly in LDS;
//   3. dy levels 1-2 written to a compact pyramid (level 1 over the x plane,
//      which is not read any more, when it fits there), deeper dy levels by the
//      butterfly;
//   4. level correlations, one band per wavefront: level 1 over T x T site
//      tiles into per-lane registers, level 2 row by row into per-lane
//      registers, deeper levels row by row into LDS.
// The sums stay in registers across the workgroup's planes and are reduced
// once, in a fixed order, into the workgroup's partials (the layout of the
// fused backward, so the same finalize applies). Both pyramids are
// unnormalised (2^l x the orthonormal coefficients); the finalize removes the
// resulting 4^l exactly.
#include "wtconv_fused.h"

namespace wtc {
namespace {

// T x T consecutive-row tile of a compact array (row pitch a multiple of 4,
// i0 a multiple of T), read with 16- or 8-byte loads.
template <int T>
DEV void load_tile(const float* __restrict__ p, int pitch, int j0, int i0, float (&v)[T][T])
{
#pragma unroll
    for (int r = 0; r < T; ++r) {
        const float* row = p + (j0 + r) * pitch + i0;
        if constexpr (T == 4) {
            const float4 f = *reinterpret_cast<const float4*>(row);
            v[r][0] = f.x, v[r][1] = f.y, v[r][2] = f.z, v[r][3] = f.w;
        } else if constexpr (T == 2) {
            const float2 f = *reinterpret_cast<const float2*>(row);
            v[r][0] = f.x, v[r][1] = f.y;
        } else {
            v[r][0] = row[0];
        }
    }
}

// Compact dy level of a plane region.
struct DyLevel {
    int off, pitch, band;
};

// Level correlation of band q over T x T site tiles of every resident plane:
//   acc[p][t] += sum over sites s of dY(s) * X(s + (p - R, t - R)),
// dY from the compact dy pyramid, X from the zero-haloed x pyramid.
// RGN: only the sites [m0, m1) x [m0, m1) of the region's grid count (the
// tile's own); the dy values of the others are taken as zero.
template <int K, int T, bool RGN>
DEV void grad_band_tiles(const float* __restrict__ region0, int stride, const LevelGeom& xl, DyLevel dl, int q,
                         int np, float (&acc)[K * K], int lane, int m0, int m1)
{
    const int tx = xl.ew / T;
    const int per = tx * (xl.eh / T);
    for (int it = lane; it < np * per; it += 64) {
        const TileIdx ti = tile_at(it, per, xl.r_tper, tx, xl.r_tx, T);
        const float* base = region0 + ti.p * stride;
        float ctr[T][T];
        load_tile<T>(base + dl.off + q * dl.band, dl.pitch, ti.j0, ti.i0, ctr);
        if constexpr (RGN) {
#pragma unroll
            for (int r = 0; r < T; ++r)
#pragma unroll
                for (int c = 0; c < T; ++c) {
                    const int j = ti.j0 + r, i = ti.i0 + c;
                    if (j < m0 || j >= m1 || i < m0 || i >= m1) ctr[r][c] = 0.f;
                }
        }
        corr_tile<K, T>(base + xl.off + q * xl.band, xl.pitch, ti.j0, ti.i0, ctr, acc);
    }
}

template <int K, bool RGN = false>
DEV void grad_band(const float* region0, int stride, const LevelGeom& xl, DyLevel dl, int q, int np,
                   float (&acc)[K * K], int lane, int m0 = 0, int m1 = 0)
{
    if (xl.T == 4)
        grad_band_tiles<K, 4, RGN>(region0, stride, xl, dl, q, np, acc, lane, m0, m1);
    else if (xl.T == 2)
        grad_band_tiles<K, 2, RGN>(region0, stride, xl, dl, q, np, acc, lane, m0, m1);
    else
        grad_band_tiles<K, 1, RGN>(region0, stride, xl, dl, q, np, acc, lane, m0, m1);
}

// One CW-site chunk of a site row for the row-wise correlation below:
//   acc[t] += sum_i dY[i] * X[i + t] (X read from its array column i0 - R).
template <int K, int CW>
DEV void grad_row_chunk(const float* __restrict__ dr, const float* __restrict__ xr, float (&acc)[K])
{
    constexpr int R = K / 2;
    constexpr int NX = ceil4c(CW + 2 * R);
    float d[CW], xv[NX];
#pragma unroll
    for (int v = 0; v < CW / 4; ++v) {
        const float4 f = reinterpret_cast<const float4*>(dr)[v];
        d[4 * v] = f.x, d[4 * v + 1] = f.y, d[4 * v + 2] = f.z, d[4 * v + 3] = f.w;
    }
#pragma unroll
    for (int v = 0; v < NX / 4; ++v) {
        const float4 f = reinterpret_cast<const float4*>(xr)[v];
        xv[4 * v] = f.x, xv[4 * v + 1] = f.y, xv[4 * v + 2] = f.z, xv[4 * v + 3] = f.w;
    }
#pragma unroll
    for (int i = 0; i < CW; ++i)
#pragma unroll
        for (int t = 0; t < K; ++t) acc[t] = __builtin_fmaf(d[i], xv[i + t], acc[t]);
}

// Level correlation of band q of a deep level, by rows: lane (tap row p, row
// group rg) accumulates into acc the K sums G[p][0..K-1] over the site rows
// rg, rg + NG, ... of the list of every resident plane's rows, walking each
// row in chunks of row_chunk(w) sites; sites past the grid width are zero on
// both sides.
// Lanes past the K tap rows read a valid row; their sums are dropped.
template <int K>
constexpr int rows_lanes() { return row_group_lanes(K); }  // lanes per row group

template <int K>
DEV void grad_rows_acc(const float* __restrict__ region0, int stride, const LevelGeom& xl, DyLevel dl, int q,
                       int np, float (&acc)[K], int lane)
{
    constexpr int R = K / 2;
    constexpr int PS = rows_lanes<K>();
    constexpr int NG = 64 / PS;  // row groups
    const int p = lane & (PS - 1), rg = lane / PS;
    const int prow = p < K ? p : R;
    const int cw = row_chunk(xl.w);
    // the (plane, row) pairs of the resident planes are dealt over the row
    // groups as one flat list, so small grids keep every group busy
    const float r_h = 1.0f / (float)xl.h;
    for (int e = rg; e < np * xl.h; e += NG) {
        const int pp = fdiv(e, r_h), j = e - pp * xl.h;
        const float* dr = region0 + pp * stride + dl.off + q * dl.band + j * dl.pitch;  // site row j, column 0
        const float* xr = region0 + pp * stride + xl.off + q * xl.band + (j + prow) * xl.pitch;  // row j + p - R
        if (cw == 4) {
            grad_row_chunk<K, 4>(dr, xr, acc);
        } else if (cw == 8) {
            for (int i0 = 0; i0 < xl.w; i0 += 8) grad_row_chunk<K, 8>(dr + i0, xr + i0, acc);
        } else {
            for (int i0 = 0; i0 < xl.w; i0 += 16) grad_row_chunk<K, 16>(dr + i0, xr + i0, acc);
        }
    }
}

// The row groups' sums of grad_rows_acc added with a fixed xor tree: lane
// p < K of every row group then holds G[p][0..K-1].
template <int K>
DEV void rows_reduce(float (&acc)[K])
{
#pragma unroll
    for (int t = 0; t < K; ++t)
#pragma unroll
        for (int m = rows_lanes<K>(); m < 64; m <<= 1) acc[t] += __shfl_xor(acc[t], m, 64);
}

// A deeper level (l >= 3): this batch's sums added to one LDS slot per tap
// (only this wavefront touches the slot), so the result does not depend on
// timing.
template <int K>
DEV void grad_band_rows(const float* __restrict__ region0, int stride, const LevelGeom& xl, DyLevel dl, int q,
                        int np, float* __restrict__ slot, int lane)
{
    constexpr int PS = rows_lanes<K>();
    const int p = lane & (PS - 1), rg = lane / PS;
    float acc[K];
#pragma unroll
    for (int t = 0; t < K; ++t) acc[t] = 0.f;
    grad_rows_acc<K>(region0, stride, xl, dl, q, np, acc, lane);
    rows_reduce<K>(acc);
    if (rg == 0 && p < K) {
#pragma unroll
        for (int t = 0; t < K; ++t) slot[p * K + t] += acc[t];
    }
}

// Zero the part of a plane's x region that the block loads do not write (the
// halo ring and the tile-alignment margin). Needed when the compact dy level 1
// was stored over the x plane in the previous batch.
DEV void zero_x_ring(float* __restrict__ reg, const PlaneGeom& g, int R, float r_sw, int tid)
{
    const int zy = 4 * g.tiles_y, zx = 4 * g.tiles_x;
    const int n_top = R * g.xpitch;
    const int n_bot = (g.xrows - R - zy) * g.xpitch;
    const int sw = g.xpitch - zx;  // ring columns of a middle row
    const int n = n_top + n_bot + zy * sw;
    for (int e = tid; e < n; e += kThreads) {
        int pos;
        if (e < n_top) {
            pos = e;
        } else if (e < n_top + n_bot) {
            pos = (R + zy) * g.xpitch + (e - n_top);
        } else {
            const int k = e - n_top - n_bot;
            const int row = fdiv(k, r_sw), col = k - row * sw;
            pos = (R + row) * g.xpitch + (col < R ? col : zx + col);
        }
        reg[pos] = 0.f;
    }
}

// The level-M (M = 1, 2) raw LL carrier sites of one 4x4 pixel block at
// (y0, x0) of a plane: 2^-M times each 2^M x 2^M block sum (pixels outside the
// plane are the zeros the block loads hold), summed in the carrier kernel's
// order (pairs within a row, then rows in order) and rounded once to the
// storage type; sites past the H1 x W1 grid are not written.
template <typename ST>
DEV void write_carrier(ST* __restrict__ out, int H1, int W1, int M, int y0, int x0, const float (&v)[4][4])
{
    if (M == 1) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int j = (y0 >> 1) + a, i = (x0 >> 1) + b;
                if (j < H1 && i < W1) {
                    const float s = (v[2 * a][2 * b] + v[2 * a][2 * b + 1]) + (v[2 * a + 1][2 * b] + v[2 * a + 1][2 * b + 1]);
                    out[(long)j * W1 + i] = from_f32<ST>(__builtin_ldexpf(s, -1));
                }
            }
    } else {
        const int j = y0 >> 2, i = x0 >> 2;
        if (j < H1 && i < W1) {
            float s = 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) s += (v[r][0] + v[r][1]) + (v[r][2] + v[r][3]);
            out[(long)j * W1 + i] = from_f32<ST>(__builtin_ldexpf(s, -2));
        }
    }
}

// At least three waves per SIMD (168 VGPRs) for k <= 5: with three
// workgroups per CU (the LDS budget of the planner) each SIMD then holds one
// wavefront of each. k = 7 keeps two; at k = 9 the 2 x 81 per-lane sums
// alone need most of a wavefront's 256 VGPRs, so one wavefront per SIMD may
// use the accumulation registers too.
template <int K>
constexpr int grad_waves_per_simd() { return K <= 5 ? 3 : (K <= 7 ? 2 : 1); }

// MR: planes with more 4x4 blocks than threads, one resident plane, block
// rounds (a separate instantiation keeps the one-round kernel's registers).
// DR: L >= 4; levels 3..5 keep their sums in registers too (another 3k per
// lane, an instantiation of its own so that shallower pyramids keep the
// smaller register budget).
// RGN: region mode (one resident region, L = 1; see GradArgs); with MR its
// blocks take several rounds (k = 7 and 9: 72 x 72 regions).
template <int K, typename ST, bool MR, bool DR, bool RGN>
__global__ void __launch_bounds__(kThreads, grad_waves_per_simd<K>()) grad_kernel(const GradArgs a)
{
    constexpr int R = K / 2, KK = K * K;
    static_assert(!RGN || !DR, "region mode takes level 1 only");
    extern __shared__ float4 lds4[];
    float* lds = reinterpret_cast<float*>(lds4);

    const PlaneGeom& g = a.g;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int C = a.C;
    const int c = blockIdx.x % C;
    const int ct = blockIdx.x / C;  // chunk (region mode: chunk * tiles + tile)
    const int ntiles = RGN ? a.rg_ntx * a.rg_nty : 1;
    const int chunk = ct / ntiles;
    const int tile = ct - chunk * ntiles;
    const int b_begin = chunk * a.nb;
    const int b_end = min(a.B, b_begin + a.nb);
    const int L = g.L;
    // region mode: origin of the region in the real plane (multiples of 4)
    const int oy = RGN ? (tile / a.rg_ntx) * a.rg_T - a.rg_h : 0;
    const int ox = RGN ? (tile % a.rg_ntx) * a.rg_T - a.rg_h : 0;
    const int PH = RGN ? a.real_H : g.H, PW = RGN ? a.real_W : g.W;  // the real plane
    const long HW = (long)PH * PW;
    const bool skip_base = a.skip_base != 0;
    const int vw = a.vec_ok == 0 ? 1 : ((PW % 4) == 0 ? 4 : ((PW % 2) == 0 ? 2 : 1));  // row vector width
    const bool alias1 = L >= 1 && a.dy_off[1] == 0;  // dy level 1 is stored over the x plane
    const int q = wave;                              // the subband this wavefront correlates

    // LDS: [deep-level kernel-gradient sums][plane regions]
    constexpr int RL = grad_reg_levels(DR);  // levels whose sums stay in registers
    const int gc_floats = L > RL ? ceil4c((L - RL) * 4 * KK) : 0;
    float* gco = lds;
    float* planes = lds + gc_floats;
    const int stride = a.stride;

    const ST* xs = reinterpret_cast<const ST*>(a.x);
    const ST* dys = reinterpret_cast<const ST*>(a.dy);

    for (int i = tid; i < a.lds_floats / 4; i += kThreads) lds4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();

    // kernel-gradient sums: base and level 1 per lane over its tiles; level 2
    // per lane (tap row, row group) over its rows (the row-wise correlation)
    constexpr int KD = DR ? K : 1;
    float g0[KK], g1[KK], g2[K], g3[KD], g4[KD], g5[KD];
#pragma unroll
    for (int t = 0; t < KK; ++t) g0[t] = g1[t] = 0.f;
#pragma unroll
    for (int t = 0; t < K; ++t) g2[t] = 0.f;
#pragma unroll
    for (int t = 0; t < KD; ++t) g3[t] = g4[t] = g5[t] = 0.f;
    float gdy = 0.f;  // sum of dy over the workgroup's pixels (bias gradient)

    const int per = g.tiles_x * g.tiles_y;
    for (int b0 = b_begin; b0 < b_end; b0 += a.PP) {
        const int np = min(a.PP, b_end - b0);
        // Per-thread LDS addresses depend only on the thread index; taking it
        // through an opaque copy inside this loop keeps the compiler from
        // hoisting them out of the loop, which would hold them across it next
        // to the kernel-gradient sums and spill them (k <= 5; at k = 7
        // the sums alone nearly fill the registers and hoisting spills less).
        int tl = threadIdx.x;
        if constexpr (K <= 5) asm volatile("" : "+v"(tl));
        const int ll = tl & 63;
        // dy levels 1-2 of one block -> the compact pyramid
        auto dy_levels = [&](const TileIdx& ti, const float (&dyb)[4][4]) {
            float* reg = planes + ti.p * stride;
            float d1[2][2][4], d2[4];
#pragma unroll
            for (int ya = 0; ya < 2; ++ya)
#pragma unroll
                for (int xb = 0; xb < 2; ++xb)
                    butterfly(dyb[2 * ya][2 * xb], dyb[2 * ya][2 * xb + 1], dyb[2 * ya + 1][2 * xb],
                              dyb[2 * ya + 1][2 * xb + 1], d1[ya][xb]);
            butterfly(d1[0][0][0], d1[0][1][0], d1[1][0][0], d1[1][1][0], d2);
            if (L >= 1) {
#pragma unroll
                for (int bq = 0; bq < 4; ++bq)
#pragma unroll
                    for (int ya = 0; ya < 2; ++ya) {
                        const float pair[2] = {d1[ya][0][bq], d1[ya][1][bq]};
                        st_row<true, 2>(reg + a.dy_off[1] + bq * a.dy_band[1] + ((ti.j0 >> 1) + ya) * a.dy_pitch[1] +
                                            (ti.i0 >> 1),
                                        pair);
                    }
            }
            if (L >= 2) {
                float* o = reg + a.dy_off[2] + (ti.j0 >> 2) * a.dy_pitch[2] + (ti.i0 >> 2);
#pragma unroll
                for (int bq = 0; bq < 4; ++bq) o[bq * a.dy_band[2]] = d2[bq];
            }
        };
        // base correlation of one block (dy centre, x window) and its dy sum
        // region mode: the blocks of the tile's own pixels (rg_h and rg_T
        // are multiples of 4, so a block is wholly inside or outside)
        auto is_inner = [&](const TileIdx& ti) {
            return !RGN || (ti.j0 >= a.rg_h && ti.j0 < a.rg_h + a.rg_T && ti.i0 >= a.rg_h && ti.i0 < a.rg_h + a.rg_T);
        };
        auto base_corr = [&](const TileIdx& ti, const float (&dyb)[4][4]) {
            corr_tile<K, 4>(planes + ti.p * stride, g.xpitch, ti.j0, ti.i0, dyb, g0);
#pragma unroll
            for (int r = 0; r < 4; ++r) gdy += (dyb[r][0] + dyb[r][1]) + (dyb[r][2] + dyb[r][3]);
        };

        if constexpr (!MR) {
            const bool mine = tl < np * per;  // at most one block per thread (planned on the host)
            const TileIdx ti = tile_at(mine ? tl : 0, per, g.r_tiles, g.tiles_x, g.r_tiles_x, 4);
            const bool inner = is_inner(ti);

            // 1. x block -> LDS with its levels 1-2; dy block in registers
            if (alias1 && b0 != b_begin)
                for (int p = 0; p < np; ++p) zero_x_ring(planes + p * stride, g, R, a.r_ring, tl);
            float dyb[4][4];
            if (mine) {
                const long plane = (long)(b0 + ti.p) * C + c;
                float v[4][4];
                fetch_block<ST>(xs + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, v);
                store_block<K>(v, planes + ti.p * stride, g, ti.j0, ti.i0);
                fetch_block<ST>(dys + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, dyb);
                if (a.cx && inner) {
                    const long co = plane * a.cH * a.cW;
                    write_carrier<ST>(reinterpret_cast<ST*>(a.cx) + co, a.cH, a.cW, a.cm, oy + ti.j0, ox + ti.i0, v);
                    write_carrier<ST>(reinterpret_cast<ST*>(a.cdy) + co, a.cH, a.cW, a.cm, oy + ti.j0, ox + ti.i0,
                                      dyb);
                }
            }
            __syncthreads();

            // 2. base correlation; x level 3
            if (mine && inner && !skip_base) base_corr(ti, dyb);
            if (L >= 3) {
                const LevelGeom& lg = g.lv[3];
                const LevelGeom& lp = g.lv[2];
                analysis_level(planes + lp.off, lp.pitch, planes + lg.off, lg, R, np, stride, tl);
            }
            __syncthreads();

            // 3. dy levels 1-2 -> compact pyramid (and a clean x-plane tail
            //    for the deeper dy levels stored there)
            for (int i = a.tail0 + tl; i < a.tail1; i += kThreads) planes[i] = 0.f;
            if (mine) dy_levels(ti, dyb);
        } else {
            // One resident plane with more 4x4 blocks than threads: each phase
            // walks the block rounds and fetches its dy blocks itself (they
            // cannot stay in registers across rounds). Every base correlation
            // reads the x plane before the barrier after which dy level 1 may
            // be stored over it.
            if (alias1 && b0 != b_begin) zero_x_ring(planes, g, R, a.r_ring, tl);
            const long plane = (long)b0 * C + c;
            const long co = plane * a.cH * a.cW;  // region mode: the plane's level-1 carriers
            for (int it = tl; it < per; it += kThreads) {
                const TileIdx ti = tile_at(it, per, g.r_tiles, g.tiles_x, g.r_tiles_x, 4);
                float v[4][4];
                fetch_block<ST>(xs + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, v);
                store_block<K>(v, planes, g, ti.j0, ti.i0);
                if (RGN && a.cx && is_inner(ti))
                    write_carrier<ST>(reinterpret_cast<ST*>(a.cx) + co, a.cH, a.cW, a.cm, oy + ti.j0, ox + ti.i0, v);
            }
            __syncthreads();
            if (!skip_base) {
                for (int it = tl; it < per; it += kThreads) {
                    const TileIdx ti = tile_at(it, per, g.r_tiles, g.tiles_x, g.r_tiles_x, 4);
                    if (!is_inner(ti)) continue;
                    float dyb[4][4];
                    fetch_block<ST>(dys + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, dyb);
                    base_corr(ti, dyb);
                }
            }
            if (L >= 3) {
                const LevelGeom& lg = g.lv[3];
                const LevelGeom& lp = g.lv[2];
                analysis_level(planes + lp.off, lp.pitch, planes + lg.off, lg, R, np, stride, tl);
            }
            __syncthreads();
            for (int i = a.tail0 + tl; i < a.tail1; i += kThreads) planes[i] = 0.f;
            for (int it = tl; it < per; it += kThreads) {
                const TileIdx ti = tile_at(it, per, g.r_tiles, g.tiles_x, g.r_tiles_x, 4);
                float dyb[4][4];
                fetch_block<ST>(dys + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, dyb);
                if (RGN && a.cx && is_inner(ti))
                    write_carrier<ST>(reinterpret_cast<ST*>(a.cdy) + co, a.cH, a.cW, a.cm, oy + ti.j0, ox + ti.i0,
                                      dyb);
                dy_levels(ti, dyb);
            }
        }
        if (L >= 4) {
            const LevelGeom& lg = g.lv[4];
            const LevelGeom& lp = g.lv[3];
            analysis_level(planes + lp.off, lp.pitch, planes + lg.off, lg, R, np, stride, tl);
        }
        __syncthreads();

        // deeper levels: dy level l (compact, from dy level l - 1) and x level l + 2
        for (int l = 3; l <= L; ++l) {
            LevelGeom dg = g.lv[l];
            dg.pitch = a.dy_pitch[l];
            dg.band = a.dy_band[l];
            analysis_level(planes + a.dy_off[l - 1], a.dy_pitch[l - 1], planes + a.dy_off[l], dg, 0, np, stride, tl);
            if (l + 2 <= L) {
                const LevelGeom& lg = g.lv[l + 2];
                const LevelGeom& lp = g.lv[l + 1];
                analysis_level(planes + lp.off, lp.pitch, planes + lg.off, lg, R, np, stride, tl);
            }
            __syncthreads();
        }

        // 4. level correlations, band q per wavefront: level 1 over register
        //    tiles, level 2 row by row into per-lane sums, the deeper levels
        //    row by row into their LDS slots
        for (int l = 1; l <= L; ++l) {
            const LevelGeom& xl = g.lv[l];
            const DyLevel dl = {a.dy_off[l], a.dy_pitch[l], a.dy_band[l]};
            if (l == 1)
                grad_band<K, RGN>(planes, stride, xl, dl, q, np, g1, ll, a.rg_h >> 1, (a.rg_h + a.rg_T) >> 1);
            else if (l == 2)
                grad_rows_acc<K>(planes, stride, xl, dl, q, np, g2, ll);
            else if (DR && l <= RL) {
                if constexpr (DR) {
                    if (l == 3)
                        grad_rows_acc<K>(planes, stride, xl, dl, q, np, g3, ll);
                    else if (l == 4)
                        grad_rows_acc<K>(planes, stride, xl, dl, q, np, g4, ll);
                    else
                        grad_rows_acc<K>(planes, stride, xl, dl, q, np, g5, ll);
                }
            } else {
                grad_band_rows<K>(planes, stride, xl, dl, q, np, gco + ((l - RL - 1) * 4 + q) * KK, ll);
            }
        }
        __syncthreads();
    }

    // fixed-order reduction of the workgroup's sums into its partials
    const int NP = partial_floats_per_channel(K, L);
    float* red = planes;  // the plane regions are free now
#pragma unroll
    for (int t = 0; t < KK; ++t) {
        const float v0 = wave_sum(g0[t]);
        const float v1 = wave_sum(g1[t]);
        if (lane == 0) {
            red[wave * KK + t] = v0;
            red[(kWaves + wave) * KK + t] = v1;
        }
    }
    rows_reduce<K>(g2);
    if constexpr (DR) {
        rows_reduce<K>(g3);
        rows_reduce<K>(g4);
        rows_reduce<K>(g5);
    }
    {
        constexpr int PS = rows_lanes<K>();
        const int p = lane & (PS - 1);
        if (lane < PS && p < K) {
#pragma unroll
            for (int t = 0; t < K; ++t) {
                red[(2 * kWaves + wave) * KK + p * K + t] = g2[t];
                if constexpr (DR) {
                    red[(3 * kWaves + wave) * KK + p * K + t] = g3[t];
                    red[(4 * kWaves + wave) * KK + p * K + t] = g4[t];
                    red[(5 * kWaves + wave) * KK + p * K + t] = g5[t];
                }
            }
        }
    }
    const float vdy = wave_sum(gdy);
    if (lane == 0) red[(RL + 1) * kWaves * KK + wave] = vdy;
    __syncthreads();
    float* dst = a.partial + ((long)ct * C + c) * NP;
    for (int t = tid; t < KK; t += kThreads) dst[t] = ((red[t] + red[KK + t]) + red[2 * KK + t]) + red[3 * KK + t];
    if (tid == 0) {
        const float* r = red + (RL + 1) * kWaves * KK;
        dst[NP - 1] = ((r[0] + r[1]) + r[2]) + r[3];
    }
    // levels 1..RL: band q's sums came from wavefront q; deeper levels from the slots
    for (int i = tid; i < 4 * KK * min(L, RL); i += kThreads) dst[KK + i] = red[kWaves * KK + i];
    for (int i = tid; i < 4 * KK * (L - RL); i += kThreads) dst[KK + 4 * RL * KK + i] = gco[i];
}

template <int K, typename ST, bool MR, bool DR, bool RGN = false>
hipError_t launch_grad_v(const GradArgs& a, int grid, hipStream_t s)
{
    const size_t bytes = (size_t)a.lds_floats * sizeof(float);
    static std::atomic<unsigned long long> lds_done{0};
    const hipError_t e = allow_full_lds(reinterpret_cast<const void*>(&grad_kernel<K, ST, MR, DR, RGN>), lds_done);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((grad_kernel<K, ST, MR, DR, RGN>), dim3(grid), dim3(kThreads), bytes, s, a);
    return hipGetLastError();
}

template <int K, typename ST>
hipError_t launch_grad_t(const GradArgs& a, int grid, hipStream_t s)
{
    if (a.rg_ntx > 0) {
        // one resident region, level 1 only (planned on the host)
        if (a.PP != 1 || a.g.L != 1) return hipErrorInvalidValue;
        return a.rounds > 1 ? launch_grad_v<K, ST, true, false, true>(a, grid, s)
                            : launch_grad_v<K, ST, false, false, true>(a, grid, s);
    }
    if (a.rounds > 1) {
        if (a.PP != 1) return hipErrorInvalidValue;  // block rounds need one resident plane
        return a.g.L >= 4 ? launch_grad_v<K, ST, true, true>(a, grid, s) : launch_grad_v<K, ST, true, false>(a, grid, s);
    }
    return a.g.L >= 4 ? launch_grad_v<K, ST, false, true>(a, grid, s) : launch_grad_v<K, ST, false, false>(a, grid, s);
}

}  // namespace

hipError_t launch_grad(int k, wtconv_dtype dt, const GradArgs& a, int grid, hipStream_t s)
{
#define WTC_GRAD_CASE(KV)                                                         \
    case KV:                                                                      \
        switch (dt) {                                                             \
            case WTCONV_F32: return launch_grad_t<KV, float>(a, grid, s);         \
            case WTCONV_BF16: return launch_grad_t<KV, uint16_t>(a, grid, s);     \
            case WTCONV_F16: return launch_grad_t<KV, _Float16>(a, grid, s);      \
        }                                                                         \
        break;
    switch (k) {
        WTC_GRAD_CASE(1)
        WTC_GRAD_CASE(3)
        WTC_GRAD_CASE(5)
        WTC_GRAD_CASE(7)
        WTC_GRAD_CASE(9)
    }
#undef WTC_GRAD_CASE
    return hipErrorInvalidValue;
}

}  // namespace wtc
