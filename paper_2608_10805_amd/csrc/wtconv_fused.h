// Fused WTConv kernels for gfx950 (MI355X): device building blocks and the
// fused kernel template, instantiated by wtconv_fwd.hip (forward) and
// wtconv_bwd.hip (backward). Internal; not part of the public ABI.
//
// One workgroup owns one channel c and a run of batch planes of that channel.
// Per plane it:
//   1. reads the plane from HBM once (coalesced, vectorised) into a zero-
//      haloed fp32 LDS array;
//   2. builds the whole Haar pyramid on chip: the butterfly of eq. (butterfly)
//      (Section 4.1) recomputed in LDS, without the 1/2 factors (they are
//      powers of two and are folded into the kernels, see below);
//   3. filters every subband of every level with its depthwise k x k kernel,
//      one band per wavefront (so each wavefront's 25 taps sit in scalar
//      registers), writing the filtered coefficients over the unfiltered ones;
//   4. forms each 4x4 output tile as the base convolution plus the
//      closed-form bit-indexed synthesis of Proposition 2 (Section 4.2) and
//      stores it to HBM once.
// Scales are folded into the kernels (eq. fold, Section 4.3): the base kernel
// becomes s0 * W0 and the level-l kernel s_l * W_l * 4^-l, where 4^-l absorbs
// the 2^-l of the unnormalised analysis pyramid and the 2^-l of Proposition 2.
// Multiplying by a power of two is exact, so only the s * W product rounds.
//
// The backward kernel runs the same pipeline on dy with the kernels rotated
// by 180 degrees (the Haar transform is symmetric and self-inverse, Section
// 2.2, so backward through synthesis is analysis and vice versa), writes dx,
// and accumulates the kernel gradients of eq. (foldgrad): correlations of the
// dy pyramid with the x pyramid (and of dy with x for the base path), held in
// registers across the workgroup's planes and reduced once per workgroup in a
// fixed order. A second small kernel sums the per-workgroup partials in a fixed
// order and unfolds them into dW and d(scale).
#pragma once

#include <stdint.h>

#include "wtconv_device.h"
#include "wtconv_internal.h"

namespace wtc {
namespace {

// Levels whose kernel gradient is accumulated in per-lane registers across a
// workgroup's planes (two in the single-round variant, which has the register
// room, one otherwise); deeper levels accumulate row by row in LDS.
template <bool ONE>
constexpr int reg_levels() { return ONE ? 2 : 1; }

// n / d for 0 <= n < 2^20 from rinv = fp32(1 / d): the exact quotient
// (n + 0.5) / d lies at least 0.5 / d away from an integer, while the two
// fp32 roundings perturb it by at most about (n / d) * 2^-23, far less.
DEV int fdiv(int n, float rinv) { return (int)(((float)n + 0.5f) * rinv); }

constexpr int ceil4c(int v) { return (v + 3) / 4 * 4; }
constexpr int ceil2c(int v) { return (v + 1) / 2 * 2; }

// Width (floats) read per window row for a T-wide tile: whole vectors.
template <int K, int T>
struct Win {
    static constexpr int R = K / 2;
    static constexpr int N = T + 2 * R;                       // taps touched
    static constexpr int NA = T == 4 ? ceil4c(N) : (T == 2 ? ceil2c(N) : N);  // loaded
};

// Load NA consecutive floats starting at an address aligned to the vector
// width used for tile edge T (16 bytes for T = 4, 8 bytes for T = 2).
template <int K, int T>
DEV void load_row(const float* __restrict__ p, float (&row)[Win<K, T>::NA])
{
    constexpr int NA = Win<K, T>::NA;
    if constexpr (T == 4) {
#pragma unroll
        for (int v = 0; v < NA / 4; ++v) {
            const float4 f = reinterpret_cast<const float4*>(p)[v];
            row[4 * v + 0] = f.x;
            row[4 * v + 1] = f.y;
            row[4 * v + 2] = f.z;
            row[4 * v + 3] = f.w;
        }
    } else if constexpr (T == 2) {
#pragma unroll
        for (int v = 0; v < NA / 2; ++v) {
            const float2 f = reinterpret_cast<const float2*>(p)[v];
            row[2 * v + 0] = f.x;
            row[2 * v + 1] = f.y;
        }
    } else {
#pragma unroll
        for (int v = 0; v < NA; ++v) row[v] = p[v];
    }
}

// Two consecutive storage elements -> fp32 (one 8-byte or 4-byte load).
DEV void load2(const float* __restrict__ p, float (&v)[2])
{
    const float2 f = *reinterpret_cast<const float2*>(p);
    v[0] = f.x;
    v[1] = f.y;
}
DEV void load2(const uint16_t* __restrict__ p, float (&v)[2])
{
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    v[0] = __uint_as_float(u << 16);
    v[1] = __uint_as_float(u & 0xffff0000u);
}
DEV void load2(const _Float16* __restrict__ p, float (&v)[2])
{
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    _Float16 h[2];
    __builtin_memcpy(h, &u, 4);
    v[0] = (float)h[0];
    v[1] = (float)h[1];
}

// Four consecutive storage elements -> fp32 (one 16-byte or 8-byte load).
DEV void load4(const float* __restrict__ p, float (&v)[4])
{
    const float4 f = *reinterpret_cast<const float4*>(p);
    v[0] = f.x;
    v[1] = f.y;
    v[2] = f.z;
    v[3] = f.w;
}
DEV void load4(const uint16_t* __restrict__ p, float (&v)[4])
{
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    v[0] = __uint_as_float(u.x << 16);
    v[1] = __uint_as_float(u.x & 0xffff0000u);
    v[2] = __uint_as_float(u.y << 16);
    v[3] = __uint_as_float(u.y & 0xffff0000u);
}
DEV void load4(const _Float16* __restrict__ p, float (&v)[4])
{
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    _Float16 h[4];
    __builtin_memcpy(h, &u, 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (float)h[i];
}

// Store N consecutive floats to LDS; with PAIRS the address is 8-byte aligned
// and pairs go out as 64-bit stores.
template <bool PAIRS, int N>
DEV void st_row(float* __restrict__ p, const float* v)
{
    if constexpr (PAIRS && N % 2 == 0) {
#pragma unroll
        for (int i = 0; i < N; i += 2) *reinterpret_cast<float2*>(p + i) = make_float2(v[i], v[i + 1]);
    } else {
#pragma unroll
        for (int i = 0; i < N; ++i) p[i] = v[i];
    }
}

// ----------------------------------------------------------------------------
// 1. one 4x4 pixel block: HBM -> LDS, plus Haar levels 1 and 2 in registers
//    (the block holds exactly four level-1 sites and one level-2 site).
//    Pixels outside the plane are zero (zero extension). Ragged sites beyond
//    the level grids are written as the zeros they are.
// ----------------------------------------------------------------------------
// A 4x4 pixel block whose top-left pixel is (y0, x0) of an H x W plane; pixels
// outside the plane (including negative coordinates) read as zero. vw is the
// vector width the plane allows: 4 (W % 4 == 0), 2 (W even: a pair starting at
// an even column lies wholly inside or wholly outside the plane) or 1; x0 is a
// multiple of 4.
template <typename T>
DEV void fetch_block(const T* __restrict__ src, int H, int W, int y0, int x0, int vw, float (&v)[4][4])
{
    if (vw == 4 && y0 >= 0 && x0 >= 0 && y0 + 4 <= H && x0 + 4 <= W) {
#pragma unroll
        for (int r = 0; r < 4; ++r) load4(src + (long)(y0 + r) * W + x0, v[r]);
    } else if (vw == 2) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int y = y0 + r;
#pragma unroll
            for (int c = 0; c < 4; c += 2) {
                const int x = x0 + c;
                if (y >= 0 && y < H && x >= 0 && x < W) {
                    float pr[2];
                    load2(src + (long)y * W + x, pr);
                    v[r][c] = pr[0];
                    v[r][c + 1] = pr[1];
                } else {
                    v[r][c] = v[r][c + 1] = 0.f;
                }
            }
        }
    } else if (y0 >= 0 && x0 >= 0 && y0 + 4 <= H && x0 + 4 <= W) {
        // a block inside the plane: element loads, no bounds checks
        const T* p = src + (long)y0 * W + x0;
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int c = 0; c < 4; ++c) v[r][c] = to_f32(p[(long)r * W + c]);
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int y = y0 + r, x = x0 + c;
                v[r][c] = (y >= 0 && y < H && x >= 0 && x < W) ? to_f32(src[(long)y * W + x]) : 0.f;
            }
    }
}

template <int K>
DEV void store_block(const float (&v)[4][4], float* __restrict__ reg, const PlaneGeom& g, int y0, int x0)
{
    constexpr int R = K / 2;
    constexpr bool PAIRS = (R % 2) == 0;  // interior origin keeps 8-byte alignment
#pragma unroll
    for (int r = 0; r < 4; ++r) st_row<PAIRS, 4>(reg + (y0 + r + R) * g.xpitch + x0 + R, v[r]);
    if (g.L < 1) return;
    const LevelGeom& l1 = g.lv[1];
    float c1[2][2][4];  // [a][b][band]
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
            butterfly(v[2 * a][2 * b], v[2 * a][2 * b + 1], v[2 * a + 1][2 * b], v[2 * a + 1][2 * b + 1], c1[a][b]);
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            const float pair[2] = {c1[a][0][q], c1[a][1][q]};
            st_row<PAIRS, 2>(reg + l1.off + q * l1.band + ((y0 >> 1) + a + R) * l1.pitch + (x0 >> 1) + R, pair);
        }
    if (g.L < 2) return;
    const LevelGeom& l2 = g.lv[2];
    float c2[4];
    butterfly(c1[0][0][0], c1[0][1][0], c1[1][0][0], c1[1][1][0], c2);
    float* o = reg + l2.off + ((y0 >> 2) + R) * l2.pitch + (x0 >> 2) + R;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q * l2.band] = c2[q];
}

// One 4x4 pixel block: HBM -> LDS, plus Haar levels 1 and 2 in registers (the
// block holds exactly four level-1 sites and one level-2 site). Pixels outside
// the plane are zero (zero extension); ragged sites beyond the level grids are
// written as the zeros they are.
template <int K, typename T>
DEV void load_block(const T* __restrict__ src, float* __restrict__ reg, const PlaneGeom& g, int y0, int x0,
                    int vw)
{
    float v[4][4];
    fetch_block<T>(src, g.H, g.W, y0, x0, vw, v);
    store_block<K>(v, reg, g, y0, x0);
}

// ----------------------------------------------------------------------------
// 2. one analysis level, all resident planes: unnormalised butterfly
//    (LL, LH, HL, HH) = (a+b+c+d, a+b-c-d, a-b+c-d, a-b-c+d), eq. (butterfly)
//    without the 1/2. Zero extension comes from the zero halo / ragged rows.
// ----------------------------------------------------------------------------
DEV void analysis_level(const float* __restrict__ src, int sp, float* __restrict__ dst, const LevelGeom& lg,
                        int R, int np, int stride, int tid)
{
    const int per = lg.h * lg.w;
    for (int e = tid; e < np * per; e += kThreads) {
        const int p = fdiv(e, lg.r_hw);
        const int r = e - p * per;
        const int j = fdiv(r, lg.r_w);
        const int i = r - j * lg.w;
        const float* s = src + p * stride + (2 * j + R) * sp + 2 * i + R;
        float co[4];
        butterfly(s[0], s[1], s[sp], s[sp + 1], co);
        float* o = dst + p * stride + (j + R) * lg.pitch + i + R;
        o[0] = co[0];
        o[lg.band] = co[1];
        o[2 * lg.band] = co[2];
        o[3 * lg.band] = co[3];
    }
}

// ----------------------------------------------------------------------------
// depthwise "same" correlation of a T x T tile of sites (or pixels):
//   out[oy][ox] = sum_{p,t} w[p][t] * src[j0+oy+p-R][i0+ox+t-R]
// `band` points at the array origin (the top-left halo element).
// ----------------------------------------------------------------------------
template <int K, int T>
DEV void conv_tile(const float* __restrict__ band, int pitch, int j0, int i0, const float (&w)[K * K],
                   float (&out)[T][T])
{
    constexpr int N = Win<K, T>::N;
#pragma unroll
    for (int oy = 0; oy < T; ++oy)
#pragma unroll
        for (int ox = 0; ox < T; ++ox) out[oy][ox] = 0.f;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float row[Win<K, T>::NA];
        load_row<K, T>(band + (j0 + r) * pitch + i0, row);
#pragma unroll
        for (int oy = 0; oy < T; ++oy) {
            const int p = r - oy;
            if (p < 0 || p >= K) continue;
#pragma unroll
            for (int ox = 0; ox < T; ++ox)
#pragma unroll
                for (int t = 0; t < K; ++t)  // the first term is a product (no zeroed accumulator)
                    out[oy][ox] = (p == 0 && t == 0) ? w[0] * row[ox]
                                                     : __builtin_fmaf(w[p * K + t], row[ox + t], out[oy][ox]);
        }
    }
}

// conv_tile that also returns the tile's own input values (the window centre).
template <int K, int T>
DEV void conv_tile_ctr(const float* __restrict__ band, int pitch, int j0, int i0, const float (&w)[K * K],
                       float (&out)[T][T], float (&ctr)[T][T])
{
    constexpr int R = K / 2, N = Win<K, T>::N;
#pragma unroll
    for (int oy = 0; oy < T; ++oy)
#pragma unroll
        for (int ox = 0; ox < T; ++ox) out[oy][ox] = 0.f;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float row[Win<K, T>::NA];
        load_row<K, T>(band + (j0 + r) * pitch + i0, row);
        if (r >= R && r < R + T) {
#pragma unroll
            for (int ox = 0; ox < T; ++ox) ctr[r - R][ox] = row[R + ox];
        }
#pragma unroll
        for (int oy = 0; oy < T; ++oy) {
            const int p = r - oy;
            if (p < 0 || p >= K) continue;
#pragma unroll
            for (int ox = 0; ox < T; ++ox)
#pragma unroll
                for (int t = 0; t < K; ++t)  // the first term is a product (no zeroed accumulator)
                    out[oy][ox] = (p == 0 && t == 0) ? w[0] * row[ox]
                                                     : __builtin_fmaf(w[p * K + t], row[ox + t], out[oy][ox]);
        }
    }
}

// Kernel-gradient correlation of one tile:
//   acc[p][t] += sum_{oy,ox} ctr[oy][ox] * src[j0+oy+p-R][i0+ox+t-R]
template <int K, int T>
DEV void corr_tile(const float* __restrict__ band, int pitch, int j0, int i0, const float (&ctr)[T][T],
                   float (&acc)[K * K])
{
    constexpr int N = Win<K, T>::N;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float row[Win<K, T>::NA];
        load_row<K, T>(band + (j0 + r) * pitch + i0, row);
#pragma unroll
        for (int oy = 0; oy < T; ++oy) {
            const int p = r - oy;
            if (p < 0 || p >= K) continue;
#pragma unroll
            for (int ox = 0; ox < T; ++ox)
#pragma unroll
                for (int t = 0; t < K; ++t) acc[p * K + t] = __builtin_fmaf(ctr[oy][ox], row[ox + t], acc[p * K + t]);
        }
    }
}

template <int K, int T>
DEV void load_center(const float* __restrict__ band, int pitch, int j0, int i0, float (&ctr)[T][T])
{
    constexpr int R = K / 2;
#pragma unroll
    for (int oy = 0; oy < T; ++oy)
#pragma unroll
        for (int ox = 0; ox < T; ++ox) ctr[oy][ox] = band[(j0 + oy + R) * pitch + i0 + ox + R];
}

// Decompose a flat tile index over (plane, tile row, tile column).
struct TileIdx {
    int p, j0, i0;
};
DEV TileIdx tile_at(int it, int per, float rper, int tx, float rtx, int T)
{
    TileIdx ti;
    ti.p = fdiv(it, rper);
    const int r = it - ti.p * per;
    const int jt = fdiv(r, rtx);
    ti.j0 = jt * T;
    ti.i0 = (r - jt * tx) * T;
    return ti;
}

// ----------------------------------------------------------------------------
// 3. filter one subband of one level in place, for all resident planes.
//    Every lane computes all of its tiles into registers first; only then are
//    the filtered values written over the unfiltered ones (one band is read
//    and written by one wavefront only, and a wavefront's LDS operations
//    complete in program order). Ragged sites outside the true grid are not
//    written, so they stay zero for the next plane.
// ----------------------------------------------------------------------------
template <int K, int T, int MAXR, bool GRAD>
DEV void filter_band_inplace(float* __restrict__ region0, const float* __restrict__ aux0, int stride,
                             const LevelGeom& lg, int q, int np, const float (&w)[K * K], float (&gacc)[K * K],
                             int lane)
{
    constexpr int R = K / 2;
    const int tx = lg.ew / T;
    const int per = tx * (lg.eh / T);
    const int total = np * per;
    float res[MAXR][T][T];
#pragma unroll
    for (int k = 0; k < MAXR; ++k) {
        const int it = lane + 64 * k;
        if (it < total) {
            const TileIdx ti = tile_at(it, per, lg.r_tper, tx, lg.r_tx, T);
            const int boff = ti.p * stride + lg.off + q * lg.band;
            if constexpr (GRAD) {
                // the kernel gradient of this band: the unfiltered tile (dZ)
                // against the partner pyramid, before the tile is overwritten
                float ctr[T][T];
                conv_tile_ctr<K, T>(region0 + boff, lg.pitch, ti.j0, ti.i0, w, res[k], ctr);
                corr_tile<K, T>(aux0 + boff, lg.pitch, ti.j0, ti.i0, ctr, gacc);
            } else {
                conv_tile<K, T>(region0 + boff, lg.pitch, ti.j0, ti.i0, w, res[k]);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < MAXR; ++k) {
        const int it = lane + 64 * k;
        if (it < total) {
            const TileIdx ti = tile_at(it, per, lg.r_tper, tx, lg.r_tx, T);
            float* band = region0 + ti.p * stride + lg.off + q * lg.band + (ti.j0 + R) * lg.pitch + ti.i0 + R;
            if (ti.j0 + T <= lg.h && ti.i0 + T <= lg.w) {
#pragma unroll
                for (int oy = 0; oy < T; ++oy) st_row<(R % 2) == 0, T>(band + oy * lg.pitch, res[k][oy]);
            } else {
#pragma unroll
                for (int oy = 0; oy < T; ++oy)
#pragma unroll
                    for (int ox = 0; ox < T; ++ox)
                        if (ti.j0 + oy < lg.h && ti.i0 + ox < lg.w) band[oy * lg.pitch + ox] = res[k][oy][ox];
            }
        }
    }
}

// Forward, single round: levels 1 and 3..L of band q in one pass over the
// wavefront, all in 4x4 site tiles. Lanes [s_l, s_l + n_l) take the n_l tiles
// of level l (level 1 first, then 3, 4, ...); every lane reads its own level's
// folded kernel from LDS and filters its tile in place once the whole
// wavefront has read its windows (levels are separate arrays, and a
// wavefront's LDS operations complete in program order).
template <int K>
DEV void filter_merged(float* __restrict__ region0, int stride, const PlaneGeom& g, const float* __restrict__ wtab,
                       int q, int np, int lane)
{
    constexpr int R = K / 2, KK = K * K;
    // this lane's level, tile index and level geometry (uniform loop, per-lane selects)
    int lvl = 0, it = 0, start = 0, off = 0, pitch = 0, band = 0, h = 0, w = 0, tx = 0, per = 0;
    float r_tper = 0.f, r_tx = 0.f;
    for (int l = 1; l <= g.L; ++l) {
        if (l == 2) continue;
        const LevelGeom& lg = g.lv[l];
        const int ltx = lg.ew / 4;
        const int n = np * ltx * (lg.eh / 4);
        if (lvl == 0 && lane < start + n) {
            lvl = l;
            it = lane - start;
            off = lg.off;
            pitch = lg.pitch;
            band = lg.band;
            h = lg.h;
            w = lg.w;
            tx = ltx;
            per = ltx * (lg.eh / 4);
            r_tper = lg.r_tper;
            r_tx = lg.r_tx;
        }
        start += n;
    }
    if (lvl == 0) return;
    float wv[KK];
    const float* wrow_p = wtab + (1 + (lvl - 1) * 4 + q) * KK;
#pragma unroll
    for (int i = 0; i < KK; ++i) wv[i] = wrow_p[i];
    const TileIdx ti = tile_at(it, per, r_tper, tx, r_tx, 4);
    float* base = region0 + ti.p * stride + off + q * band;
    float res[4][4];
    conv_tile<K, 4>(base, pitch, ti.j0, ti.i0, wv, res);
    float* dst = base + (ti.j0 + R) * pitch + ti.i0 + R;
    if (ti.j0 + 4 <= h && ti.i0 + 4 <= w) {
#pragma unroll
        for (int oy = 0; oy < 4; ++oy) st_row<(R % 2) == 0, 4>(dst + oy * pitch, res[oy]);
    } else {
#pragma unroll
        for (int oy = 0; oy < 4; ++oy)
#pragma unroll
            for (int ox = 0; ox < 4; ++ox)
                if (ti.j0 + oy < h && ti.i0 + ox < w) dst[oy * pitch + ox] = res[oy][ox];
    }
}

template <int K, bool ONE, bool GRAD>
DEV void filter_band(float* region0, const float* aux0, int stride, const LevelGeom& lg, int q, int np,
                     const float (&w)[K * K], float (&gacc)[K * K], int lane)
{
    if (lg.T == 4)
        filter_band_inplace<K, 4, ONE ? 1 : kMaxRounds4, GRAD>(region0, aux0, stride, lg, q, np, w, gacc, lane);
    else if (lg.T == 2)
        filter_band_inplace<K, 2, ONE ? 1 : kMaxRounds2, GRAD>(region0, aux0, stride, lg, q, np, w, gacc, lane);
    else
        filter_band_inplace<K, 1, ONE ? 1 : kMaxRounds1, GRAD>(region0, aux0, stride, lg, q, np, w, gacc, lane);
}

// Kernel-gradient correlation of one subband over all resident planes with
// tiles: acc += sum over sites of dZ(site) * Y(site + tap offset).
// Sites counted by a kernel-gradient correlation: [m0, m1) in both grid
// directions (region mode counts only its own tile's sites; otherwise all).
struct SiteMask {
    int m0, m1;
};

template <int K, int T>
DEV void corr_band_tiles(const float* __restrict__ dz0, const float* __restrict__ y0, int stride,
                         const LevelGeom& lg, int q, int np, float (&acc)[K * K], int lane, SiteMask mk)
{
    const int tx = lg.ew / T;
    const int per = tx * (lg.eh / T);
    const int total = np * per;
    for (int it = lane; it < total; it += 64) {
        const TileIdx ti = tile_at(it, per, lg.r_tper, tx, lg.r_tx, T);
        const int boff = ti.p * stride + lg.off + q * lg.band;
        float ctr[T][T];
        load_center<K, T>(dz0 + boff, lg.pitch, ti.j0, ti.i0, ctr);
#pragma unroll
        for (int oy = 0; oy < T; ++oy)
#pragma unroll
            for (int ox = 0; ox < T; ++ox) {
                const int j = ti.j0 + oy, i = ti.i0 + ox;
                if (j < mk.m0 || j >= mk.m1 || i < mk.m0 || i >= mk.m1) ctr[oy][ox] = 0.f;
            }
        corr_tile<K, T>(y0 + boff, lg.pitch, ti.j0, ti.i0, ctr, acc);
    }
}

template <int K>
DEV void corr_band(const float* dz0, const float* y0, int stride, const LevelGeom& lg, int q, int np,
                   float (&acc)[K * K], int lane, SiteMask mk)
{
    if (lg.T == 4)
        corr_band_tiles<K, 4>(dz0, y0, stride, lg, q, np, acc, lane, mk);
    else if (lg.T == 2)
        corr_band_tiles<K, 2>(dz0, y0, stride, lg, q, np, acc, lane, mk);
    else
        corr_band_tiles<K, 1>(dz0, y0, stride, lg, q, np, acc, lane, mk);
}

// Kernel-gradient correlation of one coarse subband, by rows: lane (tap row p,
// row group rg) keeps the K sums G[p][0..K-1] for the rows rg, rg+NG, ... of
// the list of every resident plane's site rows and walks each row in CW-site
// chunks read with 16-byte loads:
//   G[p][t] += sum_i dZ[j][i] * Y[j+p-R][i+t-R].
// Reads past the grid width hit zeros (ragged sites / halo), which contribute
// nothing. The row groups are then summed with a fixed xor tree and added to
// one LDS slot per tap, so the result does not depend on timing.
template <int K, int CW>
DEV void corr_row_chunk(const float* __restrict__ dzr, const float* __restrict__ yr, float (&acc)[K])
{
    constexpr int R = K / 2;
    constexpr int ND = ceil4c(CW + R), NY = ceil4c(CW + 2 * R);
    float d[ND], y[NY];
#pragma unroll
    for (int v = 0; v < ND / 4; ++v) {
        const float4 f = reinterpret_cast<const float4*>(dzr)[v];
        d[4 * v] = f.x, d[4 * v + 1] = f.y, d[4 * v + 2] = f.z, d[4 * v + 3] = f.w;
    }
#pragma unroll
    for (int v = 0; v < NY / 4; ++v) {
        const float4 f = reinterpret_cast<const float4*>(yr)[v];
        y[4 * v] = f.x, y[4 * v + 1] = f.y, y[4 * v + 2] = f.z, y[4 * v + 3] = f.w;
    }
#pragma unroll
    for (int i = 0; i < CW; ++i)
#pragma unroll
        for (int t = 0; t < K; ++t) acc[t] = __builtin_fmaf(d[R + i], y[i + t], acc[t]);
}

template <int K>
DEV void corr_band_rows(const float* __restrict__ dz0, const float* __restrict__ y0, int stride,
                        const LevelGeom& lg, int q, int np, float* __restrict__ slot, int lane)
{
    constexpr int R = K / 2;
    constexpr int PS = row_group_lanes(K);  // lanes per row group
    constexpr int NG = 64 / PS;                                        // row groups
    const int p = lane & (PS - 1), rg = lane / PS;
    const bool active = p < K;
    const int prow = active ? p : R;  // inactive lanes read a valid row and are dropped below
    float acc[K];
#pragma unroll
    for (int t = 0; t < K; ++t) acc[t] = 0.f;
    // the (plane, row) pairs of the resident planes are dealt over the row
    // groups as one flat list, so small grids keep every group busy
    const int cw = row_chunk(lg.w);
    const float r_h = 1.0f / (float)lg.h;
    for (int e = rg; e < np * lg.h; e += NG) {
        const int pp = fdiv(e, r_h), j = e - pp * lg.h;
        const float* dzr = dz0 + pp * stride + lg.off + q * lg.band + (j + R) * lg.pitch;  // array column 0, site row j
        const float* yr = y0 + pp * stride + lg.off + q * lg.band + (j + prow) * lg.pitch;  // site row j + p - R
        if (cw == 4) {
            corr_row_chunk<K, 4>(dzr, yr, acc);
        } else if (cw == 8) {
            for (int i0 = 0; i0 < lg.w; i0 += 8) corr_row_chunk<K, 8>(dzr + i0, yr + i0, acc);
        } else {
            for (int i0 = 0; i0 < lg.w; i0 += 16) corr_row_chunk<K, 16>(dzr + i0, yr + i0, acc);
        }
    }
#pragma unroll
    for (int t = 0; t < K; ++t)
#pragma unroll
        for (int m = PS; m < 64; m <<= 1) acc[t] += __shfl_xor(acc[t], m, 64);
    if (rg == 0 && active) {
#pragma unroll
        for (int t = 0; t < K; ++t) slot[p * K + t] += acc[t];
    }
}

// Backward, one band of one level: kernel gradient into `gl` and, if dx is
// wanted, the rotated-kernel filter for dx; one pass over the tiles when every
// level fits a single register-tile round.
template <int K, bool ONE>
DEV void grad_and_filter(float* side_in, const float* side_aux, int stride, const LevelGeom& lg, int q, int np,
                         const float (&w)[K * K], float (&gl)[K * K], bool have_out, int lane, SiteMask mk)
{
    if (ONE && have_out) {
        filter_band<K, ONE, true>(side_in, side_aux, stride, lg, q, np, w, gl, lane);
    } else {
        corr_band<K>(side_in, side_aux, stride, lg, q, np, gl, lane, mk);
        if (have_out) filter_band<K, ONE, false>(side_in, side_aux, stride, lg, q, np, w, gl, lane);
    }
}

// ----------------------------------------------------------------------------
// 4. one 4x4 output tile: base correlation + closed-form synthesis
// ----------------------------------------------------------------------------
// Base correlation of the 4x4 tile at (y0, x0); also returns the tile's own
// input values (the window centre), which the backward pass correlates with x.
template <int K>
DEV void base_tile(const float* __restrict__ xa, int xpitch, int y0, int x0, const float (&w)[K * K], float init,
                   float (&acc)[4][4], float (&ctr)[4][4])
{
    constexpr int R = K / 2, N = Win<K, 4>::N;
#pragma unroll
    for (int oy = 0; oy < 4; ++oy)
#pragma unroll
        for (int ox = 0; ox < 4; ++ox) acc[oy][ox] = 0.f;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float row[Win<K, 4>::NA];
        load_row<K, 4>(xa + (y0 + r) * xpitch + x0, row);
        if (r >= R && r < R + 4) {
#pragma unroll
            for (int ox = 0; ox < 4; ++ox) ctr[r - R][ox] = row[R + ox];
        }
#pragma unroll
        for (int oy = 0; oy < 4; ++oy) {
            const int p = r - oy;
            if (p < 0 || p >= K) continue;
#pragma unroll
            for (int ox = 0; ox < 4; ++ox)
#pragma unroll
                for (int t = 0; t < K; ++t)  // the first term starts from `init` (the folded bias)
                    acc[oy][ox] = __builtin_fmaf(w[p * K + t], row[ox + t], (p == 0 && t == 0) ? init : acc[oy][ox]);
        }
    }
}

// base_tile for TR output rows (a half tile: TR = 2), without the centre.
template <int K, int TR>
DEV void base_rows(const float* __restrict__ xa, int xpitch, int y0, int x0, const float (&w)[K * K], float init,
                   float (&acc)[TR][4])
{
    constexpr int N = TR + 2 * (K / 2);
#pragma unroll
    for (int oy = 0; oy < TR; ++oy)
#pragma unroll
        for (int ox = 0; ox < 4; ++ox) acc[oy][ox] = 0.f;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float row[Win<K, 4>::NA];
        load_row<K, 4>(xa + (y0 + r) * xpitch + x0, row);
#pragma unroll
        for (int oy = 0; oy < TR; ++oy) {
            const int p = r - oy;
            if (p < 0 || p >= K) continue;
#pragma unroll
            for (int ox = 0; ox < 4; ++ox)
#pragma unroll
                for (int t = 0; t < K; ++t)
                    acc[oy][ox] = __builtin_fmaf(w[p * K + t], row[ox + t], (p == 0 && t == 0) ? init : acc[oy][ox]);
        }
    }
}

// Proposition 2 for the 4x4 tile at (y0, x0), y0 and x0 multiples of 4, added
// to acc. Every coefficient has its 4^-l already folded into the kernels, so
// each level contributes LL + sy*LH + sx*HL + sy*sx*HH at (y >> l, x >> l) with
// sy = (-1)^bit(l-1) of y, sx likewise. For l >= 3 the whole tile shares one
// coefficient tuple and one sign pair; level 2 has one tuple and a sign pair
// per 2x2 quadrant; level 1 has a tuple per quadrant and a sign pair per pixel.
// Because the LL term of every level enters with sign +, the coarser levels'
// sum for a quadrant is simply added to that quadrant's level-1 LL.
// `carry` (nullable) is the contribution of the levels above m = cr.m (the
// synthesis of a coarse sub-problem, in orthonormal units, on the level-m
// grid, in the pass's storage type); it enters level m's LL, i.e. with the factor 2^-m of m synthesis
// steps: per quadrant for m = 1, tile-wide for m >= 2 (a 4x4 tile lies inside
// one level-2 site). (cy, cx) is the tile's first level-m site in it.
struct Carry {
    const void* p;  // elements of the pass's storage type CT
    int H, W, cy, cx, m;
};

template <int K, typename CT>
DEV void synth_tile(const float* __restrict__ reg, const PlaneGeom& g, int y0, int x0, float (&acc)[4][4],
                    const Carry& cr)
{
    const CT* carry = reinterpret_cast<const CT*>(cr.p);
    constexpr int R = K / 2;
    const int L = g.L;
    if (L < 1) return;
    float coarse = 0.f;
    if (cr.p && cr.m >= 2 && cr.cy < cr.H && cr.cx < cr.W)
        coarse = __builtin_ldexpf(to_f32(carry[(long)cr.cy * cr.W + cr.cx]), -cr.m);
    for (int l = 3; l <= L; ++l) {
        const LevelGeom& lg = g.lv[l];
        const float* z = reg + lg.off + ((y0 >> l) + R) * lg.pitch + (x0 >> l) + R;
        const float ll = z[0], lh = z[lg.band], hl = z[2 * lg.band], hh = z[3 * lg.band];
        const bool by = (y0 >> (l - 1)) & 1, bx = (x0 >> (l - 1)) & 1;
        const float t1 = by ? ll - lh : ll + lh;  // LL + sy LH
        const float t2 = by ? hl - hh : hl + hh;  // HL + sy HH
        coarse += bx ? t1 - t2 : t1 + t2;
    }
    float quad[2][2];
    if (L >= 2) {
        const LevelGeom& lg = g.lv[2];
        const float* z = reg + lg.off + ((y0 >> 2) + R) * lg.pitch + (x0 >> 2) + R;
        const float ll = z[0] + coarse, lh = z[lg.band], hl = z[2 * lg.band], hh = z[3 * lg.band];
        const float u = ll + lh, v = ll - lh, s = hl + hh, d = hl - hh;
        quad[0][0] = u + s;
        quad[0][1] = u - s;
        quad[1][0] = v + d;
        quad[1][1] = v - d;
    } else {
        quad[0][0] = quad[0][1] = quad[1][0] = quad[1][1] = coarse;
    }
    if (cr.p && cr.m == 1) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int j = cr.cy + a, i = cr.cx + b;
                if (j < cr.H && i < cr.W) quad[a][b] += 0.5f * to_f32(carry[(long)j * cr.W + i]);
            }
    }
    const LevelGeom& lg = g.lv[1];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const float* z = reg + lg.off + ((y0 >> 1) + a + R) * lg.pitch + (x0 >> 1) + b + R;
            const float ll = z[0] + quad[a][b], lh = z[lg.band], hl = z[2 * lg.band], hh = z[3 * lg.band];
            const float u = ll + lh, v = ll - lh, s = hl + hh, d = hl - hh;
            acc[2 * a][2 * b] += u + s;
            acc[2 * a][2 * b + 1] += u - s;
            acc[2 * a + 1][2 * b] += v + d;
            acc[2 * a + 1][2 * b + 1] += v - d;
        }
}

// synth_tile for half a (tile rows 2a and 2a + 1, i.e. level-1 quadrant row a)
// of the 4x4 tile at (y0, x0): the same operations, in the same order, for
// those eight pixels; acc holds their two rows.
template <int K, typename CT>
DEV void synth_half(const float* __restrict__ reg, const PlaneGeom& g, int y0, int x0, int a, float (&acc)[2][4],
                    const Carry& cr)
{
    const CT* carry = reinterpret_cast<const CT*>(cr.p);
    constexpr int R = K / 2;
    const int L = g.L;
    if (L < 1) return;
    float coarse = 0.f;
    if (cr.p && cr.m >= 2 && cr.cy < cr.H && cr.cx < cr.W)
        coarse = __builtin_ldexpf(to_f32(carry[(long)cr.cy * cr.W + cr.cx]), -cr.m);
    for (int l = 3; l <= L; ++l) {
        const LevelGeom& lg = g.lv[l];
        const float* z = reg + lg.off + ((y0 >> l) + R) * lg.pitch + (x0 >> l) + R;
        const float ll = z[0], lh = z[lg.band], hl = z[2 * lg.band], hh = z[3 * lg.band];
        const bool by = (y0 >> (l - 1)) & 1, bx = (x0 >> (l - 1)) & 1;
        const float t1 = by ? ll - lh : ll + lh;
        const float t2 = by ? hl - hh : hl + hh;
        coarse += bx ? t1 - t2 : t1 + t2;
    }
    float quad[2];
    if (L >= 2) {
        const LevelGeom& lg = g.lv[2];
        const float* z = reg + lg.off + ((y0 >> 2) + R) * lg.pitch + (x0 >> 2) + R;
        const float ll = z[0] + coarse, lh = z[lg.band], hl = z[2 * lg.band], hh = z[3 * lg.band];
        const float u = ll + lh, v = ll - lh, s = hl + hh, d = hl - hh;
        quad[0] = a ? v + d : u + s;
        quad[1] = a ? v - d : u - s;
    } else {
        quad[0] = quad[1] = coarse;
    }
    if (cr.p && cr.m == 1) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int j = cr.cy + a, i = cr.cx + b;
            if (j < cr.H && i < cr.W) quad[b] += 0.5f * to_f32(carry[(long)j * cr.W + i]);
        }
    }
    const LevelGeom& lg = g.lv[1];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const float* z = reg + lg.off + ((y0 >> 1) + a + R) * lg.pitch + (x0 >> 1) + b + R;
        const float ll = z[0] + quad[b], lh = z[lg.band], hl = z[2 * lg.band], hh = z[3 * lg.band];
        const float u = ll + lh, v = ll - lh, s = hl + hh, d = hl - hh;
        acc[0][2 * b] += u + s;
        acc[0][2 * b + 1] += u - s;
        acc[1][2 * b] += v + d;
        acc[1][2 * b + 1] += v - d;
    }
}

// Store a 4x4 output tile at (y0, x0) (non-negative, x0 a multiple of 4) of an
// H x W plane, cropped to the plane; vw as for fetch_block.
template <typename T, int TR = 4>
DEV void store_tile(T* __restrict__ plane, int H, int W, int y0, int x0, const float (&v)[TR][4], int vw)
{
#pragma unroll
    for (int oy = 0; oy < TR; ++oy) {
        const int y = y0 + oy;
        if (y >= H || x0 >= W) break;
        T* row = plane + (long)y * W + x0;
        if (vw == 2) {
#pragma unroll
            for (int c = 0; c < 4; c += 2) {
                if (x0 + c >= W) break;
                if constexpr (sizeof(T) == 4) {
                    *reinterpret_cast<float2*>(row + c) = make_float2(v[oy][c], v[oy][c + 1]);
                } else {
                    T h[2] = {from_f32<T>(v[oy][c]), from_f32<T>(v[oy][c + 1])};
                    uint32_t packed;
                    __builtin_memcpy(&packed, h, 4);
                    *reinterpret_cast<uint32_t*>(row + c) = packed;
                }
            }
        } else if (vw == 4 && x0 + 4 <= W) {
            if constexpr (sizeof(T) == 4) {
                *reinterpret_cast<float4*>(row) = make_float4(v[oy][0], v[oy][1], v[oy][2], v[oy][3]);
            } else {
                T h[4] = {from_f32<T>(v[oy][0]), from_f32<T>(v[oy][1]), from_f32<T>(v[oy][2]),
                          from_f32<T>(v[oy][3])};
                uint2 packed;
                __builtin_memcpy(&packed, h, 8);
                *reinterpret_cast<uint2*>(row) = packed;
            }
        } else if (x0 + 4 <= W) {
#pragma unroll
            for (int ox = 0; ox < 4; ++ox) row[ox] = from_f32<T>(v[oy][ox]);
        } else {
#pragma unroll
            for (int ox = 0; ox < 4; ++ox)
                if (x0 + ox < W) row[ox] = from_f32<T>(v[oy][ox]);
        }
    }
}

DEV float wave_sum(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// Sum the per-workgroup partials over chunks in increasing order, then unfold
// eq. (foldgrad): dW = s * G and ds = <G, W>, where G is the gradient of the
// folded kernel s*W (the level partials carry an extra 4^l from the
// unnormalised pyramids, removed here exactly); for the base row also the bias
// terms d b0 = s0 * sum(dy) and b0 * sum(dy) in d s0. One wavefront per
// (channel c, kernel row `band`: 0 = base, else 1 + (l-1)*4 + q); lane t
// owns tap t (lane k*k the sum of dy; at k = 9 the taps and the sum wrap
// round the 64 lanes); the d(scale) dot product is a fixed-order wavefront
// reduction.
DEV void reduce_task(const ReduceArgs& a, int c, int band, int t)
{
    const int KK = a.k * a.k;
    const int NP = partial_floats_per_channel(a.k, a.L);
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
    // lane t takes taps t, t + 64, ... (more than one only for k = 9) and the
    // bias sum at index k * k
    float prod = 0.f;
    const long step = (long)a.C * NP;
    for (int tt = t; tt <= KK; tt += 64) {
        if (tt < KK) {
            const float* src = a.partial + (long)c * NP + band * KK + tt;
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
            dw[tt] = scale * G;
            prod = tt == t ? G * w[tt] : __builtin_fmaf(G, w[tt], prod);
        } else if (band == 0) {
            // folded base bias b~ = s0 * b0: its gradient is the sum of dy, so
            // d b0 = s0 * sum(dy) and d s0 gains b0 * sum(dy) (eq. foldgrad)
            const float* src = a.partial + (long)c * NP + (NP - 1);
            float Gb = 0.f;
            for (int ch = 0; ch < a.nchunks; ++ch) Gb += src[(long)ch * step];
            if (a.db0) a.db0[c] = scale * Gb;
            if (a.p.b0) prod = tt == t ? a.p.b0[c] * Gb : __builtin_fmaf(a.p.b0[c], Gb, prod);
        }
    }
    prod = wave_sum(prod);
    if (t == 0) *ds = prod;
}

// A finalize workgroup at the head of a forward launch: wavefront w of
// workgroup b takes task 4b + w, task c * (1 + 4L) + row being (channel c,
// kernel row `row`). Dispatched first, these short, latency-bound waves
// overlap the plane work instead of trailing it.
DEV void fin_wave(const FusedArgs& a, int lane, int wave)
{
    const int rows = 1 + 4 * a.fin.L;
    const int task = 4 * (int)blockIdx.x + wave;
    if (task >= a.fin.C * rows) return;
    const int c = task / rows;
    reduce_task(a.fin, c, task - c * rows, lane);
}

// Index of the folded-weight row for the base kernel (0) or level l band q.
DEV int wrow(int l, int q) { return l == 0 ? 0 : 1 + (l - 1) * 4 + q; }

// Fetch one folded kernel into registers (the same value in every lane, read
// with broadcast LDS loads, so the FMAs take it as a VGPR operand without any
// cross-lane moves); `rot` reverses the tap order (180-degree rotation, used
// for dx).
template <int K>
DEV void fetch_weights(const float* __restrict__ wtab, int row, bool rot, int lane, float (&w)[K * K])
{
    constexpr int KK = K * K;
    (void)lane;
#pragma unroll
    for (int i = 0; i < KK; ++i) w[i] = wtab[row * KK + (rot ? KK - 1 - i : i)];
}

// ----------------------------------------------------------------------------
// the fused kernel
// ----------------------------------------------------------------------------
template <int K, typename ST, bool BWD, bool ONE, bool RGN>
__global__ void __launch_bounds__(kThreads) fused_kernel(const FusedArgs a)
{
    constexpr int R = K / 2, KK = K * K;
    extern __shared__ float4 lds4[];
    float* lds = reinterpret_cast<float*>(lds4);

    const PlaneGeom& g = a.g;  // the plane (or, in region mode, the region) held on chip
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int C = a.C;
    if constexpr (!BWD)
        if ((int)blockIdx.x < a.fin_blocks) {
            fin_wave(a, lane, wave);
            return;
        }
    const int bid = (int)blockIdx.x - a.fin_blocks;
    const int c = bid % C;
    const int ntiles = RGN ? a.rg_ntx * a.rg_nty : 1;
    const int chunk = (bid / C) / ntiles;
    const int tile = (bid / C) - chunk * ntiles;
    const int b_begin = chunk * a.nb;
    const int b_end = min(a.B, b_begin + a.nb);
    const int L = g.L;
    // region mode: origin of the region in the real plane (multiples of 4)
    const int oy = RGN ? (tile / a.rg_ntx) * a.rg_T - a.rg_h : 0;
    const int ox = RGN ? (tile % a.rg_ntx) * a.rg_T - a.rg_h : 0;
    const int PH = RGN ? a.real_H : g.H, PW = RGN ? a.real_W : g.W;  // the real plane
    const long HW = (long)PH * PW;
    const bool skip_base = a.skip_base != 0;
    // eq. (fold): the folded base bias s0 * b0 starts every output pixel's sum
    const float bias = (!BWD && !skip_base && a.p.b0) ? a.p.s0[c] * a.p.b0[c] : 0.f;

    // LDS: [folded weights][coarse kernel-gradient sums (backward)][planes]
    const int wt_floats = ceil4c((1 + 4 * L) * KK);
    const int gc_floats = BWD ? ceil4c(L * 4 * KK) : 0;
    float* wtab = lds;
    float* gco = lds + wt_floats;
    float* planes = lds + wt_floats + gc_floats;
    const int stride = BWD ? 2 * g.plane_floats : g.plane_floats;  // region of one plane
    float* side_in = planes;                                       // input side (x / dy)
    float* side_aux = planes + g.plane_floats;                     // backward: x side

    const ST* in = reinterpret_cast<const ST*>(a.in);
    const ST* aux = reinterpret_cast<const ST*>(a.aux);
    ST* out = reinterpret_cast<ST*>(a.out);
    const bool have_out = out != nullptr;
    // vector width of the plane's rows (plane bases are 16-byte aligned when vec_ok)
    const int vw = a.vec_ok == 0 ? 1 : ((PW % 4) == 0 ? 4 : ((PW % 2) == 0 ? 2 : 1));
    const int q = wave;  // the subband this wavefront filters

    for (int i = tid; i < a.lds_floats / 4; i += kThreads) lds4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();

    // eq. (fold): base s0*W0; level l band q: s_l*W_l*4^-l (taps reversed when
    // the forward pass computes dx)
    const bool rot = !BWD && a.p.rot != 0;
    for (int i = tid; i < KK; i += kThreads) wtab[i] = a.p.s0[c] * a.p.w0[c * KK + (rot ? KK - 1 - i : i)];
    for (int l = 1; l <= L; ++l) {
        const float norm = __builtin_ldexpf(1.f, -2 * l);
        const float* lw = a.p.lw[l - 1];
        const float* ls = a.p.ls[l - 1];
        for (int i = tid; i < 4 * KK; i += kThreads) {
            const int q = i / KK, t = i - q * KK;
            wtab[wrow(l, q) * KK + t] = ls[4 * c + q] * lw[(4 * c + q) * KK + (rot ? KK - 1 - t : t)] * norm;
        }
    }
    __syncthreads();

    // backward: per-lane kernel-gradient sums (base; levels 1 and 2 of band `wave`)
    float g0[KK], g1[KK], g2[KK];
#pragma unroll
    for (int t = 0; t < KK; ++t) g0[t] = g1[t] = g2[t] = 0.f;
    float gdy = 0.f;  // backward: sum of dy over the workgroup's pixels (bias gradient)

    for (int b0 = b_begin; b0 < b_end; b0 += a.PP) {
        const int np = min(a.PP, b_end - b0);

        // 1. planes -> LDS, with Haar levels 1 and 2 formed on the way in
        {
            const int tx = g.tiles_xl, per = g.tiles_xl * g.tiles_y;
            for (int it = tid; it < np * per; it += kThreads) {
                const TileIdx ti = tile_at(it, per, g.r_tiles_l, tx, g.r_tiles_xl, 4);
                if (ti.i0 >= 4 * g.tiles_x) continue;  // a padding lane of the tile row
                const long plane = (long)(b0 + ti.p) * C + c;
                float v[4][4];
                fetch_block<ST>(in + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, v);
                store_block<K>(v, side_in + ti.p * stride, g, ti.j0, ti.i0);
                if constexpr (BWD) {
                    fetch_block<ST>(aux + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, vw, v);
                    store_block<K>(v, side_aux + ti.p * stride, g, ti.j0, ti.i0);
                }
            }
        }
        __syncthreads();

        // 2. the remaining Haar levels on chip
        for (int l = 3; l <= L; ++l) {
            const LevelGeom& lg = g.lv[l];
            const LevelGeom& lp = g.lv[l - 1];
            analysis_level(side_in + lp.off, lp.pitch, side_in + lg.off, lg, R, np, stride, tid);
            if constexpr (BWD) analysis_level(side_aux + lp.off, lp.pitch, side_aux + lg.off, lg, R, np, stride, tid);
            __syncthreads();
        }

        // 3. subband filtering, one band per wavefront. In the backward pass the
        //    kernel gradient of each band is accumulated on the way: for levels
        //    1..3 in per-lane registers (in the same pass over the tiles as the
        //    dx filter when every level fits one tile round), for deeper levels
        //    row by row into LDS.
        for (int l = 1; l <= L; ++l) {
            const LevelGeom& lg = g.lv[l];
            if constexpr (!BWD && ONE) {
                // levels 1 and >= 3 in one round (see filter_merged), level 2 below
                if (a.merge_deep && l != 2) {
                    if (l == 1) filter_merged<K>(side_in, stride, g, wtab, q, np, lane);
                    continue;
                }
            }
            float w[KK];
            fetch_weights<K>(wtab, wrow(l, q), BWD, lane, w);
            if constexpr (BWD) {
                // region mode counts only the sites of its own tile
                const SiteMask mk = RGN ? SiteMask{a.rg_h >> l, (a.rg_h + a.rg_T) >> l} : SiteMask{0, 1 << 30};
                if (l <= reg_levels<ONE>()) {
                    // static choice of the accumulator array keeps it in registers
                    if (l == 1)
                        grad_and_filter<K, ONE>(side_in, side_aux, stride, lg, q, np, w, g1, have_out, lane, mk);
                    else
                        grad_and_filter<K, ONE>(side_in, side_aux, stride, lg, q, np, w, g2, have_out, lane, mk);
                } else {
                    corr_band_rows<K>(side_in, side_aux, stride, lg, q, np, gco + ((l - 1) * 4 + q) * KK, lane);
                    if (have_out) filter_band<K, ONE, false>(side_in, side_aux, stride, lg, q, np, w, g1, lane);
                }
            } else {
                filter_band<K, ONE, false>(side_in, side_aux, stride, lg, q, np, w, g1, lane);
            }
        }
        __syncthreads();

        // 4. output tiles (region mode: the tiles of the region's inner rg_T x rg_T square)
        {
            float w[KK];
            fetch_weights<K>(wtab, 0, BWD, lane, w);
            const int tx = RGN ? a.rg_T / 4 : g.tiles_xl;
            const int per = RGN ? tx * tx : g.tiles_xl * g.tiles_y;
            // Backward with at most half as many output tiles as threads: a
            // tile's dx (base correlation with rotated taps and synthesis) and
            // its base kernel-gradient correlation go to two threads, the
            // second half of the workgroup taking the correlations, instead of
            // one thread doing both while the other half idles.
            const int n = np * per;
            const bool halves = BWD && have_out && !skip_base && 2 * n <= kThreads;
            // Forward, half tiles (two rows each, two threads per tile) for
            // the tiles [nmain, n) on the threads [hbase, hbase + 2 (n - nmain)):
            //  - more tiles than threads: the tiles past the last full round,
            //    when they fill at most half a round, so that every thread's
            //    last round costs half a tile rather than half the threads
            //    paying a whole one;
            //  - a single round: the tiles of the last, partly filled
            //    wavefront, when they fill at most half of it, so that this
            //    wavefront's instructions cost half a tile.
            int nmain = n, hbase = 0;
            if constexpr (!BWD && !RGN) {
                const int rem = n % kThreads, rw = n % 64;
                if (!ONE && n > kThreads && rem != 0 && 2 * rem <= kThreads) {
                    nmain = n - rem;
                } else if (ONE && n <= kThreads && rw != 0 && 2 * rw <= 64) {
                    nmain = n - rw;
                    hbase = nmain;
                }
            }
            for (int it2 = tid; it2 < (halves ? 2 * n : nmain); it2 += kThreads) {
                const bool corr_only = halves && it2 >= n;
                const int it = corr_only ? it2 - n : it2;
                TileIdx ti = RGN ? tile_at(it, per, a.rg_r_itiles, tx, a.rg_r_itx, 4)
                                 : tile_at(it, per, g.r_tiles_l, tx, g.r_tiles_xl, 4);
                if (!RGN && ti.i0 >= 4 * g.tiles_x) continue;  // a padding lane of the tile row
                if (RGN) {
                    ti.j0 += a.rg_h;
                    ti.i0 += a.rg_h;
                }
                const float* reg = side_in + ti.p * stride;
                const long plane = (long)(b0 + ti.p) * C + c;
                float acc[4][4], ctr[4][4];
                if ((!BWD || have_out) && !corr_only) {
                    if (skip_base) {
#pragma unroll
                        for (int oy2 = 0; oy2 < 4; ++oy2)
#pragma unroll
                            for (int ox2 = 0; ox2 < 4; ++ox2) acc[oy2][ox2] = 0.f;
                    } else {
                        base_tile<K>(reg, g.xpitch, ti.j0, ti.i0, w, bias, acc, ctr);
                    }
                    Carry cr = {nullptr, 0, 0, 0, 0, 0};
                    if (a.carry) {
                        cr.p = reinterpret_cast<const ST*>(a.carry) + plane * a.carry_H * a.carry_W;
                        cr.H = a.carry_H;
                        cr.W = a.carry_W;
                        cr.m = a.carry_level;
                        cr.cy = (oy + ti.j0) >> cr.m;
                        cr.cx = (ox + ti.i0) >> cr.m;
                    }
                    synth_tile<K, ST>(reg, g, ti.j0, ti.i0, acc, cr);
                    store_tile<ST>(out + plane * HW, PH, PW, oy + ti.j0, ox + ti.i0, acc, vw);
                } else if (!skip_base) {
                    load_center<K, 4>(reg, g.xpitch, ti.j0, ti.i0, ctr);
                }
                if constexpr (BWD) {
                    if (!skip_base && (corr_only || !halves)) {
                        corr_tile<K, 4>(side_aux + ti.p * stride, g.xpitch, ti.j0, ti.i0, ctr, g0);
#pragma unroll
                        for (int oy2 = 0; oy2 < 4; ++oy2)
                            gdy += (ctr[oy2][0] + ctr[oy2][1]) + (ctr[oy2][2] + ctr[oy2][3]);
                    }
                }
            }
            if constexpr (!BWD && !RGN) {
                const int h = tid - hbase;
                if (nmain < n && h >= 0 && h < 2 * (n - nmain)) {
                    const int hrow = h & 1;  // rows 2 hrow, 2 hrow + 1 of the tile
                    const TileIdx ti = tile_at(nmain + (h >> 1), per, g.r_tiles_l, tx, g.r_tiles_xl, 4);
                    if (ti.i0 < 4 * g.tiles_x) {
                        const float* reg = side_in + ti.p * stride;
                        const long plane = (long)(b0 + ti.p) * C + c;
                        float acc2[2][4];
                        if (skip_base) {
#pragma unroll
                            for (int oy2 = 0; oy2 < 2; ++oy2)
#pragma unroll
                                for (int ox2 = 0; ox2 < 4; ++ox2) acc2[oy2][ox2] = 0.f;
                        } else {
                            base_rows<K, 2>(reg, g.xpitch, ti.j0 + 2 * hrow, ti.i0, w, bias, acc2);
                        }
                        Carry cr = {nullptr, 0, 0, 0, 0, 0};
                        if (a.carry) {
                            cr.p = reinterpret_cast<const ST*>(a.carry) + plane * a.carry_H * a.carry_W;
                            cr.H = a.carry_H;
                            cr.W = a.carry_W;
                            cr.m = a.carry_level;
                            cr.cy = ti.j0 >> cr.m;
                            cr.cx = ti.i0 >> cr.m;
                        }
                        synth_half<K, ST>(reg, g, ti.j0, ti.i0, hrow, acc2, cr);
                        store_tile<ST, 2>(out + plane * HW, PH, PW, ti.j0 + 2 * hrow, ti.i0, acc2, vw);
                    }
                }
            }
        }
        __syncthreads();
    }

    if constexpr (BWD) {
        // fixed-order reduction of the kernel-gradient sums of this workgroup
        const int NP = partial_floats_per_channel(K, L);
        float* red = planes;  // the plane regions are free now
#pragma unroll
        for (int t = 0; t < KK; ++t) {
            const float v0 = wave_sum(g0[t]);
            const float v1 = wave_sum(g1[t]);
            const float v2 = wave_sum(g2[t]);
            if (lane == 0) {
                red[wave * KK + t] = v0;
                red[(kWaves + wave) * KK + t] = v1;
                red[(2 * kWaves + wave) * KK + t] = v2;
            }
        }
        const float vdy = wave_sum(gdy);
        if (lane == 0) red[3 * kWaves * KK + wave] = vdy;
        __syncthreads();
        float* dst = a.partial + ((long)(chunk * ntiles + tile) * C + c) * NP;
        for (int t = tid; t < KK; t += kThreads)
            dst[t] = ((red[t] + red[KK + t]) + red[2 * KK + t]) + red[3 * KK + t];
        if (tid == 0) {
            const float* r = red + 3 * kWaves * KK;
            dst[NP - 1] = ((r[0] + r[1]) + r[2]) + r[3];
        }
        // register-held levels: band q's sums came from wavefront q
        for (int i = tid; i < 4 * KK * min(L, reg_levels<ONE>()); i += kThreads) dst[KK + i] = red[kWaves * KK + i];
        for (int i = 4 * KK * reg_levels<ONE>() + tid; i < 4 * L * KK; i += kThreads) dst[KK + i] = gco[i];
    }
}

template <int K, typename ST, bool BWD, bool ONE, bool RGN>
hipError_t launch_variant(const FusedArgs& a, int grid, hipStream_t s)
{
    const size_t bytes = (size_t)a.lds_floats * sizeof(float);
    static std::atomic<unsigned long long> lds_done{0};
    const hipError_t e = allow_full_lds(reinterpret_cast<const void*>(&fused_kernel<K, ST, BWD, ONE, RGN>), lds_done);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((fused_kernel<K, ST, BWD, ONE, RGN>), dim3(grid), dim3(kThreads), bytes, s, a);
    return hipGetLastError();
}

template <int K, typename ST, bool BWD>
hipError_t launch_one(const FusedArgs& a, int grid, hipStream_t s)
{
    if (a.rg_ntx > 0) {
        if constexpr (!BWD)  // forward regions whose level fits one register-tile round
            if (a.one_round) return launch_variant<K, ST, BWD, true, true>(a, grid, s);
        return launch_variant<K, ST, BWD, false, true>(a, grid, s);
    }
    return a.one_round ? launch_variant<K, ST, BWD, true, false>(a, grid, s)
                       : launch_variant<K, ST, BWD, false, false>(a, grid, s);
}

template <int K, bool BWD>
hipError_t launch_dt(wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
    switch (dt) {
        case WTCONV_F32: return launch_one<K, float, BWD>(a, grid, s);
        case WTCONV_BF16: return launch_one<K, uint16_t, BWD>(a, grid, s);
        case WTCONV_F16: return launch_one<K, _Float16, BWD>(a, grid, s);
    }
    return hipErrorInvalidValue;
}

template <bool BWD>
hipError_t dispatch(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
    switch (k) {
        case 1: return launch_dt<1, BWD>(dt, a, grid, s);
        case 3: return launch_dt<3, BWD>(dt, a, grid, s);
        case 5: return launch_dt<5, BWD>(dt, a, grid, s);
        case 7: return launch_dt<7, BWD>(dt, a, grid, s);
        case 9:
            // the k = 9 backward is compiled in a translation unit of its own
            if constexpr (BWD)
                return launch_backward_k9(dt, a, grid, s);
            else
                return launch_dt<9, false>(dt, a, grid, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace
}  // namespace wtc
