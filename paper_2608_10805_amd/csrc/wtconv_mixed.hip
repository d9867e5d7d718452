// Forward WTConv kernel with mixed task rounds for gfx950 (MI355X), for
// resident planes. Internal; not part of the public ABI.
//
// The arithmetic is fused_kernel's (wtconv_fused.h): each plane and its
// unnormalised Haar pyramid on chip, every subband filtered in place with its
// folded kernel (eq. fold, Section 4.3), each output pixel formed as the base
// correlation plus the closed-form synthesis of Proposition 2 (Section 4.2).
// What differs is how the k x k correlations are spread over lanes.
// fused_kernel gives each wavefront one subband and each thread one output
// tile, in separate rounds; a 56 x 56 plane then takes three rounds of 4 x 4
// tiles (level 1 with the deep levels, level 2, the output tiles) at 77-83 %
// lane use. Here the output tiles' base correlations and the subband tiles of
// every level and band are equal tasks (4 x 4 tiles, k^2 FMAs per element)
// packed into as few rounds of 256 lanes as possible: the 196 output tiles and
// 276 subband tiles of a 56 x 56 plane at L = 3 fill two rounds at 92 % lane
// use. A lane reads the folded kernel of its own task from LDS, so the lanes
// of one wavefront may filter different bands; the base correlation starts
// from the folded bias, a subband tile from zero (an exact product).
//
// The host packs whole (level, band) groups into rounds: a band array is read
// only by its own group's tasks, so a round's filtered tiles are written over
// the unfiltered sites right after one barrier, and no later round reads
// them. Output tiles need every level filtered, so they take the rounds from
// the last one with subband tiles (F) on: round F's output tiles wait for its
// write-back, and later rounds hold output tiles only. Each output tile is
// finished (Proposition 2, the store) in its own round, so a lane holds one
// tile's sums at a time. Within a round the tasks are split into four
// contiguous quarters, one per wavefront.
//
// Per batch of resident planes:
//   1. load the planes (levels 1 and 2 formed in registers on the way);
//   2. the remaining analysis levels in LDS;
//   3. per round: every task's 16 correlations into registers; up to round F,
//      a barrier and the round's subband tiles written in place (ragged sites
//      past the grid stay zero); from round F on (after one more barrier in
//      round F), each output tile adds Proposition 2 to its base correlation
//      (and a split's carry) and is stored once.
// The (task -> lane) assignment depends only on the thread index and the
// plan, so each thread decodes its tasks once per workgroup.
#include "wtconv_fused.h"

namespace wtc {
namespace {

// One task of a thread: a 4x4 output tile (its base correlation) or a 4x4
// tile of sites of one band of one level.
struct MixedSlot {
    int src;    // LDS float offset, from the planes array, of the window's top-left element
    int pitch;  // floats per row of the array the window lies in
    int woff;   // float offset of the task's folded kernel in the weight table
    int meta;   // kind (0 none, 1 output tile, 2 subband tile) | valid rows << 2 | valid cols << 5 | plane << 8
    int pos;    // output tile: (j0 << 16) | i0, its first pixel in the plane
};

constexpr int kSlotNone = 0, kSlotOut = 1, kSlotBand = 2;

// The task of (round r, this thread): the round's tasks in segment order,
// split into four contiguous quarters, quarter w to wavefront w.
template <int K>
DEV MixedSlot decode_slot(const FusedArgs& a, int r, int wave, int lane)
{
    constexpr int KP = ceil4c(K * K);
    const PlaneGeom& g = a.g;
    MixedSlot sl = {0, 0, 0, kSlotNone, 0};
    const int n = a.mx_ntask[r];
    const int nq = (n + 3) >> 2;
    int t = wave * nq + lane;
    if (lane >= nq || t >= n) return sl;
    // the segment of task t (uniform loop, per-lane selects); a round has at
    // most one run of output tiles, the earlier ones are counted in mx_out0
    int seg = 0, rel = 0, at = 0;
    for (int i = a.mx_seg0[r]; i < a.mx_seg0[r + 1]; ++i) {
        const int cnt = a.mx_seg[i] >> 8;
        if (t >= at && t < at + cnt) {
            seg = a.mx_seg[i];
            rel = t - at;
        }
        at += cnt;
    }
    t = rel;
    const int out_base = a.mx_out0[r];
    if ((seg & 3) == kSlotOut) {
        const TileIdx ti = tile_at(out_base + t, g.tiles_x * g.tiles_y, g.r_tiles, g.tiles_x, g.r_tiles_x, 4);
        sl.src = ti.p * g.plane_floats + ti.j0 * g.xpitch + ti.i0;
        sl.pitch = g.xpitch;
        sl.woff = 0;
        sl.meta = kSlotOut | (ti.p << 8);
        sl.pos = (ti.j0 << 16) | ti.i0;
        return sl;
    }
    const int lvl = (seg >> 2) & 15, q = (seg >> 6) & 3;
    int off = 0, band = 0, pitch = 0, h = 0, w = 0, tx = 0, per = 0;
    float r_tper = 0.f, r_tx = 0.f;
    for (int l = 1; l <= g.L; ++l) {
        if (l != lvl) continue;
        const LevelGeom& lg = g.lv[l];
        off = lg.off;
        band = lg.band;
        pitch = lg.pitch;
        h = lg.h;
        w = lg.w;
        tx = lg.ew / 4;
        per = tx * (lg.eh / 4);
        r_tper = lg.r_tper;
        r_tx = lg.r_tx;
    }
    const TileIdx ti = tile_at(t, per, r_tper, tx, r_tx, 4);
    sl.src = ti.p * g.plane_floats + off + q * band + ti.j0 * pitch + ti.i0;
    sl.pitch = pitch;
    sl.woff = wrow(lvl, q) * KP;
    const int rows = min(4, h - ti.j0), cols = min(4, w - ti.i0);
    sl.meta = kSlotBand | (rows << 2) | (cols << 5) | (ti.p << 8);
    return sl;
}

template <int K, typename ST, int NR>
__global__ void __launch_bounds__(kThreads) mixed_kernel(const FusedArgs a)
{
    constexpr int R = K / 2, KK = K * K, KP = ceil4c(KK);
    extern __shared__ float4 lds4[];
    float* lds = reinterpret_cast<float*>(lds4);

    const PlaneGeom& g = a.g;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int C = a.C;
    if ((int)blockIdx.x < a.fin_blocks) {
        fin_wave(a, lane, wave);
        return;
    }
    const int bid = (int)blockIdx.x - a.fin_blocks;
    const int c = bid % C;
    const int chunk = bid / C;
    const int b_begin = chunk * a.nb;
    const int b_end = min(a.B, b_begin + a.nb);
    const int L = g.L;
    const int PH = g.H, PW = g.W;
    const long HW = (long)PH * PW;
    const bool skip_base = a.skip_base != 0;
    // eq. (fold): the folded base bias s0 * b0 starts every output pixel's sum
    const float bias = (!skip_base && a.p.b0) ? a.p.s0[c] * a.p.b0[c] : 0.f;

    // LDS: [folded weights, one KP-float row per kernel][planes]
    float* wtab = lds;
    float* planes = lds + (1 + 4 * L) * KP;
    const int stride = g.plane_floats;

    const ST* in = reinterpret_cast<const ST*>(a.in);
    ST* out = reinterpret_cast<ST*>(a.out);
    const int vw = a.vec_ok == 0 ? 1 : ((PW % 4) == 0 ? 4 : ((PW % 2) == 0 ? 2 : 1));

    for (int i = tid; i < a.lds_floats / 4; i += kThreads) lds4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();

    // eq. (fold): base s0*W0; level l band q: s_l*W_l*4^-l (taps reversed when
    // the forward pass computes dx); rows padded to KP floats (16-byte aligned)
    const bool rot = a.p.rot != 0;
    for (int i = tid; i < KK; i += kThreads) wtab[i] = a.p.s0[c] * a.p.w0[c * KK + (rot ? KK - 1 - i : i)];
    for (int l = 1; l <= L; ++l) {
        const float norm = __builtin_ldexpf(1.f, -2 * l);
        const float* lw = a.p.lw[l - 1];
        const float* ls = a.p.ls[l - 1];
        for (int i = tid; i < 4 * KK; i += kThreads) {
            const int q = i / KK, t = i - q * KK;
            wtab[wrow(l, q) * KP + t] = ls[4 * c + q] * lw[(4 * c + q) * KK + (rot ? KK - 1 - t : t)] * norm;
        }
    }

    MixedSlot sl[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) sl[r] = decode_slot<K>(a, r, wave, lane);
    __syncthreads();

    for (int b0 = b_begin; b0 < b_end; b0 += a.PP) {
        const int np = min(a.PP, b_end - b0);

        // 1. planes -> LDS, with Haar levels 1 and 2 formed on the way in
        {
            const int tx = g.tiles_x, per = g.tiles_x * g.tiles_y;
            for (int it = tid; it < np * per; it += kThreads) {
                const TileIdx ti = tile_at(it, per, g.r_tiles, tx, g.r_tiles_x, 4);
                const long plane = (long)(b0 + ti.p) * C + c;
                float v[4][4];
                fetch_block<ST>(in + plane * HW, PH, PW, ti.j0, ti.i0, vw, v);
                store_block<K>(v, planes + ti.p * stride, g, ti.j0, ti.i0);
            }
        }
        __syncthreads();

        // 2. the remaining Haar levels on chip
        for (int l = 3; l <= L; ++l) {
            const LevelGeom& lg = g.lv[l];
            const LevelGeom& lp = g.lv[l - 1];
            analysis_level(planes + lp.off, lp.pitch, planes + lg.off, lg, R, np, stride, tid);
            __syncthreads();
        }

        // 3. task rounds
        const int F = a.mx_first_out;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            // Everything derived from the task (window row addresses, synthesis
            // addresses) is recomputed here every batch: held across the batch
            // loop (it does not change) it would take tens of registers per round.
            int src = sl[r].src, pitch = sl[r].pitch, woff = sl[r].woff, meta = sl[r].meta, pos = sl[r].pos;
            asm volatile("" : "+v"(src), "+v"(pitch), "+v"(woff), "+v"(meta), "+v"(pos));
            const int kind = meta & 3;
            const int p = meta >> 8;
            const bool live = kind != kSlotNone && p < np;
            float res[4][4];
            if (live && !(kind == kSlotOut && skip_base)) {
                float w[KK];
                {
                    const float4* wp = reinterpret_cast<const float4*>(wtab + woff);
                    float t[KP];
#pragma unroll
                    for (int v = 0; v < KP / 4; ++v) {
                        const float4 f = wp[v];
                        t[4 * v] = f.x, t[4 * v + 1] = f.y, t[4 * v + 2] = f.z, t[4 * v + 3] = f.w;
                    }
#pragma unroll
                    for (int i = 0; i < KK; ++i) w[i] = t[i];
                }
                float ctr[4][4];
                base_tile<K>(planes + src, pitch, 0, 0, w, kind == kSlotOut ? bias : 0.f, res, ctr);
            } else {
#pragma unroll
                for (int oy = 0; oy < 4; ++oy)
#pragma unroll
                    for (int ox = 0; ox < 4; ++ox) res[oy][ox] = 0.f;
            }
            if (r <= F) {
                __syncthreads();  // every window of this round's bands has been read
                if (live && kind == kSlotBand) {
                    float* dst = planes + src + R * pitch + R;
                    const int rows = (meta >> 2) & 7, cols = (meta >> 5) & 7;
                    if (rows == 4 && cols == 4) {
#pragma unroll
                        for (int oy = 0; oy < 4; ++oy) st_row<(R % 2) == 0, 4>(dst + oy * pitch, res[oy]);
                    } else {
#pragma unroll
                        for (int oy = 0; oy < 4; ++oy)
#pragma unroll
                            for (int ox = 0; ox < 4; ++ox)
                                if (oy < rows && ox < cols) dst[oy * pitch + ox] = res[oy][ox];
                    }
                }
                if (r == F) __syncthreads();  // every level is filtered
            }
            // output tiles: Proposition 2 (and the carry) added, one store per pixel
            if (r >= F && live && kind == kSlotOut) {
                const int j0 = pos >> 16, i0 = pos & 0xffff;
                const long plane = (long)(b0 + p) * C + c;
                Carry cr = {nullptr, 0, 0, 0, 0, 0};
                if (a.carry) {
                    cr.p = reinterpret_cast<const ST*>(a.carry) + plane * a.carry_H * a.carry_W;
                    cr.H = a.carry_H;
                    cr.W = a.carry_W;
                    cr.m = a.carry_level;
                    cr.cy = j0 >> cr.m;
                    cr.cx = i0 >> cr.m;
                }
                synth_tile<K, ST>(planes + p * stride, g, j0, i0, res, cr);
                store_tile<ST>(out + plane * HW, PH, PW, j0, i0, res, vw);
            }
        }
        __syncthreads();  // the next batch overwrites the planes
    }
}

template <int K, typename ST, int NR>
hipError_t launch_mixed_v(const FusedArgs& a, int grid, hipStream_t s)
{
    const size_t bytes = (size_t)a.lds_floats * sizeof(float);
    static std::atomic<unsigned long long> lds_done{0};
    const hipError_t e = allow_full_lds(reinterpret_cast<const void*>(&mixed_kernel<K, ST, NR>), lds_done);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((mixed_kernel<K, ST, NR>), dim3(grid), dim3(kThreads), bytes, s, a);
    return hipGetLastError();
}

template <int K, typename ST>
hipError_t launch_mixed_t(const FusedArgs& a, int grid, hipStream_t s)
{
    switch (a.mx_rounds) {
        case 1: return launch_mixed_v<K, ST, 1>(a, grid, s);
        case 2: return launch_mixed_v<K, ST, 2>(a, grid, s);
        case 3: return launch_mixed_v<K, ST, 3>(a, grid, s);
        case 4: return launch_mixed_v<K, ST, 4>(a, grid, s);
    }
    return hipErrorInvalidValue;
}

template <int K, typename ST, int NR>
int mixed_wgs_v(int fallback)
{
    static std::atomic<int> cache{0};
    return wgs_by_regs(reinterpret_cast<const void*>(&mixed_kernel<K, ST, NR>), cache, fallback);
}

template <int K, typename ST>
int mixed_wgs_t(int rounds, int fallback)
{
    switch (rounds) {
        case 1: return mixed_wgs_v<K, ST, 1>(fallback);
        case 2: return mixed_wgs_v<K, ST, 2>(fallback);
        case 3: return mixed_wgs_v<K, ST, 3>(fallback);
        case 4: return mixed_wgs_v<K, ST, 4>(fallback);
    }
    return fallback;
}

template <int K>
int mixed_wgs_k(wtconv_dtype dt, int rounds, int fallback)
{
    switch (dt) {
        case WTCONV_F32: return mixed_wgs_t<K, float>(rounds, fallback);
        case WTCONV_BF16: return mixed_wgs_t<K, uint16_t>(rounds, fallback);
        case WTCONV_F16: return mixed_wgs_t<K, _Float16>(rounds, fallback);
    }
    return fallback;
}

}  // namespace

hipError_t launch_forward_mixed(int k, wtconv_dtype dt, const FusedArgs& a, int grid, hipStream_t s)
{
#define WTC_MCASE(KV)                                                        \
    case KV:                                                                 \
        switch (dt) {                                                        \
            case WTCONV_F32: return launch_mixed_t<KV, float>(a, grid, s);     \
            case WTCONV_BF16: return launch_mixed_t<KV, uint16_t>(a, grid, s); \
            case WTCONV_F16: return launch_mixed_t<KV, _Float16>(a, grid, s);  \
        }                                                                    \
        break;
    switch (k) {
        WTC_MCASE(1)
        WTC_MCASE(3)
        WTC_MCASE(5)
        WTC_MCASE(7)
        WTC_MCASE(9)
    }
#undef WTC_MCASE
    return hipErrorInvalidValue;
}

int mixed_wgs_by_regs(int k, wtconv_dtype dt, int rounds, int fallback)
{
    switch (k) {
        case 1: return mixed_wgs_k<1>(dt, rounds, fallback);
        case 3: return mixed_wgs_k<3>(dt, rounds, fallback);
        case 5: return mixed_wgs_k<5>(dt, rounds, fallback);
        case 7: return mixed_wgs_k<7>(dt, rounds, fallback);
        case 9: return mixed_wgs_k<9>(dt, rounds, fallback);
    }
    return fallback;
}

}  // namespace wtc
