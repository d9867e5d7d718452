// Host side of libwtconv: argument validation (before any HIP call), on-chip
// layout planning and kernel launches. See include/wtconv.h for the contract.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "wtconv_internal.h"

namespace {

using wtc::FusedArgs;
using wtc::kMaxLevels;
using wtc::LevelGeom;
using wtc::PlaneGeom;

constexpr int kLdsFloatsMax = 160 * 1024 / 4;     // one compute unit's LDS
constexpr int kLdsFloatsShared = 64 * 1024 / 4;   // keep >= 2 workgroups per CU when possible
// A workgroup's LDS is allocated in whole granules of 1280 bytes, 128 per
// compute unit (measured on MI355X with 256-thread workgroups: three of 53760
// bytes are resident per CU, of 53888 bytes only two; two of 81920 bytes).
constexpr int kLdsGranuleFloats = 1280 / 4;
constexpr int kLdsGranules = 128;

// Workgroups the forward aims for (whole batch chunks of a channel each).
// Measured on MI355X against 4096 (us per forward, k = 5 fp32): 56 x 56 L3
// B64 C96 67.6 -> 66.9, 28 x 28 L1 B64 C192 37.2 -> 35.0, 14 x 14 L1 B128 C384
// 41.9 -> 40.6, 63 x 95 L3 B32 C128 149.4 -> 142.6, 128 x 128 L3 B8 C128
// 134.6 -> 130.7; 56 x 56 L5 bf16 B128 167.1 -> 169.2. At 1024 the small
// planes gain more but 56 x 56 loses 19 % (too few workgroups for the tail).
constexpr int kForwardTargetWorkgroups = 2048;
constexpr int kBackwardTargetWorkgroups = 1536;
// The region backward (planes beyond one CU's LDS) aims for fewer, longer
// workgroups: each carries a larger working set, and more batch planes per
// workgroup amortise its set-up. Measured (combined backward, us, 1536 ->
// 768): 224 x 224 B16 C64 L1 401.1 -> 382.3, L3 682.9 -> 669.9; B8 C32 k = 3
// 128 x 128 L1 67.6 -> 59.1, 256 x 256 L3 292.6 -> 283.4; 512 x 512 within
// 0.1 %. 3072 was slower everywhere (up to +13 %).
constexpr int kRegionBackwardTargetWorkgroups = 768;
// The gradient route over region tiles (grad_kernel, then the rotated forward
// for dx) keeps less per workgroup and, when a region is one block round
// (k <= 5), gains from a fuller grid: measured (combined backward, us, 768 ->
// 1536, k = 5 L3): 224 x 224 B16 C64 576.0 -> 541.3 (bf16 543.2 -> 504.0),
// 128 x 128 B8 C128 280.9 -> 264.9; 256 x 256 and 512 x 512 within 1 %,
// 128 x 128 B8 C32 +1.2 %. 3072 lost up to 12 %. With two block rounds (k = 7,
// 9) 768 stays ahead: 224 x 224 B16 C64 k = 7 L3 1380.3 -> 1353.1 at 768,
// k = 9 L3 2444.8 -> 2355.2, k = 9 L1 2047.0 -> 1954.4; k = 7 128 x 128 B8
// C128 751.8 -> 765.3.
constexpr int kRegionGradTargetWorkgroups = 1536;
// A region that would take two block rounds (k = 7, 9: 56 x 56 tiles in
// 72 x 72 regions) is re-tiled at 48 x 48, whose 64 x 64 regions are one
// round at the larger target: combined backward, us, 224 x 224 B16 C64 L3
// k = 7 1350.4 -> 1257.2, k = 9 2350.5 -> 2106.3; 128 x 128 B8 C128 k = 7
// 763.0 -> 548.9; 512 x 512 B8 C32 k = 7 2299.0 -> 1848.0, k = 9 4235.0 ->
// 3368.5. The multi-round region branch stays as the fallback.
constexpr bool kRegionGradSmallTiles = true;

int ceil_to(int v, int m) { return (v + m - 1) / m * m; }
int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

// Workgroups per CU that a workgroup LDS size allows.
int lds_wgs(long lds_floats)
{
    return lds_floats <= 0 ? kLdsGranules : kLdsGranules / cdiv(lds_floats, kLdsGranuleFloats);
}

// Mixed task rounds (wtconv_mixed.hip) of a forward plan: see pack_mixed().
struct MixedPlan {
    int rounds = 0;  // 0: the plan runs fused_kernel
    int first_out = 0;
    int seg0[wtc::kMixedMaxRounds + 1] = {};
    int ntask[wtc::kMixedMaxRounds] = {};
    int out0[wtc::kMixedMaxRounds] = {};
    int seg[wtc::kMixedMaxSegs] = {};
};

struct Plan {
    PlaneGeom g;
    MixedPlan mx;
    int one_round = 0;  // every level filtered in one register-tile round per lane
    int merge_deep = 0;  // forward: levels 1 and >= 3 filtered in one round (4x4 tiles)
    int PP = 1;        // planes resident at once
    int nb = 1;        // planes per workgroup
    int nchunks = 1;   // workgroups per channel
    int lds_floats = 0;
};

int window_floats(int T, int R)
{
    const int n = T + 2 * R;
    return T == 4 ? ceil_to(n, 4) : (T == 2 ? ceil_to(n, 2) : n);
}

int round_cap(int T)
{
    return T == 4 ? wtc::kMaxRounds4 : (T == 2 ? wtc::kMaxRounds2 : wtc::kMaxRounds1);
}

// Tile edge for filtering an h x w level with PP resident planes. Each of the
// four wavefronts filters one band; a round gives every lane one T x T tile.
// Per round a wavefront issues T*T*k*k FMAs on its SIMD (4 cycles each) and
// reads a (T+k-1)-row window per lane from LDS, which all four wavefronts
// share at 128 bytes per cycle (the backward pass reads two windows). The
// tile with the smallest estimated time max(FMA, LDS) wins, larger tiles on
// ties; rounds are capped by the registers that hold in-place results.
// With one_pref, tile edges that take a single round are preferred whenever
// one exists (so that the plan can use the single-round kernel variant).
int pick_tile(int h, int w, int PP, int k, bool bwd, bool one_pref = false)
{
    const int R = k / 2;
    long best_cost = -1;
    int best = 0;
    bool one_avail = false;
    for (int T : {4, 2, 1})
        if (one_pref && (long)PP * (ceil_to(h, T) / T) * (ceil_to(w, T) / T) <= 64) one_avail = true;
    for (int T : {4, 2, 1}) {
        const long tiles = (long)PP * (ceil_to(h, T) / T) * (ceil_to(w, T) / T);
        const long rounds = cdiv(tiles, 64);
        if (rounds > round_cap(T) || (one_avail && rounds > 1)) continue;
        const long fma_cycles = rounds * T * T * k * k * 4;
        const long lds_bytes = rounds * wtc::kWaves * (bwd ? 2 : 1) * (T + 2 * R) * window_floats(T, R) * 4 * 64;
        const long cost = std::max(fma_cycles, lds_bytes / 128);
        if (best_cost < 0 || cost < best_cost) {
            best_cost = cost;
            best = T;
        }
    }
    return best;
}

void set_tile_lanes(PlaneGeom& g, int lanes)
{
    g.tiles_xl = lanes;
    g.r_tiles_xl = 1.0f / (float)lanes;
    g.r_tiles_l = 1.0f / (float)(lanes * g.tiles_y);
}

// Lay out one plane's input array and pyramid for a given number of resident
// planes. Returns false if a level cannot be tiled within the register caps.
// rows_from: the first level whose kernel-gradient correlation walks whole
// rows (the fused backward and the gradient pass: 2);
// those levels' rows are padded to whole row chunks.
// share_halo: the four band arrays of a level share their zero halo rows
// (band q's last R rows are band q + 1's first R: both are zeros that nothing
// writes, and every window or row read of band q ends within them). Forward
// plans also pass rows_from = kMaxLevels + 1: only the backward runs the
// kernel-gradient row chunks that the row padding is for.
// t1_max: the largest tile edge level 1 may take (the gradient pass tries 2).
// pitch2: levels filtered in 2 x 2 or single-site tiles (8-byte and 4-byte
// LDS reads, forward only) get rows padded to 2 floats instead of 4; every
// level still starts 16-byte aligned. Smaller, but rows starting on odd
// float pairs cost 0.5-3 % in bank conflicts, and offered to the plan search
// it traded workgroups for planes badly (12 x 12 L = 3 +28 %, 14 x 14 L = 4
// +20 %), so only the merge of the deep levels below uses it.
bool layout(const wtconv_desc& d, int PP, bool bwd, PlaneGeom& g, bool t4_deep = false, bool one_pref = false,
            int rows_from = 2, bool t4_all = false, bool share_halo = false, int t1_max = 4, bool pitch2 = false)
{
    const int R = d.k / 2;
    memset(&g, 0, sizeof(g));
    g.H = d.H;
    g.W = d.W;
    g.L = d.L;
    g.xrows = ceil_to(d.H, 4) + 2 * R;
    g.xpitch = ceil_to(d.W, 4) - 4 + ceil_to(4 + 2 * R, 4);
    g.tiles_x = ceil_to(d.W, 4) / 4;
    g.tiles_y = ceil_to(d.H, 4) / 4;
    long off = (long)g.xrows * g.xpitch;
    int h = d.H, w = d.W;
    for (int l = 1; l <= d.L; ++l) {
        h = (h + 1) / 2;
        w = (w + 1) / 2;
        LevelGeom& lg = g.lv[l];
        lg.h = h;
        lg.w = w;
        lg.T = (t4_all || (t4_deep && l >= 3)) ? 4 : pick_tile(h, w, PP, d.k, bwd, one_pref);
        if (l == 1 && lg.T > t1_max) lg.T = t1_max;
        if (lg.T == 0) return false;
        lg.eh = ceil_to(h, lg.T);
        lg.ew = ceil_to(w, lg.T);
        const int rows = R + std::max(lg.eh + R, h + 1);
        int pitch = std::max(lg.ew - lg.T + window_floats(lg.T, R), R + std::max(lg.ew + R, w + 1));
        if (l >= rows_from) {  // whole-row chunks of the coarse kernel-gradient pass stay inside the row
            const int cw = wtc::row_chunk(w);
            pitch = std::max(pitch, ceil_to(w, cw) - cw + ceil_to(cw + 2 * R, 4));
        }
        lg.pitch = ceil_to(pitch, (pitch2 && lg.T < 4) ? 2 : 4);
        const int shared = share_halo ? R : 0;  // halo rows a band shares with the next
        lg.band = (rows - shared) * lg.pitch;
        lg.off = (int)off;
        lg.r_w = 1.0f / (float)w;
        lg.r_hw = 1.0f / (float)(h * w);
        lg.r_tx = 1.0f / (float)(lg.ew / lg.T);
        lg.r_tper = 1.0f / (float)((lg.ew / lg.T) * (lg.eh / lg.T));
        off += 4L * lg.band + (long)shared * lg.pitch;
        off = (off + 3) / 4 * 4;  // the next level's rows start 16-byte aligned
        if (off > (1L << 30)) return false;
    }
    g.plane_floats = (int)off;
    g.r_W = 1.0f / (float)d.W;
    g.r_tiles_x = 1.0f / (float)g.tiles_x;
    g.r_tiles = 1.0f / (float)(g.tiles_x * g.tiles_y);
    set_tile_lanes(g, g.tiles_x);
    // flat indices decomposed with fp32 reciprocals must stay below 2^20
    if ((long)PP * g.tiles_x * g.tiles_y * 16 >= (1L << 20)) return false;
    return true;
}

int lds_floats_for(const wtconv_desc& d, bool bwd, int PP, const PlaneGeom& g)
{
    const int KK = d.k * d.k;
    const int wt = ceil_to((1 + 4 * d.L) * KK, 4);
    const int gc = bwd ? ceil_to(d.L * 4 * KK, 4) : 0;
    const long planes = std::max((long)PP * (bwd ? 2 : 1) * g.plane_floats, (long)4 * wtc::kWaves * KK);
    const long total = wt + gc + ceil_to((int)std::min(planes, 1L << 30), 4);
    return total > (1L << 30) ? (1 << 30) : (int)total;
}

// Single-round variant: one 4x4 block / output tile per thread and one
// register tile per lane for every level.
bool single_round(const wtconv_desc& d, int PP, const PlaneGeom& g)
{
    if ((long)PP * g.tiles_x * g.tiles_y > wtc::kThreads) return false;
    for (int l = 1; l <= d.L; ++l) {
        const LevelGeom& lg = g.lv[l];
        if ((long)PP * (lg.eh / lg.T) * (lg.ew / lg.T) > 64) return false;
    }
    return true;
}

// Workgroups (4 wavefronts) per CU that the forward kernel's registers allow:
// 512 registers per SIMD lane over the kernel's VGPR count, queried from the
// HIP runtime for the compiled kernel. Without a device to ask, the counts of
// one gfx950 build stand in (single round: 55 / 63-68 / 100-103 / 147-148
// VGPRs for k = 1 / 3 / 5 / 7; general: 123 / 137 / 148-149 / 173); the
// forward workspace size does not depend on this choice.
int forward_wgs(const wtconv_desc& d, bool one)
{
    const int k = d.k;
    const int fallback = one ? (k <= 1 ? 8 : (k <= 3 ? 7 : (k <= 5 ? 4 : 3))) : (k <= 1 ? 4 : (k <= 5 ? 3 : 2));
    return wtc::forward_wgs_by_regs(k, d.dtype, one, fallback);
}

// Lane use of one workgroup's output-tile rounds with PP resident planes.
double tile_use(const PlaneGeom& g, int PP)
{
    const long nt = (long)PP * g.tiles_x * g.tiles_y;
    return (double)nt / ((double)wtc::kThreads * cdiv(nt, wtc::kThreads));
}

// ----------------------------------------------------------------------------
// Mixed task rounds (forward, resident planes; wtconv_mixed.hip). The output
// tiles and the 4x4 site tiles of every (level, band) are equal tasks of 16
// k^2 FMAs, dealt to 256 lanes per round. Whole (level, band) groups are packed
// into rounds first-fit by decreasing size (a group's tiles share a round: its
// band is written in place after that round's barrier, and no other round
// reads it); the output tiles then fill the rounds from the last one holding a
// group on (they need every level filtered). Fails if a group exceeds a round,
// or more than kMixedMaxRounds rounds are needed.
// ----------------------------------------------------------------------------
bool pack_mixed(const wtconv_desc& d, int PP, const PlaneGeom& g, MixedPlan& mp)
{
    constexpr int cap = wtc::kThreads;
    constexpr int RM = wtc::kMixedMaxRounds;
    struct Grp {
        int l, q, n;
    };
    Grp grp[4 * kMaxLevels];
    int ng = 0;
    for (int l = 1; l <= d.L; ++l) {
        const LevelGeom& lg = g.lv[l];
        if (lg.T != 4) return false;
        const long n = (long)PP * (lg.eh / 4) * (lg.ew / 4);
        if (n > cap) return false;
        for (int q = 0; q < 4; ++q) grp[ng++] = {l, q, (int)n};
    }
    std::stable_sort(grp, grp + ng, [](const Grp& a, const Grp& b) { return a.n > b.n; });
    int used[RM] = {};
    int rnd[4 * kMaxLevels] = {};
    int nr = 0;  // rounds holding groups
    for (int i = 0; i < ng; ++i) {
        int r = 0;
        while (r < nr && used[r] + grp[i].n > cap) ++r;
        if (r == RM) return false;
        if (r == nr) ++nr;
        used[r] += grp[i].n;
        rnd[i] = r;
    }
    const int F = nr > 0 ? nr - 1 : 0;
    long left = (long)PP * g.tiles_x * g.tiles_y;
    int outs[RM] = {};
    int r = F;
    for (; left > 0; ++r) {
        if (r >= RM) return false;
        const int take = (int)std::min<long>(left, cap - used[r]);
        outs[r] = take;
        used[r] += take;
        left -= take;
    }
    const int rounds = std::max(nr, r);
    int ns = 0, out0 = 0;
    for (int rr = 0; rr < rounds; ++rr) {
        mp.seg0[rr] = ns;
        mp.ntask[rr] = used[rr];
        mp.out0[rr] = out0;
        for (int i = 0; i < ng; ++i)
            if (rnd[i] == rr) mp.seg[ns++] = 2 | (grp[i].l << 2) | (grp[i].q << 6) | (grp[i].n << 8);
        if (outs[rr] > 0) mp.seg[ns++] = 1 | (outs[rr] << 8);
        out0 += outs[rr];
    }
    mp.seg0[rounds] = ns;
    mp.rounds = rounds;
    mp.first_out = F;
    return true;
}

// Modeled FMA issue per wavefront and resident plane of a forward plan, in
// FMAs per lane: a round of T x T site tiles costs T^2 k^2 on every lane of
// the wavefronts it occupies (masked lanes included).
double issue_fused(const wtconv_desc& d, int PP, const PlaneGeom& g, bool merged)
{
    const int KK = d.k * d.k;
    double c = (double)cdiv((long)PP * g.tiles_x * g.tiles_y, wtc::kThreads) * 16 * KK;
    for (int l = 1; l <= d.L; ++l) {
        const LevelGeom& lg = g.lv[l];
        if (merged && l != 2) {
            if (l == 1) c += 16.0 * KK;  // level 1 and the levels from 3 on: one round
            continue;
        }
        c += (double)cdiv((long)PP * (lg.eh / lg.T) * (lg.ew / lg.T), 64) * lg.T * lg.T * KK;
    }
    return c / PP;
}

double issue_mixed(const wtconv_desc& d, int PP, const MixedPlan& mp)
{
    return (double)mp.rounds * 16 * d.k * d.k / PP;
}

// Workgroups per CU that the mixed kernel's registers allow (queried from the
// runtime; without a device, the counts of one gfx950 build stand in: 75-125
// VGPRs over k = 1..7 and one to four rounds).
int mixed_wgs(const wtconv_desc& d, int rounds)
{
    return wtc::mixed_wgs_by_regs(d.k, d.dtype, rounds, d.k <= 3 ? 5 : 4);
}

// The mixed variant replaces a forward plan for planes of at most 16 x 16
// pixels (level 1 at most 8 x 8) when its modeled issue per plane is at most
// this fraction of the plan's and it keeps enough workgroups per CU. Measured
// on MI355X (k = 5 fp32 unless noted, us per forward, fused -> mixed): 14 x 14
// B128 C384 L1 46.0 -> 41.9, L2 73.2 -> 53.7, the split L3 76.1 -> 72.2, k = 7
// L3 115.5 -> 95.8; 16 x 16 B128 C384 L1 41.3 -> 38.4, L2 67.5 -> 49.2; 15 x 15
// and 13 x 13 at B128 C192 4-6 % faster; with fewer planes (B * C = 12288 or
// 24576) within 1 %. On larger planes the fused kernel's lane use is already
// 80-90 % and the extra barriers cost more than the mixed rounds save: 56 x 56
// L3 B64 C96 68.0 -> 69.2, 20 x 20 L3 36.3 -> 41.5, 63 x 95 L3 149.7 -> 176.9.
constexpr double kMixedGain = 0.95;
constexpr int kMixedMaxEdge = 16;

bool make_plan(const wtconv_desc& d, bool bwd, Plan& pl, bool allow_mixed = true)
{
    const long px = (long)ceil_to(d.H, 4) * ceil_to(d.W, 4);
    int want = std::max(1, cdiv(4096, px));  // aim for >= 256 output tiles per workgroup
    want = std::min(want, d.B);
    int PP = 0;
    for (int pp = want; pp >= 1; --pp) {
        PlaneGeom g;
        if (!layout(d, pp, bwd, g, false, false, bwd ? 2 : kMaxLevels + 1, false, !bwd)) continue;
        const int lds = lds_floats_for(d, bwd, pp, g);
        if (lds <= kLdsFloatsShared || (pp == 1 && lds <= kLdsFloatsMax)) {
            PP = pp;
            pl.g = g;
            pl.lds_floats = lds;
            break;
        }
    }
    if (PP == 0) return false;
    // Forward: every plane count up to one round of output tiles (or the
    // count above), in the default tile layout and in one preferring
    // single-round tiles, scored by output-tile lane use x workgroups per CU
    // (registers and LDS), the general kernel variant at 3/4 (its round loops);
    // more planes on ties. Measured on MI355X (us per forward, k = 5, B64 C192
    // 28 x 28 unless noted): L = 1 6 planes 54.5 -> 4 single-round 40.6; L = 3
    // 4 planes 64.7 -> 3 single-round 61.3; L = 4 70.0 -> 62.0; B128 56 x 56
    // L = 1 2 planes 153.6 -> 1 single-round 121.1; 40 x 40 k = 7 L = 4 155.9 ->
    // 81.4.
    bool pref_used = false;
    if (!bwd) {
        const long tiles = px / 16;
        const int ppmax = std::max(PP, (int)std::min<long>(d.B, wtc::kThreads / tiles));
        double best = -1.0;
        for (int pp = 1; pp <= ppmax; ++pp)
            for (int pref = 0; pref < 2; ++pref) {
                PlaneGeom g;
                if (!layout(d, pp, bwd, g, false, pref == 1, kMaxLevels + 1, false, true)) continue;
                const int lds = lds_floats_for(d, bwd, pp, g);
                if (lds > kLdsFloatsMax) continue;
                const bool one = single_round(d, pp, g);
                const int wgs = std::min(forward_wgs(d, one), lds_wgs(lds));
                const double score = tile_use(g, pp) * wgs * (one ? 1.0 : 0.75);
                if (score >= best) {
                    best = score;
                    PP = pp;
                    pl.g = g;
                    pl.lds_floats = lds;
                    pref_used = pref == 1;
                }
            }
    }
    pl.PP = PP;
    pl.one_round = single_round(d, PP, pl.g) ? 1 : 0;
    // Forward, single round, level 1 in 4x4 tiles and at least three levels:
    // the levels from 3 on (small grids, each otherwise a round of its own
    // with a handful of busy lanes) take 4x4 tiles too and share level 1's
    // round on the lanes level 1 leaves idle, if they fit (measured on MI355X:
    // the 7x7 level 3 of a 56x56 plane cost 5 us of a 73 us forward on its own).
    // It is taken if it keeps the workgroups per CU of the unmerged layout
    // (registers and LDS), with the even row padding if that is what keeps
    // them. Measured on MI355X (us per forward, k = 5): B128 C96 56 x 56 L = 5
    // 153.6 -> 137.0 (bf16 154.1 -> 136.2; merged it needs 10272 floats with
    // 4-float rows, past the 10240 of four workgroups, and 10140 with 2-float
    // rows); B64 C96 48 x 48 L = 5 79.0 -> 70.2 and 45 x 45 89.5 -> 78.3 (5
    // workgroups' LDS down to 4, which the registers allow anyway). Merged at
    // one workgroup fewer it was slower: 56 x 56 L = 5 +4.6 %, k = 7 40 x 40
    // L = 3 +12 %.
    if (!bwd && pl.one_round && d.L >= 3 && pl.g.lv[1].T == 4) {
        const int reg_wgs = forward_wgs(d, true);
        for (int p2 = 0; p2 < 2 && !pl.merge_deep; ++p2) {
            PlaneGeom gm;
            if (!layout(d, PP, bwd, gm, true, pref_used, kMaxLevels + 1, false, true, 4, p2 == 1)) continue;
            long lanes = (long)PP * (gm.lv[1].eh / 4) * (gm.lv[1].ew / 4);
            for (int l = 3; l <= d.L; ++l) lanes += (long)PP * (gm.lv[l].eh / 4) * (gm.lv[l].ew / 4);
            const int lds = lds_floats_for(d, bwd, PP, gm);
            if (lanes <= 64 && lds <= kLdsFloatsMax &&
                std::min(reg_wgs, lds_wgs(lds)) >= std::min(reg_wgs, lds_wgs(pl.lds_floats))) {
                pl.g = gm;
                pl.lds_floats = lds;
                pl.merge_deep = 1;
            }
        }
    }
    // Forward: the mixed task rounds, at the plane count that minimises their
    // modeled issue (more workgroups per CU on ties), if they beat the plan.
    if (!bwd && allow_mixed && d.L >= 1 && d.H <= kMixedMaxEdge && d.W <= kMixedMaxEdge) {
        const double cost_f = issue_fused(d, PP, pl.g, pl.merge_deep != 0);
        const int wgs_f = std::min(forward_wgs(d, pl.one_round != 0), lds_wgs(pl.lds_floats));
        const long tiles = (long)ceil_to(d.H, 4) * ceil_to(d.W, 4) / 16;
        const int ppmax = (int)std::max(1L, std::min<long>(d.B, (long)wtc::kMixedMaxRounds * wtc::kThreads / tiles));
        double best = -1.0;
        int best_wgs = 0;
        Plan mp;
        for (int pp = 1; pp <= ppmax; ++pp) {
            PlaneGeom g;
            if (!layout(d, pp, false, g, false, false, kMaxLevels + 1, true, true)) continue;
            MixedPlan m;
            if (!pack_mixed(d, pp, g, m)) continue;
            const int KP = ceil_to(d.k * d.k, 4);
            const long lds = (long)(1 + 4 * d.L) * KP + (long)pp * g.plane_floats;
            if (lds > kLdsFloatsMax) continue;
            const int wgs = std::min(mixed_wgs(d, m.rounds), lds_wgs(lds));
            // only plane counts that keep the workgroups per CU of the plan
            // compete (the cheapest count overall may not, and used to veto
            // the mixed rounds altogether: B128 C192 12 x 12 L = 2 forward
            // 30.3 -> 24.2 us, L = 3 34.5 -> 28.5, 10 x 10 L = 3 35.4 ->
            // 30.1, 9 x 9 L = 2 B64 21.2 -> 18.1, k = 3 B128 C384 14 x 14
            // L = 3 58.6 -> 49.3)
            if (wgs < std::min(wgs_f, 3)) continue;
            const double cost = issue_mixed(d, pp, m);
            if (best < 0 || cost < best || (cost == best && wgs > best_wgs)) {
                best = cost;
                best_wgs = wgs;
                mp.g = g;
                mp.mx = m;
                mp.PP = pp;
                mp.lds_floats = (int)lds;
            }
        }
        if (best >= 0 && best <= kMixedGain * cost_f) {
            pl.g = mp.g;
            pl.mx = mp.mx;
            pl.PP = PP = mp.PP;
            pl.lds_floats = mp.lds_floats;
            pl.one_round = 0;
            pl.merge_deep = 0;
        }
    }
    // Forward, single round: the rows of output tiles (and of the blocks the
    // threads load) padded to a multiple of 8 lanes, so that every group of 8
    // lanes of a 16-byte LDS access stays inside one tile row, when that keeps
    // one round and does not put work on more wavefronts. Measured on MI355X
    // (us per forward, k = 5): 56 x 56 L3 B64 C96 68.3 -> 66.6 (LDS bank
    // conflict cycles -16 %), 28 x 28 L1 B64 C192 35.4 -> 34.4, k = 3 56 x 56
    // L1 B128 79.7 -> 77.4; 12 x 12 L3, where it spread 63 tiles over three
    // wavefronts instead of one, 55.7 -> 57.9 (hence the condition). Padding
    // the subband tiles of the filter stage the same way changed nothing.
    if (!bwd && pl.one_round && pl.mx.rounds == 0) {
        const int xl = ceil_to(pl.g.tiles_x, 8);
        const long n = (long)PP * pl.g.tiles_y * pl.g.tiles_x, npad = (long)PP * pl.g.tiles_y * xl;
        if (npad <= wtc::kThreads && cdiv(npad, 64) == cdiv(n, 64)) set_tile_lanes(pl.g, xl);
    }
    const int target = bwd ? kBackwardTargetWorkgroups : kForwardTargetWorkgroups;
    const int chunks_target = std::max(1, cdiv(target, d.C));
    int nb = ceil_to(cdiv(d.B, chunks_target), PP);
    if (bwd) nb = std::max(nb, std::min(ceil_to(4, PP), ceil_to(d.B, PP)));
    pl.nb = nb;
    pl.nchunks = cdiv(d.B, nb);
    return true;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb)
{
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
    return pa < pb + nb && pb < pa + na;
}

size_t elem_size(wtconv_dtype dt) { return dt == WTCONV_F32 ? 4 : 2; }
size_t align256(size_t n) { return (n + 255) / 256 * 256; }

wtconv_status check_desc(const wtconv_desc* d)
{
    if (!d) return WTCONV_ERR_NULL;
    if (d->B < 1 || d->C < 1 || d->H < 1 || d->W < 1) return WTCONV_ERR_SHAPE;
    if ((long)d->H * d->W > (1L << 30) || (long)d->B * d->C > (1L << 30) ||
        (long)d->C * 4 * 49 > (1L << 30) || (long)d->B * d->C * d->H * d->W > (1L << 40))
        return WTCONV_ERR_SHAPE;
    if (d->k < 1 || d->k > 9 || (d->k % 2) == 0) return WTCONV_ERR_KSIZE;
    if (d->L < 0 || d->L > WTCONV_MAX_LEVELS) return WTCONV_ERR_LEVELS;
    if (d->dtype != WTCONV_F32 && d->dtype != WTCONV_BF16 && d->dtype != WTCONV_F16) return WTCONV_ERR_DTYPE;
    return WTCONV_OK;
}

wtconv_status check_levels(int L, const float* const* lw, const float* const* ls)
{
    if (L == 0) return WTCONV_OK;
    if (!lw || !ls) return WTCONV_ERR_NULL;
    for (int l = 0; l < L; ++l)
        if (!lw[l] || !ls[l]) return WTCONV_ERR_NULL;
    return WTCONV_OK;
}

void fill_params(wtc::ParamPtrs& p, int L, const float* w0, const float* s0, const float* b0, const float* const* lw,
                 const float* const* ls)
{
    memset(&p, 0, sizeof(p));
    p.w0 = w0;
    p.s0 = s0;
    p.b0 = b0;
    for (int l = 0; l < L; ++l) {
        p.lw[l] = lw[l];
        p.ls[l] = ls[l];
    }
}

// Parameter gradient destinations (device pointers).
struct Grads {
    float* dw0;
    float* ds0;
    float* db0;  // nullable
    float* dlw[kMaxLevels];
    float* dls[kMaxLevels];
};

// The same parameters, levels shifted by m: the coarse sub-problem's level l
// is the full problem's level l + m.
wtc::ParamPtrs shift_params(const wtc::ParamPtrs& p, int m)
{
    wtc::ParamPtrs s = p;
    for (int l = 0; l < kMaxLevels; ++l) {
        s.lw[l] = l + m < kMaxLevels ? p.lw[l + m] : nullptr;
        s.ls[l] = l + m < kMaxLevels ? p.ls[l + m] : nullptr;
    }
    return s;
}

Grads shift_grads(const Grads& g, int m)
{
    Grads s = g;
    for (int l = 0; l < kMaxLevels; ++l) {
        s.dlw[l] = l + m < kMaxLevels ? g.dlw[l + m] : nullptr;
        s.dls[l] = l + m < kMaxLevels ? g.dls[l + m] : nullptr;
    }
    return s;
}

int vec_ok(const void* a, const void* b, const void* c)
{
    const uintptr_t m = 15;  // 16-byte loads of the input planes
    return (((uintptr_t)a & m) == 0 && ((uintptr_t)b & m) == 0 && ((uintptr_t)c & m) == 0) ? 1 : 0;
}

// ----------------------------------------------------------------------------
// Execution choice. A problem runs in one of four ways:
//   tiny     planes of at most 8 x 8 pixels: wtconv_tiny.hip, one lane per
//            batch entry, every level in registers;
//   resident one fused pass per plane resident in LDS (wtconv_kernels.hip);
//   split    resident, but the levels above m (the first level whose grid is
//            at most 8 x 8) are a coarse sub-problem: the coarse branch is
//            exactly the WTConv, without base path, of the level-m raw LL
//            carrier X_m (2^-m times each 2^m x 2^m block sum), whose output
//            is the coarse levels' contribution at the level-m grid and whose
//            input gradient is the same contribution for dx; its kernel
//            gradients are those of levels m+1..L. The carrier is tiny, and
//            the fused pass then runs levels 1..m only and adds the carry at
//            level m. The deepest levels are the least efficient part of the
//            fused pass (a few sites per band, one barrier-separated step each,
//            and the largest LDS footprint), so this trades one extra read of
//            the input for them;
//   region   planes too large for LDS: the same split at m = 1 (the sub-
//            problem recurses until it fits), with the base path and level 1
//            run on 56 x 56 (or smaller) output tiles with a halo of 2R pixels
//            (the level-1 receptive field).
// ----------------------------------------------------------------------------
struct RegionPlan {
    Plan pl;
    int T = 0, h = 0, ntx = 0, nty = 0;
};

bool make_region_plan(const wtconv_desc& d, bool bwd, RegionPlan& rp, int target = 0, int t_max = 56)
{
    // the carrier kernel decomposes small offsets with fp32 reciprocals
    if (d.H >= (1 << 19) || d.W >= (1 << 19)) return false;
    const int R = d.k / 2;
    const int m = d.L > 0 ? 1 : 0;
    rp.h = ceil_to(m ? 2 * R : R, 4);
    for (int T : {56, 48, 40, 32, 24, 16, 8}) {
        if (T > t_max) continue;
        wtconv_desc rd = d;
        rd.B = 1;  // one region resident at a time
        rd.H = rd.W = T + 2 * rp.h;
        rd.L = m;
        Plan pl;
        if (!make_plan(rd, bwd, pl, false) || pl.PP != 1) continue;
        rp.T = T;
        rp.ntx = cdiv(d.W, T);
        rp.nty = cdiv(d.H, T);
        const long ntiles = (long)rp.ntx * rp.nty;
        if (target <= 0) target = bwd ? kRegionBackwardTargetWorkgroups : kForwardTargetWorkgroups;
        const long chunks_target = std::max(1L, (target + d.C * ntiles - 1) / (d.C * ntiles));
        pl.nb = (int)((d.B + chunks_target - 1) / chunks_target);
        pl.nchunks = cdiv(d.B, pl.nb);
        if (bwd) pl.one_round = 0;  // the forward keeps its single-round variant
        if ((long)pl.nchunks * ntiles * d.C > INT32_MAX) return false;  // grid size
        rp.pl = pl;
        return true;
    }
    return false;
}

enum class Mode { Tiny, Resident, Split, Region, None };

struct Exec {
    Mode mode = Mode::None;
    Plan pl;         // resident / split: the fused pass (split: levels 1..m)
    RegionPlan rp;   // region
    int m = 0;       // split / region: levels run by the fused pass
    bool coarse = false;  // split / region: a coarse sub-problem exists (L > m)
};

// Planes of at most 8 x 8 run one plane per lane, unless the tiny backward's
// LDS (staging rows plus every folded kernel of four channels) would not fit:
// k = 9 with L >= 6; those planes run resident like larger ones.
bool use_tiny(const wtconv_desc& d)
{
    return d.H <= wtc::kTinyMaxEdge && d.W <= wtc::kTinyMaxEdge &&
           wtc::tiny_lds_bytes(d.k, d.L, true) <= (size_t)wtc::kLdsBytesMax;
}
int tiny_groups(const wtconv_desc& d) { return cdiv(d.B, 64); }

// The first level whose grid is at most 8 x 8.
int tiny_level(const wtconv_desc& d)
{
    int m = 0, h = d.H, w = d.W;
    while (h > wtc::kTinyMaxEdge || w > wtc::kTinyMaxEdge) {
        h = (h + 1) / 2;
        w = (w + 1) / 2;
        ++m;
    }
    return m;
}

// Whether a resident problem runs its levels above m as a tiny sub-problem
// (measured on MI355X at the ConvNeXt-T shapes). The split costs one extra
// read of the input per pass (two in the backward) plus the tiny kernel; in
// the forward it pays when the fused pass loses at least three deep levels,
// and in the backward pass when it sheds any level above m = 1 or two above
// a deeper m, or when it brings the workgroup's LDS under the two-per-CU mark.
// The tiny kernel runs one lane per plane, so with few planes it cannot fill
// the chip: a forward split at m = 1 (planes of at most 16 x 16, whose whole
// pass runs in mixed task rounds) needs B * C >= 32768 (B * C / 64 = 512
// wavefronts). Measured forwards, k = 5, split against whole (us): 14 x 14 at
// B128 C384, L = 3 70.6 / 64.2 (bf16 72.6 / 63.4), L = 4 71.4 / 87.0, L = 5
// 72.4 / 96.9; L = 5 at B64 C384 66.1 / 60.3, 16 x 16 at B64 C192 65.3 /
// 59.4, 12 x 12 at B128 C192 80.1 / 74.6.
constexpr long kSplitMinPlanes = 32768;

bool want_split(const wtconv_desc& d, bool bwd, int m, int full_lds, int split_lds)
{
    if (m < 1 || m > 6 || d.L <= m) return false;
    const int deep = d.L - m;
    if (!bwd) return deep >= 3 && (m > 1 || (long)d.B * d.C >= kSplitMinPlanes);
    return m == 1 || deep >= 2 || (lds_wgs(full_lds) < 2 && lds_wgs(split_lds) >= 2);
}

// Plans by descriptor. The plan search costs tens of microseconds of host
// time for small planes (every resident-plane count, tile layout and
// mixed-round packing is tried), as long as the kernels it plans: uncached,
// a loop of 12 x 12 forwards left the GPU waiting on it. A fixed table of the
// last kSlots descriptors, replaced round-robin; lookups and inserts hold a
// mutex, the search runs outside it (two threads that miss on the same
// descriptor compute the same plan). Plans depend only on the descriptor and
// on the compiled kernels' register counts.
template <typename V>
class PlanCache {
  public:
    template <typename F>
    V get(const wtconv_desc& d, int tag, F compute)
    {
        const Key key = {{d.B, d.C, d.H, d.W, d.k, d.L, (int)d.dtype, tag}};
        {
            std::lock_guard<std::mutex> lock(mu_);
            for (int i = 0; i < n_; ++i)
                if (keys_[i] == key) return vals_[i];
        }
        const V v = compute();
        std::lock_guard<std::mutex> lock(mu_);
        const int slot = n_ < kSlots ? n_++ : (int)(next_++ % kSlots);
        keys_[slot] = key;
        vals_[slot] = v;
        return v;
    }

  private:
    struct Key {
        int v[8];
        bool operator==(const Key& o) const { return memcmp(v, o.v, sizeof(v)) == 0; }
    };
    static constexpr int kSlots = 64;
    std::mutex mu_;
    Key keys_[kSlots];
    V vals_[kSlots];
    int n_ = 0;
    unsigned next_ = 0;
};

Exec choose_uncached(const wtconv_desc& d, bool bwd);
bool region_grad_one_round(const wtconv_desc& d, const Exec& ex);

Exec choose(const wtconv_desc& d, bool bwd)
{
    static PlanCache<Exec> cache;
    return cache.get(d, bwd ? 1 : 0, [&] { return choose_uncached(d, bwd); });
}

Exec choose_uncached(const wtconv_desc& d, bool bwd)
{
    Exec ex;
    if (use_tiny(d)) {
        ex.mode = Mode::Tiny;
        return ex;
    }
    // A forward whose resident plane would leave one workgroup per CU runs in
    // regions instead, whose single-round passes fit four: measured (us per
    // forward, k = 5, B16 C64) 112 x 112 L1 76.7 -> 40.5, L3 93.3 -> 75.0;
    // 96 x 96 L1 58.3 -> 38.8, L3 73.7 -> 66.2. At two workgroups per CU the
    // resident plane stays ahead (63 x 95 L3 136.6 against 196.9, 84 x 84 L3
    // 37.0 against 61.9).
    if (make_plan(d, bwd, ex.pl) &&
        (bwd || lds_wgs(ex.pl.lds_floats) >= 2 || !make_region_plan(d, bwd, ex.rp))) {
        const int m = tiny_level(d);
        if (m >= 1 && d.L > m) {
            wtconv_desc f = d;
            f.L = m;
            Plan sp;
            if (make_plan(f, bwd, sp) && want_split(d, bwd, m, ex.pl.lds_floats, sp.lds_floats)) {
                ex.pl = sp;
                ex.mode = Mode::Split;
                ex.m = m;
                ex.coarse = true;
                return ex;
            }
        }
        ex.mode = Mode::Resident;
        return ex;
    }
    if (make_region_plan(d, bwd, ex.rp)) {
        ex.mode = Mode::Region;
        ex.m = d.L > 0 ? 1 : 0;
        ex.coarse = d.L >= 2;
        // the tile edge does not depend on the target, only the batch chunks
        if (bwd && region_grad_one_round(d, ex)) {
            make_region_plan(d, bwd, ex.rp, kRegionGradTargetWorkgroups);
        } else if (bwd && kRegionGradSmallTiles) {
            Exec alt = ex;
            if (make_region_plan(d, bwd, alt.rp, kRegionGradTargetWorkgroups, 48) && region_grad_one_round(d, alt))
                ex = alt;
        }
    }
    return ex;
}

// ----------------------------------------------------------------------------
// Kernel-gradient pass of the backward (wtconv_grad.hip). When it is used, dx
// is the forward pass on dy with rotated kernels and grad_kernel forms every
// kernel gradient. It needs every batch of resident planes to load at most
// one 4x4 block per thread; otherwise the fused backward runs.
// ----------------------------------------------------------------------------
struct GradPlan {
    PlaneGeom g;  // x side (zero-haloed)
    int tail0 = 0, tail1 = 0;  // x-plane floats past dy level 1 that hold deeper dy levels
    int dy_off[kMaxLevels + 1] = {}, dy_pitch[kMaxLevels + 1] = {}, dy_band[kMaxLevels + 1] = {};
    int stride = 0, PP = 1, nb = 1, nchunks = 1, lds_floats = 0;
    int rounds = 1;  // 4x4 block rounds per plane (more than one only with PP = 1)
};

int grad_gc_floats(const wtconv_desc& d)
{
    const int rl = wtc::grad_reg_levels(d.L >= 4);
    return d.L > rl ? ceil_to((d.L - rl) * 4 * d.k * d.k, 4) : 0;
}

// Compact dy pyramid next to the x side. A level's array covers the sites its
// tiles read (tile-aligned extents), the sites the block loads write (levels 1
// and 2), the sources of the next level's butterflies and, for levels >= 2,
// whole row chunks of the row-wise correlation. Level 1 is stored over the x
// plane when it fits and the block loads write every site that is read.
bool grad_layout(const wtconv_desc& d, int PP, GradPlan& gp, int t1_max = 4)
{
    // storing dy level 1 over the x plane costs a re-zeroing of the x plane's
    // halo ring per batch; it pays for large planes (one resident plane), where
    // it decides the number of workgroups per CU
    const bool may_alias = PP == 1;
    if (!layout(d, PP, true, gp.g, false, false, 2, false, false, t1_max)) return false;
    const PlaneGeom& g = gp.g;
    const long xplane = (long)g.xrows * g.xpitch;
    long extra = 0;
    long xfree = -1;  // with dy level 1 over the x plane: the first float of the x plane it leaves free
    for (int l = 1; l <= d.L; ++l) {
        const LevelGeom& lg = g.lv[l];
        int rows = std::max(lg.eh, l == 1 ? 2 * g.tiles_y : (l == 2 ? g.tiles_y : lg.h));
        int cols = std::max(lg.ew, l == 1 ? 2 * g.tiles_x : (l == 2 ? g.tiles_x : lg.w));
        if (l < d.L) {
            rows = std::max(rows, 2 * g.lv[l + 1].h);
            cols = std::max(cols, 2 * g.lv[l + 1].w);
        }
        if (l >= 2) cols = std::max(cols, ceil_to(lg.w, wtc::row_chunk(lg.w)));
        const int pitch = ceil_to(cols, 4);
        const long size = 4L * rows * pitch;
        gp.dy_pitch[l] = pitch;
        gp.dy_band[l] = rows * pitch;
        if (l == 1 && may_alias && size <= xplane && lg.eh <= 2 * g.tiles_y && lg.ew <= 2 * g.tiles_x) {
            gp.dy_off[l] = 0;
            xfree = size;
        } else if (l >= 3 && xfree >= 0 && xfree + size <= xplane) {
            // the x plane is dead once dy level 1 is written over it (every
            // dy level is written after the base correlation has read it), and
            // the next batch's block loads and halo re-zeroing rewrite all of it;
            // the kernel clears this tail in the phase that writes dy levels 1-2,
            // before levels >= 3 are built in it (after a barrier), so that their
            // sites past the grid read as zero
            if (gp.tail1 == 0) gp.tail0 = (int)xfree;
            gp.dy_off[l] = (int)xfree;
            xfree += size;
            gp.tail1 = (int)xfree;
        } else {
            gp.dy_off[l] = (int)(g.plane_floats + extra);
            extra += size;
        }
        if (g.plane_floats + extra > (1L << 28)) return false;
    }
    gp.stride = (int)(g.plane_floats + extra);
    const long planes = std::max((long)PP * gp.stride, 24L * d.k * d.k + 4);  // also the final reduction scratch
    const long total = grad_gc_floats(d) + ceil_to((int)std::min(planes, 1L << 28), 4);
    if (total > kLdsFloatsMax) return false;
    gp.lds_floats = (int)total;
    return true;
}

// Planes with more 4x4 blocks than a workgroup has threads take up to this
// many block rounds per plane (one resident plane): 63 x 95 and similar.
constexpr int kGradMaxRounds = 4;

// Resident planes per batch: the best of (block-load lane use) x (workgroups
// per CU, up to three) over the feasible counts; larger counts on ties.
bool make_grad_plan(const wtconv_desc& d, GradPlan& gp)
{
    const long per = (long)(ceil_to(d.H, 4) / 4) * (ceil_to(d.W, 4) / 4);
    if (per > wtc::kThreads) {
        // One resident plane, its 4x4 blocks in several rounds per thread. At
        // L = 1 beyond two rounds the region-tiled fused backward is as fast or
        // faster (measured on MI355X, k = 5, B16 C64: 96 x 96 121 vs 122 us,
        // 112 x 112 121 vs 155 us; at L = 3 the gradient pass wins: 84 x 84
        // 183 -> 127, 96 x 96 192 -> 153, 112 x 112 200 -> 189 us).
        const long rounds = cdiv(per, (long)wtc::kThreads);
        if (rounds > kGradMaxRounds || (d.L < 2 && rounds > 2) || !grad_layout(d, 1, gp)) return false;
        gp.PP = 1;
        gp.rounds = (int)rounds;
    } else {
        const int maxpp = (int)std::min<long>(d.B, wtc::kThreads / per);
        double best = -1.0;
        // Level 1 in 4 x 4 site tiles first. Tiles of 2 x 2 sites take the
        // same FMA issue in four times the rounds, but the level's arrays
        // then cover the grid rounded to 2 rather than to 4 sites (14 x 14
        // instead of 16 x 16 at 28 x 28): they replace the 4 x 4 plan when
        // that lets more planes or workgroups fit, i.e. when the score with
        // the workgroups per CU that the kernel's registers allow (3 for
        // k <= 5, 2 for k = 7, 1 for k = 9) rises without fewer workgroups.
        // Measured on MI355X (combined backward, us, 4 x 4 -> 2 x 2): B64
        // C192 28 x 28 L1 82.0 -> 74.1 (bf16 80.4 -> 71.7), B128 C192 L1 142.4
        // -> 122.6, 26 x 26 L1 95.9 -> 82.5; B64 C96 50 x 50 L3 203.3 ->
        // 168.0, 52 x 52 L5 213.2 -> 178.8, 58 x 58 L2 194.9 -> 169.3, L3
        // 224.2 -> 192.8, 49 x 49 L4 225.8 -> 187.6, 18 x 18 L3 61.5 -> 54.4;
        // k = 3 B64 C192 28 x 28 L1 65.7 -> 59.7, B64 C96 58 x 58 L3 181.3 ->
        // 153.1; k = 7 28 x 28 L2 188.6 -> 177.2, L4 229.7 -> 218.0, B128 C192
        // 26 x 26 L3 418.3 -> 390.2. Taken without the register limit it also
        // moved 12 x 12 L2 B128 C384 to more planes at fewer workgroups (101.2
        // -> 113.1) and k = 7 58 x 58 L1 to tiles that only added rounds
        // (220.4 -> 270.4).
        const int reg_wgs = d.k <= 5 ? 3 : (d.k <= 7 ? 2 : 1);
        double best_r = -1.0;
        int best_wgs = 0;
        for (int t1 : {4, 2})
            for (int pp = 1; pp <= maxpp; ++pp) {
                GradPlan c;
                if (!grad_layout(d, pp, c, t1)) continue;
                const int wgs = std::min(3, lds_wgs(c.lds_floats));
                const double lanes = (double)pp * per / wtc::kThreads;
                const double score = lanes * wgs;
                const double score_r = lanes * std::min(wgs, reg_wgs);
                if (t1 == 4 ? score >= best : (score_r > best_r && std::min(wgs, reg_wgs) >= best_wgs)) {
                    best = score;
                    best_r = score_r;
                    best_wgs = std::min(wgs, reg_wgs);
                    gp = c;
                    gp.PP = pp;
                }
            }
        if (best < 0) return false;
    }
    // One round of resident workgroups: the per-workgroup setup and the final
    // reduction of 3 x 25 sums per thread are paid once per workgroup, so few
    // long-running workgroups that fill every CU beat many short ones
    // (measured on MI355X at the ConvNeXt-T shapes). The chunk count rounds
    // down so that the grid fits the slots: rounding 512 / 192 up to 3 chunks
    // left a second round of 64 workgroups (28 x 28, L = 3: 150 -> 143 us per
    // backward at B = 64, 289 -> 250 us at B = 128 with 2 chunks).
    const int wgs_per_cu = std::max(1, std::min(3, lds_wgs(gp.lds_floats)));
    const int slots = 256 * wgs_per_cu;
    const int chunks = std::max(1, std::min(d.B, slots / d.C));
    gp.nb = ceil_to(cdiv(d.B, chunks), gp.PP);
    gp.nchunks = cdiv(d.B, gp.nb);
    return true;
}

struct GradExec {
    bool use = false;
    GradPlan gp;
    int Lf = 0;           // levels whose kernel gradients grad_kernel forms
    bool coarse = false;  // levels Lf+1..L: backward of the coarse sub-problem on X_m, dY_m
};

// The gradient pass sheds the levels above m (the first level whose grid is
// at most 8 x 8) to a coarse sub-problem on the level-m carriers of x and dy
// when that removes at least this many levels and more than one plane is
// resident per batch (each deep level is then a row pass over every resident
// plane). Measured on MI355X, backward us, split / not: 28x28 B64 L4 174 / 198,
// L5 187 / 238, B128 L5 278 / 439; 56x56 (one resident plane) B128 L5 429 / 382.
constexpr int kGradSplitMinShed = 2;
// A single level above m >= 2 is shed too once the coarse sub-problem has
// enough planes for its one-plane-per-lane kernel: at least this many. The
// gradient pass then keeps the smaller LDS of levels 1..m (the carriers come
// from the pass itself). Measured on MI355X, k = 5, L = 3, combined backward
// us, shed / not: B128 C192 18 x 18 158 / 180, 20 x 20 142 / 161, 26 x 26 216
// / 257, 28 x 28 193 / 225 (bf16 199 / 234), 30 x 30 257 / 272, 32 x 32 219 /
// 232, 24 x 24 172 / 175; B96 C192 28 x 28 155 / 173. Below it the gain
// shrinks and turns into a loss: B80 C192 28 x 28 142 / 152, B128 C128
// 32 x 32 145 / 143, B64 C192 28 x 28 124 / 122, 20 x 20 101 / 89, 24 x 24
// 110 / 99. k = 3 and 7 at B128 C192 28 x 28: within 1 %. (Shedding the level in the forward pass too
// was slower at every one of these shapes: 28 x 28 B128 108 against 83 us.)
constexpr long kGradShedOneMinPlanes = 18432;

// Measured on MI355X: the gradient pass beats the fused backward when the
// plane's first level at most 8 x 8 is level 2 or deeper (planes above 16 x 16)
// and there is at least one level (L = 1, k = 5: 28 x 28 115 -> 94 us, 40 x 40
// 130 -> 80 us, 56 x 56 B = 128 252 -> 231 us); it then handles every level
// itself. Planes whose level 1 is already at most 8 x 8 (9 x 9 to 16 x 16) take
// it at L <= 2, where it runs without a coarse sub-problem (B128 C384 14 x 14,
// k = 5: L = 1 139 -> 131 us, L = 2 196 -> 156 us). At L >= 3 it needs the
// split (carriers and the tiny kernels, for dx too), which pays only where
// the fused backward is weakest: at k = 7 (whose fused backward holds 3 x 49
// kernel-gradient sums per lane and runs one wavefront per SIMD; B128 C384
// 14 x 14 L = 3 623 -> 288 us, L = 5 629 -> 299 us, bf16 L = 3 696 -> 317 us,
// 12 x 12 and 16 x 16 L = 3 -38 %) and at k = 5 on planes of at most 3 x 3
// pixel blocks (B128 C192 L = 3: 10 x 10 126 -> 112 us, 11 x 11 140 -> 122 us,
// 12 x 12 124 -> 109 us; 10 x 10 L = 5 129 -> 124 us). Since dx takes the
// coarse sub-problem's input gradient as a carry and the finalize runs in the
// dx launch, it also wins at k = 5 up to 16 x 16 (B128 C384 14 x 14, combined
// backward: L = 3 189.9 -> 180.2 us, L = 4 191.8 -> 182.9, L = 5 193.9 ->
// 187.5, bf16 L = 3 203.4 -> 196.6; B64 C384 L = 5 129.6 -> 126.5; B64 C192
// 16 x 16 L = 3 96.1 -> 92.3, L = 5 100.3 -> 96.2). At k = 3 it does not pay
// (14 x 14 L = 3 152.9 -> 152.8 us; 12 x 12 within 2 %). L = 0 runs the fused
// backward.
bool grad_pass_pays_deep(const wtconv_desc& d)
{
    return d.k >= 5;
}

GradExec choose_grad_uncached(const wtconv_desc& d);

GradExec choose_grad(const wtconv_desc& d)
{
    static PlanCache<GradExec> cache;
    return cache.get(d, 2, [&] { return choose_grad_uncached(d); });
}

GradExec choose_grad_uncached(const wtconv_desc& d)
{
    GradExec ge;
    if (use_tiny(d) || d.L < 1) return ge;
    const int m = tiny_level(d);
    if (m < 1 || (m == 1 && d.L > 2 && !grad_pass_pays_deep(d))) return ge;
    wtconv_desc f = d;
    if (d.L - m >= kGradSplitMinShed || (m >= 2 && d.L > m && (long)d.B * d.C >= kGradShedOneMinPlanes)) {
        GradPlan full;
        if (make_grad_plan(d, full) && full.PP > 1) f.L = m;
    }
    ge.use = make_grad_plan(f, ge.gp);
    ge.Lf = f.L;
    ge.coarse = d.L > f.L;
    return ge;
}

// Sites of the level-m grid over the whole tensor.
long level_floats(const wtconv_desc& d, int m)
{
    long h = d.H, w = d.W;
    for (int l = 0; l < m; ++l) {
        h = (h + 1) / 2;
        w = (w + 1) / 2;
    }
    return (long)d.B * d.C * h * w;
}

// The coarse sub-problem of a split at level m: the operator (without base
// path) on the level-m carriers, in the problem's storage type (the carriers,
// the coarse contribution and, in the backward, the coarse dx are held in it:
// half the workspace of fp32 for 16-bit problems, at one extra rounding of
// those intermediates).
wtconv_desc coarse_desc(const wtconv_desc& d, int m)
{
    wtconv_desc s = d;
    for (int l = 0; l < m; ++l) {
        s.H = (s.H + 1) / 2;
        s.W = (s.W + 1) / 2;
    }
    s.L = d.L - m;
    return s;
}

// Bytes of one level-m carrier-sized buffer of the whole tensor (storage type).
size_t level_bytes(const wtconv_desc& d, int m)
{
    return align256((size_t)level_floats(d, m) * elem_size(d.dtype));
}

wtc::TinyArgs tiny_args(const wtconv_desc& d, const void* in, const void* aux, void* out, float* partial,
                        const wtc::ParamPtrs& p, int skip_base)
{
    wtc::TinyArgs t;
    memset(&t, 0, sizeof(t));
    t.in = in;
    t.aux = aux;
    t.out = out;
    t.partial = partial;
    t.p = p;
    t.B = d.B;
    t.C = d.C;
    t.H = d.H;
    t.W = d.W;
    t.L = d.L;
    t.skip_base = skip_base;
    return t;
}

const size_t kUnsupported = ~(size_t)0;

// Kernel-gradient partials written by the fused (or tiny) pass of `ex`.
size_t pass_partial_bytes(const wtconv_desc& d, const Exec& ex)
{
    switch (ex.mode) {
        case Mode::Tiny:
            return align256((size_t)tiny_groups(d) * d.C * wtc::partial_floats_per_channel(d.k, d.L) * 4);
        case Mode::Resident:
            return align256((size_t)ex.pl.nchunks * d.C * wtc::partial_floats_per_channel(d.k, d.L) * 4);
        case Mode::Split:
            return align256((size_t)ex.pl.nchunks * d.C * wtc::partial_floats_per_channel(d.k, ex.m) * 4);
        case Mode::Region:
            return align256((size_t)ex.rp.pl.nchunks * ex.rp.ntx * ex.rp.nty * d.C *
                            wtc::partial_floats_per_channel(d.k, ex.m) * 4);
        case Mode::None: break;
    }
    return kUnsupported;
}

// Workspace layouts.
//   forward:  [X_m][carry][sub-problem]                   (split / region with a coarse part)
//   backward: [partials][X_m][dY_m][dX_m][sub-problem]
size_t forward_ws(const wtconv_desc& d)
{
    const Exec ex = choose(d, false);
    if (ex.mode == Mode::None) return kUnsupported;
    if (!ex.coarse) return 0;
    const size_t sub = forward_ws(coarse_desc(d, ex.m));
    if (sub == kUnsupported) return kUnsupported;
    return 2 * level_bytes(d, ex.m) + sub;
}

size_t backward_ws(const wtconv_desc& d);

// Gradient-pass workspace: [partials][X_m][dY_m][coarse backward][forward workspace of dx]
size_t grad_partial_bytes(const wtconv_desc& d, const GradExec& ge)
{
    return align256((size_t)ge.gp.nchunks * d.C * wtc::partial_floats_per_channel(d.k, ge.Lf) * 4);
}


// The dx pass of a gradient-pass backward with a coarse sub-problem on levels
// above m: the forward's fused pass on levels 1..m of the resident plane (the
// coarse levels enter as a carry). False if that pass has no resident plan.
bool dx_pass_plan(const wtconv_desc& d, int m, Plan& pl)
{
    wtconv_desc f = d;
    f.L = m;
    if (m < 1 || use_tiny(d)) return false;
    struct Found {
        bool ok;
        Plan pl;
    };
    static PlanCache<Found> cache;
    const Found r = cache.get(f, 3, [&] {
        Found v;
        v.ok = make_plan(f, false, v.pl);
        return v;
    });
    if (r.ok) pl = r.pl;
    return r.ok;
}

// [X_m][dY_m][dX_m][coarse backward]
size_t grad_coarse_bytes(const wtconv_desc& d, const GradExec& ge)
{
    if (!ge.coarse) return 0;
    const size_t sub = backward_ws(coarse_desc(d, ge.Lf));
    if (sub == kUnsupported) return kUnsupported;
    return 3 * level_bytes(d, ge.Lf) + sub;
}

size_t backward_ws(const wtconv_desc& d)
{
    const GradExec ge = choose_grad(d);
    if (ge.use) {
        const size_t coarse = grad_coarse_bytes(d, ge);
        const size_t fwd = forward_ws(d);
        if (coarse == kUnsupported || fwd == kUnsupported) return kUnsupported;
        return grad_partial_bytes(d, ge) + coarse + fwd;
    }
    const Exec ex = choose(d, true);
    if (ex.mode == Mode::None) return kUnsupported;
    const size_t part = pass_partial_bytes(d, ex);
    if (!ex.coarse) return part;
    const size_t sub = backward_ws(coarse_desc(d, ex.m));
    if (sub == kUnsupported) return kUnsupported;
    return part + 3 * level_bytes(d, ex.m) + sub;
}

FusedArgs base_args(const wtconv_desc& d, const Plan& pl, const void* in, const void* aux, void* out,
                    const wtc::ParamPtrs& p, int skip_base)
{
    FusedArgs a;
    memset(&a, 0, sizeof(a));
    a.in = in;
    a.aux = aux;
    a.out = out;
    a.p = p;
    a.B = d.B;
    a.C = d.C;
    a.nb = pl.nb;
    a.PP = pl.PP;
    a.vec_ok = vec_ok(in, aux ? aux : in, out ? out : in);
    a.lds_floats = pl.lds_floats;
    a.one_round = pl.one_round;
    a.merge_deep = pl.merge_deep;
    a.skip_base = skip_base;
    a.mx_rounds = pl.mx.rounds;
    a.mx_first_out = pl.mx.first_out;
    memcpy(a.mx_seg0, pl.mx.seg0, sizeof(a.mx_seg0));
    memcpy(a.mx_ntask, pl.mx.ntask, sizeof(a.mx_ntask));
    memcpy(a.mx_out0, pl.mx.out0, sizeof(a.mx_out0));
    memcpy(a.mx_seg, pl.mx.seg, sizeof(a.mx_seg));
    a.g = pl.g;
    return a;
}

void set_region(FusedArgs& a, const wtconv_desc& d, const RegionPlan& rp)
{
    a.rg_ntx = rp.ntx;
    a.rg_nty = rp.nty;
    a.rg_T = rp.T;
    a.rg_h = rp.h;
    a.real_H = d.H;
    a.real_W = d.W;
    a.rg_r_itx = 1.0f / (float)(rp.T / 4);
    a.rg_r_itiles = 1.0f / (float)((rp.T / 4) * (rp.T / 4));
}

void set_carry(FusedArgs& a, const wtconv_desc& d, int m, const void* carry)
{
    const wtconv_desc c = coarse_desc(d, m);
    a.carry = carry;
    a.carry_H = c.H;
    a.carry_W = c.W;
    a.carry_level = m;
}

wtconv_status hip_status(hipError_t e) { return e == hipSuccess ? WTCONV_OK : WTCONV_ERR_HIP; }

wtconv_status carrier(const wtconv_desc& d, int m, const void* in, void* out, hipStream_t stream)
{
    const wtconv_desc cd = coarse_desc(d, m);
    wtc::CarrierArgs c;
    c.in = in;
    c.out = out;
    c.planes = (long)d.B * d.C;
    c.H = d.H;
    c.W = d.W;
    c.H1 = cd.H;
    c.W1 = cd.W;
    c.m = m;
    // m = 1 reads row pairs (W even suffices), deeper levels rows of 4-multiples
    c.vec_ok = (d.W % (m == 1 ? 2 : 4) == 0 && ((uintptr_t)in & (d.dtype == WTCONV_F32 ? 15 : 7)) == 0) ? 1 : 0;
    return hip_status(wtc::launch_carrier(d.dtype, c, stream));
}

// The fused pass of a resident / split / region execution (grid and plan).
struct FusedPass {
    const Plan* pl;
    int grid;
};

FusedPass fused_pass(const wtconv_desc& d, const Exec& ex)
{
    if (ex.mode == Mode::Region)
        return {&ex.rp.pl, ex.rp.pl.nchunks * ex.rp.ntx * ex.rp.nty * d.C};
    return {&ex.pl, ex.pl.nchunks * d.C};
}

wtc::ReduceArgs reduce_args(const wtconv_desc& d, int L, int nchunks, const wtc::ParamPtrs& p, const Grads& gr,
                            const char* ws, int skip_base)
{
    wtc::ReduceArgs r;
    memset(&r, 0, sizeof(r));
    r.partial = reinterpret_cast<const float*>(ws);
    r.nchunks = nchunks;
    r.C = d.C;
    r.k = d.k;
    r.L = L;
    r.skip_base = skip_base;
    r.p = p;
    r.dw0 = gr.dw0;
    r.ds0 = gr.ds0;
    r.db0 = skip_base ? nullptr : gr.db0;
    for (int l = 0; l < L; ++l) {
        r.dlw[l] = gr.dlw[l];
        r.dls[l] = gr.dls[l];
    }
    return r;
}

wtconv_status reduce(const wtconv_desc& d, int L, int nchunks, const wtc::ParamPtrs& p, const Grads& gr,
                     const char* ws, int skip_base, hipStream_t stream)
{
    return hip_status(wtc::launch_reduce(reduce_args(d, L, nchunks, p, gr, ws, skip_base), stream));
}

// A finalize reduction that the last launch of a forward pass runs in extra
// workgroups ahead of its own (dx of the combined backward); `done` tells
// whether it was attached (a tiny-plane pass takes none). Their count is
// rounded up to a multiple of 8 so that the plane workgroups keep their
// round-robin placement over the eight XCDs.
struct FinJob {
    wtc::ReduceArgs r;
    bool done;
};

void attach_fin(FusedArgs& a, int& grid, FinJob* fin)
{
    if (!fin) return;
    a.fin = fin->r;
    a.fin_blocks = ceil_to(cdiv((long)fin->r.C * (1 + 4 * fin->r.L), 4), 8);
    grid += a.fin_blocks;
    fin->done = true;
}

wtconv_status forward_impl(const wtconv_desc& d, const void* x, const wtc::ParamPtrs& p, void* y, char* ws,
                           int skip_base, hipStream_t stream, FinJob* fin = nullptr)
{
    const Exec ex = choose(d, false);
    if (ex.mode == Mode::None) return WTCONV_ERR_UNSUPPORTED;
    if (ex.mode == Mode::Tiny)
        return hip_status(
            wtc::launch_tiny(d.k, d.dtype, false, tiny_args(d, x, nullptr, y, nullptr, p, skip_base), stream));
    const void* carry = nullptr;
    if (ex.coarse) {
        const size_t n1 = level_bytes(d, ex.m);
        void* x1 = ws;
        void* c1 = ws + n1;
        wtconv_status st = carrier(d, ex.m, x, x1, stream);
        if (st != WTCONV_OK) return st;
        st = forward_impl(coarse_desc(d, ex.m), x1, shift_params(p, ex.m), c1, ws + 2 * n1, 1, stream);
        if (st != WTCONV_OK) return st;
        carry = c1;
    }
    const FusedPass fp = fused_pass(d, ex);
    FusedArgs a = base_args(d, *fp.pl, x, nullptr, y, p, skip_base);
    if (ex.mode == Mode::Region) set_region(a, d, ex.rp);
    if (carry) set_carry(a, d, ex.m, carry);
    int grid = fp.grid;
    attach_fin(a, grid, fin);
    return hip_status(wtc::launch_forward(d.k, d.dtype, a, grid, stream));
}

// cx, cdy (nullable): also write the level-cm (1 or 2) carriers of x and dy
// there, as carrier() would.
// rp (nullable): region mode, over the region tiles of rp with its chunks.
wtconv_status grad_pass(const wtconv_desc& d, const GradExec& ge, const void* x, const void* dy, float* partial,
                        int skip_base, hipStream_t stream, void* cx = nullptr, void* cdy = nullptr, int cm = 0,
                        const RegionPlan* rp = nullptr)
{
    wtc::GradArgs a;
    memset(&a, 0, sizeof(a));
    int grid = ge.gp.nchunks * d.C;
    a.nb = ge.gp.nb;
    if (rp) {
        a.rg_ntx = rp->ntx;
        a.rg_nty = rp->nty;
        a.rg_T = rp->T;
        a.rg_h = rp->h;
        a.real_H = d.H;
        a.real_W = d.W;
        a.nb = rp->pl.nb;
        grid = rp->pl.nchunks * rp->ntx * rp->nty * d.C;
    }
    if (cx) {
        const wtconv_desc cd = coarse_desc(d, cm);
        a.cx = cx;
        a.cdy = cdy;
        a.cm = cm;
        a.cH = cd.H;
        a.cW = cd.W;
    }
    a.x = x;
    a.dy = dy;
    a.partial = partial;
    a.B = d.B;
    a.C = d.C;
    a.PP = ge.gp.PP;
    a.rounds = ge.gp.rounds;
    a.vec_ok = vec_ok(x, dy, x);
    a.lds_floats = ge.gp.lds_floats;
    a.skip_base = skip_base;
    a.stride = ge.gp.stride;
    a.r_ring = 1.0f / (float)(ge.gp.g.xpitch - 4 * ge.gp.g.tiles_x);
    a.tail0 = ge.gp.tail0;
    a.tail1 = ge.gp.tail1;
    for (int l = 0; l <= kMaxLevels; ++l) {
        a.dy_off[l] = ge.gp.dy_off[l];
        a.dy_pitch[l] = ge.gp.dy_pitch[l];
        a.dy_band[l] = ge.gp.dy_band[l];
    }
    a.g = ge.gp.g;
    return hip_status(wtc::launch_grad(d.k, d.dtype, a, grid, stream));
}

// Backward of a problem in region mode by the gradient route: the gradient
// pass over the same region tiles as the fused region backward (so the
// partials and the finalize are the same), writing the level-1 carriers of x
// and dy from the tiles' own blocks; the coarse sub-problem's backward on
// them; dx as the forward on dy with rotated kernels over levels 1..1 with
// the coarse input gradient as its carry. A region of more 4x4 blocks than
// threads (k = 7 and 9) walks them in rounds. False (nothing launched) if the
// region's gradient pass needs more than one resident region.
constexpr bool kRegionGradRoute = true;

bool region_grad_exec(const wtconv_desc& d, const Exec& ex, GradExec& ge)
{
    if (!kRegionGradRoute || ex.mode != Mode::Region || ex.m != 1) return false;
    wtconv_desc rd = d;
    rd.B = 1;
    rd.H = rd.W = ex.rp.T + 2 * ex.rp.h;
    rd.L = 1;
    if (!make_grad_plan(rd, ge.gp) || ge.gp.PP != 1 || ge.gp.g.L != 1) return false;
    ge.use = true;
    ge.Lf = 1;
    ge.coarse = ex.coarse;
    return true;
}

bool region_grad_one_round(const wtconv_desc& d, const Exec& ex)
{
    GradExec ge;
    return region_grad_exec(d, ex, ge) && ge.gp.rounds == 1;
}

wtconv_status partials_impl(const wtconv_desc& d, const void* x, const void* dy, const wtc::ParamPtrs& p,
                            void* dx, char* ws, int skip_base, hipStream_t stream, const Grads* gr = nullptr,
                            bool* fin_done = nullptr);

wtconv_status region_grad_backward(const wtconv_desc& d, const Exec& ex, const GradExec& ge, const void* x,
                                   const void* dy, const wtc::ParamPtrs& p, void* dx, char* ws, int skip_base,
                                   hipStream_t stream)
{
    const size_t part = pass_partial_bytes(d, ex);
    void* x1 = nullptr;
    void* dy1 = nullptr;
    void* dx1 = nullptr;
    if (ex.coarse) {
        const size_t n1 = level_bytes(d, 1);
        x1 = ws + part;
        dy1 = ws + part + n1;
        dx1 = dx ? ws + part + 2 * n1 : nullptr;
    }
    wtconv_status st = grad_pass(d, ge, x, dy, reinterpret_cast<float*>(ws), skip_base, stream, x1, dy1, x1 ? 1 : 0,
                                 &ex.rp);
    if (st == WTCONV_OK && ex.coarse)
        st = partials_impl(coarse_desc(d, 1), x1, dy1, shift_params(p, 1), dx1, ws + part + 3 * level_bytes(d, 1), 1,
                           stream, nullptr, nullptr);
    if (st != WTCONV_OK || !dx) return st;
    wtc::ParamPtrs pr = p;
    pr.rot = 1;
    pr.b0 = nullptr;  // the bias does not reach dx
    wtconv_desc f = d;
    f.L = 1;
    const Exec fx = choose(f, false);
    if (fx.mode != Mode::Region && fx.mode != Mode::Resident) return WTCONV_ERR_UNSUPPORTED;
    const FusedPass fp = fused_pass(f, fx);
    FusedArgs a = base_args(f, *fp.pl, dy, nullptr, dx, pr, skip_base);
    if (fx.mode == Mode::Region) set_region(a, f, fx.rp);
    if (dx1) set_carry(a, d, 1, dx1);
    return hip_status(wtc::launch_forward(d.k, d.dtype, a, fp.grid, stream));
}

// With `gr` (the combined backward), the finalize of the kernel gradients of
// levels 0..Lf of the gradient route runs at the end of the dx launch when it
// can; *fin_done then tells finalize_impl to skip it.
wtconv_status partials_impl(const wtconv_desc& d, const void* x, const void* dy, const wtc::ParamPtrs& p,
                            void* dx, char* ws, int skip_base, hipStream_t stream, const Grads* gr,
                            bool* fin_done)
{
    const GradExec ge = choose_grad(d);
    if (ge.use) {
        const size_t part = grad_partial_bytes(d, ge);
        // dx is the forward pass on dy with every kernel rotated by 180
        // degrees. With a coarse sub-problem its levels above Lf are that
        // sub-problem's input gradient, which the coarse backward forms from
        // the same carriers (it is the adjoint of the coarse branch applied to
        // dY_Lf): dx is then one fused pass on levels 1..Lf with that carry,
        // instead of a forward that would take the dy carrier and run the
        // coarse forward again.
        wtc::ParamPtrs pr = p;
        pr.rot = 1;
        pr.b0 = nullptr;  // the bias does not reach dx
        Plan dxp;
        const bool dx_carry = dx && ge.coarse && dx_pass_plan(d, ge.Lf, dxp);
        wtconv_status st = WTCONV_OK;
        void* dx1 = nullptr;
        if (ge.coarse) {
            // kernel gradients of levels Lf+1..L (and the coarse part of dx):
            // the coarse sub-problem's, on the level-Lf carriers of x and dy
            // (no base path). At Lf <= 2 the gradient pass forms the carriers
            // from the blocks it loads anyway (a block covers whole carrier
            // sites), instead of two carrier launches that read x and dy again.
            const size_t n1 = level_bytes(d, ge.Lf);
            void* x1 = ws + part;
            void* dy1 = ws + part + n1;
            dx1 = dx_carry ? ws + part + 2 * n1 : nullptr;
            const bool in_pass = ge.Lf <= 2 && ge.gp.rounds == 1;
            if (in_pass) {
                st = grad_pass(d, ge, x, dy, reinterpret_cast<float*>(ws), skip_base, stream, x1, dy1, ge.Lf);
            } else {
                st = carrier(d, ge.Lf, x, x1, stream);
                if (st == WTCONV_OK) st = carrier(d, ge.Lf, dy, dy1, stream);
            }
            if (st == WTCONV_OK)
                st = partials_impl(coarse_desc(d, ge.Lf), x1, dy1, shift_params(p, ge.Lf), dx1, ws + part + 3 * n1,
                                   1, stream);
            if (st == WTCONV_OK && !in_pass) st = grad_pass(d, ge, x, dy, reinterpret_cast<float*>(ws), skip_base, stream);
        } else {
            st = grad_pass(d, ge, x, dy, reinterpret_cast<float*>(ws), skip_base, stream);
        }
        if (st != WTCONV_OK || !dx) return st;
        FinJob fin = {};
        if (gr) fin.r = reduce_args(d, ge.Lf, ge.gp.nchunks, p, *gr, ws, skip_base);
        if (dx_carry) {
            wtconv_desc f = d;
            f.L = ge.Lf;
            FusedArgs a = base_args(f, dxp, dy, nullptr, dx, pr, skip_base);
            set_carry(a, d, ge.Lf, dx1);
            int grid = dxp.nchunks * d.C;
            attach_fin(a, grid, gr ? &fin : nullptr);
            st = hip_status(wtc::launch_forward(d.k, d.dtype, a, grid, stream));
        } else {
            st = forward_impl(d, dy, pr, dx, ws + part + grad_coarse_bytes(d, ge), skip_base, stream,
                              gr ? &fin : nullptr);
        }
        if (fin_done) *fin_done = st == WTCONV_OK && fin.done;
        return st;
    }
    const Exec ex = choose(d, true);
    if (ex.mode == Mode::None) return WTCONV_ERR_UNSUPPORTED;
    if (ex.mode == Mode::Tiny)
        return hip_status(wtc::launch_tiny(
            d.k, d.dtype, true, tiny_args(d, dy, x, dx, reinterpret_cast<float*>(ws), p, skip_base), stream));
    {
        GradExec rge;
        if (region_grad_exec(d, ex, rge)) return region_grad_backward(d, ex, rge, x, dy, p, dx, ws, skip_base, stream);
    }
    const size_t part = pass_partial_bytes(d, ex);
    const void* carry = nullptr;
    if (ex.coarse) {
        const size_t n1 = level_bytes(d, ex.m);
        void* x1 = ws + part;
        void* dy1 = ws + part + n1;
        void* dx1 = dx ? ws + part + 2 * n1 : nullptr;
        wtconv_status st = carrier(d, ex.m, x, x1, stream);
        if (st == WTCONV_OK) st = carrier(d, ex.m, dy, dy1, stream);
        if (st == WTCONV_OK)
            st = partials_impl(coarse_desc(d, ex.m), x1, dy1, shift_params(p, ex.m), dx1, ws + part + 3 * n1, 1,
                               stream);
        if (st != WTCONV_OK) return st;
        carry = dx1;
    }
    const FusedPass fp = fused_pass(d, ex);
    FusedArgs a = base_args(d, *fp.pl, dy, x, dx, p, skip_base);
    if (ex.mode == Mode::Region) set_region(a, d, ex.rp);
    if (carry) set_carry(a, d, ex.m, carry);
    a.partial = reinterpret_cast<float*>(ws);
    return hip_status(wtc::launch_backward(d.k, d.dtype, a, fp.grid, stream));
}

// main_done: the reduction of levels 0..Lf of the gradient route already ran
// with the dx launch (partials_impl with `gr`).
wtconv_status finalize_impl(const wtconv_desc& d, const wtc::ParamPtrs& p, const Grads& gr, const char* ws,
                            int skip_base, hipStream_t stream, bool main_done = false)
{
    const GradExec ge = choose_grad(d);
    if (ge.use) {
        if (ge.coarse) {
            const size_t part = grad_partial_bytes(d, ge);
            const size_t n1 = level_bytes(d, ge.Lf);
            // the coarse sub-problem's workspace follows X_m, dY_m and dX_m (see partials_impl)
            const wtconv_status st = finalize_impl(coarse_desc(d, ge.Lf), shift_params(p, ge.Lf),
                                                   shift_grads(gr, ge.Lf), ws + part + 3 * n1, 1, stream);
            if (st != WTCONV_OK) return st;
        }
        if (main_done) return WTCONV_OK;
        return reduce(d, ge.Lf, ge.gp.nchunks, p, gr, ws, skip_base, stream);
    }
    const Exec ex = choose(d, true);
    switch (ex.mode) {
        case Mode::None: return WTCONV_ERR_UNSUPPORTED;
        case Mode::Tiny: return reduce(d, d.L, tiny_groups(d), p, gr, ws, skip_base, stream);
        case Mode::Resident: return reduce(d, d.L, ex.pl.nchunks, p, gr, ws, skip_base, stream);
        default: break;
    }
    if (ex.coarse) {
        const size_t part = pass_partial_bytes(d, ex);
        const size_t n1 = level_bytes(d, ex.m);
        const wtconv_status st = finalize_impl(coarse_desc(d, ex.m), shift_params(p, ex.m), shift_grads(gr, ex.m),
                                               ws + part + 3 * n1, 1, stream);
        if (st != WTCONV_OK) return st;
    }
    const int nchunks = ex.mode == Mode::Region ? ex.rp.pl.nchunks * ex.rp.ntx * ex.rp.nty : ex.pl.nchunks;
    return reduce(d, ex.m, nchunks, p, gr, ws, skip_base, stream);
}

struct Range {
    const void* p;
    size_t n;
};

bool any_overlap(const Range* outs, int no, const Range* ins, int ni)
{
    for (int i = 0; i < no; ++i) {
        for (int j = 0; j < ni; ++j)
            if (overlaps(outs[i].p, outs[i].n, ins[j].p, ins[j].n)) return true;
        for (int j = i + 1; j < no; ++j)
            if (overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return true;
    }
    return false;
}

int param_ranges(const wtconv_desc& d, const float* w0, const float* s0, const float* b0, const float* const* lw,
                 const float* const* ls, Range* r)
{
    const size_t KK = (size_t)d.k * d.k;
    int n = 0;
    r[n++] = {w0, (size_t)d.C * KK * 4};
    r[n++] = {s0, (size_t)d.C * 4};
    r[n++] = {b0, (size_t)d.C * 4};  // a null range overlaps nothing
    for (int l = 0; l < d.L; ++l) {
        r[n++] = {lw[l], (size_t)4 * d.C * KK * 4};
        r[n++] = {ls[l], (size_t)4 * d.C * 4};
    }
    return n;
}

wtconv_status check_workspace(size_t need, const void* ws, size_t bytes)
{
    if (need == kUnsupported) return WTCONV_ERR_UNSUPPORTED;
    if (need == 0) return WTCONV_OK;
    if (!ws || bytes < need || ((uintptr_t)ws & 15)) return WTCONV_ERR_WORKSPACE;
    return WTCONV_OK;
}

// Shared argument checks of the backward entry points.
wtconv_status backward_checks(const wtconv_desc* desc, const void* x, const void* dy, const float* base_w,
                              const float* base_scale, const float* base_bias, const float* const* level_w,
                              const float* const* level_scale, const void* dx, const void* workspace,
                              size_t workspace_bytes, const Range* extra_outs, int n_extra, size_t* need_out)
{
    wtconv_status st = check_desc(desc);
    if (st != WTCONV_OK) return st;
    const wtconv_desc& d = *desc;
    if (!x || !dy || !base_w || !base_scale) return WTCONV_ERR_NULL;
    if ((st = check_levels(d.L, level_w, level_scale)) != WTCONV_OK) return st;
    const size_t need = backward_ws(d);
    if ((st = check_workspace(need, workspace, workspace_bytes)) != WTCONV_OK) return st;
    if (need == 0) return WTCONV_ERR_WORKSPACE;  // the backward always writes partials
    const size_t act = (size_t)d.B * d.C * d.H * d.W * elem_size(d.dtype);
    Range ins[5 + 2 * kMaxLevels];
    int ni = 0;
    ins[ni++] = {x, act};
    ins[ni++] = {dy, act};
    ni += param_ranges(d, base_w, base_scale, base_bias, level_w, level_scale, ins + ni);
    Range outs[2 + 3 + 2 * kMaxLevels];
    int no = 0;
    outs[no++] = {dx, act};
    outs[no++] = {workspace, need};
    for (int i = 0; i < n_extra; ++i) outs[no++] = extra_outs[i];
    if (any_overlap(outs, no, ins, ni)) return WTCONV_ERR_ALIAS;
    *need_out = need;
    return WTCONV_OK;
}

Grads grads_of(int L, float* d_base_w, float* d_base_scale, float* d_base_bias, float* const* d_level_w,
               float* const* d_level_scale)
{
    Grads gr;
    memset(&gr, 0, sizeof(gr));
    gr.dw0 = d_base_w;
    gr.ds0 = d_base_scale;
    gr.db0 = d_base_bias;
    for (int l = 0; l < L; ++l) {
        gr.dlw[l] = d_level_w[l];
        gr.dls[l] = d_level_scale[l];
    }
    return gr;
}

}  // namespace

extern "C" {

int wtconv_version(void) { return 300; }

const char* wtconv_status_string(wtconv_status s)
{
    switch (s) {
        case WTCONV_OK: return "ok";
        case WTCONV_ERR_NULL: return "a required pointer is NULL";
        case WTCONV_ERR_SHAPE: return "invalid shape (B, C, H, W must be >= 1 and sizes must fit)";
        case WTCONV_ERR_KSIZE: return "unsupported kernel size (k must be 1, 3, 5, 7 or 9)";
        case WTCONV_ERR_LEVELS: return "unsupported number of levels (0 <= L <= 8)";
        case WTCONV_ERR_DTYPE: return "unknown dtype";
        case WTCONV_ERR_ALIAS: return "an output overlaps an input or another output";
        case WTCONV_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case WTCONV_ERR_UNSUPPORTED: return "no execution plan for this shape";
        case WTCONV_ERR_HIP: return "HIP runtime error";
        case WTCONV_ERR_SCRATCH: return "the problem needs more workspace than the static scratch of "
                                        "wtconv_backward_noalloc holds";
    }
    return "unknown status";
}

size_t wtconv_forward_workspace_bytes(const wtconv_desc* desc)
{
    if (check_desc(desc) != WTCONV_OK) return 0;
    const size_t n = forward_ws(*desc);
    return n == kUnsupported ? 0 : n;
}

wtconv_status wtconv_forward(const wtconv_desc* desc, const void* x, const float* base_w,
                             const float* base_scale, const float* base_bias, const float* const* level_w,
                             const float* const* level_scale, void* y, void* workspace,
                             size_t workspace_bytes, hipStream_t stream)
{
    wtconv_status st = check_desc(desc);
    if (st != WTCONV_OK) return st;
    const wtconv_desc& d = *desc;
    if (!x || !y || !base_w || !base_scale) return WTCONV_ERR_NULL;
    if ((st = check_levels(d.L, level_w, level_scale)) != WTCONV_OK) return st;
    const size_t need = forward_ws(d);
    if ((st = check_workspace(need, workspace, workspace_bytes)) != WTCONV_OK) return st;
    const size_t bytes = (size_t)d.B * d.C * d.H * d.W * elem_size(d.dtype);
    Range ins[5 + 2 * kMaxLevels];
    int ni = 0;
    ins[ni++] = {x, bytes};
    ni += param_ranges(d, base_w, base_scale, base_bias, level_w, level_scale, ins + ni);
    const Range outs[2] = {{y, bytes}, {workspace, need}};
    if (any_overlap(outs, 2, ins, ni)) return WTCONV_ERR_ALIAS;
    wtc::ParamPtrs p;
    fill_params(p, d.L, base_w, base_scale, base_bias, level_w, level_scale);
    return forward_impl(d, x, p, y, reinterpret_cast<char*>(workspace), 0, stream);
}

size_t wtconv_backward_workspace_bytes(const wtconv_desc* desc)
{
    if (check_desc(desc) != WTCONV_OK) return 0;
    const size_t n = backward_ws(*desc);
    return n == kUnsupported ? 0 : n;
}

wtconv_status wtconv_backward_partials(const wtconv_desc* desc, const void* x, const void* dy,
                                       const float* base_w, const float* base_scale,
                                       const float* const* level_w, const float* const* level_scale,
                                       void* dx, void* workspace, size_t workspace_bytes,
                                       hipStream_t stream)
{
    size_t need = 0;
    const wtconv_status st = backward_checks(desc, x, dy, base_w, base_scale, nullptr, level_w, level_scale, dx,
                                             workspace, workspace_bytes, nullptr, 0, &need);
    if (st != WTCONV_OK) return st;
    wtc::ParamPtrs p;
    fill_params(p, desc->L, base_w, base_scale, nullptr, level_w, level_scale);
    return partials_impl(*desc, x, dy, p, dx, reinterpret_cast<char*>(workspace), 0, stream);
}

wtconv_status wtconv_backward_finalize(const wtconv_desc* desc, const float* base_w, const float* base_scale,
                                       const float* base_bias, const float* const* level_w,
                                       const float* const* level_scale, float* d_base_w, float* d_base_scale,
                                       float* d_base_bias, float* const* d_level_w, float* const* d_level_scale,
                                       const void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    wtconv_status st = check_desc(desc);
    if (st != WTCONV_OK) return st;
    const wtconv_desc& d = *desc;
    if (!base_w || !base_scale || !d_base_w || !d_base_scale) return WTCONV_ERR_NULL;
    if ((st = check_levels(d.L, level_w, level_scale)) != WTCONV_OK) return st;
    if ((st = check_levels(d.L, (const float* const*)d_level_w, (const float* const*)d_level_scale)) != WTCONV_OK)
        return st;
    const size_t need = backward_ws(d);
    if ((st = check_workspace(need, workspace, workspace_bytes)) != WTCONV_OK) return st;
    if (need == 0) return WTCONV_ERR_WORKSPACE;
    Range ins[4 + 2 * kMaxLevels];
    int ni = param_ranges(d, base_w, base_scale, base_bias, level_w, level_scale, ins);
    ins[ni++] = {workspace, need};
    Range outs[3 + 2 * kMaxLevels];
    const int no = param_ranges(d, d_base_w, d_base_scale, d_base_bias, (const float* const*)d_level_w,
                                (const float* const*)d_level_scale, outs);
    if (any_overlap(outs, no, ins, ni)) return WTCONV_ERR_ALIAS;
    wtc::ParamPtrs p;
    fill_params(p, d.L, base_w, base_scale, base_bias, level_w, level_scale);
    return finalize_impl(d, p, grads_of(d.L, d_base_w, d_base_scale, d_base_bias, d_level_w, d_level_scale),
                         reinterpret_cast<const char*>(workspace), 0, stream);
}

size_t wtconv_backward_data_workspace_bytes(const wtconv_desc* desc)
{
    if (check_desc(desc) != WTCONV_OK) return 0;
    const size_t n = forward_ws(*desc);
    return n == kUnsupported ? 0 : n;
}

wtconv_status wtconv_backward_data(const wtconv_desc* desc, const void* dy, const float* base_w,
                                   const float* base_scale, const float* const* level_w,
                                   const float* const* level_scale, void* dx, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream)
{
    wtconv_status st = check_desc(desc);
    if (st != WTCONV_OK) return st;
    const wtconv_desc& d = *desc;
    if (!dy || !dx || !base_w || !base_scale) return WTCONV_ERR_NULL;
    if ((st = check_levels(d.L, level_w, level_scale)) != WTCONV_OK) return st;
    const size_t need = forward_ws(d);
    if ((st = check_workspace(need, workspace, workspace_bytes)) != WTCONV_OK) return st;
    const size_t bytes = (size_t)d.B * d.C * d.H * d.W * elem_size(d.dtype);
    Range ins[5 + 2 * kMaxLevels];
    int ni = 0;
    ins[ni++] = {dy, bytes};
    ni += param_ranges(d, base_w, base_scale, nullptr, level_w, level_scale, ins + ni);
    const Range outs[2] = {{dx, bytes}, {workspace, need}};
    if (any_overlap(outs, 2, ins, ni)) return WTCONV_ERR_ALIAS;
    wtc::ParamPtrs p;
    fill_params(p, d.L, base_w, base_scale, nullptr, level_w, level_scale);
    p.rot = 1;  // the forward pass on dy with every kernel rotated by 180 degrees
    return forward_impl(d, dy, p, dx, reinterpret_cast<char*>(workspace), 0, stream);
}

wtconv_status wtconv_backward(const wtconv_desc* desc, const void* x, const void* dy,
                              const float* base_w, const float* base_scale, const float* base_bias,
                              const float* const* level_w, const float* const* level_scale,
                              void* dx, float* d_base_w, float* d_base_scale, float* d_base_bias,
                              float* const* d_level_w, float* const* d_level_scale,
                              void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    wtconv_status st = check_desc(desc);
    if (st != WTCONV_OK) return st;
    const wtconv_desc& d = *desc;
    if (!d_base_w || !d_base_scale) return WTCONV_ERR_NULL;
    if ((st = check_levels(d.L, (const float* const*)d_level_w, (const float* const*)d_level_scale)) != WTCONV_OK)
        return st;
    if (!base_w || !base_scale) return WTCONV_ERR_NULL;
    if ((st = check_levels(d.L, level_w, level_scale)) != WTCONV_OK) return st;
    // the gradient outputs join the overlap check of the fused phase
    Range grads[3 + 2 * kMaxLevels];
    const int ng = param_ranges(d, d_base_w, d_base_scale, d_base_bias, (const float* const*)d_level_w,
                                (const float* const*)d_level_scale, grads);
    size_t need = 0;
    st = backward_checks(desc, x, dy, base_w, base_scale, base_bias, level_w, level_scale, dx, workspace,
                         workspace_bytes, grads, ng, &need);
    if (st != WTCONV_OK) return st;
    wtc::ParamPtrs p;
    fill_params(p, d.L, base_w, base_scale, base_bias, level_w, level_scale);
    char* ws = reinterpret_cast<char*>(workspace);
    const Grads gr = grads_of(d.L, d_base_w, d_base_scale, d_base_bias, d_level_w, d_level_scale);
    bool fin_done = false;
    st = partials_impl(d, x, dy, p, dx, ws, 0, stream, &gr, &fin_done);
    if (st != WTCONV_OK) return st;
    return finalize_impl(d, p, gr, ws, 0, stream, fin_done);
}

}  // extern "C"
