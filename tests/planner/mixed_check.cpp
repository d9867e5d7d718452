// Host-only check of the mixed-round forward plans (no GPU, no kernels):
// includes the library's host source with the kernel launchers stubbed out,
// and for each descriptor on stdin ("B C H W k L dtype" per line) whose forward
// plan uses mixed task rounds verifies, on the CPU, what the kernel relies on:
//   - every (level, band) group lies whole in one round, at or before the
//     first round with output tiles, and every output tile lies in a round at
//     or after it; a round holds at most 256 tasks;
//   - the groups cover every (level, band) once and the output runs cover
//     every output tile of the resident planes once;
//   - every task's correlation window (the rows and 16-byte row reads of a 4x4
//     tile) and every write-back lies inside its own array and inside the
//     workgroup's LDS.
// Prints one line per descriptor: "ok <rounds>", "fused" (not mixed) or
// "FAIL <reason>". Built and run by tests/test_planner.py.
#include "wtconv_api.cpp"

#include <stdio.h>

#include <vector>

namespace wtc {
hipError_t launch_forward(int, wtconv_dtype, const FusedArgs&, int, hipStream_t) { return hipSuccess; }
hipError_t launch_backward(int, wtconv_dtype, const FusedArgs&, int, hipStream_t) { return hipSuccess; }
hipError_t launch_reduce(const ReduceArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_grad(int, wtconv_dtype, const GradArgs&, int, hipStream_t) { return hipSuccess; }
hipError_t launch_carrier(wtconv_dtype, const CarrierArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_tiny(int, wtconv_dtype, bool, const TinyArgs&, hipStream_t) { return hipSuccess; }
int forward_wgs_by_regs(int, wtconv_dtype, bool, int fallback) { return fallback; }
hipError_t launch_forward_mixed(int, wtconv_dtype, const FusedArgs&, int, hipStream_t) { return hipSuccess; }
int mixed_wgs_by_regs(int, wtconv_dtype, int, int fallback) { return fallback; }
}  // namespace wtc

static const char* check(const wtconv_desc& d, const Plan& pl)
{
    const MixedPlan& m = pl.mx;
    const PlaneGeom& g = pl.g;
    const int R = d.k / 2, KP = ceil_to(d.k * d.k, 4), PP = pl.PP;
    const long planes_floats = (long)pl.lds_floats - (long)(1 + 4 * d.L) * KP;
    if (planes_floats < (long)PP * g.plane_floats) return "LDS smaller than the resident planes";
    if (m.rounds < 1 || m.rounds > wtc::kMixedMaxRounds || m.first_out < 0 || m.first_out >= m.rounds)
        return "round counts";
    std::vector<int> seen(4 * (d.L + 1), 0);
    long outs = 0;
    for (int r = 0; r < m.rounds; ++r) {
        long n = 0;
        for (int i = m.seg0[r]; i < m.seg0[r + 1]; ++i) {
            const int s = m.seg[i], kind = s & 3, l = (s >> 2) & 15, q = (s >> 6) & 3, cnt = s >> 8;
            n += cnt;
            if (kind == 1) {
                if (r < m.first_out) return "output tiles before the last round with groups";
                if (m.out0[r] != outs) return "output base of a round";
                outs += cnt;
                continue;
            }
            if (kind != 2 || l < 1 || l > d.L) return "segment kind / level";
            if (r > m.first_out) return "group after the first output round";
            const LevelGeom& lg = g.lv[l];
            if (lg.T != 4) return "level not in 4x4 tiles";
            const int tx = lg.ew / 4, ty = lg.eh / 4;
            if (cnt != PP * tx * ty) return "group size";
            if (seen[4 * l + q]++) return "group twice";
            // every tile of the group: window rows [j0, j0 + 4 + 2R), floats
            // [i0, i0 + ceil4(4 + 2R)) of a band array whose rows run to the
            // next band's origin plus R zero halo rows it may share with it;
            // write-back rows [j0 + R, j0 + R + 4) clipped to the grid
            const int rows = lg.band / lg.pitch + R, na = ceil_to(4 + 2 * R, 4);
            for (int t = 0; t < cnt; ++t) {
                const int p = t / (tx * ty), rem = t % (tx * ty), j0 = 4 * (rem / tx), i0 = 4 * (rem % tx);
                if (j0 + 4 + 2 * R > rows || i0 + na > lg.pitch) return "window outside its band array";
                if (j0 + R + std::min(4, lg.h - j0) > lg.band / lg.pitch) return "write-back past the band's own rows";
                const long base = (long)p * g.plane_floats + lg.off + (long)q * lg.band;
                if (base + (long)(j0 + 4 + 2 * R - 1) * lg.pitch + i0 + na > planes_floats) return "window outside LDS";
                if (std::min(4, lg.h - j0) < 1 || std::min(4, lg.w - i0) < 1) return "tile past the grid";
            }
        }
        if (n > wtc::kThreads) return "round over 256 tasks";
        if (n != m.ntask[r]) return "round task count";
    }
    for (int l = 1; l <= d.L; ++l)
        for (int q = 0; q < 4; ++q)
            if (seen[4 * l + q] != 1) return "group missing";
    if (outs != (long)PP * g.tiles_x * g.tiles_y) return "output tiles not covered once";
    // output windows in the haloed input plane
    const int na = ceil_to(4 + 2 * R, 4);
    if ((g.tiles_y * 4 + 2 * R) > g.xrows || (g.tiles_x - 1) * 4 + na > g.xpitch) return "output window";
    return nullptr;
}

int main()
{
    int B, C, H, W, k, L, dt;
    while (scanf("%d %d %d %d %d %d %d", &B, &C, &H, &W, &k, &L, &dt) == 7) {
        const wtconv_desc d = {B, C, H, W, k, L, (wtconv_dtype)dt};
        const Exec f = choose(d, false);
        if ((f.mode != Mode::Resident && f.mode != Mode::Split) || f.pl.mx.rounds == 0) {
            printf("fused\n");
            continue;
        }
        wtconv_desc pd = d;
        if (f.mode == Mode::Split) pd.L = f.m;
        const char* e = check(pd, f.pl);
        if (e)
            printf("FAIL %s\n", e);
        else
            printf("ok %d\n", f.pl.mx.rounds);
    }
    return 0;
}
