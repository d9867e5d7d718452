// Host-only view of the execution planner (no GPU, no kernels): includes the
// library's host source with the kernel launchers stubbed out, and prints the
// plan chosen for each descriptor on stdin ("B C H W k L dtype" per line) as
// one JSON object per line. Built and run by tests/test_planner.py.
#include "wtconv_api.cpp"

#include <stdio.h>

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

static const char* mode_name(Mode m)
{
    switch (m) {
        case Mode::Tiny: return "tiny";
        case Mode::Resident: return "resident";
        case Mode::Split: return "split";
        case Mode::Region: return "region";
        case Mode::None: break;
    }
    return "none";
}

int main()
{
    int B, C, H, W, k, L, dt;
    while (scanf("%d %d %d %d %d %d %d", &B, &C, &H, &W, &k, &L, &dt) == 7) {
        const wtconv_desc d = {B, C, H, W, k, L, (wtconv_dtype)dt};
        const Exec f = choose(d, false);
        const GradExec ge = choose_grad(d);
        const Exec b = choose(d, true);
        GradExec rge;
        const bool region_grad = !ge.use && region_grad_exec(d, b, rge);
        printf("{\"bwd_region_grad\": %d, ", region_grad ? 1 : 0);
        printf("\"fwd_mx_rounds\": %d, \"fwd_mx_first_out\": %d, \"fwd_mx_seg\": [", f.pl.mx.rounds,
               f.pl.mx.first_out);
        for (int r = 0; r < f.pl.mx.rounds; ++r) {
            printf("%s[", r ? ", " : "");
            for (int i = f.pl.mx.seg0[r]; i < f.pl.mx.seg0[r + 1]; ++i) {
                const int sg = f.pl.mx.seg[i];
                printf("%s[%d, %d, %d, %d]", i > f.pl.mx.seg0[r] ? ", " : "", sg & 3, (sg >> 2) & 15, (sg >> 6) & 3,
                       sg >> 8);
            }
            printf("]");
        }
        printf("], ");
        printf("\"fwd_tiles_x\": %d, \"fwd_tiles_xl\": %d, ", f.pl.g.tiles_x, f.pl.g.tiles_xl);
        printf("\"fwd_mode\": \"%s\", \"fwd_m\": %d, \"fwd_PP\": %d, \"fwd_one_round\": %d, \"fwd_merge_deep\": %d, "
               "\"fwd_lds_floats\": %d, \"fwd_nb\": %d, \"fwd_nchunks\": %d, \"grad_pass\": %d, \"grad_levels\": %d, "
               "\"grad_coarse\": %d, \"grad_PP\": %d, \"grad_rounds\": %d, \"grad_lds_floats\": %d, "
               "\"grad_nchunks\": %d, \"bwd_mode\": \"%s\", \"fwd_ws\": %zu, \"bwd_ws\": %zu}\n",
               mode_name(f.mode), f.m, f.pl.PP, f.pl.one_round, f.pl.merge_deep, f.pl.lds_floats, f.pl.nb,
               f.pl.nchunks, ge.use ? 1 : 0, ge.Lf, ge.coarse ? 1 : 0, ge.gp.PP, ge.gp.rounds, ge.gp.lds_floats,
               ge.gp.nchunks, mode_name(b.mode), wtconv_forward_workspace_bytes(&d),
               wtconv_backward_workspace_bytes(&d));
    }
    return 0;
}
