// WTConv kernels for planes of at most 8 x 8 pixels (gfx950).
//
// The last ConvNeXt-T stage has 7 x 7 planes, where the tiled kernel of
// wtconv_kernels.hip cannot fill its lanes: a plane has fewer tiles than a
// wavefront has lanes, and most Haar levels are 4 x 4 grids or smaller. Here
// a lane owns a whole plane instead: lane = batch entry, wavefront = channel,
// so every lane of a wavefront runs the same instructions with the same
// (broadcast) kernel taps on its own plane.
//
// Each plane is zero-extended to 8 x 8. The Haar levels of the extension are
// the levels of the plane followed by zeros (the grids of Alg. 1 with its
// bottom/right padding are ceil(H / 2^l) x ceil(W / 2^l)), the "same"
// correlations see zeros beyond the grid either way, and anything computed
// beyond the plane only reaches pixels that are never stored. So the whole
// computation is on fixed 8 x 8 / 4 x 4 / 2 x 2 / 1 x 1 grids: all indexing
// is compile-time, every tap that would read zero padding is skipped at
// compile time, and plane, pyramid, filtered coefficients and output stay in
// registers. The arithmetic is that of the tiled kernel: unnormalised
// butterflies (eq. butterfly without its 1/2), kernels folded as s * W and
// s_l * W_l * 4^-l (eq. fold), and the synthesis of Proposition 2 evaluated as
// its cascade from the coarsest level, which needs no 1/2 either.
//
// LDS only transposes HBM traffic -- for a fixed batch entry the four
// channels of a workgroup are one contiguous run of 4*H*W elements, read and
// written with coalesced accesses and turned into one register per lane --
// and reduces the kernel gradients across a wavefront in a fixed order.
#include <stdint.h>

#include "wtconv_device.h"
#include "wtconv_internal.h"

namespace wtc {
namespace {

constexpr int kTE = 8;             // plane edge held per lane
constexpr int kTPos = kTE * kTE;   // positions per plane
// Staging, parking and gradient-scratch rows are 65 floats apart, so that both
// the position-major accesses of the transposes (consecutive lanes = consecutive
// positions) and the lane-major ones (consecutive lanes = consecutive batch
// entries) fall in distinct LDS banks.
constexpr int kTPitch = 65;
constexpr int kTStage = 64 * kTPitch;  // floats per wavefront
static_assert(kTStage == kTinyStageFloats, "tiny_lds_bytes() sizes the staging areas");


// Index of the folded-kernel row for the base kernel (0) or level l band q.
DEV int trow(int l, int q) { return l == 0 ? 0 : 1 + (l - 1) * 4 + q; }

template <int K>
DEV void load_taps(const float* __restrict__ wt, int row, bool rot, float (&w)[K * K])
{
    constexpr int KK = K * K;
#pragma unroll
    for (int i = 0; i < KK; ++i) w[i] = wt[row * KK + (rot ? KK - 1 - i : i)];
}

// z = w (*) u on an N x N grid, "same" with zero outside the grid; rows >= rows
// of the output are not needed and are left at zero.
template <int K, int N>
DEV void grid_conv(const float (&u)[N * N], const float (&w)[K * K], float (&z)[N * N], int rows = N)
{
    constexpr int R = K / 2;
#pragma unroll
    for (int j = 0; j < N; ++j) {
        if (j >= rows) {
#pragma unroll
            for (int i = 0; i < N; ++i) z[j * N + i] = 0.f;
            continue;
        }
#pragma unroll
        for (int i = 0; i < N; ++i) {
            float acc = 0.f;  // fma(w, u, 0) rounds like the product w * u
#pragma unroll
            for (int p = 0; p < K; ++p) {
                const int y = j + p - R;
                if (y < 0 || y >= N) continue;
#pragma unroll
                for (int t = 0; t < K; ++t) {
                    const int x = i + t - R;
                    if (x < 0 || x >= N) continue;
                    acc = __builtin_fmaf(w[p * K + t], u[y * N + x], acc);
                }
            }
            z[j * N + i] = acc;
        }
    }
}

// grid_conv on the 8 x 8 grid with every output written straight to this
// lane's column of the position-major rows `park` (rows >= `rows`: zero), so
// the 64 outputs never occupy registers together.
template <int K>
DEV void grid_conv8_park(const float (&u)[64], const float (&w)[K * K], float init, float* park, int lane, int rows)
{
    constexpr int R = K / 2, N = 8;
#pragma unroll
    for (int j = 0; j < N; ++j) {
        if (j >= rows) {
#pragma unroll
            for (int i = 0; i < N; ++i) park[(j * N + i) * kTPitch + lane] = 0.f;
            continue;
        }
#pragma unroll
        for (int i = 0; i < N; ++i) {
            float acc = init;  // the folded bias (zero in the backward pass)
#pragma unroll
            for (int p = 0; p < K; ++p) {
                const int y = j + p - R;
                if (y < 0 || y >= N) continue;
#pragma unroll
                for (int t = 0; t < K; ++t) {
                    const int x = i + t - R;
                    if (x < 0 || x >= N) continue;
                    acc = __builtin_fmaf(w[p * K + t], u[y * N + x], acc);
                }
            }
            park[(j * N + i) * kTPitch + lane] = acc;
        }
    }
}

// g[p][t] += sum over sites (j < rows) of d[j][i] * u[j+p-R][i+t-R].
template <int K, int N>
DEV void grid_corr(const float (&d)[N * N], const float (&u)[N * N], float (&g)[K * K], int rows = N)
{
    constexpr int R = K / 2;
#pragma unroll
    for (int j = 0; j < N; ++j) {
        if (j >= rows) break;
#pragma unroll
        for (int i = 0; i < N; ++i)
#pragma unroll
            for (int p = 0; p < K; ++p) {
                const int y = j + p - R;
                if (y < 0 || y >= N) continue;
#pragma unroll
                for (int t = 0; t < K; ++t) {
                    const int x = i + t - R;
                    if (x < 0 || x >= N) continue;
                    g[p * K + t] = __builtin_fmaf(d[j * N + i], u[y * N + x], g[p * K + t]);
                }
            }
    }
}

// Taps of a k x k kernel that can touch an N x N grid from inside it.
template <int K, int N>
constexpr bool tap_live(int tap)
{
    const int R = K / 2, dp = tap / K - R, dt = tap % K - R;
    return dp > -N && dp < N && dt > -N && dt < N;
}

// One analysis level: unnormalised butterflies of the N x N grid u into four
// bands of the (N/2) x (N/2) grid (N = 1: the grid is zero-padded to 2 x 2).
template <int N>
DEV void analyse(const float (&u)[N * N], float (&o)[4][(N > 1 ? N / 2 : 1) * (N > 1 ? N / 2 : 1)])
{
    if constexpr (N == 1) {
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q][0] = u[0];
    } else {
        constexpr int M = N / 2;
#pragma unroll
        for (int j = 0; j < M; ++j)
#pragma unroll
            for (int i = 0; i < M; ++i) {
                float c[4];
                butterfly(u[(2 * j) * N + 2 * i], u[(2 * j) * N + 2 * i + 1], u[(2 * j + 1) * N + 2 * i],
                          u[(2 * j + 1) * N + 2 * i + 1], c);
#pragma unroll
                for (int q = 0; q < 4; ++q) o[q][j * M + i] = c[q];
            }
    }
}

// One synthesis step of the cascade: the four (filtered) bands z of an M x M
// grid, with `carry` added to LL, expanded into the 2M x 2M grid (each site
// (j, i) gives LL+LH+HL+HH, LL+LH-HL-HH, LL-LH+HL-HH, LL-LH-HL+HH at its
// pixels (0,0), (0,1), (1,0), (1,1)).
template <int M>
DEV void expand(const float (&z)[4][M * M], const float (&carry)[M * M], float (&out)[4 * M * M])
{
#pragma unroll
    for (int j = 0; j < M; ++j)
#pragma unroll
        for (int i = 0; i < M; ++i) {
            const int s = j * M + i;
            const float ll = z[0][s] + carry[s];
            const float u = ll + z[1][s], v = ll - z[1][s], a = z[2][s] + z[3][s], b = z[2][s] - z[3][s];
            out[(2 * j) * 2 * M + 2 * i] = u + a;
            out[(2 * j) * 2 * M + 2 * i + 1] = u - a;
            out[(2 * j + 1) * 2 * M + 2 * i] = v + b;
            out[(2 * j + 1) * 2 * M + 2 * i + 1] = v - b;
        }
}

// Kernel-gradient sums of one wavefront, reduced across its 64 lanes in a
// fixed order through an LDS scratch: lane l puts value n at scr[l * 65 + n];
// at a flush, lane n sums column n over l = 0..63 and writes it to the partial
// row at the offset recorded for n.
struct GradQueue {
    float* scr;  // 64 x kTPitch floats of this wavefront
    int* offs;   // 64 partial-row offsets
    int n;
};

DEV void wave_sync() { __builtin_amdgcn_wave_barrier(); }

DEV void gq_flush(GradQueue& q, float* __restrict__ dst, int lane, bool store)
{
    if (q.n == 0) return;
    wave_sync();
    if (lane < q.n) {
        float s = 0.f;
        for (int l = 0; l < 64; ++l) s += q.scr[l * kTPitch + lane];
        if (store) dst[q.offs[lane]] = s;
    }
    wave_sync();
    q.n = 0;
}

// Queue the live taps of one kernel gradient g (partial-row offset `off`) and
// write zeros for the taps that cannot be reached on an N x N grid.
template <int K, int N>
DEV void gq_put(GradQueue& q, const float (&g)[K * K], int off, float* __restrict__ dst, int lane, bool store)
{
    constexpr int KK = K * K;
    int live = 0;
#pragma unroll
    for (int t = 0; t < KK; ++t) live += tap_live<K, N>(t) ? 1 : 0;
    if (q.n + live > 64) gq_flush(q, dst, lane, store);
#pragma unroll
    for (int t = 0; t < KK; ++t) {
        if (tap_live<K, N>(t)) {
            if constexpr (KK > 64)  // k = 9: more live taps than a flush holds
                if (q.n == 64) gq_flush(q, dst, lane, store);
            q.scr[lane * kTPitch + q.n] = g[t];
            if (lane == 0) q.offs[q.n] = off + t;
            ++q.n;
        } else if (store && lane == 0) {
            dst[off + t] = 0.f;
        }
    }
}

// Queue one value (partial-row offset `off`).
DEV void gq_put1(GradQueue& q, float v, int off, float* __restrict__ dst, int lane, bool store)
{
    if (q.n + 1 > 64) gq_flush(q, dst, lane, store);
    q.scr[lane * kTPitch + q.n] = v;
    if (lane == 0) q.offs[q.n] = off;
    ++q.n;
}

template <int K, typename ST, bool BWD>
__global__ void __launch_bounds__(256) tiny_kernel(const TinyArgs a)
{
    constexpr int KK = K * K;
    extern __shared__ float4 tlds4[];
    float* lds = reinterpret_cast<float*>(tlds4);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ncg = (a.C + 3) / 4;
    const int cg = blockIdx.x % ncg, bg = blockIdx.x / ncg;
    const int c0 = cg * 4, b0 = bg * 64;
    const int nch = min(4, a.C - c0);
    const int c = c0 + wave;
    const bool cvalid = wave < nch;
    const int H = a.H, W = a.W, HW = H * W, L = a.L;
    const int nrows = 1 + 4 * L;

    float* stage = lds;                        // [4][kTStage]
    float* wtab = lds + 4 * kTStage;           // [4][nrows][KK]
    int* offs = reinterpret_cast<int*>(wtab + 4 * nrows * KK);  // [4][64]
    float* mystage = stage + wave * kTStage;
    const float* mytab = wtab + wave * nrows * KK;

    for (int i = tid; i < 4 * kTStage / 4; i += 256) tlds4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    // eq. (fold): base s0*W0; level l band q: s_l*W_l*4^-l
    const bool rot = !BWD && a.p.rot != 0;  // forward pass computing dx: taps reversed
    for (int i = tid; i < nch * nrows * KK; i += 256) {
        const int cl = i / (nrows * KK), r = i - cl * (nrows * KK);
        const int row = r / KK, tt = r - row * KK, cc = c0 + cl;
        const int t = rot ? KK - 1 - tt : tt;
        float v;
        if (row == 0) {
            v = a.p.s0[cc] * a.p.w0[cc * KK + t];
        } else {
            const int l = (row - 1) / 4 + 1, q = (row - 1) - (l - 1) * 4;
            v = a.p.ls[l - 1][4 * cc + q] * a.p.lw[l - 1][(4 * cc + q) * KK + t] * __builtin_ldexpf(1.f, -2 * l);
        }
        wtab[cl * nrows * KK + r] = v;
    }
    __syncthreads();

    // coalesced staging: thread t <-> element t of the run [b][c0 .. c0+nch-1][H][W]
    const int run = nch * HW;
    int my_slot = -1;
    if (tid < run) {
        const int cl = tid / HW, pos = tid - cl * HW, y = pos / W, x = pos - y * W;
        my_slot = cl * kTStage + (y * kTE + x) * kTPitch;
    }
    const int nb = min(64, a.B - b0);
    const long bstep = (long)a.C * HW;
    // all 64 loads are issued before any is used (addresses clamped to the last
    // batch entry; entries past it stage zeros, so they add nothing anywhere)
    auto stage_in = [&](const ST* __restrict__ src, float (&v)[kTPos]) {
        if (my_slot >= 0) {
            const ST* p = src + ((long)b0 * a.C + c0) * HW + tid;
            float t[64];
#pragma unroll
            for (int bl = 0; bl < 64; ++bl) t[bl] = to_f32(p[min(bl, nb - 1) * bstep]);
#pragma unroll
            for (int bl = 0; bl < 64; ++bl) stage[my_slot + bl] = bl < nb ? t[bl] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kTPos; ++i) v[i] = mystage[i * kTPitch + lane];
        __syncthreads();
    };
    // store the values parked at `rows` ([4][kTStage], position-major)
    auto store_out = [&](ST* __restrict__ dst, const float* rows) {
        __syncthreads();
        if (my_slot >= 0) {
            ST* p = dst + ((long)b0 * a.C + c0) * HW + tid;
            const int off = my_slot;
#pragma unroll 16
            for (int bl = 0; bl < nb; ++bl) p[bl * bstep] = from_f32<ST>(rows[off + bl]);
        }
    };
    // the last synthesis step, added onto the values parked at `park` (own rows)
    auto expand_add = [&](const float (&z)[4][16], const float (&carry)[16], float* park) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int s = j * 4 + i;
                const float ll = z[0][s] + carry[s];
                const float u = ll + z[1][s], v = ll - z[1][s], p2 = z[2][s] + z[3][s], m2 = z[2][s] - z[3][s];
                park[((2 * j) * 8 + 2 * i) * kTPitch + lane] += u + p2;
                park[((2 * j) * 8 + 2 * i + 1) * kTPitch + lane] += u - p2;
                park[((2 * j + 1) * 8 + 2 * i) * kTPitch + lane] += v + m2;
                park[((2 * j + 1) * 8 + 2 * i + 1) * kTPitch + lane] += v - m2;
            }
    };
    auto centre = [&](int l, int q) { return mytab[trow(l, q) * KK + KK / 2]; };

    const bool skip_base = a.skip_base != 0;
    float w[KK];

    if constexpr (!BWD) {
        float X[kTPos];
        stage_in(reinterpret_cast<const ST*>(a.in), X);
        // the base output is parked in this wavefront's staging rows
        if (skip_base) {
#pragma unroll
            for (int i = 0; i < kTPos; ++i) mystage[i * kTPitch + lane] = 0.f;
        } else {
            load_taps<K>(mytab, trow(0, 0), false, w);
            // eq. (fold): the folded base bias s0 * b0 starts every output pixel's sum
            const float bias = (cvalid && a.p.b0) ? a.p.s0[c] * a.p.b0[c] : 0.f;
            grid_conv8_park<K>(X, w, bias, mystage, lane, H);
        }
        if (L >= 1) {
            float U1[4][16], U2[4][4], U3[4];
            analyse<8>(X, U1);
            analyse<4>(U1[0], U2);
            {
                float t[4][1];
                analyse<2>(U2[0], t);
#pragma unroll
                for (int q = 0; q < 4; ++q) U3[q] = t[q][0];
            }
            // levels >= 4 are 1 x 1 grids whose four raw bands all equal the
            // level-3 LL (the padded butterfly of a single value); only the
            // centre tap reaches them. Cascade from the coarsest level.
            float r1 = 0.f;
#pragma unroll
            for (int l = kMaxLevels; l >= 4; --l) {
                if (l > L) continue;
                const float f0 = centre(l, 0) * U3[0], f1 = centre(l, 1) * U3[0];
                const float f2 = centre(l, 2) * U3[0], f3 = centre(l, 3) * U3[0];
                r1 = ((f0 + r1) + f1) + (f2 + f3);
            }
            float rec2[4] = {0.f, 0.f, 0.f, 0.f};
            if (L >= 3) {
                float z3[4][1];
#pragma unroll
                for (int q = 0; q < 4; ++q) z3[q][0] = centre(3, q) * U3[q];
                const float cr[1] = {r1};
                expand<1>(z3, cr, rec2);
            }
            float rec1[16];
            if (L >= 2) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float z[4];
                    load_taps<K>(mytab, trow(2, q), false, w);
                    grid_conv<K, 2>(U2[q], w, z);
#pragma unroll
                    for (int s2 = 0; s2 < 4; ++s2) U2[q][s2] = z[s2];
                }
                expand<2>(U2, rec2, rec1);
            } else {
#pragma unroll
                for (int s2 = 0; s2 < 16; ++s2) rec1[s2] = 0.f;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float z[16];
                load_taps<K>(mytab, trow(1, q), false, w);
                grid_conv<K, 4>(U1[q], w, z);
#pragma unroll
                for (int s2 = 0; s2 < 16; ++s2) U1[q][s2] = z[s2];
            }
            expand_add(U1, rec1, mystage);
        }
        store_out(reinterpret_cast<ST*>(a.out), stage);
    } else {
        // ---------------- backward ----------------
        float* park = lds + 4 * kTStage + 4 * nrows * KK + 4 * 64;  // [4][kTStage], dx accumulation
        float* mypark = park + wave * kTStage;
        float X[kTPos], D[kTPos];
        stage_in(reinterpret_cast<const ST*>(a.aux), X);
        stage_in(reinterpret_cast<const ST*>(a.in), D);
        const int NP = partial_floats_per_channel(K, L);  // KK * nrows taps, then the sum of dy
        float* prow = a.partial + ((long)bg * a.C + (cvalid ? c : 0)) * NP;
        const bool store_g = cvalid;
        GradQueue gq = {mystage, offs + wave * 64, 0};
        const bool want_dx = a.out != nullptr;

        if (skip_base) {
#pragma unroll
            for (int i = 0; i < kTPos; ++i) mypark[i * kTPitch + lane] = 0.f;
        } else {
            float g[KK];
#pragma unroll
            for (int t = 0; t < KK; ++t) g[t] = 0.f;
            grid_corr<K, 8>(D, X, g, H);
            gq_put<K, 8>(gq, g, 0, prow, lane, store_g);
            // the bias gradient: sum of this entry's dy plane (zero beyond it)
            float sdy = 0.f;
#pragma unroll
            for (int i = 0; i < kTPos; ++i) sdy += D[i];
            gq_put1(gq, sdy, NP - 1, prow, lane, store_g);
            load_taps<K>(mytab, trow(0, 0), true, w);
            grid_conv8_park<K>(D, w, 0.f, mypark, lane, H);
        }
        if (L >= 1) {
            float U1[4][16], V1[4][16];
            analyse<8>(X, U1);
            analyse<8>(D, V1);
            float U2[4][4], V2[4][4], U3[4], V3[4];
            analyse<4>(U1[0], U2);
            analyse<4>(V1[0], V2);
            {
                float tu[4][1], tv[4][1];
                analyse<2>(U2[0], tu);
                analyse<2>(V2[0], tv);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    U3[q] = tu[q][0];
                    V3[q] = tv[q][0];
                }
            }
            // levels >= 4: 1 x 1 grids, raw bands all equal to the level-3 LL;
            // only the centre tap (its own rotation) reaches them
            float r1 = 0.f;
#pragma unroll
            for (int l = kMaxLevels; l >= 4; --l) {
                if (l > L) continue;
                float f[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float g[KK];
#pragma unroll
                    for (int t = 0; t < KK; ++t) g[t] = 0.f;
                    g[KK / 2] = V3[0] * U3[0];
                    gq_put<K, 1>(gq, g, KK * trow(l, q), prow, lane, store_g);
                    f[q] = centre(l, q) * V3[0];
                }
                r1 = ((f[0] + r1) + f[1]) + (f[2] + f[3]);
            }
            float rec2[4] = {0.f, 0.f, 0.f, 0.f};
            if (L >= 3) {
                float z3[4][1];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float g[KK];
#pragma unroll
                    for (int t = 0; t < KK; ++t) g[t] = 0.f;
                    g[KK / 2] = V3[q] * U3[q];
                    gq_put<K, 1>(gq, g, KK * trow(3, q), prow, lane, store_g);
                    z3[q][0] = centre(3, q) * V3[q];
                }
                const float cr[1] = {r1};
                expand<1>(z3, cr, rec2);
            }
            float rec1[16];
            if (L >= 2) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float g[KK];
#pragma unroll
                    for (int t = 0; t < KK; ++t) g[t] = 0.f;
                    grid_corr<K, 2>(V2[q], U2[q], g);
                    gq_put<K, 2>(gq, g, KK * trow(2, q), prow, lane, store_g);
                    float z[4];
                    load_taps<K>(mytab, trow(2, q), true, w);
                    grid_conv<K, 2>(V2[q], w, z);
#pragma unroll
                    for (int s2 = 0; s2 < 4; ++s2) V2[q][s2] = z[s2];
                }
                expand<2>(V2, rec2, rec1);
            } else {
#pragma unroll
                for (int s2 = 0; s2 < 16; ++s2) rec1[s2] = 0.f;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float g[KK];
#pragma unroll
                for (int t = 0; t < KK; ++t) g[t] = 0.f;
                grid_corr<K, 4>(V1[q], U1[q], g);
                gq_put<K, 4>(gq, g, KK * trow(1, q), prow, lane, store_g);
                float z[16];
                load_taps<K>(mytab, trow(1, q), true, w);
                grid_conv<K, 4>(V1[q], w, z);
#pragma unroll
                for (int s2 = 0; s2 < 16; ++s2) V1[q][s2] = z[s2];
            }
            expand_add(V1, rec1, mypark);
        }
        gq_flush(gq, prow, lane, store_g);
        if (want_dx) store_out(reinterpret_cast<ST*>(a.out), park);
    }
}

}  // namespace


namespace {

template <int K, typename ST, bool BWD>
hipError_t launch_tiny_variant(const TinyArgs& a, hipStream_t s)
{
    const size_t bytes = tiny_lds_bytes(K, a.L, BWD);
    static std::atomic<unsigned long long> lds_done{0};
    const hipError_t e = allow_full_lds(reinterpret_cast<const void*>(&tiny_kernel<K, ST, BWD>), lds_done);
    if (e != hipSuccess) return e;
    const int grid = ((a.C + 3) / 4) * ((a.B + 63) / 64);
    hipLaunchKernelGGL((tiny_kernel<K, ST, BWD>), dim3(grid), dim3(256), bytes, s, a);
    return hipGetLastError();
}

template <bool BWD>
hipError_t tiny_dispatch(int k, wtconv_dtype dt, const TinyArgs& a, hipStream_t s)
{
#define WTC_TCASE(KV)                                                                 \
    case KV:                                                                          \
        switch (dt) {                                                                 \
            case WTCONV_F32: return launch_tiny_variant<KV, float, BWD>(a, s);        \
            case WTCONV_BF16: return launch_tiny_variant<KV, uint16_t, BWD>(a, s);    \
            case WTCONV_F16: return launch_tiny_variant<KV, _Float16, BWD>(a, s);     \
        }                                                                             \
        break;
    switch (k) {
        WTC_TCASE(1)
        WTC_TCASE(3)
        WTC_TCASE(5)
        WTC_TCASE(7)
        WTC_TCASE(9)
    }
#undef WTC_TCASE
    return hipErrorInvalidValue;
}

}  // namespace


hipError_t launch_tiny(int k, wtconv_dtype dt, bool bwd, const TinyArgs& a, hipStream_t s)
{
    return bwd ? tiny_dispatch<true>(k, dt, a, s) : tiny_dispatch<false>(k, dt, a, s);
}

}  // namespace wtc
