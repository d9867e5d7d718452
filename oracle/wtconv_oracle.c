/*
 * wtconv_oracle.c -- fp64 CPU oracle for the WTConv operator.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the correctness reference that the
 * GPU library is checked against. It shares no code, header, table or helper
 * with the GPU path, and nothing in the product path may load it: only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg do.
 *
 * What it computes (Aflalo et al., "Fast and Memory-Efficient Wavelet
 * Convolutions via I/O-Aware Reformulation"):
 *
 *   the WTConv operator of Section 2.1 (Alg. 1), materialised in float64,
 *   one (batch, channel) plane at a time. Its output is a base path plus a
 *   wavelet branch. The base path is the plane correlated with the base
 *   kernel W0, plus the bias b, times the base scale s0. The wavelet branch
 *   takes an L-level Haar pyramid of the plane (level 1 analyses the plane,
 *   level l analyses the unfiltered low-pass band of level l-1), correlates
 *   each of the four bands of every level with its own kernel and multiplies
 *   it by its own scale, and synthesises the result back level by level from
 *   the coarsest: at each level the reconstruction from below joins the
 *   filtered low-pass band before one synthesis step.
 *   A is one level of the orthonormal 2x2 Haar transform, i.e. the matrix of
 *   Proposition 1 applied to every non-overlapping 2x2 block, with the band
 *   formulas of eq. (butterfly) in Section 4.1. A^T is its synthesis.
 *   "(*)" is the depthwise k x k "same" cross-correlation with zero padding
 *   (Section 2.1 notation; PyTorch conv2d semantics).
 *
 * Readings of points the paper leaves open (each is listed in the design
 * notes of the repository):
 *   - odd sizes: before each analysis level the carrier is zero-padded at the
 *     bottom/right to even size; after each synthesis level the result is
 *     cropped back to the size of that level's input;
 *   - the four subbands of channel c at level l are convolution channels
 *     4c+q with q = 0 LL, 1 LH, 2 HL, 3 HH; the level scale has one entry per
 *     convolution channel (4C entries), the base scale one per channel;
 *   - zero padding of the convolutions in coefficient space is zero outside
 *     the level's grid;
 *   - k is odd, R = (k-1)/2.
 *
 * The backward pass is the exact reverse-mode adjoint of the steps above:
 * the adjoint of a crop is a zero pad, the adjoint of analysis-with-pad is
 * synthesis-with-crop (Section 2.2: H is symmetric and self-inverse), the
 * adjoint of a same-correlation is the correlation with the kernel rotated
 * by 180 degrees, and the parameter gradients are correlations of the
 * upstream gradient with the layer input. Per-plane parameter gradients are
 * summed over the batch in increasing batch order.
 *
 * The closed-form synthesis (Proposition 2, Section 4.2, proved in
 * Appendix A) is implemented separately, only so that tests can compare it
 * with the cascade; the forward pass above never uses it.
 *
 * Layouts: x, y, dy, dx are [B][C][H][W]; base_w [C][k][k]; base_scale [C];
 * level_w [L][4C][k][k]; level_scale [L][4C]. All float64, C-contiguous.
 */
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Rows of the Haar matrix H of Proposition 1, indexed [band q][position],
 * position = 2*ry + rx within a 2x2 block [[a,b],[c,d]] = (0,0),(0,1),(1,0),(1,1).
 * Row q reproduces eq. (butterfly): LL=a+b+c+d, LH=a+b-c-d, HL=a-b+c-d,
 * HH=a-b-c+d, each times 1/2. */
static const double HAAR[4][4] = {
    {+1.0, +1.0, +1.0, +1.0},
    {+1.0, +1.0, -1.0, -1.0},
    {+1.0, -1.0, +1.0, -1.0},
    {+1.0, -1.0, -1.0, +1.0},
};

static int half_up(int n) { return (n + 1) / 2; }

/* One analysis level (Alg. 1, Y = A X) with bottom/right zero padding to even
 * size. X is h x w; Y is 4 x ceil(h/2) x ceil(w/2), band-major. */
void oracle_haar_analysis(int h, int w, const double* X, double* Y)
{
    const int ho = half_up(h), wo = half_up(w);
    for (int q = 0; q < 4; ++q)
        for (int j = 0; j < ho; ++j)
            for (int i = 0; i < wo; ++i) {
                double acc = 0.0;
                for (int ry = 0; ry < 2; ++ry)
                    for (int rx = 0; rx < 2; ++rx) {
                        const int yy = 2 * j + ry, xx = 2 * i + rx;
                        const double v = (yy < h && xx < w) ? X[yy * w + xx] : 0.0;
                        acc += HAAR[q][2 * ry + rx] * v;
                    }
                Y[(q * ho + j) * wo + i] = 0.5 * acc;
            }
}

/* One synthesis level (Alg. 1, A^T): the 4-band coefficients on a
 * ceil(h/2) x ceil(w/2) grid are expanded to 2x2 blocks with the same matrix
 * (H^T = H), and the even-size result is cropped to h x w. */
void oracle_haar_synthesis(int h, int w, const double* Y, double* X)
{
    const int ho = half_up(h), wo = half_up(w);
    for (int yy = 0; yy < h; ++yy)
        for (int xx = 0; xx < w; ++xx) {
            const int j = yy / 2, i = xx / 2, pos = 2 * (yy % 2) + (xx % 2);
            double acc = 0.0;
            for (int q = 0; q < 4; ++q)
                acc += HAAR[q][pos] * Y[(q * ho + j) * wo + i];
            X[yy * w + xx] = 0.5 * acc;
        }
}

/* "same" cross-correlation with zero padding:
 * out[y][x] = sum_{p,t} wk[p][t] * u[y+p-R][x+t-R]. */
void oracle_corr_same(int h, int w, int k, const double* u, const double* wk, double* out)
{
    const int R = (k - 1) / 2;
    for (int y = 0; y < h; ++y)
        for (int x = 0; x < w; ++x) {
            double acc = 0.0;
            for (int p = 0; p < k; ++p) {
                const int yy = y + p - R;
                if (yy < 0 || yy >= h) continue;
                for (int t = 0; t < k; ++t) {
                    const int xx = x + t - R;
                    if (xx < 0 || xx >= w) continue;
                    acc += wk[p * k + t] * u[yy * w + xx];
                }
            }
            out[y * w + x] = acc;
        }
}

/* Adjoint of oracle_corr_same with respect to its input u:
 * out[y][x] = sum_{p,t} wk[p][t] * g[y-p+R][x-t+R]. */
static void corr_same_adjoint(int h, int w, int k, const double* g, const double* wk, double* out)
{
    const int R = (k - 1) / 2;
    for (int y = 0; y < h; ++y)
        for (int x = 0; x < w; ++x) {
            double acc = 0.0;
            for (int p = 0; p < k; ++p) {
                const int yy = y - p + R;
                if (yy < 0 || yy >= h) continue;
                for (int t = 0; t < k; ++t) {
                    const int xx = x - t + R;
                    if (xx < 0 || xx >= w) continue;
                    acc += wk[p * k + t] * g[yy * w + xx];
                }
            }
            out[y * w + x] = acc;
        }
}

/* Gradient of oracle_corr_same with respect to its kernel:
 * gw[p][t] = sum_{y,x} g[y][x] * u[y+p-R][x+t-R]. Accumulates into gw. */
static void corr_same_kernel_grad(int h, int w, int k, const double* g, const double* u, double* gw)
{
    const int R = (k - 1) / 2;
    for (int p = 0; p < k; ++p)
        for (int t = 0; t < k; ++t) {
            double acc = 0.0;
            for (int y = 0; y < h; ++y) {
                const int yy = y + p - R;
                if (yy < 0 || yy >= h) continue;
                for (int x = 0; x < w; ++x) {
                    const int xx = x + t - R;
                    if (xx < 0 || xx >= w) continue;
                    acc += g[y * w + x] * u[yy * w + xx];
                }
            }
            gw[p * k + t] += acc;
        }
}

/* Sizes of the level grids: hs[0] = H, hs[l] = ceil(hs[l-1] / 2). */
static void level_sizes(int H, int W, int L, int* hs, int* ws)
{
    hs[0] = H;
    ws[0] = W;
    for (int l = 1; l <= L; ++l) {
        hs[l] = half_up(hs[l - 1]);
        ws[l] = half_up(ws[l - 1]);
    }
}

/* Number of doubles in the concatenated coefficient pyramid of levels 1..L
 * (each level 4 x H_l x W_l, band-major). */
long oracle_pyramid_size(int H, int W, int L)
{
    int hs[64], ws[64];
    if (L < 0 || L > 60) return -1;
    level_sizes(H, W, L, hs, ws);
    long n = 0;
    for (int l = 1; l <= L; ++l) n += 4L * hs[l] * ws[l];
    return n;
}

/* The unfiltered Haar pyramid Y_1..Y_L of one plane (Alg. 1): level l is the
 * analysis of level l-1's unfiltered low-pass band (of x itself for l = 1). */
int oracle_plane_pyramid(int H, int W, int L, const double* x, double* y_out)
{
    int hs[64], ws[64];
    if (H < 1 || W < 1 || L < 0 || L > 60) return 1;
    level_sizes(H, W, L, hs, ws);
    double* carrier = (double*)malloc(sizeof(double) * (size_t)H * W);
    if (!carrier) return 2;
    memcpy(carrier, x, sizeof(double) * (size_t)H * W);
    long off = 0;
    for (int l = 1; l <= L; ++l) {
        double* Y = y_out + off;
        oracle_haar_analysis(hs[l - 1], ws[l - 1], carrier, Y);
        memcpy(carrier, Y, sizeof(double) * (size_t)hs[l] * ws[l]); /* raw LL */
        off += 4L * hs[l] * ws[l];
    }
    free(carrier);
    return 0;
}

/*
 * Synthesis cascade of Alg. 1, from the coarsest level to the finest: the
 * partial reconstruction coming up from the level below (zero under the
 * coarsest) is added to the filtered LL band of level l, the four bands are
 * synthesised one level (A^T) and cropped to the size of level l-1's grid.
 * z is the pyramid Z_1..Z_L laid out as in oracle_pyramid_size; R is H x W.
 * With L = 0, R = 0.
 */
int oracle_cascade_synthesis(int H, int W, int L, const double* z, double* R)
{
    int hs[64], ws[64];
    if (H < 1 || W < 1 || L < 0 || L > 60) return 1;
    level_sizes(H, W, L, hs, ws);
    double* U = (double*)malloc(sizeof(double) * 4 * (size_t)H * W + 8);
    double* Rn = (double*)malloc(sizeof(double) * (size_t)H * W);
    if (!U || !Rn) {
        free(U); free(Rn);
        return 2;
    }
    for (long e = 0; e < (long)H * W; ++e) R[e] = 0.0;
    long off = oracle_pyramid_size(H, W, L);
    int have_r = 0;
    for (int l = L; l >= 1; --l) {
        const int n = hs[l] * ws[l];
        off -= 4L * n;
        memcpy(U, z + off, sizeof(double) * 4 * (size_t)n);
        if (have_r)
            for (int e = 0; e < n; ++e) U[e] += Rn[e];                     /* onto the LL band */
        oracle_haar_synthesis(hs[l - 1], ws[l - 1], U, Rn);                /* one level up, cropped */
        have_r = 1;
    }
    if (have_r) memcpy(R, Rn, sizeof(double) * (size_t)H * W);
    free(U); free(Rn);
    return 0;
}

/*
 * Forward pass of one plane (the operator of Alg. 1), built from its four
 * parts in turn, each materialised in full:
 *   1. the unfiltered Haar pyramid Y_1..Y_L of x (oracle_plane_pyramid: each
 *      level analyses the raw low-pass band of the level above);
 *   2. every band of every level correlated with its own kernel and
 *      multiplied by its own scale, giving Z_1..Z_L;
 *   3. the synthesis cascade of Z_1..Z_L back to the pixel grid (R);
 *   4. the base path s0 * (x (*) W0 + b0), to which R is added.
 * Arguments:
 *   w0: k*k base kernel, s0: base scale, b0: base bias (added to the base
 *       correlation before the scale multiplies it),
 *   wl: L x 4 x k*k level kernels of this channel (row q of level l is
 *       convolution channel 4c+q), sl: L x 4 level scales,
 *   y: H x W output,
 *   z_out (nullable): the filtered, scaled coefficients Z_1..Z_L, concatenated
 *       as in oracle_pyramid_size.
 */
int oracle_plane_forward(int H, int W, int k, int L, const double* x, const double* w0, double s0,
                         const double* wl, const double* sl, double b0, double* y, double* z_out)
{
    int hs[64], ws[64];
    if (H < 1 || W < 1 || k < 1 || (k % 2) == 0 || L < 0 || L > 60) return 1;
    level_sizes(H, W, L, hs, ws);
    const int kk = k * k;
    const long npyr = oracle_pyramid_size(H, W, L);
    const size_t pyr_bytes = sizeof(double) * (size_t)(npyr > 0 ? npyr : 1);
    double* Y = (double*)malloc(pyr_bytes);
    double* Z = (double*)malloc(pyr_bytes);
    double* R = (double*)malloc(sizeof(double) * (size_t)H * W);
    if (!Y || !Z || !R) {
        free(Y); free(Z); free(R);
        return 2;
    }

    /* 1. analysis pyramid */
    int rc = oracle_plane_pyramid(H, W, L, x, Y);

    /* 2. each band filtered by its kernel, then scaled */
    long off = 0;
    for (int l = 1; l <= L && rc == 0; ++l) {
        const int n = hs[l] * ws[l];
        for (int q = 0; q < 4; ++q) {
            const long band = off + (long)q * n;
            oracle_corr_same(hs[l], ws[l], k, Y + band, wl + ((long)(l - 1) * 4 + q) * kk, Z + band);
            const double s = sl[(l - 1) * 4 + q];
            for (int e = 0; e < n; ++e) Z[band + e] *= s;
        }
        off += 4L * n;
    }

    /* 3. synthesis of the filtered pyramid */
    if (rc == 0) rc = oracle_cascade_synthesis(H, W, L, Z, R);

    /* 4. base path, plus the wavelet branch */
    if (rc == 0) {
        oracle_corr_same(H, W, k, x, w0, y);
        for (long e = 0; e < (long)H * W; ++e) y[e] = s0 * (y[e] + b0) + R[e];
        if (z_out && npyr > 0) memcpy(z_out, Z, sizeof(double) * (size_t)npyr);
    }
    free(Y); free(Z); free(R);
    return rc;
}

/*
 * Closed-form bit-indexed synthesis (Proposition 2): for every output pixel
 *   R[y][x] = sum_l 2^-l ( LL + sy*LH + sx*HL + sy*sx*HH ),
 * with the level-l coefficients read at (floor(y/2^l), floor(x/2^l)) and
 * sy = (-1)^(floor(y/2^(l-1)) mod 2), sx likewise. z is a pyramid laid out as
 * in oracle_pyramid_size. Used only by tests, to compare with the cascade.
 */
void oracle_closed_form_synthesis(int H, int W, int L, const double* z, double* R)
{
    int hs[64], ws[64];
    level_sizes(H, W, L, hs, ws);
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            double acc = 0.0;
            long off = 0;
            double scale = 1.0;
            for (int l = 1; l <= L; ++l) {
                scale *= 0.5;
                const int n = hs[l] * ws[l];
                const int j = y >> l, i = x >> l;
                const double sy = ((y >> (l - 1)) & 1) ? -1.0 : 1.0;
                const double sx = ((x >> (l - 1)) & 1) ? -1.0 : 1.0;
                const double* c = z + off;
                acc += scale * (c[0L * n + j * ws[l] + i] + sy * c[1L * n + j * ws[l] + i] +
                                sx * c[2L * n + j * ws[l] + i] + sy * sx * c[3L * n + j * ws[l] + i]);
                off += 4L * n;
            }
            R[y * W + x] = acc;
        }
}

/*
 * Backward pass of one plane: exact reverse mode through oracle_plane_forward.
 * Outputs dx (H x W) and the plane's parameter gradients:
 *   gw0 [k*k], gs0 [1], gb0 [1], gwl [L x 4 x k*k], gsl [L x 4]  (overwritten).
 * With y_base = s0 (x (*) W0 + b0): dW0 = s0 corr(dy, x), db0 = s0 sum(dy) and
 * ds0 = sum(dy (x (*) W0 + b0)), which is eq. (foldgrad)'s <dW~, W> + db~ b.
 */
int oracle_plane_backward(int H, int W, int k, int L, const double* x, const double* dy,
                          const double* w0, double s0, const double* wl, const double* sl, double b0,
                          double* dx, double* gw0, double* gs0, double* gb0, double* gwl, double* gsl)
{
    int hs[64], ws[64];
    if (H < 1 || W < 1 || k < 1 || (k % 2) == 0 || L < 0 || L > 60) return 1;
    level_sizes(H, W, L, hs, ws);
    const int kk = k * k;
    const long npyr = oracle_pyramid_size(H, W, L);
    const size_t np = (size_t)(npyr > 0 ? npyr : 1);
    const size_t HW = (size_t)H * W;

    double* Y = (double*)malloc(sizeof(double) * np);   /* unfiltered Y_l */
    double* C = (double*)malloc(sizeof(double) * np);   /* unscaled convs Y_l * W_l */
    double* dZ = (double*)malloc(sizeof(double) * np);  /* dL/dZ_l */
    double* carrier = (double*)malloc(sizeof(double) * HW);
    double* dR = (double*)malloc(sizeof(double) * HW);
    double* dYl = (double*)malloc(sizeof(double) * 4 * HW + 8);
    double* dC = (double*)malloc(sizeof(double) * HW);
    double* tmp = (double*)malloc(sizeof(double) * HW);
    double* dcar = (double*)malloc(sizeof(double) * HW);
    long* offs = (long*)malloc(sizeof(long) * (size_t)(L + 2));
    if (!Y || !C || !dZ || !carrier || !dR || !dYl || !dC || !tmp || !dcar || !offs) {
        free(Y); free(C); free(dZ); free(carrier); free(dR); free(dYl); free(dC); free(tmp);
        free(dcar); free(offs);
        return 2;
    }

    /* recompute the forward intermediates needed by the adjoint */
    memcpy(carrier, x, sizeof(double) * HW);
    long off = 0;
    for (int l = 1; l <= L; ++l) {
        const int n = hs[l] * ws[l];
        offs[l] = off;
        oracle_haar_analysis(hs[l - 1], ws[l - 1], carrier, Y + off);
        for (int q = 0; q < 4; ++q)
            oracle_corr_same(hs[l], ws[l], k, Y + off + (long)q * n, wl + ((long)(l - 1) * 4 + q) * kk,
                             C + off + (long)q * n);
        memcpy(carrier, Y + off, sizeof(double) * (size_t)n);
        off += 4L * n;
    }

    /* base path: y_base = s0 * (corr(x, w0) + b0) */
    for (int t = 0; t < kk; ++t) gw0[t] = 0.0;
    oracle_corr_same(H, W, k, x, w0, tmp);
    double g = 0.0, sdy = 0.0;
    for (size_t e = 0; e < HW; ++e) {
        g += dy[e] * (tmp[e] + b0);
        sdy += dy[e];
    }
    *gs0 = g;
    *gb0 = s0 * sdy;
    for (size_t e = 0; e < HW; ++e) dC[e] = s0 * dy[e];
    corr_same_kernel_grad(H, W, k, dC, x, gw0);
    corr_same_adjoint(H, W, k, dC, w0, dx);

    /* adjoint of the upward cascade: R_l = crop(A^T(U_l)), U_l = Z_l with LL += R_{l+1}.
     * dU_l = A(pad(dR_l)); dZ_l = dU_l; dR_{l+1} = LL(dU_l). */
    memcpy(dR, dy, sizeof(double) * HW);
    for (int l = 1; l <= L; ++l) {
        const int n = hs[l] * ws[l];
        oracle_haar_analysis(hs[l - 1], ws[l - 1], dR, dZ + offs[l]);
        memcpy(dR, dZ + offs[l], sizeof(double) * (size_t)n);
    }

    /* adjoint of the downward loop, deepest level first */
    for (int e = 0; e < (int)HW; ++e) dcar[e] = 0.0;     /* dL/dX_L = 0: the deepest raw LL is unused */
    for (int l = L; l >= 1; --l) {
        const int n = hs[l] * ws[l];
        memset(dYl, 0, sizeof(double) * 4 * (size_t)n);
        for (int e = 0; e < n; ++e) dYl[e] += dcar[e];    /* X_l = LL(Y_l) */
        for (int q = 0; q < 4; ++q) {
            const double s = sl[(l - 1) * 4 + q];
            const double* wk = wl + ((long)(l - 1) * 4 + q) * kk;
            const double* dz = dZ + offs[l] + (long)q * n;
            const double* cq = C + offs[l] + (long)q * n;
            double acc = 0.0;
            for (int e = 0; e < n; ++e) acc += dz[e] * cq[e];
            gsl[(l - 1) * 4 + q] = acc;                    /* d s_l */
            for (int e = 0; e < n; ++e) dC[e] = s * dz[e];
            double* gw = gwl + ((long)(l - 1) * 4 + q) * kk;
            for (int t = 0; t < kk; ++t) gw[t] = 0.0;
            corr_same_kernel_grad(hs[l], ws[l], k, dC, Y + offs[l] + (long)q * n, gw);
            corr_same_adjoint(hs[l], ws[l], k, dC, wk, tmp);
            for (int e = 0; e < n; ++e) dYl[(long)q * n + e] += tmp[e];
        }
        /* adjoint of Y_l = A(pad(X_{l-1})) is crop(A^T(dY_l)) */
        oracle_haar_synthesis(hs[l - 1], ws[l - 1], dYl, dcar);
    }
    if (L >= 1)
        for (size_t e = 0; e < HW; ++e) dx[e] += dcar[e];

    free(Y); free(C); free(dZ); free(carrier); free(dR); free(dYl); free(dC); free(tmp);
    free(dcar); free(offs);
    return 0;
}

/* Gather the level parameters of channel c from the [L][4C][k*k] / [L][4C]
 * layouts into [L][4][k*k] / [L][4]. */
static void channel_params(int C, int k, int L, int c, const double* level_w, const double* level_scale,
                           double* wl, double* sl)
{
    const int kk = k * k;
    for (int l = 0; l < L; ++l)
        for (int q = 0; q < 4; ++q) {
            memcpy(wl + ((long)l * 4 + q) * kk, level_w + ((long)l * 4 * C + 4L * c + q) * kk,
                   sizeof(double) * (size_t)kk);
            sl[l * 4 + q] = level_scale[(long)l * 4 * C + 4L * c + q];
        }
}

static int check_desc(int B, int C, int H, int W, int k, int L)
{
    if (B < 1 || C < 1 || H < 1 || W < 1) return 1;
    if (k < 1 || (k % 2) == 0) return 1;
    if (L < 0 || L > 60) return 1;
    return 0;
}

/* Whole-tensor forward. OpenMP over the B*C independent planes. */
int oracle_forward(int B, int C, int H, int W, int k, int L, const double* x, const double* base_w,
                   const double* base_scale, const double* base_bias, const double* level_w,
                   const double* level_scale, double* y)
{
    if (check_desc(B, C, H, W, k, L)) return 1;
    const int kk = k * k;
    const long HW = (long)H * W;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (long pl = 0; pl < (long)B * C; ++pl) {
        const int c = (int)(pl % C);
        double* wl = (double*)malloc(sizeof(double) * ((size_t)L * 4 * kk + 1));
        double* sl = (double*)malloc(sizeof(double) * ((size_t)L * 4 + 1));
        if (!wl || !sl) {
            err |= 2;
        } else {
            channel_params(C, k, L, c, level_w, level_scale, wl, sl);
            err |= oracle_plane_forward(H, W, k, L, x + pl * HW, base_w + (long)c * kk, base_scale[c], wl, sl,
                                        base_bias ? base_bias[c] : 0.0, y + pl * HW, NULL);
        }
        free(wl);
        free(sl);
    }
    return err;
}

/* Whole-tensor backward. Planes run in parallel; the per-plane parameter
 * gradients are then summed over b = 0..B-1 in that order. */
int oracle_backward(int B, int C, int H, int W, int k, int L, const double* x, const double* dy,
                    const double* base_w, const double* base_scale, const double* base_bias,
                    const double* level_w, const double* level_scale, double* dx, double* d_base_w,
                    double* d_base_scale, double* d_base_bias, double* d_level_w, double* d_level_scale)
{
    if (check_desc(B, C, H, W, k, L)) return 1;
    const int kk = k * k;
    const long HW = (long)H * W;
    const long P = (long)B * C;
    const long per = kk + 2 + (long)L * 4 * kk + (long)L * 4; /* per-plane gradient record */
    double* part = (double*)malloc(sizeof(double) * (size_t)(P * per));
    if (!part) return 2;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (long pl = 0; pl < P; ++pl) {
        const int c = (int)(pl % C);
        double* wl = (double*)malloc(sizeof(double) * ((size_t)L * 4 * kk + 1));
        double* sl = (double*)malloc(sizeof(double) * ((size_t)L * 4 + 1));
        if (!wl || !sl) {
            err |= 2;
        } else {
            channel_params(C, k, L, c, level_w, level_scale, wl, sl);
            double* rec = part + pl * per;
            err |= oracle_plane_backward(H, W, k, L, x + pl * HW, dy + pl * HW, base_w + (long)c * kk,
                                         base_scale[c], wl, sl, base_bias ? base_bias[c] : 0.0, dx + pl * HW,
                                         rec, rec + kk, rec + kk + 1, rec + kk + 2,
                                         rec + kk + 2 + (long)L * 4 * kk);
        }
        free(wl);
        free(sl);
    }
    if (err) {
        free(part);
        return err;
    }
    memset(d_base_w, 0, sizeof(double) * (size_t)C * kk);
    memset(d_base_scale, 0, sizeof(double) * (size_t)C);
    memset(d_base_bias, 0, sizeof(double) * (size_t)C);
    if (L > 0) {
        memset(d_level_w, 0, sizeof(double) * (size_t)L * 4 * C * kk);
        memset(d_level_scale, 0, sizeof(double) * (size_t)L * 4 * C);
    }
    for (int b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c) {
            const double* rec = part + ((long)b * C + c) * per;
            /* dW0 = s0 * dW~0 happens inside the plane adjoint (dC = s0*dy) */
            for (int t = 0; t < kk; ++t) d_base_w[(long)c * kk + t] += rec[t];
            d_base_scale[c] += rec[kk];
            d_base_bias[c] += rec[kk + 1];
            for (int l = 0; l < L; ++l)
                for (int q = 0; q < 4; ++q) {
                    const double* gw = rec + kk + 2 + ((long)l * 4 + q) * kk;
                    double* dst = d_level_w + ((long)l * 4 * C + 4L * c + q) * kk;
                    for (int t = 0; t < kk; ++t) dst[t] += gw[t];
                    d_level_scale[(long)l * 4 * C + 4L * c + q] += rec[kk + 2 + (long)L * 4 * kk + l * 4 + q];
                }
        }
    free(part);
    return 0;
}

/* Number of OpenMP threads the oracle will use (for reporting). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Set the number of OpenMP threads used by the whole-tensor entry points
 * (benchmark reporting of single-thread timings). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
