/*
 * PyraMiD-LSTM CPU oracle: plain, slow, fp64 nested loops.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
 * its Python binding) may include, link, load or call this file; only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg use it.  It shares
 * no code, header, table or helper with the GPU implementation.
 *
 * What it computes (Stollenga, Byeon, Liwicki, Schmidhuber, "Parallel
 * Multi-Dimensional LSTM ...", arXiv 1506.07452):
 *   - Section 2.3, direction set: six C-LSTMs, one per direction
 *     z+, z-, y+, y-, x+, x- (paper axes x,y,z = volume W,H,D), each a full LSTM
 *     RNN whose time index is bound to the sweep axis.
 *   - Section 2.3, Eq. (7)-(12): gate pre-activations are a 2D in-plane
 *     convolution of the current input plane plus a 2D in-plane convolution of
 *     the previous plane's hidden state plus a per-gate bias shared by all
 *     positions; sigmoid gates i, f, o, tanh cell input, cell and hidden update.
 *     The first plane of a sweep has no predecessor, so its recurrent term and
 *     its c_{-1} f term are absent (read here as h_{-1} = c_{-1} = 0).
 *   - Section 2.3, Eq. (13): the layer output is the sum of the six h^d.
 *   - Section 2 (Method), sigma(x) = 1 / (1 + e^{-x}).
 *   - Section 2.3, footnote on convolutions: 2D convolution, stride 1.
 *   - Section 2.3 ("Fully-Connected Layer") and Fig. 3: a per-voxel fully
 *     connected layer squashed by tanh; a softmax after the last one.
 *   - Section 3 ("Training"): the network is trained by gradient descent, which
 *     needs the gradient of all of the above (back-propagation through the
 *     sweeps); the paper does not write it out, it is the chain rule applied to
 *     Eq. (7)-(13).
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - zero "same" padding (pad K/2) for both convolutions; the volumes keep their
 *     size W x H x D (Section 2.3).
 *   - "*" is cross-correlation with weight layout [out][in][ka][kb], ka over the
 *     first and kb over the second in-plane axis, taken in (D, H, W) order:
 *     z+- -> (H, W), y+- -> (D, W), x+- -> (D, H); the same orientation for the
 *     + and - direction of an axis.
 *   - 0-based time: plane index z = t for a + direction, z = T-1-t for a -.
 *   - one bias vector per gate per direction; gate packing (i, f, g=c~, o).
 *   - six independent parameter sets (superscript d on every theta).
 *
 * Layouts (all row-major, fp64):
 *   x   [N][D][H][W][C]          wx [6][4O][C][K][K]
 *   h   [N][D][H][W][O]          wh [6][4O][O][K][K]      b [6][4O]
 *   hd  [6][N][D][H][W][O]       (optional per-direction outputs h^d)
 *   gates [6][N][D][H][W][4O]    (optional post-activation i,f,g,o)
 *   cell  [6][N][D][H][W][O]     (optional c^d)
 *
 * Parity pinning: see tests/test_oracle_pins.py (textbook LSTM reduction,
 * library-convolution reduction, zero-direction identity, mirror symmetry,
 * dependency cone, brute-force recursion, closed form at 1x1x1, finite
 * differences and autograd of the gradients).
 */
#include <math.h>
#include <omp.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

#define NDIR 6

/* Sweep axis of direction d (0 = D/z, 1 = H/y, 2 = W/x) and its sign. */
static int dir_axis(int d) { return d / 2; }
static int dir_sign(int d) { return (d % 2 == 0) ? +1 : -1; }

/* Map (sweep position s, in-plane p, in-plane q) of direction d to (z, y, x).
 * In-plane axes are the two remaining axes in (D, H, W) order. */
static void plane_to_vol(int d, int s, int p, int q, int *z, int *y, int *x)
{
    switch (dir_axis(d)) {
    case 0: *z = s; *y = p; *x = q; break;
    case 1: *z = p; *y = s; *x = q; break;
    default: *z = p; *y = q; *x = s; break;
    }
}

static void plane_dims(int d, int D, int H, int W, int *T, int *P, int *Q)
{
    switch (dir_axis(d)) {
    case 0: *T = D; *P = H; *Q = W; break;
    case 1: *T = H; *P = D; *Q = W; break;
    default: *T = W; *P = D; *Q = H; break;
    }
}

static size_t vidx(int D, int H, int W, int n, int z, int y, int x)
{
    return (((size_t)n * D + z) * H + y) * W + x;
}

/* Number of OpenMP threads the oracle's parallel loops use. */
int oracle_threads(void) { return omp_get_max_threads(); }

/* Sets that number for later calls from the calling thread (n >= 1). */
void oracle_set_threads(int n) { if (n >= 1) omp_set_num_threads(n); }

static double sigmoid(double a) { return 1.0 / (1.0 + exp(-a)); }

/* One direction, one batch element: forward sweep of Eq. (7)-(12).
 * Writes h^d, the gates and c^d of this direction in volume layout
 * (hdir [V][O], gdir [V][4O], cdir [V][O], V = D*H*W of one batch element). */
static void sweep_forward(int d, int n, int D, int H, int W, int C, int O, int K,
                          const double *x, const double *wx, const double *wh,
                          const double *b, double *hdir, double *gdir, double *cdir)
{
    int T, P, Q;
    plane_dims(d, D, H, W, &T, &P, &Q);
    const int r = K / 2;
    const int G = 4 * O;
    const double *wxd = wx + (size_t)d * G * C * K * K;
    const double *whd = wh + (size_t)d * G * O * K * K;
    const double *bd = b + (size_t)d * G;

    for (int t = 0; t < T; ++t) {
        const int s = (dir_sign(d) > 0) ? t : T - 1 - t;      /* current plane */
        const int sp = (dir_sign(d) > 0) ? s - 1 : s + 1;     /* previous plane */
#pragma omp parallel for schedule(static)
        for (int p = 0; p < P; ++p) {
            double *A = (double *)malloc(sizeof(double) * G);
            for (int q = 0; q < Q; ++q) {
                for (int gn = 0; gn < G; ++gn) {
                    double acc = bd[gn];
                    /* input convolution over the current plane */
                    for (int ka = 0; ka < K; ++ka)
                        for (int kb = 0; kb < K; ++kb) {
                            const int pp = p + ka - r, qq = q + kb - r;
                            if (pp < 0 || pp >= P || qq < 0 || qq >= Q) continue;
                            int z, y, xx;
                            plane_to_vol(d, s, pp, qq, &z, &y, &xx);
                            const double *xv = x + vidx(D, H, W, n, z, y, xx) * C;
                            for (int c = 0; c < C; ++c)
                                acc += xv[c] * wxd[(((size_t)gn * C + c) * K + ka) * K + kb];
                        }
                    /* recurrent convolution over the previous plane's h^d */
                    if (t > 0) {
                        for (int ka = 0; ka < K; ++ka)
                            for (int kb = 0; kb < K; ++kb) {
                                const int pp = p + ka - r, qq = q + kb - r;
                                if (pp < 0 || pp >= P || qq < 0 || qq >= Q) continue;
                                int z, y, xx;
                                plane_to_vol(d, sp, pp, qq, &z, &y, &xx);
                                const double *hv = hdir + vidx(D, H, W, 0, z, y, xx) * O;
                                for (int j = 0; j < O; ++j)
                                    acc += hv[j] * whd[(((size_t)gn * O + j) * K + ka) * K + kb];
                            }
                    }
                    A[gn] = acc;
                }
                int z, y, xx;
                plane_to_vol(d, s, p, q, &z, &y, &xx);
                const size_t v = vidx(D, H, W, 0, z, y, xx);
                const double *cprev = NULL;
                if (t > 0) {
                    int zp, yp, xp;
                    plane_to_vol(d, sp, p, q, &zp, &yp, &xp);
                    cprev = cdir + vidx(D, H, W, 0, zp, yp, xp) * O;
                }
                for (int o = 0; o < O; ++o) {
                    const double gi = sigmoid(A[0 * O + o]);
                    const double gf = sigmoid(A[1 * O + o]);
                    const double gg = tanh(A[2 * O + o]);
                    const double go = sigmoid(A[3 * O + o]);
                    const double c = gg * gi + (cprev ? cprev[o] * gf : 0.0);
                    cdir[v * O + o] = c;
                    hdir[v * O + o] = go * tanh(c);
                    gdir[v * G + 0 * O + o] = gi;
                    gdir[v * G + 1 * O + o] = gf;
                    gdir[v * G + 2 * O + o] = gg;
                    gdir[v * G + 3 * O + o] = go;
                }
            }
            free(A);
        }
    }
}

/* Layer forward: Eq. (7)-(13).  Returns 0, or -1 on bad arguments / no memory. */
int oracle_forward(int N, int D, int H, int W, int C, int O, int K,
                   const double *x, const double *wx, const double *wh, const double *b,
                   double *h, double *hd, double *gates, double *cell)
{
    if (N < 1 || D < 1 || H < 1 || W < 1 || C < 1 || O < 1 || K < 1 || K % 2 == 0)
        return -1;
    const size_t V = (size_t)D * H * W;
    double *hdir = (double *)malloc(sizeof(double) * V * O);
    double *cdir = (double *)malloc(sizeof(double) * V * O);
    double *gdir = (double *)malloc(sizeof(double) * V * 4 * O);
    if (!hdir || !cdir || !gdir) { free(hdir); free(cdir); free(gdir); return -1; }
    memset(h, 0, sizeof(double) * N * V * O);
    /* Directions outermost so that Eq. (13) sums in the fixed order d = 0..5. */
    for (int d = 0; d < NDIR; ++d)
        for (int n = 0; n < N; ++n) {
            sweep_forward(d, n, D, H, W, C, O, K, x, wx, wh, b, hdir, gdir, cdir);
            double *hn = h + (size_t)n * V * O;
            for (size_t i = 0; i < V * O; ++i) hn[i] += hdir[i];
            const size_t off = ((size_t)d * N + n) * V;
            if (hd) memcpy(hd + off * O, hdir, sizeof(double) * V * O);
            if (cell) memcpy(cell + off * O, cdir, sizeof(double) * V * O);
            if (gates) memcpy(gates + off * 4 * O, gdir, sizeof(double) * V * 4 * O);
        }
    free(hdir); free(cdir); free(gdir);
    return 0;
}

/* Layer backward: the chain rule through Eq. (7)-(13), back-propagation through
 * each sweep in reverse plane order.  dh = dL/dh of the summed output; since
 * h = sum_d h^d, every direction receives the same dL/dh^d = dh.
 *
 * Per direction, in reverse t (gc = dL/dc, gh = dL/dh^d of the plane):
 *   gh_t  = dh[plane t] + recurrent term from A_{t+1} (transposed convolution)
 *   gc_t  = gh_t * o_t * (1 - tanh^2 c_t) + gc_{t+1} * f_{t+1}
 *   dA_o  = gh_t * tanh c_t * o (1 - o)
 *   dA_i  = gc_t * g * i (1 - i)
 *   dA_g  = gc_t * i * (1 - g^2)
 *   dA_f  = gc_t * c_{t-1} * f (1 - f)            (c_{-1} = 0)
 * and the parameter / input gradients collect dA against the convolution inputs.
 * dx, dwx, dwh, db are overwritten; the parameter gradients are summed over
 * the batch.  dx may be NULL. */
int oracle_backward(int N, int D, int H, int W, int C, int O, int K,
                    const double *x, const double *wx, const double *wh, const double *b,
                    const double *dh, double *dx, double *dwx, double *dwh, double *db)
{
    if (N < 1 || D < 1 || H < 1 || W < 1 || C < 1 || O < 1 || K < 1 || K % 2 == 0)
        return -1;
    const size_t V = (size_t)D * H * W;
    const int G = 4 * O;
    const int r = K / 2;
    double *hdir = (double *)malloc(sizeof(double) * V * O);
    double *cdir = (double *)malloc(sizeof(double) * V * O);
    double *gdir = (double *)malloc(sizeof(double) * V * G);
    double *dA = (double *)malloc(sizeof(double) * V * G);   /* dA at every voxel */
    double *gc = (double *)malloc(sizeof(double) * V * O);   /* dL/dc at every voxel */
    if (!hdir || !cdir || !gdir || !dA || !gc) {
        free(hdir); free(cdir); free(gdir); free(dA); free(gc);
        return -1;
    }
    if (dx) memset(dx, 0, sizeof(double) * N * V * C);
    memset(dwx, 0, sizeof(double) * NDIR * G * C * K * K);
    memset(dwh, 0, sizeof(double) * NDIR * G * O * K * K);
    memset(db, 0, sizeof(double) * NDIR * G);

    for (int d = 0; d < NDIR; ++d) {
        int T, P, Q;
        plane_dims(d, D, H, W, &T, &P, &Q);
        const double *wxd = wx + (size_t)d * G * C * K * K;
        const double *whd = wh + (size_t)d * G * O * K * K;
        double *dwxd = dwx + (size_t)d * G * C * K * K;
        double *dwhd = dwh + (size_t)d * G * O * K * K;
        double *dbd = db + (size_t)d * G;
        for (int n = 0; n < N; ++n) {
            sweep_forward(d, n, D, H, W, C, O, K, x, wx, wh, b, hdir, gdir, cdir);
            const double *dhn = dh + (size_t)n * V * O;
            for (int t = T - 1; t >= 0; --t) {
                const int s = (dir_sign(d) > 0) ? t : T - 1 - t;
                const int sn = (dir_sign(d) > 0) ? s + 1 : s - 1;   /* plane t+1 */
                const int sp = (dir_sign(d) > 0) ? s - 1 : s + 1;   /* plane t-1 */
#pragma omp parallel for schedule(static)
                for (int p = 0; p < P; ++p)
                    for (int q = 0; q < Q; ++q) {
                        int z, y, xx;
                        plane_to_vol(d, s, p, q, &z, &y, &xx);
                        const size_t v = vidx(D, H, W, 0, z, y, xx);
                        size_t vn = 0, vp = 0;
                        if (t + 1 < T) {
                            int a, bb, cc;
                            plane_to_vol(d, sn, p, q, &a, &bb, &cc);
                            vn = vidx(D, H, W, 0, a, bb, cc);
                        }
                        if (t > 0) {
                            int a, bb, cc;
                            plane_to_vol(d, sp, p, q, &a, &bb, &cc);
                            vp = vidx(D, H, W, 0, a, bb, cc);
                        }
                        for (int j = 0; j < O; ++j) {
                            double gh = dhn[v * O + j];
                            if (t + 1 < T) {
                                /* h_t[p][q][j] fed A_{t+1}[p'][q'] with p' = p - (ka - r). */
                                for (int ka = 0; ka < K; ++ka)
                                    for (int kb = 0; kb < K; ++kb) {
                                        const int pp = p - (ka - r), qq = q - (kb - r);
                                        if (pp < 0 || pp >= P || qq < 0 || qq >= Q) continue;
                                        int a, bb, cc;
                                        plane_to_vol(d, sn, pp, qq, &a, &bb, &cc);
                                        const double *dAn = dA + vidx(D, H, W, 0, a, bb, cc) * G;
                                        for (int gn = 0; gn < G; ++gn)
                                            gh += dAn[gn] * whd[(((size_t)gn * O + j) * K + ka) * K + kb];
                                    }
                            }
                            const double gi = gdir[v * G + 0 * O + j];
                            const double gf = gdir[v * G + 1 * O + j];
                            const double gg = gdir[v * G + 2 * O + j];
                            const double go = gdir[v * G + 3 * O + j];
                            const double c = cdir[v * O + j];
                            const double tc = tanh(c);
                            double gcv = gh * go * (1.0 - tc * tc);
                            if (t + 1 < T) gcv += gc[vn * O + j] * gdir[vn * G + 1 * O + j];
                            gc[v * O + j] = gcv;
                            const double cprev = (t > 0) ? cdir[vp * O + j] : 0.0;
                            dA[v * G + 0 * O + j] = gcv * gg * gi * (1.0 - gi);
                            dA[v * G + 1 * O + j] = gcv * cprev * gf * (1.0 - gf);
                            dA[v * G + 2 * O + j] = gcv * gi * (1.0 - gg * gg);
                            dA[v * G + 3 * O + j] = gh * tc * go * (1.0 - go);
                        }
                    }
            }
            /* Parameter and input gradients: every plane's dA against the
             * inputs of its two convolutions (Eq. (7)-(9), (11)). */
#pragma omp parallel for schedule(static)
            for (int gn = 0; gn < G; ++gn) {
                for (int t = 0; t < T; ++t) {
                    const int s = (dir_sign(d) > 0) ? t : T - 1 - t;
                    const int sp = (dir_sign(d) > 0) ? s - 1 : s + 1;
                    for (int p = 0; p < P; ++p)
                        for (int q = 0; q < Q; ++q) {
                            int z, y, xx;
                            plane_to_vol(d, s, p, q, &z, &y, &xx);
                            const double g = dA[vidx(D, H, W, 0, z, y, xx) * G + gn];
                            dbd[gn] += g;
                            for (int ka = 0; ka < K; ++ka)
                                for (int kb = 0; kb < K; ++kb) {
                                    const int pp = p + ka - r, qq = q + kb - r;
                                    if (pp < 0 || pp >= P || qq < 0 || qq >= Q) continue;
                                    int a, bb, cc;
                                    plane_to_vol(d, s, pp, qq, &a, &bb, &cc);
                                    const double *xv = x + vidx(D, H, W, n, a, bb, cc) * C;
                                    for (int ci = 0; ci < C; ++ci)
                                        dwxd[(((size_t)gn * C + ci) * K + ka) * K + kb] += g * xv[ci];
                                    if (t > 0) {
                                        plane_to_vol(d, sp, pp, qq, &a, &bb, &cc);
                                        const double *hv = hdir + vidx(D, H, W, 0, a, bb, cc) * O;
                                        for (int j = 0; j < O; ++j)
                                            dwhd[(((size_t)gn * O + j) * K + ka) * K + kb] += g * hv[j];
                                    }
                                }
                        }
                }
            }
            if (dx) {
                /* dx[voxel (s, p', q')][c] += dA_t[p][q][gn] * wx[gn][c][ka][kb]
                 * for every (p, q, tap) with p' = p + ka - r, q' = q + kb - r. */
                double *dxn = dx + (size_t)n * V * C;
                for (int t = 0; t < T; ++t) {
                    const int s = (dir_sign(d) > 0) ? t : T - 1 - t;
#pragma omp parallel for schedule(static)
                    for (int pp = 0; pp < P; ++pp)
                        for (int qq = 0; qq < Q; ++qq) {
                            int z, y, xx;
                            plane_to_vol(d, s, pp, qq, &z, &y, &xx);
                            double *dxv = dxn + vidx(D, H, W, 0, z, y, xx) * C;
                            for (int ka = 0; ka < K; ++ka)
                                for (int kb = 0; kb < K; ++kb) {
                                    const int p = pp - (ka - r), q = qq - (kb - r);
                                    if (p < 0 || p >= P || q < 0 || q >= Q) continue;
                                    int a, bb, cc;
                                    plane_to_vol(d, s, p, q, &a, &bb, &cc);
                                    const double *dAv = dA + vidx(D, H, W, 0, a, bb, cc) * G;
                                    for (int gn = 0; gn < G; ++gn)
                                        for (int ci = 0; ci < C; ++ci)
                                            dxv[ci] += dAv[gn] * wxd[(((size_t)gn * C + ci) * K + ka) * K + kb];
                                }
                        }
                }
            }
        }
    }
    free(hdir); free(cdir); free(gdir); free(dA); free(gc);
    return 0;
}

/* Per-voxel fully connected layer squashed by tanh (Section 2.3,
 * "Fully-Connected Layer"):  y[m][o] = tanh(sum_i w[o][i] * x[m][i] + b[o]).
 * x [M][Cin], w [Cout][Cin], b [Cout], y [M][Cout]. */
void oracle_fc_tanh_forward(long M, int Cin, int Cout, const double *x,
                            const double *w, const double *b, double *y)
{
#pragma omp parallel for schedule(static)
    for (long m = 0; m < M; ++m)
        for (int o = 0; o < Cout; ++o) {
            double acc = b[o];
            for (int i = 0; i < Cin; ++i) acc += w[(size_t)o * Cin + i] * x[(size_t)m * Cin + i];
            y[(size_t)m * Cout + o] = tanh(acc);
        }
}

/* Gradient of oracle_fc_tanh_forward given its output y and dL/dy.
 * dx (nullable) [M][Cin], dw [Cout][Cin], db [Cout]; all overwritten. */
void oracle_fc_tanh_backward(long M, int Cin, int Cout, const double *x,
                             const double *w, const double *y, const double *dy,
                             double *dx, double *dw, double *db)
{
    memset(dw, 0, sizeof(double) * Cout * Cin);
    memset(db, 0, sizeof(double) * Cout);
#pragma omp parallel for schedule(static)
    for (int o = 0; o < Cout; ++o)
        for (long m = 0; m < M; ++m) {
            const double yv = y[(size_t)m * Cout + o];
            const double dz = dy[(size_t)m * Cout + o] * (1.0 - yv * yv);
            db[o] += dz;
            for (int i = 0; i < Cin; ++i) dw[(size_t)o * Cin + i] += dz * x[(size_t)m * Cin + i];
        }
    if (dx) {
#pragma omp parallel for schedule(static)
        for (long m = 0; m < M; ++m)
            for (int i = 0; i < Cin; ++i) {
                double acc = 0.0;
                for (int o = 0; o < Cout; ++o) {
                    const double yv = y[(size_t)m * Cout + o];
                    acc += dy[(size_t)m * Cout + o] * (1.0 - yv * yv) * w[(size_t)o * Cin + i];
                }
                dx[(size_t)m * Cin + i] = acc;
            }
    }
}

/* Last fully connected layer followed by a per-voxel softmax (Fig. 3 caption,
 * Section 2.3): logits[m][k] = sum_i w[k][i] x[m][i] + b[k], p = softmax.
 * With labels (nullable): returns the mean cross-entropy over the M voxels and,
 * when dx/dw/db are given, its gradient (dlogits = (p - onehot) / M). */
double oracle_softmax_ce(long M, int Cin, int Kc, const double *x, const double *w,
                         const double *b, const int *labels, double *p,
                         double *dx, double *dw, double *db)
{
    double loss = 0.0;
#pragma omp parallel for schedule(static) reduction(+ : loss)
    for (long m = 0; m < M; ++m) {
        double *pm = p + (size_t)m * Kc;
        double mx = -INFINITY;
        for (int k = 0; k < Kc; ++k) {
            double acc = b[k];
            for (int i = 0; i < Cin; ++i) acc += w[(size_t)k * Cin + i] * x[(size_t)m * Cin + i];
            pm[k] = acc;
            if (acc > mx) mx = acc;
        }
        double z = 0.0;
        for (int k = 0; k < Kc; ++k) z += exp(pm[k] - mx);
        for (int k = 0; k < Kc; ++k) pm[k] = exp(pm[k] - mx) / z;
        if (labels) loss += -log(pm[labels[m]]);
    }
    if (!labels) return 0.0;
    loss /= (double)M;
    if (dw && db) {
        memset(dw, 0, sizeof(double) * Kc * Cin);
        memset(db, 0, sizeof(double) * Kc);
        for (int k = 0; k < Kc; ++k)
            for (long m = 0; m < M; ++m) {
                const double g = (p[(size_t)m * Kc + k] - (labels[m] == k ? 1.0 : 0.0)) / (double)M;
                db[k] += g;
                for (int i = 0; i < Cin; ++i) dw[(size_t)k * Cin + i] += g * x[(size_t)m * Cin + i];
            }
    }
    if (dx) {
#pragma omp parallel for schedule(static)
        for (long m = 0; m < M; ++m)
            for (int i = 0; i < Cin; ++i) {
                double acc = 0.0;
                for (int k = 0; k < Kc; ++k) {
                    const double g = (p[(size_t)m * Kc + k] - (labels[m] == k ? 1.0 : 0.0)) / (double)M;
                    acc += g * w[(size_t)k * Cin + i];
                }
                dx[(size_t)m * Cin + i] = acc;
            }
    }
    return loss;
}
