/*
 * PVConv CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct fp64 implementation of what one
 * Point-Voxel Convolution layer computes (Liu, Tang, Lin, Han, "Point-Voxel CNN
 * for Efficient 3D Deep Learning", NeurIPS 2019, Section 4). Only the test
 * suite, the package smoke check and the benchmark's CPU-baseline leg may load
 * this library. It shares no code, header or table with the GPU library, and
 * the GPU library never calls it.
 *
 * Every step follows the paper's definition directly:
 *   ref_normalize      Section 4.1 "Normalization"
 *   ref_voxel_ids      Section 4.1 "Voxelization", the indicator of Eq. 2
 *   ref_voxelize       Section 4.1 "Voxelization", Eq. 2
 *   ref_conv3d(_at)    Section 4.1 "Feature Aggregation" with the fixed-offset
 *                      3x3x3 kernel of Section 3 (Eq. 1, "Dynamic Kernel
 *                      Computation": offsets in {0, +-1} per axis)
 *   ref_batchnorm      Section 4.1 "Feature Aggregation" (batch normalisation,
 *                      inference form with running statistics)
 *   ref_leaky_relu     Section 4.1 "Feature Aggregation" (leaky rectifier)
 *   ref_relu           Section 4.2 (point-branch MLP nonlinearity)
 *   ref_devoxelize     Section 4.1 "Devoxelization" (trilinear interpolation)
 *   ref_devoxelize_nearest  Section 4.1 "Devoxelization", the nearest-neighbour
 *                      mapping the section sets against trilinear (the
 *                      devoxelisation row of the ablation table)
 *   ref_linear         Section 4.2 "Point-Based Feature Transformation"
 *   ref_*_backward     gradients of the above with respect to their inputs
 *                      (and of the convolution with respect to its weights):
 *                      the layer is differentiable end to end (Section 4.1
 *                      "Devoxelization" relies on it for trilinear vs
 *                      nearest); each is the adjoint of the linear map the
 *                      forward step applies
 *   ref_maxpool        Section 5.1 "Models" (PointNet backbone global feature)
 *   ref_fps, ref_ball_query, ref_group, ref_three_nn, ref_three_interpolate
 *                      the PointNet++ primitives that PVCNN++ keeps around its
 *                      PVConv layers (Section 5.2 "Models": PointNet++
 *                      extended with PVConv), as PointNet++ (Qi et al., 2017)
 *                      defines them: iterative farthest point sampling, ball
 *                      query grouping, and inverse-distance interpolation
 *                      over the three nearest neighbours
 * Fusion by addition (Section 4.3) and the composition of the steps live in
 * oracle/__init__.py.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *  - the "gravity center" is the arithmetic mean of the coordinates, summed in
 *    an order-free int64 fixed-point form so that voxel indices do not depend
 *    on summation order (see centroid_axis);
 *  - max ||p||_2 is taken after centring, per cloud; the unit-sphere points are
 *    then scaled by 1/2 and shifted by 1/2 into [0,1]^3;
 *  - a cloud whose points all coincide maps every point to (1/2, 1/2, 1/2);
 *  - voxel indices use floor as Eq. 2 writes it and are clamped to [0, R-1];
 *  - voxel (u,v,w) has its centre at ((u+1/2)/R, (v+1/2)/R, (w+1/2)/R) for the
 *    trilinear interpolation, with border cells replicated;
 *  - grid layout [B][R][R][R][C] with x -> u (slowest), z -> w, C innermost.
 *
 * All arithmetic is IEEE fp64 with round-to-nearest-even and no contraction
 * (built with -ffp-contract=off), except where a floating-point comparison
 * decides an index (the farthest point, ball membership, the three nearest
 * neighbours): there the squared distance is computed in fp32 as
 * fma(dz, dz, fma(dy, dy, dx*dx)) with dx = x_j - x_c (fmaf rounds once), the
 * precision and order the GPU kernels use, so that both sides make the same
 * choices.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define PV_ORACLE_OK 0
#define PV_ORACLE_EINVAL (-1)

/* ------------------------------------------------------------------------- */
/* Section 4.1 "Normalization"                                               */
/* ------------------------------------------------------------------------- */

/* Smallest L with 2^L >= n. */
static int ceil_log2(int64_t n) {
    int L = 0;
    while (((int64_t)1 << L) < n) L++;
    return L;
}

/* Gravity centre along one axis: the mean of x_{k,a} over the cloud.
 * The sum is taken as integers at the fixed-point scale 2^S, chosen so that no
 * partial sum can overflow int64 (|x| < 2^e and N <= 2^L give |sum| < 2^62).
 * Integer addition is exact, so the result does not depend on the order in
 * which the points are added. */
static double centroid_axis(const float* xyz, int64_t N, int axis) {
    double A = 0.0;
    for (int64_t k = 0; k < N; k++) {
        double a = fabs((double)xyz[3 * k + axis]);
        if (a > A) A = a;
    }
    if (A == 0.0) return 0.0;
    int e;
    frexp(A, &e); /* A = f * 2^e, f in [1/2, 1) */
    int S = 62 - ceil_log2(N) - e;
    int64_t q = 0;
    for (int64_t k = 0; k < N; k++) q += llrint(ldexp((double)xyz[3 * k + axis], S));
    return ldexp((double)q / (double)N, -S);
}

/* coords [B][N][3] fp32 -> centroid [B][3], radius [B] (max ||p - c||_2) and
 * pnorm [B][N][3] = ((p - c) / radius) * 1/2 + 1/2.
 * Returns PV_ORACLE_EINVAL on a non-finite coordinate. */
int ref_normalize(const float* coords, int64_t B, int64_t N, double* centroid,
                  double* radius, double* pnorm) {
    for (int64_t i = 0; i < B * N * 3; i++)
        if (!isfinite(coords[i])) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++) {
        const float* p = coords + b * N * 3;
        double c[3];
        for (int a = 0; a < 3; a++) c[a] = centroid_axis(p, N, a);
        /* largest squared distance to the centre */
        double M2 = 0.0;
        for (int64_t k = 0; k < N; k++) {
            double dx = (double)p[3 * k + 0] - c[0];
            double dy = (double)p[3 * k + 1] - c[1];
            double dz = (double)p[3 * k + 2] - c[2];
            double n2 = (dx * dx + dy * dy) + dz * dz;
            if (n2 > M2) M2 = n2;
        }
        double m = sqrt(M2);
        for (int a = 0; a < 3; a++) centroid[b * 3 + a] = c[a];
        radius[b] = m;
        for (int64_t k = 0; k < N; k++) {
            for (int a = 0; a < 3; a++) {
                double d = (double)p[3 * k + a] - c[a];
                double unit = (M2 == 0.0) ? 0.0 : d / m; /* into the unit sphere */
                pnorm[(b * N + k) * 3 + a] = unit * 0.5 + 0.5; /* into [0,1] */
            }
        }
    }
    return PV_ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Section 4.1 "Voxelization", Eq. 2                                         */
/* ------------------------------------------------------------------------- */

static int64_t voxel_coord(double x, int R) {
    double f = floor(x * (double)R);
    if (f < 0.0) return 0;
    if (f > (double)(R - 1)) return R - 1;
    return (int64_t)f;
}

/* pnorm [B][N][3] -> ids [B][N], id = (u*R + v)*R + w with
 * (u, v, w) = (floor(x*R), floor(y*R), floor(z*R)) clamped to [0, R-1]. */
int ref_voxel_ids(const double* pnorm, int64_t B, int64_t N, int R, int32_t* ids) {
    if (R < 1) return PV_ORACLE_EINVAL;
    for (int64_t i = 0; i < B * N; i++) {
        int64_t u = voxel_coord(pnorm[3 * i + 0], R);
        int64_t v = voxel_coord(pnorm[3 * i + 1], R);
        int64_t w = voxel_coord(pnorm[3 * i + 2], R);
        ids[i] = (int32_t)((u * R + v) * R + w);
    }
    return PV_ORACLE_OK;
}

/* V_{u,v,w,c} = (1 / N_{u,v,w}) * sum_k [id_k = (u,v,w)] f_{k,c}, and 0 for an
 * empty voxel. feats [B][N][C] -> grid [B][R^3][C], counts [B][R^3]. */
int ref_voxelize(const int32_t* ids, const double* feats, int64_t B, int64_t N, int64_t C,
                 int R, double* grid, int32_t* counts) {
    int64_t V = (int64_t)R * R * R;
    memset(grid, 0, sizeof(double) * (size_t)(B * V * C));
    memset(counts, 0, sizeof(int32_t) * (size_t)(B * V));
    for (int64_t b = 0; b < B; b++) {
        for (int64_t k = 0; k < N; k++) {
            int64_t id = ids[b * N + k];
            if (id < 0 || id >= V) return PV_ORACLE_EINVAL;
            counts[b * V + id] += 1;
            for (int64_t c = 0; c < C; c++)
                grid[(b * V + id) * C + c] += feats[(b * N + k) * C + c];
        }
        for (int64_t v = 0; v < V; v++) {
            int32_t n = counts[b * V + v];
            if (n == 0) continue;
            for (int64_t c = 0; c < C; c++) grid[(b * V + v) * C + c] /= (double)n;
        }
    }
    return PV_ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Section 4.1 "Feature Aggregation": 3x3x3 convolution, zero padding 1      */
/* ------------------------------------------------------------------------- */

/* One output voxel (b, u, v, w), all output channels:
 * y[o] = sum over offsets (du,dv,dw) in {-1,0,1}^3 and input channels i of
 *        W[o][du+1][dv+1][dw+1][i] * X[b][u+du][v+dv][w+dw][i],
 * with X = 0 outside the grid. The kernel is indexed by the neighbour's offset
 * from the centre, as Section 3 describes for volumetric convolution. */
static void conv_one_voxel(const double* x, int64_t b, int R, int64_t Cin, int64_t Cout,
                           const double* w, int64_t u, int64_t v, int64_t ww, double* y) {
    for (int64_t o = 0; o < Cout; o++) y[o] = 0.0;
    for (int du = -1; du <= 1; du++)
        for (int dv = -1; dv <= 1; dv++)
            for (int dw = -1; dw <= 1; dw++) {
                int64_t nu = u + du, nv = v + dv, nw = ww + dw;
                if (nu < 0 || nu >= R || nv < 0 || nv >= R || nw < 0 || nw >= R) continue;
                const double* xin = x + (((b * R + nu) * R + nv) * R + nw) * Cin;
                int tap = ((du + 1) * 3 + (dv + 1)) * 3 + (dw + 1);
                for (int64_t o = 0; o < Cout; o++) {
                    const double* wk = w + (o * 27 + tap) * Cin;
                    double s = 0.0;
                    for (int64_t i = 0; i < Cin; i++) s += wk[i] * xin[i];
                    y[o] += s;
                }
            }
}

/* x [B][R][R][R][Cin], w [Cout][3][3][3][Cin] -> y [B][R][R][R][Cout]. */
int ref_conv3d(const double* x, int64_t B, int R, int64_t Cin, int64_t Cout,
               const double* w, double* y) {
    if (B < 0 || R < 1 || Cin < 1 || Cout < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t b = 0; b < B; b++)
        for (int64_t u = 0; u < R; u++)
            for (int64_t v = 0; v < R; v++)
                for (int64_t ww = 0; ww < R; ww++)
                    conv_one_voxel(x, b, R, Cin, Cout, w, u, v, ww,
                                   y + (b * V + (u * R + v) * R + ww) * Cout);
    return PV_ORACLE_OK;
}

/* The same convolution evaluated only at the selected output voxels
 * sel[j] = b * R^3 + (u * R + v) * R + w; y is [n_sel][Cout]. */
int ref_conv3d_at(const double* x, int64_t B, int R, int64_t Cin, int64_t Cout,
                  const double* w, int64_t n_sel, const int64_t* sel, double* y) {
    int64_t V = (int64_t)R * R * R;
    for (int64_t j = 0; j < n_sel; j++)
        if (sel[j] < 0 || sel[j] >= B * V) return PV_ORACLE_EINVAL;
#pragma omp parallel for schedule(dynamic)
    for (int64_t j = 0; j < n_sel; j++) {
        int64_t b = sel[j] / V, r = sel[j] % V;
        int64_t u = r / ((int64_t)R * R), v = (r / R) % R, ww = r % R;
        conv_one_voxel(x, b, R, Cin, Cout, w, u, v, ww, y + j * Cout);
    }
    return PV_ORACLE_OK;
}

/* Batch normalisation with running statistics, applied in place to
 * y [M][C]: y = gamma * (y - mean) / sqrt(var + eps) + beta. */
int ref_batchnorm(double* y, int64_t M, int64_t C, const double* gamma, const double* beta,
                  const double* mean, const double* var, double eps) {
    for (int64_t c = 0; c < C; c++)
        if (!(var[c] + eps > 0.0)) return PV_ORACLE_EINVAL;
    for (int64_t m = 0; m < M; m++)
        for (int64_t c = 0; c < C; c++)
            y[m * C + c] = gamma[c] * (y[m * C + c] - mean[c]) / sqrt(var[c] + eps) + beta[c];
    return PV_ORACLE_OK;
}

/* Leaky rectifier, in place: y >= 0 ? y : slope * y. */
void ref_leaky_relu(double* y, int64_t n, double slope) {
    for (int64_t i = 0; i < n; i++)
        if (y[i] < 0.0) y[i] = slope * y[i];
}

/* Rectifier, in place. */
void ref_relu(double* y, int64_t n) {
    for (int64_t i = 0; i < n; i++)
        if (y[i] < 0.0) y[i] = 0.0;
}

/* ------------------------------------------------------------------------- */
/* Section 4.1 "Devoxelization": trilinear interpolation                     */
/* ------------------------------------------------------------------------- */

/* For one normalised coordinate: the two neighbouring cell indices along the
 * axis and their weights. Cell i's centre is at (i + 1/2) / R, so the
 * continuous cell coordinate is t = R * x - 1/2, clamped to [0, R-1]. */
static void trilinear_axis(double x, int R, int64_t* i0, int64_t* i1, double* w0,
                           double* w1) {
    double t = x * (double)R - 0.5;
    if (t < 0.0) t = 0.0;
    if (t > (double)(R - 1)) t = (double)(R - 1);
    double f = floor(t);
    *i0 = (int64_t)f;
    *i1 = (*i0 + 1 < R) ? *i0 + 1 : R - 1;
    *w1 = t - f;
    *w0 = 1.0 - *w1;
}

/* grid [B][R^3][C], pnorm [B][N][3] -> out [B][N][C]:
 * out_k = sum over the 8 surrounding cells of (wx * wy * wz) * V[cell]. */
int ref_devoxelize(const double* grid, int64_t B, int R, int64_t C, const double* pnorm,
                   int64_t N, double* out) {
    if (R < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
    for (int64_t b = 0; b < B; b++)
        for (int64_t k = 0; k < N; k++) {
            const double* p = pnorm + (b * N + k) * 3;
            int64_t iu[2], iv[2], iw[2];
            double wu[2], wv[2], ww[2];
            trilinear_axis(p[0], R, &iu[0], &iu[1], &wu[0], &wu[1]);
            trilinear_axis(p[1], R, &iv[0], &iv[1], &wv[0], &wv[1]);
            trilinear_axis(p[2], R, &iw[0], &iw[1], &ww[0], &ww[1]);
            double* o = out + (b * N + k) * C;
            for (int64_t c = 0; c < C; c++) o[c] = 0.0;
            for (int a = 0; a < 2; a++)
                for (int e = 0; e < 2; e++)
                    for (int g = 0; g < 2; g++) {
                        double wt = (wu[a] * wv[e]) * ww[g];
                        const double* cell = grid + (b * V + (iu[a] * R + iv[e]) * R + iw[g]) * C;
                        for (int64_t c = 0; c < C; c++) o[c] += wt * cell[c];
                    }
        }
    return PV_ORACLE_OK;
}

/* Nearest-neighbour devoxelisation: every point takes the features of the
 * voxel it falls into, i.e. the voxel of its Eq. 2 index, so that all points
 * of one voxel share one feature vector.
 * grid [B][R^3][C], ids [B][N] (voxel index within the cloud) -> out [B][N][C].
 * An index outside [0, R^3) is invalid input. */
int ref_devoxelize_nearest(const double* grid, int64_t B, int R, int64_t C,
                           const int32_t* ids, int64_t N, double* out) {
    if (R < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
    for (int64_t k = 0; k < B * N; k++)
        if (ids[k] < 0 || ids[k] >= V) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++)
        for (int64_t k = 0; k < N; k++) {
            const double* row = grid + (b * V + ids[b * N + k]) * C;
            double* o = out + (b * N + k) * C;
            for (int64_t c = 0; c < C; c++) o[c] = row[c];
        }
    return PV_ORACLE_OK;
}

/* Trilinear weights of the 8 cells around each point, as ref_devoxelize uses
 * them: cells [B*N][8] (linear voxel id within the cloud) and weights [B*N][8]. */
int ref_devoxelize_weights(const double* pnorm, int64_t n_points, int R, int64_t* cells,
                           double* weights) {
    if (R < 1) return PV_ORACLE_EINVAL;
    for (int64_t k = 0; k < n_points; k++) {
        const double* p = pnorm + k * 3;
        int64_t iu[2], iv[2], iw[2];
        double wu[2], wv[2], ww[2];
        trilinear_axis(p[0], R, &iu[0], &iu[1], &wu[0], &wu[1]);
        trilinear_axis(p[1], R, &iv[0], &iv[1], &wv[0], &wv[1]);
        trilinear_axis(p[2], R, &iw[0], &iw[1], &ww[0], &ww[1]);
        int j = 0;
        for (int a = 0; a < 2; a++)
            for (int e = 0; e < 2; e++)
                for (int g = 0; g < 2; g++, j++) {
                    cells[k * 8 + j] = (iu[a] * R + iv[e]) * R + iw[g];
                    weights[k * 8 + j] = (wu[a] * wv[e]) * ww[g];
                }
    }
    return PV_ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Section 4.2 "Point-Based Feature Transformation": shared per-point Linear  */
/* ------------------------------------------------------------------------- */

/* x [M][Cin], w [Cout][Cin], bias [Cout] or NULL -> y [M][Cout] = x w^T + bias. */
int ref_linear(const double* x, int64_t M, int64_t Cin, int64_t Cout, const double* w,
               const double* bias, double* y) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; m++)
        for (int64_t o = 0; o < Cout; o++) {
            double s = 0.0;
            for (int64_t i = 0; i < Cin; i++) s += x[m * Cin + i] * w[o * Cin + i];
            y[m * Cout + o] = bias ? s + bias[o] : s;
        }
    return PV_ORACLE_OK;
}

/* Per-cloud maximum over the points: x [B][N][C] -> out [B][C]. */
int ref_maxpool(const double* x, int64_t B, int64_t N, int64_t C, double* out) {
    if (N < 1) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++)
        for (int64_t c = 0; c < C; c++) {
            double m = x[(b * N) * C + c];
            for (int64_t k = 1; k < N; k++) {
                double v = x[(b * N + k) * C + c];
                if (v > m) m = v;
            }
            out[b * C + c] = m;
        }
    return PV_ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Backward pass: gradients of the steps above. Each forward step is linear  */
/* in the input it is differentiated by, so each gradient is the adjoint     */
/* (transpose) of that linear map, written out from its definition.          */
/* ------------------------------------------------------------------------- */

/* Eq. 2 averages the features of the points in each voxel, so
 * dL/df[b][k][c] = dL/dV[b][id_k][c] / N[b][id_k].
 * dgrid [B][R^3][C], ids [B][N], counts [B][R^3] -> dfeats [B][N][C]. */
int ref_voxelize_backward(const double* dgrid, const int32_t* ids, const int32_t* counts,
                          int64_t B, int64_t N, int64_t C, int R, double* dfeats) {
    if (R < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
    for (int64_t b = 0; b < B; b++)
        for (int64_t k = 0; k < N; k++) {
            int64_t id = ids[b * N + k];
            if (id < 0 || id >= V || counts[b * V + id] < 1) return PV_ORACLE_EINVAL;
            double n = (double)counts[b * V + id];
            for (int64_t c = 0; c < C; c++)
                dfeats[(b * N + k) * C + c] = dgrid[(b * V + id) * C + c] / n;
        }
    return PV_ORACLE_OK;
}

/* Trilinear devoxelisation: out_k = sum over its 8 cells of w(k, cell) V[cell],
 * so dL/dV[cell] = sum over the points k of w(k, cell) dL/dout_k.
 * dout [B][N][C], pnorm [B][N][3] -> dgrid [B][R^3][C]. */
int ref_devoxelize_backward(const double* dout, const double* pnorm, int64_t B, int64_t N,
                            int64_t C, int R, double* dgrid) {
    if (R < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
    memset(dgrid, 0, sizeof(double) * (size_t)(B * V * C));
    for (int64_t b = 0; b < B; b++)
        for (int64_t k = 0; k < N; k++) {
            const double* p = pnorm + (b * N + k) * 3;
            int64_t iu[2], iv[2], iw[2];
            double wu[2], wv[2], ww[2];
            trilinear_axis(p[0], R, &iu[0], &iu[1], &wu[0], &wu[1]);
            trilinear_axis(p[1], R, &iv[0], &iv[1], &wv[0], &wv[1]);
            trilinear_axis(p[2], R, &iw[0], &iw[1], &ww[0], &ww[1]);
            const double* g = dout + (b * N + k) * C;
            for (int a = 0; a < 2; a++)
                for (int e = 0; e < 2; e++)
                    for (int f = 0; f < 2; f++) {
                        double wt = (wu[a] * wv[e]) * ww[f];
                        double* cell = dgrid + (b * V + (iu[a] * R + iv[e]) * R + iw[f]) * C;
                        for (int64_t c = 0; c < C; c++) cell[c] += wt * g[c];
                    }
        }
    return PV_ORACLE_OK;
}

/* Nearest-neighbour devoxelisation copies V[id_k] to point k, so
 * dL/dV[cell] = sum of dL/dout_k over the points k with id_k = cell. */
int ref_devoxelize_nearest_backward(const double* dout, const int32_t* ids, int64_t B,
                                    int64_t N, int64_t C, int R, double* dgrid) {
    if (R < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
    for (int64_t k = 0; k < B * N; k++)
        if (ids[k] < 0 || ids[k] >= V) return PV_ORACLE_EINVAL;
    memset(dgrid, 0, sizeof(double) * (size_t)(B * V * C));
    for (int64_t b = 0; b < B; b++)
        for (int64_t k = 0; k < N; k++) {
            double* cell = dgrid + (b * V + ids[b * N + k]) * C;
            const double* g = dout + (b * N + k) * C;
            for (int64_t c = 0; c < C; c++) cell[c] += g[c];
        }
    return PV_ORACLE_OK;
}

/* Convolution, gradient with respect to its input. Output voxel p reads
 * input voxel p + d through W[o][d][i], so
 * dL/dx[b][q][i] = sum over offsets d and output channels o of
 *                  W[o][d][i] * dL/dy[b][q - d][o], for q - d inside the grid.
 * dy [B][R^3][Cout], w [Cout][27][Cin] -> dx [B][R^3][Cin]. */
int ref_conv3d_backward_data(const double* dy, int64_t B, int R, int64_t Cin, int64_t Cout,
                             const double* w, double* dx) {
    if (B < 0 || R < 1 || Cin < 1 || Cout < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t b = 0; b < B; b++)
        for (int64_t u = 0; u < R; u++)
            for (int64_t v = 0; v < R; v++)
                for (int64_t ww = 0; ww < R; ww++) {
                    double* out = dx + (b * V + (u * R + v) * R + ww) * Cin;
                    for (int64_t i = 0; i < Cin; i++) out[i] = 0.0;
                    for (int du = -1; du <= 1; du++)
                        for (int dv = -1; dv <= 1; dv++)
                            for (int dw = -1; dw <= 1; dw++) {
                                int64_t pu = u - du, pv = v - dv, pw = ww - dw;
                                if (pu < 0 || pu >= R || pv < 0 || pv >= R || pw < 0 || pw >= R)
                                    continue;
                                int tap = ((du + 1) * 3 + (dv + 1)) * 3 + (dw + 1);
                                const double* g = dy + (b * V + (pu * R + pv) * R + pw) * Cout;
                                for (int64_t o = 0; o < Cout; o++) {
                                    const double* wk = w + (o * 27 + tap) * Cin;
                                    for (int64_t i = 0; i < Cin; i++) out[i] += wk[i] * g[o];
                                }
                            }
                }
    return PV_ORACLE_OK;
}

/* Convolution, gradient with respect to its weights:
 * dL/dW[o][d][i] = sum over clouds b and output voxels p of
 *                  dL/dy[b][p][o] * x[b][p + d][i], for p + d inside the grid.
 * dy [B][R^3][Cout], x [B][R^3][Cin] -> dw [Cout][27][Cin]. */
int ref_conv3d_backward_weight(const double* dy, const double* x, int64_t B, int R, int64_t Cin,
                               int64_t Cout, double* dw) {
    if (B < 0 || R < 1 || Cin < 1 || Cout < 1) return PV_ORACLE_EINVAL;
    int64_t V = (int64_t)R * R * R;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t o = 0; o < Cout; o++)
        for (int tap = 0; tap < 27; tap++) {
            int du = tap / 9 - 1, dv = (tap / 3) % 3 - 1, dw_ = tap % 3 - 1;
            double* out = dw + (o * 27 + tap) * Cin;
            for (int64_t i = 0; i < Cin; i++) out[i] = 0.0;
            for (int64_t b = 0; b < B; b++)
                for (int64_t u = 0; u < R; u++)
                    for (int64_t v = 0; v < R; v++)
                        for (int64_t ww = 0; ww < R; ww++) {
                            int64_t nu = u + du, nv = v + dv, nw = ww + dw_;
                            if (nu < 0 || nu >= R || nv < 0 || nv >= R || nw < 0 || nw >= R)
                                continue;
                            double g = dy[(b * V + (u * R + v) * R + ww) * Cout + o];
                            if (g == 0.0) continue;
                            const double* xin = x + (b * V + (nu * R + nv) * R + nw) * Cin;
                            for (int64_t i = 0; i < Cin; i++) out[i] += g * xin[i];
                        }
        }
    return PV_ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* PointNet++ primitives (PVCNN++, Section 5.2 "Models")                     */
/* ------------------------------------------------------------------------- */

/* Squared distance between two points of fp32 coordinates, in fp32, in the
 * form the kernels use: fused multiply-adds, each rounded once. */
static float sqdist_f32(const float* a, const float* b) {
    const float dx = a[0] - b[0];
    const float dy = a[1] - b[1];
    const float dz = a[2] - b[2];
    return fmaf(dz, dz, fmaf(dy, dy, dx * dx));
}

/* Iterative farthest point sampling. The first sample is point 0; each next
 * one is the point whose distance to the samples taken so far (the minimum
 * over them) is largest, the lowest index among equals. xyz [B][N][3],
 * idx out [B][npoint]. 1 <= npoint <= N. */
int ref_fps(const float* xyz, int64_t B, int64_t N, int64_t npoint, int32_t* idx) {
    if (B < 0 || N < 1 || npoint < 1 || npoint > N) return PV_ORACLE_EINVAL;
    float* dmin = (float*)malloc((size_t)N * sizeof(float));
    if (!dmin) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++) {
        const float* p = xyz + b * N * 3;
        int32_t* out = idx + b * npoint;
        for (int64_t j = 0; j < N; j++) dmin[j] = INFINITY;
        int64_t last = 0;
        out[0] = 0;
        for (int64_t s = 1; s < npoint; s++) {
            int64_t best = 0;
            float bestd = -1.0f;
            for (int64_t j = 0; j < N; j++) {
                const float d = sqdist_f32(p + j * 3, p + last * 3);
                if (d < dmin[j]) dmin[j] = d;
                if (dmin[j] > bestd) {
                    bestd = dmin[j];
                    best = j;
                }
            }
            out[s] = (int32_t)best;
            last = best;
        }
    }
    free(dmin);
    return PV_ORACLE_OK;
}

/* Ball query: for each centre, the first nsample points (in index order)
 * whose squared distance to it is below radius^2 (radius^2 formed in fp32);
 * a centre with fewer repeats its first neighbour in the remaining slots, and
 * one with none gets point 0 in every slot. xyz [B][N][3], centers
 * [B][npoint][3], idx out [B][npoint][nsample]. */
int ref_ball_query(const float* xyz, int64_t B, int64_t N, const float* centers,
                   int64_t npoint, float radius, int64_t nsample, int32_t* idx) {
    if (B < 0 || N < 1 || npoint < 0 || nsample < 1 || !(radius >= 0.0f))
        return PV_ORACLE_EINVAL;
    const float r2 = radius * radius;
    for (int64_t b = 0; b < B; b++)
        for (int64_t i = 0; i < npoint; i++) {
            const float* c = centers + (b * npoint + i) * 3;
            int32_t* out = idx + (b * npoint + i) * nsample;
            int64_t cnt = 0;
            for (int64_t j = 0; j < N && cnt < nsample; j++)
                if (sqdist_f32(xyz + (b * N + j) * 3, c) < r2) out[cnt++] = (int32_t)j;
            const int32_t fill = cnt > 0 ? out[0] : 0;
            for (int64_t k = cnt; k < nsample; k++) out[k] = fill;
        }
    return PV_ORACLE_OK;
}

/* Grouping: for centre i and slot k with neighbour j = idx[b][i][k], the row
 * (x_j - c_i, feats_j): the neighbour's coordinates relative to the centre,
 * then its C features. out [B][npoint][nsample][3 + C]. */
int ref_group(const float* xyz, const double* feats, int64_t B, int64_t N, int64_t C,
              const float* centers, int64_t npoint, const int32_t* idx, int64_t nsample,
              double* out) {
    if (B < 0 || N < 1 || C < 0 || npoint < 0 || nsample < 1) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++)
        for (int64_t i = 0; i < npoint; i++) {
            const float* cf = centers + (b * npoint + i) * 3;
            for (int64_t k = 0; k < nsample; k++) {
                const int64_t j = idx[(b * npoint + i) * nsample + k];
                if (j < 0 || j >= N) return PV_ORACLE_EINVAL;
                double* o = out + ((b * npoint + i) * nsample + k) * (3 + C);
                const float* p = xyz + (b * N + j) * 3;
                for (int a = 0; a < 3; a++) o[a] = (double)p[a] - (double)cf[a];
                for (int64_t ch = 0; ch < C; ch++) o[3 + ch] = feats[(b * N + j) * C + ch];
            }
        }
    return PV_ORACLE_OK;
}

/* Three nearest neighbours: for each of the n unknown points, the three known
 * points (of m >= 3) with the smallest squared distance, nearest first, the
 * lower index first among equals; and the inverse-distance weights
 * w_k = (1 / (d_k + 1e-8)) / sum_l (1 / (d_l + 1e-8)) with d the Euclidean
 * distance. unknown [B][n][3], known [B][m][3]; idx out [B][n][3], weight out
 * [B][n][3]. */
int ref_three_nn(const float* unknown, int64_t B, int64_t n, const float* known, int64_t m,
                 int32_t* idx, double* weight) {
    if (B < 0 || n < 0 || m < 3) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++)
        for (int64_t i = 0; i < n; i++) {
            const float* u = unknown + (b * n + i) * 3;
            float bd[3] = {INFINITY, INFINITY, INFINITY};
            int64_t bi[3] = {0, 0, 0};
            for (int64_t j = 0; j < m; j++) {
                const float d = sqdist_f32(known + (b * m + j) * 3, u);
                /* strictly smaller moves ahead: among equals the earlier
                 * (lower) index stays in front */
                if (d < bd[0]) {
                    bd[2] = bd[1]; bi[2] = bi[1];
                    bd[1] = bd[0]; bi[1] = bi[0];
                    bd[0] = d; bi[0] = j;
                } else if (d < bd[1]) {
                    bd[2] = bd[1]; bi[2] = bi[1];
                    bd[1] = d; bi[1] = j;
                } else if (d < bd[2]) {
                    bd[2] = d; bi[2] = j;
                }
            }
            double inv[3], sum = 0.0;
            for (int k = 0; k < 3; k++) {
                inv[k] = 1.0 / (sqrt((double)bd[k]) + 1e-8);
                sum += inv[k];
            }
            for (int k = 0; k < 3; k++) {
                idx[(b * n + i) * 3 + k] = (int32_t)bi[k];
                weight[(b * n + i) * 3 + k] = inv[k] / sum;
            }
        }
    return PV_ORACLE_OK;
}

/* Inverse-distance interpolation: out[b][i][c] = sum_k weight[b][i][k] *
 * feats[b][idx[b][i][k]][c]. feats [B][m][C], out [B][n][C]. */
int ref_three_interpolate(const double* feats, int64_t B, int64_t m, int64_t C,
                          const int32_t* idx, const double* weight, int64_t n, double* out) {
    if (B < 0 || m < 1 || C < 1 || n < 0) return PV_ORACLE_EINVAL;
    for (int64_t b = 0; b < B; b++)
        for (int64_t i = 0; i < n; i++)
            for (int64_t c = 0; c < C; c++) {
                double acc = 0.0;
                for (int k = 0; k < 3; k++) {
                    const int64_t j = idx[(b * n + i) * 3 + k];
                    if (j < 0 || j >= m) return PV_ORACLE_EINVAL;
                    acc += weight[(b * n + i) * 3 + k] * feats[(b * m + j) * C + c];
                }
                out[(b * n + i) * C + c] = acc;
            }
    return PV_ORACLE_OK;
}
