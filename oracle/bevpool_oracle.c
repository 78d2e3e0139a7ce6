/*
 * CPU oracle for BEV pooling (BEVFusion, arXiv 2205.13542, Sec. III-B).
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke entry point and the
 * benchmark's CPU-baseline leg may load this library. It shares no code,
 * header or constant with the GPU library; the two are compared, never mixed.
 *
 * What is computed, as plain definitions written out:
 *
 *   - The camera feature point cloud (Sec. III-B, first paragraph): every
 *     camera n, depth bin d, feature pixel (h, w) gives one point, N*D*H*W in
 *     all. Its feature is P[n,d,h,w] * F[n,h,w,:] (depth probability times the
 *     pixel's feature vector).
 *   - Its 3-D position: the pixel's camera ray at depth d, mapped to the ego
 *     frame by the camera's extrinsics (same paragraph; the "Precomputation"
 *     paragraph computes this coordinate once per calibration).
 *   - Quantisation to a BEV cell of step r along x and y, and flattening along
 *     z (first paragraph). Points outside the grid are dropped.
 *   - The association: grid index per point, points ordered by grid index,
 *     each point's rank recorded ("Precomputation" paragraph). After it, the
 *     points of one cell are consecutive ("Interval Reduction" paragraph).
 *   - Pooling by sum, one of the symmetric functions the "Interval Reduction"
 *     paragraph allows, with no approximation ("Takeaways" paragraph: the
 *     method is exact); and by mean and max, the other two it names.
 *
 * Readings where the paper is silent (each one is also listed with the design
 * notes of the GPU library, which implements the same readings independently):
 *   - depth of bin k: d_k = depth_min + k * depth_step, k in [0, D);
 *   - depth is camera-frame z (the ray point is d * K^-1 [u, v, 1]);
 *   - pixel (h, w) sits at u = w + pixel_offset, v = h + pixel_offset;
 *   - extrinsics map camera to ego: p_ego = R p_cam + t;
 *   - quantisation uses floor, and the range test is done on the floored
 *     index, so each cell is half-open [min + i*r, min + (i+1)*r);
 *   - z is quantised like x and y: iz = floor((z - z_min) / z_cell); with one
 *     z slab a point is kept only if iz == 0, with nz slabs if 0 <= iz < nz;
 *   - cell id = iy * nx + ix; output layout [B][ny][nx][C]; with nz slabs the
 *     cell id is (iy * nx + ix) * nz + iz, so a [B][ny][nx][nz][C] map is the
 *     slabs' features concatenated along channels (flattening along z);
 *   - ties in the sort are broken by point id (a stable sort);
 *   - all geometry is IEEE double, evaluated in the fixed order below, with
 *     no fused multiply-add (this file is built with -ffp-contract=off);
 *   - sums are accumulated in double from zero and rounded once to float.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Field order is part of the ctypes contract in oracle/__init__.py. */
typedef struct {
    int32_t n_cams, feat_h, feat_w, n_depth;
    double depth_min, depth_step, pixel_offset;
    int32_t nx, ny;
    double x_min, y_min, cell_x, cell_y;
    double z_min, z_cell;
} oracle_geometry;

static int64_t n_points_of(const oracle_geometry *g) {
    return (int64_t)g->n_cams * g->n_depth * g->feat_h * g->feat_w;
}

/*
 * Grid index of every frustum point, in point-id order
 * p = ((n*D + d)*H + h)*W + w. Dropped points get -1.
 * intrinsics: [N][4] = fx, fy, cx, cy (feature-grid pixels).
 * extrinsics: [N][12] = row-major [R | t], camera to ego.
 * Returns the number of kept points.
 */
/*
 * Grid index of every frustum point over nz stacked z slabs (nz >= 1):
 * iz = floor((z - z_min) / z_cell) in [0, nz), cell (iy * nx + ix) * nz + iz.
 * Returns the number of kept points.
 */
int64_t oracle_cell_map_slabs(const double *intrinsics, const double *extrinsics,
                              const oracle_geometry *g, int32_t nz, int32_t *cell_of_point) {
    int64_t kept = 0;
    int64_t p = 0;
    for (int n = 0; n < g->n_cams; ++n) {
        const double fx = intrinsics[4 * n + 0];
        const double fy = intrinsics[4 * n + 1];
        const double cx = intrinsics[4 * n + 2];
        const double cy = intrinsics[4 * n + 3];
        const double *E = extrinsics + 12 * n;
        for (int d = 0; d < g->n_depth; ++d) {
            const double depth = g->depth_min + (double)d * g->depth_step;
            for (int h = 0; h < g->feat_h; ++h) {
                for (int w = 0; w < g->feat_w; ++w, ++p) {
                    /* point on the pixel's ray at camera-frame depth `depth` */
                    const double u = (double)w + g->pixel_offset;
                    const double v = (double)h + g->pixel_offset;
                    const double xc = depth * ((u - cx) / fx);
                    const double yc = depth * ((v - cy) / fy);
                    const double zc = depth;
                    /* camera frame -> ego frame */
                    const double X = ((E[0] * xc + E[1] * yc) + E[2] * zc) + E[3];
                    const double Y = ((E[4] * xc + E[5] * yc) + E[6] * zc) + E[7];
                    const double Z = ((E[8] * xc + E[9] * yc) + E[10] * zc) + E[11];
                    /* quantise; keep only points inside the grid and the slabs */
                    const double qx = floor((X - g->x_min) / g->cell_x);
                    const double qy = floor((Y - g->y_min) / g->cell_y);
                    const double qz = floor((Z - g->z_min) / g->z_cell);
                    int32_t cell = -1;
                    if (qx >= 0.0 && qx < (double)g->nx &&
                        qy >= 0.0 && qy < (double)g->ny && qz >= 0.0 && qz < (double)nz) {
                        cell = ((int32_t)qy * g->nx + (int32_t)qx) * nz + (int32_t)qz;
                        ++kept;
                    }
                    cell_of_point[p] = cell;
                }
            }
        }
    }
    return kept;
}

/* One z slab: a point is kept only if iz == 0; cell id iy * nx + ix. */
int64_t oracle_cell_map(const double *intrinsics, const double *extrinsics,
                        const oracle_geometry *g, int32_t *cell_of_point) {
    return oracle_cell_map_slabs(intrinsics, extrinsics, g, 1, cell_of_point);
}

/*
 * Points ordered by grid index, ties by point id (stable counting placement),
 * and the interval table: cell_start[c] .. cell_start[c+1] is cell c's run.
 * sorted_point receives the kept points only (cell_start[n_cells] of them).
 */
void oracle_sort_by_cell(const int32_t *cell_of_point, int64_t n_points,
                         int32_t n_cells, int32_t *sorted_point,
                         int32_t *cell_start) {
    int64_t *count = (int64_t *)calloc((size_t)n_cells + 1, sizeof(int64_t));
    for (int64_t p = 0; p < n_points; ++p)
        if (cell_of_point[p] >= 0) count[cell_of_point[p]] += 1;
    int64_t run = 0;
    for (int32_t c = 0; c < n_cells; ++c) {
        cell_start[c] = (int32_t)run;
        run += count[c];
    }
    cell_start[n_cells] = (int32_t)run;
    /* place each point after the earlier points of its cell */
    memset(count, 0, ((size_t)n_cells + 1) * sizeof(int64_t));
    for (int64_t p = 0; p < n_points; ++p) {
        const int32_t c = cell_of_point[p];
        if (c < 0) continue;
        sorted_point[cell_start[c] + count[c]] = (int32_t)p;
        count[c] += 1;
    }
    free(count);
}

/*
 * Sum pooling: out[b][cell][:] = sum over kept points p of that cell of
 * P[b][p] * F[b][pixel(p)][:], accumulated in double over points in id order.
 * P: [B][N][D][H][W], F: [B][N][H][W][C], both float (reduced-precision
 * inputs are widened exactly by the caller). out: [B][ny][nx][C] float.
 * out64 (optional) receives the double sums before rounding, abs64
 * (optional) the sums of |P * F| per element, a scale for error bounds.
 * Channels are split across threads; every element keeps the same
 * summation order, so the result does not depend on the thread count.
 */
void oracle_pool(const float *P, const float *F, const int32_t *cell_of_point,
                 const oracle_geometry *g, int32_t batch, int32_t channels,
                 float *out, double *out64, double *abs64) {
    const int64_t NP = n_points_of(g);
    const int64_t HW = (int64_t)g->feat_h * g->feat_w;
    const int64_t DHW = (int64_t)g->n_depth * HW;
    const int64_t n_pix = (int64_t)g->n_cams * HW;
    const int64_t n_cells = (int64_t)g->nx * g->ny;
    const int64_t C = channels;
    for (int32_t b = 0; b < batch; ++b) {
        const float *Pb = P + (size_t)b * NP;
        const float *Fb = F + (size_t)b * n_pix * C;
        float *ob = out + (size_t)b * n_cells * C;
        double *acc = (double *)calloc((size_t)n_cells * C, sizeof(double));
        double *aacc = abs64 ? (double *)calloc((size_t)n_cells * C, sizeof(double)) : NULL;
#pragma omp parallel
        {
            int64_t c0 = 0, c1 = C;
#ifdef _OPENMP
            const int64_t nt = omp_get_num_threads(), t = omp_get_thread_num();
            const int64_t slice = (C + nt - 1) / nt;
            c0 = t * slice < C ? t * slice : C;
            c1 = c0 + slice < C ? c0 + slice : C;
#endif
            for (int64_t p = 0; p < NP && c0 < c1; ++p) {
                const int32_t cell = cell_of_point[p];
                if (cell < 0) continue;
                const int64_t n = p / DHW;
                const int64_t hw = p % HW;
                const double prob = (double)Pb[p];
                const float *feat = Fb + (n * HW + hw) * C;
                double *a = acc + (int64_t)cell * C;
                double *aa = aacc ? aacc + (int64_t)cell * C : NULL;
                for (int64_t c = c0; c < c1; ++c) {
                    const double term = prob * (double)feat[c];
                    a[c] += term;
                    if (aa) aa[c] += fabs(term);
                }
            }
        }
        for (int64_t i = 0; i < n_cells * C; ++i) ob[i] = (float)acc[i];
        if (out64) memcpy(out64 + (size_t)b * n_cells * C, acc, (size_t)n_cells * C * sizeof(double));
        if (abs64) memcpy(abs64 + (size_t)b * n_cells * C, aacc, (size_t)n_cells * C * sizeof(double));
        free(acc);
        free(aacc);
    }
}

/*
 * Mean and max pooling: the other two symmetric functions the "Interval
 * Reduction" paragraph names for aggregating a cell's points.
 *   mode 1 (mean): out = (sum over the cell's kept points of P * F) divided
 *                  by the number of those points, in double;
 *   mode 2 (max):  out = the largest P * F over those points, per channel;
 *                  each product is exact in double (a float times a float
 *                  has at most 48 significant bits).
 * A cell without points gets 0 in both modes. P, F and the layouts are those
 * of oracle_pool; out64: [B][ny][nx][C] double. Channels are split across
 * threads as in oracle_pool.
 */
void oracle_pool_reduce(const float *P, const float *F, const int32_t *cell_of_point,
                        const oracle_geometry *g, int32_t batch, int32_t channels,
                        int32_t mode, double *out64) {
    const int64_t NP = n_points_of(g);
    const int64_t HW = (int64_t)g->feat_h * g->feat_w;
    const int64_t DHW = (int64_t)g->n_depth * HW;
    const int64_t n_pix = (int64_t)g->n_cams * HW;
    const int64_t n_cells = (int64_t)g->nx * g->ny;
    const int64_t C = channels;
    int64_t *count = (int64_t *)calloc((size_t)n_cells, sizeof(int64_t));
    for (int64_t p = 0; p < NP; ++p) {
        if (cell_of_point[p] >= 0) ++count[cell_of_point[p]];
    }
    for (int32_t b = 0; b < batch; ++b) {
        const float *Pb = P + (size_t)b * NP;
        const float *Fb = F + (size_t)b * n_pix * C;
        double *acc = out64 + (size_t)b * n_cells * C;
        const double init = mode == 2 ? -INFINITY : 0.0;
        for (int64_t i = 0; i < n_cells * C; ++i) acc[i] = init;
#pragma omp parallel
        {
            int64_t c0 = 0, c1 = C;
#ifdef _OPENMP
            const int64_t nt = omp_get_num_threads(), t = omp_get_thread_num();
            const int64_t slice = (C + nt - 1) / nt;
            c0 = t * slice < C ? t * slice : C;
            c1 = c0 + slice < C ? c0 + slice : C;
#endif
            for (int64_t p = 0; p < NP && c0 < c1; ++p) {
                const int32_t cell = cell_of_point[p];
                if (cell < 0) continue;
                const int64_t n = p / DHW;
                const int64_t hw = p % HW;
                const double prob = (double)Pb[p];
                const float *feat = Fb + (n * HW + hw) * C;
                double *a = acc + (int64_t)cell * C;
                for (int64_t c = c0; c < c1; ++c) {
                    const double term = prob * (double)feat[c];
                    if (mode == 2) {
                        if (term > a[c]) a[c] = term;
                    } else {
                        a[c] += term;
                    }
                }
            }
        }
        for (int64_t cell = 0; cell < n_cells; ++cell) {
            double *a = acc + cell * C;
            for (int64_t c = 0; c < C; ++c) {
                if (count[cell] == 0) a[c] = 0.0;
                else if (mode == 1) a[c] = a[c] / (double)count[cell];
            }
        }
    }
    free(count);
}

/*
 * Gradients of sum pooling. The forward map is bilinear in (P, F): each kept
 * point p adds P[p] * F[pixel(p)][:] to its cell's row (Sec. III-B; the
 * paper trains the whole model end to end, so the pooling is differentiated
 * like any other layer). With G = d loss / d out [B][ny][nx][C]:
 *   dP[b][p]        = sum_c F[b][pixel(p)][c] * G[b][cell(p)][c]  (kept p; 0 if dropped)
 *   dF[b][pix][c]   = sum over kept points p of the pixel of P[b][p] * G[b][cell(p)][c]
 * accumulated in double: dP over channels in channel order, dF over the
 * pixel's depth bins in bin order. Each pixel owns its D points and its dF
 * row, so pixels are split across threads without any shared sum.
 * dP64: [B][N][D][H][W] double, dF64: [B][N][H][W][C] double.
 */
void oracle_backward(const float *P, const float *F, const float *G,
                     const int32_t *cell_of_point, const oracle_geometry *g,
                     int32_t batch, int32_t channels, double *dP64, double *dF64) {
    const int64_t NP = n_points_of(g);
    const int64_t HW = (int64_t)g->feat_h * g->feat_w;
    const int64_t D = g->n_depth;
    const int64_t n_pix = (int64_t)g->n_cams * HW;
    const int64_t n_cells = (int64_t)g->nx * g->ny;
    const int64_t C = channels;
    for (int32_t b = 0; b < batch; ++b) {
        const float *Pb = P + (size_t)b * NP;
        const float *Fb = F + (size_t)b * n_pix * C;
        const float *Gb = G + (size_t)b * n_cells * C;
        double *dPb = dP64 + (size_t)b * NP;
        double *dFb = dF64 + (size_t)b * n_pix * C;
#pragma omp parallel for schedule(static)
        for (int64_t pix = 0; pix < n_pix; ++pix) {
            const int64_t n = pix / HW, hw = pix % HW;
            const float *feat = Fb + pix * C;
            double *df = dFb + pix * C;
            for (int64_t c = 0; c < C; ++c) df[c] = 0.0;
            for (int64_t d = 0; d < D; ++d) {
                const int64_t p = (n * D + d) * HW + hw;
                const int32_t cell = cell_of_point[p];
                if (cell < 0) {
                    dPb[p] = 0.0;
                    continue;
                }
                const float *grad = Gb + (int64_t)cell * C;
                const double prob = (double)Pb[p];
                double dot = 0.0;
                for (int64_t c = 0; c < C; ++c) {
                    dot += (double)feat[c] * (double)grad[c];
                    df[c] += prob * (double)grad[c];
                }
                dPb[p] = dot;
            }
        }
    }
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of later parallel regions started from the calling thread (n >= 1);
 * every function above gives bitwise the same result for any count. */
void oracle_set_threads(int n) {
#ifdef _OPENMP
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}
