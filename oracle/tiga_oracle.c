/*
 * CPU oracle for fused message passing -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests, the smoke check and the benchmark's CPU-baseline leg may load
 * this library.  It shares no code, header, table or constant with the HIP
 * library; the two only consume the same seeded inputs.
 *
 * Everything here is the plain definition of what fused message passing
 * computes (Tiga, "Compiling Graph Message Passing at Scale"):
 *
 *   m_e = f(x_{s(e)}, z_{d(e)}, a_e),   y_i = finalize( combine_{d(e)=i} m_e )
 *   (Section 3.1, the message/update equation)
 *
 * with the relation given as destination-major CSR (Section 3.1 and 4.3:
 * row i owns edge positions [row_ptr[i], row_ptr[i+1]); the edge position
 * indexes edge fields and col[e] is the source id), as a radius predicate over
 * positions (Section 4.9, generated relations), or as all ordered pairs j != i.
 *
 * Floating point: inputs are fp32; every sum is accumulated in fp64 (fp32 x
 * fp32 products are exact in fp64) and returned in fp64, together with the
 * sum of absolute values of its terms, so a caller can bound the error of any
 * fp32 summation order.  The max reducer and the radius membership test are
 * decisions, so they are evaluated in fp32 exactly as the message is defined
 * (one fp32 multiply; an fp32 squared distance without contraction).  Build
 * with -ffp-contract=off.
 *
 * Parity pins for every function are in the CPU test suite (worked example of
 * Section 3.1, library routines, brute force, invariants, finite differences).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

int tiga_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for the following calls: n >= 1 sets that many, n <= 0 restores the default (all host
 * cores).  Only the timing of the baseline uses it; every result is independent of it (each
 * output is summed by one thread in a fixed order). */
static int default_threads = 0;
void tiga_oracle_set_threads(int n) {
#ifdef _OPENMP
    if (default_threads == 0) default_threads = omp_get_max_threads();
    omp_set_num_threads(n >= 1 ? n : default_threads);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Stored CSR relation, weighted-sum message                                 */
/* ------------------------------------------------------------------------ */

/* Sum reducer (Section 3.1; identity 0, so an empty row finalizes to 0):
 *   y[i,f] = sum_{e in row i} w[e] * x[col[e], f]     (w == NULL means w = 1)
 * Rows are taken from `rows` (nrows entries) or, if rows == NULL, all rows
 * 0..nrows-1.  Output k belongs to row rows[k]. */
void tiga_oracle_csr_sum_fwd(int64_t nrows, const int64_t *rows, int32_t F,
                             const int64_t *row_ptr, const int32_t *col,
                             const float *x, const float *w,
                             double *y, double *yabs) {
    int64_t k;
#pragma omp parallel for schedule(dynamic, 64)
    for (k = 0; k < nrows; ++k) {
        int64_t i = rows ? rows[k] : k;
        for (int32_t f = 0; f < F; ++f) {
            double acc = 0.0, mag = 0.0;
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                double term = (w ? (double)w[e] : 1.0) * (double)x[(int64_t)col[e] * F + f];
                acc += term;
                mag += fabs(term);
            }
            y[k * F + f] = acc;
            if (yabs) yabs[k * F + f] = mag;
        }
    }
}

/* Max reducer.  The paper leaves max undefined beyond "an empty row starts
 * from the identity and finalization fixes the empty-row convention"
 * (Section 3.1).  Reading: identity -inf; the message is the fp32 product
 * w[e]*x[col[e],f]; edges are visited in ascending CSR position and a later
 * edge replaces the best only if strictly greater, so ties keep the lowest
 * edge position (+0 and -0 compare equal); an empty row finalizes to value 0
 * and argmax -1. */
void tiga_oracle_csr_max_fwd(int64_t nrows, const int64_t *rows, int32_t F,
                             const int64_t *row_ptr, const int32_t *col,
                             const float *x, const float *w,
                             float *y, int32_t *arg) {
    int64_t k;
#pragma omp parallel for schedule(dynamic, 64)
    for (k = 0; k < nrows; ++k) {
        int64_t i = rows ? rows[k] : k;
        for (int32_t f = 0; f < F; ++f) {
            int have = 0;
            float best = 0.0f;
            int64_t best_e = -1;
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                float xv = x[(int64_t)col[e] * F + f];
                float v = w ? w[e] * xv : xv;
                if (!have || v > best) {
                    best = v;
                    best_e = e;
                    have = 1;
                }
            }
            y[k * F + f] = have ? best : 0.0f;
            arg[k * F + f] = (int32_t)best_e;
        }
    }
}

/* Vector-Jacobian product of the weighted sum (Section 5, adjoint equation):
 *   dx[j,f] = sum_{e : col[e] = j} w[e] * dy[d(e), f]
 *   dw[e]   = sum_f x[col[e], f] * dy[d(e), f]
 * (the paper writes dw for one feature; a per-edge scalar weight broadcast
 * over F features collects the sum over f).  Repeated sources accumulate,
 * edges of empty rows do not exist.  dx is over all num_src sources, dw over
 * all edges; either may be NULL.  A plain serial walk over rows and edges. */
void tiga_oracle_csr_sum_bwd(int64_t num_dst, int64_t num_src, int32_t F,
                             const int64_t *row_ptr, const int32_t *col,
                             const float *x, const float *w, const float *dy,
                             double *dx, double *dxabs, double *dw, double *dwabs) {
    if (dx) {
        memset(dx, 0, sizeof(double) * (size_t)num_src * F);
        if (dxabs) memset(dxabs, 0, sizeof(double) * (size_t)num_src * F);
        for (int64_t i = 0; i < num_dst; ++i)
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
                for (int32_t f = 0; f < F; ++f) {
                    double term = (w ? (double)w[e] : 1.0) * (double)dy[i * F + f];
                    dx[(int64_t)col[e] * F + f] += term;
                    if (dxabs) dxabs[(int64_t)col[e] * F + f] += fabs(term);
                }
    }
    if (dw) {
        int64_t i;
#pragma omp parallel for schedule(dynamic, 64)
        for (i = 0; i < num_dst; ++i)
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                double acc = 0.0, mag = 0.0;
                for (int32_t f = 0; f < F; ++f) {
                    double term = (double)x[(int64_t)col[e] * F + f] * (double)dy[i * F + f];
                    acc += term;
                    mag += fabs(term);
                }
                dw[e] = acc;
                if (dwabs) dwabs[e] = mag;
            }
    }
}

/* Vector-Jacobian product of the max reducer: y[i,f] depends only on the
 * selected edge e* = arg[i,f] (the derivative of max with respect to the
 * selected message is 1 and 0 for the others), so
 *   dx[col[e*], f] += w[e*] * dy[i,f],   dw[e*] += x[col[e*], f] * dy[i,f]
 * for every (i,f) with e* >= 0.  Empty rows contribute nothing. */
void tiga_oracle_csr_max_bwd(int64_t num_dst, int64_t num_src, int64_t num_edges, int32_t F,
                             const int64_t *row_ptr, const int32_t *col,
                             const float *x, const float *w, const int32_t *arg,
                             const float *dy,
                             double *dx, double *dxabs, double *dw, double *dwabs) {
    (void)row_ptr;
    if (dx) {
        memset(dx, 0, sizeof(double) * (size_t)num_src * F);
        if (dxabs) memset(dxabs, 0, sizeof(double) * (size_t)num_src * F);
    }
    if (dw) {
        memset(dw, 0, sizeof(double) * (size_t)num_edges);
        if (dwabs) memset(dwabs, 0, sizeof(double) * (size_t)num_edges);
    }
    for (int64_t i = 0; i < num_dst; ++i)
        for (int32_t f = 0; f < F; ++f) {
            int64_t e = arg[i * F + f];
            if (e < 0) continue;
            int64_t j = col[e];
            double g = (double)dy[i * F + f];
            if (dx) {
                double term = (w ? (double)w[e] : 1.0) * g;
                dx[j * F + f] += term;
                if (dxabs) dxabs[j * F + f] += fabs(term);
            }
            if (dw) {
                double term = (double)x[j * F + f] * g;
                dw[e] += term;
                if (dwabs) dwabs[e] += fabs(term);
            }
        }
}

/* ------------------------------------------------------------------------ */
/* Generated radius relation (Section 4.9)                                   */
/* ------------------------------------------------------------------------ */

/* Membership: j != i and the fp32 squared distance, formed from direct
 * coordinate differences (the evaluation protocol uses direct differences,
 * not the |a|^2+|b|^2-2ab identity), is strictly below fp32(r*r).  Each
 * operation is one fp32 rounding; nothing is contracted. */
static int within(const float *pi, const float *pj, float r2) {
    float dx = pj[0] - pi[0];
    float dy = pj[1] - pi[1];
    float dz = pj[2] - pi[2];
    float sx = dx * dx;
    float sy = dy * dy;
    float sz = dz * dz;
    float d2 = (sx + sy) + sz;
    return d2 < r2;
}

/* A uniform cell directory: per axis, the box [lo, hi] is cut into cells no
 * smaller than r (with a 1e-3 relative margin), so every accepted neighbour
 * of a point lies in the 27 cells around the point's own cell.  Cells only
 * restrict the candidates; the predicate alone decides membership. */
typedef struct {
    int64_t n;
    double lo[3], h[3];
    int64_t dim[3];
    int64_t *start; /* ncell + 1 */
    int64_t *items; /* point ids, grouped by cell, ascending within a cell */
} grid_t;

static int64_t cell_coord(const grid_t *g, int a, float p) {
    int64_t c = (int64_t)floor(((double)p - g->lo[a]) / g->h[a]);
    if (c < 0) c = 0;
    if (c >= g->dim[a]) c = g->dim[a] - 1;
    return c;
}

static int grid_build(grid_t *g, int64_t n, const float *pos, float radius) {
    g->n = n;
    for (int a = 0; a < 3; ++a) {
        double lo = INFINITY, hi = -INFINITY;
        for (int64_t i = 0; i < n; ++i) {
            double v = pos[i * 3 + a];
            if (v < lo) lo = v;
            if (v > hi) hi = v;
        }
        if (n == 0) lo = hi = 0.0;
        double ext = hi - lo;
        double hmin = (double)radius * 1.001;
        int64_t d = (hmin > 0.0) ? (int64_t)floor(ext / hmin) : 1;
        if (d < 1) d = 1;
        if (d > 1024) d = 1024;
        g->lo[a] = lo;
        g->h[a] = (ext > 0.0) ? ext / (double)d : 1.0;
        g->dim[a] = d;
    }
    int64_t ncell = g->dim[0] * g->dim[1] * g->dim[2];
    g->start = (int64_t *)calloc((size_t)ncell + 1, sizeof(int64_t));
    g->items = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n ? n : 1));
    int64_t *cell = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n ? n : 1));
    if (!g->start || !g->items || !cell) return -1;
    for (int64_t i = 0; i < n; ++i) {
        const float *p = pos + i * 3;
        cell[i] = (cell_coord(g, 2, p[2]) * g->dim[1] + cell_coord(g, 1, p[1])) * g->dim[0] +
                  cell_coord(g, 0, p[0]);
        g->start[cell[i] + 1]++;
    }
    for (int64_t c = 0; c < ncell; ++c) g->start[c + 1] += g->start[c];
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)ncell);
    if (!fill) return -1;
    memcpy(fill, g->start, sizeof(int64_t) * (size_t)ncell);
    for (int64_t i = 0; i < n; ++i) g->items[fill[cell[i]]++] = i;
    free(fill);
    free(cell);
    return 0;
}

static void grid_free(grid_t *g) {
    free(g->start);
    free(g->items);
}

/* Visit the accepted neighbours of point i in ascending index order.  With
 * use_grid == 0 this is the plain O(N) scan over all j. */
typedef void (*visit_fn)(void *ctx, int64_t i, int64_t j);

static int cmp_i64(const void *a, const void *b) {
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

static int64_t neighbours(const grid_t *g, int use_grid, int64_t n, const float *pos, float r2,
                          int64_t i, int64_t *buf, int64_t cap) {
    int64_t cnt = 0;
    const float *pi = pos + i * 3;
    if (!use_grid) {
        for (int64_t j = 0; j < n; ++j)
            if (j != i && within(pi, pos + j * 3, r2)) {
                if (cnt < cap) buf[cnt] = j;
                cnt++;
            }
        return cnt;
    }
    int64_t c[3];
    for (int a = 0; a < 3; ++a) c[a] = cell_coord(g, a, pi[a]);
    for (int64_t cz = c[2] - 1; cz <= c[2] + 1; ++cz) {
        if (cz < 0 || cz >= g->dim[2]) continue;
        for (int64_t cy = c[1] - 1; cy <= c[1] + 1; ++cy) {
            if (cy < 0 || cy >= g->dim[1]) continue;
            for (int64_t cx = c[0] - 1; cx <= c[0] + 1; ++cx) {
                if (cx < 0 || cx >= g->dim[0]) continue;
                int64_t cell = (cz * g->dim[1] + cy) * g->dim[0] + cx;
                for (int64_t t = g->start[cell]; t < g->start[cell + 1]; ++t) {
                    int64_t j = g->items[t];
                    if (j != i && within(pi, pos + j * 3, r2)) {
                        if (cnt < cap) buf[cnt] = j;
                        cnt++;
                    }
                }
            }
        }
    }
    if (cnt <= cap) qsort(buf, (size_t)cnt, sizeof(int64_t), cmp_i64);
    return cnt;
}

/* Shared driver: for each requested point, gather its sorted neighbour list
 * and hand it to `body`. */
typedef void (*point_body)(void *ctx, int64_t k, int64_t i, const int64_t *nb, int64_t cnt);

static int for_each_point(int64_t n, const float *pos, float radius, int64_t npts,
                          const int64_t *pts, point_body body, void *ctx) {
    float r2 = radius * radius;
    grid_t g;
    memset(&g, 0, sizeof g);
    int use_grid = n > 4096;
    if (use_grid && grid_build(&g, n, pos, radius) != 0) return -1;
    int err = 0;
    int64_t k;
#pragma omp parallel
    {
        int64_t cap = 256;
        int64_t *buf = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
#pragma omp for schedule(dynamic, 64)
        for (k = 0; k < npts; ++k) {
            int64_t i = pts ? pts[k] : k;
            int64_t cnt = neighbours(&g, use_grid, n, pos, r2, i, buf, cap);
            if (cnt > cap) {
                free(buf);
                cap = cnt;
                buf = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
                if (!buf) {
#pragma omp atomic write
                    err = 1;
                    cap = 0;
                    continue;
                }
                cnt = neighbours(&g, use_grid, n, pos, r2, i, buf, cap);
            }
            body(ctx, k, i, buf, cnt);
        }
        free(buf);
    }
    if (use_grid) grid_free(&g);
    return err ? -1 : 0;
}

/* Gaussian weight of an accepted pair, from the fp64 displacement. */
static double kernel_weight(const float *pi, const float *pj, double inv_s2, double d[3]) {
    d[0] = (double)pj[0] - (double)pi[0];
    d[1] = (double)pj[1] - (double)pi[1];
    d[2] = (double)pj[2] - (double)pi[2];
    return exp(-(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]) * inv_s2);
}

typedef struct {
    int32_t F;
    const float *pos, *x, *dy;
    double inv_s2;
    double *y, *yabs, *dx, *dxabs, *dp, *dpabs;
    int32_t *count;
} radius_ctx;

/* Forward: y_i = sum_{j in N(i)} exp(-|p_i - p_j|^2 / sigma^2) x_j, with
 * N(i) = { j != i : |p_j - p_i|^2 < r^2 }; count_i = |N(i)|. */
static void radius_fwd_body(void *vctx, int64_t k, int64_t i, const int64_t *nb, int64_t cnt) {
    radius_ctx *c = (radius_ctx *)vctx;
    const int32_t F = c->F;
    double *y = c->y + k * F;
    double *ya = c->yabs ? c->yabs + k * F : NULL;
    for (int32_t f = 0; f < F; ++f) {
        y[f] = 0.0;
        if (ya) ya[f] = 0.0;
    }
    const float *pi = c->pos + i * 3;
    for (int64_t t = 0; t < cnt; ++t) {
        int64_t j = nb[t];
        double d[3];
        double kw = kernel_weight(pi, c->pos + j * 3, c->inv_s2, d);
        for (int32_t f = 0; f < F; ++f) {
            double term = kw * (double)c->x[j * F + f];
            y[f] += term;
            if (ya) ya[f] += fabs(term);
        }
    }
    if (c->count) c->count[k] = (int32_t)cnt;
}

int tiga_oracle_radius_fwd(int64_t n, int32_t F, const float *pos, const float *x,
                           float radius, float sigma, int64_t npts, const int64_t *pts,
                           double *y, double *yabs, int32_t *count) {
    radius_ctx c;
    memset(&c, 0, sizeof c);
    c.F = F;
    c.pos = pos;
    c.x = x;
    c.inv_s2 = 1.0 / ((double)sigma * (double)sigma);
    c.y = y;
    c.yabs = yabs;
    c.count = count;
    return for_each_point(n, pos, radius, npts, pts, radius_fwd_body, &c);
}

/* Backward with membership held fixed (Section 5: radius cutoff membership is
 * discrete and not differentiated).  With k_ij = exp(-|p_i-p_j|^2/sigma^2)
 * and the loss L = sum_i <dy_i, y_i>:
 *   dx_j = sum_{i : j in N(i)} k_ij dy_i = sum_{i in N(j)} k_ij dy_i
 *          (the relation and the weight are symmetric in i, j),
 *   dp_i = sum_{j in N(i)} (2 k_ij / sigma^2) (p_j - p_i) (<dy_i, x_j> + <dy_j, x_i>)
 *          (p_i enters k_ij as destination and k_ji as source; dk/dp_i =
 *          (2k/sigma^2)(p_j - p_i) in both). */
static void radius_bwd_body(void *vctx, int64_t k, int64_t i, const int64_t *nb, int64_t cnt) {
    radius_ctx *c = (radius_ctx *)vctx;
    const int32_t F = c->F;
    const float *pi = c->pos + i * 3;
    if (c->dx) {
        for (int32_t f = 0; f < F; ++f) {
            c->dx[k * F + f] = 0.0;
            if (c->dxabs) c->dxabs[k * F + f] = 0.0;
        }
    }
    double gp[3] = {0, 0, 0}, ga[3] = {0, 0, 0};
    for (int64_t t = 0; t < cnt; ++t) {
        int64_t j = nb[t];
        double d[3];
        double kw = kernel_weight(pi, c->pos + j * 3, c->inv_s2, d);
        if (c->dx) {
            for (int32_t f = 0; f < F; ++f) {
                double term = kw * (double)c->dy[j * F + f];
                c->dx[k * F + f] += term;
                if (c->dxabs) c->dxabs[k * F + f] += fabs(term);
            }
        }
        if (c->dp) {
            double s = 0.0, sa = 0.0;
            for (int32_t f = 0; f < F; ++f) {
                double a = (double)c->dy[i * F + f] * (double)c->x[j * F + f];
                double b = (double)c->dy[j * F + f] * (double)c->x[i * F + f];
                s += a + b;
                sa += fabs(a) + fabs(b);
            }
            double coef = 2.0 * kw * c->inv_s2;
            for (int a = 0; a < 3; ++a) {
                gp[a] += coef * d[a] * s;
                ga[a] += fabs(coef * d[a]) * sa;
            }
        }
    }
    if (c->dp)
        for (int a = 0; a < 3; ++a) {
            c->dp[k * 3 + a] = gp[a];
            if (c->dpabs) c->dpabs[k * 3 + a] = ga[a];
        }
}

int tiga_oracle_radius_bwd(int64_t n, int32_t F, const float *pos, const float *x,
                           const float *dy, float radius, float sigma, int64_t npts,
                           const int64_t *pts, double *dx, double *dxabs, double *dp,
                           double *dpabs) {
    radius_ctx c;
    memset(&c, 0, sizeof c);
    c.F = F;
    c.pos = pos;
    c.x = x;
    c.dy = dy;
    c.inv_s2 = 1.0 / ((double)sigma * (double)sigma);
    c.dx = dx;
    c.dxabs = dxabs;
    c.dp = dp;
    c.dpabs = dpabs;
    return for_each_point(n, pos, radius, npts, pts, radius_bwd_body, &c);
}

typedef struct {
    int64_t *ptr;
    int32_t *idx;
    int32_t *count;
} nbr_ctx;

static void nbr_body(void *vctx, int64_t k, int64_t i, const int64_t *nb, int64_t cnt) {
    nbr_ctx *c = (nbr_ctx *)vctx;
    (void)i;
    if (c->count) c->count[k] = (int32_t)cnt;
    if (c->idx)
        for (int64_t t = 0; t < cnt; ++t) c->idx[c->ptr[k] + t] = (int32_t)nb[t];
}

/* Accepted neighbour lists, ascending per point.  Call once with idx == NULL
 * to obtain counts, then with ptr (exclusive prefix of counts) and idx. */
int tiga_oracle_radius_neighbors(int64_t n, const float *pos, float radius, int64_t npts,
                                 const int64_t *pts, int32_t *count, const int64_t *ptr,
                                 int32_t *idx) {
    nbr_ctx c = {(int64_t *)ptr, idx, count};
    return for_each_point(n, pos, radius, npts, pts, nbr_body, &c);
}

/* ------------------------------------------------------------------------ */
/* Dense all-pairs relation (no edge array; Section 1: a dense relation may  */
/* need no edge array)                                                       */
/* ------------------------------------------------------------------------ */

/* Softened inverse-square message summed over all j != i:
 *   y_i = sum_{j != i} q_j (p_j - p_i) / (|p_j - p_i|^2 + eps^2)^(3/2).
 * The softening constant is given as the fp32 value eps; its square enters as
 * the fp32 product eps*eps (one rounding), the constant a single-precision
 * implementation of the message is handed.  Everything else is fp64. */
void tiga_oracle_dense_fwd(int64_t n, const float *pos, const float *q, float eps,
                           int64_t npts, const int64_t *pts, double *y, double *yabs) {
    const float e2f = eps * eps;
    const double e2 = (double)e2f;
    int64_t k;
#pragma omp parallel for schedule(dynamic, 16)
    for (k = 0; k < npts; ++k) {
        int64_t i = pts ? pts[k] : k;
        double acc[3] = {0, 0, 0}, mag[3] = {0, 0, 0};
        for (int64_t j = 0; j < n; ++j) {
            if (j == i) continue;
            double d[3];
            for (int a = 0; a < 3; ++a) d[a] = (double)pos[j * 3 + a] - (double)pos[i * 3 + a];
            double s = d[0] * d[0] + d[1] * d[1] + d[2] * d[2] + e2;
            double coef = (double)q[j] / (s * sqrt(s));
            for (int a = 0; a < 3; ++a) {
                acc[a] += coef * d[a];
                mag[a] += fabs(coef * d[a]);
            }
        }
        for (int a = 0; a < 3; ++a) {
            y[k * 3 + a] = acc[a];
            if (yabs) yabs[k * 3 + a] = mag[a];
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Online-softmax reducer over an implicit triangular or dense relation      */
/* (Section 5.2, online softmax; appendix "Causal attention as message       */
/* passing")                                                                 */
/* ------------------------------------------------------------------------ */

/* IEEE 754 binary16: sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Every value is exactly representable in double. */
double tiga_oracle_f16_to_double(uint16_t h) {
    int s = h >> 15, e = (h >> 10) & 31, f = h & 1023;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);            /* subnormal: f * 2^-24 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25); /* (1 + f / 2^10) * 2^(e - 15) */
    return s ? -v : v;
}

/* bfloat16: the upper 16 bits of an IEEE 754 binary32. */
double tiga_oracle_bf16_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float x;
    memcpy(&x, &u, sizeof x);
    return (double)x;
}

/* Attention as message passing, one head at a time.  Destination i supplies the
 * query q_i, source j the key k_j and value v_j; the relation is
 *   triangular (relation 0):  N(i) = {0, ..., i}   (the diagonal is included)
 *   dense      (relation 1):  N(i) = {0, ..., n-1}
 * the message is the pair (score s_ij = scale * <q_i, k_j>, value v_j), and the
 * online-softmax reducer finalizes to
 *   y_i = sum_{j in N(i)} exp(s_ij) v_j / sum_{j in N(i)} exp(s_ij).
 * The sums are evaluated after subtracting the row maximum of the scores, which
 * changes nothing mathematically.  Inputs are [H][n][D] bit patterns (dtype 0 =
 * binary16, 1 = bfloat16), widened exactly to double; all arithmetic is fp64.
 * For each requested query row pts[k] (all rows if pts == NULL) and head h:
 *   y   [k][h][d] = y_i,
 *   yabs[k][h][d] = sum_j p_ij |v_jd| with p_ij the normalized weights,
 *   lse [k][h]    = log sum_{j in N(i)} exp(s_ij).
 * yabs and lse may be NULL.  Returns 0, or -1 for an unknown dtype/relation. */
int tiga_oracle_attention_fwd(int64_t n, int32_t H, int32_t D, int dtype, const uint16_t *q,
                              const uint16_t *k, const uint16_t *v, double scale, int relation,
                              int64_t npts, const int64_t *pts, double *y, double *yabs, double *lse) {
    if ((dtype != 0 && dtype != 1) || (relation != 0 && relation != 1)) return -1;
    double (*cvt)(uint16_t) = dtype == 0 ? tiga_oracle_f16_to_double : tiga_oracle_bf16_to_double;
    int64_t t;
#pragma omp parallel for schedule(dynamic, 1)
    for (t = 0; t < npts * H; ++t) {
        int64_t kk = t / H, h = t % H;
        int64_t i = pts ? pts[kk] : kk;
        int64_t last = relation == 0 ? i : n - 1;       /* N(i) = {0, ..., last} */
        const uint16_t *qi = q + (h * n + i) * D;
        double *out = y + (kk * H + h) * D;
        double *mag = yabs ? yabs + (kk * H + h) * D : NULL;
        double mx = -INFINITY, den = 0.0;
        for (int64_t j = 0; j <= last; ++j) {          /* pass 1: the row maximum */
            const uint16_t *kj = k + (h * n + j) * D;
            double s = 0.0;
            for (int d = 0; d < D; ++d) s += cvt(qi[d]) * cvt(kj[d]);
            s *= scale;
            if (s > mx) mx = s;
        }
        for (int d = 0; d < D; ++d) {
            out[d] = 0.0;
            if (mag) mag[d] = 0.0;
        }
        for (int64_t j = 0; j <= last; ++j) {          /* pass 2: weights and sums */
            const uint16_t *kj = k + (h * n + j) * D;
            const uint16_t *vj = v + (h * n + j) * D;
            double s = 0.0;
            for (int d = 0; d < D; ++d) s += cvt(qi[d]) * cvt(kj[d]);
            s *= scale;
            double p = exp(s - mx);
            den += p;
            for (int d = 0; d < D; ++d) {
                out[d] += p * cvt(vj[d]);
                if (mag) mag[d] += p * fabs(cvt(vj[d]));
            }
        }
        for (int d = 0; d < D; ++d) {
            out[d] /= den;
            if (mag) mag[d] /= den;
        }
        if (lse) lse[kk * H + h] = mx + log(den);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Generated exact kNN relation (Section 4.9, generated relations; the      */
/* exact-kNN workload of Section 7)                                         */
/* ------------------------------------------------------------------------ */

/* Squared distance in fp32 from direct differences, no contraction:
 *   d2 = fl(fl(fl(dx*dx) + fl(dy*dy)) + fl(dz*dz)),  dx = fl(p_j.x - p_i.x), ... */
static float knn_d2(const float *pi, const float *pj) {
    float dx = pj[0] - pi[0], dy = pj[1] - pi[1], dz = pj[2] - pi[2];
    float sx = dx * dx, sy = dy * dy, sz = dz * dz;
    float s = sx + sy;
    return s + sz;
}

/* Exact k nearest neighbours over one point set, self excluded.  Source j is
 * ranked by the key (d2_ij, j) in lexicographic order (a distance tie keeps the
 * lower index); a key with a non-finite d2 is never selected.  S_i holds the k
 * smallest keys (fewer if fewer sources have a finite d2).  For each requested
 * query pts[k'] (all points if pts == NULL):
 *   nbr [k'][t] = the t-th selected source in key order, -1 past |S_i|  (may be NULL)
 *   y   [k'][f] = sum_{j in S_i} x[j][f]       (fp64; x == NULL or F == 0 skips y)
 *   yabs[k'][f] = sum_{j in S_i} |x[j][f]|     (may be NULL)
 * Returns 0, or -1 if a scratch allocation fails. */
int tiga_oracle_knn(int64_t n, int32_t F, const float *pos, const float *x, int32_t k, int64_t npts,
                    const int64_t *pts, int32_t *nbr, double *y, double *yabs) {
    int fail = 0;
    int64_t q;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : fail)
    for (q = 0; q < npts; ++q) {
        int64_t i = pts ? pts[q] : q;
        float *bd = (float *)malloc(sizeof(float) * (size_t)(k > 0 ? k : 1));
        int64_t *bj = (int64_t *)malloc(sizeof(int64_t) * (size_t)(k > 0 ? k : 1));
        if (!bd || !bj) {
            free(bd);
            free(bj);
            fail = 1;
            continue;
        }
        int cnt = 0;
        for (int64_t j = 0; j < n && k > 0; ++j) {
            if (j == i) continue;
            float d2 = knn_d2(pos + i * 3, pos + j * 3);
            if (!isfinite(d2)) continue;
            /* j grows, so among equal distances the retained (lower) index stays first:
             * the new key goes after every retained key with d2 <= its own */
            if (cnt == k && !(d2 < bd[k - 1])) continue;
            int at = cnt < k ? cnt : k - 1;
            while (at > 0 && d2 < bd[at - 1]) {
                bd[at] = bd[at - 1];
                bj[at] = bj[at - 1];
                --at;
            }
            bd[at] = d2;
            bj[at] = j;
            if (cnt < k) ++cnt;
        }
        if (nbr)
            for (int t = 0; t < k; ++t) nbr[q * k + t] = t < cnt ? (int32_t)bj[t] : -1;
        if (y && x)
            for (int f = 0; f < F; ++f) {
                double acc = 0.0, mag = 0.0;
                for (int t = 0; t < cnt; ++t) {
                    acc += (double)x[bj[t] * F + f];
                    mag += fabs((double)x[bj[t] * F + f]);
                }
                y[q * F + f] = acc;
                if (yabs) yabs[q * F + f] = mag;
            }
        free(bd);
        free(bj);
    }
    return fail ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Edge-local MLP message over a given relation (appendix "A differentiable */
/* EdgeNN example"; Section 5 for the vector-Jacobian product)              */
/* ------------------------------------------------------------------------ */

/* For the destination-major relation (ptr, idx) -- row i lists the sources j of
 * destination i -- with the message
 *   in_ij = [p_j - p_i ; x_j]                       (3 + F values, fp64)
 *   a_ij  = W1 in_ij + b1,  r_ij = max(a_ij, 0)     (H values)
 *   m_ij  = W2 r_ij + b2                            (O values; the final bias is
 *                                                    part of every message)
 *   y_i   = sum_{j in row i} m_ij                   (an empty row gives 0)
 * W1 is [H][3 + F], b1 [H], W2 [O][H], b2 [O], all fp32 row-major.  If dy
 * ([n][O], fp32) is given, the gradients of L = sum_i <dy_i, y_i> with the
 * relation held fixed are formed as well:
 *   dm = dy_i;  dW2 += dm r^T;  db2 += dm;  da = (W2^T dm) * [a > 0];
 *   dW1 += da in^T;  db1 += da;  din = W1^T da;
 *   dp_j += din[0..3);  dp_i -= din[0..3);  dx_j += din[3..3+F).
 * The derivative of max(a, 0) at a = 0 is taken as 0.  Serial over
 * destinations in ascending order; all arithmetic fp64.
 *
 * Outputs come as three arrays of seven pointers, in the order
 *   y [n][O], dx [n][F], dp [n][3], dW1 [H][3+F], db1 [H], dW2 [O][H], db2 [O]
 * (any pointer, or the whole mag / slack array, may be NULL):
 *   val:   the values above;
 *   mag:   for every output, its absolute-value evaluation with this oracle's
 *          ReLU decisions held: every input, weight, bias and cotangent is
 *          replaced by its absolute value, the output of an active unit by the
 *          absolute-value evaluation of its pre-activation
 *          aa = |b1| + sum_c |W1[h][c]| |in_c|, and an inactive unit
 *          contributes nothing.  It bounds the rounding error of any fp32
 *          evaluation order, as the sum of |terms| does for a plain sum;
 *   slack: the absolute-value evaluation of what reaches the output through
 *          units whose ReLU decision fp32 cannot settle, |a| <= 2^-14 aa (an
 *          fp32 evaluation of a with up to 3 + F + 1 roundings is off by at
 *          most about 2^-17 aa), taken as if the unit were active.  A unit's
 *          decision flipping changes an output by at most its slack. */
enum { EN_Y, EN_DX, EN_DP, EN_DW1, EN_DB1, EN_DW2, EN_DB2, EN_OUTS };

static void en_zero(double *p, int64_t count) {
    if (p) memset(p, 0, sizeof(double) * (size_t)count);
}

void tiga_oracle_edgenn(int64_t n, int32_t F, int32_t H, int32_t O, const float *pos, const float *x,
                        const int64_t *ptr, const int32_t *idx, const float *W1, const float *b1,
                        const float *W2, const float *b2, const float *dy, double *const *val,
                        double *const *mag, double *const *slack) {
    const int32_t D = 3 + F;
    const double unsettled = ldexp(1.0, -14);
    const int64_t sizes[EN_OUTS] = {n * O, n * F, n * 3, (int64_t)H * D, H, (int64_t)O * H, O};
    double *v[EN_OUTS], *m[EN_OUTS], *sl[EN_OUTS];
    for (int k = 0; k < EN_OUTS; ++k) {
        v[k] = val ? val[k] : NULL;
        m[k] = mag ? mag[k] : NULL;
        sl[k] = slack ? slack[k] : NULL;
        en_zero(v[k], sizes[k]);
        en_zero(m[k], sizes[k]);
        en_zero(sl[k], sizes[k]);
    }
    double *in = (double *)malloc(sizeof(double) * (size_t)D);
    double *ina = (double *)malloc(sizeof(double) * (size_t)D);
    double *a = (double *)malloc(sizeof(double) * (size_t)H);
    double *aa = (double *)malloc(sizeof(double) * (size_t)H);
    double *da = (double *)malloc(sizeof(double) * (size_t)H);
    double *ga = (double *)malloc(sizeof(double) * (size_t)H);
    for (int64_t i = 0; i < n; ++i) {
        for (int64_t e = ptr[i]; e < ptr[i + 1]; ++e) {
            const int64_t j = idx[e];
            for (int c = 0; c < 3; ++c) in[c] = (double)pos[j * 3 + c] - (double)pos[i * 3 + c];
            for (int c = 0; c < F; ++c) in[3 + c] = (double)x[j * F + c];
            for (int c = 0; c < D; ++c) ina[c] = fabs(in[c]);
            for (int h = 0; h < H; ++h) {
                double s = (double)b1[h], sa = fabs((double)b1[h]);
                for (int c = 0; c < D; ++c) {
                    s += (double)W1[h * D + c] * in[c];
                    sa += fabs((double)W1[h * D + c]) * ina[c];
                }
                a[h] = s;
                aa[h] = sa;
            }
#define ACTIVE(h) (a[h] > 0.0)
#define UNSETTLED(h) (fabs(a[h]) <= unsettled * aa[h])
            /* forward */
            for (int o = 0; o < O; ++o) {
                double s = (double)b2[o], sa = fabs((double)b2[o]), su = 0.0;
                for (int h = 0; h < H; ++h) {
                    const double w2 = (double)W2[o * H + h];
                    s += w2 * (ACTIVE(h) ? a[h] : 0.0);
                    sa += fabs(w2) * (ACTIVE(h) ? aa[h] : 0.0);
                    if (UNSETTLED(h)) su += fabs(w2) * aa[h];
                }
                if (v[EN_Y]) v[EN_Y][i * O + o] += s;
                if (m[EN_Y]) m[EN_Y][i * O + o] += sa;
                if (sl[EN_Y]) sl[EN_Y][i * O + o] += su;
            }
            if (!dy) continue;
            const float *dm = dy + i * O;
            for (int o = 0; o < O; ++o) {
                const double g = (double)dm[o], gabs = fabs(g);
                for (int h = 0; h < H; ++h) {
                    if (v[EN_DW2]) v[EN_DW2][o * H + h] += g * (ACTIVE(h) ? a[h] : 0.0);
                    if (m[EN_DW2]) m[EN_DW2][o * H + h] += gabs * (ACTIVE(h) ? aa[h] : 0.0);
                    if (sl[EN_DW2] && UNSETTLED(h)) sl[EN_DW2][o * H + h] += gabs * aa[h];
                }
                if (v[EN_DB2]) v[EN_DB2][o] += g;
                if (m[EN_DB2]) m[EN_DB2][o] += gabs;
            }
            for (int h = 0; h < H; ++h) {
                double s = 0.0, sa = 0.0;
                for (int o = 0; o < O; ++o) {
                    s += (double)W2[o * H + h] * (double)dm[o];
                    sa += fabs((double)W2[o * H + h]) * fabs((double)dm[o]);
                }
                da[h] = ACTIVE(h) ? s : 0.0;
                ga[h] = sa; /* the absolute-value evaluation of da, mask open */
                const double gm = ACTIVE(h) ? sa : 0.0, gu = UNSETTLED(h) ? sa : 0.0;
                if (v[EN_DB1]) v[EN_DB1][h] += da[h];
                if (m[EN_DB1]) m[EN_DB1][h] += gm;
                if (sl[EN_DB1]) sl[EN_DB1][h] += gu;
                for (int c = 0; c < D; ++c) {
                    if (v[EN_DW1]) v[EN_DW1][h * D + c] += da[h] * in[c];
                    if (m[EN_DW1]) m[EN_DW1][h * D + c] += gm * ina[c];
                    if (sl[EN_DW1]) sl[EN_DW1][h * D + c] += gu * ina[c];
                }
            }
            for (int c = 0; c < D; ++c) {
                double s = 0.0, sa = 0.0, su = 0.0;
                for (int h = 0; h < H; ++h) {
                    const double w1 = (double)W1[h * D + c];
                    s += w1 * da[h];
                    sa += fabs(w1) * (ACTIVE(h) ? ga[h] : 0.0);
                    if (UNSETTLED(h)) su += fabs(w1) * ga[h];
                }
                if (c < 3) {
                    if (v[EN_DP]) {
                        v[EN_DP][j * 3 + c] += s;
                        v[EN_DP][i * 3 + c] -= s;
                    }
                    if (m[EN_DP]) {
                        m[EN_DP][j * 3 + c] += sa;
                        m[EN_DP][i * 3 + c] += sa;
                    }
                    if (sl[EN_DP]) {
                        sl[EN_DP][j * 3 + c] += su;
                        sl[EN_DP][i * 3 + c] += su;
                    }
                } else {
                    if (v[EN_DX]) v[EN_DX][j * F + (c - 3)] += s;
                    if (m[EN_DX]) m[EN_DX][j * F + (c - 3)] += sa;
                    if (sl[EN_DX]) sl[EN_DX][j * F + (c - 3)] += su;
                }
            }
#undef ACTIVE
#undef UNSETTLED
        }
    }
    free(in);
    free(ina);
    free(a);
    free(aa);
    free(da);
    free(ga);
}
