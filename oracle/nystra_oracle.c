/*
 * PnP-Nystra float64 CPU oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code, header, table or helper with the
 * HIP library under paper_2506_08520_amd/, and it is deliberately plain:
 * straight loops in float64, one (window, head) unit at a time, in the order
 * the paper states the method, with no blocking, fusion or re-association.
 *
 * Paper: "Plug-and-Play Linear Attention with Provable Guarantees for
 * Training-Free Image Restoration" (PnP-Nystra).  Citations name its
 * sections, equations and Algorithm 1.
 *
 * Readings taken where the paper is silent (each is listed in the design doc):
 *  - softmax scale: 1/sqrt(d_h) per head unless the caller passes one (Sec. 1
 *    writes 1/sqrt(d); with h heads each head attends in d_h = d/h dims).
 *  - landmark pooling (Sec. 2.2, "average pooling over non-overlapping
 *    windows"): mode 0 = 2-D patches of the sqrt(N) x sqrt(N) token window,
 *    mode 1 = contiguous 1-D token segments.  See oracle_geometry().
 *  - pseudo-inverse (Sec. 2.2, Step 4): the iteration of Razavi et al. 2014,
 *    Z <- Z (13I - AZ(15I - AZ(7I - AZ))) / 4, started from
 *    Z_0 = A^T / (||A||_1 ||A||_inf) computed per unit.
 *  - the matrix that is pseudo-inverted is the normalised core block G_A^n
 *    (Sec. 2.2 stabilised form, Eq. (8)), whose rows are divided by the row
 *    maxima m_U taken over the G_U rows.
 *  - no epsilon and no clamp in the final row-wise division (Step 7).
 *
 * Parity status of each function is stated in its comment and in the design doc.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_EARG 1
#define ORC_EGEOM 2
#define ORC_ENOMEM 3

/* ------------------------------------------------------------------------ */
/* Landmark geometry (Sec. 2.2: landmarks are averages over non-overlapping  */
/* windows of tokens).                                                        */
/*                                                                            */
/* mode 0 (2-D): the N tokens form a w x w window in row-major order         */
/*   (w = sqrt(N)).  The m landmarks form a g_r x g_c grid of equal patches. */
/*   g_c is the largest divisor of m with g_c * g_c <= m such that both g_c  */
/*   and g_r = m / g_c divide w.  A patch is (w/g_r) rows x (w/g_c) columns. */
/*   For square m this is ordinary 2-D average pooling.                       */
/* mode 1 (1-D): m contiguous segments of N/m tokens (requires m | N).       */
/* Landmarks are numbered row-major over the patch grid.                      */
/* out[0..4] = rows, cols, patch_rows, patch_cols, grid_cols.                 */
/* Parity: pinned by hand-written maps (tests/golden) and by torch's         */
/* avg_pool2d / avg_pool1d on the pooled means.                               */
/* ------------------------------------------------------------------------ */
int oracle_geometry(int N, int m, int mode, int *out)
{
    if (N < 1 || m < 1 || m > N || out == NULL)
        return ORC_EARG;
    if (mode == 0) {
        int w = 0;
        while ((w + 1) * (w + 1) <= N)
            ++w;
        if (w * w != N)
            return ORC_EGEOM;
        int best = 0;
        for (int gc = 1; gc * gc <= m; ++gc) {
            if (m % gc != 0)
                continue;
            int gr = m / gc;
            if (w % gc == 0 && w % gr == 0)
                best = gc;
        }
        if (best == 0)
            return ORC_EGEOM;
        out[0] = w;
        out[1] = w;
        out[2] = w / (m / best);
        out[3] = w / best;
        out[4] = best;
        return ORC_OK;
    }
    if (mode == 1) {
        if (N % m != 0)
            return ORC_EGEOM;
        out[0] = 1;
        out[1] = N;
        out[2] = 1;
        out[3] = N / m;
        out[4] = m;
        return ORC_OK;
    }
    return ORC_EARG;
}

/* map[t] = landmark that token t is averaged into (Step 1). */
int oracle_landmark_map(int N, int m, int mode, int32_t *map)
{
    int g[5];
    int rc = oracle_geometry(N, m, mode, g);
    if (rc != ORC_OK)
        return rc;
    if (map == NULL)
        return ORC_EARG;
    for (int t = 0; t < N; ++t) {
        int r = t / g[1];
        int c = t % g[1];
        map[t] = (r / g[2]) * g[4] + (c / g[3]);
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Step 4: iterative pseudo-inverse of the m x m matrix A (row-major).       */
/* Z_0 = A^T / (||A||_1 ||A||_inf), then `iters` times                        */
/*   X = A Z;  Z <- 1/4 Z (13 I - X (15 I - X (7 I - X))).                    */
/* Parity: pinned by the residual identity E_{k+1} = 3/4 E_k^3 + 1/4 E_k^4    */
/* (E_k = I - A Z_k), by convergence to the LAPACK pseudo-inverse, and by    */
/* the symmetry of A Z_0.                                                      */
/* ------------------------------------------------------------------------ */
static void matmul(const double *A, const double *B, double *C, int n, int k, int p)
{
    /* C (n x p) = A (n x k) * B (k x p), all row-major. */
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < p; ++j) {
            double acc = 0.0;
            for (int q = 0; q < k; ++q)
                acc += A[i * k + q] * B[q * p + j];
            C[i * p + j] = acc;
        }
}

int oracle_pinv(const double *A, double *Z, int m, int iters)
{
    if (A == NULL || Z == NULL || m < 1 || iters < 0)
        return ORC_EARG;
    size_t mm = (size_t)m * m;
    double *X = malloc(mm * sizeof(double));
    double *Y = malloc(mm * sizeof(double));
    double *T = malloc(mm * sizeof(double));
    if (!X || !Y || !T) {
        free(X);
        free(Y);
        free(T);
        return ORC_ENOMEM;
    }
    double norm1 = 0.0, norminf = 0.0;
    for (int j = 0; j < m; ++j) {
        double s = 0.0;
        for (int i = 0; i < m; ++i)
            s += fabs(A[i * m + j]);
        if (s > norm1)
            norm1 = s;
    }
    for (int i = 0; i < m; ++i) {
        double s = 0.0;
        for (int j = 0; j < m; ++j)
            s += fabs(A[i * m + j]);
        if (s > norminf)
            norminf = s;
    }
    double a0 = 1.0 / (norm1 * norminf);
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < m; ++j)
            Z[i * m + j] = a0 * A[j * m + i];
    for (int it = 0; it < iters; ++it) {
        matmul(A, Z, X, m, m, m);                 /* X = A Z            */
        for (size_t e = 0; e < mm; ++e)           /* Y = 7I - X         */
            Y[e] = -X[e];
        for (int i = 0; i < m; ++i)
            Y[i * m + i] += 7.0;
        matmul(X, Y, T, m, m, m);                 /* T = X (7I - X)     */
        for (size_t e = 0; e < mm; ++e)           /* Y = 15I - T        */
            Y[e] = -T[e];
        for (int i = 0; i < m; ++i)
            Y[i * m + i] += 15.0;
        matmul(X, Y, T, m, m, m);                 /* T = X (15I - ...)  */
        for (size_t e = 0; e < mm; ++e)           /* Y = 13I - T        */
            Y[e] = -T[e];
        for (int i = 0; i < m; ++i)
            Y[i * m + i] += 13.0;
        matmul(Z, Y, T, m, m, m);                 /* T = Z (13I - ...)  */
        for (size_t e = 0; e < mm; ++e)
            Z[e] = 0.25 * T[e];
    }
    free(X);
    free(Y);
    free(T);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* One (window, head) unit of PnP-Nystra, Algorithm 1 computed in the        */
/* stabilised form of Eq. (8) (Sec. 2.2).                                     */
/*   Q, K, V: N x d row-major.  O: N x d.                                     */
/* Optional trace outputs (any may be NULL):                                  */
/*   Qbar, Kbar (m x d), mL (N), mU (m), GL (N x m), GU (m x N), GA (m x m),  */
/*   Z (m x m), P (N x m), ON (N x d), OD (N).                                */
/* ------------------------------------------------------------------------ */
typedef struct {
    double *Qbar, *Kbar, *mL, *mU, *GL, *GU, *GA, *Z, *P, *ON, *OD;
} unit_bufs;

static int unit_alloc(unit_bufs *b, int N, int d, int m)
{
    memset(b, 0, sizeof(*b));
    b->Qbar = malloc((size_t)m * d * sizeof(double));
    b->Kbar = malloc((size_t)m * d * sizeof(double));
    b->mL = malloc((size_t)N * sizeof(double));
    b->mU = malloc((size_t)m * sizeof(double));
    b->GL = malloc((size_t)N * m * sizeof(double));
    b->GU = malloc((size_t)m * N * sizeof(double));
    b->GA = malloc((size_t)m * m * sizeof(double));
    b->Z = malloc((size_t)m * m * sizeof(double));
    b->P = malloc((size_t)N * m * sizeof(double));
    b->ON = malloc((size_t)N * d * sizeof(double));
    b->OD = malloc((size_t)N * sizeof(double));
    if (!b->Qbar || !b->Kbar || !b->mL || !b->mU || !b->GL || !b->GU || !b->GA ||
        !b->Z || !b->P || !b->ON || !b->OD)
        return ORC_ENOMEM;
    return ORC_OK;
}

static void unit_free(unit_bufs *b)
{
    free(b->Qbar);
    free(b->Kbar);
    free(b->mL);
    free(b->mU);
    free(b->GL);
    free(b->GU);
    free(b->GA);
    free(b->Z);
    free(b->P);
    free(b->ON);
    free(b->OD);
}

static double dot(const double *a, const double *b, int d)
{
    double acc = 0.0;
    for (int k = 0; k < d; ++k)
        acc += a[k] * b[k];
    return acc;
}

/* Steps 1-7 for one unit into the buffers b; O receives the output. */
static int unit_compute(const double *Q, const double *K, const double *V, double *O,
                        int N, int d, int m, int iters, const int32_t *map,
                        double scale, unit_bufs *b)
{
    /* Step 1: landmarks = means of the tokens of each pooling window. */
    int *count = calloc((size_t)m, sizeof(int));
    if (!count)
        return ORC_ENOMEM;
    memset(b->Qbar, 0, (size_t)m * d * sizeof(double));
    memset(b->Kbar, 0, (size_t)m * d * sizeof(double));
    for (int t = 0; t < N; ++t) {
        int l = map[t];
        count[l] += 1;
        for (int k = 0; k < d; ++k) {
            b->Qbar[l * d + k] += Q[t * d + k];
            b->Kbar[l * d + k] += K[t * d + k];
        }
    }
    for (int l = 0; l < m; ++l)
        for (int k = 0; k < d; ++k) {
            b->Qbar[l * d + k] /= count[l];
            b->Kbar[l * d + k] /= count[l];
        }
    free(count);

    /* Step 3 with the row-max stabilisation of Sec. 2.2:
     *   m_L(i) = max_j (Q Kbar^T / sqrt d)_ij,  G_L^n = exp(. - m_L(i))
     *   m_U(i) = max_j (Qbar K^T / sqrt d)_ij,  G_U^n = exp(. - m_U(i))   */
    for (int i = 0; i < N; ++i) {
        double mx = -INFINITY;
        for (int j = 0; j < m; ++j) {
            double a = scale * dot(Q + (size_t)i * d, b->Kbar + (size_t)j * d, d);
            b->GL[i * m + j] = a;
            if (a > mx)
                mx = a;
        }
        b->mL[i] = mx;
        for (int j = 0; j < m; ++j)
            b->GL[i * m + j] = exp(b->GL[i * m + j] - mx);
    }
    for (int i = 0; i < m; ++i) {
        double mx = -INFINITY;
        for (int j = 0; j < N; ++j) {
            double a = scale * dot(b->Qbar + (size_t)i * d, K + (size_t)j * d, d);
            b->GU[(size_t)i * N + j] = a;
            if (a > mx)
                mx = a;
        }
        b->mU[i] = mx;
        for (int j = 0; j < N; ++j)
            b->GU[(size_t)i * N + j] = exp(b->GU[(size_t)i * N + j] - mx);
    }
    /* Step 2, normalised as G_A^n = M_U^{-1} G_A (rows divided by exp(m_U)). */
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < m; ++j)
            b->GA[i * m + j] =
                exp(scale * dot(b->Qbar + (size_t)i * d, b->Kbar + (size_t)j * d, d) - b->mU[i]);

    /* Step 4: Z ~ (G_A^n)^dagger. */
    int rc = oracle_pinv(b->GA, b->Z, m, iters);
    if (rc != ORC_OK)
        return rc;

    /* Step 5: premultiplier P = G_L^n Z (N x m). */
    matmul(b->GL, b->Z, b->P, N, m, m);

    /* Step 6: O_N = P (G_U^n V), O_D = P (G_U^n 1_N). */
    double *GUV = malloc((size_t)m * d * sizeof(double));
    double *GU1 = malloc((size_t)m * sizeof(double));
    if (!GUV || !GU1) {
        free(GUV);
        free(GU1);
        return ORC_ENOMEM;
    }
    matmul(b->GU, V, GUV, m, N, d);
    for (int i = 0; i < m; ++i) {
        double s = 0.0;
        for (int j = 0; j < N; ++j)
            s += b->GU[(size_t)i * N + j];
        GU1[i] = s;
    }
    matmul(b->P, GUV, b->ON, N, m, d);
    for (int i = 0; i < N; ++i) {
        double s = 0.0;
        for (int j = 0; j < m; ++j)
            s += b->P[i * m + j] * GU1[j];
        b->OD[i] = s;
    }
    free(GUV);
    free(GU1);

    /* Step 7: row-wise division. */
    for (int i = 0; i < N; ++i)
        for (int k = 0; k < d; ++k)
            O[(size_t)i * d + k] = b->ON[(size_t)i * d + k] / b->OD[i];
    return ORC_OK;
}

static void copy_opt(double *dst, const double *src, size_t n)
{
    if (dst)
        memcpy(dst, src, n * sizeof(double));
}

/* One unit with every intermediate exposed (NULL pointers are skipped). */
int oracle_unit_trace(const double *Q, const double *K, const double *V, double *O,
                      int N, int d, int m, int iters, int mode, double scale,
                      double *Qbar, double *Kbar, double *mL, double *mU,
                      double *GL, double *GU, double *GA, double *Z, double *P,
                      double *ON, double *OD)
{
    if (!Q || !K || !V || !O || d < 1 || iters < 0)
        return ORC_EARG;
    int32_t *map = malloc((size_t)N * sizeof(int32_t));
    if (!map)
        return ORC_ENOMEM;
    int rc = oracle_landmark_map(N, m, mode, map);
    if (rc != ORC_OK) {
        free(map);
        return rc;
    }
    unit_bufs b;
    rc = unit_alloc(&b, N, d, m);
    if (rc == ORC_OK)
        rc = unit_compute(Q, K, V, O, N, d, m, iters, map, scale, &b);
    if (rc == ORC_OK) {
        copy_opt(Qbar, b.Qbar, (size_t)m * d);
        copy_opt(Kbar, b.Kbar, (size_t)m * d);
        copy_opt(mL, b.mL, (size_t)N);
        copy_opt(mU, b.mU, (size_t)m);
        copy_opt(GL, b.GL, (size_t)N * m);
        copy_opt(GU, b.GU, (size_t)m * N);
        copy_opt(GA, b.GA, (size_t)m * m);
        copy_opt(Z, b.Z, (size_t)m * m);
        copy_opt(P, b.P, (size_t)N * m);
        copy_opt(ON, b.ON, (size_t)N * d);
        copy_opt(OD, b.OD, (size_t)N);
    }
    unit_free(&b);
    free(map);
    return rc;
}

/* Frobenius norm of the Step 4 residual I - A Z (A, Z: m x m, row-major). */
/* Parity: pinned by the residual recurrence E_{k+1} = 3/4 E_k^3 + 1/4 E_k^4 */
/* run from E_0 = I - A Z_0 (a derivation from the update, not the update).  */
static double residual_fro(const double *A, const double *Z, int m)
{
    double acc = 0.0;
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < m; ++j) {
            double x = (i == j) ? 1.0 : 0.0;
            for (int q = 0; q < m; ++q)
                x -= A[i * m + q] * Z[q * m + j];
            acc += x * x;
        }
    return sqrt(acc);
}

/* ------------------------------------------------------------------------ */
/* Batched forward over `units` independent (window, head) units laid out    */
/* contiguously as [units][N][d].  diag (optional, units x 3) receives per    */
/* unit the minimum and maximum of O_D and the Frobenius norm of the Step 4   */
/* residual I - G_A^n Z_K.  n_threads <= 0 uses the OpenMP default.  Returns  */
/* the first nonzero status of any unit.                                      */
/* ------------------------------------------------------------------------ */
int oracle_forward(const double *Q, const double *K, const double *V, double *O,
                   long units, int N, int d, int m, int iters, int mode, double scale,
                   int n_threads, double *diag)
{
    if (units < 0 || d < 1 || iters < 0)
        return ORC_EARG;
    if (units == 0)
        return ORC_OK;
    if (!Q || !K || !V || !O)
        return ORC_EARG;
    int32_t *map = malloc((size_t)N * sizeof(int32_t));
    if (!map)
        return ORC_ENOMEM;
    int rc = oracle_landmark_map(N, m, mode, map);
    if (rc != ORC_OK) {
        free(map);
        return rc;
    }
    int status = ORC_OK;
#ifdef _OPENMP
    if (n_threads <= 0)
        n_threads = omp_get_max_threads();
#pragma omp parallel num_threads(n_threads)
#endif
    {
        unit_bufs b;
        int lrc = unit_alloc(&b, N, d, m);
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (long u = 0; u < units; ++u) {
            if (lrc != ORC_OK)
                continue;
            size_t off = (size_t)u * N * d;
            int urc = unit_compute(Q + off, K + off, V + off, O + off, N, d, m, iters, map,
                                   scale, &b);
            if (urc != ORC_OK) {
                lrc = urc;
                continue;
            }
            if (diag) {
                double lo = INFINITY, hi = -INFINITY;
                for (int i = 0; i < N; ++i) {
                    if (b.OD[i] < lo)
                        lo = b.OD[i];
                    if (b.OD[i] > hi)
                        hi = b.OD[i];
                }
                diag[3 * u] = lo;
                diag[3 * u + 1] = hi;
                diag[3 * u + 2] = residual_fro(b.GA, b.Z, m);
            }
        }
        unit_free(&b);
        if (lrc != ORC_OK) {
#ifdef _OPENMP
#pragma omp critical
#endif
            if (status == ORC_OK)
                status = lrc;
        }
    }
    free(map);
    return status;
}

/* ------------------------------------------------------------------------ */
/* Exact softmax self-attention, Eq. (1), per unit, with the usual row-max   */
/* shift inside the softmax:  O = softmax(scale Q K^T) V.                     */
/* Parity: pinned against torch's scaled_dot_product_attention in float64.   */
/* ------------------------------------------------------------------------ */
int oracle_exact(const double *Q, const double *K, const double *V, double *O, long units,
                 int N, int d, double scale, int n_threads)
{
    if (units < 0 || N < 1 || d < 1)
        return ORC_EARG;
    if (units == 0)
        return ORC_OK;
    if (!Q || !K || !V || !O)
        return ORC_EARG;
    int status = ORC_OK;
#ifdef _OPENMP
    if (n_threads <= 0)
        n_threads = omp_get_max_threads();
#pragma omp parallel num_threads(n_threads)
#endif
    {
        double *row = malloc((size_t)N * sizeof(double));
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (long u = 0; u < units; ++u) {
            if (!row)
                continue;
            size_t off = (size_t)u * N * d;
            const double *q = Q + off, *k = K + off, *v = V + off;
            double *o = O + off;
            for (int i = 0; i < N; ++i) {
                double mx = -INFINITY;
                for (int j = 0; j < N; ++j) {
                    row[j] = scale * dot(q + (size_t)i * d, k + (size_t)j * d, d);
                    if (row[j] > mx)
                        mx = row[j];
                }
                double den = 0.0;
                for (int j = 0; j < N; ++j) {
                    row[j] = exp(row[j] - mx);
                    den += row[j];
                }
                for (int c = 0; c < d; ++c) {
                    double acc = 0.0;
                    for (int j = 0; j < N; ++j)
                        acc += row[j] * v[(size_t)j * d + c];
                    o[(size_t)i * d + c] = acc / den;
                }
            }
        }
        if (!row) {
#ifdef _OPENMP
#pragma omp critical
#endif
            status = ORC_ENOMEM;
        }
        free(row);
    }
    return status;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
