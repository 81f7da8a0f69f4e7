/*
 * ks_oracle.c -- reference CPU implementation of Kronecker-sparse (KS)
 * matrix multiplication, in double precision.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header or table with the HIP path.
 *
 * What it computes (paper, Section 1 "Scope of this work" and Definition 2.1):
 *   K is an (a*b*d) x (a*c*d) matrix whose support lies in
 *   I_a (x) 1_{b x c} (x) I_d, and the product is  Y = X K^T  for a batch
 *   X of B row vectors of length N = a*c*d, giving Y of B rows of length
 *   M = a*b*d.
 *
 * The nonzeros of K are passed packed, one dense b x c block per (i, j) in
 * [a] x [d], stored as Kv[(i*d + j)][k][l] (row-major (a*d, b, c)); this is the
 * pre-permuted "(ad, b, c)" storage of the batched-GEMM baseline (paper,
 * Appendix A.1, and Table 1).  The block (i, j) holds the entries of K on the
 * rows  i*b*d + k*d + j  (k < b)  and the columns  i*c*d + l*d + j  (l < c)
 * (paper, Section 4.1, the row/col index sets of Algorithm 2).
 *
 * Because those row sets partition [M] and the column sets partition [N]
 * (Section 4.1), every entry of K off these positions is zero, so the plain
 * definition  Y[beta, m] = sum_n K[m, n] X[beta, n]  reduces, for
 * m = i*b*d + k*d + j, to
 *      Y[beta, m] = sum_{l < c} Kv[i*d+j][k][l] * X[beta, i*c*d + l*d + j].
 * This file evaluates exactly that sum, in fp64, in ascending l.
 *
 * Layouts (paper, Section 2.2):  batch-size-first (BSF): X is (B, N) and Y is
 * (B, M), row-major;  batch-size-last (BSL): X is (N, B) and Y is (M, B),
 * row-major.  The layout only changes the index arithmetic.
 *
 * Chains (paper, Section 1 and Appendix B.1, Table 5): W = K_1 K_2 ... K_L and
 * Y = X W^T = (((X K_L^T) K_{L-1}^T) ... ) K_1^T, i.e. K_L is applied first.
 * Intermediates are kept in fp64.
 *
 * Build: a plain C compiler with OpenMP, e.g.
 *   gcc -O2 -fopenmp -fPIC -shared ks_oracle.c -o libks_oracle.so
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define KSO_BSF 0
#define KSO_BSL 1

/* Index of logical element (beta, n) of a (rows = batch) x (cols = width)
 * matrix stored in the given layout. */
static int64_t kso_index(int layout, int64_t beta, int64_t n, int64_t batch, int64_t width)
{
    if (layout == KSO_BSF)
        return beta * width + n;
    return n * batch + beta;
}

/* Number of OpenMP threads the oracle will use (0 when built without OpenMP
 * reports 1). */
int kso_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Y = X K^T for one KS factor (pattern (a,b,c,d)).
 *   Kv : a*d*b*c doubles, packed as described above.
 *   X  : batch*a*c*d doubles in `layout`.
 *   Y  : batch*a*b*d doubles in `layout` (overwritten).
 *   nthreads <= 0 means "use the OpenMP default".
 * Returns 0, or -1 on an invalid argument.
 */
int kso_matmul(int64_t a, int64_t b, int64_t c, int64_t d,
               const double *Kv, const double *X, double *Y,
               int64_t batch, int layout, int nthreads)
{
    if (a < 1 || b < 1 || c < 1 || d < 1 || batch < 0)
        return -1;
    if (layout != KSO_BSF && layout != KSO_BSL)
        return -1;
    const int64_t N = a * c * d;
    const int64_t M = a * b * d;
    (void)nthreads;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#endif
    /* One task per (i, j, beta); every output of a task is computed as the
     * plain sum over l. */
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t ij = 0; ij < a * d; ++ij) {
        for (int64_t beta = 0; beta < batch; ++beta) {
            const int64_t i = ij / d;
            const int64_t j = ij % d;
            const double *block = Kv + ij * b * c;
            for (int64_t k = 0; k < b; ++k) {
                double acc = 0.0;
                for (int64_t l = 0; l < c; ++l) {
                    const int64_t n = i * c * d + l * d + j;
                    acc += block[k * c + l] * X[kso_index(layout, beta, n, batch, N)];
                }
                const int64_t m = i * b * d + k * d + j;
                Y[kso_index(layout, beta, m, batch, M)] = acc;
            }
        }
    }
    return 0;
}

/*
 * Selected entries of Y = X K^T: out[t] = Y[beta[t], m[t]], computed one by
 * one from the definition (used to check very large outputs on a sample).
 */
int kso_entries(int64_t a, int64_t b, int64_t c, int64_t d,
                const double *Kv, const double *X, int64_t batch, int layout,
                const int64_t *beta, const int64_t *m, int64_t count, double *out)
{
    if (a < 1 || b < 1 || c < 1 || d < 1 || batch < 0)
        return -1;
    if (layout != KSO_BSF && layout != KSO_BSL)
        return -1;
    const int64_t N = a * c * d;
    const int64_t M = a * b * d;
    for (int64_t t = 0; t < count; ++t) {
        if (beta[t] < 0 || beta[t] >= batch || m[t] < 0 || m[t] >= M)
            return -1;
    }
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < count; ++t) {
        /* m = i*b*d + k*d + j with k < b, j < d */
        const int64_t i = m[t] / (b * d);
        const int64_t k = (m[t] % (b * d)) / d;
        const int64_t j = m[t] % d;
        const double *block = Kv + (i * d + j) * b * c;
        double acc = 0.0;
        for (int64_t l = 0; l < c; ++l) {
            const int64_t n = i * c * d + l * d + j;
            acc += block[k * c + l] * X[kso_index(layout, beta[t], n, batch, N)];
        }
        out[t] = acc;
    }
    return 0;
}

/*
 * Materialise the dense (a*b*d) x (a*c*d) matrix K from its packed values,
 * row-major.  Entries off the KS support are set to zero.
 */
int kso_dense(int64_t a, int64_t b, int64_t c, int64_t d, const double *Kv, double *K)
{
    if (a < 1 || b < 1 || c < 1 || d < 1)
        return -1;
    const int64_t N = a * c * d;
    const int64_t M = a * b * d;
    memset(K, 0, (size_t)(M * N) * sizeof(double));
    for (int64_t i = 0; i < a; ++i)
        for (int64_t j = 0; j < d; ++j)
            for (int64_t k = 0; k < b; ++k)
                for (int64_t l = 0; l < c; ++l)
                    K[(i * b * d + k * d + j) * N + (i * c * d + l * d + j)] =
                        Kv[((i * d + j) * b + k) * c + l];
    return 0;
}

/*
 * Chain: Y = X (K_1 K_2 ... K_L)^T with factor f = 0 .. L-1 holding K_{f+1}.
 * pat holds 4*L integers (a,b,c,d per factor, in product order) and Kvs the L
 * packed value arrays.  Consecutive factors must satisfy
 *   a_f c_f d_f == a_{f+1} b_{f+1} d_{f+1}
 * (Appendix B.1, Table 5, deformable-butterfly row).  K_L is applied first;
 * intermediates are fp64.  Returns 0, or -1 on an invalid argument.
 */
int kso_chain(int nfactors, const int64_t *pat, const double *const *Kvs,
              const double *X, double *Y, int64_t batch, int layout, int nthreads)
{
    if (nfactors < 1 || batch < 0)
        return -1;
    for (int f = 0; f + 1 < nfactors; ++f) {
        const int64_t *p = pat + 4 * f, *q = pat + 4 * (f + 1);
        if (p[0] * p[2] * p[3] != q[0] * q[1] * q[3])
            return -2;
    }
    int64_t width_max = 0;
    for (int f = 0; f < nfactors; ++f) {
        const int64_t *p = pat + 4 * f;
        if (p[0] * p[1] * p[3] > width_max) width_max = p[0] * p[1] * p[3];
        if (p[0] * p[2] * p[3] > width_max) width_max = p[0] * p[2] * p[3];
    }
    double *cur = NULL, *nxt = NULL;
    if (nfactors > 1) {
        cur = (double *)malloc((size_t)(width_max * (batch > 0 ? batch : 1)) * sizeof(double));
        nxt = (double *)malloc((size_t)(width_max * (batch > 0 ? batch : 1)) * sizeof(double));
        if (!cur || !nxt) { free(cur); free(nxt); return -1; }
    }
    const double *in = X;
    int rc = 0;
    for (int f = nfactors - 1; f >= 0 && rc == 0; --f) {
        const int64_t *p = pat + 4 * f;
        double *out = (f == 0) ? Y : nxt;
        rc = kso_matmul(p[0], p[1], p[2], p[3], Kvs[f], in, out, batch, layout, nthreads);
        if (f != 0) {
            double *t = cur; cur = nxt; nxt = t;
            in = cur;
        }
    }
    free(cur);
    free(nxt);
    return rc;
}

/*
 * Output epilogue of a Transformer MLP layer built from a KS factor (paper
 * appendix, ViT-S/16 submodule table: "Linear + bias" rows, and the
 * feed-forward block Linear + GELU): in place on Y (batch x M in `layout`),
 *     Y[beta, m] = act(Y[beta, m] + bias[m]),
 * with bias NULL for no bias, act 0 for none and 1 for the exact GELU
 * x * Phi(x) = 0.5 * x * (1 + erf(x / sqrt(2))).  fp64.
 */
int kso_bias_act(double *Y, const double *bias, int64_t M, int64_t batch, int layout, int act)
{
    if (M < 1 || batch < 0 || (act != 0 && act != 1))
        return -1;
    if (layout != KSO_BSF && layout != KSO_BSL)
        return -1;
    for (int64_t beta = 0; beta < batch; ++beta) {
        for (int64_t m = 0; m < M; ++m) {
            double *y = &Y[kso_index(layout, beta, m, batch, M)];
            double v = *y + (bias ? bias[m] : 0.0);
            if (act == 1)
                v = 0.5 * v * (1.0 + erf(v / sqrt(2.0)));
            *y = v;
        }
    }
    return 0;
}
