/*
 * Gram-Space oracle: plain, slow, fp64 reference of the operators.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links or calls
 * this file; only the test-suite, the smoke check and the CPU-baseline leg of
 * the benchmark load it.  It shares no code with the HIP path.
 *
 * Notation: the codebook is C (M rows of length D; row j is codebook vector
 * c_j, i.e. column j of the paper's W).  The orthonormal basis is Q (r rows of
 * length D, Q = U^T) and the Gram-loc coordinates are R (M x r, R = T^T), so
 * that C = R Q.  All matrices are dense row-major fp64.
 *
 * Every sum runs in index order, one scalar accumulator, no blocking.  The
 * only parallelism is over independent output rows (OpenMP), which leaves the
 * result bit-identical to a serial run.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

int gso_threads(void) { return omp_get_max_threads(); }
void gso_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }

/*
 * Gram-Space compression (Sec. 3.1, Eq. 1; rank = algebraic rank, Sec. 3.2;
 * finite-precision construction by Householder QR, Sec. 3.2).
 *
 * Householder QR of W = C^T with column skipping: codebook vectors are taken
 * in index order.  Vector i is transformed by the reflectors built so far; if
 * the part of it not yet spanned has norm rho <= tau * ||c_i|| it is
 * dependent (its coordinates are the first r transformed entries), otherwise
 * a new reflector maps that part onto +-rho e_r and the basis grows by one.
 * The sign of each basis vector is chosen so the pivot R[i, r] is +rho.
 *
 * Outputs: Q (capacity M x D, rows 0..r-1 written, the rest zeroed),
 *          R (M x M; R[i, k] for k < r, zeros elsewhere),
 *          kept[0..r-1] = index of the codebook vector that produced basis
 *          vector k, *rank = r.
 * Returns 0, or -1 on allocation failure.
 */
int gso_compress(const double *C, long M, long D, double tau,
                 double *Q, double *R, int *kept, int *rank)
{
    double *W = (double *)malloc(sizeof(double) * (size_t)M * (size_t)D);
    double *U = (double *)malloc(sizeof(double) * (size_t)M * (size_t)D);
    double *sgn = (double *)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1));
    if (!W || !U || !sgn) { free(W); free(U); free(sgn); return -1; }
    memcpy(W, C, sizeof(double) * (size_t)M * (size_t)D);
    memset(U, 0, sizeof(double) * (size_t)M * (size_t)D);
    memset(R, 0, sizeof(double) * (size_t)M * (size_t)M);
    memset(Q, 0, sizeof(double) * (size_t)M * (size_t)D);

    long r = 0;
    for (long i = 0; i < M; ++i) {
        const double *ci = C + i * D;
        double *w = W + i * D;
        double cn2 = 0.0;
        for (long d = 0; d < D; ++d) cn2 += ci[d] * ci[d];
        double rho2 = 0.0;
        for (long d = r; d < D; ++d) rho2 += w[d] * w[d];
        double rho = sqrt(rho2);
        for (long k = 0; k < r; ++k) R[i * M + k] = sgn[k] * w[k];
        if (r >= D || rho <= tau * sqrt(cn2)) continue;   /* dependent */

        /* reflector H = I - 2 u u^T acting on entries r..D-1 with
           H w[r:] = alpha e_0, alpha = -sign(w[r]) rho (no cancellation). */
        double alpha = (w[r] >= 0.0) ? -rho : rho;
        double *u = U + r * D;
        for (long d = r; d < D; ++d) u[d] = w[d];
        u[r] -= alpha;
        double unorm2 = 0.0;
        for (long d = r; d < D; ++d) unorm2 += u[d] * u[d];
        double unorm = sqrt(unorm2);
        for (long d = r; d < D; ++d) u[d] /= unorm;
        sgn[r] = (alpha > 0.0) ? 1.0 : -1.0;
        R[i * M + r] = rho;                  /* = sgn[r] * alpha */
        kept[r] = (int)i;

        /* apply the new reflector to every later codebook vector */
        #pragma omp parallel for schedule(static)
        for (long j = i + 1; j < M; ++j) {
            double *wj = W + j * D;
            double s = 0.0;
            for (long d = r; d < D; ++d) s += u[d] * wj[d];
            for (long d = r; d < D; ++d) wj[d] -= 2.0 * s * u[d];
        }
        ++r;
    }

    /* basis vector k = sgn[k] * H_0 H_1 ... H_k e_k (later reflectors leave
       e_k unchanged); apply them to e_k from the innermost outwards */
    #pragma omp parallel for schedule(dynamic, 1)
    for (long k = 0; k < r; ++k) {
        double *q = Q + k * D;
        memset(q, 0, sizeof(double) * (size_t)D);
        q[k] = 1.0;
        for (long j = k; j >= 0; --j) {
            const double *u = U + j * D;
            double s = 0.0;
            for (long d = j; d < D; ++d) s += u[d] * q[d];
            for (long d = j; d < D; ++d) q[d] -= 2.0 * s * u[d];
        }
        for (long d = 0; d < D; ++d) q[d] *= sgn[k];
    }
    *rank = (int)r;
    free(W); free(U); free(sgn);
    return 0;
}

/* Probability vectorisation (Sec. 2.2): v_b = sum_j P[b, j] c_j.
   P is B x M, C is M x D, V is B x D.  The scaled codebook vectors are added
   to v_b one after the other, j = 0 .. M - 1, so every component is summed
   in index order. */
void gso_prob2vec(const double *P, long B, long M, const double *C, long D,
                  double *V)
{
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b) {
        double *v = V + b * D;
        for (long d = 0; d < D; ++d) v[d] = 0.0;
        for (long j = 0; j < M; ++j) {
            const double p = P[b * M + j];
            const double *c = C + j * D;
            for (long d = 0; d < D; ++d) v[d] += p * c[d];
        }
    }
}

/* Euclidean row norms of a B x D matrix. */
void gso_row_norms(const double *X, long B, long D, double *out)
{
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b) {
        double s = 0.0;
        for (long d = 0; d < D; ++d) s += X[b * D + d] * X[b * D + d];
        out[b] = sqrt(s);
    }
}

/*
 * Similarity against the codebook in the original D-dimensional space
 * (Sec. 2.2; Sec. 3.2 Eq. 2-3).  mode 0 (dot):    S = scale * <x_b, c_j>
 *                                   mode 1 (cosine): S = scale * <x_b, c_j> /
 *                                                        (||x_b|| ||c_j||)
 * with a cosine of 0 where either norm is zero.  X is B x D, C is M x D.
 */
void gso_similarity(const double *X, long B, long D, const double *C, long M,
                    int mode, double scale, double *S)
{
    double *cn = (double *)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1));
    gso_row_norms(C, M, D, cn);
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b) {
        double xn2 = 0.0;
        for (long d = 0; d < D; ++d) xn2 += X[b * D + d] * X[b * D + d];
        double xn = sqrt(xn2);
        for (long j = 0; j < M; ++j) {
            double s = 0.0;
            for (long d = 0; d < D; ++d) s += X[b * D + d] * C[j * D + d];
            if (mode == 1) {
                double den = xn * cn[j];
                s = (den > 0.0) ? s / den : 0.0;
            }
            S[b * M + j] = scale * s;
        }
    }
    free(cn);
}

/* Row argmax, the lowest index winning an exact tie. */
void gso_argmax(const double *S, long B, long M, int *idx)
{
    for (long b = 0; b < B; ++b) {
        long best = 0;
        for (long j = 1; j < M; ++j)
            if (S[b * M + j] > S[b * M + best]) best = j;
        idx[b] = (int)best;
    }
}

/* Attention score (Sec. 2.2): a_b = softmax over the M entries of beta*s_b,
   computed with the row maximum subtracted. */
void gso_softmax(const double *S, long B, long M, double beta, double *A)
{
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b) {
        double m = -INFINITY;
        for (long j = 0; j < M; ++j)
            if (beta * S[b * M + j] > m) m = beta * S[b * M + j];
        double z = 0.0;
        for (long j = 0; j < M; ++j) z += exp(beta * S[b * M + j] - m);
        for (long j = 0; j < M; ++j) A[b * M + j] = exp(beta * S[b * M + j] - m) / z;
    }
}

/* Gram-loc of a batch (Sec. 3.1): t_b = U^T x_b, i.e. T[b, k] = <x_b, q_k>.
   X is B x D, Q is r x D, T is B x r. */
void gso_project(const double *X, long B, long D, const double *Q, long r,
                 double *T)
{
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b)
        for (long k = 0; k < r; ++k) {
            double s = 0.0;
            for (long d = 0; d < D; ++d) s += X[b * D + d] * Q[k * D + d];
            T[b * r + k] = s;
        }
}

/* Restore to the original domain (Sec. 3.1, Sec. 3.3): x_b = U t_b, i.e.
   X[b, d] = sum_k T[b, k] Q[k, d].  T is B x r, Q is r x D, X is B x D.  The
   scaled basis vectors are added one after the other, k = 0 .. r - 1, so
   every component is summed in index order. */
void gso_reconstruct(const double *T, long B, long r, const double *Q, long D,
                     double *X)
{
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b) {
        double *x = X + b * D;
        for (long d = 0; d < D; ++d) x[d] = 0.0;
        for (long k = 0; k < r; ++k) {
            const double t = T[b * r + k];
            const double *q = Q + k * D;
            for (long d = 0; d < D; ++d) x[d] += t * q[d];
        }
    }
}

/* Component-wise binding by element-wise product (Sec. 2.2; Table 1). */
void gso_bind(const double *X, const double *Y, long n, double *Z)
{
    #pragma omp parallel for schedule(static)
    for (long i = 0; i < n; ++i) Z[i] = X[i] * Y[i];
}

/* Blockwise circular convolution (binding) and circular correlation
   (unbinding) of restored vectors, the component-wise "modulo-style"
   operators that follow a restore (Sec. 2.2, Sec. 3.3).  Each row of D
   values splits into D / L consecutive blocks of length L; within a block,
     conv: Z[i] = sum_j X[j] Y[(i - j) mod L]
     corr: Z[i] = sum_j X[j] Y[(j - i) mod L]
   summed in index order j = 0 .. L - 1.  X, Y, Z are B x D. */
void gso_circular(const double *X, const double *Y, long B, long D, long L, int corr, double *Z)
{
    #pragma omp parallel for schedule(static)
    for (long b = 0; b < B; ++b)
        for (long s0 = 0; s0 < D; s0 += L) {
            const double *x = X + b * D + s0, *y = Y + b * D + s0;
            for (long i = 0; i < L; ++i) {
                double acc = 0.0;
                for (long j = 0; j < L; ++j) {
                    long k = corr ? (j - i) : (i - j);
                    k %= L;
                    if (k < 0) k += L;
                    acc += x[j] * y[k];
                }
                Z[b * D + s0 + i] = acc;
            }
        }
}

/* Exclusive-or binding of binary vectors: each restored value is read as the
   bit (value >= 0.5), Z = 1 where the two bits differ, else 0. */
void gso_xor(const double *X, const double *Y, long n, double *Z)
{
    #pragma omp parallel for schedule(static)
    for (long i = 0; i < n; ++i) Z[i] = ((X[i] >= 0.5) != (Y[i] >= 0.5)) ? 1.0 : 0.0;
}
