/*
 * cola_oracle.c -- plain fp64 CPU oracle for the CoLA layer.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * definition that the GPU library is checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark load it; the GPU
 * product path never links, imports or calls it, and it shares no code,
 * header, table or helper with that path.
 *
 * What it computes (CoLA, arXiv 2502.10940):
 *   - the CoLA layer h = B sigma(A x)                     (Sec. 3.2, Eq. main-fwd)
 *   - the dense layers h = W x used as the baseline       (Sec. 3.2, Eq. full-rank-linear)
 *   - their gradients by the chain rule, the "2x rule":
 *     grad_x = W^T grad_h and grad_W = grad_h x^T per GEMM (Sec. 3.4, the
 *     gradient equation under Table "compute breakdown")
 *   - CoLA-M keeps only the r-wide pre-activation A x and recomputes
 *     sigma(A x) in backward (Sec. 4.2 and App. C); the values are those of
 *     CoLA, so the backward below takes the saved pre-activation Z as input.
 *
 * Layout (the paper stores one token per column, X in R^{d_in x n}; this
 * oracle stores the transpose, one token per row, which is what the GPU
 * library uses):
 *   X[T][d_in], A[r][d_in], B[d_out][r], Z,H,dZ[T][r], Y,dY[T][d_out],
 *   dX[T][d_in], dA[r][d_in], dB[d_out][r], W[d_out][d_in], dW[d_out][d_in].
 * All arrays are dense row-major fp64.  So Z = X A^T is (A X_paper)^T.
 *
 * sigma: act 0 = identity, act 1 = SiLU (Swish with beta = 1), the
 * activation the paper names for its LLaMA runs (Sec. 5.2, the closing remark
 * naming GeLU and Swish).  SiLU(z) = z s(z), s = logistic sigmoid,
 * SiLU'(z) = s(z) (1 + z (1 - s(z))).  act 2 = GeLU, the other activation
 * that remark names (the BERT runs, App. D); the paper does not say which
 * form, this is the exact one: GeLU(z) = z Phi(z), Phi the standard normal
 * CDF, GeLU'(z) = Phi(z) + z phi(z), phi its density.
 *
 * Every matrix product is a textbook triple loop, no blocking, no BLAS,
 * no fast-math; OpenMP splits only the outermost output-row loop, so each
 * output element is one sequential sum in fp64.
 *
 * The "both sigma" variant of the ablation (an outer nonlinearity sigma_out
 * on the layer output, App. ablation) is the composition of the layer with
 * sigma_out; its backward is the chain rule through that composition.
 *
 * Pins (tests/test_oracle_*.py): identity-sigma closed form against the
 * conventional low-rank product B A X (Sec. 3.3), central finite differences,
 * torch fp64 autograd, the Prop. 1 limit construction, the Lemma
 * (E_sigma = 0) construction, SiLU special values, and the FLOP counts of
 * Table "compute all methods" (Sec. 3.4) and App. B.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* multiply-add counter: each GEMM adds its loop trip count M*N*K once.      */
/* ------------------------------------------------------------------------ */
static int64_t g_mac_count = 0;

void oracle_reset_macs(void) { g_mac_count = 0; }
int64_t oracle_macs(void) { return g_mac_count; }

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* the pointwise nonlinearity                                               */
/* ------------------------------------------------------------------------ */

/* logistic sigmoid, evaluated so that exp never overflows */
static double logistic(double z) {
    if (z >= 0.0) return 1.0 / (1.0 + exp(-z));
    double e = exp(z);
    return e / (1.0 + e);
}

/* standard normal CDF through erfc (no cancellation for negative z) and density */
static double normal_cdf(double z) { return 0.5 * erfc(-z * 0.70710678118654752440); }
static double normal_pdf(double z) { return 0.39894228040143267794 * exp(-0.5 * z * z); }

double oracle_sigma(int act, double z) {
    if (act == 0) return z;
    if (act == 2) return z * normal_cdf(z);
    return z * logistic(z);
}

double oracle_sigma_prime(int act, double z) {
    if (act == 0) return 1.0;
    if (act == 2) return normal_cdf(z) + z * normal_pdf(z);
    double s = logistic(z);
    return s * (1.0 + z * (1.0 - s));
}

/* ------------------------------------------------------------------------ */
/* the three GEMM shapes the layer needs, each a plain triple loop           */
/* ------------------------------------------------------------------------ */

/* C[M][N] = sum_k P[M][K] * Q[N][K]          (P Q^T) */
static void gemm_nt(int64_t M, int64_t N, int64_t K,
                    const double* P, const double* Q, double* C) {
    g_mac_count += M * N * K;
    #pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            double s = 0.0;
            for (int64_t k = 0; k < K; ++k) s += P[m * K + k] * Q[n * K + k];
            C[m * N + n] = s;
        }
}

/* C[M][N] = sum_k P[M][K] * Q[K][N]          (P Q) */
static void gemm_nn(int64_t M, int64_t N, int64_t K,
                    const double* P, const double* Q, double* C) {
    g_mac_count += M * N * K;
    #pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        double* c = C + m * N;
        for (int64_t n = 0; n < N; ++n) c[n] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double p = P[m * K + k];
            const double* q = Q + k * N;
            for (int64_t n = 0; n < N; ++n) c[n] += p * q[n];
        }
    }
}

/* C[M][N] = sum_k P[K][M] * Q[K][N]          (P^T Q) */
static void gemm_tn(int64_t M, int64_t N, int64_t K,
                    const double* P, const double* Q, double* C) {
    g_mac_count += M * N * K;
    #pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        double* c = C + m * N;
        for (int64_t n = 0; n < N; ++n) c[n] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double p = P[k * M + m];
            const double* q = Q + k * N;
            for (int64_t n = 0; n < N; ++n) c[n] += p * q[n];
        }
    }
}

/* ------------------------------------------------------------------------ */
/* CoLA layer                                                               */
/* ------------------------------------------------------------------------ */

/* Forward, Eq. main-fwd: Z = A x, H = sigma(Z), Y = B H  (token-major). */
void oracle_cola_fwd(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int act,
                     const double* X, const double* A, const double* B,
                     double* Z, double* H, double* Y) {
    gemm_nt(T, r, d_in, X, A, Z);                 /* Z[t][j] = sum_k X[t][k] A[j][k] */
    for (int64_t i = 0; i < T * r; ++i) H[i] = oracle_sigma(act, Z[i]);
    gemm_nt(T, d_out, r, H, B, Y);                /* Y[t][o] = sum_j H[t][j] B[o][j] */
}

/* Backward from the saved pre-activation Z (what CoLA-M keeps; CoLA keeps
 * H = sigma(Z) as well, which is the same value).  Chain rule through
 * Y = B sigma(Z), Z = A x, each GEMM giving its two gradient GEMMs:
 *   dH = dY B, dZ = dH * sigma'(Z), dX = dZ A, dA = dZ^T X, dB = dY^T H.
 * dZ_out may be NULL.  dA and dB are overwritten. */
void oracle_cola_bwd(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int act,
                     const double* X, const double* Z,
                     const double* A, const double* B, const double* dY,
                     double* dZ_out, double* dX, double* dA, double* dB,
                     double* scratch /* 2*T*r doubles */) {
    double* H = scratch;
    double* dZ = scratch + T * r;
    for (int64_t i = 0; i < T * r; ++i) H[i] = oracle_sigma(act, Z[i]);
    gemm_nn(T, r, d_out, dY, B, dZ);              /* dH[t][j] = sum_o dY[t][o] B[o][j] */
    for (int64_t i = 0; i < T * r; ++i) dZ[i] *= oracle_sigma_prime(act, Z[i]);
    gemm_nn(T, d_in, r, dZ, A, dX);               /* dX[t][k] = sum_j dZ[t][j] A[j][k] */
    gemm_tn(r, d_in, T, dZ, X, dA);               /* dA[j][k] = sum_t dZ[t][j] X[t][k] */
    gemm_tn(d_out, r, T, dY, H, dB);              /* dB[o][j] = sum_t dY[t][o] H[t][j] */
    if (dZ_out) memcpy(dZ_out, dZ, (size_t)(T * r) * sizeof(double));
}

/* ------------------------------------------------------------------------ */
/* "both sigma" variant (App. ablation, Table "ablation"): the nonlinearity */
/* that followed the original linear layer is kept on top of the layer,      */
/* Y = sigma_out(B sigma(A x)).  The layer output before sigma_out, P, is    */
/* what the backward needs.                                                  */
/* ------------------------------------------------------------------------ */

/* Forward: Z, H as in oracle_cola_fwd, P = H B^T, Y = sigma_out(P). */
void oracle_cola_fwd_outer(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int act, int outer,
                           const double* X, const double* A, const double* B,
                           double* Z, double* H, double* P, double* Y) {
    oracle_cola_fwd(T, d_in, d_out, r, act, X, A, B, Z, H, P);
    for (int64_t i = 0; i < T * d_out; ++i) Y[i] = oracle_sigma(outer, P[i]);
}

/* Backward: the chain rule through sigma_out gives dP = dY * sigma_out'(P);
 * the layer's own backward then runs on dP.  dP_out may be NULL. */
void oracle_cola_bwd_outer(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int act, int outer,
                           const double* X, const double* Z, const double* P,
                           const double* A, const double* B, const double* dY,
                           double* dP_out, double* dZ_out, double* dX, double* dA, double* dB,
                           double* scratch /* 2*T*r + T*d_out doubles */) {
    double* dP = scratch + 2 * T * r;
    for (int64_t i = 0; i < T * d_out; ++i) dP[i] = dY[i] * oracle_sigma_prime(outer, P[i]);
    oracle_cola_bwd(T, d_in, d_out, r, act, X, Z, A, B, dP, dZ_out, dX, dA, dB, scratch);
    if (dP_out) memcpy(dP_out, dP, (size_t)(T * d_out) * sizeof(double));
}

/* CoLA-M's recompute of a layer output from its saved pre-activation (Sec.
 * 4.2, App. C: only the r-wide activation is kept, the up projection B h is
 * recomputed in backward): H = sigma(Z), Y = H B^T. */
void oracle_cola_up_from_z(int64_t T, int64_t d_out, int64_t r, int act,
                           const double* Z, const double* B, double* H, double* Y) {
    for (int64_t i = 0; i < T * r; ++i) H[i] = oracle_sigma(act, Z[i]);
    /* the up projection */
    gemm_nt(T, d_out, r, H, B, Y);                /* Y[t][o] = sum_j H[t][j] B[o][j] */
}

/* ------------------------------------------------------------------------ */
/* dense baseline, Eq. full-rank-linear and the 2x rule                      */
/* ------------------------------------------------------------------------ */

void oracle_dense_fwd(int64_t T, int64_t d_in, int64_t d_out,
                      const double* X, const double* W, double* Y) {
    gemm_nt(T, d_out, d_in, X, W, Y);             /* Y[t][o] = sum_k X[t][k] W[o][k] */
}

void oracle_dense_bwd(int64_t T, int64_t d_in, int64_t d_out,
                      const double* X, const double* W, const double* dY,
                      double* dX, double* dW) {
    gemm_nn(T, d_in, d_out, dY, W, dX);           /* dX[t][k] = sum_o dY[t][o] W[o][k] */
    gemm_tn(d_out, d_in, T, dY, X, dW);           /* dW[o][k] = sum_t dY[t][o] X[t][k] */
}

/* ------------------------------------------------------------------------ */
/* sampled evaluation for shapes too large for the full oracle               */
/* ------------------------------------------------------------------------ */

/* Dense layer, per selected token t = rows[i]: the rows Y[t][:] and dX[t][:]
 * from the definition on that token alone.  Outputs are [nrows][width]. */
void oracle_dense_rows(int64_t T, int64_t d_in, int64_t d_out,
                       const double* X, const double* W, const double* dY,
                       int64_t nrows, const int64_t* rows, double* Yr, double* dXr) {
    (void)T;
    g_mac_count += nrows * (d_out * d_in + d_in * d_out);
    #pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < nrows; ++i) {
        const double* x = X + rows[i] * d_in;
        const double* dy = dY + rows[i] * d_out;
        for (int64_t o = 0; o < d_out; ++o) {        /* Y[t][o] = sum_k X[t][k] W[o][k] */
            double s = 0.0;
            for (int64_t k = 0; k < d_in; ++k) s += x[k] * W[o * d_in + k];
            Yr[i * d_out + o] = s;
        }
        for (int64_t k = 0; k < d_in; ++k) {         /* dX[t][k] = sum_o dY[t][o] W[o][k] */
            double s = 0.0;
            for (int64_t o = 0; o < d_out; ++o) s += dy[o] * W[o * d_in + k];
            dXr[i * d_in + k] = s;
        }
    }
}

/* Dense weight gradient, per selected output index o = outs[i]: the row
 * dW[o][:] = sum_t dY[t][o] X[t][:].  Output is [nouts][d_in]. */
void oracle_dense_wgrad_rows(int64_t T, int64_t d_in, int64_t d_out,
                             const double* X, const double* dY,
                             int64_t nouts, const int64_t* outs, double* dWr) {
    g_mac_count += nouts * d_in * T;
    #pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < nouts; ++i) {
        const int64_t o = outs[i];
        for (int64_t k = 0; k < d_in; ++k) {
            double s = 0.0;
            for (int64_t t = 0; t < T; ++t) s += dY[t * d_out + o] * X[t * d_in + k];
            dWr[i * d_in + k] = s;
        }
    }
}

/* Per selected token t = rows[i]: Z, H, Y, dZ and dX rows, each computed from
 * the definition on that token alone (every output row of the layer depends
 * only on its own input row).  Outputs are [nrows][width]. */
void oracle_cola_rows(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int act,
                      const double* X, const double* A, const double* B, const double* dY,
                      int64_t nrows, const int64_t* rows,
                      double* Zr, double* Hr, double* Yr, double* dZr, double* dXr) {
    (void)T;
    g_mac_count += nrows * (r * d_in + d_out * r + d_out * r + d_in * r);
    #pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < nrows; ++i) {
        const double* x = X + rows[i] * d_in;
        const double* dy = dY + rows[i] * d_out;
        double* z = Zr + i * r;
        double* h = Hr + i * r;
        double* y = Yr + i * d_out;
        double* dz = dZr + i * r;
        double* dx = dXr + i * d_in;
        for (int64_t j = 0; j < r; ++j) {
            double s = 0.0;
            for (int64_t k = 0; k < d_in; ++k) s += x[k] * A[j * d_in + k];
            z[j] = s;
            h[j] = oracle_sigma(act, s);
        }
        for (int64_t o = 0; o < d_out; ++o) {
            double s = 0.0;
            for (int64_t j = 0; j < r; ++j) s += h[j] * B[o * r + j];
            y[o] = s;
        }
        for (int64_t j = 0; j < r; ++j) {
            double s = 0.0;
            for (int64_t o = 0; o < d_out; ++o) s += dy[o] * B[o * r + j];
            dz[j] = s * oracle_sigma_prime(act, z[j]);
        }
        for (int64_t k = 0; k < d_in; ++k) {
            double s = 0.0;
            for (int64_t j = 0; j < r; ++j) s += dz[j] * A[j * d_in + k];
            dx[k] = s;
        }
    }
}

/* Per selected rank index j = cols[c]: the full row dA[j][:] and the full
 * column dB[:][j].  Both need the whole token column Z[:, j]:
 *   Z[t][j] = sum_k X[t][k] A[j][k],  dZ[t][j] = (sum_o dY[t][o] B[o][j]) sigma'(Z[t][j]),
 *   dA[j][k] = sum_t dZ[t][j] X[t][k], dB[o][j] = sum_t dY[t][o] sigma(Z[t][j]).
 * Outputs dA_rows[ncols][d_in], dB_cols[ncols][d_out].  Returns 0, or -1 if
 * the temporary token columns cannot be allocated. */
int oracle_cola_wgrad_cols(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int act,
                           const double* X, const double* A, const double* B, const double* dY,
                           int64_t ncols, const int64_t* cols,
                           double* dA_rows, double* dB_cols) {
    double* H = (double*)malloc((size_t)(2 * T) * sizeof(double));
    if (!H) return -1;
    double* dZ = H + T;
    g_mac_count += ncols * T * (2 * d_in + 2 * d_out);
    for (int64_t c = 0; c < ncols; ++c) {
        int64_t j = cols[c];
        double* da = dA_rows + c * d_in;
        double* db = dB_cols + c * d_out;
        #pragma omp parallel for schedule(static)
        for (int64_t t = 0; t < T; ++t) {
            double z = 0.0;
            for (int64_t k = 0; k < d_in; ++k) z += X[t * d_in + k] * A[j * d_in + k];
            double dh = 0.0;
            for (int64_t o = 0; o < d_out; ++o) dh += dY[t * d_out + o] * B[o * r + j];
            H[t] = oracle_sigma(act, z);
            dZ[t] = dh * oracle_sigma_prime(act, z);
        }
        #pragma omp parallel for schedule(static)
        for (int64_t k = 0; k < d_in; ++k) {
            double s = 0.0;
            for (int64_t t = 0; t < T; ++t) s += dZ[t] * X[t * d_in + k];
            da[k] = s;
        }
        #pragma omp parallel for schedule(static)
        for (int64_t o = 0; o < d_out; ++o) {
            double s = 0.0;
            for (int64_t t = 0; t < T; ++t) s += dY[t * d_out + o] * H[t];
            db[o] = s;
        }
    }
    free(H);
    return 0;
}
