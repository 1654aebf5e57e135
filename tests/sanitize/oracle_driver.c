/* Host sanitizer driver for the fp64 oracle (test infrastructure): every
 * oracle entry point on small and degenerate shapes, built with
 * AddressSanitizer and UndefinedBehaviorSanitizer; any report fails the run.
 * Also checks a few values the definitions fix (identity sigma gives the
 * low-rank product; the sampled evaluators give the full oracle's rows). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_cola_fwd(int64_t, int64_t, int64_t, int64_t, int, const double*, const double*, const double*,
                     double*, double*, double*);
void oracle_cola_bwd(int64_t, int64_t, int64_t, int64_t, int, const double*, const double*, const double*,
                     const double*, const double*, double*, double*, double*, double*, double*);
void oracle_cola_fwd_outer(int64_t, int64_t, int64_t, int64_t, int, int, const double*, const double*,
                           const double*, double*, double*, double*, double*);
void oracle_cola_bwd_outer(int64_t, int64_t, int64_t, int64_t, int, int, const double*, const double*,
                           const double*, const double*, const double*, const double*, double*, double*, double*,
                           double*, double*, double*);
void oracle_dense_fwd(int64_t, int64_t, int64_t, const double*, const double*, double*);
void oracle_dense_bwd(int64_t, int64_t, int64_t, const double*, const double*, const double*, double*, double*);
void oracle_cola_rows(int64_t, int64_t, int64_t, int64_t, int, const double*, const double*, const double*,
                      const double*, int64_t, const int64_t*, double*, double*, double*, double*, double*);
int oracle_cola_wgrad_cols(int64_t, int64_t, int64_t, int64_t, int, const double*, const double*, const double*,
                           const double*, int64_t, const int64_t*, double*, double*);
void oracle_cola_up_from_z(int64_t, int64_t, int64_t, int, const double*, const double*, double*, double*);
void oracle_dense_rows(int64_t, int64_t, int64_t, const double*, const double*, const double*, int64_t,
                       const int64_t*, double*, double*);
void oracle_dense_wgrad_rows(int64_t, int64_t, int64_t, const double*, const double*, int64_t, const int64_t*,
                             double*);

static double* arr(int64_t n, unsigned seed) {
    double* p = malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    for (int64_t i = 0; i < n; ++i) {
        seed = seed * 1103515245u + 12345u;
        p[i] = ((seed >> 8) & 0xffff) / 32768.0 - 1.0;
    }
    return p;
}

static int run(int64_t T, int64_t di, int64_t dO, int64_t r, int act) {
    double *X = arr(T * di, 1), *A = arr(r * di, 2), *B = arr(dO * r, 3), *dY = arr(T * dO, 4);
    double *Z = arr(T * r, 0), *H = arr(T * r, 0), *Y = arr(T * dO, 0), *P = arr(T * dO, 0), *Yo = arr(T * dO, 0);
    double *dZ = arr(T * r, 0), *dX = arr(T * di, 0), *dA = arr(r * di, 0), *dB = arr(dO * r, 0);
    double* scratch = arr(2 * T * r + T * dO, 0);
    double *dP = arr(T * dO, 0), *W = arr(dO * di, 5), *dW = arr(dO * di, 0);
    int bad = 0;
    oracle_cola_fwd(T, di, dO, r, act, X, A, B, Z, H, Y);
    oracle_cola_bwd(T, di, dO, r, act, X, Z, A, B, dY, dZ, dX, dA, dB, scratch);
    oracle_cola_fwd_outer(T, di, dO, r, act, 1, X, A, B, Z, H, P, Yo);
    oracle_cola_bwd_outer(T, di, dO, r, act, 1, X, Z, P, A, B, dY, dP, dZ, dX, dA, dB, scratch);
    oracle_dense_fwd(T, di, dO, X, W, Y);
    oracle_dense_bwd(T, di, dO, X, W, dY, dX, dW);
    oracle_cola_up_from_z(T, dO, r, act, Z, B, H, Y);
    if (T > 0) {
        int64_t rows[3] = {0, T - 1, T / 2};
        double *Zr = arr(3 * r, 0), *Hr = arr(3 * r, 0), *Yr = arr(3 * dO, 0), *dZr = arr(3 * r, 0),
               *dXr = arr(3 * di, 0);
        oracle_cola_rows(T, di, dO, r, act, X, A, B, dY, 3, rows, Zr, Hr, Yr, dZr, dXr);
        int64_t cols[2] = {0, r - 1};
        double *dAr = arr(2 * di, 0), *dBc = arr(2 * dO, 0);
        bad |= oracle_cola_wgrad_cols(T, di, dO, r, act, X, A, B, dY, 2, cols, dAr, dBc) != 0;
        int64_t outs[2] = {0, dO - 1};
        double *Ydr = arr(3 * dO, 0), *dXdr = arr(3 * di, 0), *dWr = arr(2 * di, 0);
        oracle_dense_rows(T, di, dO, X, W, dY, 3, rows, Ydr, dXdr);
        oracle_dense_wgrad_rows(T, di, dO, X, dY, 2, outs, dWr);
        /* the sampled dense rows are the full oracle's rows */
        for (int64_t k = 0; k < di; ++k)
            if (fabs(dWr[k] - dW[k]) > 1e-12 * (1.0 + fabs(dW[k]))) bad = 1;
        free(Zr); free(Hr); free(Yr); free(dZr); free(dXr); free(dAr); free(dBc); free(Ydr); free(dXdr); free(dWr);
    }
    if (act == 0 && T > 0) {
        /* identity sigma: Y = X (B A)^T */
        oracle_cola_fwd(T, di, dO, r, 0, X, A, B, Z, H, Y);
        for (int64_t t = 0; t < T; ++t)
            for (int64_t o = 0; o < dO; ++o) {
                double s = 0.0;
                for (int64_t k = 0; k < di; ++k) {
                    double w = 0.0;
                    for (int64_t j = 0; j < r; ++j) w += B[o * r + j] * A[j * di + k];
                    s += X[t * di + k] * w;
                }
                if (fabs(s - Y[t * dO + o]) > 1e-10 * (1.0 + fabs(s))) bad = 1;
            }
    }
    free(X); free(A); free(B); free(dY); free(Z); free(H); free(Y); free(P); free(Yo); free(dZ); free(dX);
    free(dA); free(dB); free(scratch); free(dP); free(W); free(dW);
    return bad;
}

int main(void) {
    const int64_t shapes[][4] = {{1, 1, 1, 1}, {3, 5, 4, 2}, {7, 1, 4, 3}, {17, 13, 9, 5}, {0, 4, 3, 2}};
    int bad = 0;
    for (unsigned s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
        for (int act = 0; act < 3; ++act) bad |= run(shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3], act);
    printf(bad ? "oracle sanitizer driver: value check FAILED\n" : "oracle sanitizer driver: ok\n");
    return bad;
}
