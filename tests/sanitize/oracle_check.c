/* Runs every oracle function on small shapes under AddressSanitizer and
 * UndefinedBehaviorSanitizer (zero-padded widths and n_dyad above a width
 * included), and checks the forward pass and its gradients against a dense
 * weight built by pushing unit vectors through the oracle's own forward pass
 * (a consistency check; the pins against the paper live in the Python tests). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_forward(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M, const double *X,
                    const double *W1, const double *W2, const double *bias, int act, double *Y, double *H);
void oracle_backward_dx(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M, const double *dZ,
                        const double *W1, const double *W2, int act_in, const double *H_in, double *dX);
void oracle_backward_dw(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M, const double *dZ,
                        const double *X, double *dW1, double *dW2, double *db);
void oracle_bias_grad(int64_t n_out, int64_t M, const double *dZ, double *db);
void oracle_backward_dw_entries(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M,
                                const double *dZ, const double *X, int64_t n, const int32_t *comp,
                                const int64_t *i, const int64_t *j, const int64_t *k, double *out);

static uint64_t state = 88172645463325252ull;
static double rnd(void) {   /* xorshift64, uniform in [-1, 1) */
    state ^= state << 13; state ^= state >> 7; state ^= state << 17;
    return (double)(state >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}
static double *vec(int64_t n) {
    double *p = malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    for (int64_t q = 0; q < n; ++q) p[q] = rnd();
    return p;
}

static int check(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M) {
    const int64_t bi = (n_in + D - 1) / D, bo = (n_out + D - 1) / D, nw = D * bo * bi;
    double *X = vec(M * n_in), *W1 = vec(nw), *W2 = vec(nw), *b = vec(n_out), *dZ = vec(M * n_out);
    double *H = vec(M * n_in), *Y = vec(M * n_out), *Hs = vec(M * n_out), *dX = vec(M * n_in);
    double *dW1 = vec(nw), *dW2 = vec(nw), *db = vec(n_out), *db2 = vec(n_out);
    double *E = calloc((size_t)n_in * n_in, sizeof(double)), *Wd = vec(n_in * n_out);
    for (int64_t c = 0; c < n_in; ++c) E[c * n_in + c] = 1.0;
    /* dense W (as Wd[c][f]) from unit inputs, no bias */
    oracle_forward(variant, n_in, n_out, D, n_in, E, W1, W2, NULL, 0, Wd, NULL);
    oracle_forward(variant, n_in, n_out, D, M, X, W1, W2, b, 1, Y, Hs);
    oracle_backward_dx(variant, n_in, n_out, D, M, dZ, W1, W2, 1, H, dX);
    oracle_backward_dw(variant, n_in, n_out, D, M, dZ, X, dW1, dW2, db);
    oracle_bias_grad(n_out, M, dZ, db2);
    int bad = 0;
    for (int64_t m = 0; m < M; ++m)
        for (int64_t f = 0; f < n_out; ++f) {
            double s = b[f];
            for (int64_t c = 0; c < n_in; ++c) s += Wd[c * n_out + f] * X[m * n_in + c];
            if (fabs(Hs[m * n_out + f] - s) > 1e-12 * (1 + fabs(s))) bad = 1;
        }
    for (int64_t m = 0; m < M; ++m)
        for (int64_t c = 0; c < n_in; ++c) {
            double s = 0;
            for (int64_t f = 0; f < n_out; ++f) s += Wd[c * n_out + f] * dZ[m * n_out + f];
            const double h = H[m * n_in + c];
            s *= 0.5 * erfc(-h / sqrt(2.0)) + h * exp(-0.5 * h * h) * 0.39894228040143267794;   /* 1 / sqrt(2 pi) */
            if (fabs(dX[m * n_in + c] - s) > 1e-12 * (1 + fabs(s))) bad = 1;
        }
    for (int64_t f = 0; f < n_out; ++f)
        if (fabs(db[f] - db2[f]) > 1e-12 * (1 + fabs(db[f]))) bad = 1;
    /* every entry of dW through the sampled-entry form */
    int32_t *comp = malloc(2 * nw * sizeof(int32_t));
    int64_t *ii = malloc(2 * nw * sizeof(int64_t)), *jj = malloc(2 * nw * sizeof(int64_t)),
            *kk = malloc(2 * nw * sizeof(int64_t));
    double *ent = malloc(2 * nw * sizeof(double));
    for (int64_t q = 0; q < 2 * nw; ++q) {
        const int64_t e = q % nw;
        comp[q] = q < nw ? 1 : 2; ii[q] = e / (bo * bi); jj[q] = (e / bi) % bo; kk[q] = e % bi;
    }
    oracle_backward_dw_entries(variant, n_in, n_out, D, M, dZ, X, 2 * nw, comp, ii, jj, kk, ent);
    for (int64_t q = 0; q < 2 * nw; ++q) {
        const double ref = q < nw ? dW1[q] : dW2[q - nw];
        if (fabs(ent[q] - ref) > 1e-12 * (1 + fabs(ref))) bad = 1;
    }
    free(X); free(W1); free(W2); free(b); free(dZ); free(H); free(Y); free(Hs); free(dX);
    free(dW1); free(dW2); free(db); free(db2); free(E); free(Wd);
    free(comp); free(ii); free(jj); free(kk); free(ent);
    if (bad) fprintf(stderr, "mismatch: variant %d, %lld -> %lld, n_dyad %lld, M %lld\n", variant,
                     (long long)n_in, (long long)n_out, (long long)D, (long long)M);
    return bad;
}

int main(void) {
    static const int64_t shapes[][4] = {
        {64, 256, 4, 9}, {16, 16, 4, 3}, {12, 18, 3, 4}, {7, 6, 2, 5}, {5, 9, 8, 3},
        {100, 36, 8, 2}, {10, 6, 1, 4}, {32, 16, 16, 2}, {24, 40, 8, 0},
    };
    int bad = 0;
    for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
        for (int v = 0; v < 3; ++v) bad |= check(v, shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3]);
    if (bad) return 1;
    printf("oracle sanitized ok\n");
    return 0;
}
