/*
 * CPU oracle for the Dyad layer (arXiv 2312.06881) -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load this file's library.  It is a plain, slow, obviously-correct statement of
 * what the Dyad layer computes, in fp64, with no blocking, fusion or reordering.
 * It shares no code, header or constant with the GPU library.
 *
 * Notation (token-major, row-major, as PyTorch stores activations; the paper's
 * Sec. 2.1 uses the transposed, feature-major convention -- every reshape in the
 * paper acts on the feature index only, so the arithmetic is identical):
 *   D  = n_dyad, the number of blocks per component
 *   n_in, n_out = full layer widths; bi = ceil(n_in / D), bo = ceil(n_out / D)
 *   (bi, bo are what the paper calls n_in, n_out: the size of one block, Sec. 2.2)
 *   X[M][n_in], Y[M][n_out], W1[D][bo][bi] (BlockDiag), W2[D][bo][bi] (BlockTrans)
 *
 * Each stored weight W_c[i][j][k] is one entry of the dense weight W at
 * (row, col) given by the index maps below; Y[m] = W X[m] + b (Sec. 2.2, Eq. 1).
 *   BlockDiag, every variant:   row = i*bo + j, col = i*bi + k          (Eq. 2)
 *   BlockTrans, Dyad-IT:        row = i*bo + j, col = k*D  + i          (Eq. 9-10)
 *   BlockTrans, Dyad-OT:        row = j*D  + i, col = i*bi + k          (Sec. 2.4.1, Eq. 11-13)
 *   BlockTrans, Dyad-DT:        row = j*D  + i, col = k*D  + i          (Sec. 2.4.2, Eq. 14-16)
 * Readings where the paper is silent or inconsistent:
 *   - Dyad-IT input map: the strided view of Eq. 9 (reshape to (bi, D, .) then
 *     swap the first two axes) is taken as binding; it equals P X for the P of
 *     Eq. 5, where Eq. 6 writes P^T X.  The two agree only when bi == D.
 *   - Dyad-OT output map: the mirror image of Eq. 9 applied to the output, i.e.
 *     the block output Z2[i][j] lands on feature j*D + i (Eq. 13 with the P of
 *     Eq. 5 built for block size bo).
 *   - The paper never names the activation between fc1 and fc2; this oracle
 *     offers the exact (erf) GELU, x * Phi(x).
 *   - The backward pass is not described in the paper; it is the gradient of
 *     Y = W X + b: dX = W^T dZ, dW_c[i][j][k] = sum_m dZ[m][row] X[m][col],
 *     db = sum_m dZ[m].  Weight gradients are overwritten, not accumulated.
 *   - Widths that n_dyad does not divide are zero-padded up to the next
 *     multiple of n_dyad (appendix, caveat on rectangular W): the layer is the
 *     one of widths D*bi -> D*bo applied to X with zero columns appended, and
 *     only its first n_out outputs are kept.  An entry whose col is >= n_in
 *     therefore meets a zero input, and one whose row is >= n_out feeds a
 *     dropped output: both contribute nothing, and their gradients are zero.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <omp.h>

#define ORACLE_IT 0
#define ORACLE_OT 1
#define ORACLE_DT 2

#define ORACLE_ACT_NONE 0
#define ORACLE_ACT_GELU 1

/* Dense-W row of stored entry W_c[i][j][.] (maps in the header). */
static int64_t entry_row(int variant, int comp, int64_t D, int64_t bo, int64_t i, int64_t j)
{
    if (comp == 1 || variant == ORACLE_IT)
        return i * bo + j;
    return j * D + i;
}

/* Dense-W column of stored entry W_c[i][.][k] (maps in the header). */
static int64_t entry_col(int variant, int comp, int64_t D, int64_t bi, int64_t i, int64_t k)
{
    if (comp == 1 || variant == ORACLE_OT)
        return i * bi + k;
    return k * D + i;
}

/* Per-block size of a width zero-padded up to a multiple of D. */
static int64_t block_size(int64_t n, int64_t D)
{
    return (n + D - 1) / D;
}

/* Standard normal CDF, Phi(x) = erfc(-x / sqrt 2) / 2 (no cancellation for x << 0). */
static double normal_cdf(double x)
{
    return 0.5 * erfc(-x / sqrt(2.0));
}

/* Exact GELU, x * Phi(x). */
double oracle_gelu(double x)
{
    return x * normal_cdf(x);
}

/* d/dx [x * Phi(x)] = Phi(x) + x * phi(x). */
double oracle_gelu_grad(double x)
{
    const double pi = 3.14159265358979323846;
    return normal_cdf(x) + x * exp(-0.5 * x * x) / sqrt(2.0 * pi);
}

/* out[e] = GELU(in[e]) for n values: the activated input of a layer that
 * follows a GELU (fc2 of a feed-forward block), formed elementwise. */
void oracle_gelu_vec(int64_t n, const double *in, double *out)
{
    int64_t e;
#pragma omp parallel for schedule(static)
    for (e = 0; e < n; ++e)
        out[e] = oracle_gelu(in[e]);
}

int oracle_threads(void)
{
    return omp_get_max_threads();
}

/*
 * Forward: Y[m] = W X[m] + b, then optionally H = Y (pre-activation) and
 * Y = GELU(H).  bias may be NULL (no bias); H may be NULL.
 */
void oracle_forward(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M,
                    const double *X, const double *W1, const double *W2, const double *bias,
                    int act, double *Y, double *H)
{
    const int64_t bi = block_size(n_in, D), bo = block_size(n_out, D);
    int64_t m;
#pragma omp parallel for schedule(static)
    for (m = 0; m < M; ++m) {
        const double *x = X + m * n_in;
        double *y = Y + m * n_out;
        for (int64_t f = 0; f < n_out; ++f)
            y[f] = bias ? bias[f] : 0.0;
        for (int comp = 1; comp <= 2; ++comp) {
            const double *W = comp == 1 ? W1 : W2;
            for (int64_t i = 0; i < D; ++i)
                for (int64_t j = 0; j < bo; ++j)
                    for (int64_t k = 0; k < bi; ++k) {
                        int64_t row = entry_row(variant, comp, D, bo, i, j);
                        int64_t col = entry_col(variant, comp, D, bi, i, k);
                        if (row >= n_out || col >= n_in) /* padded output or zero input */
                            continue;
                        y[row] += W[(i * bo + j) * bi + k] * x[col];
                    }
        }
        if (act == ORACLE_ACT_GELU) {
            for (int64_t f = 0; f < n_out; ++f) {
                if (H)
                    H[m * n_out + f] = y[f];
                y[f] = oracle_gelu(y[f]);
            }
        }
    }
}

/*
 * Input gradient: dX[m] = W^T dZ[m], then optionally dX *= GELU'(H_in) when the
 * layer's input X was GELU(H_in).  H_in must be non-NULL when act_in is GELU.
 */
void oracle_backward_dx(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M,
                        const double *dZ, const double *W1, const double *W2,
                        int act_in, const double *H_in, double *dX)
{
    const int64_t bi = block_size(n_in, D), bo = block_size(n_out, D);
    int64_t m;
#pragma omp parallel for schedule(static)
    for (m = 0; m < M; ++m) {
        const double *dz = dZ + m * n_out;
        double *dx = dX + m * n_in;
        for (int64_t c = 0; c < n_in; ++c)
            dx[c] = 0.0;
        for (int comp = 1; comp <= 2; ++comp) {
            const double *W = comp == 1 ? W1 : W2;
            for (int64_t i = 0; i < D; ++i)
                for (int64_t j = 0; j < bo; ++j)
                    for (int64_t k = 0; k < bi; ++k) {
                        int64_t row = entry_row(variant, comp, D, bo, i, j);
                        int64_t col = entry_col(variant, comp, D, bi, i, k);
                        if (row >= n_out || col >= n_in) /* no gradient through padding */
                            continue;
                        dx[col] += W[(i * bo + j) * bi + k] * dz[row];
                    }
        }
        if (act_in == ORACLE_ACT_GELU)
            for (int64_t c = 0; c < n_in; ++c)
                dx[c] *= oracle_gelu_grad(H_in[m * n_in + c]);
    }
}

/* Bias gradient: db[f] = sum_m dZ[m][f]. */
void oracle_bias_grad(int64_t n_out, int64_t M, const double *dZ, double *db)
{
    int64_t f;
#pragma omp parallel for schedule(static)
    for (f = 0; f < n_out; ++f) {
        double s = 0.0;
        for (int64_t m = 0; m < M; ++m)
            s += dZ[m * n_out + f];
        db[f] = s;
    }
}

/*
 * Weight and bias gradients: dW_c[i][j][k] = sum_m dZ[m][row] X[m][col],
 * db[f] = sum_m dZ[m][f].  db may be NULL.
 */
void oracle_backward_dw(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M,
                        const double *dZ, const double *X, double *dW1, double *dW2, double *db)
{
    const int64_t bi = block_size(n_in, D), bo = block_size(n_out, D);
    int64_t t;
#pragma omp parallel for schedule(static)
    for (t = 0; t < 2 * D * bo; ++t) {
        int comp = t < D * bo ? 1 : 2;
        int64_t ij = t % (D * bo), i = ij / bo, j = ij % bo;
        double *dW = comp == 1 ? dW1 : dW2;
        int64_t row = entry_row(variant, comp, D, bo, i, j);
        for (int64_t k = 0; k < bi; ++k) {
            int64_t col = entry_col(variant, comp, D, bi, i, k);
            double s = 0.0;
            if (row < n_out && col < n_in) /* else the entry touches only padding */
                for (int64_t m = 0; m < M; ++m)
                    s += dZ[m * n_out + row] * X[m * n_in + col];
            dW[(i * bo + j) * bi + k] = s;
        }
    }
    if (db)
        oracle_bias_grad(n_out, M, dZ, db);
}

/*
 * Selected weight-gradient entries, for checks at sizes where the full dW is
 * too slow: out[e] = dW_{comp[e]}[i[e]][j[e]][k[e]] by the same sum as above.
 */
void oracle_backward_dw_entries(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M,
                                const double *dZ, const double *X, int64_t n_entries,
                                const int32_t *comp, const int64_t *i, const int64_t *j,
                                const int64_t *k, double *out)
{
    const int64_t bi = block_size(n_in, D), bo = block_size(n_out, D);
    int64_t e;
#pragma omp parallel for schedule(static)
    for (e = 0; e < n_entries; ++e) {
        int64_t row = entry_row(variant, comp[e], D, bo, i[e], j[e]);
        int64_t col = entry_col(variant, comp[e], D, bi, i[e], k[e]);
        double s = 0.0;
        if (row < n_out && col < n_in)
            for (int64_t m = 0; m < M; ++m)
                s += dZ[m * n_out + row] * X[m * n_in + col];
        out[e] = s;
    }
}
