/*
 * scd_oracle.c -- plain, sequential, fp64 reference of stochastic coordinate
 * descent/ascent for generalized linear models.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark use it.  It shares no code with the HIP library.
 *
 * Source: Parnell, Duenner, Atasu, Sifalakis, Pozidis, "Large-Scale Stochastic
 * Learning using GPUs" (arXiv 1702.07005).
 *   - Ridge primal objective: Sec. II-A, eq. (primal_obj).
 *   - Primal coordinate step and shared-vector update: Sec. II-A, eq. (update_primal)
 *     and the line that follows it.
 *   - Ridge dual objective and dual step: Sec. II-B, eqs. (dual_obj), (update_dual).
 *   - Duality gap: Sec. II-C (G_P, G_D built from eqs. duality-1/2).
 *   - Sequential SCD with a fresh random permutation per epoch: Sec. III-A, Alg. 1.
 *   - Hinge-loss SVM dual (SDCA-style box-constrained ascent): the paper names SVMs as
 *     another problem solved by stochastic coordinate methods (Sec. I) and takes its dual
 *     step from SDCA (Sec. II-B); the hinge dual below is derived from first principles:
 *       P(w) = (1/N) sum_i max(0, 1 - y_i x_i.w) + (lambda/2) |w|^2
 *       D(a) = (1/N) sum_i a_i - (lambda/2) |w(a)|^2,  w(a) = (1/(lambda N)) sum_i a_i y_i x_i,
 *       0 <= a_i <= 1; exact 1-D maximisation of D over a_i gives
 *       a_i <- clip(a_i + lambda N (1 - y_i x_i.w) / |x_i|^2, 0, 1).
 *
 * The visiting order is a keyed bijection of [0, C) per (seed, epoch); the paper only
 * says "generate random permutation" (Alg. 1, Alg. 2).  The construction (a 4-round
 * balanced Feistel network with cycle-walking, SplitMix64-derived round keys and the
 * MurmurHash3 32-bit finaliser as round function) is written out in full below.
 *
 * All arithmetic is IEEE double, except in oracle_epochs_f32 (a single-precision
 * copy of the epochs, for timing only).  fp32 inputs are promoted exactly.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Permutation of the coordinates (one per epoch).                            */
/* ------------------------------------------------------------------------- */

/* SplitMix64 output function (Steele, Lea, Flood, OOPSLA 2014): the generator's
 * state advances by the golden-ratio increment; each output is this mix of the state. */
static const uint64_t SM64_GAMMA = 0x9E3779B97F4A7C15ULL;

uint64_t oracle_splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* n-th output (n >= 1) of SplitMix64 started from state s. */
uint64_t oracle_splitmix64_nth(uint64_t s, uint64_t n)
{
    return oracle_splitmix64_mix(s + SM64_GAMMA * n);
}

/* MurmurHash3 32-bit finaliser (Appleby, public domain). */
uint32_t oracle_fmix32(uint32_t h)
{
    h ^= h >> 16;
    h *= 0x85EBCA6BU;
    h ^= h >> 13;
    h *= 0xC2B2AE35U;
    h ^= h >> 16;
    return h;
}

/* Round keys of epoch t: base = SplitMix64 output number t+1 from state seed;
 * key r = low 32 bits of SplitMix64 output number r+1 from state base. */
void oracle_perm_keys(uint64_t seed, uint64_t epoch, uint32_t keys[4])
{
    uint64_t base = oracle_splitmix64_nth(seed, epoch + 1);
    for (int r = 0; r < 4; ++r)
        keys[r] = (uint32_t)oracle_splitmix64_nth(base, (uint64_t)r + 1);
}

/* Half width h: the smallest h >= 1 with 2^(2h) >= C. */
int oracle_perm_half_bits(uint64_t C)
{
    int b = 0;
    while (b < 64 && ((uint64_t)1 << b) < C)
        ++b;
    int h = (b + 1) / 2;
    return h < 1 ? 1 : h;
}

/* One Feistel encryption of x in [0, 2^(2h)):
 *   (L, R) = (x >> h, x mod 2^h);  4 times: (L, R) <- (R, L xor (fmix32(R xor k_r) mod 2^h)). */
static uint64_t feistel_encrypt(uint64_t x, int h, const uint32_t keys[4])
{
    uint64_t mask = ((uint64_t)1 << h) - 1;
    uint64_t L = x >> h;
    uint64_t R = x & mask;
    for (int r = 0; r < 4; ++r) {
        uint64_t f = (uint64_t)oracle_fmix32((uint32_t)R ^ keys[r]) & mask;
        uint64_t newL = R;
        uint64_t newR = L ^ f;
        L = newL;
        R = newR;
    }
    return (L << h) | R;
}

/* pi_{seed,epoch}(j): apply the Feistel map until the value falls into [0, C)
 * (cycle-walking, Black & Rogaway 2002). */
uint64_t oracle_perm_at(uint64_t seed, uint64_t epoch, uint64_t C, uint64_t j)
{
    uint32_t keys[4];
    oracle_perm_keys(seed, epoch, keys);
    int h = oracle_perm_half_bits(C);
    uint64_t x = feistel_encrypt(j, h, keys);
    while (x >= C)
        x = feistel_encrypt(x, h, keys);
    return x;
}

/* The whole visiting order of one epoch: out[j] = pi(j), j = 0..C-1. */
void oracle_permutation(uint64_t seed, uint64_t epoch, int64_t C, int64_t *out)
{
    for (int64_t j = 0; j < C; ++j)
        out[j] = (int64_t)oracle_perm_at(seed, epoch, (uint64_t)C, (uint64_t)j);
}

/* ------------------------------------------------------------------------- */
/* Sparse segments.  A coordinate's data is one segment [ptr[c], ptr[c+1]) of   */
/* (idx, val): a column of A in CSC (primal), a row of A in CSR (dual).          */
/* ------------------------------------------------------------------------- */

/* |a_c|^2 for every coordinate: the denominator terms of eqs. (update_primal),
 * (update_dual) and of the hinge step. */
void oracle_norms(int64_t C, const int64_t *ptr, const float *val, double *out)
{
    for (int64_t c = 0; c < C; ++c) {
        double s = 0.0;
        for (int64_t k = ptr[c]; k < ptr[c + 1]; ++k)
            s += (double)val[k] * (double)val[k];
        out[c] = s;
    }
}

/* out[c] = <a_c, u> and cond[c] = sum |a_c| |u| over the segment (fp64). */
void oracle_gather_dots(int64_t C, const int64_t *ptr, const int32_t *idx, const float *val,
                        const float *u, double *out, double *cond)
{
    for (int64_t c = 0; c < C; ++c) {
        double s = 0.0, a = 0.0;
        for (int64_t k = ptr[c]; k < ptr[c + 1]; ++k) {
            double p = (double)val[k] * (double)u[idx[k]];
            s += p;
            a += fabs(p);
        }
        out[c] = s;
        if (cond)
            cond[c] = a;
    }
}

/* ------------------------------------------------------------------------- */
/* Ridge regression, primal form, A given by columns (CSC).                   */
/* ------------------------------------------------------------------------- */

/* Visit the coordinates coords[0..n) in order, each with the exact step of
 * eq. (update_primal):
 *   dbeta = (<y - w, a_m> - lambda N beta_m) / (|a_m|^2 + lambda N),
 *   beta_m += dbeta,  w += a_m dbeta      (w = A beta, the shared vector). */
void oracle_ridge_primal_visit(int64_t N, const int64_t *col_ptr, const int32_t *row_idx,
                               const float *val, const float *y, double lambda,
                               const int64_t *coords, int64_t n, const double *norms,
                               double *beta, double *w)
{
    double lN = lambda * (double)N;
    for (int64_t t = 0; t < n; ++t) {
        int64_t m = coords[t];
        double g = 0.0;
        for (int64_t k = col_ptr[m]; k < col_ptr[m + 1]; ++k)
            g += ((double)y[row_idx[k]] - w[row_idx[k]]) * (double)val[k];
        double d = (g - lN * beta[m]) / (norms[m] + lN);
        beta[m] += d;
        for (int64_t k = col_ptr[m]; k < col_ptr[m + 1]; ++k)
            w[row_idx[k]] += (double)val[k] * d;
    }
}

/* Alg. 1: n_epochs passes, epoch e (global index epoch0 + e) visiting pi_{seed,e}. */
void oracle_ridge_primal_epochs(int64_t N, int64_t M, const int64_t *col_ptr, const int32_t *row_idx,
                                const float *val, const float *y, double lambda, uint64_t seed,
                                int64_t epoch0, int32_t n_epochs, double *beta, double *w)
{
    double *norms = (double *)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1));
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(M > 0 ? M : 1));
    oracle_norms(M, col_ptr, val, norms);
    for (int32_t e = 0; e < n_epochs; ++e) {
        oracle_permutation(seed, (uint64_t)(epoch0 + e), M, order);
        oracle_ridge_primal_visit(N, col_ptr, row_idx, val, y, lambda, order, M, norms, beta, w);
    }
    free(order);
    free(norms);
}

/* ------------------------------------------------------------------------- */
/* Ridge regression, dual form, A given by rows (CSR).                        */
/* ------------------------------------------------------------------------- */

/* Eq. (update_dual), coordinate n:
 *   dalpha = (lambda y_n - <wbar, abar_n> - lambda N alpha_n) / (lambda N + |abar_n|^2),
 *   alpha_n += dalpha,  wbar += abar_n dalpha      (wbar = A^T alpha). */
void oracle_ridge_dual_visit(int64_t N, const int64_t *row_ptr, const int32_t *col_idx,
                             const float *val, const float *y, double lambda,
                             const int64_t *coords, int64_t n, const double *norms,
                             double *alpha, double *wbar)
{
    double lN = lambda * (double)N;
    for (int64_t t = 0; t < n; ++t) {
        int64_t i = coords[t];
        double g = 0.0;
        for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
            g += wbar[col_idx[k]] * (double)val[k];
        double d = (lambda * (double)y[i] - g - lN * alpha[i]) / (lN + norms[i]);
        alpha[i] += d;
        for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
            wbar[col_idx[k]] += (double)val[k] * d;
    }
}

void oracle_ridge_dual_epochs(int64_t N, int64_t M, const int64_t *row_ptr, const int32_t *col_idx,
                              const float *val, const float *y, double lambda, uint64_t seed,
                              int64_t epoch0, int32_t n_epochs, double *alpha, double *wbar)
{
    (void)M;
    double *norms = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
    oracle_norms(N, row_ptr, val, norms);
    for (int32_t e = 0; e < n_epochs; ++e) {
        oracle_permutation(seed, (uint64_t)(epoch0 + e), N, order);
        oracle_ridge_dual_visit(N, row_ptr, col_idx, val, y, lambda, order, N, norms, alpha, wbar);
    }
    free(order);
    free(norms);
}

/* ------------------------------------------------------------------------- */
/* Hinge-loss SVM, dual form, A given by rows (CSR), y in {-1, +1}.           */
/* ------------------------------------------------------------------------- */

/* Exact maximisation of D over alpha_i on [0, 1]:
 *   g = x_i.w;  a = clip(alpha_i + lambda N (1 - y_i g) / |x_i|^2, 0, 1);
 *   for |x_i| = 0, D is linear in alpha_i with slope 1/N, so a = 1;
 *   w += (a - alpha_i) y_i x_i / (lambda N);  alpha_i = a. */
void oracle_svm_dual_visit(int64_t N, const int64_t *row_ptr, const int32_t *col_idx,
                           const float *val, const float *y, double lambda,
                           const int64_t *coords, int64_t n, const double *norms,
                           double *alpha, double *w)
{
    double lN = lambda * (double)N;
    for (int64_t t = 0; t < n; ++t) {
        int64_t i = coords[t];
        double g = 0.0;
        for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
            g += w[col_idx[k]] * (double)val[k];
        double a;
        if (norms[i] > 0.0) {
            a = alpha[i] + lN * (1.0 - (double)y[i] * g) / norms[i];
            if (a < 0.0)
                a = 0.0;
            if (a > 1.0)
                a = 1.0;
        } else {
            a = 1.0;
        }
        double d = a - alpha[i];
        alpha[i] = a;
        double c = d * (double)y[i] / lN;
        for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
            w[col_idx[k]] += (double)val[k] * c;
    }
}

void oracle_svm_dual_epochs(int64_t N, int64_t M, const int64_t *row_ptr, const int32_t *col_idx,
                            const float *val, const float *y, double lambda, uint64_t seed,
                            int64_t epoch0, int32_t n_epochs, double *alpha, double *w)
{
    (void)M;
    double *norms = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
    oracle_norms(N, row_ptr, val, norms);
    for (int32_t e = 0; e < n_epochs; ++e) {
        oracle_permutation(seed, (uint64_t)(epoch0 + e), N, order);
        oracle_svm_dual_visit(N, row_ptr, col_idx, val, y, lambda, order, N, norms, alpha, w);
    }
    free(order);
    free(norms);
}

/* ------------------------------------------------------------------------- */
/* The same sequential epochs in single precision (timing reference).         */
/* ------------------------------------------------------------------------- */

/* The paper computes in single precision on the CPU and the GPU (Sec. III-A, III-C)
 * and quotes its speed-ups against one thread running Alg. 1.  This is Alg. 1 once
 * more, with the model, the shared vector, the norms and every operation in float,
 * so that that baseline can be timed; the correctness reference is the fp64 code
 * above.  form: 0 ridge primal (CSC columns), 1 hinge SVM dual (CSR rows),
 * 2 ridge dual (CSR rows).  The steps are those of the three visit functions above. */
void oracle_epochs_f32(int form, int64_t N, int64_t M, const int64_t *ptr, const int32_t *idx,
                       const float *val, const float *y, double lambda, uint64_t seed,
                       int64_t epoch0, int32_t n_epochs, float *model, float *shared)
{
    int64_t C = form == 0 ? M : N;
    float lN = (float)(lambda * (double)N);
    float lam = (float)lambda;
    float *norms = (float *)malloc(sizeof(float) * (size_t)(C > 0 ? C : 1));
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(C > 0 ? C : 1));
    for (int64_t c = 0; c < C; ++c) {
        float s = 0.0f;
        for (int64_t k = ptr[c]; k < ptr[c + 1]; ++k)
            s += val[k] * val[k];
        norms[c] = s;
    }
    for (int32_t e = 0; e < n_epochs; ++e) {
        oracle_permutation(seed, (uint64_t)(epoch0 + e), C, order);
        for (int64_t t = 0; t < C; ++t) {
            int64_t m = order[t];
            float g = 0.0f, coef;
            if (form == 0) {
                for (int64_t k = ptr[m]; k < ptr[m + 1]; ++k)
                    g += (y[idx[k]] - shared[idx[k]]) * val[k];
                float d = (g - lN * model[m]) / (norms[m] + lN);
                model[m] += d;
                coef = d;
            } else if (form == 1) {
                for (int64_t k = ptr[m]; k < ptr[m + 1]; ++k)
                    g += shared[idx[k]] * val[k];
                float a = 1.0f;
                if (norms[m] > 0.0f) {
                    a = model[m] + lN * (1.0f - y[m] * g) / norms[m];
                    if (a < 0.0f)
                        a = 0.0f;
                    if (a > 1.0f)
                        a = 1.0f;
                }
                coef = (a - model[m]) * y[m] / lN;
                model[m] = a;
            } else {
                for (int64_t k = ptr[m]; k < ptr[m + 1]; ++k)
                    g += shared[idx[k]] * val[k];
                float d = (lam * y[m] - g - lN * model[m]) / (lN + norms[m]);
                model[m] += d;
                coef = d;
            }
            for (int64_t k = ptr[m]; k < ptr[m + 1]; ++k)
                shared[idx[k]] += val[k] * coef;
        }
    }
    free(order);
    free(norms);
}

/* ------------------------------------------------------------------------- */
/* Objectives and duality gaps.                                                */
/* ------------------------------------------------------------------------- */

/* Ridge, model beta in R^M, A in CSC.  If w is NULL, w = A beta is recomputed fresh;
 * otherwise the given shared vector stands in for A beta.
 *   P(beta)  = 1/(2N) |A beta - y|^2 + lambda/2 |beta|^2                 (primal_obj)
 *   alpha    = (y - A beta) / N                                          (duality-2)
 *   D(alpha) = -N/2 |alpha|^2 - 1/(2 lambda) |A^T alpha|^2 + alpha^T y    (dual_obj)
 *   G_P      = |P - D|                                                   (Sec. II-C) */
void oracle_ridge_primal_objectives(int64_t N, int64_t M, const int64_t *col_ptr,
                                    const int32_t *row_idx, const float *val, const float *y,
                                    double lambda, const double *beta, const double *w_in,
                                    double *primal, double *dual, double *gap)
{
    double *w = (double *)calloc((size_t)(N > 0 ? N : 1), sizeof(double));
    if (w_in) {
        memcpy(w, w_in, sizeof(double) * (size_t)N);
    } else {
        for (int64_t m = 0; m < M; ++m)
            for (int64_t k = col_ptr[m]; k < col_ptr[m + 1]; ++k)
                w[row_idx[k]] += (double)val[k] * beta[m];
    }
    double res2 = 0.0, beta2 = 0.0, a2 = 0.0, ay = 0.0, ata2 = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        double r = w[i] - (double)y[i];
        res2 += r * r;
        double a = ((double)y[i] - w[i]) / (double)N;
        a2 += a * a;
        ay += a * (double)y[i];
    }
    for (int64_t m = 0; m < M; ++m) {
        beta2 += beta[m] * beta[m];
        double d = 0.0;
        for (int64_t k = col_ptr[m]; k < col_ptr[m + 1]; ++k)
            d += (double)val[k] * ((double)y[row_idx[k]] - w[row_idx[k]]) / (double)N;
        ata2 += d * d;
    }
    double P = res2 / (2.0 * (double)N) + 0.5 * lambda * beta2;
    double D = -0.5 * (double)N * a2 - ata2 / (2.0 * lambda) + ay;
    if (primal)
        *primal = P;
    if (dual)
        *dual = D;
    if (gap)
        *gap = fabs(P - D);
    free(w);
}

/* Ridge, dual model alpha in R^N, A in CSR.  wbar = A^T alpha (fresh if wbar_in is NULL).
 *   beta = A^T alpha / lambda                                             (duality-1)
 *   G_D  = |P(beta) - D(alpha)|                                           (Sec. II-C) */
void oracle_ridge_dual_objectives(int64_t N, int64_t M, const int64_t *row_ptr,
                                  const int32_t *col_idx, const float *val, const float *y,
                                  double lambda, const double *alpha, const double *wbar_in,
                                  double *primal, double *dual, double *gap)
{
    double *wbar = (double *)calloc((size_t)(M > 0 ? M : 1), sizeof(double));
    if (wbar_in) {
        memcpy(wbar, wbar_in, sizeof(double) * (size_t)M);
    } else {
        for (int64_t i = 0; i < N; ++i)
            for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
                wbar[col_idx[k]] += (double)val[k] * alpha[i];
    }
    double a2 = 0.0, ay = 0.0, wb2 = 0.0, res2 = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        a2 += alpha[i] * alpha[i];
        ay += alpha[i] * (double)y[i];
    }
    for (int64_t m = 0; m < M; ++m)
        wb2 += wbar[m] * wbar[m];
    /* A beta with beta = wbar / lambda, row by row. */
    for (int64_t i = 0; i < N; ++i) {
        double ab = 0.0;
        for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
            ab += (double)val[k] * wbar[col_idx[k]] / lambda;
        double r = ab - (double)y[i];
        res2 += r * r;
    }
    double beta2 = wb2 / (lambda * lambda);
    double P = res2 / (2.0 * (double)N) + 0.5 * lambda * beta2;
    double D = -0.5 * (double)N * a2 - wb2 / (2.0 * lambda) + ay;
    if (primal)
        *primal = P;
    if (dual)
        *dual = D;
    if (gap)
        *gap = fabs(P - D);
    free(wbar);
}

/* Hinge SVM, dual model alpha in [0,1]^N, A in CSR.  w = w(alpha) (fresh if w_in is NULL).
 *   P(w) = (1/N) sum_i max(0, 1 - y_i x_i.w) + lambda/2 |w|^2
 *   D(a) = (1/N) sum_i a_i - lambda/2 |w|^2
 *   G    = P - D  (non-negative by weak duality). */
void oracle_svm_dual_objectives(int64_t N, int64_t M, const int64_t *row_ptr,
                                const int32_t *col_idx, const float *val, const float *y,
                                double lambda, const double *alpha, const double *w_in,
                                double *primal, double *dual, double *gap)
{
    double lN = lambda * (double)N;
    double *w = (double *)calloc((size_t)(M > 0 ? M : 1), sizeof(double));
    if (w_in) {
        memcpy(w, w_in, sizeof(double) * (size_t)M);
    } else {
        for (int64_t i = 0; i < N; ++i)
            for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
                w[col_idx[k]] += (double)val[k] * alpha[i] * (double)y[i] / lN;
    }
    double hinge = 0.0, asum = 0.0, w2 = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        double g = 0.0;
        for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k)
            g += (double)val[k] * w[col_idx[k]];
        double l = 1.0 - (double)y[i] * g;
        hinge += l > 0.0 ? l : 0.0;
        asum += alpha[i];
    }
    for (int64_t m = 0; m < M; ++m)
        w2 += w[m] * w[m];
    double P = hinge / (double)N + 0.5 * lambda * w2;
    double D = asum / (double)N - 0.5 * lambda * w2;
    if (primal)
        *primal = P;
    if (dual)
        *dual = D;
    if (gap)
        *gap = P - D;
    free(w);
}
