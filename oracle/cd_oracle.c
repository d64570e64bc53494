/*
 * COUNTDOWN sparse Gated-MLP FFN -- CPU reference oracle, fp64.
 *
 * TEST INFRASTRUCTURE ONLY. The test suite, the smoke check and the
 * bench's CPU-baseline leg are the only callers. The product path never
 * loads this library, and the oracle shares no code, header, table or
 * helper with the HIP kernels.
 *
 * Every routine is a plain loop over the paper's definitions
 * (arXiv 2505.17701, "COUNTDOWN"):
 *   Sec. 3 "Problem Formulation": u = x.W_up, h = sigma(x.W_gate), s = u (.) h;
 *   Eq. (1) dense Gated-MLP;  Eq. (2)-(3) sparse evaluation on an index set;
 *   Eq. (5) y as a linear combination of the rows of W_down^T;
 *   Eq. (6b) M-CountDown index set {i : |u[i]| > tau_M};
 *   Eq. (6c) D-CountDown index set {i : |s[i]| > tau_D};
 *   Eq. (6a) CATS index set {i : |h[i]| > tau_C} (comparison baseline);
 *   Sec. 4 "Constructing SP^Prac": layerwise constant threshold
 *     tau_hat = (1/T) sum_t Quantile(k, |u^(t)|) and the low-rank predictor
 *     s_hat = x.theta_A.theta_B with predicted set {i : s_hat[i] > tau};
 *   Sec. 6 "Possible Predictor Candidate: TernaryLinear" (Table 4): the
 *     predictor score s_hat = x.theta with theta in {-1, 0, +1}, thresholded
 *     like the low-rank score;
 *   Limitations section: batch > 1 takes the union of the index sets;
 *   the per-token form of Eq. (6): each token's threshold is the quantile of
 *   its own coefficients (cdo_ffn_topk).
 *
 * Inputs are the exact bf16 values the GPU consumes (uint16 bit patterns),
 * widened exactly to double; thresholds arrive as the fp32 value the GPU
 * gets, widened to double. All arithmetic is double. Sums run in ascending
 * index order. Matrices are neuron-major [d_ff][d_model] row-major (row i is
 * the weight vector of intermediate neuron i); the predictor is A_t
 * [d_rank][d_model] and B_t [d_ff][d_rank]; the ternary predictor is int8
 * theta_t [d_ff][d_model] (theta transposed, entries -1, 0, +1).
 *
 * Readings of points the paper leaves open (strict '>' of Eq. (6) rather
 * than the listings' '>=', linear-interpolation quantiles, mean of
 * per-token quantiles, fp64 intermediates, union over a batch) are the
 * ones documented with the project design notes.
 *
 * OpenMP only splits loops over independent rows or output columns; the
 * result does not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define CDO_OK 0
#define CDO_EINVAL (-1)
#define CDO_ENOMEM (-2)

enum {
    CDO_COEF_ABS_U = 0,
    CDO_COEF_ABS_S = 1,
    CDO_COEF_SHAT = 2,
    CDO_COEF_ABS_H = 3,
    CDO_COEF_TERN = 4
};

/* exact widening of a bf16 bit pattern */
static double wide(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int cdo_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* threads of the following calls (timing only; results do not depend on it) */
void cdo_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* SiLU(z) = z * sigmoid(z) = z / (1 + e^-z), the activation of Sec. 3
 * (sigma = SiLU). For z < 0 the form z e^z / (1 + e^z) avoids e^-z overflow. */
double cdo_silu(double z)
{
    if (z >= 0.0)
        return z / (1.0 + exp(-z));
    double e = exp(z);
    return z * e / (1.0 + e);
}

/* out[i] = sum_j v[j] * W[i][j]: the vector-matrix product v.W of Sec. 3
 * with W stored neuron-major (W[i] = the i-th column of the paper's matrix). */
static void project_bf16(const uint16_t *v, const uint16_t *W, int64_t rows, int64_t cols,
                         double *out)
{
    double *vd = (double *)malloc(sizeof(double) * (size_t)cols);
    for (int64_t j = 0; j < cols; j++)
        vd[j] = wide(v[j]);
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < rows; i++) {
        const uint16_t *w = W + i * cols;
        double acc = 0.0;
        for (int64_t j = 0; j < cols; j++)
            acc += vd[j] * wide(w[j]);
        out[i] = acc;
    }
    free(vd);
}

/* same product with a double left operand (the latent of the predictor) */
static void project_f64(const double *v, const uint16_t *W, int64_t rows, int64_t cols,
                        double *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < rows; i++) {
        const uint16_t *w = W + i * cols;
        double acc = 0.0;
        for (int64_t j = 0; j < cols; j++)
            acc += v[j] * wide(w[j]);
        out[i] = acc;
    }
}

/* one row-dot x . W[i] (used for the index-restricted products of Eq. (2)) */
static double row_dot(const uint16_t *x, const uint16_t *W, int64_t i, int64_t cols)
{
    const uint16_t *w = W + i * cols;
    double acc = 0.0;
    for (int64_t j = 0; j < cols; j++)
        acc += wide(x[j]) * wide(w[j]);
    return acc;
}

/* Sec. 3: u = x.W_up, g = x.W_gate (the pre-activation h_pre), s = u (.) SiLU(g),
 * for B tokens. Any output pointer may be NULL. Arrays are [B][d_ff]. */
int cdo_coefficients(const uint16_t *x, int B, const uint16_t *W_gate, const uint16_t *W_up,
                     int d_model, int d_ff, double *u, double *g, double *s)
{
    if (!x || !W_gate || !W_up || B < 1 || d_model < 1 || d_ff < 1)
        return CDO_EINVAL;
    double *uu = (double *)malloc(sizeof(double) * (size_t)d_ff);
    double *gg = (double *)malloc(sizeof(double) * (size_t)d_ff);
    if (!uu || !gg) {
        free(uu);
        free(gg);
        return CDO_ENOMEM;
    }
    for (int b = 0; b < B; b++) {
        const uint16_t *xb = x + (int64_t)b * d_model;
        project_bf16(xb, W_up, d_ff, d_model, uu);
        project_bf16(xb, W_gate, d_ff, d_model, gg);
        for (int64_t i = 0; i < d_ff; i++) {
            if (u) u[(int64_t)b * d_ff + i] = uu[i];
            if (g) g[(int64_t)b * d_ff + i] = gg[i];
            if (s) s[(int64_t)b * d_ff + i] = uu[i] * cdo_silu(gg[i]);
        }
    }
    free(uu);
    free(gg);
    return CDO_OK;
}

/* Sec. 4: the low-rank predictor score s_hat = (x.theta_A).theta_B for B tokens.
 * latent [B][d_rank] and shat [B][d_ff]; latent may be NULL. */
int cdo_predictor(const uint16_t *x, int B, const uint16_t *A_t, const uint16_t *B_t,
                  int d_model, int d_rank, int d_ff, double *latent, double *shat)
{
    if (!x || !A_t || !B_t || !shat || B < 1 || d_model < 1 || d_rank < 1 || d_ff < 1)
        return CDO_EINVAL;
    double *l = (double *)malloc(sizeof(double) * (size_t)d_rank);
    if (!l)
        return CDO_ENOMEM;
    for (int b = 0; b < B; b++) {
        project_bf16(x + (int64_t)b * d_model, A_t, d_rank, d_model, l);
        if (latent)
            memcpy(latent + (int64_t)b * d_rank, l, sizeof(double) * (size_t)d_rank);
        project_f64(l, B_t, d_ff, d_rank, shat + (int64_t)b * d_ff);
    }
    free(l);
    return CDO_OK;
}

/* Sec. 6, TernaryLinear: s_hat_b[i] = sum_j x_b[j] theta[j][i], theta in {-1, 0, +1},
 * given transposed as theta_t [d_ff][d_model]; shat [B][d_ff]. Entries outside
 * {-1, 0, +1} are rejected. */
int cdo_ternary_predictor(const uint16_t *x, int B, const int8_t *theta_t, int d_model, int d_ff,
                          double *shat)
{
    if (!x || !theta_t || !shat || B < 1 || d_model < 1 || d_ff < 1)
        return CDO_EINVAL;
    for (int64_t e = 0; e < (int64_t)d_ff * d_model; e++)
        if (theta_t[e] < -1 || theta_t[e] > 1)
            return CDO_EINVAL;
    for (int b = 0; b < B; b++) {
        const uint16_t *xb = x + (int64_t)b * d_model;
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < d_ff; i++) {
            double t = 0.0;
            for (int64_t j = 0; j < d_model; j++)
                t += wide(xb[j]) * (double)theta_t[i * d_model + j];
            shat[(int64_t)b * d_ff + i] = t;
        }
    }
    return CDO_OK;
}

/* Eq. (6) with a constant threshold, and the union over a batch: IDX holds
 * every i for which some token b has coefficient c_b[i] > thld, in ascending
 * order. use_abs selects |c| (Eq. 6a-6c) or the signed score (predictor).
 * Returns |IDX|, or a negative error. */
int64_t cdo_select(const double *c, int B, int64_t d_ff, int use_abs, double thld, int32_t *idx)
{
    if (!c || !idx || B < 1 || d_ff < 1 || isnan(thld))
        return CDO_EINVAL;
    int64_t n = 0;
    for (int64_t i = 0; i < d_ff; i++) {
        int keep = 0;
        for (int b = 0; b < B; b++) {
            double v = c[(int64_t)b * d_ff + i];
            if (use_abs)
                v = fabs(v);
            if (v > thld)
                keep = 1;
        }
        if (keep)
            idx[n++] = (int32_t)i;
    }
    return n;
}

/* Eq. (5) restricted to an index set: y_b = sum over t of s_b[idx[t]] * W_down^T[idx[t]],
 * summed in the order of idx. s is [B][d_ff], y is [B][d_model]. */
int cdo_combine(const double *s, int B, int64_t d_ff, const uint16_t *W_down, int d_model,
                const int32_t *idx, int64_t n, double *y)
{
    if (!s || !W_down || !y || B < 1 || d_ff < 1 || d_model < 1 || n < 0 || (n > 0 && !idx))
        return CDO_EINVAL;
    for (int64_t t = 0; t < n; t++)
        if (idx[t] < 0 || idx[t] >= d_ff)
            return CDO_EINVAL;
    for (int b = 0; b < B; b++) {
        const double *sb = s + (int64_t)b * d_ff;
        double *yb = y + (int64_t)b * d_model;
        #pragma omp parallel for schedule(static)
        for (int64_t j = 0; j < d_model; j++) {
            double acc = 0.0;
            for (int64_t t = 0; t < n; t++)
                acc += sb[idx[t]] * wide(W_down[(int64_t)idx[t] * d_model + j]);
            yb[j] = acc;
        }
    }
    return CDO_OK;
}

/* Eq. (1): the dense Gated-MLP y = ((x.W_up) (.) SiLU(x.W_gate)) . W_down^T,
 * every neuron in ascending order. y is [B][d_model]. */
int cdo_dense(const uint16_t *x, int B, const uint16_t *W_gate, const uint16_t *W_up,
              const uint16_t *W_down, int d_model, int d_ff, double *y)
{
    if (!x || !W_gate || !W_up || !W_down || !y || B < 1 || d_model < 1 || d_ff < 1)
        return CDO_EINVAL;
    double *s = (double *)malloc(sizeof(double) * (size_t)d_ff);
    if (!s)
        return CDO_ENOMEM;
    for (int b = 0; b < B; b++) {
        const uint16_t *xb = x + (int64_t)b * d_model;
        #pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < d_ff; i++) {
            double uu = row_dot(xb, W_up, i, d_model);
            double gg = row_dot(xb, W_gate, i, d_model);
            s[i] = uu * cdo_silu(gg);
        }
        double *yb = y + (int64_t)b * d_model;
        #pragma omp parallel for schedule(static)
        for (int64_t j = 0; j < d_model; j++) {
            double acc = 0.0;
            for (int64_t i = 0; i < d_ff; i++)
                acc += s[i] * wide(W_down[i * d_model + j]);
            yb[j] = acc;
        }
    }
    free(s);
    return CDO_OK;
}

/* Eq. (2)-(3) on a given index set: gate and up are evaluated only on the
 * rows in idx (W^I = W[:, IDX]), then Eq. (5) over idx. s_c (optional) gets
 * the coefficients s_b[idx[t]] as [B][n]. */
int cdo_ffn_on_idx(const uint16_t *x, int B, const uint16_t *W_gate, const uint16_t *W_up,
                   const uint16_t *W_down, int d_model, int d_ff, const int32_t *idx, int64_t n,
                   double *y, double *s_c)
{
    if (!x || !W_gate || !W_up || !W_down || !y || B < 1 || d_model < 1 || d_ff < 1 || n < 0 ||
        (n > 0 && !idx))
        return CDO_EINVAL;
    for (int64_t t = 0; t < n; t++)
        if (idx[t] < 0 || idx[t] >= d_ff)
            return CDO_EINVAL;
    double *s = (double *)calloc((size_t)B * (size_t)d_ff, sizeof(double));
    if (!s)
        return CDO_ENOMEM;
    for (int b = 0; b < B; b++) {
        const uint16_t *xb = x + (int64_t)b * d_model;
        #pragma omp parallel for schedule(static)
        for (int64_t t = 0; t < n; t++) {
            int64_t i = idx[t];
            double uu = row_dot(xb, W_up, i, d_model);
            double gg = row_dot(xb, W_gate, i, d_model);
            s[(int64_t)b * d_ff + i] = uu * cdo_silu(gg);
        }
        if (s_c)
            for (int64_t t = 0; t < n; t++)
                s_c[(int64_t)b * n + t] = s[(int64_t)b * d_ff + idx[t]];
    }
    int rc = cdo_combine(s, B, d_ff, W_down, d_model, idx, n, y);
    free(s);
    return rc;
}

/* M-CountDown (Eq. 6b, Sec. 4): u = x.W_up densely; IDX = {i : exists b, |u_b[i]| > thld};
 * gate only on IDX; y by Eq. (5). coef (optional) receives u [B][d_ff].
 * Returns |IDX| or a negative error; idx must hold d_ff entries. */
int64_t cdo_ffn_mono(const uint16_t *x, int B, const uint16_t *W_gate, const uint16_t *W_up,
                     const uint16_t *W_down, int d_model, int d_ff, double thld, int32_t *idx,
                     double *y, double *coef)
{
    if (!x || !W_gate || !W_up || !W_down || !y || !idx || B < 1 || d_model < 1 || d_ff < 1 ||
        isnan(thld))
        return CDO_EINVAL;
    double *u = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d_ff);
    if (!u)
        return CDO_ENOMEM;
    for (int b = 0; b < B; b++)
        project_bf16(x + (int64_t)b * d_model, W_up, d_ff, d_model, u + (int64_t)b * d_ff);
    if (coef)
        memcpy(coef, u, sizeof(double) * (size_t)B * (size_t)d_ff);
    int64_t n = cdo_select(u, B, d_ff, 1, thld, idx);
    free(u);
    if (n < 0)
        return n;
    int rc = cdo_ffn_on_idx(x, B, W_gate, W_up, W_down, d_model, d_ff, idx, n, y, NULL);
    return rc < 0 ? rc : n;
}

/* CATS, the comparison method (Eq. 6a): h = SiLU(x.W_gate) densely;
 * IDX = {i : exists b, |h_b[i]| > thld}; up only on IDX; y by Eq. (5).
 * coef (optional) receives h [B][d_ff]. Returns |IDX| or a negative error. */
int64_t cdo_ffn_cats(const uint16_t *x, int B, const uint16_t *W_gate, const uint16_t *W_up,
                     const uint16_t *W_down, int d_model, int d_ff, double thld, int32_t *idx,
                     double *y, double *coef)
{
    if (!x || !W_gate || !W_up || !W_down || !y || !idx || B < 1 || d_model < 1 || d_ff < 1 ||
        isnan(thld))
        return CDO_EINVAL;
    double *h = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d_ff);
    if (!h)
        return CDO_ENOMEM;
    for (int b = 0; b < B; b++) {
        double *hb = h + (int64_t)b * d_ff;
        project_bf16(x + (int64_t)b * d_model, W_gate, d_ff, d_model, hb);
        for (int64_t i = 0; i < d_ff; i++)
            hb[i] = cdo_silu(hb[i]);
    }
    if (coef)
        memcpy(coef, h, sizeof(double) * (size_t)B * (size_t)d_ff);
    int64_t n = cdo_select(h, B, d_ff, 1, thld, idx);
    free(h);
    if (n < 0)
        return n;
    int rc = cdo_ffn_on_idx(x, B, W_gate, W_up, W_down, d_model, d_ff, idx, n, y, NULL);
    return rc < 0 ? rc : n;
}

/* D-CountDown, ideal (Eq. 6c): s computed densely; IDX = {i : exists b, |s_b[i]| > thld};
 * y by Eq. (5) over IDX. coef (optional) receives s [B][d_ff]. */
int64_t cdo_ffn_dual_ideal(const uint16_t *x, int B, const uint16_t *W_gate,
                           const uint16_t *W_up, const uint16_t *W_down, int d_model, int d_ff,
                           double thld, int32_t *idx, double *y, double *coef)
{
    if (!x || !W_gate || !W_up || !W_down || !y || !idx || B < 1 || d_model < 1 || d_ff < 1 ||
        isnan(thld))
        return CDO_EINVAL;
    double *s = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d_ff);
    if (!s)
        return CDO_ENOMEM;
    int rc = cdo_coefficients(x, B, W_gate, W_up, d_model, d_ff, NULL, NULL, s);
    if (rc < 0) {
        free(s);
        return rc;
    }
    if (coef)
        memcpy(coef, s, sizeof(double) * (size_t)B * (size_t)d_ff);
    int64_t n = cdo_select(s, B, d_ff, 1, thld, idx);
    if (n >= 0)
        rc = cdo_combine(s, B, d_ff, W_down, d_model, idx, n, y);
    free(s);
    if (n < 0)
        return n;
    return rc < 0 ? rc : n;
}

/* D-CountDown, practical (Sec. 4): the predictor score s_hat decides
 * IDX = {i : exists b, s_hat_b[i] > thld} (signed); gate and up only on IDX;
 * y by Eq. (5). coef (optional) receives s_hat [B][d_ff]. */
int64_t cdo_ffn_dual_pred(const uint16_t *x, int B, const uint16_t *W_gate,
                          const uint16_t *W_up, const uint16_t *W_down, const uint16_t *A_t,
                          const uint16_t *B_t, int d_model, int d_rank, int d_ff, double thld,
                          int32_t *idx, double *y, double *coef)
{
    if (!x || !W_gate || !W_up || !W_down || !A_t || !B_t || !y || !idx || B < 1 ||
        d_model < 1 || d_rank < 1 || d_ff < 1 || isnan(thld))
        return CDO_EINVAL;
    double *sh = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d_ff);
    if (!sh)
        return CDO_ENOMEM;
    int rc = cdo_predictor(x, B, A_t, B_t, d_model, d_rank, d_ff, NULL, sh);
    if (rc < 0) {
        free(sh);
        return rc;
    }
    if (coef)
        memcpy(coef, sh, sizeof(double) * (size_t)B * (size_t)d_ff);
    int64_t n = cdo_select(sh, B, d_ff, 0, thld, idx);
    free(sh);
    if (n < 0)
        return n;
    rc = cdo_ffn_on_idx(x, B, W_gate, W_up, W_down, d_model, d_ff, idx, n, y, NULL);
    return rc < 0 ? rc : n;
}

/* D-CountDown with the ternary predictor (Sec. 6): IDX = {i : exists b,
 * s_hat_b[i] > thld} with s_hat = x.theta (signed); gate and up only on IDX;
 * y by Eq. (5). coef (optional) receives s_hat [B][d_ff]. */
int64_t cdo_ffn_dual_tern(const uint16_t *x, int B, const uint16_t *W_gate,
                          const uint16_t *W_up, const uint16_t *W_down, const int8_t *theta_t,
                          int d_model, int d_ff, double thld, int32_t *idx, double *y,
                          double *coef)
{
    if (!x || !W_gate || !W_up || !W_down || !theta_t || !y || !idx || B < 1 || d_model < 1 ||
        d_ff < 1 || isnan(thld))
        return CDO_EINVAL;
    double *sh = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d_ff);
    if (!sh)
        return CDO_ENOMEM;
    int rc = cdo_ternary_predictor(x, B, theta_t, d_model, d_ff, sh);
    if (rc < 0) {
        free(sh);
        return rc;
    }
    if (coef)
        memcpy(coef, sh, sizeof(double) * (size_t)B * (size_t)d_ff);
    int64_t n = cdo_select(sh, B, d_ff, 0, thld, idx);
    free(sh);
    if (n < 0)
        return n;
    rc = cdo_ffn_on_idx(x, B, W_gate, W_up, W_down, d_model, d_ff, idx, n, y, NULL);
    return rc < 0 ? rc : n;
}

static int cmp_double(const void *a, const void *b)
{
    double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

/* Quantile(k, v) of Sec. 3 with linear interpolation between order
 * statistics: sorted v, h = k (n - 1), q = v[floor h] + (h - floor h)(v[floor h + 1] - v[floor h]). */
double cdo_quantile_linear(double k, const double *v, int64_t n)
{
    if (!v || n < 1 || !(k >= 0.0 && k <= 1.0))
        return NAN;
    double *w = (double *)malloc(sizeof(double) * (size_t)n);
    if (!w)
        return NAN;
    memcpy(w, v, sizeof(double) * (size_t)n);
    qsort(w, (size_t)n, sizeof(double), cmp_double);
    double h = k * (double)(n - 1);
    int64_t lo = (int64_t)floor(h);
    if (lo >= n - 1)
        lo = n - 1;
    double q = w[lo];
    if (lo + 1 < n)
        q = w[lo] + (h - (double)lo) * (w[lo + 1] - w[lo]);
    free(w);
    return q;
}

/* Per-token coefficient vector for calibration: |u| (M, Eq. 6b), |s| (D ideal,
 * Eq. 6c), s_hat signed (low-rank predictor, Sec. 4; ternary predictor, Sec. 6)
 * or |h| = |SiLU(x.W_gate)| (CATS, Eq. 6a). */
static int token_coef(int kind, const uint16_t *x, const uint16_t *W_gate, const uint16_t *W_up,
                      const uint16_t *A_t, const uint16_t *B_t, const int8_t *theta_t,
                      int d_model, int d_rank, int d_ff, double *c)
{
    int rc;
    if (kind == CDO_COEF_SHAT)
        return cdo_predictor(x, 1, A_t, B_t, d_model, d_rank, d_ff, NULL, c);
    if (kind == CDO_COEF_TERN)
        return cdo_ternary_predictor(x, 1, theta_t, d_model, d_ff, c);
    if (kind == CDO_COEF_ABS_U) {
        if (!W_up)
            return CDO_EINVAL;
        project_bf16(x, W_up, d_ff, d_model, c);
    } else if (kind == CDO_COEF_ABS_S) {
        rc = cdo_coefficients(x, 1, W_gate, W_up, d_model, d_ff, NULL, NULL, c);
        if (rc < 0)
            return rc;
    } else if (kind == CDO_COEF_ABS_H) {
        if (!W_gate)
            return CDO_EINVAL;
        project_bf16(x, W_gate, d_ff, d_model, c);
        for (int64_t i = 0; i < d_ff; i++)
            c[i] = cdo_silu(c[i]);
    } else {
        return CDO_EINVAL;
    }
    for (int64_t i = 0; i < d_ff; i++)
        c[i] = fabs(c[i]);
    return CDO_OK;
}

/* Sec. 4 calibration: tau_hat = (1/T) sum_t Quantile(k, c^(t)) over T tokens,
 * c^(t) the coefficient vector of token t for the chosen variant. q_out
 * (optional) receives the T per-token quantiles. The mean is summed in token
 * order. Returns NAN on bad arguments. */
double cdo_calibrate(int kind, const uint16_t *X, int T, const uint16_t *W_gate,
                     const uint16_t *W_up, const uint16_t *A_t, const uint16_t *B_t, int d_model,
                     int d_rank, int d_ff, double k, double *q_out, const int8_t *theta_t)
{
    if (!X || T < 1 || d_model < 1 || d_ff < 1 || !(k >= 0.0 && k <= 1.0))
        return NAN;
    double *c = (double *)malloc(sizeof(double) * (size_t)d_ff);
    if (!c)
        return NAN;
    double sum = 0.0;
    for (int t = 0; t < T; t++) {
        if (token_coef(kind, X + (int64_t)t * d_model, W_gate, W_up, A_t, B_t, theta_t, d_model,
                       d_rank, d_ff, c) < 0) {
            free(c);
            return NAN;
        }
        double q = cdo_quantile_linear(k, c, d_ff);
        if (q_out)
            q_out[t] = q;
        sum += q;
    }
    free(c);
    return sum / (double)T;
}

/* Per-token threshold: Eq. (6) with each token's threshold taken as the
 * quantile of its own coefficient vector (the ideal, per-token form of the
 * sparsity definition, Sec. 3; Sec. 4 replaces it by the calibrated mean):
 *   thld_b = Quantile(k, c_b),  IDX = {i : exists b, c_b[i] > thld_b},
 * c_b the variant's coefficient vector of token b (kind as in cdo_calibrate:
 * |u|, |s|, signed s_hat of either predictor, or |h|), union over the batch; y by Eq. (5) over IDX
 * with the dense-equivalent s. q_out (optional) receives the B thresholds.
 * Returns |IDX| or a negative status. */
int64_t cdo_ffn_topk(int kind, const uint16_t *x, int B, const uint16_t *W_gate,
                     const uint16_t *W_up, const uint16_t *W_down, const uint16_t *A_t,
                     const uint16_t *B_t, int d_model, int d_rank, int d_ff, double k,
                     int32_t *idx, double *y, double *q_out, const int8_t *theta_t)
{
    if (!x || !W_gate || !W_up || !W_down || !idx || !y || B < 1 || d_model < 1 || d_ff < 1 ||
        !(k >= 0.0 && k <= 1.0))
        return CDO_EINVAL;
    double *c = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d_ff);
    double *q = (double *)malloc(sizeof(double) * (size_t)B);
    if (!c || !q) {
        free(c);
        free(q);
        return CDO_ENOMEM;
    }
    for (int b = 0; b < B; b++) {
        double *cb = c + (int64_t)b * d_ff;
        int rc = token_coef(kind, x + (int64_t)b * d_model, W_gate, W_up, A_t, B_t, theta_t,
                            d_model, d_rank, d_ff, cb);
        if (rc < 0) {
            free(c);
            free(q);
            return rc;
        }
        q[b] = cdo_quantile_linear(k, cb, d_ff);
    }
    int64_t n = 0;
    for (int64_t i = 0; i < d_ff; i++) {
        int keep = 0;
        for (int b = 0; b < B; b++)
            if (c[(int64_t)b * d_ff + i] > q[b])
                keep = 1;
        if (keep)
            idx[n++] = (int32_t)i;
    }
    free(c);
    int rc = cdo_ffn_on_idx(x, B, W_gate, W_up, W_down, d_model, d_ff, idx, n, y, NULL);
    if (rc >= 0 && q_out)
        for (int b = 0; b < B; b++)
            q_out[b] = q[b];
    free(q);
    return rc < 0 ? rc : n;
}

/* Residual + RMSNorm between stacked layers (not part of the paper; used by the
 * 32-layer stack workload): h += y; r = h / sqrt(mean(h^2) + eps) (gain 1).
 * h is updated in place, r receives the normalised vector. */
int cdo_residual_rmsnorm(double *h, const double *y, int d_model, double eps, double *r)
{
    if (!h || !r || d_model < 1 || !(eps >= 0.0))
        return CDO_EINVAL;
    if (y)
        for (int64_t j = 0; j < d_model; j++)
            h[j] += y[j];
    double ss = 0.0;
    for (int64_t j = 0; j < d_model; j++)
        ss += h[j] * h[j];
    double inv = 1.0 / sqrt(ss / (double)d_model + eps);
    for (int64_t j = 0; j < d_model; j++)
        r[j] = h[j] * inv;
    return CDO_OK;
}
