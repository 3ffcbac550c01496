/*
 * QuantEase CPU oracle (arXiv 2309.01885) -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, double-precision loops that restate the paper's definitions and
 * algorithm steps.  Only tests/, the smoke check and the benchmark's CPU-baseline
 * leg may load this library; the product path never does.  It shares no source,
 * header, table or helper with the HIP library.
 *
 * Notation follows the paper (Sec. 2.1, "Problem Formulation: Layerwise Quantization"):
 *   W  (q x p)  layer weights, row-major;  X (p x n) layer input;
 *   Sigma = X X^T (p x p);  What = the quantized weights;
 *   per-row grid Q_i = { s_i (k - z_i) : k = 0 .. 2^b - 1 }.
 *
 * Everything here is fp64 except grid_minmax, which deliberately works in fp32:
 * its floating-point results decide an integer (the zero point), and both sides
 * of a parity comparison must take that decision in the same precision.
 *
 * Built with: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC (no fast-math:
 * every sum is taken in the written order).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Gram matrix, Lemma 1 (Sigma = X X^T): Sigma_ab = sum_t X_at X_bt in fp64.   */
/* layout 0: X is p x n (channel-major); layout 1: X is n x p (token-major).   */
/* ------------------------------------------------------------------------- */
static inline double x_at(const float* X, int64_t p, int64_t n, int layout, int64_t a, int64_t t)
{
    return layout == 0 ? (double)X[a * n + t] : (double)X[t * p + a];
}

void qeo_gram(const float* X, int64_t p, int64_t n, int layout, double* Sigma)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t a = 0; a < p; ++a) {
        for (int64_t b = a; b < p; ++b) {
            double acc = 0.0;
            for (int64_t t = 0; t < n; ++t)
                acc += x_at(X, p, n, layout, a, t) * x_at(X, p, n, layout, b, t);
            Sigma[a * p + b] = acc;
            Sigma[b * p + a] = acc;
        }
    }
}

/* Selected entries (a[m], b[m]) of X X^T, one dot product each. */
void qeo_gram_entries(const float* X, int64_t p, int64_t n, int layout,
                      const int64_t* ia, const int64_t* ib, int64_t m, double* out)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t e = 0; e < m; ++e) {
        double acc = 0.0;
        for (int64_t t = 0; t < n; ++t)
            acc += x_at(X, p, n, layout, ia[e], t) * x_at(X, p, n, layout, ib[e], t);
        out[e] = acc;
    }
}

/* ------------------------------------------------------------------------- */
/* Per-row uniform grid (Sec. 2.1: levels uniformly spaced, per output channel). */
/* The paper does not print the formula; the reading used is the asymmetric     */
/* min/max grid: lo = min(0, min_j W_ij), hi = max(0, max_j W_ij) over the      */
/* entries not excluded, scale = (hi - lo) / (2^b - 1), zero = rint(-lo/scale); */
/* an all-zero row uses lo = -1, hi = +1.  Entries with H_ij != 0 are left out  */
/* (outlier-aware grid, Sec. 4.3: the top-s weights are removed from the pool). */
/* Computed in fp32 on purpose (see the file header).                           */
/* ------------------------------------------------------------------------- */
void qeo_grid_minmax(const float* W, int64_t q, int64_t p, int bits, const float* H,
                     float* scale, float* zero)
{
    const float maxq = (float)((1 << bits) - 1);
    for (int64_t i = 0; i < q; ++i) {
        float lo = 0.0f, hi = 0.0f;
        for (int64_t j = 0; j < p; ++j) {
            if (H && H[i * p + j] != 0.0f) continue;
            float w = W[i * p + j];
            if (w < lo) lo = w;
            if (w > hi) hi = w;
        }
        if (lo == 0.0f && hi == 0.0f) { lo = -1.0f; hi = 1.0f; }
        float s = (hi - lo) / maxq;
        float negq = -lo / s;
        scale[i] = s;
        zero[i] = rintf(negq);
    }
}

/* ------------------------------------------------------------------------- */
/* The quantizer q_i (Sec. 2.1, eq. quant) with the modified-CD tie rule          */
/* (Sec. 3.3): the coordinate moves only if the move strictly decreases f.      */
/* t is the unconstrained minimiser expressed in grid units, t = beta/s + z.    */
/* The 1-D objective is proportional to (s (k - z) - beta)^2 = s^2 (k - t)^2,    */
/* so the nearest grid code is the exact minimiser over Q_i; ties between two   */
/* codes at equal distance go to the even code (round half to even), except    */
/* that a valid current code at equal distance is kept.                        */
/* ------------------------------------------------------------------------- */
static int grid_decide(double t, int maxq, int have_code, int code)
{
    double k = nearbyint(t);           /* default rounding mode: half to even */
    if (k < 0.0) k = 0.0;
    if (k > (double)maxq) k = (double)maxq;
    int kk = (int)k;
    if (have_code && kk != code && fabs(t - (double)code) <= fabs(t - (double)kk))
        kk = code;
    return kk;
}

/* Distance of t from the nearest decision boundary between two grid codes
 * (boundaries sit at m + 1/2, m = 0 .. maxq-1).  Used by the parity protocol to
 * show that a code on which two implementations disagree was a near tie. */
static double boundary_margin(double t, int maxq)
{
    if (maxq < 1) return INFINITY;
    double u = t - 0.5;
    double m = nearbyint(u);
    if (m < 0.0) m = 0.0;
    if (m > (double)(maxq - 1)) m = (double)(maxq - 1);
    return fabs(u - m);
}

/* ------------------------------------------------------------------------- */
/* One cyclic CD sweep in the direct form of Lemma 1:                           */
/*   beta = -[ sum_{k != j} Sigma_jk What_ik - T_ij ] / Sigma_jj,               */
/*   What_ij <- q_i(beta),                                                      */
/* for j = 1..p in order, all rows i (rows are independent, Sec. 3.2).          */
/* T = W Sigma for the basic problem, T = (W - H) Sigma for the outlier-aware    */
/* CD step (Sec. 4.3 / Algorithm "Outlier-Aware QuantEase").                     */
/* valid[i*p+j] != 0 means What_ij currently sits on grid code codes[i*p+j].    */
/* relax != 0 writes beta unquantized (the paper's occasional unquantized pass, */
/* Sec. 3.2 "Initialization") and marks the codes invalid.                      */
/* margin (nullable) receives boundary_margin(t) of every decision.             */
/* j0 > 0 starts the pass at column j0 (the rest of a sweep whose first j0      */
/* coordinates are already done; the parity protocol uses it to follow another  */
/* implementation's choice at a tie and carry on from there).                   */
/* Returns 0, or 1 if some Sigma_jj <= 0 (Lemma 1 footnote).                    */
/* ------------------------------------------------------------------------- */
int qeo_cd_sweep_lemma1(const double* T, const double* S, int64_t q, int64_t p, int bits,
                        const double* scale, const double* zero, double* Wh, int32_t* codes,
                        uint8_t* valid, double* margin, int relax, int64_t j0)
{
    for (int64_t j = 0; j < p; ++j)
        if (!(S[j * p + j] > 0.0)) return 1;
    const int maxq = (1 << bits) - 1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < q; ++i) {
        double* w = Wh + i * p;
        for (int64_t j = j0; j < p; ++j) {
            const double* Sj = S + j * p;
            double c = 0.0;
            for (int64_t l = 0; l < p; ++l)
                if (l != j) c += Sj[l] * w[l];
            double beta = -(c - T[i * p + j]) / Sj[j];
            if (relax) {
                w[j] = beta;
                valid[i * p + j] = 0;
                if (margin) margin[i * p + j] = INFINITY;
                continue;
            }
            double t = beta / scale[i] + zero[i];
            int k = grid_decide(t, maxq, valid[i * p + j], codes[i * p + j]);
            if (margin) margin[i * p + j] = boundary_margin(t, maxq);
            codes[i * p + j] = k;
            valid[i * p + j] = 1;
            w[j] = scale[i] * ((double)k - zero[i]);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* One sweep of Algorithm "QuantEase" (rank-1 bookkeeping of What Sigma).      */
/* M = What Sigma is carried across columns; for each column j:                */
/*   u = [M_:,j - Sigma_jj What_:,j - T_:,j] / Sigma_jj                          */
/*   M -= What_:,j Sigma_j,:          (part A of the rank-1 identity)            */
/*   What_ij = q_i(-u_i)                                                        */
/*   M += What_:,j Sigma_j,:          (part B)                                   */
/* ------------------------------------------------------------------------- */
int qeo_cd_sweep_alg1(const double* T, const double* S, int64_t q, int64_t p, int bits,
                      const double* scale, const double* zero, double* Wh, int32_t* codes,
                      uint8_t* valid, double* M)
{
    for (int64_t j = 0; j < p; ++j)
        if (!(S[j * p + j] > 0.0)) return 1;
    const int maxq = (1 << bits) - 1;
    for (int64_t j = 0; j < p; ++j) {
        const double* Sj = S + j * p;
        const double sjj = Sj[j];
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < q; ++i) {
            double* m = M + i * p;
            double u = (m[j] - sjj * Wh[i * p + j] - T[i * p + j]) / sjj;
            double old = Wh[i * p + j];
            for (int64_t l = 0; l < p; ++l) m[l] -= old * Sj[l];
            double t = -u / scale[i] + zero[i];
            int k = grid_decide(t, maxq, valid[i * p + j], codes[i * p + j]);
            codes[i * p + j] = k;
            valid[i * p + j] = 1;
            double nw = scale[i] * ((double)k - zero[i]);
            Wh[i * p + j] = nw;
            for (int64_t l = 0; l < p; ++l) m[l] += nw * Sj[l];
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* One sweep of Algorithm "Accelerated QuantEase with partial update".          */
/* N is Sigma^norm (column j divided by Sigma_jj) with its diagonal already      */
/* set to zero; P = W Sigma^norm was formed before the diagonal was zeroed.      */
/* Per sweep: dW = What (a copy); Phat = What N; then for each column j:         */
/*   beta = P_:,j - Phat_:,j + dW_:,1:j N_1:j,j ;  What_:,j = q(beta);           */
/*   dW_:,j -= What_:,j.                                                         */
/* dW and Phat are caller-provided q x p scratch.                               */
/* ------------------------------------------------------------------------- */
void qeo_cd_sweep_alg2(const double* P, const double* N, int64_t q, int64_t p, int bits,
                       const double* scale, const double* zero, double* Wh, int32_t* codes,
                       uint8_t* valid, double* dW, double* Phat)
{
    const int maxq = (1 << bits) - 1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < q; ++i) {
        for (int64_t l = 0; l < p; ++l) dW[i * p + l] = Wh[i * p + l];
        for (int64_t j = 0; j < p; ++j) {
            double acc = 0.0;
            for (int64_t l = 0; l < p; ++l) acc += Wh[i * p + l] * N[l * p + j];
            Phat[i * p + j] = acc;
        }
        for (int64_t j = 0; j < p; ++j) {
            double part = 0.0;
            for (int64_t l = 0; l <= j; ++l) part += dW[i * p + l] * N[l * p + j];
            double beta = P[i * p + j] - Phat[i * p + j] + part;
            double t = beta / scale[i] + zero[i];
            int k = grid_decide(t, maxq, valid[i * p + j], codes[i * p + j]);
            codes[i * p + j] = k;
            valid[i * p + j] = 1;
            Wh[i * p + j] = scale[i] * ((double)k - zero[i]);
            dW[i * p + j] -= Wh[i * p + j];
        }
    }
}

/* ------------------------------------------------------------------------- */
/* P_s (Sec. 4.3, eq. iht-update): keep the s entries of V largest in absolute  */
/* value, zero the rest.  Ties in |V| go to the lower linear index i*p+j;       */
/* entries equal to zero are never part of the support.                         */
/* Writes the support as ascending linear indices; returns its size.            */
/* ------------------------------------------------------------------------- */
typedef struct { double key; int64_t idx; } qeo_kv;

static int kv_cmp(const void* a, const void* b)
{
    const qeo_kv* x = (const qeo_kv*)a;
    const qeo_kv* y = (const qeo_kv*)b;
    if (x->key > y->key) return -1;
    if (x->key < y->key) return 1;
    return (x->idx < y->idx) ? -1 : (x->idx > y->idx);
}

static int idx_cmp(const void* a, const void* b)
{
    int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
    return (x < y) ? -1 : (x > y);
}

int64_t qeo_topk_abs(const double* V, int64_t count, int64_t s, int64_t* support)
{
    qeo_kv* kv = (qeo_kv*)malloc(sizeof(qeo_kv) * (size_t)(count > 0 ? count : 1));
    if (!kv) return -1;
    for (int64_t e = 0; e < count; ++e) { kv[e].key = fabs(V[e]); kv[e].idx = e; }
    qsort(kv, (size_t)count, sizeof(qeo_kv), kv_cmp);
    int64_t nnz = 0;
    for (int64_t r = 0; r < s && r < count; ++r) {
        if (kv[r].key == 0.0) break;
        support[nnz++] = kv[r].idx;
    }
    free(kv);
    qsort(support, (size_t)nnz, sizeof(int64_t), idx_cmp);
    return nnz;
}

/* Number of OpenMP threads the loops above run with (for reporting). */
#include <omp.h>
int qeo_num_threads(void) { return omp_get_max_threads(); }
