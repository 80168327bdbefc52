/*
 * Dense DKM oracle, fp64, plain C.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the test-suite, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code with the HIP library.
 *
 * What it computes (DKM over the full N x k attention map, the form that the
 * paper's Sec. 2 says costs O(|W||C|) memory, and that Sec. 2.2's
 * uniquification reproduces exactly because equal 16-bit patterns give equal
 * attention rows):
 *
 *   v_i          = the real value of the i-th weight: an fp16 (IEEE 754
 *                  binary16) pattern for the keyed entry points; bf16 patterns
 *                  are decoded by dkm_decode_bf16 and passed as values
 *   for t = 1..T:
 *     D_ij       = -|v_i - C^(t-1)_j| / tau
 *     A^(t)_ij   = exp(D_ij) / sum_m exp(D_im)          (softmax over centroids)
 *     S^(t)_j    = sum_i A^(t)_ij,  P^(t)_j = sum_i A^(t)_ij v_i
 *     C^(t)_j    = P^(t)_j / S^(t)_j                     (S_j = 0: keep C^(t-1)_j)
 *     stop early when eps > 0 and max_j |C^(t)_j - C^(t-1)_j| <= eps
 *   W~_i         = sum_j A^(T)_ij C^(T)_j
 *
 * and the reverse-mode derivative of L = sum_i g_i W~_i with respect to every
 * v_i and to C^(0), through every executed iteration (the paper's Sec. 2.2
 * requires the backward to agree with ordinary autograd of the dense map).
 * d|x|/dx at x = 0 is taken as 0.
 *
 * Sums over weights use fixed blocks of DKM_BLK weights, each summed in index
 * order, then the block partials in block order, so results do not depend on
 * the OpenMP thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define DKM_BLK 65536
#define DKM_KMAX 256

/* IEEE 754 binary16 -> double, by its definition (exact for every pattern). */
double dkm_fp16_value(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int m = h & 0x3FF;
    double mag;
    if (e == 0)
        mag = ldexp((double)m, -24);               /* subnormal: m * 2^-24 */
    else if (e == 31)
        mag = m ? NAN : INFINITY;
    else
        mag = ldexp((double)(1024 + m), e - 25);   /* (1 + m/1024) * 2^(e-15) */
    return sign ? -mag : mag;
}

void dkm_decode_fp16(const uint16_t* keys, int64_t n, double* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = dkm_fp16_value(keys[i]);
}

/* bfloat16 -> double, by its definition: 1 sign, 8 exponent (bias 127) and 7
 * mantissa bits (the upper half of an IEEE 754 binary32); exact for every
 * pattern. */
double dkm_bf16_value(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 7) & 0xFF;
    int m = h & 0x7F;
    double mag;
    if (e == 0)
        mag = ldexp((double)m, -133);              /* subnormal: m * 2^-126 * 2^-7 */
    else if (e == 0xFF)
        mag = m ? NAN : INFINITY;
    else
        mag = ldexp((double)(m + 128), e - 134);   /* (1 + m/128) * 2^(e-127) */
    return sign ? -mag : mag;
}

void dkm_decode_bf16(const uint16_t* keys, int64_t n, double* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = dkm_bf16_value(keys[i]);
}

int dkm_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for later calls (timing only: the fixed-block sums make every
 * result independent of the thread count). */
void dkm_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

static double sgn(double x) { return (x > 0.0) - (x < 0.0); }

/* One row of the attention map: softmax_j(-|v - c_j| / tau). */
static void attn_row(double v, const double* c, int k, double tau, double* a)
{
    double dmax = -INFINITY;
    for (int j = 0; j < k; ++j) {
        a[j] = -fabs(v - c[j]) / tau;
        if (a[j] > dmax) dmax = a[j];
    }
    double sum = 0.0;
    for (int j = 0; j < k; ++j) {
        a[j] = exp(a[j] - dmax);
        sum += a[j];
    }
    for (int j = 0; j < k; ++j) a[j] /= sum;
}

static int64_t nblocks(int64_t n) { return (n + DKM_BLK - 1) / DKM_BLK; }

/*
 * Forward.  c_hist and s_hist hold (max_iter + 1) rows of k values: row t is
 * C^(t) and S^(t) (row 0 of s_hist is unused and set to 0).  w_tilde gets N
 * values; attn (nullable) gets A^(T) as an N x k row-major array.  Returns T,
 * the number of iterations executed.
 */
int dkm_dense_forward_f64(const double* v, int64_t n, int k, double tau, int max_iter,
                          double eps, const double* c0, double* c_hist, double* s_hist,
                          double* w_tilde, double* attn)
{
    if (k < 1 || k > DKM_KMAX || max_iter < 1 || n < 1 || !(tau > 0.0)) return -1;
    const int64_t nb = nblocks(n);
    double* part = (double*)calloc((size_t)nb * 2 * k, sizeof(double));
    if (!part) return -2;
    memcpy(c_hist, c0, sizeof(double) * k);
    memset(s_hist, 0, sizeof(double) * k);
    int T = max_iter;
    for (int t = 1; t <= max_iter; ++t) {
        const double* cp = c_hist + (size_t)(t - 1) * k;
        double* cn = c_hist + (size_t)t * k;
        double* st = s_hist + (size_t)t * k;
#pragma omp parallel for schedule(static)
        for (int64_t b = 0; b < nb; ++b) {
            double a[DKM_KMAX];
            double* Sb = part + (size_t)b * 2 * k;
            double* Pb = Sb + k;
            for (int j = 0; j < 2 * k; ++j) Sb[j] = 0.0;
            int64_t hi = (b + 1) * DKM_BLK < n ? (b + 1) * DKM_BLK : n;
            for (int64_t i = b * DKM_BLK; i < hi; ++i) {
                attn_row(v[i], cp, k, tau, a);
                for (int j = 0; j < k; ++j) {
                    Sb[j] += a[j];
                    Pb[j] += a[j] * v[i];
                }
            }
        }
        double dmax = 0.0;
        for (int j = 0; j < k; ++j) {
            double S = 0.0, P = 0.0;
            for (int64_t b = 0; b < nb; ++b) {
                S += part[(size_t)b * 2 * k + j];
                P += part[(size_t)b * 2 * k + k + j];
            }
            st[j] = S;
            cn[j] = S > 0.0 ? P / S : cp[j];
            double d = fabs(cn[j] - cp[j]);
            if (d > dmax) dmax = d;
        }
        if (eps > 0.0 && dmax <= eps) { T = t; break; }
    }
    free(part);
    const double* cT = c_hist + (size_t)T * k;
    const double* cTm1 = c_hist + (size_t)(T - 1) * k;
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < nb; ++b) {
        double a[DKM_KMAX];
        int64_t hi = (b + 1) * DKM_BLK < n ? (b + 1) * DKM_BLK : n;
        for (int64_t i = b * DKM_BLK; i < hi; ++i) {
            attn_row(v[i], cTm1, k, tau, a);
            double w = 0.0;
            for (int j = 0; j < k; ++j) w += a[j] * cT[j];
            w_tilde[i] = w;
            if (attn)
                for (int j = 0; j < k; ++j) attn[(size_t)i * k + j] = a[j];
        }
    }
    return T;
}

/*
 * Backward of L = sum_i g_i W~_i.  Needs the history written by the forward
 * (c_hist rows 0..T, s_hist rows 1..T).  Writes dL/dv (N values) and dL/dC^(0).
 *
 * Adjoint bookkeeping, in the forward's own notation: gam_j holds dL/dC^(t)_j.
 * At t = T the map A^(T) is also used directly by W~, which adds
 * g_i C^(T)_j to the adjoint of A^(T)_ij.  Through C^(t) = P/S the adjoint
 * of A^(t)_ij gains gam_j (v_i - C^(t)_j) / S_j and v_i gains A_ij gam_j / S_j;
 * through the softmax and D_ij = -|v_i - C^(t-1)_j| / tau the adjoint reaches
 * v_i with factor -sgn/tau and C^(t-1)_j with factor +sgn/tau.
 */
int dkm_dense_backward_f64(const double* v, int64_t n, int k, double tau, int T,
                           const double* c_hist, const double* s_hist, const double* g,
                           double* grad_w, double* grad_c0)
{
    if (k < 1 || k > DKM_KMAX || T < 1 || n < 1 || !(tau > 0.0)) return -1;
    const int64_t nb = nblocks(n);
    double* part = (double*)calloc((size_t)nb * 2 * k, sizeof(double));
    if (!part) return -2;
    double gam[DKM_KMAX], E[DKM_KMAX];

    /* Direct use of A^(T) and C^(T) by W~. */
    {
        const double* cT = c_hist + (size_t)T * k;
        const double* cTm1 = c_hist + (size_t)(T - 1) * k;
#pragma omp parallel for schedule(static)
        for (int64_t b = 0; b < nb; ++b) {
            double a[DKM_KMAX];
            double* Gb = part + (size_t)b * 2 * k;
            double* Eb = Gb + k;
            for (int j = 0; j < 2 * k; ++j) Gb[j] = 0.0;
            int64_t hi = (b + 1) * DKM_BLK < n ? (b + 1) * DKM_BLK : n;
            for (int64_t i = b * DKM_BLK; i < hi; ++i) {
                attn_row(v[i], cTm1, k, tau, a);
                double w = 0.0;
                for (int j = 0; j < k; ++j) w += a[j] * cT[j];
                double h = 0.0;
                for (int j = 0; j < k; ++j) {
                    double s = sgn(v[i] - cTm1[j]);
                    double q = a[j] * (cT[j] - w) * s;   /* softmax-Jacobian term */
                    h += q;
                    Gb[j] += g[i] * a[j];
                    Eb[j] += g[i] * q;
                }
                grad_w[i] = -g[i] * h / tau;
            }
        }
        for (int j = 0; j < k; ++j) {
            double G = 0.0, Es = 0.0;
            for (int64_t b = 0; b < nb; ++b) {
                G += part[(size_t)b * 2 * k + j];
                Es += part[(size_t)b * 2 * k + k + j];
            }
            gam[j] = G;
            E[j] = Es / tau;
        }
    }

    /* Iterations t = T .. 1, each mapping dL/dC^(t) to dL/dC^(t-1). */
    for (int t = T; t >= 1; --t) {
        const double* ct = c_hist + (size_t)t * k;
        const double* cp = c_hist + (size_t)(t - 1) * k;
        const double* S = s_hist + (size_t)t * k;
#pragma omp parallel for schedule(static)
        for (int64_t b = 0; b < nb; ++b) {
            double a[DKM_KMAX], al[DKM_KMAX];
            double* Gb = part + (size_t)b * k;
            for (int j = 0; j < k; ++j) Gb[j] = 0.0;
            int64_t hi = (b + 1) * DKM_BLK < n ? (b + 1) * DKM_BLK : n;
            for (int64_t i = b * DKM_BLK; i < hi; ++i) {
                attn_row(v[i], cp, k, tau, a);
                double abar = 0.0, direct = 0.0;
                for (int j = 0; j < k; ++j) {
                    al[j] = S[j] > 0.0 ? gam[j] * (v[i] - ct[j]) / S[j] : 0.0;
                    abar += a[j] * al[j];
                    if (S[j] > 0.0) direct += a[j] * gam[j] / S[j];
                }
                double r = 0.0;
                for (int j = 0; j < k; ++j) {
                    double s = sgn(v[i] - cp[j]);
                    double d = a[j] * (al[j] - abar) * s;
                    r += d;
                    Gb[j] += d;
                }
                grad_w[i] += direct - r / tau;
            }
        }
        double nxt[DKM_KMAX];
        for (int j = 0; j < k; ++j) {
            double s = 0.0;
            for (int64_t b = 0; b < nb; ++b) s += part[(size_t)b * k + j];
            nxt[j] = s / tau;
            if (t == T) nxt[j] += E[j];
            if (!(S[j] > 0.0)) nxt[j] += gam[j];   /* C^(t)_j = C^(t-1)_j */
        }
        memcpy(gam, nxt, sizeof(double) * k);
    }
    memcpy(grad_c0, gam, sizeof(double) * k);
    free(part);
    return 0;
}

/* Keyed wrappers: the inputs are raw fp16 bit patterns. */
int dkm_dense_forward(const uint16_t* keys, int64_t n, int k, double tau, int max_iter,
                      double eps, const double* c0, double* c_hist, double* s_hist,
                      double* w_tilde, double* attn)
{
    double* v = (double*)malloc(sizeof(double) * (size_t)n);
    if (!v) return -2;
    dkm_decode_fp16(keys, n, v);
    int r = dkm_dense_forward_f64(v, n, k, tau, max_iter, eps, c0, c_hist, s_hist, w_tilde, attn);
    free(v);
    return r;
}

int dkm_dense_backward(const uint16_t* keys, int64_t n, int k, double tau, int T,
                       const double* c_hist, const double* s_hist, const double* g,
                       double* grad_w, double* grad_c0)
{
    double* v = (double*)malloc(sizeof(double) * (size_t)n);
    if (!v) return -2;
    dkm_decode_fp16(keys, n, v);
    int r = dkm_dense_backward_f64(v, n, k, tau, T, c_hist, s_hist, g, grad_w, grad_c0);
    free(v);
    return r;
}
