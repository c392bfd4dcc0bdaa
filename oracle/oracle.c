/*
 * oracle.c -- plain, slow, scalar CPU oracle for the few-bit activation path
 * of "Few-Bit Backward: Quantized Gradients of Activation Functions for
 * Memory Footprint Reduction" (Novikov et al., ICML 2022).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file.  Only the test suite, the smoke check of the entry module
 * and the CPU-baseline leg of the benchmark may use it.  It shares no source,
 * header, table or constant with the HIP library: the only things both sides
 * agree on are the data formats (IEEE bit patterns, the packed-code stream)
 * and the seeded synthetic inputs, which are generated elsewhere.
 *
 * Arithmetic is IEEE double throughout; results are rounded exactly once to
 * the requested storage type with this file's own round-to-nearest-even
 * conversions.  There is no blocking, fusion or reordering beyond what each
 * definition states, so every function can be checked against the paper by
 * eye.
 *
 * What each function follows:
 *   activations f and f'   -- Sec. 2 (pointwise activations, GELU, ReLU) and
 *                             Table 1's list of activations; Swish is defined
 *                             in Sec. 4 (ResNet paragraph) as x*sigmoid(x).
 *   weight w               -- Sec. 3, Eq. (3): uniform on [A,B] or a density.
 *   prefix integrals       -- Sec. 3, Eqs. (8)-(9) (F^2, W, FW recursions).
 *   interval cost T, y     -- Sec. 3, Eqs. (4), (7), (8).
 *   dynamic programme      -- Sec. 3, Eqs. (6)-(7).
 *   symmetric fit          -- Fig. 3 caption: for an even f' only [0, inf)
 *                             is quantised, the bins apply to |x|.
 *   classify / forward     -- Listing 1 (forward: bin index by sorted search,
 *                             keep indices, return f(X)); Eq. (2).
 *   packing                -- Sec. 2: log2(k) bits per element.  The paper
 *                             does not fix a layout; this oracle defines it
 *                             as a dense little-endian LSB-first bit stream.
 *   backward               -- Eq. (1) with f' replaced by the stored value
 *                             y[idx] (Listing 1, backward).
 *   refinement             -- Sec. 3: y(s) by Eq. (4), the analytic gradient
 *                             of L(s, y(s)) in s, gradient descent from the
 *                             DP result (reading R14).
 *
 * Readings where the paper is silent or garbled (each one is listed in the
 * design notes of the repository, whose numbering these keep; R9-R13 there
 * concern the GELU variant, the symmetric fit, the code layout and the
 * workloads, and are stated at the functions they shape):
 *   R1  Eq. (7) prints the same k on both sides of the recurrence; it is read
 *       as DP(i,k+1) = min_{j<i} DP(j,k) + T(j,i), matching Eq. (6).
 *   R2  Eq. (6) prints y(t',t) without the normalising integral of w; it is
 *       read as the optimal value of Eq. (4).
 *   R3  The grid is uniform, t_i = A + i (B-A)/n, and each cell integral is
 *       an 8-point Gauss-Legendre rule (the paper only says "numerically").
 *   R4  Interval costs are clamped: T := max(T, 0); an interval with zero
 *       weight gets T := 0 and y := f'(midpoint).  Prefix sums of a normal
 *       density saturate in double far in the tails, which otherwise yields
 *       0/0 and negative costs.
 *   R5  Every interval holds at least one grid cell (j ranges over
 *       k-1 <= j < i); ties keep the smallest j.
 *   R6  Only interior boundaries are stored; the outer bins are unbounded,
 *       so inputs outside [A,B] take the first or last value.
 *   R7  Bin membership is half-open, [s_m, s_{m+1}): idx(x) counts the
 *       boundaries s_m <= x.  NaN compares false (idx 0); -0 == +0.
 *   R8  Half-precision gradients are rounded twice by definition: the fp32
 *       product widen(g)*v[idx], then round-to-nearest-even to the dtype.
 *   R14 The paper leaves the gradient method open; the refinement here is
 *       steepest descent with Armijo backtracking, integrals at off-grid
 *       boundaries taken as the grid prefix plus the partial cell by the
 *       same 8-point rule.
 *
 * Parity status: activations, weights, fit, classify, pack/unpack and
 * backward are pinned by the CPU tests (closed forms, central differences,
 * the paper's Table 1, Lloyd-Max tables, brute force, hand-made bit vectors,
 * exhaustive or sampled conversions against other libraries).  The weight
 * functions are pinned by the normal cdf and the moments of truncated
 * normals, SELU's f by the self-normalising property its constants are
 * defined by.  The fp32 value of y is compared to the GPU within a
 * tolerance only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

/* ------------------------------------------------------------------ */
/* Activation identifiers (oracle-local numbering, same values as the  */
/* public ABI enumerations so tests can pass one integer around).      */
/* ------------------------------------------------------------------ */
enum {
    OR_GELU = 0, OR_SILU = 1, OR_SIGMOID = 2, OR_TANH = 3,
    OR_RELU = 4, OR_SELU = 5, OR_SOFTPLUS = 6,
    OR_HALFSQ = 7   /* f(x) = x^2/2, f'(x) = x: the Lloyd-Max special case */
};
enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };
enum { OR_W_UNIFORM = 0, OR_W_NORMAL = 1, OR_W_MIXTURE = 2 };

static const double OR_PI = 3.14159265358979323846;

/* SELU constants (Klambauer et al., 2017). */
static const double SELU_LAMBDA = 1.0507009873554804934193349852946;
static const double SELU_ALPHA = 1.6732632423543772848170429916717;

/* logistic sigmoid, evaluated on the side that cannot overflow */
static double or_sigmoid(double x)
{
    if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
    double e = exp(x);
    return e / (1.0 + e);
}

/* standard normal cdf and pdf: Phi(x) = erfc(-x/sqrt 2)/2 */
static double or_Phi(double x) { return 0.5 * erfc(-x / sqrt(2.0)); }
static double or_phi(double x) { return exp(-0.5 * x * x) / sqrt(2.0 * OR_PI); }

/* f(x): the activation itself (Sec. 2; Table 1 rows). */
double oracle_f(int act, double x)
{
    if (isnan(x)) return x;
    switch (act) {
    case OR_GELU:
        if (isinf(x)) return x > 0 ? x : -0.0;      /* limits of x*Phi(x) */
        return x * or_Phi(x);
    case OR_SILU:
        if (isinf(x)) return x > 0 ? x : -0.0;      /* limits of x*sigma(x) */
        return x * or_sigmoid(x);
    case OR_SIGMOID:
        return or_sigmoid(x);
    case OR_TANH:
        return tanh(x);
    case OR_RELU:
        return x > 0 ? x : 0.0;
    case OR_SELU:
        return x > 0 ? SELU_LAMBDA * x : SELU_LAMBDA * SELU_ALPHA * expm1(x);
    case OR_SOFTPLUS:
        return x > 0 ? x + log1p(exp(-x)) : log1p(exp(x));
    case OR_HALFSQ:
        return 0.5 * x * x;
    }
    return NAN;
}

/* f'(x): closed-form derivatives. */
double oracle_df(int act, double x)
{
    switch (act) {
    case OR_GELU:                                   /* Phi(x) + x phi(x) */
        return or_Phi(x) + x * or_phi(x);
    case OR_SILU: {                                 /* s (1 + x (1 - s)) */
        double s = or_sigmoid(x);
        return s * (1.0 + x * (1.0 - s));
    }
    case OR_SIGMOID: {                              /* s (1 - s) */
        double s = or_sigmoid(x);
        return s * (1.0 - s);
    }
    case OR_TANH: {                                 /* 1 - tanh^2 */
        double t = tanh(x);
        return 1.0 - t * t;
    }
    case OR_RELU:
        return x > 0 ? 1.0 : 0.0;
    case OR_SELU:
        return x > 0 ? SELU_LAMBDA : SELU_LAMBDA * SELU_ALPHA * exp(x);
    case OR_SOFTPLUS:
        return or_sigmoid(x);
    case OR_HALFSQ:
        return x;
    }
    return NAN;
}

/* ------------------------------------------------------------------ */
/* Weight functions (Sec. 3, Eq. (3)); w = 0 outside [A, B].           */
/* ------------------------------------------------------------------ */
typedef struct {
    int32_t kind;      /* OR_W_UNIFORM, OR_W_NORMAL, OR_W_MIXTURE */
    int32_t pad;
    double A, B;       /* support */
    double mu, sigma;  /* normal: N(mu, sigma^2) */
    double p, sigma2;  /* mixture: (1-p) N(mu,sigma^2) + p N(mu,sigma2^2) */
} oracle_weight;

static double or_normal_pdf(double x, double mu, double sigma)
{
    double z = (x - mu) / sigma;
    return exp(-0.5 * z * z) / (sigma * sqrt(2.0 * OR_PI));
}

static double or_w(const oracle_weight* w, double x)
{
    if (x < w->A || x > w->B) return 0.0;
    switch (w->kind) {
    case OR_W_UNIFORM: return 1.0;
    case OR_W_NORMAL: return or_normal_pdf(x, w->mu, w->sigma);
    case OR_W_MIXTURE:
        return (1.0 - w->p) * or_normal_pdf(x, w->mu, w->sigma)
             + w->p * or_normal_pdf(x, w->mu, w->sigma2);
    }
    return 0.0;
}

/* 8-point Gauss-Legendre rule on [-1, 1]: nodes and weights as tabulated in
 * Abramowitz & Stegun, Table 25.4. */
static const double GL8_X[4] = {0.183434642495649804939476142360184,
                                0.525532409916328985817739049189246,
                                0.796666477413626739591553936475830,
                                0.960289856497536231683560868569473};
static const double GL8_W[4] = {0.362683783378361982965150449277196,
                                0.313706645877887287337962201986601,
                                0.222381034453374470544355994426241,
                                0.101228536290376259152531354309962};

/* Cell integrals over [a, b] of w, f' w and f'^2 w (reading R3). */
static void or_cell(int act, const oracle_weight* w, double a, double b,
                    double* iw, double* ifw, double* if2w)
{
    double c = 0.5 * (a + b), h = 0.5 * (b - a);
    double sw = 0, sfw = 0, sf2w = 0;
    for (int k = 0; k < 4; ++k) {
        for (int sgn = -1; sgn <= 1; sgn += 2) {
            double x = c + sgn * h * GL8_X[k];
            double wx = or_w(w, x), d = oracle_df(act, x);
            sw += GL8_W[k] * wx;
            sfw += GL8_W[k] * d * wx;
            sf2w += GL8_W[k] * d * d * wx;
        }
    }
    *iw = h * sw;
    *ifw = h * sfw;
    *if2w = h * sf2w;
}

/* Prefix integrals W(i), FW(i), F2(i), i = 0..n, on the uniform grid over
 * [A, B] (Sec. 3, Eqs. (8)-(9)).  Arrays have n+1 entries.  Returns 0. */
int oracle_prefix(int act, const oracle_weight* w, int64_t n,
                  double* W, double* FW, double* F2)
{
    if (n < 1) return -1;
    double A = w->A, B = w->B;
    W[0] = FW[0] = F2[0] = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double a = A + (double)i * (B - A) / (double)n;
        double b = A + (double)(i + 1) * (B - A) / (double)n;
        double iw, ifw, if2w;
        or_cell(act, w, a, b, &iw, &ifw, &if2w);
        W[i + 1] = W[i] + iw;
        FW[i + 1] = FW[i] + ifw;
        F2[i + 1] = F2[i] + if2w;
    }
    return 0;
}

/* Optimal value and cost of one interval [t_j, t_i] (Eqs. (4), (7), (8),
 * with reading R4). */
static void or_interval(const double* W, const double* FW, const double* F2,
                        int64_t j, int64_t i, int act, double tj, double ti,
                        double* y_out, double* T_out)
{
    double dW = W[i] - W[j];
    double dFW = FW[i] - FW[j];
    double dF2 = F2[i] - F2[j];
    if (!(dW > 0.0)) {
        *y_out = oracle_df(act, 0.5 * (tj + ti));
        *T_out = 0.0;
        return;
    }
    double y = dFW / dW;
    double T = dF2 - y * y * dW;
    *y_out = y;
    *T_out = T > 0.0 ? T : 0.0;
}

/* Exposed for the brute-force test: cost of interval (j, i) on the grid. */
double oracle_interval_cost(const double* W, const double* FW, const double* F2,
                            int64_t j, int64_t i, int act, double tj, double ti)
{
    double y, T;
    or_interval(W, FW, F2, j, i, act, tj, ti, &y, &T);
    return T;
}

/*
 * The optimal piecewise-constant fit of f' (Sec. 3): dynamic programme over
 * the grid, Eqs. (6)-(7) with readings R1, R4, R5.
 *
 *   act, bits      activation and bit width (K = 2^bits intervals)
 *   w              weight and support [A, B]; for symmetric = 1 the fit is
 *                  made on [max(A,0), B] and the reported loss doubled
 *   n              number of grid cells
 *   s_out[K-1]     interior boundaries rounded to fp32 (reading R6)
 *   v_out[K]       interval values rounded to fp32
 *   loss_out       DP(n, K) (doubled for the symmetric fit)
 *   cuts_out[K+1]  grid indices j_0 = 0 < j_1 < ... < j_K = n (may be NULL)
 *   dp_last[K]     DP(n, k) for k = 1..K (may be NULL)
 *   vd_out[K]      interval values in double (may be NULL)
 * Returns 0, or -1 for bad arguments / allocation failure, -2 when the fp32
 * boundaries are not strictly increasing.
 */
int oracle_fit(int act, int bits, const oracle_weight* w_in, int64_t n,
               int symmetric, float* s_out, float* v_out, double* loss_out,
               int64_t* cuts_out, double* dp_last, double* vd_out)
{
    if (bits < 1 || bits > 4 || n < 2) return -1;
    const int K = 1 << bits;
    if (n < K) return -1;
    oracle_weight w = *w_in;
    if (symmetric && w.A < 0.0) w.A = 0.0;
    const double A = w.A, B = w.B;

    double* W = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* FW = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* F2 = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* DP = (double*)malloc(sizeof(double) * (size_t)(n + 1) * (size_t)(K + 1));
    int64_t* BP = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n + 1) * (size_t)(K + 1));
    if (!W || !FW || !F2 || !DP || !BP) {
        free(W); free(FW); free(F2); free(DP); free(BP);
        return -1;
    }
    oracle_prefix(act, &w, n, W, FW, F2);

#define T_AT(i) (A + (double)(i) * (B - A) / (double)n)
#define DPX(k, i) DP[(size_t)(k) * (size_t)(n + 1) + (size_t)(i)]
#define BPX(k, i) BP[(size_t)(k) * (size_t)(n + 1) + (size_t)(i)]

    /* one interval: DP(i, 1) = T(0, i) */
    for (int64_t i = 1; i <= n; ++i) {
        double y, T;
        or_interval(W, FW, F2, 0, i, act, T_AT(0), T_AT(i), &y, &T);
        DPX(1, i) = T;
        BPX(1, i) = 0;
    }
    /* k intervals: DP(i, k) = min over k-1 <= j < i of DP(j, k-1) + T(j, i) */
    for (int k = 2; k <= K; ++k) {
        for (int64_t i = k; i <= n; ++i) {
            double best = INFINITY;
            int64_t arg = -1;
            for (int64_t j = k - 1; j < i; ++j) {
                double y, T;
                or_interval(W, FW, F2, j, i, act, T_AT(j), T_AT(i), &y, &T);
                double c = DPX(k - 1, j) + T;
                if (c < best) { best = c; arg = j; }
            }
            DPX(k, i) = best;
            BPX(k, i) = arg;
        }
    }

    /* backtrack the cut points j_K = n, j_{m-1} = BP(m, j_m), j_0 = 0 */
    int64_t cuts[17];
    cuts[K] = n;
    for (int m = K; m >= 1; --m) cuts[m - 1] = BPX(m, cuts[m]);
    /* cuts[0] is BP(1, .) = 0 */

    double scale = symmetric ? 2.0 : 1.0;
    if (loss_out) *loss_out = scale * DPX(K, n);
    if (dp_last)
        for (int k = 1; k <= K; ++k) dp_last[k - 1] = scale * DPX(k, n);
    if (cuts_out)
        for (int m = 0; m <= K; ++m) cuts_out[m] = cuts[m];

    int rc = 0;
    for (int m = 1; m <= K; ++m) {
        double y, T;
        or_interval(W, FW, F2, cuts[m - 1], cuts[m], act, T_AT(cuts[m - 1]),
                    T_AT(cuts[m]), &y, &T);
        v_out[m - 1] = (float)y;
        if (vd_out) vd_out[m - 1] = y;
    }
    for (int m = 1; m < K; ++m) s_out[m - 1] = (float)T_AT(cuts[m]);
    for (int m = 1; m + 1 < K; ++m)
        if (!(s_out[m - 1] < s_out[m])) rc = -2;
#undef T_AT
#undef DPX
#undef BPX
    free(W); free(FW); free(F2); free(DP); free(BP);
    return rc;
}

/* ------------------------------------------------------------------ */
/* Gradient refinement of the boundaries (Sec. 3: y(s) of Eq. (4), the   */
/* analytic gradient of L(s, y(s)) with respect to s, and the remark     */
/* that the DP result may be finetuned by any gradient method).          */
/* ------------------------------------------------------------------ */

/* Integrals of w, f' w and f'^2 w over [A, x], A <= x <= B: the grid prefix
 * up to the cell holding x plus the part of that cell below x, by the same
 * 8-point rule (reading R3). */
static void or_prefix_at(int act, const oracle_weight* w, int64_t n,
                         const double* W, const double* FW, const double* F2,
                         double x, double* pw, double* pfw, double* pf2w)
{
    double A = w->A, B = w->B;
    int64_t j = (int64_t)floor((x - A) / (B - A) * (double)n);
    if (j < 0) j = 0;
    if (j > n) j = n;
    double tj = A + (double)j * (B - A) / (double)n;
    if (tj > x && j > 0) {          /* rounding put x just below t_j */
        j -= 1;
        tj = A + (double)j * (B - A) / (double)n;
    }
    double iw = 0.0, ifw = 0.0, if2w = 0.0;
    if (j < n && x > tj) or_cell(act, w, tj, x, &iw, &ifw, &if2w);
    *pw = W[j] + iw;
    *pfw = FW[j] + ifw;
    *pf2w = F2[j] + if2w;
}

/* L(s, y(s)) of Eq. (3) for interior boundaries s[0..K-2] (s_0 = A and
 * s_K = B bound the outer intervals, reading R6), the values y(s) of
 * Eq. (4) and, if grad != NULL, the gradient of Sec. 3:
 *   dL/ds_i = (2 f'(s_i) - y_i - y_{i-1}) (y_i - y_{i-1}) w(s_i),
 * y_{i-1} the value left of s_i and y_i the value right of it.
 * Intervals without weight take f' at their midpoint and cost 0 (R4). */
static double or_loss_at(int act, const oracle_weight* w, int64_t n,
                         const double* W, const double* FW, const double* F2,
                         int K, const double* s, double* y, double* grad)
{
    double edge[17];
    edge[0] = w->A;
    for (int m = 1; m < K; ++m) edge[m] = s[m - 1];
    edge[K] = w->B;
    double pw[17], pfw[17], pf2w[17];
    for (int m = 0; m <= K; ++m)
        or_prefix_at(act, w, n, W, FW, F2, edge[m], &pw[m], &pfw[m], &pf2w[m]);
    double L = 0.0;
    for (int m = 0; m < K; ++m) {
        double dW = pw[m + 1] - pw[m];
        double dFW = pfw[m + 1] - pfw[m];
        double dF2 = pf2w[m + 1] - pf2w[m];
        if (!(dW > 0.0)) {
            y[m] = oracle_df(act, 0.5 * (edge[m] + edge[m + 1]));
            continue;
        }
        y[m] = dFW / dW;
        double T = dF2 - y[m] * y[m] * dW;
        L += T > 0.0 ? T : 0.0;
    }
    if (grad)
        for (int i = 1; i < K; ++i) {
            double d = oracle_df(act, s[i - 1]);
            grad[i - 1] = (2.0 * d - y[i] - y[i - 1]) * (y[i] - y[i - 1]) * or_w(w, s[i - 1]);
        }
    return L;
}

/* Exposed for the finite-difference test: L(s) (doubled for the symmetric
 * fit), y(s) and dL/ds at the given boundaries. */
int oracle_loss_at(int act, int bits, const oracle_weight* w_in, int64_t n,
                   int symmetric, const double* s, double* y_out,
                   double* grad_out, double* loss_out)
{
    if (bits < 1 || bits > 4 || n < 2) return -1;
    const int K = 1 << bits;
    oracle_weight w = *w_in;
    if (symmetric && w.A < 0.0) w.A = 0.0;
    double* W = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* FW = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* F2 = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    if (!W || !FW || !F2) { free(W); free(FW); free(F2); return -1; }
    oracle_prefix(act, &w, n, W, FW, F2);
    double scale = symmetric ? 2.0 : 1.0;
    double L = or_loss_at(act, &w, n, W, FW, F2, K, s, y_out, grad_out);
    if (grad_out)
        for (int i = 0; i < K - 1; ++i) grad_out[i] *= scale;
    *loss_out = scale * L;
    free(W); free(FW); free(F2);
    return 0;
}

/*
 * The DP fit of oracle_fit, then gradient descent on the boundaries with
 * the analytic gradient: from the DP cut points, step s <- s - t g, with t
 * halved until the step keeps the boundaries strictly increasing inside
 * (A, B) and decreases L, by at least 1e-4 t |g|^2 (Armijo), and doubled
 * after each accepted step; the first step moves no boundary by more than
 * one grid cell.  Stops after max_iter steps, or when no step decreases L.
 *
 *   s_out[K-1], v_out[K]  refined boundaries and values (fp32)
 *   sd_out[K-1]           refined boundaries in double (may be NULL)
 *   vd_out[K]             refined values in double (may be NULL)
 *   loss_out              L after refinement (doubled for symmetric)
 *   loss_dp_out           L of the DP result, same scale (may be NULL)
 *   iters_out             accepted steps (may be NULL)
 * Returns 0, -1 for bad arguments / allocation failure, -2 when the fp32
 * boundaries are not strictly increasing.
 */
int oracle_fit_refined(int act, int bits, const oracle_weight* w_in, int64_t n,
                       int symmetric, int max_iter, float* s_out, float* v_out,
                       double* sd_out, double* vd_out, double* loss_out,
                       double* loss_dp_out, int* iters_out)
{
    if (bits < 1 || bits > 4 || n < 2 || max_iter < 0) return -1;
    const int K = 1 << bits;
    int64_t cuts[17];
    float s_dp[15], v_dp[16];
    double loss_dp;
    int rc = oracle_fit(act, bits, w_in, n, symmetric, s_dp, v_dp, &loss_dp, cuts,
                        NULL, NULL);
    if (rc == -1) return -1;

    oracle_weight w = *w_in;
    if (symmetric && w.A < 0.0) w.A = 0.0;
    const double A = w.A, B = w.B, h = (B - A) / (double)n;
    double* W = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* FW = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    double* F2 = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    if (!W || !FW || !F2) { free(W); free(FW); free(F2); return -1; }
    oracle_prefix(act, &w, n, W, FW, F2);

    double s[15], trial[15], g[15], y[16];
    for (int m = 1; m < K; ++m) s[m - 1] = A + (double)cuts[m] * (B - A) / (double)n;
    double L = or_loss_at(act, &w, n, W, FW, F2, K, s, y, g);
    double gmax = 0.0;
    for (int i = 0; i < K - 1; ++i) gmax = fmax(gmax, fabs(g[i]));
    double t0 = gmax > 0.0 ? h / gmax : 0.0;
    int it = 0;
    while (it < max_iter && gmax > 0.0) {
        double g2 = 0.0;
        for (int i = 0; i < K - 1; ++i) g2 += g[i] * g[i];
        double t = t0;
        int accepted = 0;
        for (int tries = 0; tries < 80; ++tries) {
            int ok = 1;
            for (int i = 0; i < K - 1; ++i) {
                trial[i] = s[i] - t * g[i];
                if (!(trial[i] > A && trial[i] < B)) ok = 0;
                if (i > 0 && !(trial[i] > trial[i - 1])) ok = 0;
            }
            if (ok) {
                double y_try[16];
                double L_try = or_loss_at(act, &w, n, W, FW, F2, K, trial, y_try, NULL);
                if (L_try < L && L_try <= L - 1e-4 * t * g2) { accepted = 1; break; }
            }
            t *= 0.5;
        }
        if (!accepted) break;
        for (int i = 0; i < K - 1; ++i) s[i] = trial[i];
        L = or_loss_at(act, &w, n, W, FW, F2, K, s, y, g);
        gmax = 0.0;
        for (int i = 0; i < K - 1; ++i) gmax = fmax(gmax, fabs(g[i]));
        t0 = 2.0 * t;
        ++it;
    }

    double scale = symmetric ? 2.0 : 1.0;
    *loss_out = scale * L;
    if (loss_dp_out) *loss_dp_out = loss_dp;
    if (iters_out) *iters_out = it;
    rc = 0;
    for (int m = 0; m < K; ++m) {
        v_out[m] = (float)y[m];
        if (vd_out) vd_out[m] = y[m];
    }
    for (int m = 0; m < K - 1; ++m) {
        s_out[m] = (float)s[m];
        if (sd_out) sd_out[m] = s[m];
    }
    for (int m = 1; m + 1 < K; ++m)
        if (!(s_out[m - 1] < s_out[m])) rc = -2;
    free(W); free(FW); free(F2);
    return rc;
}

/* ------------------------------------------------------------------ */
/* Storage types: this file's own conversions.                         */
/* ------------------------------------------------------------------ */
static uint32_t or_f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float or_bits_f32(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* Round a double to the nearest value of a binary format with p explicit
 * mantissa bits, minimum normal exponent emin and maximum finite value vmax,
 * ties to even; returns the rounded magnitude (or INFINITY on overflow). */
static double or_round_format(double a, int p, int emin, double vmax)
{
    /* a >= 0, finite */
    if (a == 0.0) return 0.0;
    int e;
    frexp(a, &e);          /* a = m 2^e, m in [0.5, 1): floor(log2 a) = e-1 */
    int ex = e - 1;
    if (ex < emin) ex = emin;                /* subnormal quantum */
    double q = ldexp(1.0, ex - p);           /* spacing of the format at a */
    double r = rint(a / q) * q;              /* ties to even (default mode) */
    /* overflow: values at or beyond the midpoint above vmax round to inf */
    if (r > vmax) return INFINITY;
    return r;
}

/* double -> bfloat16 bits, one rounding (ties to even). */
uint16_t oracle_double_to_bf16(double d)
{
    if (isnan(d)) return (uint16_t)(signbit(d) ? 0xFFC0u : 0x7FC0u);
    uint16_t sign = signbit(d) ? 0x8000u : 0u;
    double a = fabs(d);
    if (isinf(a)) return sign | 0x7F80u;
    /* bf16: 7 explicit bits, emin = -126, max = (2 - 2^-7) 2^127 */
    double r = or_round_format(a, 7, -126, ldexp(255.0, 120));
    if (isinf(r)) return sign | 0x7F80u;
    /* r is exactly representable in fp32 with the low 16 bits zero */
    uint32_t u = or_f32_bits((float)r);
    return sign | (uint16_t)(u >> 16);
}

/* double -> IEEE binary16 bits, one rounding (ties to even). */
uint16_t oracle_double_to_f16(double d)
{
    if (isnan(d)) return (uint16_t)(signbit(d) ? 0xFE00u : 0x7E00u);
    uint16_t sign = signbit(d) ? 0x8000u : 0u;
    double a = fabs(d);
    if (isinf(a)) return sign | 0x7C00u;
    double r = or_round_format(a, 10, -14, 65504.0);
    if (isinf(r)) return sign | 0x7C00u;
    if (r == 0.0) return sign;
    if (r < ldexp(1.0, -14))                         /* subnormal: r = m 2^-24 */
        return sign | (uint16_t)(r / ldexp(1.0, -24));
    int e;
    double m = frexp(r, &e);                         /* r = m 2^e, m in [0.5,1) */
    int ex = e - 1;                                  /* r = (2m) 2^ex */
    uint16_t mant = (uint16_t)((2.0 * m - 1.0) * 1024.0);
    return sign | (uint16_t)((ex + 15) << 10) | mant;
}

/* double -> fp32 bits: C's conversion rounds to nearest even. */
uint32_t oracle_double_to_f32(double d)
{
    float f = (float)d;
    return or_f32_bits(f);
}

double oracle_bf16_to_double(uint16_t h)
{
    return (double)or_bits_f32((uint32_t)h << 16);
}

double oracle_f16_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1, ex = (h >> 10) & 0x1F, mant = h & 0x3FF;
    double v;
    if (ex == 0x1F) v = mant ? NAN : INFINITY;
    else if (ex == 0) v = ldexp((double)mant, -24);
    else v = ldexp(1024.0 + (double)mant, ex - 25);
    return sign ? -v : v;
}

static double or_load(int dtype, const void* p, int64_t i)
{
    switch (dtype) {
    case OR_F32: return (double)((const float*)p)[i];
    case OR_F16: return oracle_f16_to_double(((const uint16_t*)p)[i]);
    case OR_BF16: return oracle_bf16_to_double(((const uint16_t*)p)[i]);
    }
    return NAN;
}

static void or_store(int dtype, void* p, int64_t i, double v)
{
    switch (dtype) {
    case OR_F32: ((uint32_t*)p)[i] = oracle_double_to_f32(v); break;
    case OR_F16: ((uint16_t*)p)[i] = oracle_double_to_f16(v); break;
    case OR_BF16: ((uint16_t*)p)[i] = oracle_double_to_bf16(v); break;
    }
}

/* ------------------------------------------------------------------ */
/* Classification, packing, forward and backward.                      */
/* ------------------------------------------------------------------ */

/* idx(x) = number of boundaries s_m (m = 1..K-1) with s_m <= x (reading R7),
 * on |x| for the symmetric fit.  Compared in double: x is exact, s is fp32. */
int oracle_classify(double x, const float* s, int bits, int symmetric)
{
    const int K = 1 << bits;
    double xx = symmetric ? fabs(x) : x;
    int idx = 0;
    for (int m = 0; m < K - 1; ++m)
        if ((double)s[m] <= xx) idx += 1;
    return idx;
}

/* Words needed for n codes of b bits. */
int64_t oracle_packed_words(int64_t n, int bits)
{
    return (n * (int64_t)bits + 31) / 32;
}

/* Dense little-endian LSB-first stream: bit t of code i is stream bit
 * p = bits*i + t, stored in word p/32 at bit position p%32.  Words are
 * cleared first, so unused high bits of the last word are zero. */
void oracle_pack(const uint8_t* idx, int64_t n, int bits, uint32_t* words)
{
    int64_t nw = oracle_packed_words(n, bits);
    for (int64_t k = 0; k < nw; ++k) words[k] = 0u;
    for (int64_t i = 0; i < n; ++i)
        for (int t = 0; t < bits; ++t)
            if ((idx[i] >> t) & 1u) {
                int64_t p = (int64_t)bits * i + t;
                words[p >> 5] |= 1u << (p & 31);
            }
}

void oracle_unpack(const uint32_t* words, int64_t n, int bits, uint8_t* idx)
{
    for (int64_t i = 0; i < n; ++i) {
        unsigned c = 0;
        for (int t = 0; t < bits; ++t) {
            int64_t p = (int64_t)bits * i + t;
            c |= ((words[p >> 5] >> (p & 31)) & 1u) << t;
        }
        idx[i] = (uint8_t)c;
    }
}

/* Forward (Listing 1): y = f(x) rounded once to the dtype; idx = sorted
 * search of x among the boundaries; indices packed.  When idx_out is not
 * NULL the unpacked indices are returned too. */
int oracle_fwd(int act, int dtype, int bits, int symmetric, const float* s,
               const void* x, void* y, uint32_t* codes, uint8_t* idx_out,
               int64_t n)
{
    if (bits < 1 || bits > 4 || n < 0) return -1;
    uint8_t* idx = idx_out ? idx_out : (uint8_t*)calloc((size_t)(n > 0 ? n : 1), 1);
    if (!idx) return -1;
    for (int64_t i = 0; i < n; ++i) {
        double xi = or_load(dtype, x, i);
        idx[i] = (uint8_t)oracle_classify(xi, s, bits, symmetric);
        or_store(dtype, y, i, oracle_f(act, xi));
    }
    oracle_pack(idx, n, bits, codes);
    if (!idx_out) free(idx);
    return 0;
}

/* Backward (Eq. (1), Listing 1): grad_in = grad_out * v[idx], with the
 * product formed in fp32 and then rounded to the dtype (reading R8). */
int oracle_bwd(int dtype, int bits, const float* v, const void* g,
               const uint32_t* codes, void* gin, int64_t n)
{
    if (bits < 1 || bits > 4 || n < 0) return -1;
    for (int64_t i = 0; i < n; ++i) {
        unsigned c = 0;
        for (int t = 0; t < bits; ++t) {
            int64_t p = (int64_t)bits * i + t;
            c |= ((codes[p >> 5] >> (p & 31)) & 1u) << t;
        }
        double gi = or_load(dtype, g, i);
        /* product of two fp32 values is exact in double; (float) rounds it
         * once, which is the fp32 product */
        float prod = (float)(gi * (double)v[c]);
        or_store(dtype, gin, i, (double)prod);
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Threaded drivers for large parity cases: the range is cut into      */
/* chunks of whole 32-element groups, so each packed word has exactly  */
/* one writer.  Each chunk runs the scalar functions above unchanged.  */
/* ------------------------------------------------------------------ */
typedef struct {
    int fwd, act, dtype, bits, symmetric;
    const float* s; const float* v;
    const uint8_t* in; uint8_t* out; uint32_t* codes; const uint32_t* ccodes;
    int64_t lo, hi;   /* element range, lo a multiple of 32 */
    int rc;
} or_job;

static size_t or_esize(int dtype) { return dtype == OR_F32 ? 4 : 2; }

static void* or_worker(void* arg)
{
    or_job* j = (or_job*)arg;
    int64_t cnt = j->hi - j->lo;
    size_t es = or_esize(j->dtype);
    int64_t w0 = j->lo / 32 * j->bits;   /* first word of this chunk */
    if (j->fwd) {
        j->rc = oracle_fwd(j->act, j->dtype, j->bits, j->symmetric, j->s,
                           j->in + (size_t)j->lo * es, j->out + (size_t)j->lo * es,
                           j->codes + w0, NULL, cnt);
    } else {
        j->rc = oracle_bwd(j->dtype, j->bits, j->v, j->in + (size_t)j->lo * es,
                           j->ccodes + w0, j->out + (size_t)j->lo * es, cnt);
    }
    return NULL;
}

static int or_run_mt(or_job proto, int64_t n, int threads)
{
    if (threads < 1) threads = 1;
    if (threads > 256) threads = 256;
    int64_t groups = (n + 31) / 32;
    int64_t per = (groups + threads - 1) / threads;
    pthread_t tid[256];
    or_job jobs[256];
    int started = 0, rc = 0;
    for (int t = 0; t < threads; ++t) {
        int64_t lo = (int64_t)t * per * 32, hi = lo + per * 32;
        if (lo >= n) break;
        if (hi > n) hi = n;
        jobs[t] = proto;
        jobs[t].lo = lo; jobs[t].hi = hi; jobs[t].rc = 0;
        if (pthread_create(&tid[t], NULL, or_worker, &jobs[t]) != 0) { rc = -1; break; }
        ++started;
    }
    for (int t = 0; t < started; ++t) {
        pthread_join(tid[t], NULL);
        if (jobs[t].rc) rc = jobs[t].rc;
    }
    return rc;
}

int oracle_fwd_mt(int act, int dtype, int bits, int symmetric, const float* s,
                  const void* x, void* y, uint32_t* codes, int64_t n, int threads)
{
    if (bits < 1 || bits > 4 || n < 0) return -1;
    if (n == 0) return 0;
    or_job p;
    memset(&p, 0, sizeof p);
    p.fwd = 1; p.act = act; p.dtype = dtype; p.bits = bits; p.symmetric = symmetric;
    p.s = s; p.in = (const uint8_t*)x; p.out = (uint8_t*)y; p.codes = codes;
    return or_run_mt(p, n, threads);
}

int oracle_bwd_mt(int dtype, int bits, const float* v, const void* g,
                  const uint32_t* codes, void* gin, int64_t n, int threads)
{
    if (bits < 1 || bits > 4 || n < 0) return -1;
    if (n == 0) return 0;
    or_job p;
    memset(&p, 0, sizeof p);
    p.fwd = 0; p.dtype = dtype; p.bits = bits; p.v = v;
    p.in = (const uint8_t*)g; p.out = (uint8_t*)gin; p.ccodes = codes;
    return or_run_mt(p, n, threads);
}

/* Batch conversions for the tests: double -> storage bits of the dtype, and
 * storage bits -> double.  Same scalar functions as above. */
void oracle_round_array(int dtype, const double* in, void* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) or_store(dtype, out, i, in[i]);
}

void oracle_widen_array(int dtype, const void* in, double* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = or_load(dtype, in, i);
}
