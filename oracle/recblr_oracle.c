/*
 * fp64 CPU oracle for the BD-LRU (behavior-dependent linear recurrent unit)
 * of RecBLR, "Behavior-Dependent Linear Recurrent Units for Efficient
 * Sequential Recommendation" (CIKM 2024, arXiv 2406.12580).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or constant with the HIP library and must never be reached from it.
 *
 * What it computes (section 3.2, equation eq:linrnn and the gate equations):
 *   r_t = sigma(W_r x_t + b_r),  i_t = sigma(W_i x_t + b_i)
 *   alpha_t = exp(-softplus(Lambda) * r_t)
 *   beta_t  = sqrt(1 - alpha_t^2) * i_t
 *   h_t     = alpha_t * h_{t-1} + beta_t * x_t
 * The parallel scan of section 3.3 (operator "bullet", equation eq:h_scan)
 * reaches exactly this sequential result, so the oracle is the plain
 * sequential loop over t for every channel (b, d), in double precision.
 *
 * Layout: every [B][L][D] tensor is row-major with D fastest; [B][D] and
 * [D][D] likewise.  W is stored [out][in] so z[d] = sum_k W[d][k] x[k] + b[d].
 * h0 == NULL means a zero initial state (the paper's c_1 = beta'_1).
 *
 * Readings of the paper that this file takes (the paper is silent on them):
 *   - 1 - alpha^2 is evaluated as -expm1(-2q), q = softplus(Lambda) * r;
 *     it is the same number, without the cancellation of 1 - alpha*alpha.
 *   - The backward pass is the exact adjoint of the forward recurrence
 *     (derived here; the paper gives no backward formulas).
 *   - Gated recurrent layer core (Algorithm alg:gated_recurrent):
 *     the causal Conv1d is depthwise with K taps and a bias per channel,
 *     c_t[d] = b[d] + sum_{j<K} w[d][j] hx_{t-j}[d] with hx_{t<0} = 0 (the
 *     kernel size is not stated); x' = SiLU(c) feeds both the gate
 *     projections and the recurrence; the output is y = h (x) SiLU(hz).
 *     Its backward is the chain rule through those three lines.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double sigmoid(double z) { return 1.0 / (1.0 + exp(-z)); }

/* softplus(v) = log(1 + e^v), evaluated without overflow. */
static double softplus(double v) { return (v > 0.0 ? v : 0.0) + log1p(exp(-fabs(v))); }

/* Gate values of one element from its two pre-activations (section 3.2). */
typedef struct {
    double r, i, q, alpha, m, beta; /* m = 1 - alpha^2 */
} gates;

static gates gate_values(double zr, double zi, double s) {
    gates g;
    g.r = sigmoid(zr);
    g.i = sigmoid(zi);
    g.q = s * g.r;
    g.alpha = exp(-g.q);
    g.m = -expm1(-2.0 * g.q);
    g.beta = sqrt(g.m) * g.i;
    return g;
}

/* ------------------------------------------------------------------ */
/* Raw first-order recurrence h_t = a_t * h_{t-1} + u_t (eq:linrnn with
 * alpha_t = a_t and beta'_t = u_t given directly).                     */
void oracle_linear_scan(int64_t B, int64_t L, int64_t D, const double* a, const double* u,
                        const double* h0, double* h, double* hT) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t d = 0; d < D; ++d) {
            double state = h0 ? h0[b * D + d] : 0.0;
            for (int64_t t = 0; t < L; ++t) {
                int64_t k = (b * L + t) * D + d;
                state = a[k] * state + u[k];
                h[k] = state;
            }
            if (hT) hT[b * D + d] = state;
        }
}

/* ------------------------------------------------------------------ */
/* Gated scan with given pre-activations zr = W_r x + b_r, zi = W_i x + b_i. */
void oracle_scan_forward(int64_t B, int64_t L, int64_t D, const double* x, const double* zr,
                         const double* zi, const double* lambda, const double* h0, double* h,
                         double* hT) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t d = 0; d < D; ++d) {
            double s = softplus(lambda[d]);
            double state = h0 ? h0[b * D + d] : 0.0;
            for (int64_t t = 0; t < L; ++t) {
                int64_t k = (b * L + t) * D + d;
                gates g = gate_values(zr[k], zi[k], s);
                state = g.alpha * state + g.beta * x[k];
                h[k] = state;
            }
            if (hT) hT[b * D + d] = state;
        }
}

/* One recurrent step (inference): h_next = alpha * h_prev + beta * x over [B][D]. */
void oracle_scan_step(int64_t B, int64_t D, const double* x, const double* zr, const double* zi,
                      const double* lambda, const double* h_prev, double* h_next) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t d = 0; d < D; ++d) {
            int64_t k = b * D + d;
            gates g = gate_values(zr[k], zi[k], softplus(lambda[d]));
            h_next[k] = g.alpha * h_prev[k] + g.beta * x[k];
        }
}

/*
 * Backward of oracle_scan_forward.  Given G = dLoss/dh for every output h_t
 * (and optionally dhT = dLoss/dh_T for the final-state output) it returns
 *   dx   : the direct part dLoss/dx_t = delta_t * beta_t (x enters the
 *          recurrence only through beta'_t = beta_t * x_t)
 *   dzr, dzi : dLoss/dz for both gate pre-activations
 *   dlambda  : dLoss/dLambda, summed over b and t          ([D])
 *   dh0      : dLoss/dh0                                    ([B][D], may be NULL)
 * Adjoint of h_t = alpha_t h_{t-1} + beta_t x_t:
 *   delta_t = G_t + alpha_{t+1} delta_{t+1},  delta_{L+1} = 0, dhT added at t = L
 *   dLoss/dalpha_t = delta_t h_{t-1},  dLoss/dbeta_t = delta_t x_t
 *   alpha = exp(-q): dalpha/dq = -alpha
 *   beta = sqrt(1 - exp(-2q)) i: dbeta/dq = i alpha^2 / sqrt(1 - alpha^2), dbeta/di = sqrt(m)
 *   q = softplus(Lambda) r: dq/dr = softplus(Lambda), dq/dLambda = sigma(Lambda) r
 *   r = sigma(zr): dr/dzr = r (1 - r);  i = sigma(zi): di/dzi = i (1 - i)
 * The forward states are recomputed here in double precision.
 */
void oracle_scan_backward(int64_t B, int64_t L, int64_t D, const double* x, const double* zr,
                          const double* zi, const double* lambda, const double* h0,
                          const double* G, const double* dhT, double* dx, double* dzr,
                          double* dzi, double* dlambda, double* dh0) {
    double* dlam_bd = (double*)calloc((size_t)(B * D), sizeof(double));
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t d = 0; d < D; ++d) {
            double s = softplus(lambda[d]);
            double init = h0 ? h0[b * D + d] : 0.0;
            double* hs = (double*)malloc((size_t)(L > 0 ? L : 1) * sizeof(double));
            double state = init;
            for (int64_t t = 0; t < L; ++t) {
                int64_t k = (b * L + t) * D + d;
                gates g = gate_values(zr[k], zi[k], s);
                state = g.alpha * state + g.beta * x[k];
                hs[t] = state;
            }
            double delta_next = 0.0, alpha_next = 0.0, ds = 0.0;
            for (int64_t t = L - 1; t >= 0; --t) {
                int64_t k = (b * L + t) * D + d;
                gates g = gate_values(zr[k], zi[k], s);
                double delta = G[k] + alpha_next * delta_next;
                if (t == L - 1 && dhT) delta += dhT[b * D + d];
                double h_prev = t > 0 ? hs[t - 1] : init;
                double g_alpha = delta * h_prev;
                double g_beta = delta * x[k];
                dx[k] = delta * g.beta;
                double g_q = -g.alpha * g_alpha + g_beta * g.i * g.alpha * g.alpha / sqrt(g.m);
                dzr[k] = g_q * s * g.r * (1.0 - g.r);
                dzi[k] = g_beta * sqrt(g.m) * g.i * (1.0 - g.i);
                ds += g_q * g.r;
                delta_next = delta;
                alpha_next = g.alpha;
            }
            if (dh0) {
                /* dLoss/dh0 = alpha_1 * delta_1; with L = 0 the state passes through. */
                double pass = (L == 0 && dhT) ? dhT[b * D + d] : 0.0;
                dh0[b * D + d] = L > 0 ? alpha_next * delta_next : pass;
            }
            dlam_bd[b * D + d] = ds * sigmoid(lambda[d]);
            free(hs);
        }
    for (int64_t d = 0; d < D; ++d) {
        double acc = 0.0;
        for (int64_t b = 0; b < B; ++b) acc += dlam_bd[b * D + d];
        dlambda[d] = acc;
    }
    free(dlam_bd);
}

/* ------------------------------------------------------------------ */
/* Gate pre-activation projection z = x W^T + b over M rows (section 3.2). */
void oracle_project(int64_t M, int64_t D, const double* x, const double* W, const double* bias,
                    double* z) {
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < M; ++row)
        for (int64_t o = 0; o < D; ++o) {
            double acc = bias ? bias[o] : 0.0;
            for (int64_t k = 0; k < D; ++k) acc += W[o * D + k] * x[row * D + k];
            z[row * D + o] = acc;
        }
}

/* Full forward: projections, then the gated scan. */
void oracle_forward(int64_t B, int64_t L, int64_t D, const double* x, const double* Wr,
                    const double* br, const double* Wi, const double* bi, const double* lambda,
                    const double* h0, double* h, double* hT) {
    size_t n = (size_t)(B * L * D);
    double* zr = (double*)malloc((n ? n : 1) * sizeof(double));
    double* zi = (double*)malloc((n ? n : 1) * sizeof(double));
    oracle_project(B * L, D, x, Wr, br, zr);
    oracle_project(B * L, D, x, Wi, bi, zi);
    oracle_scan_forward(B, L, D, x, zr, zi, lambda, h0, h, hT);
    free(zr);
    free(zi);
}

/*
 * Full backward: the scan backward, then the projection backward
 *   dx += dzr W_r + dzi W_i,  dW = sum_rows dz^T x,  db = sum_rows dz.
 * dx receives the total gradient with respect to x.
 */
void oracle_backward(int64_t B, int64_t L, int64_t D, const double* x, const double* Wr,
                     const double* br, const double* Wi, const double* bi, const double* lambda,
                     const double* h0, const double* G, const double* dhT, double* dx,
                     double* dWr, double* dbr, double* dWi, double* dbi, double* dlambda,
                     double* dh0) {
    int64_t M = B * L;
    size_t n = (size_t)(M * D);
    double* zr = (double*)malloc((n ? n : 1) * sizeof(double));
    double* zi = (double*)malloc((n ? n : 1) * sizeof(double));
    double* dzr = (double*)malloc((n ? n : 1) * sizeof(double));
    double* dzi = (double*)malloc((n ? n : 1) * sizeof(double));
    oracle_project(M, D, x, Wr, br, zr);
    oracle_project(M, D, x, Wi, bi, zi);
    oracle_scan_backward(B, L, D, x, zr, zi, lambda, h0, G, dhT, dx, dzr, dzi, dlambda, dh0);
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < M; ++row)
        for (int64_t k = 0; k < D; ++k) {
            double acc = 0.0;
            for (int64_t o = 0; o < D; ++o)
                acc += dzr[row * D + o] * Wr[o * D + k] + dzi[row * D + o] * Wi[o * D + k];
            dx[row * D + k] += acc;
        }
    /* dW[o][k] = sum over rows (ascending) of dz[row][o] x[row][k]; the row loop
     * sits outside the k loop only so that x is read along its rows. */
#pragma omp parallel for schedule(static)
    for (int64_t o = 0; o < D; ++o) {
        double* wr = dWr + o * D;
        double* wi = dWi + o * D;
        for (int64_t k = 0; k < D; ++k) {
            wr[k] = 0.0;
            wi[k] = 0.0;
        }
        double sr = 0.0, si = 0.0;
        for (int64_t row = 0; row < M; ++row) {
            const double gr = dzr[row * D + o], gi = dzi[row * D + o];
            const double* xr = x + row * D;
            for (int64_t k = 0; k < D; ++k) {
                wr[k] += gr * xr[k];
                wi[k] += gi * xr[k];
            }
            sr += gr;
            si += gi;
        }
        dbr[o] = sr;
        dbi[o] = si;
    }
    free(zr);
    free(zi);
    free(dzr);
    free(dzi);
}

/*
 * Gated recurrent layer core (Algorithm alg:gated_recurrent):
 *   x'_t = SiLU(conv_b + sum_{j<K} conv_w[.][j] * hx_{t-j})   (causal, depthwise)
 *   h    = BD-LRU(x') with z = x' W^T + b                    (section 3.2)
 *   y_t  = h_t * SiLU(hz_t)
 * hx, hz, y, h: [B][L][D]; conv_w: [D][K]; conv_b: [D] or NULL.  h may be NULL.
 */
static double silu(double v) { return v / (1.0 + exp(-v)); }

void oracle_gated_forward(int64_t B, int64_t L, int64_t D, int64_t K, const double* hx,
                          const double* hz, const double* conv_w, const double* conv_b,
                          const double* Wr, const double* br, const double* Wi,
                          const double* bi, const double* lambda, const double* h0, double* y,
                          double* h, double* hT) {
    size_t n = (size_t)(B * L * D);
    double* xp = (double*)malloc((n ? n : 1) * sizeof(double));
    double* hh = (double*)malloc((n ? n : 1) * sizeof(double));
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t d = 0; d < D; ++d)
            for (int64_t t = 0; t < L; ++t) {
                double c = conv_b ? conv_b[d] : 0.0;
                for (int64_t j = 0; j < K && j <= t; ++j)
                    c += conv_w[d * K + j] * hx[(b * L + t - j) * D + d];
                xp[(b * L + t) * D + d] = silu(c);
            }
    oracle_forward(B, L, D, xp, Wr, br, Wi, bi, lambda, h0, hh, hT);
    for (size_t e = 0; e < n; ++e) {
        y[e] = hh[e] * silu(hz[e]);
        if (h) h[e] = hh[e];
    }
    free(xp);
    free(hh);
}

/*
 * Backward of oracle_gated_forward (the paper states no backward; this is the
 * exact adjoint of the three lines, by the chain rule):
 *   dh    = dy * SiLU(hz)                      (plus dhT on the final state)
 *   dhz   = dy * h * SiLU'(hz),  SiLU'(v) = s (1 + v (1 - s)), s = sigma(v)
 *   dx', dW_r, db_r, dW_i, db_i, dLambda, dh0 = oracle_backward at x' with dh
 *   dc    = dx' * SiLU'(c)                     (c: the conv output, x' = SiLU(c))
 *   dhx_t = sum_{j<K, t+j<L} conv_w[.][j] dc_{t+j}     (the causal conv's transpose)
 *   dconv_w[d][j] = sum_{b, t>=j} dc_t[d] hx_{t-j}[d],  dconv_b[d] = sum_{b,t} dc_t[d]
 * dy, dhx, dhz: [B][L][D]; dhT, h0, dh0: [B][D] or NULL; dconv_w: [D][K];
 * dconv_b: [D] (always written).
 */
static double dsilu(double v) {
    double s = sigmoid(v);
    return s * (1.0 + v * (1.0 - s));
}

void oracle_gated_backward(int64_t B, int64_t L, int64_t D, int64_t K, const double* hx,
                           const double* hz, const double* conv_w, const double* conv_b,
                           const double* Wr, const double* br, const double* Wi,
                           const double* bi, const double* lambda, const double* h0,
                           const double* dy, const double* dhT, double* dhx, double* dhz,
                           double* dconv_w, double* dconv_b, double* dWr, double* dbr,
                           double* dWi, double* dbi, double* dlambda, double* dh0) {
    size_t n = (size_t)(B * L * D);
    size_t nb = (n ? n : 1) * sizeof(double);
    double* c = (double*)malloc(nb);
    double* xp = (double*)malloc(nb);
    double* hh = (double*)malloc(nb);
    double* dh = (double*)malloc(nb);
    double* dxp = (double*)malloc(nb);
    double* hT = (double*)malloc((size_t)(B * D ? B * D : 1) * sizeof(double));
    /* forward recomputation: the conv, x' and h */
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < L; ++t)
            for (int64_t d = 0; d < D; ++d) {
                double acc = conv_b ? conv_b[d] : 0.0;
                for (int64_t j = 0; j < K && j <= t; ++j)
                    acc += conv_w[d * K + j] * hx[(b * L + t - j) * D + d];
                c[(b * L + t) * D + d] = acc;
                xp[(b * L + t) * D + d] = silu(acc);
            }
    oracle_forward(B, L, D, xp, Wr, br, Wi, bi, lambda, h0, hh, hT);
    /* output gate */
    for (size_t e = 0; e < n; ++e) {
        dh[e] = dy[e] * silu(hz[e]);
        dhz[e] = dy[e] * hh[e] * dsilu(hz[e]);
    }
    /* BD-LRU with its projections */
    oracle_backward(B, L, D, xp, Wr, br, Wi, bi, lambda, h0, dh, dhT, dxp, dWr, dbr, dWi, dbi,
                    dlambda, dh0);
    /* SiLU and the causal depthwise conv */
    for (size_t e = 0; e < n; ++e) dxp[e] *= dsilu(c[e]);  /* now dc */
    for (int64_t d = 0; d < D; ++d) {
        for (int64_t j = 0; j < K; ++j) dconv_w[d * K + j] = 0.0;
        dconv_b[d] = 0.0;
    }
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < L; ++t)
            for (int64_t d = 0; d < D; ++d) {
                double acc = 0.0;
                for (int64_t j = 0; j < K && t + j < L; ++j)
                    acc += conv_w[d * K + j] * dxp[(b * L + t + j) * D + d];
                dhx[(b * L + t) * D + d] = acc;
                double g = dxp[(b * L + t) * D + d];
                dconv_b[d] += g;
                for (int64_t j = 0; j < K && j <= t; ++j)
                    dconv_w[d * K + j] += g * hx[(b * L + t - j) * D + d];
            }
    free(c);
    free(xp);
    free(hh);
    free(dh);
    free(dxp);
    free(hT);
}

/* Full single step: projections of x_t, then one recurrence step. */
void oracle_step(int64_t B, int64_t D, const double* x, const double* Wr, const double* br,
                 const double* Wi, const double* bi, const double* lambda, const double* h_prev,
                 double* h_next) {
    size_t n = (size_t)(B * D);
    double* zr = (double*)malloc((n ? n : 1) * sizeof(double));
    double* zi = (double*)malloc((n ? n : 1) * sizeof(double));
    oracle_project(B, D, x, Wr, br, zr);
    oracle_project(B, D, x, Wi, bi, zi);
    oracle_scan_step(B, D, x, zr, zi, lambda, h_prev, h_next);
    free(zr);
    free(zi);
}
