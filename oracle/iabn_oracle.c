/*
 * Oracle for In-Place Activated Batch Normalization (InPlace-ABN),
 * Rota Bulo, Porzi, Kontschieder, "In-Place Activated BatchNorm for
 * Memory-Optimized Training of DNNs", CVPR 2018 (arXiv:1712.02616).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * CPU definition that the GPU library is checked against.  Only the tests,
 * the smoke check and the benchmark's CPU-baseline leg load it; the product
 * library never calls, links or includes anything from here, and nothing
 * here comes from the GPU library.
 *
 * Everything is computed in double precision.  Tensors are NCHW, viewed as
 * [N][C][HW] with HW = H*W contiguous; a BN "unit" is a channel, so each
 * channel owns m = N*HW values (Sec. 3.1 fixes one unit and its m minibatch
 * values; parameters are channel-specific).
 *
 * Parity status of each function (what pins it is in the tests):
 *   oracle_batch_stats            pinned: exact rational arithmetic, closed forms
 *   oracle_forward_train          pinned: closed forms, invariants, hand-derived
 *                                 worked example, exact rational arithmetic
 *   oracle_forward_eval           pinned: equals the training forward when the
 *                                 running statistics equal the batch statistics
 *   oracle_backward_i             pinned: central finite differences of the
 *                                 forward, equality with three other
 *                                 formulations, closed-form invariants
 *   oracle_backward_ii            pinned: as above
 *   oracle_backward_standard      pinned: as above; with z given, equal to the
 *                                 backward from z and y-based form where signs agree
 *   oracle_normalize              pinned: closed form, invariants (sum xhat = 0,
 *                                 mean xhat^2 = sigma^2/(sigma^2 + eps))
 *   oracle_scale_shift_act        pinned: equals the training forward's z on
 *                                 the normalised input; dyadic exact case
 *   oracle_backward_from_xhat     pinned: central finite differences, equality
 *                                 with the backward from z and from x
 *   oracle_leaky_relu(_inv)       pinned: exact round trip for dyadic slopes
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define IDX(n, c, i) ((((size_t)(n)) * (size_t)C + (size_t)(c)) * (size_t)HW + (size_t)(i))

/* Neumaier's compensated summation, used so that the oracle's sums carry
 * (almost) no rounding error of their own. */
typedef struct {
    double s;
    double comp;
} csum_t;

static void csum_add(csum_t *a, double v) {
    double t = a->s + v;
    if (fabs(a->s) >= fabs(v))
        a->comp += (a->s - t) + v;
    else
        a->comp += (v - t) + a->s;
    a->s = t;
}

static double csum_value(const csum_t *a) { return a->s + a->comp; }

/* Threads the OpenMP loops below use (1 when built without OpenMP). */
int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Leaky ReLU with slope a for negative inputs, and its inverse (Sec. 3.3,
 * "Invertible activation function"): f(y) = y for y >= 0, a*y otherwise;
 * f^-1(z) = z for z >= 0, z/a otherwise. */
double oracle_leaky_relu(double y, double a) { return (y >= 0.0) ? y : a * y; }

double oracle_leaky_relu_inv(double z, double a) { return (z >= 0.0) ? z : z / a; }

/* Derivative of the leaky ReLU, as the activation's backward step of
 * Algorithm 2 uses it: 1 on the identity branch, a on the scaled branch.  The
 * branch is taken from the stored output z; since f preserves sign for a > 0,
 * z >= 0 exactly when y >= 0. */
static double leaky_relu_slope_from_z(double z, double a) { return (z >= 0.0) ? 1.0 : a; }

/* Per-channel minibatch mean and biased variance (Sec. 3.1):
 *   mu = (1/m) sum_j x_j,   sigma^2 = (1/m) sum_j (x_j - mu)^2.
 * Two passes, compensated sums. */
void oracle_batch_stats(const double *x, int64_t N, int64_t C, int64_t HW,
                        double *mean, double *var) {
    const double m = (double)(N * HW);
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        csum_t s = {0.0, 0.0};
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) csum_add(&s, x[IDX(n, c, i)]);
        const double mu = csum_value(&s) / m;
        csum_t q = {0.0, 0.0};
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const double d = x[IDX(n, c, i)] - mu;
                csum_add(&q, d * d);
            }
        mean[c] = mu;
        var[c] = csum_value(&q) / m;
    }
}

/* Training-mode forward of the fused BN + activation layer (Algorithm 1):
 *   y = BN_{gamma,beta}(x) with batch statistics (Eq. 1 and the scale-and-shift
 *   of Sec. 3.1), z = f(y).  z is the only activation kept for the backward;
 *   mean and var (biased) are returned as the small per-channel buffers.
 * The running statistics are blended with the batch statistics,
 *   running_mean <- (1 - momentum) * running_mean + momentum * mu,
 *   running_var  <- (1 - momentum) * running_var  + momentum * sigma^2 * m/(m-1),
 * i.e. a running average of the minibatch statistics (Sec. 3.1, test-time
 * statistics) with the unbiased variance estimate used at inference by the
 * original BatchNorm paper.  Normalisation itself uses the biased variance.
 * x and z may be the same array (the layer computes in place). */
void oracle_forward_train(const double *x, int64_t N, int64_t C, int64_t HW,
                          const double *gamma, const double *beta, double eps,
                          double momentum, double slope, double *running_mean,
                          double *running_var, double *z, double *mean, double *var) {
    const double m = (double)(N * HW);
    oracle_batch_stats(x, N, C, HW, mean, var);
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        const double denom = sqrt(var[c] + eps);
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double xhat = (x[k] - mean[c]) / denom;
                const double y = gamma[c] * xhat + beta[c];
                z[k] = oracle_leaky_relu(y, slope);
            }
        running_mean[c] = (1.0 - momentum) * running_mean[c] + momentum * mean[c];
        running_var[c] = (1.0 - momentum) * running_var[c] + momentum * var[c] * m / (m - 1.0);
    }
}

/* Inference-mode forward (Sec. 3.1, last paragraph): the statistics are fixed
 * to the running estimates, z = f(gamma * (x - mu_T) / sqrt(sigma_T^2 + eps) + beta). */
void oracle_forward_eval(const double *x, int64_t N, int64_t C, int64_t HW,
                         const double *gamma, const double *beta,
                         const double *running_mean, const double *running_var,
                         double eps, double slope, double *z) {
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        const double denom = sqrt(running_var[c] + eps);
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double y = gamma[c] * (x[k] - running_mean[c]) / denom + beta[c];
                z[k] = oracle_leaky_relu(y, slope);
            }
    }
}

/* Backward of InPlace-ABN I (Algorithm 2, first branch; Sec. 3.3 "Backward
 * pass through BN"), from the stored output z and the biased variance only:
 *   dL/dy = dL/dz * f'(y)                (activation backward)
 *   y     = f^-1(z)                      (invert the activation)
 *   xhat  = (y - beta) / gamma           (invert the scale-and-shift)
 *   dL/dbeta  = sum_i dL/dy_i,  dL/dgamma = sum_i dL/dy_i * xhat_i
 *   dL/dx_i = (dL/dy_i - dL/dgamma * xhat_i / m - dL/dbeta / m) * gamma / sqrt(sigma^2 + eps).
 * dgamma and dbeta are written, not accumulated.  dz and dx may be the same
 * array. */
void oracle_backward_i(const double *z, const double *dz, int64_t N, int64_t C, int64_t HW,
                       const double *gamma, const double *beta, const double *var,
                       double eps, double slope, double *dx, double *dgamma, double *dbeta) {
    const double m = (double)(N * HW);
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        csum_t sdy = {0.0, 0.0}, sdyx = {0.0, 0.0};
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double dy = dz[k] * leaky_relu_slope_from_z(z[k], slope);
                const double y = oracle_leaky_relu_inv(z[k], slope);
                const double xhat = (y - beta[c]) / gamma[c];
                csum_add(&sdy, dy);
                csum_add(&sdyx, dy * xhat);
            }
        const double db = csum_value(&sdy);
        const double dg = csum_value(&sdyx);
        const double scale = gamma[c] / sqrt(var[c] + eps);
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double dy = dz[k] * leaky_relu_slope_from_z(z[k], slope);
                const double y = oracle_leaky_relu_inv(z[k], slope);
                const double xhat = (y - beta[c]) / gamma[c];
                dx[k] = (dy - dg * xhat / m - db / m) * scale;
            }
        dgamma[c] = dg;
        dbeta[c] = db;
    }
}

/* Backward of InPlace-ABN II (Algorithm 2, second branch; Sec. 3.3 and the
 * Appendix): the same gradients written as functions of y, so that the
 * inversion of the scale-and-shift never happens per element:
 *   dL/dbeta  = sum_i dL/dy_i
 *   dL/dgamma = (sum_i dL/dy_i * y_i - beta * dL/dbeta) / gamma
 *   dL/dx_i = [dL/dy_i - dL/dgamma * y_i / (gamma m)
 *              - (dL/dbeta - beta * dL/dgamma / gamma) / m] * gamma / sqrt(sigma^2 + eps). */
void oracle_backward_ii(const double *z, const double *dz, int64_t N, int64_t C, int64_t HW,
                        const double *gamma, const double *beta, const double *var,
                        double eps, double slope, double *dx, double *dgamma, double *dbeta) {
    const double m = (double)(N * HW);
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        csum_t sdy = {0.0, 0.0}, sdyy = {0.0, 0.0};
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double dy = dz[k] * leaky_relu_slope_from_z(z[k], slope);
                const double y = oracle_leaky_relu_inv(z[k], slope);
                csum_add(&sdy, dy);
                csum_add(&sdyy, dy * y);
            }
        const double db = csum_value(&sdy);
        const double dg = (csum_value(&sdyy) - beta[c] * db) / gamma[c];
        const double scale = gamma[c] / sqrt(var[c] + eps);
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double dy = dz[k] * leaky_relu_slope_from_z(z[k], slope);
                const double y = oracle_leaky_relu_inv(z[k], slope);
                dx[k] = (dy - dg * y / (gamma[c] * m) - (db - beta[c] * dg / gamma[c]) / m) * scale;
            }
        dgamma[c] = dg;
        dbeta[c] = db;
    }
}

/* Backward of the standard BN + activation block (Sec. 3.2, "Standard"), which
 * keeps the BN input x and the batch mean as well as the variance.  That block
 * also keeps the activation's output z for the activation's backward: when z
 * is given, the derivative of f is taken from it (as in the backward from z,
 * 1 where z >= 0); with z == NULL it is taken on the recomputed y.  The BN gradient is
 * assembled with the chain rule of the original BatchNorm paper as laid out in
 * the Appendix: dL/dxhat_j = dL/dy_j * gamma,
 *   dL/dsigma^2 = sum_j dL/dxhat_j * (x_j - mu) * (-1/2) (sigma^2 + eps)^(-3/2),
 *   dL/dmu      = -sum_j dL/dxhat_j / sqrt(sigma^2 + eps)
 *                 + dL/dsigma^2 * sum_j (-2 (x_j - mu)) / m,
 *   dL/dx_i = dL/dxhat_i / sqrt(sigma^2 + eps) + dL/dsigma^2 * 2 (x_i - mu) / m + dL/dmu / m. */
void oracle_backward_standard(const double *x, const double *z, const double *dz, int64_t N,
                              int64_t C, int64_t HW, const double *gamma, const double *beta,
                              const double *mean, const double *var, double eps,
                              double slope, double *dx, double *dgamma, double *dbeta) {
    const double m = (double)(N * HW);
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        const double denom = sqrt(var[c] + eps);
        csum_t sdy = {0.0, 0.0}, sdyx = {0.0, 0.0}, sdvar = {0.0, 0.0}, sdmu = {0.0, 0.0},
               sxc = {0.0, 0.0};
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double xc = x[k] - mean[c];
                const double xhat = xc / denom;
                const double y = gamma[c] * xhat + beta[c];
                const double dy = dz[k] * (z ? leaky_relu_slope_from_z(z[k], slope)
                                             : ((y >= 0.0) ? 1.0 : slope));
                const double dxhat = dy * gamma[c];
                csum_add(&sdy, dy);
                csum_add(&sdyx, dy * xhat);
                csum_add(&sdvar, dxhat * xc * (-0.5) * pow(var[c] + eps, -1.5));
                csum_add(&sdmu, -dxhat / denom);
                csum_add(&sxc, -2.0 * xc);
            }
        const double dvar = csum_value(&sdvar);
        const double dmu = csum_value(&sdmu) + dvar * csum_value(&sxc) / m;
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double xc = x[k] - mean[c];
                const double y = gamma[c] * xc / denom + beta[c];
                const double dy = dz[k] * (z ? leaky_relu_slope_from_z(z[k], slope)
                                             : ((y >= 0.0) ? 1.0 : slope));
                const double dxhat = dy * gamma[c];
                dx[k] = dxhat / denom + dvar * 2.0 * xc / m + dmu / m;
            }
        dgamma[c] = csum_value(&sdyx);
        dbeta[c] = csum_value(&sdy);
    }
}

/* The normalised input of Eq. (1), xhat = (x - mu)/sqrt(sigma^2 + eps), for
 * given per-channel mu and sigma^2: what the proposed checkpointing keeps for
 * the backward (Sec. 3.2, "Checkpointing (proposed version)"). */
void oracle_normalize(const double *x, int64_t N, int64_t C, int64_t HW, const double *mean,
                      const double *var, double eps, double *xhat) {
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        const double denom = sqrt(var[c] + eps);
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                xhat[k] = (x[k] - mean[c]) / denom;
            }
    }
}

/* z = f(pi(xhat)) = f(gamma*xhat + beta): the recomputation of z from the
 * stored xhat in the backward of the proposed checkpointing (Sec. 3.2). */
void oracle_scale_shift_act(const double *xhat, int64_t N, int64_t C, int64_t HW,
                            const double *gamma, const double *beta, double slope, double *z) {
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                z[k] = oracle_leaky_relu(gamma[c] * xhat[k] + beta[c], slope);
            }
}

/* Backward of the proposed checkpointing from the stored xhat (BN* of
 * Sec. 3.2, with the BN backward of Sec. 3.3): y = gamma*xhat + beta,
 * dy = dz * f'(y) (1 for y >= 0, slope otherwise),
 *   dbeta = sum dy,  dgamma = sum dy*xhat,
 *   dx = (dy - dgamma*xhat/m - dbeta/m) * gamma/sqrt(sigma^2 + eps). */
void oracle_backward_from_xhat(const double *xhat, const double *dz, int64_t N, int64_t C,
                               int64_t HW, const double *gamma, const double *beta,
                               const double *var, double eps, double slope, double *dx,
                               double *dgamma, double *dbeta) {
    const double m = (double)(N * HW);
    int64_t c;
#pragma omp parallel for schedule(dynamic, 1)
    for (c = 0; c < C; ++c) {
        csum_t sdy = {0.0, 0.0}, sdyx = {0.0, 0.0};
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double y = gamma[c] * xhat[k] + beta[c];
                const double dy = dz[k] * ((y >= 0.0) ? 1.0 : slope);
                csum_add(&sdy, dy);
                csum_add(&sdyx, dy * xhat[k]);
            }
        const double db = csum_value(&sdy), dg = csum_value(&sdyx);
        const double scale = gamma[c] / sqrt(var[c] + eps);
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const size_t k = IDX(n, c, i);
                const double y = gamma[c] * xhat[k] + beta[c];
                const double dy = dz[k] * ((y >= 0.0) ? 1.0 : slope);
                dx[k] = (dy - dg * xhat[k] / m - db / m) * scale;
            }
        dgamma[c] = dg;
        dbeta[c] = db;
    }
}
