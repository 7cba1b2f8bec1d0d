/*
 * CPU oracle for one step of LAMB, N-LAMB, NN-LAMB and LARS.
 *
 * You, Li, Reddi, Hseu, Kumar, Bhojanapalli, Song, Demmel, Keutzer, Hsieh:
 * "Large Batch Optimization for Deep Learning: Training BERT in 76 minutes",
 * ICLR 2020 (arXiv:1904.00962).
 *
 * TEST INFRASTRUCTURE ONLY. This file is the reference the HIP library is
 * checked against; it is not part of the product. Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it. It shares
 * no code, header, table or helper with the HIP library, and it includes
 * nothing from it.
 *
 * Plain single-threaded C. Every quantity of the method is computed in
 * double; inputs are widened exactly (fp32 -> double, bf16 -> fp32 -> double)
 * and each stored value (x, m, v) is rounded to fp32 once per step, with the
 * C conversion's round-to-nearest-even. One call handles one layer block
 * x^(i) (Section 2, Notation): blocks never interact within a step, so a
 * multi-tensor step is a loop over blocks in any order.
 *
 * Readings of the paper taken here (the paper is silent or ambiguous):
 *  - m_hat and v_hat of Algorithm 2 are temporaries; the stored moments stay
 *    uncorrected (Appendix E names the division "adam-correction", as in
 *    Adam, where the corrected values are not stored).
 *  - epsilon is added after the square root of the bias-corrected v_hat.
 *  - the weight-decay term lambda * x uses the pre-update x_t, and lambda is
 *    replaced by 0 for blocks whose mask is 0 (biases and norm parameters).
 *  - a zero update norm (||r + lambda x|| = 0, or ||m|| = 0 for LARS) means
 *    every element of the update is 0: the step leaves x unchanged and the
 *    reported trust ratio is 0. Any other norm, NaN included, is divided by
 *    as written, so NaN and Inf propagate by IEEE rules.
 *  - phi(z) = min(max(z, gamma_l), gamma_u) (Section 3), evaluated with
 *    comparisons so that a NaN norm stays NaN.
 *  - LARS: the trust coefficient kappa multiplies phi (kappa = 1 is
 *    Algorithm 1 exactly); the epsilon listed among Algorithm 1's inputs is
 *    never used by the algorithm and is not taken here.
 *
 *  - g_t is the mean of the per-sample gradients (Algorithms 1 and 2); the
 *    caller may hand over the sum (or a loss-scaled value) and grad_scale,
 *    so that g_t = grad_scale * g. Whether a scaled gradient is finite is
 *    decided on the fp32 product fp32(g) * fp32(grad_scale), the precision
 *    the GPU path computes it in.
 *  - Layer norms (Appendix F): L2 is the default; the paper does not name
 *    the other norms it tried, so L1 and L-infinity are offered, used for
 *    both ||x|| and ||u||. The L-infinity maximum keeps NaN.
 *  - N-LAMB / NN-LAMB (Appendix D): the inputs {beta1^t} form a per-step
 *    sequence of momentum parameters; the paper's experiments hold it
 *    constant (beta1 = 0.975), and that constant sequence is what is taken
 *    here, so the products prod_{i<=k} beta1^i are the powers beta1^k. The
 *    moment recursions use the constant beta1 and beta2 as printed.
 *
 * Parity is pinned by the closed forms, invariants and hand-worked examples
 * in the test suite; no function here is unpinned.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-2)

/* Exact widening of a bf16 bit pattern: it is the high half of an fp32. */
static double widen_bf16(uint16_t bits)
{
    uint32_t word = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &word, sizeof f);
    return (double)f;
}

static double gradient_at(const void *g, int g_is_bf16, int64_t j)
{
    if (g_is_bf16)
        return widen_bf16(((const uint16_t *)g)[j]);
    return (double)((const float *)g)[j];
}

/* Round a double to the fp32 stored state (round to nearest, ties to even). */
static float store_f32(double a)
{
    return (float)a;
}

/* Section 3: phi(z) = min{max{z, gamma_l}, gamma_u}. */
static double phi(double z, double gamma_l, double gamma_u)
{
    double p = z;
    if (p < gamma_l)
        p = gamma_l;
    if (p > gamma_u)
        p = gamma_u;
    return p;
}

#define ORACLE_NORM_L2 0
#define ORACLE_NORM_L1 1
#define ORACLE_NORM_LINF 2

/* Add one element to a running layer norm (Appendix F). */
static double norm_add(int norm, double acc, double a)
{
    if (norm == ORACLE_NORM_L1)
        return acc + fabs(a);
    if (norm == ORACLE_NORM_LINF) {
        double b = fabs(a);
        return (isnan(b) || b > acc) ? b : acc;
    }
    return acc + a * a;
}

static double norm_finish(int norm, double acc)
{
    return norm == ORACLE_NORM_L2 ? sqrt(acc) : acc;
}

/*
 * 1 if every scaled gradient element fp32(g_j) * fp32(grad_scale), computed
 * in fp32, is finite; 0 if any is NaN or infinite.
 */
int oracle_gradient_finite(int64_t d, const void *g, int g_is_bf16, double grad_scale)
{
    float s = (float)grad_scale;
    for (int64_t j = 0; j < d; ++j) {
        float gj = (float)gradient_at(g, g_is_bf16, j);
        float p = gj * s;
        if (!isfinite(p))
            return 0;
    }
    return 1;
}

/*
 * One LAMB step (Algorithm 2) on one layer block of d elements.
 *
 *   m_t   = beta1 m_{t-1} + (1 - beta1) g_t
 *   v_t   = beta2 v_{t-1} + (1 - beta2) g_t^2
 *   m_hat = m_t / (1 - beta1^t),  v_hat = v_t / (1 - beta2^t)
 *   r_t   = m_hat / (sqrt(v_hat) + eps)
 *   u     = r_t + lambda x_t
 *   x_{t+1} = x_t - eta_t phi(||x_t||) / ||u|| * u
 *
 * bias_correction = 0 drops the two divisions (Appendix E).
 * x, m, v are updated in place; g is fp32 or, with g_is_bf16, bf16 bits, and
 * g_t = grad_scale * g. norm selects the layer norm (ORACLE_NORM_*).
 * out[0] = trust ratio phi(||x_t||)/||u||, out[1] = ||x_t||, out[2] = ||u||.
 */
int oracle_lamb_layer(int64_t d, float *x, const void *g, int g_is_bf16,
                      float *m, float *v,
                      double lr, double beta1, double beta2, double eps,
                      double weight_decay, int wd, double gamma_l,
                      double gamma_u, int64_t t, int bias_correction,
                      double grad_scale, int norm, double *out)
{
    if (d < 1 || !x || !g || !m || !v || !out || t < 1 || norm < 0 || norm > 2)
        return ORACLE_EINVAL;
    double *u = (double *)malloc((size_t)d * sizeof(double));
    if (!u)
        return ORACLE_ENOMEM;

    double c1 = 1.0, c2 = 1.0;
    if (bias_correction) {
        c1 = 1.0 - pow(beta1, (double)t);
        c2 = 1.0 - pow(beta2, (double)t);
    }
    double lam = wd ? weight_decay : 0.0;

    double sum_xx = 0.0, sum_uu = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        double gj = grad_scale * gradient_at(g, g_is_bf16, j);
        double xj = (double)x[j];
        double mj = beta1 * (double)m[j] + (1.0 - beta1) * gj;
        double vj = beta2 * (double)v[j] + (1.0 - beta2) * (gj * gj);
        double m_hat = mj / c1;
        double v_hat = vj / c2;
        double r = m_hat / (sqrt(v_hat) + eps);
        u[j] = r + lam * xj;
        sum_xx = norm_add(norm, sum_xx, xj);
        sum_uu = norm_add(norm, sum_uu, u[j]);
        m[j] = store_f32(mj);
        v[j] = store_f32(vj);
    }

    double norm_x = norm_finish(norm, sum_xx);
    double norm_u = norm_finish(norm, sum_uu);
    double ratio = (norm_u == 0.0) ? 0.0 : phi(norm_x, gamma_l, gamma_u) / norm_u;
    for (int64_t j = 0; j < d; ++j)
        x[j] = store_f32((double)x[j] - lr * ratio * u[j]);

    out[0] = ratio;
    out[1] = norm_x;
    out[2] = norm_u;
    free(u);
    return ORACLE_OK;
}

/*
 * One LARS step (Algorithm 1) on one layer block of d elements.
 *
 *   m_t     = beta1 m_{t-1} + (1 - beta1) (g_t + lambda x_t)
 *   x_{t+1} = x_t - eta_t kappa phi(||x_t||) / ||m_t|| * m_t
 *
 * x and m are updated in place; g_t = grad_scale * g; norm as for LAMB.
 * out[0] = trust ratio kappa phi/||m_t||, out[1] = ||x_t||, out[2] = ||m_t||.
 */
int oracle_lars_layer(int64_t d, float *x, const void *g, int g_is_bf16,
                      float *m, double lr, double beta1, double weight_decay,
                      int wd, double gamma_l, double gamma_u,
                      double trust_coef, double grad_scale, int norm, double *out)
{
    if (d < 1 || !x || !g || !m || !out || norm < 0 || norm > 2)
        return ORACLE_EINVAL;
    double *mt = (double *)malloc((size_t)d * sizeof(double));
    if (!mt)
        return ORACLE_ENOMEM;

    double lam = wd ? weight_decay : 0.0;
    double sum_xx = 0.0, sum_mm = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        double gj = grad_scale * gradient_at(g, g_is_bf16, j);
        double xj = (double)x[j];
        mt[j] = beta1 * (double)m[j] + (1.0 - beta1) * (gj + lam * xj);
        sum_xx = norm_add(norm, sum_xx, xj);
        sum_mm = norm_add(norm, sum_mm, mt[j]);
    }

    double norm_x = norm_finish(norm, sum_xx);
    double norm_m = norm_finish(norm, sum_mm);
    double ratio = (norm_m == 0.0)
                       ? 0.0
                       : trust_coef * phi(norm_x, gamma_l, gamma_u) / norm_m;
    for (int64_t j = 0; j < d; ++j) {
        x[j] = store_f32((double)x[j] - lr * ratio * mt[j]);
        m[j] = store_f32(mt[j]);
    }

    out[0] = ratio;
    out[1] = norm_x;
    out[2] = norm_m;
    free(mt);
    return ORACLE_OK;
}

/*
 * One N-LAMB step (Algorithm 3) or, with nesterov_v, one NN-LAMB step
 * (Algorithm 4) on one layer block of d elements, at step t:
 *
 *   m_t   = beta1 m_{t-1} + (1 - beta1) g_t
 *   m_hat = beta1 m_t / (1 - beta1^(t+1)) + (1 - beta1) g_t / (1 - beta1^t)
 *   v_t   = beta2 v_{t-1} + (1 - beta2) g_t^2
 *   v_hat = beta2 v_t / (1 - beta2^t)                               (N-LAMB)
 *   v_hat = beta2 v_t / (1 - beta2^(t+1))
 *           + (1 - beta2) g_t^2 / (1 - beta2^t)                     (NN-LAMB)
 *   r_t   = m_hat / (sqrt(v_hat) + eps)
 *   u     = r_t + lambda x_t
 *   x_{t+1} = x_t - eta_t phi(||x_t||) / ||u|| * u
 *
 * Arguments and outputs as oracle_lamb_layer (bias correction is part of
 * these algorithms and always on).
 */
int oracle_nlamb_layer(int64_t d, float *x, const void *g, int g_is_bf16,
                       float *m, float *v,
                       double lr, double beta1, double beta2, double eps,
                       double weight_decay, int wd, double gamma_l,
                       double gamma_u, int64_t t, int nesterov_v,
                       double grad_scale, int norm, double *out)
{
    if (d < 1 || !x || !g || !m || !v || !out || t < 1 || norm < 0 || norm > 2)
        return ORACLE_EINVAL;
    double *u = (double *)malloc((size_t)d * sizeof(double));
    if (!u)
        return ORACLE_ENOMEM;

    double b1_t = pow(beta1, (double)t);
    double b1_next = pow(beta1, (double)(t + 1));
    double b2_t = pow(beta2, (double)t);
    double b2_next = pow(beta2, (double)(t + 1));
    double lam = wd ? weight_decay : 0.0;

    double sum_xx = 0.0, sum_uu = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        double gj = grad_scale * gradient_at(g, g_is_bf16, j);
        double xj = (double)x[j];
        double mj = beta1 * (double)m[j] + (1.0 - beta1) * gj;
        double m_hat = beta1 * mj / (1.0 - b1_next) + (1.0 - beta1) * gj / (1.0 - b1_t);
        double vj = beta2 * (double)v[j] + (1.0 - beta2) * (gj * gj);
        double v_hat;
        if (nesterov_v)
            v_hat = beta2 * vj / (1.0 - b2_next) + (1.0 - beta2) * (gj * gj) / (1.0 - b2_t);
        else
            v_hat = beta2 * vj / (1.0 - b2_t);
        double r = m_hat / (sqrt(v_hat) + eps);
        u[j] = r + lam * xj;
        sum_xx = norm_add(norm, sum_xx, xj);
        sum_uu = norm_add(norm, sum_uu, u[j]);
        m[j] = store_f32(mj);
        v[j] = store_f32(vj);
    }

    double norm_x = norm_finish(norm, sum_xx);
    double norm_u = norm_finish(norm, sum_uu);
    double ratio = (norm_u == 0.0) ? 0.0 : phi(norm_x, gamma_l, gamma_u) / norm_u;
    for (int64_t j = 0; j < d; ++j)
        x[j] = store_f32((double)x[j] - lr * ratio * u[j]);

    out[0] = ratio;
    out[1] = norm_x;
    out[2] = norm_u;
    free(u);
    return ORACLE_OK;
}

/*
 * The bf16 working copy of updated parameters: each fp32 x_j rounded to the
 * nearest bf16, ties to even; every NaN becomes the quiet NaN 0x7fc0.
 */
void oracle_round_bf16(int64_t d, const float *x, uint16_t *out)
{
    for (int64_t j = 0; j < d; ++j) {
        if (isnan(x[j])) {
            out[j] = 0x7fc0;
            continue;
        }
        uint32_t bits;
        memcpy(&bits, &x[j], sizeof bits);
        uint32_t low = bits & 0xffffu;            /* the 16 bits dropped */
        uint32_t high = bits >> 16;
        if (low > 0x8000u || (low == 0x8000u && (high & 1u)))
            high += 1u;                           /* carries into the exponent as needed */
        out[j] = (uint16_t)high;
    }
}
