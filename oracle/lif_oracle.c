/*
 * CPU ORACLE for the temporally fused LIF layer -- TEST INFRASTRUCTURE ONLY.
 * See lif_oracle.h for scope, layout, precision and pins.  Build with
 * -O2 -ffp-contract=off and without fast-math.
 */
#include "lif_oracle.h"

#include <math.h>

/* Forward: Sec. 3.1.
 * Eq. (1), hard reset: v^t = k v^{t-1} (1 - y^{t-1}) + V_rest y^{t-1} + x^t, with
 * v^0 = V_rest.  Written as a select on y^{t-1}; for finite v the two forms give
 * the same floats (k v * 1 and k v * 0 + V_rest), and the select keeps an
 * infinite membrane from turning into inf * 0 = NaN after its spike.
 * Soft reset (no equation in the paper): v^t = k (v^{t-1} - V_th y^{t-1}) + x^t.
 * Eq. (2): y^t = H(v^t - V_th), with H(0) = 1.
 * Before the first step no spike has happened: y^0 = 0. */
void lif_oracle_forward(const lif_oracle_params *p, int64_t T, int64_t N, const float *x,
                        const float *v_init, const uint8_t *y_init, uint8_t *y, float *v)
{
    const float k = p->decay, th = p->v_th, rest = p->v_rest;
    for (int64_t n = 0; n < N; ++n) {
        float vt = v_init ? v_init[n] : rest;
        int yt = y_init ? (y_init[n] != 0) : 0;
        for (int64_t t = 0; t < T; ++t) {
            const float xt = x[t * N + n];
            if (p->soft_reset) {
                float w = yt ? vt - th : vt;
                vt = k * w + xt;
            } else {
                vt = yt ? rest + xt : k * vt + xt;
            }
            yt = (vt - th >= 0.0f) ? 1 : 0;
            v[t * N + n] = vt;
            y[t * N + n] = (uint8_t)yt;
        }
    }
}

/* Sec. 5.2: delta(u) = alpha e^{-alpha u} / (1 + e^{-alpha u})^2, the derivative of
 * sigmoid(alpha u).  It is even in u, so it is evaluated at |u|, which cannot
 * overflow.  Eq. (2) fires on v - V_th, so the surrogate is taken at u = v - V_th. */
static double surrogate(double alpha, double u)
{
    const double e = exp(-alpha * fabs(u));
    return alpha * e / ((1.0 + e) * (1.0 + e));
}

/* Backward: Eq. (3), generalised to any V_rest and to the soft reset.
 * dL/dx^t = dL/dv^t, because dv^t/dx^t = 1 in Eq. (1), and
 *   dL/dv^t = dL/dy^t * delta^t + dL/dv^{t+1} * dv^{t+1}/dv^t,
 * where, with y^t differentiated through the surrogate (the reset is not detached):
 *   hard:  dv^{t+1}/dv^t = k (1 - y^t) + (V_rest - k v^t) delta^t
 *          (= k [1 - y^t - v^t delta^t] at V_rest = 0, Eq. (3) as printed),
 *   soft:  dv^{t+1}/dv^t = k (1 - V_th delta^t).
 * dL/dv^{T+1} = g_next (0 for the last layer of time).
 * The bound gx_mag runs the same recurrence with every term in absolute value (each term
 * of dv^{t+1}/dv^t separately), so it bounds the rounding error of any evaluation of
 * Eq. (3) that rounds each term with a small relative error, even where terms cancel. */
void lif_oracle_backward(const lif_oracle_params *p, int64_t T, int64_t N, const float *v,
                         const uint8_t *y, const double *gy, const double *gy_mag,
                         const double *g_next, double *gx, double *gx_mag)
{
    const double k = p->decay, th = p->v_th, rest = p->v_rest, alpha = p->alpha;
    for (int64_t n = 0; n < N; ++n) {
        double g_after = g_next ? g_next[n] : 0.0;
        double m_after = g_next ? fabs(g_next[n]) : 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int64_t i = t * N + n;
            const double vt = v[i];
            const double d = surrogate(alpha, vt - th);
            double dv_next, dv_next_mag;
            if (p->soft_reset) {
                dv_next = k * (1.0 - th * d);
                dv_next_mag = k * (1.0 + fabs(th) * d);
            } else {
                dv_next = k * (1.0 - (double)y[i]) + (rest - k * vt) * d;
                dv_next_mag = k * (1.0 - (double)y[i]) + fabs(rest - k * vt) * d;
            }
            const double g = gy[i] * d + dv_next * g_after;
            const double m = gy_mag[i] * d + dv_next_mag * m_after;
            gx[i] = g;
            gx_mag[i] = m;
            g_after = g;
            m_after = m;
        }
    }
}

void lif_oracle_gain_forward(int64_t T, int64_t B, int64_t F, const uint8_t *y,
                             const float *gain, float *x_next)
{
    for (int64_t t = 0; t < T; ++t)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t f = 0; f < F; ++f) {
                const int64_t i = (t * B + b) * F + f;
                x_next[i] = gain[f] * (float)y[i];
            }
}

void lif_oracle_gain_backward(int64_t T, int64_t B, int64_t F, const double *gx_next,
                              const double *gx_next_mag, const float *gain, double *gy,
                              double *gy_mag)
{
    for (int64_t t = 0; t < T; ++t)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t f = 0; f < F; ++f) {
                const int64_t i = (t * B + b) * F + f;
                gy[i] = (double)gain[f] * gx_next[i];
                gy_mag[i] = fabs((double)gain[f]) * gx_next_mag[i];
            }
}
