/*
 * CPU ORACLE for the temporally fused LIF layer -- TEST INFRASTRUCTURE ONLY.
 * See lif_oracle.h for scope, layout, precision and pins.  Build with
 * -O2 -ffp-contract=off and without fast-math.
 */
#include "lif_oracle.h"

#include <math.h>
#include <stdlib.h>

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
 * dL/dv^{T+1} = g_next (0 for the last step of the sequence).
 *
 * Error budgets (for comparing a finite-precision evaluation with this one).  With
 * D^t = dv^{t+1}/dv^t and g^t = dL/dv^t:
 *   err^t = gy_err^t delta^t + |gy^t| delta^t c^t + m^t |g^{t+1}| + |D^t| err^{t+1},
 *   rnd^t = gy_rnd^t delta^t + |D^t| rnd^{t+1},                    err = rnd = 0 after T.
 * c^t = 1 + alpha |v^t - V_th| is the condition number of delta (the relative change of
 * delta per relative change of its argument, plus one), and m^t is D^t with each of its
 * terms in absolute value: k (1 - y^t) + (|V_rest| + |k v^t|) delta^t c^t (hard),
 * k (1 + |V_th| delta^t c^t) (soft).  An evaluation whose every operation errs by at most
 * a relative eps, and whose input gy errs by at most eps gy_err + eps' gy_rnd, then errs by
 * at most (a small multiple of) eps err + eps' rnd: the terms of step t bound that step's
 * own rounding, and an error entering at step t + 1 reaches step t multiplied by exactly
 * D^t.  gy_err and gy_rnd may be NULL (an exact input). */
void lif_oracle_backward(const lif_oracle_params *p, int64_t T, int64_t N, const float *v,
                         const uint8_t *y, const double *gy, const double *gy_err,
                         const double *gy_rnd, const double *g_next, double *gx, double *gx_err,
                         double *gx_rnd)
{
    const double k = p->decay, th = p->v_th, rest = p->v_rest, alpha = p->alpha;
    for (int64_t n = 0; n < N; ++n) {
        double g_after = g_next ? g_next[n] : 0.0;
        double e_after = 0.0, r_after = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int64_t i = t * N + n;
            const double vt = v[i];
            const double d = surrogate(alpha, vt - th);
            /* d alpha |u| -> 0 as |u| -> inf: an infinite membrane adds nothing (not 0 * inf) */
            const double dc = d > 0.0 ? d * (1.0 + alpha * fabs(vt - th)) : 0.0;
            double D, m;
            if (p->soft_reset) {
                D = k * (1.0 - th * d);
                m = k * (1.0 + fabs(th) * dc);
            } else {
                D = k * (1.0 - (double)y[i]) + (rest - k * vt) * d;
                m = k * (1.0 - (double)y[i]) + (fabs(rest) + fabs(k * vt)) * dc;
            }
            const double g = gy[i] * d + D * g_after;
            const double e = (gy_err ? gy_err[i] * d : 0.0) + fabs(gy[i]) * dc + m * fabs(g_after) +
                             fabs(D) * e_after;
            const double r = (gy_rnd ? gy_rnd[i] * d : 0.0) + fabs(D) * r_after;
            gx[i] = g;
            gx_err[i] = e;
            if (gx_rnd)
                gx_rnd[i] = r;
            g_after = g;
            e_after = e;
            r_after = r;
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

/* dL/dy[t][b][f] = gain[f] dL/dx_next[t][b][f]: the transpose of the forward.  An error in
 * dL/dx_next reaches dL/dy multiplied by |gain[f]|, in both budgets. */
void lif_oracle_gain_backward(int64_t T, int64_t B, int64_t F, const double *gx_next,
                              const double *gx_next_err, const double *gx_next_rnd,
                              const float *gain, double *gy, double *gy_err, double *gy_rnd)
{
    for (int64_t t = 0; t < T; ++t)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t f = 0; f < F; ++f) {
                const int64_t i = (t * B + b) * F + f;
                const double a = (double)gain[f];
                gy[i] = a * gx_next[i];
                gy_err[i] = fabs(a) * gx_next_err[i];
                gy_rnd[i] = fabs(a) * gx_next_rnd[i];
            }
}

/* A stack of L layers joined by per-feature gains, the stand-in for the operator between
 * spiking layers of a network: layer 0 is fed x; layer l > 0 is fed
 * x_l[t][b][f] = gain_{l-1}[f] y_{l-1}[t][b][f].  Layers run one after the other over all
 * T steps (the temporal-major order of Sec. 3.2).  xs, y, v are [L][T][N], N = B F;
 * xs[0] is a copy of x. */
void lif_oracle_stack_forward(const lif_oracle_params *p, int L, int64_t T, int64_t B, int64_t F,
                              const float *x, const float *gains, float *xs, uint8_t *y, float *v)
{
    const int64_t TN = T * B * F;
    for (int64_t i = 0; i < TN; ++i)
        xs[i] = x[i];
    for (int l = 0; l < L; ++l) {
        lif_oracle_forward(p, T, B * F, xs + l * TN, NULL, NULL, y + l * TN, v + l * TN);
        if (l + 1 < L)
            lif_oracle_gain_forward(T, B, F, y + l * TN, gains + l * F, xs + (l + 1) * TN);
    }
}

/* Its backward, last layer first: layer L-1 takes dL/dy = gy; layer l < L-1 takes
 * gain_l[f] dL/dx_{l+1}.  gx, gx_err, gx_rnd are [L][T][N] (dL/dx of every layer and its
 * error budgets, as lif_oracle_backward).  rounded_handoff != 0: the gradient handed down
 * from layer to layer is stored in a lower precision, so its own magnitude joins the
 * rounding budget of the layer below.  Returns 0, or -1 if scratch memory is unavailable. */
int lif_oracle_stack_backward(const lif_oracle_params *p, int L, int64_t T, int64_t B, int64_t F,
                              const float *v, const uint8_t *y, const float *gains, const double *gy,
                              int rounded_handoff, double *gx, double *gx_err, double *gx_rnd)
{
    const int64_t N = B * F, TN = T * N;
    double *h = malloc(3 * (size_t)TN * sizeof(double));
    if (!h && TN > 0)
        return -1;
    double *h_g = h, *h_err = h + TN, *h_rnd = h + 2 * TN;
    for (int l = L - 1; l >= 0; --l) {
        const int64_t o = l * TN;
        if (l == L - 1) {
            lif_oracle_backward(p, T, N, v + o, y + o, gy, NULL, NULL, NULL, gx + o, gx_err + o, gx_rnd + o);
        } else {
            lif_oracle_gain_backward(T, B, F, gx + o + TN, gx_err + o + TN, gx_rnd + o + TN, gains + l * F, h_g,
                                     h_err, h_rnd);
            if (rounded_handoff)
                for (int64_t i = 0; i < TN; ++i)
                    h_rnd[i] += fabs(h_g[i]);
            lif_oracle_backward(p, T, N, v + o, y + o, h_g, h_err, h_rnd, NULL, gx + o, gx_err + o, gx_rnd + o);
        }
    }
    free(h);
    return 0;
}
