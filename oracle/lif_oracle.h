/*
 * CPU ORACLE for the temporally fused LIF layer -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded reference of what the fused LIF forward and
 * backward compute, written from the equations of Li et al., "Towards Scalable
 * GPU-Accelerated SNN Training via Temporal Fusion" (Sec. 3.1, Eqs. (1)-(3);
 * Sec. 5.2, the sigmoid surrogate).  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may call it.  It shares no code, header, table or
 * constant with the HIP library, and the HIP library never calls it.
 *
 * Layout: every tensor is time-major [T][N]; element (t, n) sits at t*N + n,
 * and t = 0..T-1 stands for the paper's time steps 1..T.
 *
 * Precision: the forward runs in fp32 with exactly one rounding per written
 * operation (built with -ffp-contract=off: no fused multiply-add).  It has to:
 * the membrane decides an integer (the spike), and that decision is taken in
 * the GPU kernel's precision.  The backward runs in fp64 on the fp32 membrane
 * trajectory and also returns running error budgets that scale the comparison
 * tolerance (the local rounding terms of each step, carried back through the
 * true factor dv^{t+1}/dv^t).
 *
 * Pins (tests/test_oracle_pins.py): constant-input spike periods (hard reset,
 * and soft reset at k = 1), the T = 1 Heaviside, the geometric leak below
 * threshold, the memoryless k = 0 case, hand-derived T = 2 examples, the
 * closed-form soft-reset trajectories for k < 1, a finite-difference identity
 * for the whole backward and for the stack, brute force in fp64, and the error
 * budgets against adversarially rounded fp32 evaluations.  No function here is
 * "parity unpinned".
 */
#ifndef LIF_ORACLE_H
#define LIF_ORACLE_H

#include <stdint.h>

typedef struct {
    float decay;    /* k_tau of Eq. (1) */
    float v_th;     /* V_th of Eq. (2) */
    float v_rest;   /* V_rest of Eq. (1): the initial membrane and the hard-reset value */
    float alpha;    /* sharpness of the sigmoid surrogate (Sec. 5.2) */
    int soft_reset; /* 0: Eq. (1); 1: subtract V_th on a spike, then leak (not in the paper) */
} lif_oracle_params;

/* Forward over T steps for N independent neurons (Eqs. (1), (2)).
 * x[T][N] input current; y[T][N] spikes (0/1); v[T][N] membrane after input
 * integration, before any reset.  v_init/y_init (nullable, [N]) give the state
 * before the first step; NULL means v = V_rest, y = 0. */
void lif_oracle_forward(const lif_oracle_params *p, int64_t T, int64_t N, const float *x,
                        const float *v_init, const uint8_t *y_init, uint8_t *y, float *v);

/* Backward (Eq. (3) with the surrogate of Sec. 5.2), in reverse time, fp64.
 * v, y: the forward's outputs.  gy[T][N] = dL/dy.  g_next (nullable, [N]) is dL/dv at
 * step T+1 (0 if NULL).  Writes gx[T][N] = dL/dx and two running error budgets:
 * gx_err[T][N] (arithmetic: scaled by the evaluation's per-operation relative error) and,
 * if gx_rnd is not NULL, gx_rnd[T][N] (scaled by the unit roundoff of a lower-precision
 * copy that fed gy).  gy_err / gy_rnd (nullable) are the same budgets of gy itself, for a
 * gy computed by an earlier layer; NULL means gy is exact.  gx_err >= |gx| everywhere. */
void lif_oracle_backward(const lif_oracle_params *p, int64_t T, int64_t N, const float *v,
                         const uint8_t *y, const double *gy, const double *gy_err,
                         const double *gy_rnd, const double *g_next, double *gx, double *gx_err,
                         double *gx_rnd);

/* Per-feature gain between stacked layers: x_next[t][b][f] = gain[f] * y[t][b][f] (fp32). */
void lif_oracle_gain_forward(int64_t T, int64_t B, int64_t F, const uint8_t *y,
                             const float *gain, float *x_next);

/* Its backward: gy[t][b][f] = gain[f] * gx_next[t][b][f] (fp64); the error budgets of
 * gx_next scale by |gain[f]|. */
void lif_oracle_gain_backward(int64_t T, int64_t B, int64_t F, const double *gx_next,
                              const double *gx_next_err, const double *gx_next_rnd,
                              const float *gain, double *gy, double *gy_err, double *gy_rnd);

/* L layers joined by the gain: layer 0 fed x[T][N], layer l > 0 fed gains[l-1][f] * y_{l-1}
 * (N = B F).  xs (input currents, xs[0] = x), y, v: [L][T][N]. */
void lif_oracle_stack_forward(const lif_oracle_params *p, int L, int64_t T, int64_t B, int64_t F,
                              const float *x, const float *gains, float *xs, uint8_t *y, float *v);

/* Backward through the stack from the last layer's dL/dy gy[T][N]: gx, gx_err, gx_rnd are
 * [L][T][N], dL/dx of every layer with its error budgets.  rounded_handoff != 0: the
 * gradient passed from layer l+1 to layer l is stored in a lower precision (its magnitude
 * joins gx_rnd below).  Returns 0, or -1 when out of memory. */
int lif_oracle_stack_backward(const lif_oracle_params *p, int L, int64_t T, int64_t B, int64_t F,
                              const float *v, const uint8_t *y, const float *gains, const double *gy,
                              int rounded_handoff, double *gx, double *gx_err, double *gx_rnd);

#endif
