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
 * trajectory and also returns a magnitude bound (the same recurrence with every
 * term in absolute value) that scales the comparison tolerance.
 *
 * Pins (tests/test_oracle_pins.py): constant-input spike periods (hard reset,
 * and soft reset at k = 1), the T = 1 Heaviside, the geometric leak below
 * threshold, the memoryless k = 0 case, hand-derived T = 2 examples, the
 * closed-form soft-reset trajectories for k < 1, a finite-difference identity
 * for the whole backward, and brute force in fp64.  No function here is
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

/* Backward (Eq. (3) with the surrogate of Sec. 5.2), in reverse time.
 * v, y: the forward's outputs.  gy[T][N] = dL/dy; gy_mag[T][N] = bound on |gy|'s
 * error-free magnitude (pass |gy| for a leaf).  g_next (nullable, [N]) is
 * dL/dv at step T+1 (0 if NULL).  Writes gx[T][N] = dL/dx and gx_mag[T][N]. */
void lif_oracle_backward(const lif_oracle_params *p, int64_t T, int64_t N, const float *v,
                         const uint8_t *y, const double *gy, const double *gy_mag,
                         const double *g_next, double *gx, double *gx_mag);

/* Per-feature gain between stacked layers: x_next[t][b][f] = gain[f] * y[t][b][f] (fp32). */
void lif_oracle_gain_forward(int64_t T, int64_t B, int64_t F, const uint8_t *y,
                             const float *gain, float *x_next);

/* Its backward: gy[t][b][f] = gain[f] * gx_next[t][b][f] (fp64), and the same for the bound. */
void lif_oracle_gain_backward(int64_t T, int64_t B, int64_t F, const double *gx_next,
                              const double *gx_next_mag, const float *gain, double *gy,
                              double *gy_mag);

#endif
