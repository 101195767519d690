/*
 * snn_lif.h -- C ABI of the temporally fused LIF spiking-neuron layer for MI355X (gfx950).
 *
 * What it computes (Li et al., "Towards Scalable GPU-Accelerated SNN Training via
 * Temporal Fusion"):
 *   forward  -- for every neuron, all T time steps of the iterative LIF model in one
 *               kernel (temporal fusion, Sec. 3.2): the membrane update of Sec. 3.1
 *               Eq. (1) (leak, input integration, reset) and the Heaviside spike of
 *               Eq. (2), with H(0) = 1;
 *   backward -- the surrogate-gradient recurrence of Eq. (3), run in reverse time in one
 *               kernel, with the sigmoid surrogate of Sec. 5.2 evaluated at v - V_th.
 *
 * Conventions shared by every entry point:
 *   - Tensors are dense and time-major, [T][N]: row t (the paper's step t+1) starts at
 *     element t*N.  A per-step shape such as [B][C][H][W] is contiguous, so N = B*C*H*W.
 *   - Every data pointer is a DEVICE pointer owned by the caller and 16-byte aligned.
 *   - The library never allocates, never synchronizes, keeps no pointer after it returns
 *     and has no mutable global state: calls are re-entrant and thread-safe.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL = null stream)
 *     and runs asynchronously with respect to the host.
 *   - Arguments are validated before anything is launched.  On error nothing is written
 *     and a negative snn_status is returned; a rejected launch returns SNN_E_LAUNCH.
 *     Faults inside a kernel surface at the caller's next synchronization.
 *   - T == 0 or N == 0 is an empty problem: SNN_OK, nothing is launched and the data
 *     pointers are not used (they may be NULL).
 *   - Limits: 0 <= T <= 2^31 - 1, 0 <= N <= 2^31, T * N <= 2^44 (SNN_E_SHAPE beyond).
 */
#ifndef SNN_LIF_H
#define SNN_LIF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SNN_OK = 0,
    SNN_E_NULL = -1,        /* a required pointer is NULL */
    SNN_E_SHAPE = -2,       /* negative or too large T, N, B, F */
    SNN_E_PARAM = -3,       /* a hyper-parameter or enum value out of range */
    SNN_E_ALIGN = -4,       /* a data pointer is not 16-byte aligned */
    SNN_E_UNSUPPORTED = -5, /* a combination the library does not implement */
    SNN_E_LAUNCH = -6       /* the HIP runtime rejected the kernel launch */
} snn_status;

typedef enum {
    SNN_RESET_HARD = 0, /* Eq. (1): after a spike the membrane restarts at V_rest (+ input) */
    SNN_RESET_SOFT = 1  /* not in the paper: subtract V_th, then leak:
                           v^t = k (v^{t-1} - V_th y^{t-1}) + x^t; backward factor k (1 - V_th delta) */
} snn_reset;

typedef enum {
    SNN_IO_F32 = 0,  /* x, dL/dy and dL/dx are float32 */
    SNN_IO_BF16 = 1  /* bfloat16 bit patterns (uint16); widened exactly, membrane kept in fp32,
                        dL/dx rounded to nearest even when stored */
} snn_io;

typedef enum {
    SNN_SPK_U8 = 0,   /* one byte per neuron (0 or 1): row t at byte t*N */
    SNN_SPK_BITS = 1, /* one bit per neuron: neuron n of row t is bit (n & 7) of byte
                         t*row_bytes + (n >> 3), row_bytes = 8*ceil(N/64) (whole little-endian
                         64-bit words), padding bits are written as 0 */
    SNN_SPK_IO = 2    /* 0.0 / 1.0 in the I/O dtype, [T][N] like x: the layer's output as a
                         tensor a following ANN operator can consume directly */
} snn_spk;

typedef struct {
    float decay;   /* k_tau of Eq. (1), in [0, 1]; the paper relates it to tau as k = 1 - 1/tau */
    float v_th;    /* V_th of Eq. (2), finite */
    float v_reset; /* V_rest of Eq. (1): membrane before step 1 and the hard-reset value, finite */
    float alpha;   /* surrogate sharpness (Sec. 5.2): delta(u) = alpha e^{-alpha u}/(1+e^{-alpha u})^2,
                      > 0 and finite */
    int32_t reset; /* snn_reset */
    int32_t io;    /* snn_io */
    int32_t spk;   /* snn_spk */
} snn_lif_cfg;

/* Bytes of one spike row for N neurons in cfg->spk's format (N, 8*ceil(N/64), or N times
 * the I/O element size).
 * Host-only; SNN_E_NULL / SNN_E_PARAM / SNN_E_SHAPE on bad arguments. */
snn_status snn_spike_row_bytes(const snn_lif_cfg *cfg, int64_t N, size_t *bytes);

/* Bytes of the forward-to-backward state for a [T][N] layer.  The content is opaque
 * (fp32 membrane checkpoints at fixed step intervals; 0 bytes when T is short enough that
 * the backward recomputes the whole trajectory from x).  Host-only. */
snn_status snn_lif_saved_bytes(const snn_lif_cfg *cfg, int64_t T, int64_t N, size_t *bytes);

/* Forward of one LIF layer over all T steps (Eqs. (1), (2); temporal fusion, Sec. 3.2).
 *   x       [T][N] in cfg->io dtype: input current x_i^(t).
 *   spikes  [T][row_bytes] out: y_i^(t) in cfg->spk format.
 *   saved   snn_lif_saved_bytes() bytes out (may be NULL when that size is 0).
 *   v_out   NULLABLE [T][N] float32 out: membrane after input integration, before any
 *           reset (the v_i^(t) of Eq. (1)).  Meant for tests; pass NULL otherwise.
 * x, spikes and saved must not be modified between this call and the matching backward. */
snn_status snn_lif_forward(const snn_lif_cfg *cfg, int64_t T, int64_t N, const void *x,
                           void *spikes, void *saved, float *v_out, void *stream);

/* Backward of the same layer (Eq. (3), reverse time, surrogate of Sec. 5.2).
 *   x, saved  exactly as passed to / written by snn_lif_forward with the same cfg, T, N.
 *   grad_s    [T][N] in cfg->io dtype: dL/dy_i^(t).
 *   grad_x    [T][N] in cfg->io dtype out: dL/dx_i^(t) (= dL/dv_i^(t)).  May be the same
 *             buffer as grad_s (in place); any other overlap is undefined.
 * The membrane trajectory is recomputed from x and the checkpoints, bit-identical to the
 * forward's.  Only grad_x is produced: k_tau, V_th, V_rest get no gradient. */
snn_status snn_lif_backward(const snn_lif_cfg *cfg, int64_t T, int64_t N, const void *x,
                            const void *saved, const void *grad_s, void *grad_x, void *stream);

/* The same layer over one time segment of a longer sequence: the state handoff of the
 * temporal split (Sec. 3.3, Fig. 1(b)), where consecutive segments of one layer run one
 * after the other (on one GPU, or on neighbouring GPUs with the four [N] fp32 vectors
 * below exchanged between them).  Running a sequence as segments T = T_1 + T_2 + ...
 * with the handoff gives the same spikes, membranes and gradients, bit for bit, as one
 * call over all T.  Each of the four pointers may be NULL; all are [N] float32, 16-byte
 * aligned, device memory:
 *   v_in    the membrane the preceding segment ended with (its v_last): v^0 of this
 *           segment, whose spike state is taken as v_in >= V_th (Eq. (2)).  NULL: the
 *           sequence starts here (v^0 = V_rest, no spike).
 *   v_last  out: the membrane after the segment's last step, v^T.
 *   g_in    dL/dv^{T+1}, handed back by the following segment (its g_out).  NULL: 0, the
 *           sequence ends here.
 *   g_out   out: dL/dv^1 of this segment in fp32 (= dL/dx^1 before rounding to cfg->io).
 * forward_seg / backward_seg of one segment must get the same v_in.  With T == 0 nothing
 * is written.  snn_lif_forward / snn_lif_backward are these calls with all four NULL. */
snn_status snn_lif_forward_seg(const snn_lif_cfg *cfg, int64_t T, int64_t N, const void *x,
                               const float *v_in, void *spikes, void *saved, float *v_last,
                               float *v_out, void *stream);
snn_status snn_lif_backward_seg(const snn_lif_cfg *cfg, int64_t T, int64_t N, const void *x,
                                const float *v_in, const void *saved, const void *grad_s,
                                const float *g_in, void *grad_x, float *g_out, void *stream);

/* Stand-in for the ANN operator between stacked LIF layers (not part of the paper's
 * method): a per-feature gain, N = B*F neurons per step, neuron (b, f) at b*F + f.
 *   forward:  x_next[t][b][f] = gain[f] * y[t][b][f]   (spikes in cfg->spk format,
 *             x_next in cfg->io dtype, product in fp32 then rounded to the io dtype; y is
 *             0 or 1, so this is gain[f] rounded to the io dtype, times y);
 *   backward: grad_s[t][b][f] = g[f] * grad_x_next[t][b][f], g[f] = gain[f] rounded to the
 *             io dtype as the forward applies it (io dtype in and out; product in fp32,
 *             rounded once; may be the same buffer).
 * gain is a device float32 [F] array. */
snn_status snn_gain_spikes_forward(const snn_lif_cfg *cfg, int64_t T, int64_t B, int64_t F,
                                   const void *spikes, const float *gain, void *x_next,
                                   void *stream);
snn_status snn_gain_grad_backward(const snn_lif_cfg *cfg, int64_t T, int64_t B, int64_t F,
                                  const void *grad_x_next, const float *gain, void *grad_s,
                                  void *stream);

/* A LIF layer fused with the gain in front of it: the layer whose input current is
 * x[t][b][f] = gain[f] * spikes_in[t][b][f], read directly from the previous layer's spikes
 * instead of from a stored x.  Sec. 5 feeds LIF layers from an ANN operator (Listing 1's
 * nn.Sequential); fusing that operator into the layer goes beyond the paper and is
 * offered for the per-feature gain above only.  Same shapes as the gain functions
 * (N = B*F, neuron (b, f) at b*F + f); everything else as snn_lif_forward / backward.
 *   spikes_in  previous layer's spikes, in THIS cfg's spike format (u8, bits, or 0/1
 *              values of the I/O dtype shaped [T][N] as the autograd path passes them).
 *   gain       device float32 [F].  The input current uses gain[f] rounded to cfg->io,
 *              so the layer's spikes, membranes and checkpoints equal, bit for bit, those
 *              of snn_gain_spikes_forward followed by snn_lif_forward.
 * forward_gain: spikes, saved, v_out as in snn_lif_forward.
 * backward_gain: spikes_in, gain, saved exactly as in the matching forward_gain; grad_s
 *              [T][N] io: dL/dy of this layer; grad_s_in [T][N] io out: dL/d spikes_in =
 *              g[f] * dL/dx with g[f] = gain[f] rounded to cfg->io (the factor the input
 *              current was formed with), formed in fp32 and rounded once to the io dtype
 *              (the unfused pair rounds dL/dx first, so bf16 results may differ there in
 *              the last bit).  grad_s_in may be the same buffer as grad_s; no other overlap.
 * x is never materialised: per (t, n) the forward reads 1 B (u8) or 1/8 B (bits) of input
 * instead of 4 B or 2 B (with I/O-dtype spikes it saves the glue kernel's write and read of
 * x). */
snn_status snn_lif_forward_gain(const snn_lif_cfg *cfg, int64_t T, int64_t B, int64_t F,
                                const void *spikes_in, const float *gain, void *spikes,
                                void *saved, float *v_out, void *stream);
snn_status snn_lif_backward_gain(const snn_lif_cfg *cfg, int64_t T, int64_t B, int64_t F,
                                 const void *spikes_in, const float *gain, const void *saved,
                                 const void *grad_s, void *grad_s_in, void *stream);

/* A stack of L = 2 or 3 LIF layers joined by per-feature gains, fused across the layers as
 * well as across time: layer 0 is fed x, layer l > 0 is fed gain[l-1][f] * y_{l-1} of the
 * same step, and one kernel per direction carries every neuron through all L layers with
 * the L membranes on chip.  The layers are those of snn_gain_spikes_forward +
 * snn_lif_forward applied in turn (same cfg for every layer); fusing across layers goes
 * beyond the paper (Sec. 5 puts an ANN operator between layers) and is offered for this
 * elementwise operator only.  Shapes as the gain functions: N = B*F, neuron (b, f) at b*F + f.
 *   x          [T][N] io dtype: layer 0's input current.
 *   gains      device float32 [L-1][F].  As in snn_lif_forward_gain, a gain multiplies a
 *              spike after rounding to cfg->io, so spikes and membranes equal those of the
 *              layer-by-layer run bit for bit.
 *   spikes     [T][row_bytes] out: the last layer's spikes in cfg->spk format.
 *   hidden_spikes  NULLABLE [L-1][T][row_bytes] out: the other layers' spikes.
 *   saved      snn_lif_stack_saved_bytes() bytes out (every layer's membrane checkpoints;
 *              may be NULL when that size is 0).
 *   v_out      NULLABLE [L][T][N] float32 out: every layer's membranes (tests).
 * backward: x, gains, saved exactly as in the forward; grad_s [T][N] io: dL/dy of the last
 * layer; grad_x [T][N] io out: dL/dx of layer 0 (may be the same buffer as grad_s).  The
 * gradient handed from layer l down to layer l-1, g dL/dx_l with g the gain rounded to
 * cfg->io, stays in fp32 (the layer-by-layer run stores it in the io dtype).  Other L: SNN_E_UNSUPPORTED. */
snn_status snn_lif_stack_saved_bytes(const snn_lif_cfg *cfg, int32_t L, int64_t T, int64_t N,
                                     size_t *bytes);
snn_status snn_lif_stack_forward(const snn_lif_cfg *cfg, int32_t L, int64_t T, int64_t B, int64_t F,
                                 const void *x, const float *gains, void *spikes,
                                 void *hidden_spikes, void *saved, float *v_out, void *stream);
snn_status snn_lif_stack_backward(const snn_lif_cfg *cfg, int32_t L, int64_t T, int64_t B,
                                  int64_t F, const void *x, const float *gains, const void *saved,
                                  const void *grad_s, void *grad_x, void *stream);

/* Serial (per-time-step) baseline of the same layer: the "serial training" method that
 * temporal fusion is compared against (Sec. 3.2, Fig. 3) -- one launch per time step, the
 * membrane round-tripping through memory between steps.  Kept as an ablation baseline.
 * Its arithmetic is the fused kernels' own, so a step-by-step run reproduces the fused
 * forward and backward bit for bit.
 *   forward step t:  x_t [N] (io dtype), v_prev [N] fp32 membrane after step t-1 (NULL for
 *                    the first step: V_rest and no spike) -> v_t [N] fp32 (needed by the
 *                    backward and the next step), spikes_t (one row in cfg->spk format).
 *   backward step t: v_t [N] fp32, grad_s_t [N] io dtype, g_next [N] fp32 = dL/dv of step
 *                    t+1 (NULL at the last step) -> grad_x_t [N] io dtype = dL/dv of step t,
 *                    and the same value in fp32 into g_out [N] when g_out is not NULL (pass
 *                    it as the next call's g_next; for fp32 I/O grad_x_t itself can be).
 * The step pointers are rows of [T][N] tensors, so they need only their element alignment
 * (and 8 bytes for bit-packed spike rows), not the 16 bytes the other entry points require. */
snn_status snn_lif_serial_forward_step(const snn_lif_cfg *cfg, int64_t N, const void *x_t,
                                       const float *v_prev, float *v_t, void *spikes_t,
                                       void *stream);
snn_status snn_lif_serial_backward_step(const snn_lif_cfg *cfg, int64_t N, const float *v_t,
                                        const void *grad_s_t, const float *g_next, void *grad_x_t,
                                        float *g_out, void *stream);

/* Static text for a status code. */
const char *snn_status_str(snn_status status);

#ifdef __cplusplus
}
#endif

#endif /* SNN_LIF_H */
