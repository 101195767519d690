/* A plain-C client of libsnnlif: device memory from hipMalloc, a stream from
 * hipStreamCreate, and nothing but the C ABI of include/snn_lif.h -- no Python, no torch.
 * It runs the fused forward and backward of several layers (fp32 and bf16 I/O, u8 and bit
 * spikes, hard and soft reset, one and several chunks, ragged N) and compares them with
 * the CPU oracle (test infrastructure) on the same seeded inputs: spikes exactly (a
 * mismatch is forgiven only strictly within 1e-5 of V_th, and that neuron is then left
 * out), membranes bit for bit, dL/dx within the oracle's error budget: |gpu - ref| <=
 * q |ref| + (1 + q) 1e-5 err, q = 2^-8 for bf16 storage and 0 for fp32.  It does the same
 * for the stack fused across depth against the oracle's stack, checks that a sequence run
 * as segments with the state handoff equals the single call bit for bit, and checks
 * argument errors.  Exit status 0 when everything matches. */
#include <hip/hip_runtime_api.h>

#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "lif_oracle.h"
#include "snn_lif.h"

/* the seeded input generator (synth/gen.c) */
void synth_fill_f32(uint64_t seed, uint64_t stream, int kind, double a, double b, int64_t start, int64_t count,
                    float *out);
void synth_f32_to_bf16(const float *in, uint16_t *out, int64_t count);

#define HIP_OK(call)                                                              \
    do {                                                                          \
        hipError_t e_ = (call);                                                   \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));     \
            exit(3);                                                              \
        }                                                                         \
    } while (0)

typedef struct {
    int64_t T, N;
    int32_t reset, io, spk;
    float decay, v_th, v_reset, alpha;
    uint64_t seed;
} layer_case;

static float widen_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static void *dev_alloc(size_t bytes)
{
    void *p = NULL;
    if (bytes) HIP_OK(hipMalloc(&p, bytes));
    return p;
}

static int run_case(const layer_case *c, hipStream_t stream)
{
    const int64_t T = c->T, N = c->N, TN = T * N;
    const int bf16 = c->io == SNN_IO_BF16;
    const size_t esz = bf16 ? 2 : 4;
    snn_lif_cfg cfg = {c->decay, c->v_th, c->v_reset, c->alpha, c->reset, c->io, c->spk};

    /* inputs: x ~ N(0.5, 0.5), dL/dy ~ N(0, 1); bf16 I/O rounds them, the oracle gets the
     * exact widened values */
    float *x = malloc(TN * 4), *gs = malloc(TN * 4);
    uint16_t *x16 = malloc(TN * 2), *gs16 = malloc(TN * 2);
    synth_fill_f32(c->seed, 0, 0, 0.5, 0.5, 0, TN, x);
    synth_fill_f32(c->seed, 1, 0, 0.0, 1.0, 0, TN, gs);
    if (bf16) {
        synth_f32_to_bf16(x, x16, TN);
        synth_f32_to_bf16(gs, gs16, TN);
        for (int64_t i = 0; i < TN; ++i) {
            x[i] = widen_bf16(x16[i]);
            gs[i] = widen_bf16(gs16[i]);
        }
    }

    size_t row = 0, saved_bytes = 0;
    if (snn_spike_row_bytes(&cfg, N, &row) != SNN_OK || snn_lif_saved_bytes(&cfg, T, N, &saved_bytes) != SNN_OK) {
        fprintf(stderr, "size queries failed\n");
        return 1;
    }
    void *dx = dev_alloc(TN * esz), *dgs = dev_alloc(TN * esz), *dgx = dev_alloc(TN * esz);
    void *dspk = dev_alloc(T * row), *dsaved = dev_alloc(saved_bytes);
    float *dv = dev_alloc(TN * 4);
    HIP_OK(hipMemcpy(dx, bf16 ? (void *)x16 : (void *)x, TN * esz, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dgs, bf16 ? (void *)gs16 : (void *)gs, TN * esz, hipMemcpyHostToDevice));

    snn_status st = snn_lif_forward(&cfg, T, N, dx, dspk, dsaved, dv, stream);
    if (st == SNN_OK) st = snn_lif_backward(&cfg, T, N, dx, dsaved, dgs, dgx, stream);
    if (st != SNN_OK) {
        fprintf(stderr, "library call failed: %s\n", snn_status_str(st));
        return 1;
    }
    HIP_OK(hipStreamSynchronize(stream));

    uint8_t *spk = malloc(T * row);
    float *v = malloc(TN * 4), *gx = malloc(TN * 4);
    uint16_t *gx16 = malloc(TN * 2);
    HIP_OK(hipMemcpy(spk, dspk, T * row, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(v, dv, TN * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(bf16 ? (void *)gx16 : (void *)gx, dgx, TN * esz, hipMemcpyDeviceToHost));
    if (bf16)
        for (int64_t i = 0; i < TN; ++i) gx[i] = widen_bf16(gx16[i]);

    /* the oracle on the same inputs */
    lif_oracle_params p = {c->decay, c->v_th, c->v_reset, c->alpha, c->reset == SNN_RESET_SOFT};
    uint8_t *y_ref = malloc(TN);
    float *v_ref = malloc(TN * 4);
    double *gsd = malloc(TN * 8), *g_ref = malloc(TN * 8), *err = malloc(TN * 8);
    for (int64_t i = 0; i < TN; ++i) gsd[i] = gs[i];
    lif_oracle_forward(&p, T, N, x, NULL, NULL, y_ref, v_ref);
    lif_oracle_backward(&p, T, N, v_ref, y_ref, gsd, NULL, NULL, NULL, g_ref, err, NULL);

    const double q = bf16 ? 1.0 / 256.0 : 0.0;
    int64_t hard = 0, forgiven = 0, v_bad = 0, g_bad = 0, ties = 0;
    uint8_t *excluded = calloc(N, 1);
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t n = 0; n < N; ++n) {
            if (excluded[n]) continue;
            const int64_t i = t * N + n;
            const int y = c->spk == SNN_SPK_U8 ? spk[t * row + n] : (spk[t * row + (n >> 3)] >> (n & 7)) & 1;
            const double dist = fabs((double)v_ref[i] - (double)c->v_th);
            ties += v_ref[i] == c->v_th;
            if (y != y_ref[i]) {
                if (dist > 0 && dist < 1e-5) {
                    ++forgiven;
                    excluded[n] = 1;
                    continue;
                }
                ++hard;
            }
            if (memcmp(&v[i], &v_ref[i], 4) != 0) ++v_bad;
        }
    }
    for (int64_t i = 0; i < TN; ++i) {
        if (excluded[i % N]) continue;
        const double tol = q * fabs(g_ref[i]) + (1.0 + q) * 1e-5 * err[i] + 1e-30;
        if (!(fabs((double)gx[i] - g_ref[i]) <= tol)) ++g_bad;
    }
    printf("T=%lld N=%lld %s %s %s: ties=%lld forgiven=%lld hard=%lld v_unequal=%lld grad_bad=%lld\n",
           (long long)T, (long long)N, c->reset == SNN_RESET_SOFT ? "soft" : "hard", bf16 ? "bf16" : "f32",
           c->spk == SNN_SPK_U8 ? "u8" : "bits", (long long)ties, (long long)forgiven, (long long)hard,
           (long long)v_bad, (long long)g_bad);

    HIP_OK(hipFree(dx));
    HIP_OK(hipFree(dgs));
    HIP_OK(hipFree(dgx));
    HIP_OK(hipFree(dspk));
    if (dsaved) HIP_OK(hipFree(dsaved));
    HIP_OK(hipFree(dv));
    free(x), free(gs), free(x16), free(gs16), free(spk), free(v), free(gx), free(gx16);
    free(y_ref), free(v_ref), free(gsd), free(g_ref), free(err), free(excluded);
    return (hard || v_bad || g_bad) ? 1 : 0;
}

/* Spike (t, n) of a [T][row] buffer in format spk. */
static int spike_at(const uint8_t *s, int spk, int64_t row, int64_t t, int64_t n)
{
    return spk == SNN_SPK_U8 ? s[t * row + n] : (s[t * row + (n >> 3)] >> (n & 7)) & 1;
}

/* A stack of L layers joined by per-feature gains, fused across depth (one kernel per
 * direction), against the oracle's layer-by-layer stack: every layer's spikes and
 * membranes, and dL/dx of layer 0 within the oracle's error budget.  The gains are rounded
 * to the I/O dtype on the oracle's side, as the kernels apply them. */
static int run_stack_case(int32_t L, int64_t T, int64_t B, int64_t F, int32_t reset, int32_t io, int32_t spk,
                          uint64_t seed, hipStream_t stream)
{
    const int64_t N = B * F, TN = T * N;
    const int bf16 = io == SNN_IO_BF16;
    const size_t esz = bf16 ? 2 : 4;
    snn_lif_cfg cfg = {0.5f, 1.0f, 0.0f, 4.0f, reset, io, spk};
    float *x = malloc(TN * 4), *gs = malloc(TN * 4), *gains = malloc((L - 1) * F * 4);
    uint16_t *x16 = malloc(TN * 2), *gs16 = malloc(TN * 2), *g16 = malloc((L - 1) * F * 2);
    synth_fill_f32(seed, 0, 0, 0.4, 0.6, 0, TN, x);
    synth_fill_f32(seed, 1, 0, 0.0, 1.0, 0, TN, gs);
    for (int32_t l = 0; l + 1 < L; ++l) synth_fill_f32(seed, 3 + l, 1, 0.5, 2.0, 0, F, gains + l * F);
    float *gains_io = malloc((L - 1) * F * 4);   /* as the kernels apply them */
    memcpy(gains_io, gains, (L - 1) * F * 4);
    if (bf16) {
        synth_f32_to_bf16(x, x16, TN);
        synth_f32_to_bf16(gs, gs16, TN);
        synth_f32_to_bf16(gains, g16, (L - 1) * F);
        for (int64_t i = 0; i < TN; ++i) {
            x[i] = widen_bf16(x16[i]);
            gs[i] = widen_bf16(gs16[i]);
        }
        for (int64_t i = 0; i < (L - 1) * F; ++i) gains_io[i] = widen_bf16(g16[i]);
    }
    size_t row = 0, saved_bytes = 0;
    if (snn_spike_row_bytes(&cfg, N, &row) != SNN_OK ||
        snn_lif_stack_saved_bytes(&cfg, L, T, N, &saved_bytes) != SNN_OK) {
        fprintf(stderr, "stack size queries failed\n");
        return 1;
    }
    void *dx = dev_alloc(TN * esz), *dgs = dev_alloc(TN * esz), *dgx = dev_alloc(TN * esz);
    void *dspk = dev_alloc(T * row), *dhid = dev_alloc((L - 1) * T * row), *dsaved = dev_alloc(saved_bytes);
    float *dv = dev_alloc(L * TN * 4), *dgains = dev_alloc((L - 1) * F * 4);
    HIP_OK(hipMemcpy(dx, bf16 ? (void *)x16 : (void *)x, TN * esz, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dgs, bf16 ? (void *)gs16 : (void *)gs, TN * esz, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dgains, gains, (L - 1) * F * 4, hipMemcpyHostToDevice));
    snn_status st = snn_lif_stack_forward(&cfg, L, T, B, F, dx, dgains, dspk, dhid, dsaved, dv, stream);
    if (st == SNN_OK) st = snn_lif_stack_backward(&cfg, L, T, B, F, dx, dgains, dsaved, dgs, dgx, stream);
    if (st != SNN_OK) {
        fprintf(stderr, "stack call failed: %s\n", snn_status_str(st));
        return 1;
    }
    HIP_OK(hipStreamSynchronize(stream));
    uint8_t *spk_last = malloc(T * row), *hid = malloc((L - 1) * T * row);
    float *v = malloc(L * TN * 4), *gx = malloc(TN * 4);
    uint16_t *gx16 = malloc(TN * 2);
    HIP_OK(hipMemcpy(spk_last, dspk, T * row, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hid, dhid, (L - 1) * T * row, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(v, dv, L * TN * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(bf16 ? (void *)gx16 : (void *)gx, dgx, TN * esz, hipMemcpyDeviceToHost));
    if (bf16)
        for (int64_t i = 0; i < TN; ++i) gx[i] = widen_bf16(gx16[i]);

    lif_oracle_params p = {cfg.decay, cfg.v_th, cfg.v_reset, cfg.alpha, reset == SNN_RESET_SOFT};
    float *xs = malloc(L * TN * 4), *v_ref = malloc(L * TN * 4);
    uint8_t *y_ref = malloc(L * TN);
    double *gsd = malloc(TN * 8), *g_ref = malloc(L * TN * 8), *err = malloc(L * TN * 8), *rnd = malloc(L * TN * 8);
    for (int64_t i = 0; i < TN; ++i) gsd[i] = gs[i];
    lif_oracle_stack_forward(&p, L, T, B, F, x, gains_io, xs, y_ref, v_ref);
    if (lif_oracle_stack_backward(&p, L, T, B, F, v_ref, y_ref, gains_io, gsd, 0, g_ref, err, rnd) != 0) {
        fprintf(stderr, "oracle out of memory\n");
        return 1;
    }
    int64_t hard = 0, forgiven = 0, v_bad = 0, g_bad = 0;
    uint8_t *excluded = calloc(N, 1);
    for (int32_t l = 0; l < L; ++l) {
        const uint8_t *s = l == L - 1 ? spk_last : hid + (int64_t)l * T * row;
        for (int64_t t = 0; t < T; ++t)
            for (int64_t n = 0; n < N; ++n) {
                if (excluded[n]) continue;
                const int64_t i = l * TN + t * N + n;
                if (spike_at(s, spk, row, t, n) != y_ref[i]) {
                    const double dist = fabs((double)v_ref[i] - (double)cfg.v_th);
                    if (dist > 0 && dist < 1e-5) {
                        ++forgiven;
                        excluded[n] = 1;
                        continue;
                    }
                    ++hard;
                }
                if (memcmp(&v[i], &v_ref[i], 4) != 0) ++v_bad;
            }
    }
    const double q = bf16 ? 1.0 / 256.0 : 0.0;
    for (int64_t i = 0; i < TN; ++i) {
        if (excluded[i % N]) continue;
        const double tol = q * fabs(g_ref[i]) + (1.0 + q) * (1e-5 * err[i] + rnd[i] / 256.0) + 1e-30;
        if (!(fabs((double)gx[i] - g_ref[i]) <= tol)) ++g_bad;
    }
    printf("stack L=%d T=%lld B=%lld F=%lld %s %s %s: forgiven=%lld hard=%lld v_unequal=%lld grad_bad=%lld\n", L,
           (long long)T, (long long)B, (long long)F, reset == SNN_RESET_SOFT ? "soft" : "hard", bf16 ? "bf16" : "f32",
           spk == SNN_SPK_U8 ? "u8" : "bits", (long long)forgiven, (long long)hard, (long long)v_bad, (long long)g_bad);
    HIP_OK(hipFree(dx));
    HIP_OK(hipFree(dgs));
    HIP_OK(hipFree(dgx));
    HIP_OK(hipFree(dspk));
    HIP_OK(hipFree(dhid));
    if (dsaved) HIP_OK(hipFree(dsaved));
    HIP_OK(hipFree(dv));
    HIP_OK(hipFree(dgains));
    free(x), free(gs), free(gains), free(gains_io), free(x16), free(gs16), free(g16), free(spk_last), free(hid);
    free(v), free(gx), free(gx16), free(xs), free(v_ref), free(y_ref), free(gsd), free(g_ref), free(err), free(rnd);
    free(excluded);
    return (hard || v_bad || g_bad) ? 1 : 0;
}

/* A sequence split into segments (snn_lif_forward_seg / snn_lif_backward_seg, the state
 * handoff of the temporal split) against the single call over all T: spikes and dL/dx bit
 * for bit, and the last segment's v_last equal to the single call's last membrane. */
static int run_segment_case(int64_t T, int64_t N, const int64_t *lens, int nseg, int32_t io, hipStream_t stream)
{
    const int64_t TN = T * N;
    const int bf16 = io == SNN_IO_BF16;
    const size_t esz = bf16 ? 2 : 4;
    snn_lif_cfg cfg = {0.75f, 1.0f, 0.0f, 4.0f, SNN_RESET_SOFT, io, SNN_SPK_BITS};
    float *x = malloc(TN * 4), *gs = malloc(TN * 4);
    uint16_t *x16 = malloc(TN * 2), *gs16 = malloc(TN * 2);
    synth_fill_f32(77, 0, 0, 0.5, 0.5, 0, TN, x);
    synth_fill_f32(77, 1, 0, 0.0, 1.0, 0, TN, gs);
    synth_f32_to_bf16(x, x16, TN);
    synth_f32_to_bf16(gs, gs16, TN);
    size_t row = 0, saved_bytes = 0;
    if (snn_spike_row_bytes(&cfg, N, &row) != SNN_OK || snn_lif_saved_bytes(&cfg, T, N, &saved_bytes) != SNN_OK)
        return 1;
    char *dx = dev_alloc(TN * esz), *dgs = dev_alloc(TN * esz), *dgx = dev_alloc(TN * esz), *dgx2 = dev_alloc(TN * esz);
    char *dspk = dev_alloc(T * row), *dspk2 = dev_alloc(T * row), *dsaved = dev_alloc(saved_bytes);
    float *dv = dev_alloc(TN * 4), *dstate = dev_alloc((nseg + 1) * N * 4), *dg = dev_alloc(2 * N * 4);
    HIP_OK(hipMemcpy(dx, bf16 ? (void *)x16 : (void *)x, TN * esz, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dgs, bf16 ? (void *)gs16 : (void *)gs, TN * esz, hipMemcpyHostToDevice));
    snn_status st = snn_lif_forward(&cfg, T, N, dx, dspk, dsaved, dv, stream);
    if (st == SNN_OK) st = snn_lif_backward(&cfg, T, N, dx, dsaved, dgs, dgx, stream);
    /* segment s covers steps [t0, t0 + lens[s]); its saved state is its own */
    int64_t t0s[16];
    for (int s = 0, t0 = 0; s < nseg; t0 += lens[s], ++s) t0s[s] = t0;
    void *seg_saved[16] = {0};
    for (int s = 0; s < nseg && st == SNN_OK; ++s) {
        size_t b = 0;
        st = snn_lif_saved_bytes(&cfg, lens[s], N, &b);
        seg_saved[s] = dev_alloc(b);
        const float *v_in = s ? dstate + (int64_t)(s - 1) * N : NULL;
        if (st == SNN_OK)
            st = snn_lif_forward_seg(&cfg, lens[s], N, dx + t0s[s] * N * esz, v_in, dspk2 + t0s[s] * row, seg_saved[s],
                                     dstate + (int64_t)s * N, NULL, stream);
    }
    for (int s = nseg - 1, i = 0; s >= 0 && st == SNN_OK; --s, ++i) {
        const float *v_in = s ? dstate + (int64_t)(s - 1) * N : NULL;
        const float *g_in = i ? dg + (int64_t)(i % 2) * N : NULL;
        st = snn_lif_backward_seg(&cfg, lens[s], N, dx + t0s[s] * N * esz, v_in, seg_saved[s], dgs + t0s[s] * N * esz,
                                  g_in, dgx2 + t0s[s] * N * esz, dg + (int64_t)((i + 1) % 2) * N, stream);
    }
    if (st != SNN_OK) {
        fprintf(stderr, "segment call failed: %s\n", snn_status_str(st));
        return 1;
    }
    HIP_OK(hipStreamSynchronize(stream));
    uint8_t *a = malloc(T * row), *b = malloc(T * row);
    char *ga = malloc(TN * esz), *gb = malloc(TN * esz);
    float *v_last = malloc(N * 4), *v = malloc(TN * 4);
    HIP_OK(hipMemcpy(a, dspk, T * row, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(b, dspk2, T * row, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(ga, dgx, TN * esz, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gb, dgx2, TN * esz, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(v_last, dstate + (int64_t)(nseg - 1) * N, N * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(v, dv, TN * 4, hipMemcpyDeviceToHost));
    const int fail = memcmp(a, b, T * row) != 0 || memcmp(ga, gb, TN * esz) != 0 ||
                     memcmp(v_last, v + (T - 1) * N, N * 4) != 0;
    printf("segments T=%lld N=%lld %s in %d parts: %s\n", (long long)T, (long long)N, bf16 ? "bf16" : "f32", nseg,
           fail ? "DIFFER from the single call" : "equal to the single call bit for bit");
    HIP_OK(hipFree(dx));
    HIP_OK(hipFree(dgs));
    HIP_OK(hipFree(dgx));
    HIP_OK(hipFree(dgx2));
    HIP_OK(hipFree(dspk));
    HIP_OK(hipFree(dspk2));
    if (dsaved) HIP_OK(hipFree(dsaved));
    HIP_OK(hipFree(dv));
    HIP_OK(hipFree(dstate));
    HIP_OK(hipFree(dg));
    for (int s = 0; s < nseg; ++s)
        if (seg_saved[s]) HIP_OK(hipFree(seg_saved[s]));
    free(x), free(gs), free(x16), free(gs16), free(a), free(b), free(ga), free(gb), free(v_last), free(v);
    return fail;
}

/* argument errors come back as status codes, before anything is launched */
static int check_errors(hipStream_t stream)
{
    snn_lif_cfg cfg = {0.5f, 1.0f, 0.0f, 4.0f, SNN_RESET_HARD, SNN_IO_F32, SNN_SPK_U8};
    snn_lif_cfg bad = cfg;
    bad.decay = 2.0f;
    char *buf = dev_alloc(4096);
    int fails = 0;
    fails += snn_lif_forward(NULL, 4, 64, buf, buf, NULL, NULL, stream) != SNN_E_NULL;
    fails += snn_lif_forward(&bad, 4, 64, buf, buf, NULL, NULL, stream) != SNN_E_PARAM;
    fails += snn_lif_forward(&cfg, -1, 64, buf, buf, NULL, NULL, stream) != SNN_E_SHAPE;
    fails += snn_lif_forward(&cfg, 4, 64, buf + 4, buf + 1024, NULL, NULL, stream) != SNN_E_ALIGN;
    fails += snn_lif_backward(&cfg, 4, 64, buf, NULL, NULL, buf, stream) != SNN_E_NULL;
    fails += snn_lif_forward(&cfg, 0, 64, NULL, NULL, NULL, NULL, stream) != SNN_OK;
    fails += snn_status_str(SNN_E_ALIGN) == NULL;
    HIP_OK(hipFree(buf));
    printf("argument errors: %s\n", fails ? "FAILED" : "ok");
    return fails ? 1 : 0;
}

int main(void)
{
    const layer_case cases[] = {
        {40, 5003, SNN_RESET_HARD, SNN_IO_F32, SNN_SPK_U8, 0.5f, 1.0f, 0.0f, 4.0f, 11},
        {33, 65536, SNN_RESET_HARD, SNN_IO_F32, SNN_SPK_BITS, 0.2f, 0.3f, 0.0f, 4.0f, 12},
        {20, 4096, SNN_RESET_SOFT, SNN_IO_BF16, SNN_SPK_BITS, 0.75f, 1.0f, 0.0f, 4.0f, 13},
        {4, 1 << 20, SNN_RESET_HARD, SNN_IO_BF16, SNN_SPK_U8, 0.5f, 1.0f, 0.25f, 2.0f, 14},
        {48, 3 << 18, SNN_RESET_SOFT, SNN_IO_F32, SNN_SPK_U8, 0.75f, 1.0f, 0.0f, 4.0f, 15},
    };
    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    int fails = check_errors(stream);
    for (size_t i = 0; i < sizeof cases / sizeof cases[0]; ++i) fails += run_case(&cases[i], stream);
    fails += run_stack_case(3, 32, 6, 1000, SNN_RESET_HARD, SNN_IO_F32, SNN_SPK_U8, 21, stream);
    fails += run_stack_case(2, 40, 3, 4097, SNN_RESET_SOFT, SNN_IO_BF16, SNN_SPK_BITS, 22, stream);
    /* past 2^20 neurons the stack takes 2 neurons per lane (one below): N = 2^20 + 2 */
    fails += run_stack_case(2, 17, 2, 524289, SNN_RESET_SOFT, SNN_IO_F32, SNN_SPK_U8, 23, stream);
    const int64_t cuts_a[] = {1, 31, 32, 16}, cuts_b[] = {64, 16, 17};
    /* segment starts must stay 16-byte aligned: N = 64 * 1564, whose fp32 rows (400384 B) and
     * bit-spike rows (12512 B) are multiples of 16 bytes */
    fails += run_segment_case(80, 100096, cuts_a, 4, SNN_IO_F32, stream);
    fails += run_segment_case(97, 1 << 20, cuts_b, 3, SNN_IO_BF16, stream);
    HIP_OK(hipStreamDestroy(stream));
    printf("%s\n", fails ? "FAILED" : "all cases match the oracle");
    return fails ? 1 : 0;
}
