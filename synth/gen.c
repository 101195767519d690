/*
 * Seeded synthetic inputs for the fused LIF layer: the ONE module shared by the
 * GPU path's tests/benchmark and the CPU oracle. It holds no LIF arithmetic.
 *
 * Every value is a pure function f(seed, stream, index), so any subset of a
 * tensor (a strided neuron sample, one time row) can be regenerated on its own
 * and matches the full tensor bit for bit, whatever the thread count.
 *
 *   bits(i)    = splitmix64 finaliser of (key + (i+1) * golden_gamma)
 *                (Steele, Lea & Flood, "Fast splittable pseudorandom number
 *                generators", OOPSLA 2014), key derived from (seed, stream)
 *   uniform(i) = ((bits(i) >> 11) + 0.5) * 2^-53, strictly inside (0, 1)
 *   normal(i)  = Box-Muller (1958) on the uniform pair (2*floor(i/2), 2*floor(i/2)+1):
 *                r = sqrt(-2 ln u1); even i -> r cos(2 pi u2), odd i -> r sin(2 pi u2)
 *
 * All transforms are computed in double and rounded once to float (RNE);
 * bf16 tensors are rounded from that float by RNE.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define SYNTH_GAMMA 0x9e3779b97f4a7c15ULL

static uint64_t synth_fmix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

static uint64_t synth_key(uint64_t seed, uint64_t stream)
{
    return synth_fmix(synth_fmix(seed + SYNTH_GAMMA) ^ (stream * 0xd1b54a32d192ed03ULL + 0x632be59bd9b4e019ULL));
}

static double synth_u01(uint64_t key, uint64_t i)
{
    uint64_t b = synth_fmix(key + (i + 1) * SYNTH_GAMMA);
    return ((double)(b >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

static double synth_std_normal(uint64_t key, uint64_t i)
{
    const double two_pi = 6.283185307179586476925286766559;
    uint64_t p = i & ~1ULL;
    double u1 = synth_u01(key, p), u2 = synth_u01(key, p + 1);
    double r = sqrt(-2.0 * log(u1));
    return (i & 1ULL) ? r * sin(two_pi * u2) : r * cos(two_pi * u2);
}

/* kind: 0 = normal(a = mean, b = standard deviation), 1 = uniform(a = low, b = high) */
static float synth_value(int kind, uint64_t key, uint64_t i, double a, double b)
{
    if (kind == 0)
        return (float)(a + b * synth_std_normal(key, i));
    return (float)(a + (b - a) * synth_u01(key, i));
}

/* out[j] = value at index start + j, for j in [0, count) */
void synth_fill_f32(uint64_t seed, uint64_t stream, int kind, double a, double b,
                    int64_t start, int64_t count, float *out)
{
    uint64_t key = synth_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < count; ++j)
        out[j] = synth_value(kind, key, (uint64_t)(start + j), a, b);
}

/* out[j] = value at index idx[j] */
void synth_gather_f32(uint64_t seed, uint64_t stream, int kind, double a, double b,
                      const int64_t *idx, int64_t count, float *out)
{
    uint64_t key = synth_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < count; ++j)
        out[j] = synth_value(kind, key, (uint64_t)idx[j], a, b);
}

/* Bernoulli overwrite: out[j] = value where uniform(stream, start + j) < p, else unchanged. */
void synth_bernoulli_set_f32(uint64_t seed, uint64_t stream, double p, float value,
                             int64_t start, int64_t count, float *out)
{
    uint64_t key = synth_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < count; ++j)
        if (synth_u01(key, (uint64_t)(start + j)) < p)
            out[j] = value;
}

void synth_bernoulli_set_gather_f32(uint64_t seed, uint64_t stream, double p, float value,
                                    const int64_t *idx, int64_t count, float *out)
{
    uint64_t key = synth_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < count; ++j)
        if (synth_u01(key, (uint64_t)idx[j]) < p)
            out[j] = value;
}

/* float -> bf16 bit pattern, round to nearest even; NaN stays a quiet NaN. */
void synth_f32_to_bf16(const float *in, uint16_t *out, int64_t count)
{
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < count; ++j) {
        uint32_t u;
        memcpy(&u, &in[j], 4);
        if ((u & 0x7fffffffu) > 0x7f800000u)
            out[j] = (uint16_t)((u >> 16) | 0x0040u);
        else
            out[j] = (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
    }
}

/* Raw 64-bit output for tests of the generator itself. */
uint64_t synth_bits(uint64_t seed, uint64_t stream, uint64_t i)
{
    return synth_fmix(synth_key(seed, stream) + (i + 1) * SYNTH_GAMMA);
}
