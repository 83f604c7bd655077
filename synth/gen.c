/*
 * Seeded, counter-based synthetic input generator.
 *
 * This file holds no arithmetic of the hook step: it only draws the
 * activations, parameters, subscriptions and request layouts that both the
 * CPU oracle and the GPU path consume.  Every element is a pure function of
 * (stream key, element index), so any element can be regenerated alone and
 * the output does not depend on the thread count.
 *
 * Random bits: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  Output i of a stream with
 * seed `key` is mix(key + (i + 1) * 0x9E3779B97F4A7C15).
 * Normals: the Box-Muller transform (Box and Muller, 1958), cosine branch
 * only, fed by outputs 2i and 2i+1 of the stream.
 * bf16: round-to-nearest-even of the double value, done directly from double
 * (no detour through float, which would round twice).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t sm_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static inline uint64_t sm_at(uint64_t key, uint64_t i) {
    return sm_mix(key + (i + 1ull) * 0x9E3779B97F4A7C15ull);
}

/* Uniform double in the open interval (0, 1). */
static inline double u01_open(uint64_t x) {
    return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

static inline double normal_at(uint64_t key, uint64_t i) {
    double u1 = u01_open(sm_at(key, 2 * i));
    double u2 = u01_open(sm_at(key, 2 * i + 1));
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925 * u2);
}

/* Round a double to the nearest bf16 (ties to even) and return its bits. */
static uint16_t gen_bf16_rne(double x) {
    if (isnan(x)) return 0x7FC0;
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    double a = fabs(x);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);               /* a = f * 2^e, f in [0.5, 1) */
    int q = e - 8;              /* quantum exponent for 8 significant bits */
    if (q < -133) q = -133;     /* bf16 subnormal quantum is 2^-133 */
    double r = nearbyint(ldexp(a, -q));   /* exact scaling, RNE */
    double v = ldexp(r, q);
    if (v >= 0x1p128) return sign | 0x7F80;
    float f = (float)v;         /* exact: v has <= 8 significant bits */
    uint32_t b;
    memcpy(&b, &f, 4);
    return (uint16_t)(b >> 16) | sign;
}

/* out[i] = bf16(mean + std * (scale_of_channel) * N(0,1)) for i < n.
 * If `chan_scale` is non-null it holds `row_len` per-channel multipliers
 * applied to element i via channel i % row_len. */
void synth_normal_bf16(uint64_t key, int64_t n, double mean, double std,
                       const double *chan_scale, int64_t row_len, uint16_t *out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double s = std;
        if (chan_scale) s *= chan_scale[i % row_len];
        out[i] = gen_bf16_rne(mean + s * normal_at(key, (uint64_t)i));
    }
}

void synth_normal_f32(uint64_t key, int64_t n, double mean, double std,
                      const double *chan_scale, int64_t row_len, float *out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double s = std;
        if (chan_scale) s *= chan_scale[i % row_len];
        out[i] = (float)(mean + s * normal_at(key, (uint64_t)i));
    }
}

void synth_uniform_f32(uint64_t key, int64_t n, double lo, double hi, float *out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)(lo + (hi - lo) * u01_open(sm_at(key, (uint64_t)i)));
}

/* Uniform doubles in (0,1), used for Bernoulli draws and choices. */
void synth_uniform_f64(uint64_t key, int64_t n, double *out) {
    for (int64_t i = 0; i < n; ++i) out[i] = u01_open(sm_at(key, (uint64_t)i));
}

/* Raw 64-bit draws. */
void synth_bits(uint64_t key, int64_t n, uint64_t *out) {
    for (int64_t i = 0; i < n; ++i) out[i] = sm_at(key, (uint64_t)i);
}

/* Rows of a [rows, cols] bf16 matrix scaled to unit L2 norm (norm taken in
 * double over the bf16 values), then rounded to bf16.  Used to materialise a
 * decoder dictionary from an encoder dictionary. */
void synth_rownorm_bf16(const uint16_t *in, int64_t rows, int64_t cols, uint16_t *out) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const uint16_t *src = in + r * cols;
        double ss = 0.0;
        for (int64_t c = 0; c < cols; ++c) {
            uint32_t b = (uint32_t)src[c] << 16;
            float f;
            memcpy(&f, &b, 4);
            ss += (double)f * (double)f;
        }
        double nrm = sqrt(ss);
        for (int64_t c = 0; c < cols; ++c) {
            uint32_t b = (uint32_t)src[c] << 16;
            float f;
            memcpy(&f, &b, 4);
            out[r * cols + c] = gen_bf16_rne(nrm > 0.0 ? (double)f / nrm : 0.0);
        }
    }
}

uint16_t synth_bf16_from_double(double x) { return gen_bf16_rne(x); }
