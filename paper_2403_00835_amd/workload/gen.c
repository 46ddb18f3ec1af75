/*
 * Seeded synthetic inputs: model weights, prompt token ids, prompt lengths.
 *
 * This module only draws random numbers. It holds none of the decoding
 * method's arithmetic and is linked by neither the GPU library nor the CPU
 * oracle: Python code calls it to fill arrays, then hands the same arrays to
 * both sides.
 *
 * Generator (counter based, so every element can be drawn independently and
 * in parallel):
 *   mix(x)   = the SplitMix64 output function applied to the state x
 *              (Steele, Lea and Flood, "Fast splittable pseudorandom number
 *              generators", OOPSLA 2014): add the golden gamma, then two
 *              xor-shift-multiply rounds and a final xor-shift.
 *   key(seed, stream) = mix(mix(seed) ^ stream)
 *   bits(seed, stream, i) = mix(key(seed, stream) ^ i)
 *
 * Normal deviates use the Box-Muller transform in double precision on the
 * pair j = i / 2: u1 = (top 53 bits of bits(.., 2j) + 1) * 2^-53 in (0, 1],
 * u2 = (top 53 bits of bits(.., 2j + 1)) * 2^-53 in [0, 1);
 * r = sqrt(-2 ln u1); element 2j takes r cos(2 pi u2), element 2j+1 takes
 * r sin(2 pi u2). The deviate is scaled by std, rounded to fp32 (nearest
 * even) and, for bf16 outputs, rounded again to bf16 (nearest even).
 *
 * Uniform ids in [0, V): the top 32 bits times V, shifted right by 32.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <stddef.h>

static inline uint64_t wl_mix(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t wl_bits(uint64_t seed, uint64_t stream, uint64_t index) {
    uint64_t key = wl_mix(wl_mix(seed) ^ stream);
    return wl_mix(key ^ index);
}

static inline uint16_t wl_f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u) { /* inf or nan: keep, quiet nan */
        uint16_t h = (uint16_t)(u >> 16);
        if (u & 0x007FFFFFu) h |= 0x0040u;
        return h;
    }
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

static inline double wl_normal(uint64_t key, uint64_t i) {
    uint64_t j = i >> 1;
    uint64_t b1 = wl_mix(key ^ (2 * j));
    uint64_t b2 = wl_mix(key ^ (2 * j + 1));
    double u1 = ((double)(b1 >> 11) + 1.0) * 0x1.0p-53;
    double u2 = (double)(b2 >> 11) * 0x1.0p-53;
    double r = sqrt(-2.0 * log(u1));
    double a = 6.283185307179586476925286766559 * u2;
    return (i & 1) ? r * sin(a) : r * cos(a);
}

/* out[i] = fp32(std * N_i) for i in [0, n). */
void wl_fill_normal_f32(uint64_t seed, uint64_t stream, double std, float *out, int64_t n) {
    uint64_t key = wl_mix(wl_mix(seed) ^ stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)(std * wl_normal(key, (uint64_t)i));
}

/* out[i] = bf16 bits of bf16(fp32(std * N_i)). */
void wl_fill_normal_bf16(uint64_t seed, uint64_t stream, double std, uint16_t *out, int64_t n) {
    uint64_t key = wl_mix(wl_mix(seed) ^ stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = wl_f32_to_bf16_rne((float)(std * wl_normal(key, (uint64_t)i)));
}

/* out[i] = uniform id in [0, vocab). */
void wl_fill_uniform_ids(uint64_t seed, uint64_t stream, int32_t vocab, int32_t *out, int64_t n) {
    uint64_t key = wl_mix(wl_mix(seed) ^ stream);
    for (int64_t i = 0; i < n; ++i) {
        uint64_t b = wl_mix(key ^ (uint64_t)i);
        out[i] = (int32_t)(((b >> 32) * (uint64_t)(uint32_t)vocab) >> 32);
    }
}

/* out[i] = lo + uniform integer in [0, hi - lo]. */
void wl_fill_uniform_range(uint64_t seed, uint64_t stream, int32_t lo, int32_t hi, int32_t *out, int64_t n) {
    uint64_t key = wl_mix(wl_mix(seed) ^ stream);
    uint64_t span = (uint64_t)(int64_t)(hi - lo) + 1u;
    for (int64_t i = 0; i < n; ++i) {
        uint64_t b = wl_mix(key ^ (uint64_t)i);
        out[i] = lo + (int32_t)(((b >> 32) * span) >> 32);
    }
}

/* out[i] = u in [0, 1) with 53 random bits. */
void wl_fill_uniform_f64(uint64_t seed, uint64_t stream, double *out, int64_t n) {
    uint64_t key = wl_mix(wl_mix(seed) ^ stream);
    for (int64_t i = 0; i < n; ++i) out[i] = (double)(wl_mix(key ^ (uint64_t)i) >> 11) * 0x1.0p-53;
}

/* Constant fill (norm gains are 1.0): fp32 and bf16 variants. */
void wl_fill_const_f32(float v, float *out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = v;
}
void wl_fill_const_bf16(float v, uint16_t *out, int64_t n) {
    uint16_t h = wl_f32_to_bf16_rne(v);
    for (int64_t i = 0; i < n; ++i) out[i] = h;
}
