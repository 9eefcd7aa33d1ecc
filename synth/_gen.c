/*
 * Seeded synthetic inputs: a counter-based Gaussian generator.
 *
 * This file only draws random numbers; it holds none of the diffusion-LLM
 * arithmetic.  Both the CPU oracle and the GPU path receive the arrays it
 * writes, so they see bit-identical weights.
 *
 * Element i of stream s under seed S is a pure function of (S, s, i):
 *   key    = mix64(S ^ mix64(s + 0x9E3779B97F4A7C15))
 *   z_a    = mix64(key + (2j)   * 0x9E3779B97F4A7C15),  j = i / 2
 *   z_b    = mix64(key + (2j+1) * 0x9E3779B97F4A7C15)
 *   u1     = ((z_a >> 40) + 1) * 2^-24          in (0, 1]
 *   u2     =  (z_b >> 40)      * 2^-24          in [0, 1)
 *   r      = sqrt(-2 ln u1)
 *   n      = r cos(2 pi u2)  (i even)   or   r sin(2 pi u2)  (i odd)
 * which is the Box-Muller transform (Box and Muller, 1958) fed by the
 * SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014), all in
 * float with the C library's logf/sincosf/sqrtf.  The value is multiplied by
 * `stdev` in float and, for the bf16 variant, rounded to bfloat16 to
 * nearest-even.  The 24-bit u1 bounds |n| below about 5.8.
 * Because every element depends only on its index, any sub-range can be
 * regenerated on its own and threads may split the work freely.
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <omp.h>

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
    return mix64(seed ^ mix64(stream + 0x9E3779B97F4A7C15ULL));
}

static inline void normal_pair(uint64_t key, uint64_t j, float* n0, float* n1) {
    const uint64_t g = 0x9E3779B97F4A7C15ULL;
    uint64_t za = mix64(key + (2 * j) * g);
    uint64_t zb = mix64(key + (2 * j + 1) * g);
    float u1 = ((float)(za >> 40) + 1.0f) * (1.0f / 16777216.0f);
    float u2 = (float)(zb >> 40) * (1.0f / 16777216.0f);
    float r = sqrtf(-2.0f * logf(u1));
    float s, c;
    sincosf(6.28318530717958647692f * u2, &s, &c);
    *n0 = r * c;
    *n1 = r * s;
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)(u >> 16); /* inf / nan */
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

#define CHUNK 65536

static void fill(uint64_t seed, uint64_t stream, uint64_t offset, uint64_t n,
                 float stdev, float* out_f32, uint16_t* out_bf16) {
    const uint64_t key = stream_key(seed, stream);
    const int64_t nchunks = (int64_t)((n + CHUNK - 1) / CHUNK);
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < nchunks; ++c) {
        uint64_t b = (uint64_t)c * CHUNK;
        uint64_t e = b + CHUNK < n ? b + CHUNK : n;
        uint64_t t = b;
        while (t < e) {
            uint64_t i = offset + t;
            float n[2];
            normal_pair(key, i >> 1, &n[0], &n[1]);
            for (int h = (int)(i & 1); h < 2 && t < e; ++h, ++t) {
                float v = n[h] * stdev;
                if (out_f32) out_f32[t] = v;
                else out_bf16[t] = f32_to_bf16_rne(v);
            }
        }
    }
}

void synth_normal_f32(uint64_t seed, uint64_t stream, uint64_t offset, uint64_t n,
                      float stdev, float* out) {
    fill(seed, stream, offset, n, stdev, out, 0);
}

void synth_normal_bf16(uint64_t seed, uint64_t stream, uint64_t offset, uint64_t n,
                       float stdev, uint16_t* out) {
    fill(seed, stream, offset, n, stdev, 0, out);
}

/* Uniform integers in [0, hi): (mix64(key + i * golden) >> 11) mod hi. */
void synth_uniform_int(uint64_t seed, uint64_t stream, uint64_t offset, uint64_t n,
                       uint64_t hi, int32_t* out) {
    const uint64_t key = stream_key(seed, stream);
    for (uint64_t t = 0; t < n; ++t)
        out[t] = (int32_t)((mix64(key + (offset + t) * 0x9E3779B97F4A7C15ULL) >> 11) % hi);
}

void synth_set_threads(int n) { omp_set_num_threads(n); }
