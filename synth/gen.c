/*
 * Seeded synthetic inputs for the tree-verification workloads.
 *
 * This file holds no arithmetic of the verification method: it only turns
 * (seed, tensor id, element index) into numbers.  The stream is the
 * splitmix64 generator (Steele, Lea and Flood, "Fast splittable pseudorandom
 * number generators", OOPSLA 2014; constants as in Vigna's public-domain
 * reference), used counter-style: element i of a stream keyed by k is
 * mix(k + (i + 1) * golden).  Normals come from the Box-Muller transform
 * (Box and Muller, 1958) over the two 32-bit halves of one draw.
 *
 * Both the GPU path and the CPU oracle consume the bytes this writes; neither
 * calls it directly for arithmetic.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t dvs_key(uint64_t seed, uint64_t tensor)
{
    return mix64(mix64(seed + GOLDEN) ^ (tensor * GOLDEN));
}

static inline uint64_t draw(uint64_t key, uint64_t i)
{
    return mix64(key + (i + 1) * GOLDEN);
}

/* fp32 -> bf16 bit pattern, round to nearest even (finite inputs only). */
static inline uint16_t f32_to_bf16_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* Normal pair from draw j: (r cos t, r sin t), r = sqrt(-2 ln u1), t = 2 pi u2,
 * evaluated in single precision. */
static inline void normal_pair(uint64_t key, uint64_t j, float *z0, float *z1)
{
    uint64_t r = draw(key, j);
    float u1 = ((float)(uint32_t)(r >> 40) + 0.5f) * (1.0f / 16777216.0f);
    float u2 = ((float)(uint32_t)((r >> 8) & 0xFFFFFFu) + 0.5f) * (1.0f / 16777216.0f);
    float rad = sqrtf(-2.0f * logf(u1));
    float t = 6.28318530717958647692f * u2;
    *z0 = rad * cosf(t);
    *z1 = rad * sinf(t);
}

/* Element i of the normal stream scaled by sigma, as fp32; draws are consumed
 * in pairs (element 2j and 2j+1 share draw j). */
#define NORMAL_LOOP(STORE)                                                    \
    uint64_t key = dvs_key(seed, tensor);                                     \
    uint64_t end = start + n;                                                 \
    long long p0 = (long long)(start >> 1), p1 = (long long)((end + 1) >> 1); \
    _Pragma("omp parallel for schedule(static, 32768)")                       \
    for (long long j = p0; j < p1; ++j) {                                     \
        float z[2];                                                           \
        normal_pair(key, (uint64_t)j, &z[0], &z[1]);                          \
        for (int h = 0; h < 2; ++h) {                                         \
            uint64_t i = 2 * (uint64_t)j + (uint64_t)h;                       \
            if (i >= start && i < end) {                                      \
                float v = (float)sigma * z[h];                                \
                STORE;                                                        \
            }                                                                 \
        }                                                                     \
    }

/* out[e] = bf16(sigma * N_{start+e}), e < n. */
void dvs_normal_bf16(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n,
                     double sigma, uint16_t *out)
{
    NORMAL_LOOP(out[i - start] = f32_to_bf16_bits(v))
}

/* out[e] = fp32(sigma * N_{start+e}), e < n. */
void dvs_normal_f32(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n,
                    double sigma, float *out)
{
    NORMAL_LOOP(out[i - start] = v)
}

/* Norm gains scattered around 1: out[e] = bf16(1 + sigma * N_{start+e}). */
void dvs_gain_bf16(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n,
                   double sigma, uint16_t *out)
{
    NORMAL_LOOP(out[i - start] = f32_to_bf16_bits(1.0f + v))
}

/* The same as fp32: out[e] = fp32(1 + sigma * N_{start+e}). */
void dvs_gain_f32(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n,
                  double sigma, float *out)
{
    NORMAL_LOOP(out[i - start] = 1.0f + v)
}

/* out[e] = int8(clamp(rint(sigma * N_{start+e}), -127, 127)), e < n: integer
 * codes with a Gaussian profile (sigma = 127/4 puts the clip at 4 standard
 * deviations). */
void dvs_normal_i8(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n,
                   double sigma, int8_t *out)
{
    NORMAL_LOOP({
        float r = rintf(v);
        r = r > 127.f ? 127.f : (r < -127.f ? -127.f : r);
        out[i - start] = (int8_t)r;
    })
}

/* Raw 64-bit draws (for small host-side choices such as tree shapes). */
void dvs_u64(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n, uint64_t *out)
{
    uint64_t key = dvs_key(seed, tensor);
    for (uint64_t e = 0; e < n; ++e)
        out[e] = draw(key, start + e);
}

/* Uniform integers in [0, hi): multiply-shift of the high 32 bits. */
void dvs_uniform_int(uint64_t seed, uint64_t tensor, uint64_t start, uint64_t n,
                     uint32_t hi, int32_t *out)
{
    uint64_t key = dvs_key(seed, tensor);
    for (uint64_t e = 0; e < n; ++e)
        out[e] = (int32_t)(((draw(key, start + e) >> 32) * (uint64_t)hi) >> 32);
}
