/*
 * synth_host.c -- fast host implementation of the seeded N(0,1) bf16
 * generator defined in synth.py (SplitMix64 draw, Box-Muller cosine branch
 * in double, rounded to float then to bf16, nearest even).  It holds none of
 * the attention arithmetic; synth.py falls back to numpy when it is not
 * built, and a test checks both give the same bits.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static uint16_t normal_bf16(uint64_t z)
{
    double u1 = ((double)(z >> 32) + 1.0) * 0x1p-32;
    double u2 = (double)(z & 0xffffffffull) * 0x1p-32;
    double x = sqrt(-2.0 * log(u1)) * cos(u2 * 6.283185307179586);
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

/* out[i] = value number (start + i) of stream (seed, stream). */
void ts_synth_normal_bf16_host(uint64_t seed, uint32_t stream, int64_t start, int64_t count,
                               uint16_t *out)
{
    const uint64_t key = mix64(((seed & ((1ull << 56) - 1)) << 8) + stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; i++)
        out[i] = normal_bf16(mix64(key + ((uint64_t)(start + i) + 1) * 0x9E3779B97F4A7C15ull));
}
