/*
 * Seeded synthetic input generator for the minimal executable programs of the
 * dense matrix-vector family (the Input Data Generator of Sec. 3.1.2, Eq. 2).
 *
 * This module only draws numbers: it holds none of the matrix-vector
 * arithmetic, so that both the GPU path and the CPU oracle can be fed the
 * very same bits without sharing any computation.
 *
 * Generator: SplitMix64 (G. L. Steele, D. Lea, C. H. Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used in counter form:
 *   gamma   = 0x9E3779B97F4A7C15
 *   mix(z)  = z ^= z >> 30; z *= 0xBF58476D1CE4E5B9;
 *             z ^= z >> 27; z *= 0x94D049BB133111EB; z ^= z >> 31
 *   key(seed, a)   = mix(seed + (a + 1) * gamma)     (a = array number)
 *   bits(seed,a,k) = mix(key(seed, a) + (k + 1) * gamma)
 * so element k of array a never depends on how many elements are drawn or on
 * the number of threads drawing them.
 *
 * Conversions (all exact, no rounding):
 *   uniform[-1,1) f32: (int64)(bits >> 40) - 2^23, times 2^-23
 *   uniform[-1,1) f64: (int64)(bits >> 11) - 2^52, times 2^-52
 *   ternary {-1,0,1}:  ((bits >> 32) mod 3) - 1
 * normal(0,1): Box-Muller in fp64 on draws 2k and 2k+1,
 *   u1 = ((bits >> 11) + 1) * 2^-53 in (0,1], u2 = (bits >> 11) * 2^-53,
 *   z  = sqrt(-2 ln u1) * cos(2 pi u2), then rounded to the element type.
 *
 * Build: gcc -O2 -fopenmp -fPIC -shared (no HIP, no other sources).
 */
#include <math.h>
#include <stdint.h>

#define DG_GAMMA 0x9E3779B97F4A7C15ULL

static uint64_t dg_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static uint64_t dg_key(uint64_t seed, uint64_t array_id)
{
    return dg_mix(seed + (array_id + 1) * DG_GAMMA);
}

/* Every draw below fills out[k] with element first + k of the array, so a
 * large array can be drawn in pieces that match one whole draw bit for bit. */

/* Raw 64-bit draws: out[k] = bits(seed, array_id, first + k). */
void mep_dg_bits(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, uint64_t* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k)
        out[k] = dg_mix(key + (first + (uint64_t)k + 1) * DG_GAMMA);
}

void mep_dg_uniform_f32(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, float* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k) {
        uint64_t b = dg_mix(key + (first + (uint64_t)k + 1) * DG_GAMMA);
        int64_t v = (int64_t)(b >> 40) - (int64_t)(1LL << 23);
        out[k] = (float)v * 0x1p-23f;
    }
}

void mep_dg_uniform_f64(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, double* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k) {
        uint64_t b = dg_mix(key + (first + (uint64_t)k + 1) * DG_GAMMA);
        int64_t v = (int64_t)(b >> 11) - (int64_t)(1LL << 52);
        out[k] = (double)v * 0x1p-52;
    }
}

static double dg_normal(uint64_t key, int64_t k)
{
    uint64_t b1 = dg_mix(key + ((uint64_t)(2 * k) + 1) * DG_GAMMA);
    uint64_t b2 = dg_mix(key + ((uint64_t)(2 * k + 1) + 1) * DG_GAMMA);
    double u1 = (double)((b1 >> 11) + 1) * 0x1p-53;
    double u2 = (double)(b2 >> 11) * 0x1p-53;
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925286766559 * u2);
}

void mep_dg_normal_f32(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, float* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k)
        out[k] = (float)dg_normal(key, (int64_t)first + k);
}

void mep_dg_normal_f64(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, double* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k)
        out[k] = dg_normal(key, (int64_t)first + k);
}

void mep_dg_ternary_f32(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, float* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k) {
        uint64_t b = dg_mix(key + (first + (uint64_t)k + 1) * DG_GAMMA);
        out[k] = (float)((int)((b >> 32) % 3) - 1);
    }
}

void mep_dg_ternary_f64(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, double* out)
{
    const uint64_t key = dg_key(seed, array_id);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k) {
        uint64_t b = dg_mix(key + (first + (uint64_t)k + 1) * DG_GAMMA);
        out[k] = (double)((int)((b >> 32) % 3) - 1);
    }
}
