/*
 * Seeded synthetic inputs for the ASD verifier: target logit rows with a
 * planted greedy peak, and uniform draws for drafts and per-request controls.
 *
 * This file holds no verifier arithmetic.  Both the CPU oracle and the GPU
 * library consume the buffers it writes (the very same host buffer), so the
 * generator is shared by construction and takes no part in either side's
 * computation.
 *
 * Random numbers come from one counter-based generator: the k-th output of
 * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014) seeded with `seed` is
 *     mix(seed + (k + 1) * 0x9E3779B97F4A7C15)
 * with mix the SplitMix64 output function.  Normal draws use the Box-Muller
 * transform (Box and Muller, 1958) on one 64-bit output: the upper 32 bits
 * give u1 in (0, 1), the lower 32 bits give u2 in [0, 1).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define GEN_F32 0
#define GEN_BF16 1

static uint64_t splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t gen_splitmix64_at(uint64_t seed, uint64_t k)
{
    return splitmix64_mix(seed + (k + 1) * 0x9E3779B97F4A7C15ull);
}

/* out[j] = the (k0 + j)-th output as a double in [0, 1) with 53 random bits. */
void gen_u01(uint64_t seed, uint64_t k0, int64_t n, double *out)
{
    for (int64_t j = 0; j < n; ++j)
        out[j] = (double)(gen_splitmix64_at(seed, k0 + (uint64_t)j) >> 11) * 0x1.0p-53;
}

static uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    u += 0x7fffu + ((u >> 16) & 1u);          /* finite inputs only */
    return (uint16_t)(u >> 16);
}

static float bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/*
 * Rows [row0, row0 + nrows) of a [*, vocab] matrix of N(0, sigma^2) draws
 * (sigma is the standard deviation), written to `out` (nrows x vocab).
 * Columns 2j and 2j+1 of global row r share Box-Muller pair number
 * r * ceil(vocab / 2) + j.  Values are rounded double -> binary32 -> bf16
 * (round to nearest even at each step) for dtype 1.
 */
void gen_normal_rows(uint64_t seed, int dtype, int64_t vocab, int64_t row0,
                     int64_t nrows, double sigma, void *out)
{
    const int64_t pairs = (vocab + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t lr = 0; lr < nrows; ++lr) {
        const uint64_t base = (uint64_t)(row0 + lr) * (uint64_t)pairs;
        for (int64_t j = 0; j < pairs; ++j) {
            uint64_t h = gen_splitmix64_at(seed, base + (uint64_t)j);
            double u1 = ((double)(h >> 32) + 0.5) * 0x1.0p-32;
            double u2 = (double)(h & 0xffffffffull) * 0x1.0p-32;
            double rad = sqrt(-2.0 * log(u1));
            double ang = 6.283185307179586 * u2;
            float v[2];
            v[0] = (float)(sigma * rad * cos(ang));
            v[1] = (float)(sigma * rad * sin(ang));
            for (int e = 0; e < 2; ++e) {
                int64_t col = 2 * j + e;
                if (col >= vocab)
                    break;
                if (dtype == GEN_BF16)
                    ((uint16_t *)out)[lr * vocab + col] = f32_to_bf16_rne(v[e]);
                else
                    ((float *)out)[lr * vocab + col] = v[e];
            }
        }
    }
}

/*
 * Plant a peak in every row of `logits` (nrows x vocab): with p = peak_col[r]
 * and m the greatest value among the other columns (first such column w),
 * set z[p] = round(m + margin[r]) (binary32 addition, then bf16 rounding for
 * dtype 1) and report w in runner_col[r].  A margin of 0 makes z[p] equal to
 * z[w].  Rows hold finite values only.
 */
void gen_plant_rows(int dtype, int64_t vocab, int64_t nrows, void *logits,
                    const int64_t *peak_col, const float *margin,
                    int32_t *runner_col)
{
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t p = peak_col[r];
        int64_t w = -1;
        float m = 0.0f;
        for (int64_t c = 0; c < vocab; ++c) {
            float v;
            if (c == p)
                continue;
            v = dtype == GEN_BF16 ? bf16_to_f32(((const uint16_t *)logits)[r * vocab + c])
                                  : ((const float *)logits)[r * vocab + c];
            if (w < 0 || v > m) {
                m = v;
                w = c;
            }
        }
        if (w < 0) {            /* vocab == 1: nothing else in the row */
            runner_col[r] = (int32_t)p;
            continue;
        }
        {
            float top = m + margin[r];
            if (dtype == GEN_BF16)
                ((uint16_t *)logits)[r * vocab + p] = f32_to_bf16_rne(top);
            else
                ((float *)logits)[r * vocab + p] = top;
        }
        runner_col[r] = (int32_t)w;
    }
}

int gen_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
