/*
 * Oracle-side implementation of the seeded random-init spec (test infrastructure;
 * never linked into the product library).
 *
 * The paper states only that instances hold model weights (Sec. 3.2); the
 * spec below is this project's reading: every element is an independent
 * standard normal drawn by Box-Muller (Box & Muller, 1958) from two outputs of
 * the SplitMix64 output function (Steele, Lea & Flood, OOPSLA 2014), keyed by
 * (seed, tensor uid, element index), scaled, rounded fp64 -> fp32 -> bf16
 * (round to nearest even at each step).
 *
 * Written from that definition, independently of the library's generator.
 * glibc's log/cos are used so both sides see the same libm on one host.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static uint64_t sm64_out(uint64_t state)
{
    /* output of one SplitMix64 step taken from `state` */
    uint64_t x = state + 0x9E3779B97F4A7C15ULL;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ULL;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBULL;
    return x ^ (x >> 31);
}

uint64_t oracle_mix64(uint64_t z) { return sm64_out(z); }

uint64_t oracle_tensor_key(uint64_t seed, uint32_t layer, uint32_t slot)
{
    uint64_t uid = 32ULL * (uint64_t)layer + (uint64_t)slot;
    return sm64_out(seed ^ sm64_out(uid));
}

static double std_normal_at(uint64_t key, uint64_t e)
{
    const double two_pi = 6.283185307179586;    /* fl(2*pi) = 2*fl(pi) */
    const double inv2_53 = 1.0 / 9007199254740992.0;
    uint64_t a = sm64_out(key + 2u * e);
    uint64_t b = sm64_out(key + 2u * e + 1u);
    double u1 = (double)((a >> 11) + 1u) * inv2_53;   /* (0, 1] */
    double u2 = (double)(b >> 11) * inv2_53;          /* [0, 1) */
    return sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
}

static uint16_t f32_to_bf16_rne(float f)
{
    uint32_t bits;
    memcpy(&bits, &f, 4);
    /* round half to even on the 16 dropped bits (inputs are finite) */
    uint32_t keep_lsb = (bits >> 16) & 1u;
    bits += 0x7FFFu + keep_lsb;
    return (uint16_t)(bits >> 16);
}

/* bf16 weight tensor, logical [rows, cols] row-major. Columns [0, qk_cols) use
 * sigma_qk when it is non-zero (the Q and K blocks of the fused QKV weight). */
void oracle_gen_bf16(uint64_t key, uint64_t rows, uint64_t cols, uint64_t qk_cols,
                     double sigma, double sigma_qk, uint16_t *out)
{
    const uint64_t n = rows * cols;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        uint64_t e = (uint64_t)i;
        uint64_t c = e % cols;
        double s = (c < qk_cols && sigma_qk != 0.0) ? sigma_qk : sigma;
        float v = (float)(s * std_normal_at(key, e));
        out[i] = f32_to_bf16_rne(v);
    }
}

/* fp32 LayerNorm parameter: gamma = 1 + sigma*n (offset = 1) or beta = sigma*n. */
void oracle_gen_f32(uint64_t key, uint64_t n, double offset, double sigma, float *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)n; ++i)
        out[i] = (float)(offset + sigma * std_normal_at(key, (uint64_t)i));
}

/* raw standard normals (fp64), for distribution checks */
void oracle_std_normals(uint64_t key, uint64_t n, double *out)
{
    for (uint64_t i = 0; i < n; ++i)
        out[i] = std_normal_at(key, i);
}
