/*
 * philox_gen.h -- the seeded synthetic-input generator shared by the tests,
 * the benchmark and the CPU oracle's callers.  It holds none of the MoE
 * layer's arithmetic: it only turns (seed, stream, element index) into the
 * bits of an input tensor element.  The same source is compiled by gcc for
 * the host library and by hipcc for the device kernel, and every operation
 * below is exact integer work or a single IEEE-754 double multiply, so both
 * produce identical bits.
 *
 * Generator definition
 *   1. Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers:
 *      as easy as 1, 2, 3", SC'11): key = (seed, stream), counter =
 *      (index mod 2^32, index div 2^32, 0, 0).  Ten rounds with multipliers
 *      0xD2511F53 / 0xCD9E8D57 and Weyl key increments 0x9E3779B9 /
 *      0xBB67AE85.
 *   2. The 128 output bits are read as eight 16-bit unsigned integers u_i;
 *      S = sum u_i (Irwin-Hall sum of eight uniforms, an approximately normal
 *      variable with support of +-4.9 standard deviations).
 *   3. z = 2*S - 8*65535 is an exact even integer with mean 0 and standard
 *      deviation 2*sqrt(8*(65536^2-1)/12).
 *   4. value = (double)z * c, where the caller passes c = sigma / sd(z), so
 *      the value has mean 0 and standard deviation sigma.  One rounding.
 *   5. bf16 tensors take the round-to-nearest-even bf16 of that double
 *      (integer implementation below); fp32 tensors take (float)value.
 */
#ifndef MOE_INPUTS_PHILOX_GEN_H
#define MOE_INPUTS_PHILOX_GEN_H

#include <stdint.h>

#if defined(__HIPCC__)
#define MOE_GEN_FN static inline __host__ __device__
#else
#define MOE_GEN_FN static inline
#endif

MOE_GEN_FN void moe_gen_philox4x32_10(const uint32_t ctr_in[4],
                                      const uint32_t key_in[2],
                                      uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; ++r) {
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Steps 1-3: the exact integer z for one element. */
MOE_GEN_FN int32_t moe_gen_z(uint32_t seed, uint32_t stream, uint64_t index)
{
    uint32_t ctr[4] = {(uint32_t)index, (uint32_t)(index >> 32), 0u, 0u};
    uint32_t key[2] = {seed, stream};
    uint32_t r[4];
    moe_gen_philox4x32_10(ctr, key, r);
    int32_t s = 0;
    for (int i = 0; i < 4; ++i)
        s += (int32_t)(r[i] & 0xFFFFu) + (int32_t)(r[i] >> 16);
    return 2 * s - 8 * 65535;
}

/* Step 5 for bf16: round-to-nearest-even of a double, integer-only. */
MOE_GEN_FN uint16_t moe_gen_bf16_rne(double v)
{
    union { double d; uint64_t u; } cv;
    cv.d = v;
    uint64_t b = cv.u;
    uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
    uint64_t a = b & 0x7FFFFFFFFFFFFFFFull;
    if (a > 0x7FF0000000000000ull)
        return (uint16_t)(sign | 0x7FC0u);                 /* NaN */
    if (a == 0x7FF0000000000000ull)
        return (uint16_t)(sign | 0x7F80u);                 /* inf */
    int bexp = (int)(a >> 52);
    if (bexp == 0)
        return sign;                      /* below 2^-1022: rounds to zero */
    uint64_t mant = (a & 0x000FFFFFFFFFFFFFull) | 0x0010000000000000ull;
    int e_unb = bexp - 1023;              /* v in [2^e_unb, 2^(e_unb+1)) */
    int qexp = (e_unb < -126 ? -126 : e_unb) - 7;   /* bf16 quantum 2^qexp */
    int shift = qexp - (bexp - 1075);     /* low significand bits to drop */
    if (shift > 54)
        return sign;                      /* below a quarter quantum */
    uint64_t q = mant >> shift;
    uint64_t rem = mant & ((1ull << shift) - 1ull);
    uint64_t half = 1ull << (shift - 1);
    if (rem > half || (rem == half && (q & 1ull)))
        q += 1ull;
    if (q >= 256ull) {                    /* carried into the next binade */
        q >>= 1;
        qexp += 1;
    }
    if (q >= 128ull) {                    /* normal bf16 */
        int biased = qexp + 7 + 127;
        if (biased >= 255)
            return (uint16_t)(sign | 0x7F80u);
        return (uint16_t)(sign | (uint16_t)(biased << 7) | (uint16_t)(q & 127ull));
    }
    return (uint16_t)(sign | (uint16_t)q); /* subnormal bf16, quantum 2^-133 */
}

MOE_GEN_FN uint16_t moe_gen_bf16(uint32_t seed, uint32_t stream, uint64_t index,
                                 double c)
{
    return moe_gen_bf16_rne((double)moe_gen_z(seed, stream, index) * c);
}

MOE_GEN_FN float moe_gen_f32(uint32_t seed, uint32_t stream, uint64_t index,
                             double c)
{
    return (float)((double)moe_gen_z(seed, stream, index) * c);
}

#endif /* MOE_INPUTS_PHILOX_GEN_H */
