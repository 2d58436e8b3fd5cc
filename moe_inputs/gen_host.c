/* Host build of the seeded input generator (definition in philox_gen.h). */
#include "philox_gen.h"

void moe_gen_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    moe_gen_philox4x32_10(ctr, key, out);
}

int32_t moe_gen_z_at(uint32_t seed, uint32_t stream, uint64_t index)
{
    return moe_gen_z(seed, stream, index);
}

uint16_t moe_gen_bf16_rne_host(double v)
{
    return moe_gen_bf16_rne(v);
}

/* out[i] = element (start + i) of stream (seed, stream), i in [0, n). */
void moe_gen_fill_bf16(uint32_t seed, uint32_t stream, uint64_t start, int64_t n,
                       double c, uint16_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = moe_gen_bf16(seed, stream, start + (uint64_t)i, c);
}

void moe_gen_fill_f32(uint32_t seed, uint32_t stream, uint64_t start, int64_t n,
                      double c, float *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = moe_gen_f32(seed, stream, start + (uint64_t)i, c);
}
