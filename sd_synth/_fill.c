/* Seeded synthetic-input filler shared by the oracle side and the GPU side.
 *
 * Holds no arithmetic of the decoding method: element i of a tensor with
 * 64-bit key K is table[h(i, K) >> 16], where h is two rounds of a 32-bit
 * integer mixer and table holds the 65536 equiprobable quantiles of the
 * target distribution.  This is inverse-transform sampling with a 16-bit
 * uniform; integer-only, so every machine produces the same bits.
 */
#include <stdint.h>

static inline uint32_t mix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352dU;
    x ^= x >> 15;
    x *= 0x846ca68bU;
    x ^= x >> 16;
    return x;
}

static inline uint32_t draw16(int64_t i, uint64_t key)
{
    uint32_t h = mix32((uint32_t)i + (uint32_t)key);
    h = mix32(h ^ (uint32_t)(key >> 32) ^ (uint32_t)((uint64_t)i >> 32) * 0x9e3779b9U);
    return h >> 16;
}

void sdsynth_fill_u16(uint16_t *out, int64_t n, uint64_t key, const uint16_t *table)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = table[draw16(i, key)];
}

void sdsynth_fill_f32(float *out, int64_t n, uint64_t key, const float *table)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = table[draw16(i, key)];
}
