/*
 * Seeded synthetic-input generator shared by the CPU oracle and the GPU
 * path.  It holds no arithmetic of the delta-extraction method: it only
 * turns (seed, tensor, kind, element index) into a reproducible value.
 *
 * Generator: Philox4x32-10, the counter-based generator of Salmon, Moraes,
 * Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC 2011):
 * ten rounds of two 32x32->64 multiplies by 0xD2511F53 and 0xCD9E8D57,
 * word shuffling with XOR of the round key, and a Weyl key schedule with
 * increments 0x9E3779B9 and 0xBB67AE85.
 *
 * Transform: the four 32-bit output words are summed exactly in 64-bit
 * integers and centred, giving an Irwin-Hall(4) variate (sum of four
 * uniforms).  One multiplication in binary64 by sigma*sqrt(3)*2^-32 gives
 * standard deviation sigma; one conversion rounds it to binary32.  Every
 * step is exact or a single IEEE round-to-nearest-even operation, so a
 * C build and a HIP build produce identical bits.  The variate is bounded
 * by 2*sqrt(3) sigma; it stands in for a normal draw.
 *
 * The file is plain C99; a HIP translation unit includes it after defining
 * SYNTH_FN as "__host__ __device__ static inline".
 */
#ifndef SYNTH_PHILOX_H
#define SYNTH_PHILOX_H

#include <stdint.h>

#ifndef SYNTH_FN
#define SYNTH_FN static inline
#endif

typedef struct {
    uint32_t w[4];
} synth_block;

/* Philox4x32-10 on counter (c0,c1,c2,c3) under key (k0,k1). */
SYNTH_FN synth_block synth_philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                         uint32_t c3, uint32_t k0, uint32_t k1)
{
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t prod0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        const uint64_t prod1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        const uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
        const uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
        const uint32_t n0 = hi1 ^ c1 ^ k0;
        const uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    synth_block out;
    out.w[0] = c0;
    out.w[1] = c1;
    out.w[2] = c2;
    out.w[3] = c3;
    return out;
}

/* Counter layout of one draw: element index (low, high word), draw kind,
 * tensor ordinal; key = the 64-bit workload seed. */
SYNTH_FN synth_block synth_block_at(uint64_t seed, uint32_t tensor, uint32_t kind,
                                    uint64_t index)
{
    return synth_philox4x32_10((uint32_t)index, (uint32_t)(index >> 32), kind, tensor,
                               (uint32_t)seed, (uint32_t)(seed >> 32));
}

/* Centred sum of the four words: an integer in [-2(2^32-1), 2(2^32-1)]. */
SYNTH_FN int64_t synth_centred_sum(synth_block b)
{
    const uint64_t s = (uint64_t)b.w[0] + (uint64_t)b.w[1] + (uint64_t)b.w[2] +
                       (uint64_t)b.w[3];
    return (int64_t)s - (int64_t)0x1FFFFFFFEull;
}

/* One binary32 draw; scale = sigma*sqrt(3)*2^-32 computed once in binary64
 * by synth_scale(); absval != 0 folds the draw to its magnitude. */
SYNTH_FN float synth_draw(uint64_t seed, uint32_t tensor, uint32_t kind, uint64_t index,
                          double scale, int absval)
{
    const int64_t c = synth_centred_sum(synth_block_at(seed, tensor, kind, index));
    const float x = (float)((double)c * scale);
    return absval ? (x < 0.0f ? -x : x) : x;
}

#endif /* SYNTH_PHILOX_H */
