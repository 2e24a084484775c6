/*
 * Host build of the seeded synthetic-input generator (see philox.h).
 * Built with gcc into synth/libsynth_cpu.so; used by the CPU oracle and by
 * host-side tests.  Holds no arithmetic of the delta-extraction method.
 */
#include <math.h>
#include <stdint.h>

#include "philox.h"

/* sigma*sqrt(3)*2^-32 in binary64: scales a centred Irwin-Hall(4) sum of
 * 32-bit words to standard deviation sigma. */
double synth_scale(double sigma)
{
    return (sigma * sqrt(3.0)) * 0x1p-32;
}

/* Raw Philox4x32-10 block, exposed for known-answer tests. */
void synth_philox_block(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    const synth_block b = synth_philox4x32_10(ctr[0], ctr[1], ctr[2], ctr[3], key[0], key[1]);
    for (int i = 0; i < 4; ++i) out[i] = b.w[i];
}

/* First output word of the block at (seed, tensor, kind, index). */
uint32_t synth_word(uint64_t seed, uint32_t tensor, uint32_t kind, uint64_t index)
{
    return synth_block_at(seed, tensor, kind, index).w[0];
}

/* out[i] = draw(seed, tensor, kind, index_base + i) for i in [0, n). */
void synth_fill_cpu(float* out, int64_t n, uint64_t seed, uint32_t tensor, uint32_t kind,
                    uint64_t index_base, double scale, int absval)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = synth_draw(seed, tensor, kind, index_base + (uint64_t)i, scale, absval);
}
