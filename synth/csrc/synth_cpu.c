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

/* 2-D block: out[r * row_stride + c] = draw at canonical flat index
 * (row0 + r) * canon_ncols + col0 + c, for r < nrows, c < ncols. */
void synth_fill_2d_cpu(float* out, int64_t nrows, int64_t ncols, int64_t row_stride,
                       uint64_t seed, uint32_t tensor, uint32_t kind, int64_t row0, int64_t col0,
                       int64_t canon_ncols, double scale, int absval)
{
    for (int64_t r = 0; r < nrows; ++r) {
        const uint64_t base = (uint64_t)((row0 + r) * canon_ncols + col0);
        for (int64_t c = 0; c < ncols; ++c)
            out[r * row_stride + c] = synth_draw(seed, tensor, kind, base + (uint64_t)c, scale, absval);
    }
}
