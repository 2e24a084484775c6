/*
 * Device build of the seeded synthetic-input generator (see philox.h).
 * Built with hipcc for gfx950 into synth/libsynth_hip.so; fills device
 * buffers with the same bits as the host build.  Holds no arithmetic of
 * the delta-extraction method.
 */
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SYNTH_FN __host__ __device__ static inline
#include "philox.h"

namespace {

__global__ __launch_bounds__(256) void synth_fill_kernel(float* __restrict__ out, int64_t n,
                                                          uint64_t seed, uint32_t tensor,
                                                          uint32_t kind, uint64_t index_base,
                                                          double scale, int absval)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = synth_draw(seed, tensor, kind, index_base + (uint64_t)i, scale, absval);
}

__global__ __launch_bounds__(256) void synth_fill_2d_kernel(float* __restrict__ out, int64_t nrows,
                                                             int64_t ncols, int64_t row_stride,
                                                             uint64_t seed, uint32_t tensor,
                                                             uint32_t kind, int64_t row0, int64_t col0,
                                                             int64_t canon_ncols, double scale,
                                                             int absval)
{
    const int64_t n = nrows * ncols;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int64_t r = i / ncols, c = i - r * ncols;
        out[r * row_stride + c] = synth_draw(seed, tensor, kind,
                                             (uint64_t)((row0 + r) * canon_ncols + col0 + c), scale,
                                             absval);
    }
}

}  // namespace

/* Device fill: out[i] = draw(seed, tensor, kind, index_base + i), i in
 * [0, n), on the given stream.  Returns a hipError_t value (0 = success). */
extern "C" int synth_fill_hip(float* out, int64_t n, uint64_t seed, uint32_t tensor,
                              uint32_t kind, uint64_t index_base, double scale, int absval,
                              void* stream)
{
    if (n <= 0) return 0;
    if (out == nullptr) return (int)hipErrorInvalidValue;
    const int64_t want = (n + 255) / 256;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(synth_fill_kernel, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, n,
                       seed, tensor, kind, index_base, scale, absval);
    return (int)hipGetLastError();
}

/* Device 2-D block fill: out[r * row_stride + c] = draw at canonical flat
 * index (row0 + r) * canon_ncols + col0 + c.  Returns a hipError_t value. */
extern "C" int synth_fill_2d_hip(float* out, int64_t nrows, int64_t ncols, int64_t row_stride,
                                 uint64_t seed, uint32_t tensor, uint32_t kind, int64_t row0,
                                 int64_t col0, int64_t canon_ncols, double scale, int absval,
                                 void* stream)
{
    if (nrows <= 0 || ncols <= 0) return 0;
    if (out == nullptr || row_stride < ncols) return (int)hipErrorInvalidValue;
    const int64_t want = (nrows * ncols + 255) / 256;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(synth_fill_2d_kernel, dim3(grid), dim3(256), 0, (hipStream_t)stream, out,
                       nrows, ncols, row_stride, seed, tensor, kind, row0, col0, canon_ncols, scale,
                       absval);
    return (int)hipGetLastError();
}
