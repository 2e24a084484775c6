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
