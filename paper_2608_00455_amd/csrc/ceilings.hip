// Reference kernels that bound what the hot path's kernels can reach on
// this GPU, for the benchmark's second roofline denominators.  They are
// measurement aids, not steps of the method, and live in their own library
// (libceilings.so), outside the C ABI of include/dte.h.
//
//  - ceil_read3: a plain read of three binary32 arrays (the 12 bytes per
//    element that delta extraction must read), in extract's access pattern
//    (persistent grid, each wave a contiguous range of 2048-element tiles,
//    eight 16-byte non-temporal loads per lane and array in flight) with no
//    arithmetic beyond folding the loaded bits, and no stores;
//    ceil_read3_dynamic: the same read by one 12-wave block per CU taking
//    four tiles per wave at a time from a counter (the CUs do not stream at
//    one rate, so a static split ends unevenly);
//  - ceil_read3_write: the same read, plus the output extraction writes
//    for a delta of a given size: 8-byte offsets (non-temporal stores) and
//    2-byte values, spread evenly over the tiles, each wave writing its
//    tiles' share contiguously, with no atomics, no selection and nothing
//    else: the read and write mix that extraction's bytes make, issued
//    naively; ceil_write_entries: the same entries written alone, each wave
//    one contiguous range.  A read stream and a write stream, one after the
//    other, bound any kernel that moves extraction's bytes over the one
//    memory bus;
//  - ceil_line_writes: for every bucket entry of every rank, a whole 64-byte
//    line written at the line that holds the entry's element (four 16-byte
//    stores), into a buffer of the shard's size: the rate of scattered
//    line updates at apply's addresses, without the read-modify-write that
//    a 2-byte store costs.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kVec = 8;
constexpr int kTile = 64 * 4 * kVec;   // elements per wave tile

__global__ __launch_bounds__(kBlock) void read3_kernel(const float* __restrict__ a,
                                                       const float* __restrict__ b,
                                                       const float* __restrict__ c, int64_t tiles,
                                                       uint32_t* __restrict__ sink)
{
    const int lane = threadIdx.x & 63;
    const int64_t g = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    const int64_t per = (tiles + nw - 1) / nw;
    const int64_t first = g * per;
    const int64_t last = first + per < tiles ? first + per : tiles;
    uint32_t acc = 0;
    for (int64_t t = first; t < last; ++t) {
        f32x4 A[kVec], B[kVec], C[kVec];
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
            const int64_t e = t * kTile + (int64_t)(j * 64 + lane) * 4;
            A[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a + e));
            B[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(b + e));
            C[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(c + e));
        }
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
            const u32x4 x = __builtin_bit_cast(u32x4, A[j]) ^ __builtin_bit_cast(u32x4, B[j]) ^
                            __builtin_bit_cast(u32x4, C[j]);
            acc ^= x.x ^ x.y ^ x.z ^ x.w;
        }
    }
    // a store the compiler cannot rule out keeps the loads; it practically
    // never happens
    if (acc == 0x9E3779B9u) sink[g * 64 + lane] = acc;
}

// read3_kernel's read with blocks of 12 waves taking 4 tiles per wave at a
// time: chunk k (from the counter) is tiles [48 k, 48 k + 48).
constexpr int kDynWaves = 12;
constexpr int kDynTiles = 4;

__global__ __launch_bounds__(64 * kDynWaves) void read3_dynamic_kernel(
    const float* __restrict__ a, const float* __restrict__ b, const float* __restrict__ c,
    int64_t tiles, unsigned long long* __restrict__ counter, uint32_t* __restrict__ sink)
{
    __shared__ int64_t s_chunk;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    uint32_t acc = 0;
    for (;;) {
        if (threadIdx.x == 0) s_chunk = (int64_t)atomicAdd(counter, 1ull);
        __syncthreads();
        const int64_t c0 = s_chunk * (kDynWaves * kDynTiles);   // block-uniform
        __syncthreads();                                        // s_chunk is rewritten next
        if (c0 >= tiles) break;
        for (int i = 0; i < kDynTiles; ++i) {
            const int64_t t = c0 + (int64_t)wave * kDynTiles + i;
            if (t >= tiles) break;
            f32x4 A[kVec], B[kVec], C[kVec];
#pragma unroll
            for (int j = 0; j < kVec; ++j) {
                const int64_t e = t * kTile + (int64_t)(j * 64 + lane) * 4;
                A[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a + e));
                B[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(b + e));
                C[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(c + e));
            }
#pragma unroll
            for (int j = 0; j < kVec; ++j) {
                const u32x4 x = __builtin_bit_cast(u32x4, A[j]) ^ __builtin_bit_cast(u32x4, B[j]) ^
                                __builtin_bit_cast(u32x4, C[j]);
                acc ^= x.x ^ x.y ^ x.z ^ x.w;
            }
        }
    }
    const int64_t g = (int64_t)blockIdx.x * kDynWaves + wave;
    if (acc == 0x9E3779B9u) sink[g * 64 + lane] = acc;
}

// read3_kernel plus, for tile t, entries [E t / tiles, E (t+1) / tiles) of
// out_idx / out_val written (values independent of the loads, so that the
// stores wait for nothing).
__global__ __launch_bounds__(kBlock) void read3_write_kernel(const float* __restrict__ a,
                                                             const float* __restrict__ b,
                                                             const float* __restrict__ c,
                                                             int64_t tiles, int64_t entries,
                                                             int64_t* __restrict__ out_idx,
                                                             uint16_t* __restrict__ out_val,
                                                             uint32_t* __restrict__ sink)
{
    const int lane = threadIdx.x & 63;
    const int64_t g = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    const int64_t per = (tiles + nw - 1) / nw;
    const int64_t first = g * per;
    const int64_t last = first + per < tiles ? first + per : tiles;
    uint32_t acc = 0;
    for (int64_t t = first; t < last; ++t) {
        f32x4 A[kVec], B[kVec], C[kVec];
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
            const int64_t e = t * kTile + (int64_t)(j * 64 + lane) * 4;
            A[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a + e));
            B[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(b + e));
            C[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(c + e));
        }
        const int64_t e0 = entries * t / tiles, e1 = entries * (t + 1) / tiles;
        for (int64_t e = e0 + lane; e < e1; e += 64) {
            __builtin_nontemporal_store(t * kTile + (e - e0), out_idx + e);
            out_val[e] = (uint16_t)e;
        }
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
            const u32x4 x = __builtin_bit_cast(u32x4, A[j]) ^ __builtin_bit_cast(u32x4, B[j]) ^
                            __builtin_bit_cast(u32x4, C[j]);
            acc ^= x.x ^ x.y ^ x.z ^ x.w;
        }
    }
    if (acc == 0x9E3779B9u) sink[g * 64 + lane] = acc;
}

// Entries [E g / waves, E (g+1) / waves) of out_idx / out_val written by
// wave g, 64 at a time.
__global__ __launch_bounds__(kBlock) void write_entries_kernel(int64_t entries,
                                                               int64_t* __restrict__ out_idx,
                                                               uint16_t* __restrict__ out_val)
{
    const int lane = threadIdx.x & 63;
    const int64_t g = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    const int64_t e1 = entries * (g + 1) / nw;
    for (int64_t e = entries * g / nw + lane; e < e1; e += 64) {
        __builtin_nontemporal_store(e, out_idx + e);
        out_val[e] = (uint16_t)e;
    }
}

constexpr int kMaxRanks = 16;
constexpr int kUnroll = 8;

struct LineSlice {
    int32_t count;
    uint16_t* dst[kMaxRanks];
    const int64_t* off[kMaxRanks];
    int64_t cap[kMaxRanks];
    int64_t numel[kMaxRanks];
};

__global__ __launch_bounds__(kBlock) void line_write_kernel(LineSlice s,
                                                            const int64_t* __restrict__ count)
{
    const int64_t nthreads = (int64_t)gridDim.x * kBlock;
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const u32x4 pat = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
    for (int r = 0; r < s.count; ++r) {
        int64_t n = count[r];
        if (n > s.cap[r]) n = s.cap[r];
        const int64_t* off = s.off[r];
        uint16_t* dst = s.dst[r];
        const int64_t lines = s.numel[r] / 32;   // whole 64-byte lines of the buffer
        for (int64_t e0 = t; e0 < n; e0 += nthreads * kUnroll) {
            int64_t j[kUnroll];
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int64_t e = e0 + k * nthreads;
                j[k] = e < n ? off[e] : -1;
            }
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int64_t line = j[k] >= 0 ? j[k] >> 5 : -1;
                if (line >= 0 && line < lines) {
                    u32x4* q = reinterpret_cast<u32x4*>(dst + line * 32);
                    q[0] = pat;
                    q[1] = pat;
                    q[2] = pat;
                    q[3] = pat;
                }
            }
        }
    }
}

int cus_of_current()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return 256;
    return n;
}

}  // namespace

extern "C" {

// Waves that ceil_read3 launches for blocks_per_cu (the size of `sink` it
// needs is 64 uint32 per wave).
int64_t ceil_read3_waves(int32_t blocks_per_cu)
{
    return blocks_per_cu > 0 ? (int64_t)cus_of_current() * blocks_per_cu * kWaves : -1;
}

// Read a, b, c (device, binary32, 16-byte aligned) over the whole tiles of
// n elements (n rounded down to a multiple of 2048); grid of blocks_per_cu
// blocks of 256 threads per CU; sink: device uint32[64 * ceil_read3_waves].
// Returns 0, 1 on a bad argument, 4 on a HIP error.
int ceil_read3(const float* a, const float* b, const float* c, int64_t n, int32_t blocks_per_cu,
               uint32_t* sink, void* stream)
{
    if (!a || !b || !c || !sink || n < 0 || blocks_per_cu <= 0 ||
        ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
          reinterpret_cast<uintptr_t>(c)) & 15u) != 0)
        return 1;
    const int64_t tiles = n / kTile;
    if (tiles == 0) return 0;
    const dim3 grid((unsigned)(cus_of_current() * blocks_per_cu));
    hipLaunchKernelGGL(read3_kernel, grid, dim3(kBlock), 0, (hipStream_t)stream, a, b, c, tiles,
                       sink);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

// ceil_read3 with the dynamic split of read3_dynamic_kernel: one block of
// 12 waves per CU; counter: device uint64, zero on entry (the call leaves
// it at the number of chunks taken); sink: device uint32[64 *
// ceil_read3_waves(3)].  Returns 0, 1 on a bad argument, 4 on a HIP error.
int ceil_read3_dynamic(const float* a, const float* b, const float* c, int64_t n,
                       unsigned long long* counter, uint32_t* sink, void* stream)
{
    if (!a || !b || !c || !sink || !counter || n < 0 ||
        ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
          reinterpret_cast<uintptr_t>(c)) & 15u) != 0)
        return 1;
    const int64_t tiles = n / kTile;
    if (tiles == 0) return 0;
    hipLaunchKernelGGL(read3_dynamic_kernel, dim3((unsigned)cus_of_current()),
                       dim3(64 * kDynWaves), 0, (hipStream_t)stream, a, b, c, tiles, counter, sink);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

// ceil_read3 plus writes of `entries` (offset, value) pairs to out_idx[0,
// entries) and out_val[0, entries) (device; out_idx 8-byte aligned), spread
// evenly over the tiles.  The written values are meaningless.  Returns 0, 1
// on a bad argument, 4 on a HIP error.
int ceil_read3_write(const float* a, const float* b, const float* c, int64_t n, int64_t entries,
                     int64_t* out_idx, uint16_t* out_val, int32_t blocks_per_cu, uint32_t* sink,
                     void* stream)
{
    if (!a || !b || !c || !sink || !out_idx || !out_val || n < 0 || entries < 0 ||
        entries > ((int64_t)1 << 40) || blocks_per_cu <= 0 ||
        ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
          reinterpret_cast<uintptr_t>(c)) & 15u) != 0 ||
        (reinterpret_cast<uintptr_t>(out_idx) & 7u) != 0 ||
        (reinterpret_cast<uintptr_t>(out_val) & 1u) != 0)
        return 1;
    const int64_t tiles = n / kTile;
    if (tiles == 0) return 0;
    if (entries > 0 && tiles > ((int64_t)1 << 62) / entries) return 1;   // E (t+1) fits int64
    const dim3 grid((unsigned)(cus_of_current() * blocks_per_cu));
    hipLaunchKernelGGL(read3_write_kernel, grid, dim3(kBlock), 0, (hipStream_t)stream, a, b, c,
                       tiles, entries, out_idx, out_val, sink);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

// The (offset, value) writes of ceil_read3_write alone: entries [0,
// entries) of out_idx / out_val (device; out_idx 8-byte aligned), each wave
// one contiguous range; blocks_per_cu blocks of 256 threads per CU.  The
// written values are meaningless.  Returns 0, 1 on a bad argument, 4 on a
// HIP error.
int ceil_write_entries(int64_t entries, int64_t* out_idx, uint16_t* out_val,
                       int32_t blocks_per_cu, void* stream)
{
    if (!out_idx || !out_val || entries < 0 || entries > ((int64_t)1 << 40) ||
        blocks_per_cu <= 0 || (reinterpret_cast<uintptr_t>(out_idx) & 7u) != 0 ||
        (reinterpret_cast<uintptr_t>(out_val) & 1u) != 0)
        return 1;
    if (entries == 0) return 0;
    const dim3 grid((unsigned)(cus_of_current() * blocks_per_cu));
    hipLaunchKernelGGL(write_entries_kernel, grid, dim3(kBlock), 0, (hipStream_t)stream, entries,
                       out_idx, out_val);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

// For r < nranks (<= 16): for k < min(count[r], cap[r]), write the 64-byte
// line of dst[r] (device, 64-byte aligned, numel[r] uint16) holding element
// off[r][k]; entries whose line is not whole inside the buffer are skipped.
// dst, off, cap, numel: host arrays; count: device int64[nranks].  The
// buffer's contents afterwards are a fixed pattern at those lines.
int ceil_line_writes(int32_t nranks, uint16_t* const* dst, const int64_t* const* off,
                     const int64_t* count, const int64_t* cap, const int64_t* numel,
                     int32_t blocks_per_cu, void* stream)
{
    if (nranks < 1 || nranks > kMaxRanks || !dst || !off || !count || !cap || !numel ||
        blocks_per_cu <= 0)
        return 1;
    LineSlice s{};
    s.count = nranks;
    for (int r = 0; r < nranks; ++r) {
        if (!dst[r] || !off[r] || (reinterpret_cast<uintptr_t>(dst[r]) & 63u) != 0) return 1;
        s.dst[r] = dst[r];
        s.off[r] = off[r];
        s.cap[r] = cap[r];
        s.numel[r] = numel[r];
    }
    const dim3 grid((unsigned)(cus_of_current() * blocks_per_cu));
    hipLaunchKernelGGL(line_write_kernel, grid, dim3(kBlock), 0, (hipStream_t)stream, s, count);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

}  // extern "C"
