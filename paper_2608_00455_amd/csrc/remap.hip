// Receiver-space remap (paper sec. 4.2.2) and direct sparse apply (sec. 4.3,
// eq. direct_sparse_apply) for gfx950.
//
// Remap: every entry (flat trainer offset i, BF16 value) finds its segment
// through a direct-mapped bucket table (bucket = i >> shift holds the
// segment of its first element; a short forward scan finishes the search),
// unravels i - flat_begin over the segment's row-major shape
// (eq. canonical_unravel), and for each operation of the segment tests
// containment a_s <= u < a_s + e and ravels u - a_s + a_r over the
// receiver view (eq. receiver_local_remapping).
//
// Work unit: a wave takes 512 consecutive entries (8 per lane) into
// registers, and keeps them there from counting to writing.  Extract emits local ascending runs, so a chunk usually lies in
// one segment: then each operation of the segment is loaded once (into
// scalar registers) and tested against all eight slots, one ballot per slot.
// Chunks that span segments route slot by slot, lanes grouped by segment.
// Each block owns a contiguous slice of the entries, taken 2048 at a time
// (one chunk per wave): count the outputs per rank, reserve bucket space
// with one atomicAdd per touched rank, recompute and write (offset, value)
// at the reserved positions from the same registers (a few atomics per
// block: same-address atomics serialise at the memory side, so they are
// kept out of the inner loops).
//
// Apply: shard[off] = val; each lane keeps eight independent
// load-then-store chains in flight (the scattered 2-byte stores are
// read-modify-write at the memory side, so parallelism is what matters);
// ranks with dense updates or shards larger than 1 GiB store past the cache.
#include <hip/hip_runtime.h>

#include "dte_internal.h"
#include "route.h"

namespace dte {
namespace {

using namespace rt;

constexpr int kBlock = 256;

__global__ void zero_i64_kernel(int64_t* p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

constexpr int kWaves = kBlock / 64;
constexpr int kRemapSlots = 8;                     // entries per lane per chunk
constexpr int kChunk = 64 * kRemapSlots;           // entries per wave per chunk
constexpr int64_t kGroup = (int64_t)kWaves * kChunk;  // entries per block per reservation
// Slice size and grid of remap: many small slices balance the uneven cost
// of routing (segments differ in operation count) better than one slice
// per resident block, but every block costs a reservation round trip, so a
// block takes about kBlockEntries entries, or fewer (down to
// kMinBlockEntries) while that leaves CUs idle.  The count is on the
// device: the grid is sized for the capacity and surplus blocks leave at
// once.
constexpr int64_t kBlockEntries = 4096;
constexpr int64_t kMinBlockEntries = 64;
constexpr int kRemapBlocksPerCU = 128;               // grid cap; larger deltas give each block more groups
constexpr int kRemapFillPerCU = 5;                 // blocks per CU that keep the chip busy

// Whole chunk inside one segment of kNd dimensions: each
// operation is loaded once (scalar registers) and tested against all slots,
// whose coordinates stay in registers.  The counting pass only tests
// containment; the writing pass ravels the contained coordinates.
template <bool kWrite, int kNd>
__device__ __forceinline__ void route_chunk(const PlanView& pl, const RankSlice& out, int lane,
                                            const SegInfo& sg, const int64_t* x, const uint16_t* y,
                                            const uint32_t (*u)[DTE_MAX_DIMS], int& runv,
                                            int64_t basev)
{
    for (int32_t k = sg.k0; k < sg.k1; ++k) {
        const DevOp o = load_op(pl.ops, k);
        const int r = o.rank - out.first;
        if (r < 0 || r >= out.count) continue;
        int run = __builtin_amdgcn_readlane(runv, r);
        int64_t* const off = out.off[r];
        uint16_t* const val = out.val[r];
        const int64_t cap = out.cap[r];
        const int64_t base = kWrite ? readlane64(basev, r) : 0;
#pragma unroll
        for (int j = 0; j < kRemapSlots; ++j) {
            const bool in = x[j] >= 0 && inside<kNd>(o, u[j]);
            const uint64_t b = __ballot(in);
            if (kWrite && in) {
                const int64_t pos = base + run + lane_prefix(b);
                if (pos < cap) {
                    off[pos] = ravel<kNd>(o, u[j]);
                    val[pos] = y[j];
                }
            }
            run += __popcll(b);
        }
        if (lane == r) runv = run;
    }
}

template <bool kWrite, int kNd>
__device__ __forceinline__ void route_chunk_in(const PlanView& pl, const RankSlice& out, int lane,
                                               const SegInfo& sg, const int64_t* x,
                                               const uint16_t* y, int& runv, int64_t basev)
{
    uint32_t u[kRemapSlots][DTE_MAX_DIMS];
#pragma unroll
    for (int j = 0; j < kRemapSlots; ++j) unravel<kNd>((uint32_t)(x[j] - sg.lo), kNd, sg.shape, u[j]);
    route_chunk<kWrite, kNd>(pl, out, lane, sg, x, y, u, runv, basev);
}

// Load the chunk of entries [c0, c1) (empty when c0 >= c1) into eight
// slots per lane; offsets outside the plan become -1 (ignored).
__device__ __forceinline__ void load_chunk(const PlanView& pl, const int64_t* __restrict__ idx,
                                           const uint16_t* __restrict__ val, int64_t c0,
                                           int64_t c1, int lane, int64_t* x, uint16_t* y)
{
    if (c0 >= c1) {
#pragma unroll
        for (int j = 0; j < kRemapSlots; ++j) {
            x[j] = -1;
            y[j] = 0;
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < kRemapSlots; ++j) {     // all loads of the chunk in flight
        int64_t e = c0 + j * 64 + lane;
        const bool ok = e < c1;
        e = ok ? e : c0;
        x[j] = idx[e];
        y[j] = val[e];
        x[j] = (ok && x[j] >= 0 && x[j] < pl.total) ? x[j] : -1;   // outside: ignored
    }
}

// Route a loaded chunk: counting pass (kWrite == false) or writing pass.
// Wave-uniform.
template <bool kWrite>
__device__ __forceinline__ void route_loaded(const PlanView& pl, const RankSlice& out, int lane,
                                             const int64_t* x, const uint16_t* y, int& runv,
                                             int64_t basev, SegInfo& cache)
{
    // does one segment hold the whole chunk?
    uint64_t any = 0;
    int64_t i0 = 0;
#pragma unroll
    for (int j = kRemapSlots - 1; j >= 0; --j) {
        const uint64_t b = __ballot(x[j] >= 0);
        if (b) {
            any = b;
            i0 = readlane64(x[j], __builtin_ctzll(b));
        }
    }
    if (any == 0) return;
    if (!(i0 >= cache.lo && i0 < cache.hi)) cache = find_segment(pl, i0);
    bool inside = true;
#pragma unroll
    for (int j = 0; j < kRemapSlots; ++j)
        inside = inside && (x[j] < 0 || (x[j] >= cache.lo && x[j] < cache.hi));
    const bool one = __ballot(!inside) == 0;
    // matrices and vectors (nearly every segment) get straight-line code
    if (one && cache.nd == 2) {
        route_chunk_in<kWrite, 2>(pl, out, lane, cache, x, y, runv, basev);
    } else if (one && cache.nd == 1) {
        route_chunk_in<kWrite, 1>(pl, out, lane, cache, x, y, runv, basev);
    } else {
#pragma unroll 1
        for (int j = 0; j < kRemapSlots; ++j)
            route_slot<kWrite>(pl, out, lane, x[j], y[j], runv, basev, cache);
    }
}

// G blocks take part (see kBlockEntries).  Block b < G owns entries
// [total b / G, total (b+1) / G), both ends rounded down to whole groups
// (kGroup: one chunk per wave) when the delta has at least two groups per
// block, else to whole chunks when it has four chunks per block (the last
// block ends at total).  Per group, each wave loads its chunk into
// registers once, counts its outputs per rank, the block reserves bucket
// space with one atomicAdd per touched rank, and each wave writes from the
// same registers after the outputs of waves 0..w-1.
__global__ __launch_bounds__(kBlock) void remap_kernel(PlanView pl, const int64_t* __restrict__ idx,
                                                       const uint16_t* __restrict__ val,
                                                       const int64_t* __restrict__ count,
                                                       int64_t in_capacity, RankSlice out,
                                                       int64_t* __restrict__ rank_count,
                                                       int64_t fill)
{
    __shared__ int s_cnt[kWaves][kRanksPerLaunch];
    __shared__ int64_t s_base[kRanksPerLaunch];

    int64_t total = *count;
    if (total > in_capacity) total = in_capacity;
    if (total < 0) total = 0;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    // slices start on group (else chunk) boundaries when each block gets
    // several: no group is left partly empty, and since extract writes each
    // wave's entries in ascending runs of hundreds to thousands, a chunk
    // then usually lies in one run (one segment); small deltas are split
    // evenly instead
    // blocks in use: about kBlockEntries entries each, more (at least
    // kMinBlockEntries each) up to `fill` blocks, at most the grid
    int64_t g = (total + kBlockEntries - 1) / kBlockEntries;
    const int64_t gmin = (total + kMinBlockEntries - 1) / kMinBlockEntries;
    const int64_t gfill = gmin < fill ? gmin : fill;
    g = g > gfill ? g : gfill;
    g = g < 1 ? 1 : (g > (int64_t)gridDim.x ? (int64_t)gridDim.x : g);
    if ((int64_t)blockIdx.x >= g) return;
    const int64_t align = total >= g * 2 * kGroup ? kGroup : (total >= g * 4 * kChunk ? kChunk : 1);
    const int64_t lo = total * blockIdx.x / g / align * align;
    const int64_t hi = blockIdx.x + 1 == g ? total : total * (blockIdx.x + 1) / g / align * align;
    SegInfo cache{};
    for (int64_t g0 = lo; g0 < hi; g0 += kGroup) {     // block-uniform trip count
        int64_t x[kRemapSlots];
        uint16_t y[kRemapSlots];
        const int64_t c0 = g0 + (int64_t)wave * kChunk;
        load_chunk(pl, idx, val, c0, c0 + kChunk < hi ? c0 + kChunk : hi, lane, x, y);
        int runv = 0;                                   // lane r: outputs for rank first + r
        route_loaded<false>(pl, out, lane, x, y, runv, 0, cache);
        if (lane < kRanksPerLaunch) s_cnt[wave][lane] = lane < out.count ? runv : 0;
        __syncthreads();
        if (wave == 0 && lane < out.count) {
            int64_t n = 0;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) n += s_cnt[w][lane];
            s_base[lane] = n > 0 ? (int64_t)atomicAdd(reinterpret_cast<unsigned long long*>(
                                                          &rank_count[out.first + lane]),
                                                      (unsigned long long)n)
                                 : 0;
        }
        __syncthreads();
        int64_t basev = 0;
        if (lane < out.count) {
            basev = s_base[lane];
            for (int w = 0; w < wave; ++w) basev += s_cnt[w][lane];
        }
        runv = 0;
        route_loaded<true>(pl, out, lane, x, y, runv, basev, cache);
        __syncthreads();                                // s_cnt and s_base are reused
    }
}

constexpr int kApplyUnroll = 8;
constexpr int64_t kDenseApply = 64;
constexpr int64_t kCachedApplyBytes = (int64_t)1 << 30;

__global__ __launch_bounds__(kBlock) void apply_kernel(ApplySlice s,
                                                      const int64_t* __restrict__ rank_count)
{
    const int64_t nthreads = (int64_t)gridDim.x * kBlock;
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (int r = 0; r < s.count; ++r) {
        int64_t n = rank_count[s.first + r];
        if (n > s.cap[r]) n = s.cap[r];
        const int64_t* off = s.off[r];
        const uint16_t* val = s.val[r];
        uint16_t* shard = s.shard[r];
        const int64_t numel = s.numel[r];
        // a rank that receives more than one entry per kDenseApply shard
        // elements, or whose shard is larger than kCachedApplyBytes, takes
        // non-temporal stores: sparse updates of a shard that the caches
        // can hold gain from their write-back, denser ones and larger
        // shards measured faster without it
        const bool stream = n * kDenseApply > numel || numel * 2 > kCachedApplyBytes;
        for (int64_t e0 = t; e0 < n; e0 += nthreads * kApplyUnroll) {
            int64_t j[kApplyUnroll];
            uint16_t v[kApplyUnroll];
#pragma unroll
            for (int k = 0; k < kApplyUnroll; ++k) {
                const int64_t e = e0 + k * nthreads;
                j[k] = e < n ? off[e] : -1;
                v[k] = e < n ? val[e] : (uint16_t)0;
            }
            if (stream) {
#pragma unroll
                for (int k = 0; k < kApplyUnroll; ++k)
                    if (j[k] >= 0 && j[k] < numel) __builtin_nontemporal_store(v[k], shard + j[k]);
            } else {
#pragma unroll
                for (int k = 0; k < kApplyUnroll; ++k)
                    if (j[k] >= 0 && j[k] < numel) shard[j[k]] = v[k];
            }
        }
    }
}

// Blocks of `kernel` that fit on one CU at once (register- and LDS-bound),
// so that a grid of cus * resident blocks runs in a single round: a grid of
// equal slices that needs a second, partial round of blocks leaves most of
// the chip idle during that round.
template <typename Kernel>
int resident_blocks(Kernel kernel)
{
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, 0) != hipSuccess || n < 1)
        n = 1;
    return n;
}

}  // namespace

hipError_t launch_zero_i64(int64_t* p, int64_t n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(zero_i64_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                       p, n);
    return hipGetLastError();
}

hipError_t launch_remap(const PlanView& plan, const int64_t* idx, const uint16_t* val,
                        const int64_t* count, int64_t in_capacity, const RankSlice& out,
                        int64_t* rank_count, int cus, hipStream_t stream)
{
    if (in_capacity <= 0) return hipSuccess;
    // the most blocks the kernel can use for in_capacity entries (its rule
    // for G with total = in_capacity)
    const int64_t fill = (int64_t)cus * kRemapFillPerCU;
    int64_t blocks = (in_capacity + kBlockEntries - 1) / kBlockEntries;
    const int64_t gmin = (in_capacity + kMinBlockEntries - 1) / kMinBlockEntries;
    blocks = blocks > (gmin < fill ? gmin : fill) ? blocks : (gmin < fill ? gmin : fill);
    if (blocks > (int64_t)cus * kRemapBlocksPerCU) blocks = (int64_t)cus * kRemapBlocksPerCU;
    const dim3 grid((unsigned)blocks);
    hipLaunchKernelGGL(remap_kernel, grid, dim3(kBlock), 0, stream, plan, idx, val, count,
                       in_capacity, out, rank_count, fill);
    return hipGetLastError();
}

hipError_t launch_apply(const ApplySlice& s, const int64_t* rank_count, int cus,
                        hipStream_t stream)
{
    static const int per_cu = resident_blocks(apply_kernel);
    const dim3 grid((unsigned)(cus * per_cu));
    hipLaunchKernelGGL(apply_kernel, grid, dim3(kBlock), 0, stream, s, rank_count);
    return hipGetLastError();
}

}  // namespace dte
