// Receiver-space remap (paper sec. 3.2.2) and direct sparse apply (sec. 3.3,
// eq. direct_sparse_apply) for gfx950.
//
// Remap: every entry (flat trainer offset i, BF16 value) finds its segment
// through a direct-mapped bucket table (bucket = i >> shift holds the
// segment of its first element; a short forward scan finishes the search),
// unravels i - flat_begin over the segment's row-major shape
// (eq. canonical_unravel), and for each operation of the segment tests
// containment a_s <= u < a_s + e and ravels u - a_s + a_r over the
// receiver view (eq. receiver_local_remapping).  Blocks own contiguous
// slices of the entry list; a first pass counts each rank's outputs in LDS,
// one atomicAdd per rank per block reserves bucket space, and a second pass
// writes (offset, value) pairs.
//
// Apply: shard[off] = val, grid-stride over each rank's bucket.
#include <hip/hip_runtime.h>

#include "dte_internal.h"

namespace dte {
namespace {

constexpr int kBlock = 256;
constexpr int kBlocksPerCU = 8;

__global__ void zero_i64_kernel(int64_t* p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

struct Located {
    int32_t seg;        // -1: outside the plan
    uint32_t u[DTE_MAX_DIMS];
};

__device__ __forceinline__ Located locate(const PlanView& pl, int64_t i)
{
    Located r;
    r.seg = -1;
    if (i < 0 || i >= pl.total) return r;
    int32_t s = pl.lookup[i >> pl.shift];
    while (pl.seg_begin[s + 1] <= i) ++s;                    // tiles [0, total)
    uint32_t li = (uint32_t)(i - pl.seg_begin[s]);           // < 2^32 (validated)
    const int nd = pl.seg_ndim[s];
    const uint32_t* shape = pl.seg_shape + (int64_t)s * DTE_MAX_DIMS;
#pragma unroll
    for (int d = DTE_MAX_DIMS - 1; d >= 0; --d) {
        if (d < nd) {
            if (d == 0) {
                r.u[0] = li;
            } else {
                const uint32_t q = li / shape[d];
                r.u[d] = li - q * shape[d];
                li = q;
            }
        } else {
            r.u[d] = 0;
        }
    }
    r.seg = s;
    return r;
}

// Receiver offset of coordinate u under op o, or -1 when u is outside o.
__device__ __forceinline__ int64_t route(const DevOp& o, const uint32_t* u)
{
    int64_t j = 0;
#pragma unroll
    for (int d = 0; d < DTE_MAX_DIMS; ++d) {
        if (d < o.ndim) {
            const uint32_t rel = u[d] - o.src_origin[d];    // wraps when u < a_s
            if (rel >= o.extent[d]) return -1;
            j = j * (int64_t)o.dst_shape[d] + (int64_t)(rel + o.dst_origin[d]);
        }
    }
    return o.dst_base + j;
}

__global__ __launch_bounds__(kBlock) void remap_kernel(PlanView pl, const int64_t* __restrict__ idx,
                                                       const uint16_t* __restrict__ val,
                                                       const int64_t* __restrict__ count,
                                                       int64_t in_capacity, RankSlice out,
                                                       int64_t* __restrict__ rank_count)
{
    __shared__ int s_cnt[kRanksPerLaunch];
    __shared__ int64_t s_base[kRanksPerLaunch];

    int64_t total = *count;
    if (total > in_capacity) total = in_capacity;
    if (total < 0) total = 0;
    const int64_t lo = total * blockIdx.x / gridDim.x;
    const int64_t hi = total * (blockIdx.x + 1) / gridDim.x;
    if (threadIdx.x < kRanksPerLaunch) s_cnt[threadIdx.x] = 0;
    __syncthreads();

    // pass 1: count this block's outputs per rank
    for (int64_t e = lo + threadIdx.x; e < hi; e += kBlock) {
        const Located L = locate(pl, idx[e]);
        if (L.seg < 0) continue;
        for (int32_t k = pl.seg_ops[L.seg]; k < pl.seg_ops[L.seg + 1]; ++k) {
            const DevOp& o = pl.ops[k];
            const int r = o.rank - out.first;
            if (r < 0 || r >= out.count) continue;
            if (route(o, L.u) >= 0) atomicAdd(&s_cnt[r], 1);
        }
    }
    __syncthreads();
    if (threadIdx.x < out.count && s_cnt[threadIdx.x] > 0)
        s_base[threadIdx.x] = (int64_t)atomicAdd(
            reinterpret_cast<unsigned long long*>(&rank_count[out.first + threadIdx.x]),
            (unsigned long long)s_cnt[threadIdx.x]);
    __syncthreads();
    if (threadIdx.x < kRanksPerLaunch) s_cnt[threadIdx.x] = 0;
    __syncthreads();

    // pass 2: write (receiver offset, value)
    for (int64_t e = lo + threadIdx.x; e < hi; e += kBlock) {
        const Located L = locate(pl, idx[e]);
        if (L.seg < 0) continue;
        const uint16_t v = val[e];
        for (int32_t k = pl.seg_ops[L.seg]; k < pl.seg_ops[L.seg + 1]; ++k) {
            const DevOp& o = pl.ops[k];
            const int r = o.rank - out.first;
            if (r < 0 || r >= out.count) continue;
            const int64_t j = route(o, L.u);
            if (j < 0) continue;
            const int64_t pos = s_base[r] + atomicAdd(&s_cnt[r], 1);
            if (pos < out.cap[r]) {
                out.off[r][pos] = j;
                out.val[r][pos] = v;
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void apply_kernel(ApplySlice s,
                                                      const int64_t* __restrict__ rank_count)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (int r = 0; r < s.count; ++r) {
        int64_t n = rank_count[s.first + r];
        if (n > s.cap[r]) n = s.cap[r];
        const int64_t* off = s.off[r];
        const uint16_t* val = s.val[r];
        uint16_t* shard = s.shard[r];
        const int64_t numel = s.numel[r];
        for (int64_t e = t; e < n; e += stride) {
            const int64_t j = off[e];
            if (j >= 0 && j < numel) shard[j] = val[e];
        }
    }
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
    const int64_t want = (int64_t)cus * kBlocksPerCU;
    const int64_t need = (in_capacity + kBlock - 1) / kBlock;
    const dim3 grid((unsigned)(need < want ? need : want));
    hipLaunchKernelGGL(remap_kernel, grid, dim3(kBlock), 0, stream, plan, idx, val, count,
                       in_capacity, out, rank_count);
    return hipGetLastError();
}

hipError_t launch_apply(const ApplySlice& s, const int64_t* rank_count, int cus,
                        hipStream_t stream)
{
    const dim3 grid((unsigned)cus * kBlocksPerCU);
    hipLaunchKernelGGL(apply_kernel, grid, dim3(kBlock), 0, stream, s, rank_count);
    return hipGetLastError();
}

}  // namespace dte
