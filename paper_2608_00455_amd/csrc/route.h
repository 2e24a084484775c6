// Device-side routing of delta entries through a transfer plan (paper
// sec. 4.2.2): segment lookup, unravel (eq. canonical_unravel), containment
// and ravel (eq. receiver_local_remapping).  Shared by the remap kernel and
// the extract kernel's routing flush; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dte_internal.h"

namespace dte {
namespace rt {

__device__ __forceinline__ int lane_prefix(uint64_t mask)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Containment a_s <= u < a_s + e of coordinate u in operation o, without
// branches (u < a_s wraps to a large value).  kNd > 0: the segment's
// dimension count, known at compile time; kNd == 0: o.ndim (wave-uniform).
template <int kNd>
__device__ __forceinline__ bool inside(const DevOp& o, const uint32_t* u)
{
    bool in = true;
#pragma unroll
    for (int d = 0; d < DTE_MAX_DIMS; ++d)
        if (kNd > 0 ? d < kNd : d < o.ndim) in = in & (u[d] - o.src_origin[d] < o.extent[d]);
    return in;
}

// Receiver offset of a contained coordinate: u - a_s + a_r raveled over the
// receiver view n_r, plus the view's base (eq. receiver_local_remapping).
template <int kNd>
__device__ __forceinline__ int64_t ravel(const DevOp& o, const uint32_t* u)
{
    uint64_t j = 0;
#pragma unroll
    for (int d = 0; d < DTE_MAX_DIMS; ++d)
        if (kNd > 0 ? d < kNd : d < o.ndim)
            j = j * o.dst_shape[d] + (uint32_t)(u[d] - o.src_origin[d] + o.dst_origin[d]);
    return o.dst_base + (int64_t)j;
}

__device__ __forceinline__ int64_t readlane64(int64_t x, int lane)
{
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)x >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Wave-uniform description of the current segment (scalar registers).
struct SegInfo {
    int64_t lo, hi;      // flat range [lo, hi); empty before the first lookup
    int32_t seg, k0, k1; // operations [k0, k1)
    int32_t nd;          // dimensions of the segment's shape
    uint32_t shape[DTE_MAX_DIMS];
};

// Segment holding the uniform flat offset i0 (0 <= i0 < total).
__device__ __forceinline__ SegInfo find_segment(const PlanView& pl, int64_t i0)
{
    int32_t s = __builtin_amdgcn_readfirstlane(pl.lookup[i0 >> pl.shift]);
    while (readlane64(pl.seg_begin[s + 1], 0) <= i0) ++s;
    SegInfo g;
    g.lo = readlane64(pl.seg_begin[s], 0);
    g.hi = readlane64(pl.seg_begin[s + 1], 0);
    g.seg = s;
    g.k0 = __builtin_amdgcn_readfirstlane(pl.seg_ops[s]);
    g.k1 = __builtin_amdgcn_readfirstlane(pl.seg_ops[s + 1]);
    g.nd = __builtin_amdgcn_readfirstlane(pl.seg_ndim[s]);
#pragma unroll
    for (int d = 0; d < DTE_MAX_DIMS; ++d)
        g.shape[d] = __builtin_amdgcn_readfirstlane(pl.seg_shape[(int64_t)s * DTE_MAX_DIMS + d]);
    return g;
}

// One operation with every field made wave-uniform (scalar registers).
__device__ __forceinline__ DevOp load_op(const DevOp* ops, int32_t k)
{
    const uint32_t* w = reinterpret_cast<const uint32_t*>(ops + k);
    DevOp o;
    uint32_t* d = reinterpret_cast<uint32_t*>(&o);
#pragma unroll
    for (int i = 0; i < (int)(sizeof(DevOp) / 4); ++i) d[i] = __builtin_amdgcn_readfirstlane(w[i]);
    return o;
}

// Unravel a segment-local offset over a row-major shape of nd dimensions
// (eq. canonical_unravel); kNd as for `inside` (kNd == 0: nd).
template <int kNd>
__device__ __forceinline__ void unravel(uint32_t li, int nd, const uint32_t* shape, uint32_t* u)
{
#pragma unroll
    for (int d = DTE_MAX_DIMS - 1; d >= 0; --d) {
        if (kNd > 0 ? d < kNd : d < nd) {
            if (d == 0) {
                u[0] = li;
            } else {
                const uint32_t q = li / shape[d];
                u[d] = li - q * shape[d];
                li = q;
            }
        } else {
            u[d] = 0;
        }
    }
}

// Route one slot lane by lane in groups sharing a segment (used when a
// chunk spans several segments).  Counters: lane r of `runv` holds the
// running count of rank first + r, lane r of `basev` the reserved bucket
// start.  kWrite == false counts outputs; kWrite == true writes them.
// kShapeRegs: unravel over the shape cached in `cache` (else re-read it,
// which needs fewer registers).
template <bool kWrite, bool kShapeRegs = true>
__device__ __forceinline__ void route_slot(const PlanView& pl, const RankSlice& out, int lane,
                                           int64_t i, uint16_t v, int& runv, int64_t basev,
                                           SegInfo& cache)
{
    bool pending = i >= 0;
    uint64_t pmask = __ballot(pending);
    while (pmask != 0) {
        const int src = __builtin_ctzll(pmask);
        const int64_t i0 = readlane64(i, src);
        if (!(i0 >= cache.lo && i0 < cache.hi)) cache = find_segment(pl, i0);
        const bool mine = pending && i >= cache.lo && i < cache.hi;
        pending = pending && !mine;
        pmask = __ballot(pending);
        uint32_t u[DTE_MAX_DIMS];
        if (kShapeRegs)
            unravel<0>((uint32_t)(i - cache.lo), cache.nd, cache.shape, u);
        else
            unravel<0>((uint32_t)(i - cache.lo),
                       __builtin_amdgcn_readfirstlane(pl.seg_ndim[cache.seg]),
                       pl.seg_shape + (int64_t)cache.seg * DTE_MAX_DIMS, u);
        for (int32_t k = cache.k0; k < cache.k1; ++k) {
            const DevOp o = load_op(pl.ops, k);
            const int r = o.rank - out.first;
            if (r < 0 || r >= out.count) continue;
            const bool in = mine && inside<0>(o, u);
            const uint64_t b = __ballot(in);
            if (b == 0) continue;
            const int start = __builtin_amdgcn_readlane(runv, r);
            if (lane == r) runv += __popcll(b);
            if (kWrite) {
                int64_t* const off = out.off[r];
                uint16_t* const val = out.val[r];
                const int64_t cap = out.cap[r];
                const int64_t pos = readlane64(basev, r) + start + lane_prefix(b);
                if (in && pos < cap) {
                    off[pos] = ravel<0>(o, u);
                    val[pos] = v;
                }
            }
        }
    }
}

}  // namespace rt
}  // namespace dte
