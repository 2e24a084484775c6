// Delta extraction for gfx950: AdamW inversion (paper sec. 3.1,
// eq. adamw_inverse), BF16 quantisation and bit comparison (sec. 3.2.1,
// eq. canonical_delta_detection) and stream compaction of the changed
// elements, fused in one streaming pass over theta, m, v.
//
// Design (HBM-bound: 12 bytes read per element, ~10 bytes written per
// changed element):
//  - persistent grid (4 blocks of 256 threads per CU), each block walks
//    4096-element tiles; each thread holds four float4 of p, m and v (twelve
//    16-byte loads in flight per lane, non-temporal: the stream is read once);
//  - the change predicate of each element slot is a wave64 ballot; a lane's
//    output slot is the popcount of the ballots before it plus mbcnt within
//    its ballot; wave totals are combined through LDS (one barrier per tile);
//  - changed entries are staged in LDS (4096 entries); a block reserves
//    global output space with one atomicAdd on the 64-bit cursor per flush
//    of its staging buffer, then copies the staged entries out coalesced.
//    The number of atomics is bounded by (entries / 4096) + blocks.
#include <hip/hip_runtime.h>

#include "dte_internal.h"

#pragma clang fp contract(off)

namespace dte {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kVec = 4;                       // float4 per thread per tile
constexpr int kSlots = 4 * kVec;              // elements per thread per tile
constexpr int kTile = kBlock * kSlots;        // 4096 elements
constexpr int kStage = kTile;                 // staging entries (>= one tile)
constexpr int kBlocksPerCU = 4;               // 40 KB LDS each

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Adaptive step term u = (lrb1*m) / (sqrt(v*rbc2) + eps): four binary32
// operations, each rounded once (sqrt and divide correctly rounded).
__device__ __forceinline__ float step_term(float m, float v, float lrb1, float rbc2, float eps)
{
    const float vh = v * rbc2;
    const float sq = __builtin_sqrtf(vh);
    const float den = sq + eps;
    const float num = lrb1 * m;
    return num / den;
}

// BF16 pattern of x: round to nearest even on the binary32 pattern; any NaN
// gives 0x7FC0.  (For non-NaN x the 32-bit sum cannot wrap.)
__device__ __forceinline__ uint32_t bf16_bits(float x)
{
    const uint32_t u = __float_as_uint(x);
    const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    return (x != x) ? 0x7FC0u : r;
}

__device__ __forceinline__ int lane_prefix(uint64_t mask)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

template <bool kVecLoads>
__device__ __forceinline__ f32x4 load4(const float* base, int64_t e, int64_t n)
{
    f32x4 r = {0.0f, 0.0f, 0.0f, 0.0f};
    if (kVecLoads && e + 3 < n) {
        r = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(base + e));
    } else {
        if (e + 0 < n) r.x = base[e + 0];
        if (e + 1 < n) r.y = base[e + 1];
        if (e + 2 < n) r.z = base[e + 2];
        if (e + 3 < n) r.w = base[e + 3];
    }
    return r;
}

// Copy `staged` LDS entries to the global output at a reserved offset.
// Block-uniform: every thread of the block calls it.
__device__ void flush(const ExtractParams& a, const int64_t* s_idx, const uint16_t* s_val,
                      int64_t* s_base, int staged)
{
    if (threadIdx.x == 0)
        *s_base = (int64_t)atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor),
                                     (unsigned long long)staged);
    __syncthreads();
    const int64_t base = *s_base;
    for (int i = threadIdx.x; i < staged; i += kBlock) {
        const int64_t pos = base + i;
        if (pos < a.capacity) {
            a.out_idx[pos] = s_idx[i];
            a.out_val[pos] = s_val[i];
        }
    }
    __syncthreads();
}

// BF16 pattern without the NaN rule (callers apply it when a NaN is present).
__device__ __forceinline__ uint32_t bf16_raw(float x)
{
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// One 4096-element tile: loads, inversion, change ballots, staging.
// kFull: the whole tile lies inside [0, n) (no per-element bounds tests).
template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev>
__device__ __forceinline__ void extract_tile(const ExtractParams& a, int64_t t0, int tid,
                                             int lane, int wave, int& staged, int& par,
                                             int64_t* s_idx, uint16_t* s_val,
                                             int (*s_tot)[kWaves], int64_t* s_base)
{
    // uniform tile base: 32-bit lane offsets from a scalar base address
    const float* tp = a.p + t0;
    const float* tm = a.m + t0;
    const float* tv = a.v + t0;
    const int64_t rem = a.n - t0;
    f32x4 P[kVec], M[kVec], V[kVec];
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int off = (j * kBlock + tid) * 4;
        if (kFull) {
            P[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(tp + off));
            M[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(tm + off));
            V[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(tv + off));
        } else {
            P[j] = load4<kVecLoads>(tp, off, rem);
            M[j] = load4<kVecLoads>(tm, off, rem);
            V[j] = load4<kVecLoads>(tv, off, rem);
        }
    }

    uint64_t mask[kSlots];
    int wave_total = 0;
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int off = (j * kBlock + tid) * 4;
        f32x4 prev;
        float ph4[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float u = step_term(M[j][c], V[j][c], a.lrb1, a.rbc2, a.eps);
            const float num = P[j][c] + u;
            ph4[c] = kDecayOne ? num : num / a.decay;
            prev[c] = ph4[c];
        }
        if (kWritePrev) {
            if (kFull || (kVecLoads && off + 3 < rem)) {
                __builtin_nontemporal_store(prev, reinterpret_cast<f32x4*>(a.out_prev + t0 + off));
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    if (off + c < rem) a.out_prev[t0 + off + c] = prev[c];
            }
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float ph = ph4[c];
            const float pc = P[j][c];
            bool changed = bf16_raw(ph) != bf16_raw(pc);
            // NaN rule, only for waves that hold a NaN (unordered pair)
            if (__builtin_expect(__ballot(__builtin_isunordered(ph, pc)) != 0, 0))
                changed = bf16_bits(ph) != bf16_bits(pc);
            if (!kFull) changed = changed && (off + c < rem);
            mask[4 * j + c] = __ballot(changed);
            wave_total += __popcll(mask[4 * j + c]);
        }
    }

    if (lane == 0) s_tot[par][wave] = wave_total;
    __syncthreads();
    int wave_off = 0, block_total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        const int c = s_tot[par][w];
        wave_off += (w < wave) ? c : 0;
        block_total += c;
    }
    par ^= 1;
    if (block_total == 0) return;

    if (staged + block_total > kStage) {
        flush(a, s_idx, s_val, s_base, staged);
        staged = 0;
    }
    int run = staged + wave_off;
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        const uint64_t k = mask[s];
        if (k != 0) {
            if ((k >> lane) & 1ull) {
                const int pos = run + lane_prefix(k);
                const int e = ((s >> 2) * kBlock + tid) * 4 + (s & 3);
                s_idx[pos] = a.index_base + t0 + e;
                s_val[pos] = (uint16_t)bf16_bits(P[s >> 2][s & 3]);
            }
            run += __popcll(k);
        }
    }
    staged += block_total;
}

// Tiles [first, last) of the range; kFull: every such tile lies inside [0, n).
template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev>
__global__ __launch_bounds__(kBlock) void extract_kernel(ExtractParams a, int64_t first,
                                                         int64_t last)
{
    __shared__ int64_t s_idx[kStage];
    __shared__ uint16_t s_val[kStage];
    __shared__ int s_tot[2][kWaves];
    __shared__ int64_t s_base;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int staged = 0;
    int par = 0;
    for (int64_t tile = first + blockIdx.x; tile < last; tile += gridDim.x)
        extract_tile<kFull, kVecLoads, kDecayOne, kWritePrev>(
            a, tile * kTile, tid, lane, wave, staged, par, s_idx, s_val, s_tot, &s_base);
    if (staged > 0) flush(a, s_idx, s_val, &s_base, staged);
}

template <bool kVecLoads>
__global__ __launch_bounds__(256) void adamw_forward_kernel(ForwardParams a)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
    for (int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; e < a.n; e += stride) {
        f32x4 P = load4<kVecLoads>(a.p, e, a.n);
        f32x4 M = load4<kVecLoads>(a.m, e, a.n);
        f32x4 V = load4<kVecLoads>(a.v, e, a.n);
        const f32x4 G = load4<kVecLoads>(a.g, e, a.n);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float g = G[c];
            const float m1 = a.b1 * M[c];
            const float m2 = a.omb1 * g;
            const float mt = m1 + m2;
            const float g2 = g * g;
            const float v1 = a.b2 * V[c];
            const float v2 = a.omb2 * g2;
            const float vt = v1 + v2;
            const float u = step_term(mt, vt, a.lrb1, a.rbc2, a.eps);
            const float dp = a.decay * P[c];
            P[c] = dp - u;
            M[c] = mt;
            V[c] = vt;
        }
        if (kVecLoads && e + 3 < a.n) {
            *reinterpret_cast<f32x4*>(a.p + e) = P;
            *reinterpret_cast<f32x4*>(a.m + e) = M;
            *reinterpret_cast<f32x4*>(a.v + e) = V;
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if (e + c < a.n) {
                    a.p[e + c] = P[c];
                    a.m[e + c] = M[c];
                    a.v[e + c] = V[c];
                }
            }
        }
    }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <bool F, bool V, bool D>
void launch_tiles(const ExtractParams& a, int64_t first, int64_t last, int64_t max_grid,
                  hipStream_t s)
{
    if (last <= first) return;
    const dim3 grid((unsigned)(last - first < max_grid ? last - first : max_grid));
    if (a.out_prev)
        hipLaunchKernelGGL((extract_kernel<F, V, D, true>), grid, dim3(kBlock), 0, s, a, first,
                           last);
    else
        hipLaunchKernelGGL((extract_kernel<F, V, D, false>), grid, dim3(kBlock), 0, s, a, first,
                           last);
}

template <bool D>
void launch_all(const ExtractParams& a, bool vec, int64_t max_grid, hipStream_t s)
{
    const int64_t full = a.n / kTile;
    const int64_t ntiles = (a.n + kTile - 1) / kTile;
    if (vec) {
        launch_tiles<true, true, D>(a, 0, full, max_grid, s);       // unguarded body
        launch_tiles<false, true, D>(a, full, ntiles, max_grid, s); // ragged last tile
    } else {
        launch_tiles<false, false, D>(a, 0, ntiles, max_grid, s);   // scalar loads
    }
}

}  // namespace

hipError_t launch_extract(const ExtractParams& a, int cus, hipStream_t stream)
{
    if (a.n <= 0) return hipSuccess;
    const int64_t max_grid = (int64_t)cus * kBlocksPerCU;
    const bool vec = aligned16(a.p) && aligned16(a.m) && aligned16(a.v) &&
                     (a.out_prev == nullptr || aligned16(a.out_prev));
    if (a.decay == 1.0f)
        launch_all<true>(a, vec, max_grid, stream);
    else
        launch_all<false>(a, vec, max_grid, stream);
    return hipGetLastError();
}

hipError_t launch_adamw_forward(const ForwardParams& a, int cus, hipStream_t stream)
{
    if (a.n <= 0) return hipSuccess;
    const int64_t quads = (a.n + 3) / 4;
    const int64_t blocks = (quads + 255) / 256;
    const int64_t want = (int64_t)cus * 8;
    const dim3 grid((unsigned)(blocks < want ? blocks : want));
    const bool vec = aligned16(a.p) && aligned16(a.m) && aligned16(a.v) && aligned16(a.g);
    if (vec)
        hipLaunchKernelGGL(adamw_forward_kernel<true>, grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(adamw_forward_kernel<false>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace dte
