// Delta extraction for gfx950: AdamW inversion (paper sec. 3.1,
// eq. adamw_inverse), BF16 quantisation and bit comparison (sec. 3.2.1,
// eq. canonical_delta_detection) and stream compaction of the changed
// elements, fused in one streaming pass over theta, m, v.
//
// Design (HBM-bound: 12 bytes read per element, ~10 bytes written per
// changed element):
//  - persistent grid; every wave walks its own 1024-element tiles (four
//    float4 of p, m and v per lane: twelve 16-byte non-temporal loads in
//    flight per lane);
//  - proof of "unchanged" before exact arithmetic: with DECAY == 1 the
//    reconstruction is ph = RN(p + u), where u has the sign of m and
//    |u| <= B, B computed from the hardware square root and reciprocal
//    (about 1 ulp each) and inflated by 2^-16; RN and BF16 rounding are
//    monotone, so if RN(p + sign(m) B) has the BF16 pattern of p, so has ph.
//    (DECAY != 1: the same interval is pushed through the division with
//    bracketing reciprocals of DECAY.)  Only lanes without that proof run the
//    correctly rounded sqrt / divide of the exact inverse; the result is
//    bit-identical to evaluating every element exactly.  When theta_hat is
//    requested every element takes the exact path;
//  - each element slot's change predicate is a wave64 ballot; a lane's
//    staging slot is the popcount of the earlier ballots plus mbcnt in its
//    own; changed entries are staged per wave in LDS (1024 entries) and a
//    wave reserves global output space with one atomicAdd on the 64-bit
//    cursor per flush of its staging area, then copies the entries out
//    coalesced.  No block-wide barrier in the main loop.  The number of
//    atomics is bounded by entries / 1024 + waves.
#include <hip/hip_runtime.h>

#include "dte_internal.h"

#pragma clang fp contract(off)

namespace dte {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kVec = 4;                       // float4 per lane per array per tile
constexpr int kSlots = 4 * kVec;              // elements per lane per tile
constexpr int kWaveTile = 64 * kSlots;        // 1024 elements per wave tile
constexpr int kWaveStage = kWaveTile;         // staging entries per wave (>= one tile)
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

// Same rounding without the NaN rule (used where NaN is excluded).
__device__ __forceinline__ uint32_t bf16_raw(float x)
{
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
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

// True only if b(ph) == b(p) is proven without the exact inverse (see the
// header).  B bounds |u| from above: hardware sqrt / reciprocal (about one
// ulp each) and two roundings, covered by the factor 1 + 2^-16; flushed or
// overflowing intermediates make B non-finite or too large, never too small,
// except a reciprocal flushed to zero, covered by the floor 2^-126 (a |u|
// below it cannot move a |p| >= 2^-100, and a smaller |p| fails the test).
template <bool kDecayOne>
__device__ __forceinline__ bool proven_unchanged(float p, float m, float v, const ExtractParams& a)
{
    const float num = a.lrb1 * m;
    const float vh = v * a.rbc2;
    const float den = __builtin_amdgcn_sqrtf(vh) + a.eps;
    const float bound = __builtin_fabsf(num) * __builtin_amdgcn_rcpf(den) * 1.0000153f;
    const bool finite = bound < __builtin_inff();           // false for NaN
    const float b = __builtin_fmaxf(bound, 0x1p-126f);
    const float lo = p + __builtin_copysignf(0.0f, m);      // RN(p + u) for u = +-0
    const float hi = p + __builtin_copysignf(b, m);         // RN(p + u) for |u| = B
    const uint32_t bp = bf16_raw(p);
    if (kDecayOne)
        return finite && (p == p) && bf16_raw(lo) == bp && bf16_raw(hi) == bp;
    // ph = RN(n / DECAY), monotone in n; bracket 1/DECAY by rd_lo <= 1/DECAY <= rd_hi
    const float x0 = lo * a.rd_lo, x1 = lo * a.rd_hi, x2 = hi * a.rd_lo, x3 = hi * a.rd_hi;
    const float mn = __builtin_fminf(__builtin_fminf(x0, x1), __builtin_fminf(x2, x3));
    const float mx = __builtin_fmaxf(__builtin_fmaxf(x0, x1), __builtin_fmaxf(x2, x3));
    return finite && (p == p) && (mn == mn) && (mx == mx) && bf16_raw(mn) == bp &&
           bf16_raw(mx) == bp;
}

// Exact inverse and change test of one element (sec. 3.1 / 3.2.1).
template <bool kDecayOne>
__device__ __forceinline__ float exact_prev(float p, float m, float v, const ExtractParams& a)
{
    const float u = step_term(m, v, a.lrb1, a.rbc2, a.eps);
    const float num = p + u;
    return kDecayOne ? num : num / a.decay;
}

struct WaveStage {
    int64_t* idx;     // this wave's kWaveStage entries in LDS
    uint16_t* val;
};

// Copy a wave's `staged` LDS entries to the reserved global range.
__device__ void flush_wave(const ExtractParams& a, const WaveStage& st, int staged, int lane)
{
    // make every lane's LDS stores visible to the other lanes of the wave
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    unsigned long long base = 0;
    if (lane == 0)
        base = atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor),
                         (unsigned long long)staged);
    base = __shfl(base, 0);
    for (int i = lane; i < staged; i += 64) {
        const int64_t pos = (int64_t)base + i;
        if (pos < a.capacity) {
            a.out_idx[pos] = st.idx[i];
            a.out_val[pos] = st.val[i];
        }
    }
    // the staging area is rewritten next: finish these reads first
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One wave tile of kWaveTile elements starting at element t0 of the range.
// kFull: the tile lies inside [0, n) (no per-element bounds tests).
template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev>
__device__ __forceinline__ void extract_wave_tile(const ExtractParams& a, int64_t t0, int lane,
                                                  int& staged, const WaveStage& st)
{
    const float* tp = a.p + t0;
    const float* tm = a.m + t0;
    const float* tv = a.v + t0;
    const int64_t rem = a.n - t0;
    f32x4 P[kVec], M[kVec], V[kVec];
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int off = (j * 64 + lane) * 4;
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
        const int off = (j * 64 + lane) * 4;
        f32x4 prev;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float p = P[j][c];
            bool changed = false;
            if (kWritePrev) {
                const float ph = exact_prev<kDecayOne>(p, M[j][c], V[j][c], a);
                prev[c] = ph;
                changed = bf16_bits(ph) != bf16_bits(p);
            } else {
                const bool cand = !proven_unchanged<kDecayOne>(p, M[j][c], V[j][c], a);
                if (__ballot(cand) != 0) {
                    if (cand) {
                        const float ph = exact_prev<kDecayOne>(p, M[j][c], V[j][c], a);
                        changed = bf16_bits(ph) != bf16_bits(p);
                    }
                }
            }
            if (!kFull) changed = changed && (off + c < rem);
            mask[4 * j + c] = __ballot(changed);
            wave_total += __popcll(mask[4 * j + c]);
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
    }
    if (wave_total == 0) return;

    if (staged + wave_total > kWaveStage) {
        flush_wave(a, st, staged, lane);
        staged = 0;
    }
    int run = staged;
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        const uint64_t k = mask[s];
        if (k != 0) {
            if ((k >> lane) & 1ull) {
                const int pos = run + lane_prefix(k);
                const int e = ((s >> 2) * 64 + lane) * 4 + (s & 3);
                st.idx[pos] = a.index_base + t0 + e;
                st.val[pos] = (uint16_t)bf16_bits(P[s >> 2][s & 3]);
            }
            run += __popcll(k);
        }
    }
    staged += wave_total;
}

// Wave tiles [first, last) of the range; kFull: each lies inside [0, n).
template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev>
__global__ __launch_bounds__(kBlock) void extract_kernel(ExtractParams a, int64_t first,
                                                         int64_t last)
{
    __shared__ int64_t s_idx[kWaves][kWaveStage];
    __shared__ uint16_t s_val[kWaves][kWaveStage];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const WaveStage st{s_idx[wave], s_val[wave]};
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    int staged = 0;
    for (int64_t t = first + (int64_t)blockIdx.x * kWaves + wave; t < last; t += nwaves)
        extract_wave_tile<kFull, kVecLoads, kDecayOne, kWritePrev>(a, t * kWaveTile, lane, staged,
                                                                   st);
    if (staged > 0) flush_wave(a, st, staged, lane);
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
    const int64_t blocks = (last - first + kWaves - 1) / kWaves;
    const dim3 grid((unsigned)(blocks < max_grid ? blocks : max_grid));
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
    const int64_t full = a.n / kWaveTile;
    const int64_t ntiles = (a.n + kWaveTile - 1) / kWaveTile;
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
