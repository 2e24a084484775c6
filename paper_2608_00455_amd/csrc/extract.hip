// Delta extraction for gfx950: AdamW inversion (paper sec. 3.1,
// eq. adamw_inverse), BF16 quantisation and bit comparison (sec. 3.2.1,
// eq. canonical_delta_detection) and stream compaction of the changed
// elements, fused in one streaming pass over theta, m, v.
//
// Design (HBM-bound: 12 bytes read per element, ~10 bytes written per
// changed element):
//  - persistent grid (3 blocks of 4 waves per CU); each block owns one
//    contiguous range of 2048-element tiles and its waves take every fourth
//    tile of it (so entries leave each wave as local, ascending runs);
//    a wave loads eight float4 of p, m and v per lane, i.e. 24 16-byte
//    non-temporal loads in flight per lane, which is what keeps the HBM
//    queues full at this occupancy;
//  - proof of "unchanged" before exact arithmetic: with DECAY == 1 the
//    reconstruction is ph = RN(p + u), where u has the sign of m and
//    |u| <= B; B comes from the hardware square root and reciprocal (about
//    1 ulp each), inflated by 2^-16, plus 2^-126; RN and BF16 rounding are
//    monotone, so if RN(p + sign(m) B) has the BF16 pattern of p, so has ph.
//    (DECAY != 1: the same interval is pushed through the division with
//    bracketing reciprocals of DECAY.)  Lanes without that proof
//    (candidates, about as many as the changed elements) queue
//    (p, m, v, position) in LDS; a wave evaluates 64 queued candidates at a
//    time with the correctly rounded inverse.  The result is bit-identical
//    to evaluating every element exactly.  When theta_hat is requested every
//    element takes the exact path;
//  - the change predicate of 64 elements is one ballot; a lane's staging
//    slot is the running count plus mbcnt within the ballot; changed entries
//    (packed 32-bit position + BF16 value) are staged per wave in LDS and a
//    wave reserves global output space with one atomicAdd on the 64-bit
//    cursor per flush of its staging area (1024 entries), then writes the
//    entries out coalesced.  No block-wide barrier anywhere; the number of
//    atomics is bounded by entries / 1024 + waves.
#include <hip/hip_runtime.h>

#include "dte_internal.h"

#pragma clang fp contract(off)

namespace dte {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kVec = 8;                       // float4 per lane per array per tile
constexpr int kSlots = 4 * kVec;              // elements per lane per tile
constexpr int kWaveTile = 64 * kSlots;        // 1024 elements per wave tile
constexpr int kWaveStage = 1024;              // staged output entries per wave (6 bytes each)
constexpr int kQueue = 128;                   // queued candidates per wave (16 bytes each)
constexpr int kBlocksPerCU = 3;               // 3 waves per SIMD (VGPR-bound), 32 KB LDS

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
    const float q = __builtin_fabsf(num) * __builtin_amdgcn_rcpf(den);
    const float b = __builtin_fmaf(q, 1.0000153f, 0x1p-126f);   // NaN stays NaN
    const float hi = p + __builtin_copysignf(b, m);
    const uint32_t up = __float_as_uint(p), uh = __float_as_uint(hi);
    const uint32_t rp = up + 0x7FFFu + ((up >> 16) & 1u);
    const uint32_t rh = uh + 0x7FFFu + ((uh >> 16) & 1u);
    if (kDecayOne) return (rp ^ rh) < 0x10000u;
    const float x0 = p * a.rd_lo, x1 = p * a.rd_hi, x2 = hi * a.rd_lo, x3 = hi * a.rd_hi;
    const float mn = __builtin_fminf(__builtin_fminf(x0, x1), __builtin_fminf(x2, x3));
    const float mx = __builtin_fmaxf(__builtin_fmaxf(x0, x1), __builtin_fmaxf(x2, x3));
    const uint32_t un = __float_as_uint(mn), ux = __float_as_uint(mx);
    const uint32_t rn = un + 0x7FFFu + ((un >> 16) & 1u);
    const uint32_t rx = ux + 0x7FFFu + ((ux >> 16) & 1u);
    return (rp ^ rn) < 0x10000u && (rp ^ rx) < 0x10000u && (mn == mn) && (mx == mx) && (hi == hi);
}

// Exact inverse and change test of one element (sec. 3.1 / 3.2.1).
template <bool kDecayOne>
__device__ __forceinline__ float exact_prev(float p, float m, float v, const ExtractParams& a)
{
    const float u = step_term(m, v, a.lrb1, a.rbc2, a.eps);
    const float num = p + u;
    return kDecayOne ? num : num / a.decay;
}

constexpr int kTileBits = __builtin_ctz(kWaveTile);
static_assert((1 << kTileBits) == kWaveTile, "wave tile must be a power of two");
// Per-wave LDS areas.  Keys are (wave iteration << kTileBits) | element in
// the tile; the wave's tiles are t_first + iteration * nwaves.
struct WaveStage {
    uint32_t* key;    // output staging: changed entries awaiting a flush
    uint16_t* val;
    float* qp;        // candidate queue: elements without an "unchanged" proof
    float* qm;
    float* qv;
    uint32_t* qkey;
    int64_t t_first;
    int64_t nwaves;
};

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Copy a wave's `staged` LDS entries to the reserved global range.
__device__ void flush_wave(const ExtractParams& a, const WaveStage& st, int staged, int lane)
{
    wave_sync();   // every lane's LDS stores visible to the other lanes
    unsigned long long base = 0;
    if (lane == 0)
        base = atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor),
                         (unsigned long long)staged);
    base = __shfl(base, 0);
    for (int i = lane; i < staged; i += 64) {
        const int64_t pos = (int64_t)base + i;
        if (pos < a.capacity) {
            const uint32_t key = st.key[i];
            const int64_t t = st.t_first + (int64_t)(key >> kTileBits) * st.nwaves;
            a.out_idx[pos] = a.index_base + t * kWaveTile + (key & (kWaveTile - 1));
            a.out_val[pos] = st.val[i];
        }
    }
    wave_sync();   // the staging area is rewritten next: finish these reads first
}

// Stage one ballot of changed entries (at most 64), flushing first when the
// staging area would overflow.  Wave-uniform control flow.
__device__ __forceinline__ void stage_changed(const ExtractParams& a, const WaveStage& st,
                                              int& staged, int lane, bool changed,
                                              uint32_t key, uint16_t val)
{
    const uint64_t k = __ballot(changed);
    if (k == 0) return;
    const int cnt = __popcll(k);
    if (staged + cnt > kWaveStage) {
        flush_wave(a, st, staged, lane);
        staged = 0;
    }
    if (changed) {
        const int pos = staged + lane_prefix(k);
        st.key[pos] = key;
        st.val[pos] = val;
    }
    staged += cnt;
}

// Exact inverse of every queued candidate, 64 per pass; changed ones are
// staged.  Empties the queue.
template <bool kDecayOne>
__device__ void drain_queue(const ExtractParams& a, const WaveStage& st, int& queued, int& staged,
                            int lane)
{
    wave_sync();
    for (int base = 0; base < queued; base += 64) {
        const int i = base + lane;
        bool changed = false;
        uint32_t key = 0;
        uint16_t bn = 0;
        if (i < queued) {
            const float p = st.qp[i];
            const float ph = exact_prev<kDecayOne>(p, st.qm[i], st.qv[i], a);
            bn = (uint16_t)bf16_bits(p);
            changed = bf16_bits(ph) != bn;
            key = st.qkey[i];
        }
        stage_changed(a, st, staged, lane, changed, key, bn);
    }
    queued = 0;
    wave_sync();
}

// One wave tile of kWaveTile elements starting at element t0 of the range.
// kFull: the tile lies inside [0, n) (no per-element bounds tests).
template <bool kFull, bool kVecLoads>
__device__ __forceinline__ void load_tile(const ExtractParams& a, int64_t t0, int lane,
                                          f32x4* P, f32x4* M, f32x4* V)
{
    const float* tp = a.p + t0;
    const float* tm = a.m + t0;
    const float* tv = a.v + t0;
    const int64_t rem = a.n - t0;
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
}

template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev>
__device__ __forceinline__ void process_tile(const ExtractParams& a, int64_t t0, int lane,
                                             int& staged, int& queued, const WaveStage& st,
                                             uint32_t iter, const f32x4* P, const f32x4* M,
                                             const f32x4* V)
{
    const int64_t rem = a.n - t0;
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int off = (j * 64 + lane) * 4;
        f32x4 prev;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float p = P[j][c];
            const bool in = kFull || (off + c < rem);
            const uint32_t key = (iter << kTileBits) | (uint32_t)(off + c);
            if (kWritePrev) {
                // theta_hat requested: the exact path for every element
                const float ph = exact_prev<kDecayOne>(p, M[j][c], V[j][c], a);
                prev[c] = ph;
                const uint32_t bn = bf16_bits(p);
                stage_changed(a, st, staged, lane, in && bf16_bits(ph) != bn, key, (uint16_t)bn);
            } else {
                const bool cand = in && !proven_unchanged<kDecayOne>(p, M[j][c], V[j][c], a);
                const uint64_t ck = __ballot(cand);
                if (ck != 0) {
                    const int cnt = __popcll(ck);
                    if (queued + cnt > kQueue) drain_queue<kDecayOne>(a, st, queued, staged, lane);
                    if (cand) {
                        const int pos = queued + lane_prefix(ck);
                        st.qp[pos] = p;
                        st.qm[pos] = M[j][c];
                        st.qv[pos] = V[j][c];
                        st.qkey[pos] = key;
                    }
                    queued += cnt;
                }
            }
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
}

// Wave tiles [first, last) of the range; kFull: each lies inside [0, n).
template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev>
__global__ __launch_bounds__(kBlock) void extract_kernel(ExtractParams a, int64_t first,
                                                         int64_t last)
{
    __shared__ uint32_t s_key[kWaves][kWaveStage];
    __shared__ uint16_t s_val[kWaves][kWaveStage];
    __shared__ float s_qp[kWaves][kQueue];
    __shared__ float s_qm[kWaves][kQueue];
    __shared__ float s_qv[kWaves][kQueue];
    __shared__ uint32_t s_qkey[kWaves][kQueue];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    // block b owns the contiguous tile range [b per, (b+1) per); its waves
    // take every kWaves-th tile of it, so the four waves of a block stream
    // neighbouring tiles and each wave's output is a local, ascending run
    const int64_t per = (last - first + gridDim.x - 1) / gridDim.x;
    const int64_t b_first = first + (int64_t)blockIdx.x * per;
    const int64_t b_last = (b_first + per < last) ? b_first + per : last;
    int64_t t = b_first + wave;
    int staged = 0;
    const WaveStage st{s_key[wave], s_val[wave], s_qp[wave], s_qm[wave], s_qv[wave],
                       s_qkey[wave], t, kWaves};
    uint32_t iter = 0;
    int queued = 0;
    for (; t < b_last; t += kWaves) {
        f32x4 P[kVec], M[kVec], V[kVec];
        load_tile<kFull, kVecLoads>(a, t * kWaveTile, lane, P, M, V);
        process_tile<kFull, kVecLoads, kDecayOne, kWritePrev>(a, t * kWaveTile, lane, staged,
                                                             queued, st, iter++, P, M, V);
    }
    if (queued > 0) drain_queue<kDecayOne>(a, st, queued, staged, lane);
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
