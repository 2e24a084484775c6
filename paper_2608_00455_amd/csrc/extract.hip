// Delta extraction for gfx950: AdamW inversion (paper sec. 4.1,
// eq. adamw_inverse), BF16 quantisation and bit comparison (sec. 4.2.1,
// eq. canonical_delta_detection) and stream compaction of the changed
// elements, fused in one streaming pass over theta, m, v.
//
// Design (HBM-bound: 12 bytes read per element, ~10 bytes written per
// changed element):
//  - persistent grid of one block of 12 waves per CU (three per SIMD, the
//    VGPR limit; the block holds the CU's whole LDS) over the full tiles,
//    three blocks of 4 waves per CU over ragged ones; each wave owns one
//    contiguous range of 2048-element tiles, ranges ascending with the
//    global wave number, so every wave's entries leave in ascending order;
//    in the unordered call the static ranges leave out the last 1/16 of
//    the full tiles, which blocks then take four tiles per wave at a time
//    from a counter (the CUs do not stream at one rate, and a static split
//    leaves the fast ones idle at the end);
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
//  - the predicate of one float4 slot of the wave (256 consecutive
//    elements) is four ballots; an element's position among the slot's
//    selected elements is the sum of mbcnt over the four ballots (lanes
//    before it) plus its own selected predecessors in the lane, so
//    candidates are queued, and changed entries (packed 32-bit position +
//    BF16 value) staged in LDS, in ascending element order: every wave's
//    output is ascending.  In the unordered call the waves of a block meet
//    every four tiles and, once they hold enough entries, reserve output
//    space for all of them with one atomicAdd on the 64-bit cursor
//    (block_round below); each wave writes its run after those of the waves
//    before it, coalesced.  A wave whose staging area (kWaveStage entries)
//    fills between two meetings flushes exactly kWaveStage entries on its
//    own with one atomicAdd;
//  - ordered mode: the waves of a block still meet every four tiles (a
//    barrier alone), which keeps them in step; each wave writes its
//    flushes to a region of the workspace of its own (no atomics) and,
//    once that is full, to a shared
//    area, recording (position, entries of the wave before it, count,
//    wave); a scan of the wave totals and a copy of the regions and
//    recorded runs then give the entries in ascending offset order
//    (order_scan_kernel, order_copy_kernel below), deterministic whatever
//    the timing of the atomics.
#include <hip/hip_runtime.h>

#include "dte_internal.h"
#include "route.h"

#pragma clang fp contract(off)

namespace dte {
namespace {

// Waves per block: 12 (one block per CU) for full tiles; the ragged-tile
// kernels need more VGPRs than 12 waves per CU leave without spilling, and
// run as 4-wave blocks, three per CU.  Either way 3 waves per SIMD.
template <bool kFull> constexpr int kWavesOf = kFull ? 12 : 4;
constexpr int kWavesPerCU = 12;
constexpr int kVec = 8;                       // float4 per lane per array per tile
constexpr int kSlots = 4 * kVec;              // elements per lane per tile
constexpr int kWaveTile = 64 * kSlots;        // 2048 elements per wave tile
constexpr int kQueue = 256;                   // queued candidates per wave (16 bytes each)
// a float4 slot selects up to 4 x 64 elements at once: they must fit an
// empty candidate queue, and the part left after one flush of the staging
// area must fit the emptied area
static_assert(kQueue >= 4 * 64, "a slot's candidates must fit the queue");
static_assert(kWaveStage >= 4 * 64, "a slot's changed entries must fit after one flush");

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

// The same term in the literal order of eq. adamw_inverse:
// lr * ((m / bc1) / (sqrt(v / bc2) + eps)), six binary32 operations.
__device__ __forceinline__ float step_term_literal(float m, float v, float lr, float bc1, float bc2,
                                                   float eps)
{
    const float mh = m / bc1;
    const float vq = v / bc2;
    const float sq = __builtin_sqrtf(vq);
    const float d = sq + eps;
    const float r = mh / d;
    return lr * r;
}

// BF16 pattern of x: round to nearest even on the binary32 pattern; any NaN
// gives 0x7FC0.  (For non-NaN x the 32-bit sum cannot wrap.)
__device__ __forceinline__ uint32_t bf16_bits(float x)
{
    const uint32_t u = __float_as_uint(x);
    const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    return (x != x) ? 0x7FC0u : r;
}

using rt::lane_prefix;   // set lanes of the mask below this lane

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
//
// Literal order: the same B bounds the literal u when every intermediate of
// both evaluations is a normal number (each then carries one rounding of
// relative error, about ten in all, far inside 2^-16).  The host allows the
// proof only when eps >= 2^-40, lr <= 2^20 and both bias corrections are
// >= 2^-20.  Then d = sqrt(v/bc2) + eps >= 2^-40, so a subnormal v/bc2
// moves d by at most 2^-75 (relative 2^-35); subnormal m/bc1, lrb1*m or
// m/bc1/d move u by at most 2^-125/eps in all, the floor (`floor`, set by
// the host) used instead of 2^-126; |m| <= 2^64 keeps m/bc1 and m/bc1/d
// finite (other elements take the exact path); v*rbc2 is clamped to the
// largest finite value so that it cannot overflow where v/bc2 does not
// (a NaN stays NaN).
template <bool kDecayOne, bool kLit>
__device__ __forceinline__ bool proven_unchanged(float p, float m, float v, const ExtractParams& a)
{
    const float num = a.lrb1 * m;
    float vh = v * a.rbc2;
    if (kLit) vh = vh > 0x1.fffffep127f ? 0x1.fffffep127f : vh;
    const bool in_range = !kLit || (__float_as_uint(m) & 0x7FFFFFFFu) <= 0x5F800000u;
    const float den = __builtin_amdgcn_sqrtf(vh) + a.eps;
    const float q = __builtin_fabsf(num) * __builtin_amdgcn_rcpf(den);
    const float b = __builtin_fmaf(q, 1.0000153f, kLit ? a.floor : 0x1p-126f);   // NaN stays NaN
    const float hi = p + __builtin_copysignf(b, m);
    const uint32_t up = __float_as_uint(p), uh = __float_as_uint(hi);
    const uint32_t rp = up + 0x7FFFu + ((up >> 16) & 1u);
    const uint32_t rh = uh + 0x7FFFu + ((uh >> 16) & 1u);
    if (kDecayOne) return in_range & ((rp ^ rh) < 0x10000u);
    const float x0 = p * a.rd_lo, x1 = p * a.rd_hi, x2 = hi * a.rd_lo, x3 = hi * a.rd_hi;
    const float mn = __builtin_fminf(__builtin_fminf(x0, x1), __builtin_fminf(x2, x3));
    const float mx = __builtin_fmaxf(__builtin_fmaxf(x0, x1), __builtin_fmaxf(x2, x3));
    const uint32_t un = __float_as_uint(mn), ux = __float_as_uint(mx);
    const uint32_t rn = un + 0x7FFFu + ((un >> 16) & 1u);
    const uint32_t rx = ux + 0x7FFFu + ((ux >> 16) & 1u);
    return in_range & ((rp ^ rn) < 0x10000u) & ((rp ^ rx) < 0x10000u) & (mn == mn) & (mx == mx) &
           (hi == hi);
}

// Exact inverse and change test of one element (sec. 4.1 / 4.2.1).
template <bool kDecayOne, bool kLit>
__device__ __forceinline__ float exact_prev(float p, float m, float v, const ExtractParams& a)
{
    const float u = kLit ? step_term_literal(m, v, a.lr, a.bc1, a.bc2, a.eps)
                         : step_term(m, v, a.lrb1, a.rbc2, a.eps);
    const float num = p + u;
    return kDecayOne ? num : num / a.decay;
}

constexpr int kTileBits = __builtin_ctz(kWaveTile);
constexpr int64_t kDenseRatio = 64;             // see flush_wave
static_assert((1 << kTileBits) == kWaveTile, "wave tile must be a power of two");

// Dynamic tail of the unordered call over full tiles: when the waves have
// at least kTailDiv tiles each, the last total / kTailDiv tiles (at most
// 2^20, so that a tile's offset from the tail's start fits a staging key)
// go to blocks four tiles per wave (one flush round) per grab.  A grab adds 2^kGrabShift to the caller's cursor, whose bits below
// kGrabShift count the entries (a delta never reaches 2^36 entries): the
// old value's high bits number the chunk, every reservation masks them off,
// and clear_grabs_kernel clears them once the kernel is done.
constexpr int64_t kTailDiv = 16;
constexpr int64_t kMaxTailTiles = (int64_t)1 << 20;
constexpr int kGrabShift = 36;
constexpr unsigned long long kCountMask = (1ull << kGrabShift) - 1;

__host__ __device__ inline int64_t tail_tiles(int64_t tiles, int64_t waves, bool dynamic)
{
    const int64_t d = dynamic && tiles >= kTailDiv * waves ? tiles / kTailDiv : 0;
    return d < kMaxTailTiles ? d : kMaxTailTiles;
}
// Per-wave LDS areas.  Keys are (wave iteration << kTileBits) | element in
// the tile; the wave's tiles are t_first + iteration.
struct WaveStage {
    uint32_t* key;    // output staging: changed entries awaiting a flush
    uint16_t* val;
    float* qp;        // candidate queue: elements without an "unchanged" proof
    float* qm;
    float* qv;
    uint32_t* qkey;
    int64_t t_first;
    int32_t wave;     // global wave number
};

// Wave-uniform output state: entries staged in LDS, entries flushed so far;
// ordered mode: entries written to the wave's region, and whether the region
// is exhausted (then every later flush goes to the shared area).
struct Staging {
    int staged;
    int64_t flushed;
    int64_t in_region;
    int spilled;
};

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Write staged entries [0, staged) to out_idx / out_val from position
// base, dropping those at or beyond capacity; kStream: offsets with
// non-temporal stores.
template <bool kStream>
__device__ __forceinline__ void write_out(const ExtractParams& a, const WaveStage& st, int64_t base,
                                          int staged, int lane)
{
    for (int i = lane; i < staged; i += 64) {
        const int64_t pos = base + i;
        if (pos < a.capacity) {
            const uint32_t key = st.key[i];
            const int64_t t = st.t_first + (int64_t)(key >> kTileBits);
            const int64_t x = a.index_base + t * kWaveTile + (int64_t)(key & (kWaveTile - 1));
            if (kStream)
                __builtin_nontemporal_store(x, a.out_idx + pos);
            else
                a.out_idx[pos] = x;
            a.out_val[pos] = st.val[i];
        }
    }
}

// Write a wave's staged entries (so.staged > 0) to positions base, base + 1,
// ...  A wave that has so far found more than one changed element per
// kDenseRatio elements scanned writes its offsets with non-temporal stores
// (measured faster on deltas of several percent of the state, slower on
// sparse ones); the choice is wave-uniform.
__device__ __forceinline__ void write_staged(const ExtractParams& a, const WaveStage& st,
                                             Staging& so, int64_t base, int lane)
{
    const int staged = so.staged;
    const uint32_t last = __builtin_amdgcn_readfirstlane(st.key[staged - 1]);
    const int64_t scanned = ((int64_t)(last >> kTileBits) + 1) * kWaveTile;
    if ((so.flushed + staged) * kDenseRatio > scanned)
        write_out<true>(a, st, base, staged, lane);
    else
        write_out<false>(a, st, base, staged, lane);
    so.flushed += staged;
    so.staged = 0;
    wave_sync();   // the staging area is rewritten next: finish these reads first
}

// Copy a wave's staged LDS entries to the reserved global range (and, in
// ordered mode, record the run).  Routing mode: route them through the plan
// into the receiver buckets instead (count, one reservation per rank, write).
template <bool kRoute>
__device__ void flush_wave(const ExtractParams& a, const WaveStage& st, Staging& so, int lane)
{
    const int staged = so.staged;
    wave_sync();   // every lane's LDS stores visible to the other lanes
    if (kRoute) {
        if (lane == 0)
            atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor), (unsigned long long)staged);
        rt::SegInfo cache{};
        int runv = 0;                            // lane r: entries for rank out.first + r
#pragma unroll 1
        for (int pass = 0; pass < 2; ++pass) {
            int64_t basev = 0;
            if (pass == 1) {
                if (lane < a.out.count && runv > 0)
                    basev = (int64_t)atomicAdd(reinterpret_cast<unsigned long long*>(
                                                   &a.rank_count[a.out.first + lane]),
                                               (unsigned long long)runv);
                runv = 0;
            }
#pragma unroll 1
            for (int g = 0; g < staged; g += 64) {
                const int i = g + lane;
                int64_t x = -1;
                uint16_t y = 0;
                if (i < staged) {
                    const uint32_t key = st.key[i];
                    const int64_t t = st.t_first + (int64_t)(key >> kTileBits);
                    x = a.index_base + t * kWaveTile + (key & (kWaveTile - 1));
                    y = st.val[i];
                    if (x >= a.plan.total) x = -1;
                }
                if (pass == 0)
                    rt::route_slot<false, false>(a.plan, a.out, lane, x, y, runv, 0, cache);
                else
                    rt::route_slot<true, false>(a.plan, a.out, lane, x, y, runv, basev, cache);
            }
        }
        so.flushed += staged;
        so.staged = 0;
        wave_sync();
        return;
    }
    if (a.runs && !so.spilled) {
        if (so.flushed + staged <= a.region_size) {
            // ordered mode: the wave's own region, no atomics (reservations
            // that every wave takes from one address slow the whole stream)
            const int64_t r0 = (int64_t)st.wave * a.region_size + so.flushed;
            for (int i = lane; i < staged; i += 64) {
                const uint32_t key = st.key[i];
                const int64_t t = st.t_first + (int64_t)(key >> kTileBits);
                a.region_idx[r0 + i] = a.index_base + t * kWaveTile + (key & (kWaveTile - 1));
                a.region_val[r0 + i] = st.val[i];
            }
            so.flushed += staged;
            so.in_region = so.flushed;
            so.staged = 0;
            wave_sync();
            return;
        }
        so.spilled = 1;
    }
    unsigned long long base = 0;
    if (lane == 0) {
        base = atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor),
                         (unsigned long long)staged) & kCountMask;
        if (a.runs) {
            const unsigned long long r =
                atomicAdd(reinterpret_cast<unsigned long long*>(a.run_cursor), 1ull);
            if ((int64_t)r < a.max_runs) {
                OrderRun run;
                run.src = (int64_t)base;
                run.woff = so.flushed;
                run.count = staged;
                run.wave = st.wave;
                a.runs[r] = run;
            }
        }
    }
    base = __shfl(base, 0);
    write_staged(a, st, so, (int64_t)base, lane);
}

// Selection of the four elements of each lane's float4 slot (256
// consecutive elements per wave): one ballot per element of the float4 and
// the slot's count.
struct Slot4 {
    uint64_t ball[4];
    int count;
};

__device__ __forceinline__ Slot4 select4(const bool (&sel)[4])
{
    Slot4 r;
    r.count = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        r.ball[c] = __ballot(sel[c]);
        r.count += __popcll(r.ball[c]);
    }
    return r;
}

// Selected elements of the slot in lanes below this one: the position of
// this lane's first selected element; its others follow in element order.
__device__ __forceinline__ int lanes_before(const Slot4& r)
{
    int before = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) before += lane_prefix(r.ball[k]);
    return before;
}

// Stage one ballot of changed entries (at most 64), flushing first when the
// staging area would overflow.  Wave-uniform control flow.
template <bool kRoute>
__device__ __forceinline__ void stage_changed(const ExtractParams& a, const WaveStage& st,
                                              Staging& so, int lane, bool changed,
                                              uint32_t key, uint16_t val)
{
    const uint64_t k = __ballot(changed);
    if (k == 0) return;
    const int cnt = __popcll(k);
    const int before = so.staged;
    const int pos = before + lane_prefix(k);
    if (changed && pos < kWaveStage) {
        st.key[pos] = key;
        st.val[pos] = val;
    }
    if (before + cnt < kWaveStage) {
        so.staged = before + cnt;
        return;
    }
    // the staging area is full: flush exactly kWaveStage entries (so every
    // flush but a wave's last is one full, aligned block), then stage the rest
    so.staged = kWaveStage;
    flush_wave<kRoute>(a, st, so, lane);
    if (changed && pos >= kWaveStage) {
        st.key[pos - kWaveStage] = key;
        st.val[pos - kWaveStage] = val;
    }
    so.staged = before + cnt - kWaveStage;
}

// Combined flushes of the unordered call.  Every kRound tiles, and once at
// the end, the kW waves of a block meet at a barrier; when they hold at
// least kBlockFlush staged entries (at the end: any), one atomicAdd on the
// cursor reserves room for all of them and each wave writes its entries
// after those of the waves before it.  Every wave of the device reserving
// its own space from the one cursor address is what slows the stream (the
// atomics, not the stores), so fewer, larger reservations are the point; a
// wave whose staging area fills between two meetings still flushes on its
// own.  Block-uniform control flow; the two LDS slots alternate, so a slot
// is rewritten only after every wave has passed a later barrier.
constexpr int kRound = 4;
constexpr int kFlushPerWave = 768;            // block flush threshold per wave

template <int kW>
__device__ void block_round(const ExtractParams& a, const WaveStage& st, Staging& so, int lane,
                            int wave, int (*s_cnt)[kW], unsigned long long* s_base, int slot,
                            bool last_round)
{
    if (lane == 0) s_cnt[slot][wave] = so.staged;
    __syncthreads();
    int total = 0, before = 0;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
        const int c = s_cnt[slot][w];
        total += c;
        before += w < wave ? c : 0;
    }
    if (total == 0 || (!last_round && total < kW * kFlushPerWave)) return;
    if (threadIdx.x == 0)
        s_base[slot] = atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor),
                                 (unsigned long long)total) & kCountMask;
    __syncthreads();
    if (so.staged > 0) write_staged(a, st, so, (int64_t)s_base[slot] + before, lane);
}

// Exact inverse of every queued candidate, 64 per pass; changed ones are
// staged.  Empties the queue.
template <bool kDecayOne, bool kLit, bool kRoute>
__device__ void drain_queue(const ExtractParams& a, const WaveStage& st, int& queued, Staging& so,
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
            const float ph = exact_prev<kDecayOne, kLit>(p, st.qm[i], st.qv[i], a);
            bn = (uint16_t)bf16_bits(p);
            changed = bf16_bits(ph) != bn;
            key = st.qkey[i];
        }
        stage_changed<kRoute>(a, st, so, lane, changed, key, bn);
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

template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev, bool kLit, bool kRoute>
__device__ __forceinline__ void process_tile(const ExtractParams& a, int64_t t0, int lane,
                                             Staging& so, int& queued, const WaveStage& st,
                                             uint32_t iter, const f32x4* P, const f32x4* M,
                                             const f32x4* V)
{
    const int64_t rem = a.n - t0;
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int off = (j * 64 + lane) * 4;
        const uint32_t key0 = (iter << kTileBits) | (uint32_t)off;
        if (kWritePrev) {
            // theta_hat requested: the exact path for every element
            f32x4 prev;
            bool sel[4];
            uint32_t bn[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float p = P[j][c];
                const float ph = exact_prev<kDecayOne, kLit>(p, M[j][c], V[j][c], a);
                prev[c] = ph;
                bn[c] = bf16_bits(p);
                sel[c] = (kFull || off + c < rem) && bf16_bits(ph) != bn[c];
            }
            const Slot4 r = select4(sel);
            if (r.count != 0) {
                const int before = so.staged;
                const int base = before + lanes_before(r);
                int k = 0;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    if (sel[c]) {
                        if (base + k < kWaveStage) {
                            st.key[base + k] = key0 + c;
                            st.val[base + k] = (uint16_t)bn[c];
                        }
                        ++k;
                    }
                }
                if (before + r.count < kWaveStage) {
                    so.staged = before + r.count;
                } else {   // full: flush one whole block, then stage the rest
                    so.staged = kWaveStage;
                    flush_wave<kRoute>(a, st, so, lane);
                    k = 0;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if (sel[c]) {
                            if (base + k >= kWaveStage) {
                                st.key[base + k - kWaveStage] = key0 + c;
                                st.val[base + k - kWaveStage] = (uint16_t)bn[c];
                            }
                            ++k;
                        }
                    }
                    so.staged = before + r.count - kWaveStage;
                }
            }
            if (kFull || (kVecLoads && off + 3 < rem)) {
                __builtin_nontemporal_store(prev, reinterpret_cast<f32x4*>(a.out_prev + t0 + off));
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    if (off + c < rem) a.out_prev[t0 + off + c] = prev[c];
            }
        } else {
            bool sel[4];
#pragma unroll
            for (int c = 0; c < 4; ++c)
                sel[c] = (kFull || off + c < rem) &&
                         ((kLit && !a.lit_filter) ||
                          !proven_unchanged<kDecayOne, kLit>(P[j][c], M[j][c], V[j][c], a));
            const Slot4 r = select4(sel);
            if (r.count != 0) {
                if (queued + r.count > kQueue)
                    drain_queue<kDecayOne, kLit, kRoute>(a, st, queued, so, lane);
                const int base = queued + lanes_before(r);
                int k = 0;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    if (sel[c]) {
                        st.qp[base + k] = P[j][c];
                        st.qm[base + k] = M[j][c];
                        st.qv[base + k] = V[j][c];
                        st.qkey[base + k] = key0 + c;
                        ++k;
                    }
                }
                queued += r.count;
            }
        }
    }
}

// Wave tiles [first, last) of the range; kFull: each lies inside [0, n).
template <bool kFull, bool kVecLoads, bool kDecayOne, bool kWritePrev, bool kLit, bool kRoute>
__global__ __launch_bounds__(64 * kWavesOf<kFull>) void extract_kernel(ExtractParams a,
                                                                      int64_t first, int64_t last)
{
    constexpr int kWaves = kWavesOf<kFull>;
    __shared__ uint32_t s_key[kWaves][kWaveStage];
    __shared__ uint16_t s_val[kWaves][kWaveStage];
    __shared__ float s_qp[kWaves][kQueue];
    __shared__ float s_qm[kWaves][kQueue];
    __shared__ float s_qv[kWaves][kQueue];
    __shared__ uint32_t s_qkey[kWaves][kQueue];
    __shared__ int s_cnt[2][kWaves];
    __shared__ unsigned long long s_base[2];
    __shared__ int64_t s_chunk;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t g = (int64_t)blockIdx.x * kWaves + wave;
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    // unordered output: combined flushes (block_round); every wave of the
    // block runs the same iterations, so the barriers match
    const bool combine = !kRoute && a.runs == nullptr;
    // wave g owns the contiguous tile range [g per, (g+1) per) of the
    // static part [first, s_last); the tail [s_last, last) is dynamic
    constexpr bool kTail = kFull && !kRoute;     // a dynamic tail is possible
    const int64_t tail = kTail ? tail_tiles(last - first, nw, combine) : 0;
    const int64_t s_last = last - tail;
    const int64_t per = (s_last - first + nw - 1) / nw;
    const int64_t w_first = first + g * per;
    const int64_t w_last = (w_first + per < s_last) ? w_first + per : s_last;
    Staging so{0, 0, 0, 0};
    const WaveStage st{s_key[wave], s_val[wave], s_qp[wave], s_qm[wave], s_qv[wave],
                       s_qkey[wave], w_first, a.wave0 + (int32_t)g};
    int queued = 0;
    int round = 0;                               // block_round calls so far (LDS slot parity)
    for (int64_t it = 0; it < per; ++it) {
        const int64_t t = w_first + it;
        if (t < w_last) {
            f32x4 P[kVec], M[kVec], V[kVec];
            load_tile<kFull, kVecLoads>(a, t * kWaveTile, lane, P, M, V);
            process_tile<kFull, kVecLoads, kDecayOne, kWritePrev, kLit, kRoute>(
                a, t * kWaveTile, lane, so, queued, st, (uint32_t)it, P, M, V);
        }
        if (it % kRound == kRound - 1) {
            if (combine)
                block_round(a, st, so, lane, wave, s_cnt, s_base, (round++) & 1, false);
            else if (!kRoute)
                __syncthreads();   // ordered: keeps the block's waves in step
        }
    }
    if (queued > 0) drain_queue<kDecayOne, kLit, kRoute>(a, st, queued, so, lane);
    if (kTail && tail > 0) {
        // staged keys count tiles from the stage's first tile: empty the
        // staging areas, then count from the tail's start
        block_round(a, st, so, lane, wave, s_cnt, s_base, (round++) & 1, true);
        const WaveStage tst{s_key[wave], s_val[wave], s_qp[wave], s_qm[wave], s_qv[wave],
                            s_qkey[wave], s_last, st.wave};
        for (;;) {
            if (threadIdx.x == 0)
                s_chunk = (int64_t)(atomicAdd(reinterpret_cast<unsigned long long*>(a.cursor),
                                              1ull << kGrabShift) >> kGrabShift);
            __syncthreads();
            const int64_t c = s_chunk * (kWaves * kRound);   // block-uniform
            __syncthreads();                                 // s_chunk is rewritten next
            if (c >= tail) break;
            for (int i = 0; i < kRound; ++i) {
                const int64_t rel = c + (int64_t)wave * kRound + i;   // tile s_last + rel
                if (rel < tail) {
                    f32x4 P[kVec], M[kVec], V[kVec];
                    load_tile<kFull, kVecLoads>(a, (s_last + rel) * kWaveTile, lane, P, M, V);
                    process_tile<kFull, kVecLoads, kDecayOne, kWritePrev, kLit, kRoute>(
                        a, (s_last + rel) * kWaveTile, lane, so, queued, tst, (uint32_t)rel, P,
                        M, V);
                }
            }
            block_round(a, tst, so, lane, wave, s_cnt, s_base, (round++) & 1, false);
        }
        if (queued > 0) drain_queue<kDecayOne, kLit, kRoute>(a, tst, queued, so, lane);
        block_round(a, tst, so, lane, wave, s_cnt, s_base, (round++) & 1, true);
    } else if (combine) {
        block_round(a, st, so, lane, wave, s_cnt, s_base, (round++) & 1, true);
    } else if (so.staged > 0) {
        flush_wave<kRoute>(a, st, so, lane);
    }
    if (a.runs && lane == 0) {
        a.wave_count[st.wave] = so.flushed;
        a.region_count[st.wave] = so.in_region;
    }
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
            const float u = a.literal ? step_term_literal(mt, vt, a.lr, a.bc1, a.bc2, a.eps)
                                      : step_term(mt, vt, a.lrb1, a.rbc2, a.eps);
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

// After an unordered launch with a dynamic tail: the grab count leaves the
// cursor's high bits (single thread; runs after the extract kernel on the
// same stream).
__global__ void clear_grabs_kernel(int64_t* cursor)
{
    *cursor = (int64_t)((unsigned long long)*cursor & kCountMask);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Blocks that one launch over wave tiles [first, last) uses, at most
// max_waves waves.
template <bool F>
int64_t blocks_of(int64_t first, int64_t last, int64_t max_waves)
{
    if (last <= first) return 0;
    const int64_t b = (last - first + kWavesOf<F> - 1) / kWavesOf<F>;
    const int64_t cap = max_waves / kWavesOf<F>;
    return b < cap ? b : cap;
}

// Launch over wave tiles [first, last); returns the number of waves.
template <bool F, bool V, bool D, bool L, bool R>
int32_t launch_tiles(ExtractParams a, int64_t first, int64_t last, int64_t max_waves,
                     int32_t wave0, hipStream_t s)
{
    if (last <= first) return 0;
    constexpr int kBlock = 64 * kWavesOf<F>;
    const dim3 grid((unsigned)blocks_of<F>(first, last, max_waves));
    a.wave0 = wave0;
    if (R)   // routing mode: no theta_hat output
        hipLaunchKernelGGL((extract_kernel<F, V, D, false, L, R>), grid, dim3(kBlock), 0, s, a, first,
                           last);
    else if (a.out_prev)
        hipLaunchKernelGGL((extract_kernel<F, V, D, true, L, false>), grid, dim3(kBlock), 0, s, a,
                           first, last);
    else
        hipLaunchKernelGGL((extract_kernel<F, V, D, false, L, false>), grid, dim3(kBlock), 0, s, a,
                           first, last);
    if (F && !R && a.runs == nullptr &&
        tail_tiles(last - first, (int64_t)grid.x * kWavesOf<F>, true) > 0)
        hipLaunchKernelGGL(clear_grabs_kernel, dim3(1), dim3(1), 0, s, a.cursor);
    return (int32_t)grid.x * kWavesOf<F>;
}

template <bool D, bool L, bool R>
int32_t launch_all(const ExtractParams& a, bool vec, int64_t max_waves, hipStream_t s)
{
    const int64_t full = a.n / kWaveTile;
    const int64_t ntiles = (a.n + kWaveTile - 1) / kWaveTile;
    if (vec) {
        const int32_t w = launch_tiles<true, true, D, L, R>(a, 0, full, max_waves, 0, s);  // unguarded
        return w + launch_tiles<false, true, D, L, R>(a, full, ntiles, max_waves, w, s);   // ragged
    }
    return launch_tiles<false, false, D, L, R>(a, 0, ntiles, max_waves, 0, s);           // scalar loads
}

// ---- ordered mode: runs to ascending positions ----------------------------

// One block: wave_base = *cursor + exclusive prefix of the wave totals; then
// the cursor advances by their sum, the true total of the call.
__global__ __launch_bounds__(1024) void order_scan_kernel(OrderParams o)
{
    constexpr int kThreads = 1024;
    constexpr int kPer = kMaxOrderedWaves / kThreads;
    __shared__ int64_t part[kThreads];
    const int tid = threadIdx.x;
    const int lo = tid * kPer;
    int64_t sum = 0;
    for (int i = 0; i < kPer; ++i)
        if (lo + i < o.waves) sum += o.wave_count[lo + i];
    part[tid] = sum;
    __syncthreads();
    for (int d = 1; d < kThreads; d <<= 1) {      // inclusive scan of the partial sums
        const int64_t x = (tid >= d) ? part[tid - d] : 0;
        __syncthreads();
        part[tid] += x;
        __syncthreads();
    }
    const int64_t c0 = *o.cursor;
    int64_t run = c0 + part[tid] - sum;
    for (int i = 0; i < kPer; ++i) {
        if (lo + i < o.waves) {
            o.wave_base[lo + i] = run;
            run += o.wave_count[lo + i];
        }
    }
    __syncthreads();                              // every thread has read the cursor
    if (tid == 0) *o.cursor = c0 + part[kThreads - 1];
}

constexpr int kCopyBlock = 256;
constexpr int kCopySlots = 8;                  // entries per lane per copy chunk
constexpr int kCopyChunk = 64 * kCopySlots;

// Regions: the waves take chunks of kCopyChunk entries (chunk c of extract
// wave g's region: its entries c kCopyChunk + i, which move to wave_base[g]
// + c kCopyChunk + i), all loads of a chunk before its stores.  Then whole
// recorded runs: entry i of a run moves from src + i to wave_base[wave] +
// woff + i.
__global__ __launch_bounds__(kCopyBlock) void order_copy_kernel(OrderParams o)
{
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * (kCopyBlock / 64) + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * (kCopyBlock / 64);
    const int64_t per_region = (o.region_size + kCopyChunk - 1) / kCopyChunk;
    const int64_t chunks = (int64_t)o.waves * per_region;
    const int64_t* __restrict__ ridx = o.region_idx;
    const uint16_t* __restrict__ rval = o.region_val;
    for (int64_t k = w; k < chunks; k += nw) {
        const int64_t g = k / per_region;
        const int64_t c0 = (k - g * per_region) * kCopyChunk;
        const int64_t cnt = o.region_count[g];
        if (c0 >= cnt) continue;
        const int64_t src0 = g * o.region_size + c0;
        const int64_t dst0 = o.wave_base[g] + c0;
        int64_t x[kCopySlots];
        uint16_t y[kCopySlots];
#pragma unroll
        for (int j = 0; j < kCopySlots; ++j) {
            const int64_t i = j * 64 + lane;
            x[j] = c0 + i < cnt ? ridx[src0 + i] : 0;
            y[j] = c0 + i < cnt ? rval[src0 + i] : (uint16_t)0;
        }
#pragma unroll
        for (int j = 0; j < kCopySlots; ++j) {
            const int64_t i = j * 64 + lane;
            if (c0 + i < cnt && dst0 + i < o.capacity) {
                o.out_idx[dst0 + i] = x[j];
                o.out_val[dst0 + i] = y[j];
            }
        }
    }
    int64_t nruns = *o.run_cursor;
    if (nruns > o.max_runs) nruns = o.max_runs;
    for (int64_t r = w; r < nruns; r += nw) {
        const OrderRun run = o.runs[r];
        const int64_t dst0 = o.wave_base[run.wave] + run.woff;
        for (int i = lane; i < run.count; i += 64) {
            const int64_t src = run.src + i;
            const int64_t dst = dst0 + i;
            if (src < o.src_capacity && dst < o.capacity) {
                o.out_idx[dst] = o.src_idx[src];
                o.out_val[dst] = o.src_val[src];
            }
        }
    }
}

}  // namespace

hipError_t launch_order(const OrderParams& o, int cus, hipStream_t stream)
{
    if (o.waves <= 0) return hipSuccess;
    hipLaunchKernelGGL(order_scan_kernel, dim3(1), dim3(1024), 0, stream, o);
    hipLaunchKernelGGL(order_copy_kernel, dim3((unsigned)cus * 8), dim3(kCopyBlock), 0, stream, o);
    return hipGetLastError();
}

namespace {

// Waves that launch_all launches (its grid rule).
int64_t waves_of(int64_t n, bool vec, int64_t max_waves)
{
    const int64_t full = n / kWaveTile;
    const int64_t ntiles = (n + kWaveTile - 1) / kWaveTile;
    if (vec)
        return blocks_of<true>(0, full, max_waves) * kWavesOf<true> +
               blocks_of<false>(full, ntiles, max_waves) * kWavesOf<false>;
    return blocks_of<false>(0, ntiles, max_waves) * kWavesOf<false>;
}

// Waves per launch at most.  Ordered mode: both launches together stay
// within kMaxOrderedWaves (the ragged launch covers one tile: one block).
int64_t max_waves_of(const ExtractParams& a, int cus)
{
    int64_t max_waves = (int64_t)cus * kWavesPerCU;
    const int64_t ordered_cap = kMaxOrderedWaves - kWavesOf<false>;
    if (a.runs && max_waves > ordered_cap) max_waves = ordered_cap;
    return max_waves;
}

bool vector_loads(const ExtractParams& a)
{
    return aligned16(a.p) && aligned16(a.m) && aligned16(a.v) &&
           (a.out_prev == nullptr || aligned16(a.out_prev));
}

}  // namespace

int64_t extract_waves(const ExtractParams& a, int cus)
{
    return a.n > 0 ? waves_of(a.n, vector_loads(a), max_waves_of(a, cus)) : 0;
}

hipError_t launch_extract(const ExtractParams& a, int cus, hipStream_t stream, int32_t* waves)
{
    if (waves) *waves = 0;
    if (a.n <= 0) return hipSuccess;
    const int64_t max_waves = max_waves_of(a, cus);
    const bool vec = vector_loads(a);
    int32_t w;
    const bool one = a.decay == 1.0f;
    if (a.route) {
        if (a.literal)
            w = one ? launch_all<true, true, true>(a, vec, max_waves, stream)
                    : launch_all<false, true, true>(a, vec, max_waves, stream);
        else
            w = one ? launch_all<true, false, true>(a, vec, max_waves, stream)
                    : launch_all<false, false, true>(a, vec, max_waves, stream);
    } else if (a.literal) {
        w = one ? launch_all<true, true, false>(a, vec, max_waves, stream)
                : launch_all<false, true, false>(a, vec, max_waves, stream);
    } else {
        w = one ? launch_all<true, false, false>(a, vec, max_waves, stream)
                : launch_all<false, false, false>(a, vec, max_waves, stream);
    }
    if (waves) *waves = w;
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
