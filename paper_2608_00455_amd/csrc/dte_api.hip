// Host side of the C ABI declared in include/dte.h: argument validation,
// step-scalar derivation, transfer-plan validation and upload, and kernel
// launches.  No call here allocates or synchronises except
// dte_plan_create / dte_plan_destroy.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <memory>
#include <vector>

#include "abi_guard.h"
#include "dte_internal.h"

struct dte_plan {
    int device;
    int32_t nseg;
    int32_t nop;
    int32_t nranks;
    int32_t max_replication;
    int64_t total;
    std::vector<int64_t> rank_numel;
    void* dev_mem;          // one allocation holding every table
    dte::PlanView view;
};

namespace {

// Compute units of a device, queried once per device (calls may come from
// several host threads: the cache is atomic; a race only repeats the query).
int cu_count(int device)
{
    static std::atomic<int> cache[64];
    if (device < 0 || device >= 64) return 256;
    int n = cache[device].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) !=
                hipSuccess || n <= 0)
            n = 256;
        cache[device].store(n, std::memory_order_relaxed);
    }
    return n;
}

// The plan's tables live on the device it was created on; the hot calls
// launch on the current device, which must be that one.
bool on_plan_device(const dte_plan* plan)
{
    int dev = -1;
    return hipGetDevice(&dev) == hipSuccess && dev == plan->device;
}

int current_cus()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    return cu_count(dev);
}

bool valid_hp(const dte_adamw_step* hp)
{
    if (!hp) return false;
    if (!(std::isfinite(hp->lr) && hp->lr >= 0.0)) return false;
    if (!(hp->beta1 >= 0.0 && hp->beta1 < 1.0)) return false;
    if (!(hp->beta2 >= 0.0 && hp->beta2 < 1.0)) return false;
    if (!(std::isfinite(hp->eps) && hp->eps >= 0.0)) return false;
    if (!std::isfinite(hp->weight_decay)) return false;
    if (hp->step < 1) return false;
    if (!(1.0 - hp->lr * hp->weight_decay > 0.0)) return false;
    if (hp->order != DTE_ORDER_FOLDED && hp->order != DTE_ORDER_LITERAL) return false;
    if (hp->reserved != 0) return false;
    return true;
}

struct AllScalars {
    dte_scalars s;
    float b1, b2, omb1, omb2;
};

// Binary64 evaluation, one rounding to binary32 per scalar.
AllScalars derive(const dte_adamw_step& hp)
{
    AllScalars a;
    const double bc1 = 1.0 - std::pow(hp.beta1, (double)hp.step);
    const double bc2 = 1.0 - std::pow(hp.beta2, (double)hp.step);
    a.s.lrb1 = (float)(hp.lr / bc1);
    a.s.rbc2 = (float)(1.0 / bc2);
    a.s.eps = (float)hp.eps;
    a.s.decay = (float)(1.0 - hp.lr * hp.weight_decay);
    a.s.lr = (float)hp.lr;
    a.s.bc1 = (float)bc1;
    a.s.bc2 = (float)bc2;
    a.s.order = hp.order;
    a.b1 = (float)hp.beta1;
    a.b2 = (float)hp.beta2;
    a.omb1 = (float)(1.0 - hp.beta1);
    a.omb2 = (float)(1.0 - hp.beta2);
    return a;
}

bool bias_ok(const dte_adamw_step& hp)
{
    const double bc1 = 1.0 - std::pow(hp.beta1, (double)hp.step);
    const double bc2 = 1.0 - std::pow(hp.beta2, (double)hp.step);
    return bc1 > 0.0 && bc2 > 0.0;
}

struct Box {
    int64_t lo[DTE_MAX_DIMS];
    int64_t hi[DTE_MAX_DIMS];
};

bool boxes_overlap(const Box& a, const Box& b, int nd)
{
    for (int d = 0; d < nd; ++d)
        if (a.hi[d] <= b.lo[d] || b.hi[d] <= a.lo[d]) return false;
    return true;
}

int64_t prod(const int64_t* s, int nd)
{
    int64_t n = 1;
    for (int d = 0; d < nd; ++d) n *= s[d];
    return n;
}

// Exact coverage of a segment by its source boxes, by coordinate
// compression: every cell of the grid cut at all box faces must lie in a
// box.  Also returns the largest number of boxes covering one cell.
bool covers(const int64_t* shape, int nd, const std::vector<Box>& boxes, int32_t* max_cover)
{
    std::vector<int64_t> cuts[DTE_MAX_DIMS];
    for (int d = 0; d < nd; ++d) {
        cuts[d].push_back(0);
        cuts[d].push_back(shape[d]);
        for (const Box& b : boxes) {
            cuts[d].push_back(b.lo[d]);
            cuts[d].push_back(b.hi[d]);
        }
        std::sort(cuts[d].begin(), cuts[d].end());
        cuts[d].erase(std::unique(cuts[d].begin(), cuts[d].end()), cuts[d].end());
    }
    size_t ncell[DTE_MAX_DIMS] = {1, 1, 1, 1};
    size_t cells = 1;
    for (int d = 0; d < nd; ++d) {
        ncell[d] = cuts[d].size() - 1;
        cells *= ncell[d];
    }
    int32_t best = 0;
    for (size_t c = 0; c < cells; ++c) {
        size_t rem = c;
        int64_t pt[DTE_MAX_DIMS];
        for (int d = nd - 1; d >= 0; --d) {
            pt[d] = cuts[d][rem % ncell[d]];   // the cell's lower corner
            rem /= ncell[d];
        }
        int32_t cover = 0;
        for (const Box& b : boxes) {
            bool in = true;
            for (int d = 0; d < nd && in; ++d) in = b.lo[d] <= pt[d] && pt[d] < b.hi[d];
            cover += in ? 1 : 0;
        }
        if (cover == 0) return false;
        best = std::max(best, cover);
    }
    *max_cover = std::max(*max_cover, best);
    return true;
}

dte_status validate_plan(const dte_segment* segs, int32_t nseg, const dte_op* ops, int32_t nop,
                         int32_t nranks, const int64_t* rank_numel, int64_t* total_out,
                         int32_t* max_rep)
{
    int64_t pos = 0;
    for (int32_t s = 0; s < nseg; ++s) {
        const dte_segment& g = segs[s];
        if (g.ndim < 1 || g.ndim > DTE_MAX_DIMS || g.flat_begin != pos) return DTE_ERR_PLAN;
        for (int d = 0; d < g.ndim; ++d)
            if (g.shape[d] < 1 || g.shape[d] >= (int64_t(1) << 31)) return DTE_ERR_PLAN;
        const int64_t n = prod(g.shape, g.ndim);
        if (n >= (int64_t(1) << 32)) return DTE_ERR_PLAN;
        pos += n;
    }
    *total_out = pos;

    struct View {
        int32_t rank;
        int64_t base;
        int32_t nd;
        int64_t shape[DTE_MAX_DIMS];
        std::vector<Box> boxes;
    };
    std::vector<View> views;
    std::vector<std::vector<int32_t>> by_seg(nseg);
    for (int32_t k = 0; k < nop; ++k) {
        const dte_op& o = ops[k];
        if (o.segment < 0 || o.segment >= nseg || o.rank < 0 || o.rank >= nranks)
            return DTE_ERR_PLAN;
        const dte_segment& g = segs[o.segment];
        const int nd = g.ndim;
        for (int d = 0; d < nd; ++d) {
            if (o.extent[d] < 1 || o.src_origin[d] < 0 || o.dst_origin[d] < 0) return DTE_ERR_PLAN;
            if (o.dst_shape[d] < 1 || o.dst_shape[d] >= (int64_t(1) << 31)) return DTE_ERR_PLAN;
            if (o.src_origin[d] + o.extent[d] > g.shape[d]) return DTE_ERR_PLAN;
            if (o.dst_origin[d] + o.extent[d] > o.dst_shape[d]) return DTE_ERR_PLAN;
        }
        const int64_t vsize = prod(o.dst_shape, nd);
        if (o.dst_base < 0 || o.dst_base + vsize > rank_numel[o.rank]) return DTE_ERR_PLAN;
        by_seg[o.segment].push_back(k);
        // find or add the destination view
        View* vw = nullptr;
        for (View& w : views)
            if (w.rank == o.rank && w.base == o.dst_base) {
                vw = &w;
                break;
            }
        if (!vw) {
            View w;
            w.rank = o.rank;
            w.base = o.dst_base;
            w.nd = nd;
            for (int d = 0; d < DTE_MAX_DIMS; ++d) w.shape[d] = d < nd ? o.dst_shape[d] : 1;
            views.push_back(w);
            vw = &views.back();
        } else {
            if (vw->nd != nd) return DTE_ERR_PLAN;
            for (int d = 0; d < nd; ++d)
                if (vw->shape[d] != o.dst_shape[d]) return DTE_ERR_PLAN;
        }
        Box b;
        for (int d = 0; d < DTE_MAX_DIMS; ++d) {
            b.lo[d] = d < nd ? o.dst_origin[d] : 0;
            b.hi[d] = d < nd ? o.dst_origin[d] + o.extent[d] : 1;
        }
        for (const Box& other : vw->boxes)
            if (boxes_overlap(b, other, nd)) return DTE_ERR_PLAN;   // two writers
        vw->boxes.push_back(b);
    }
    // distinct views of one rank: disjoint flat ranges
    std::sort(views.begin(), views.end(), [](const View& a, const View& b) {
        return a.rank != b.rank ? a.rank < b.rank : a.base < b.base;
    });
    for (size_t i = 1; i < views.size(); ++i) {
        const View& a = views[i - 1];
        const View& b = views[i];
        if (a.rank == b.rank && a.base + prod(a.shape, a.nd) > b.base) return DTE_ERR_PLAN;
    }
    // per segment: per-rank source boxes disjoint; union covers the segment
    *max_rep = 0;
    for (int32_t s = 0; s < nseg; ++s) {
        const dte_segment& g = segs[s];
        std::vector<Box> src;
        std::vector<int32_t> rank_of;
        for (int32_t k : by_seg[s]) {
            const dte_op& o = ops[k];
            Box b;
            for (int d = 0; d < DTE_MAX_DIMS; ++d) {
                b.lo[d] = d < g.ndim ? o.src_origin[d] : 0;
                b.hi[d] = d < g.ndim ? o.src_origin[d] + o.extent[d] : 1;
            }
            for (size_t i = 0; i < src.size(); ++i)
                if (rank_of[i] == o.rank && boxes_overlap(b, src[i], g.ndim)) return DTE_ERR_PLAN;
            src.push_back(b);
            rank_of.push_back(o.rank);
        }
        if (src.empty() || !covers(g.shape, g.ndim, src, max_rep)) return DTE_ERR_PLAN;
    }
    return DTE_OK;
}

size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

extern "C" {

const char* dte_status_string(dte_status status)
{
    switch (status) {
    case DTE_OK: return "DTE_OK";
    case DTE_ERR_ARG: return "DTE_ERR_ARG: invalid argument";
    case DTE_ERR_PLAN: return "DTE_ERR_PLAN: transfer plan failed validation";
    case DTE_ERR_CAPACITY: return "DTE_ERR_CAPACITY: output capacity exceeded";
    case DTE_ERR_HIP: return "DTE_ERR_HIP: HIP runtime error";
    case DTE_ERR_IO: return "DTE_ERR_IO: file read or write failed";
    case DTE_ERR_CORRUPT: return "DTE_ERR_CORRUPT: stored data failed its checksum or format check";
    case DTE_ERR_CHAIN: return "DTE_ERR_CHAIN: version does not extend the local base version";
    case DTE_ERR_UNSUPPORTED: return "DTE_ERR_UNSUPPORTED: codec not available";
    case DTE_ERR_HOST: return "DTE_ERR_HOST: host memory or thread could not be obtained";
    default: return "unknown dte_status";
    }
}

dte_status dte_derive_scalars(const dte_adamw_step* hp, dte_scalars* out)
{
    if (!out || !valid_hp(hp) || !bias_ok(*hp)) return DTE_ERR_ARG;
    *out = derive(*hp).s;
    return DTE_OK;
}

namespace {

bool extract_args_ok(const float* p, const float* m, const float* v, int64_t n,
                     int64_t index_base, const dte_adamw_step* hp, int64_t* out_idx,
                     uint16_t* out_val, int64_t capacity, int64_t* cursor)
{
    if (n < 0 || index_base < 0 || capacity < 0 || !valid_hp(hp) || !bias_ok(*hp)) return false;
    if (n == 0) return true;
    if (!p || !m || !v || !cursor) return false;
    if (capacity > 0 && (!out_idx || !out_val)) return false;
    if (index_base > INT64_MAX - n) return false;
    return true;
}

dte::ExtractParams extract_params(const float* p, const float* m, const float* v, int64_t n,
                                  int64_t index_base, const dte_adamw_step* hp,
                                  int64_t* out_idx, uint16_t* out_val, int64_t capacity,
                                  int64_t* cursor, float* out_prev)
{
    const AllScalars sc = derive(*hp);
    dte::ExtractParams a{};
    a.p = p;
    a.m = m;
    a.v = v;
    a.n = n;
    a.index_base = index_base;
    a.lrb1 = sc.s.lrb1;
    a.rbc2 = sc.s.rbc2;
    a.eps = sc.s.eps;
    a.decay = sc.s.decay;
    {
        // one binary32 step below and above the binary64 reciprocal: a
        // bracket of 1/decay whatever the binary64 rounding did
        const float r = (float)(1.0 / (double)sc.s.decay);
        a.rd_lo = std::nextafter(r, 0.0f);
        a.rd_hi = std::nextafter(r, INFINITY);
    }
    a.literal = sc.s.order == DTE_ORDER_LITERAL;
    a.lr = sc.s.lr;
    a.bc1 = sc.s.bc1;
    a.bc2 = sc.s.bc2;
    // literal order: the "unchanged" proof holds only for these scalars
    // (extract.hip, proven_unchanged)
    a.lit_filter = a.eps >= 0x1p-40f && a.lr <= 0x1p20f && a.bc1 >= 0x1p-20f && a.bc2 >= 0x1p-20f;
    a.floor = a.lit_filter
                  ? std::nextafter((float)(0x1p-124 / std::min(1.0, (double)a.eps)), INFINITY)
                  : 0x1p-126f;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.capacity = capacity;
    a.cursor = cursor;
    a.out_prev = out_prev;
    a.runs = nullptr;
    a.route = 0;
    return a;
}

// Ordered-mode workspace: per-wave regions (capacity entries in all), the
// shared area for flushes that do not fit their region (capacity entries),
// run records, wave totals, region fills and bases, two counters; every
// part 256-byte aligned.
struct OrderedWorkspace {
    int64_t ridx, rval, idx, val, runs, wave_count, region_count, wave_base, counters, total;
    int64_t max_runs;
};

int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Bytes of the static workspace of dte_extract_delta_ordered_noalloc.
constexpr int64_t kNoallocBytes = (int64_t)64 << 20;

OrderedWorkspace ordered_layout(int64_t capacity)
{
    OrderedWorkspace w;
    // every flush but a wave's last holds exactly kWaveStage entries
    w.max_runs = capacity / dte::kWaveStage + dte::kMaxOrderedWaves + 1;
    w.ridx = 0;
    w.rval = align256(w.ridx + capacity * (int64_t)sizeof(int64_t));
    w.idx = align256(w.rval + capacity * (int64_t)sizeof(uint16_t));
    w.val = align256(w.idx + capacity * (int64_t)sizeof(int64_t));
    w.runs = align256(w.val + capacity * (int64_t)sizeof(uint16_t));
    w.wave_count = align256(w.runs + w.max_runs * (int64_t)sizeof(dte::OrderRun));
    w.region_count = align256(w.wave_count + dte::kMaxOrderedWaves * (int64_t)sizeof(int64_t));
    w.wave_base = align256(w.region_count + dte::kMaxOrderedWaves * (int64_t)sizeof(int64_t));
    w.counters = align256(w.wave_base + dte::kMaxOrderedWaves * (int64_t)sizeof(int64_t));
    w.total = align256(w.counters + 2 * (int64_t)sizeof(int64_t));
    return w;
}

}  // namespace

dte_status dte_extract_delta(const float* p, const float* m, const float* v, int64_t n,
                             int64_t index_base, const dte_adamw_step* hp, int64_t* out_idx,
                             uint16_t* out_val, int64_t capacity, int64_t* cursor,
                             float* out_prev, void* stream)
{
    if (!extract_args_ok(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor))
        return DTE_ERR_ARG;
    if (n == 0) return DTE_OK;
    const dte::ExtractParams a = extract_params(p, m, v, n, index_base, hp, out_idx, out_val,
                                                capacity, cursor, out_prev);
    return dte::launch_extract(a, current_cus(), (hipStream_t)stream) == hipSuccess ? DTE_OK
                                                                                     : DTE_ERR_HIP;
}

int64_t dte_ordered_workspace_bytes(int64_t capacity)
{
    if (capacity < 0 || capacity > ((int64_t)1 << 40)) return -1;
    return ordered_layout(capacity).total;
}

namespace {

// The ordered call on a workspace of workspace_bytes at `workspace`
// (device, 256-byte aligned, at least dte_ordered_workspace_bytes(capacity)).
dte_status extract_ordered(const float* p, const float* m, const float* v, int64_t n,
                           int64_t index_base, const dte_adamw_step* hp, int64_t* out_idx,
                           uint16_t* out_val, int64_t capacity, int64_t* cursor, void* workspace,
                           float* out_prev, hipStream_t s)
{
    const OrderedWorkspace w = ordered_layout(capacity);
    char* base = static_cast<char*>(workspace);
    int64_t* counters = reinterpret_cast<int64_t*>(base + w.counters);
    const int cus = current_cus();
    // unordered fill level and run count start at zero (a fill kernel)
    if (dte::launch_zero_i64(counters, 2, s) != hipSuccess) return DTE_ERR_HIP;
    dte::ExtractParams a = extract_params(p, m, v, n, index_base, hp,
                                          reinterpret_cast<int64_t*>(base + w.idx),
                                          reinterpret_cast<uint16_t*>(base + w.val), capacity,
                                          counters, out_prev);
    a.runs = reinterpret_cast<dte::OrderRun*>(base + w.runs);
    a.max_runs = w.max_runs;
    a.run_cursor = counters + 1;
    a.wave_count = reinterpret_cast<int64_t*>(base + w.wave_count);
    a.region_idx = reinterpret_cast<int64_t*>(base + w.ridx);
    a.region_val = reinterpret_cast<uint16_t*>(base + w.rval);
    a.region_count = reinterpret_cast<int64_t*>(base + w.region_count);
    a.region_size = capacity / dte::extract_waves(a, cus);
    int32_t waves = 0;
    if (dte::launch_extract(a, cus, s, &waves) != hipSuccess) return DTE_ERR_HIP;
    dte::OrderParams o;
    o.runs = a.runs;
    o.run_cursor = a.run_cursor;
    o.max_runs = w.max_runs;
    o.wave_count = a.wave_count;
    o.wave_base = reinterpret_cast<int64_t*>(base + w.wave_base);
    o.waves = waves;
    o.src_idx = a.out_idx;
    o.src_val = a.out_val;
    o.src_capacity = capacity;
    o.region_idx = a.region_idx;
    o.region_val = a.region_val;
    o.region_count = a.region_count;
    o.region_size = a.region_size;
    o.out_idx = out_idx;
    o.out_val = out_val;
    o.capacity = capacity;
    o.cursor = cursor;
    return dte::launch_order(o, cus, s) == hipSuccess ? DTE_OK : DTE_ERR_HIP;
}

}  // namespace

dte_status dte_extract_delta_ordered(const float* p, const float* m, const float* v, int64_t n,
                                     int64_t index_base, const dte_adamw_step* hp,
                                     int64_t* out_idx, uint16_t* out_val, int64_t capacity,
                                     int64_t* cursor, void* workspace, int64_t workspace_bytes,
                                     float* out_prev, void* stream)
{
    if (!extract_args_ok(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor))
        return DTE_ERR_ARG;
    if (n == 0) return DTE_OK;
    const int64_t need = dte_ordered_workspace_bytes(capacity);
    if (need < 0 || !workspace || workspace_bytes < need ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return DTE_ERR_ARG;
    return extract_ordered(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor,
                           workspace, out_prev, (hipStream_t)stream);
}

// ---- the ordered call without allocation ---------------------------------

// Its workspace: one array per device in the code object's own storage,
// held while the library is loaded.  Host code never uses this name as an
// address (it is a host-side stand-in); the device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[kNoallocBytes];

namespace {

// Device address of `scratch` on the current device (nullptr if it cannot
// be obtained).  Threads racing on the first call both store the same value.
void* scratch_address()
{
    static std::atomic<void*> cache[64];
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    void* ptr = cache[dev].load(std::memory_order_acquire);
    if (ptr == nullptr) {
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        cache[dev].store(ptr, std::memory_order_release);
    }
    return ptr;
}

}  // namespace

int64_t dte_ordered_noalloc_max_capacity(void)
{
    // the largest capacity whose workspace fits (the size grows with it)
    int64_t lo = 0, hi = kNoallocBytes;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo + 1) / 2;
        if (ordered_layout(mid).total <= kNoallocBytes)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

dte_status dte_extract_delta_ordered_noalloc(const float* p, const float* m, const float* v,
                                             int64_t n, int64_t index_base,
                                             const dte_adamw_step* hp, int64_t* out_idx,
                                             uint16_t* out_val, int64_t capacity,
                                             int64_t* cursor, float* out_prev, void* stream)
{
    if (!extract_args_ok(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor))
        return DTE_ERR_ARG;
    if (capacity > dte_ordered_noalloc_max_capacity()) return DTE_ERR_CAPACITY;
    if (n == 0) return DTE_OK;
    void* ws = scratch_address();
    if (ws == nullptr) return DTE_ERR_HIP;
    return extract_ordered(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor, ws,
                           out_prev, (hipStream_t)stream);
}

dte_status dte_adamw_forward(float* p, float* m, float* v, const float* g, int64_t n,
                             const dte_adamw_step* hp, void* stream)
{
    if (n < 0 || !valid_hp(hp) || !bias_ok(*hp)) return DTE_ERR_ARG;
    if (n == 0) return DTE_OK;
    if (!p || !m || !v || !g) return DTE_ERR_ARG;
    const AllScalars sc = derive(*hp);
    dte::ForwardParams a;
    a.p = p;
    a.m = m;
    a.v = v;
    a.g = g;
    a.n = n;
    a.lrb1 = sc.s.lrb1;
    a.rbc2 = sc.s.rbc2;
    a.eps = sc.s.eps;
    a.decay = sc.s.decay;
    a.b1 = sc.b1;
    a.b2 = sc.b2;
    a.omb1 = sc.omb1;
    a.omb2 = sc.omb2;
    a.literal = sc.s.order == DTE_ORDER_LITERAL;
    a.lr = sc.s.lr;
    a.bc1 = sc.s.bc1;
    a.bc2 = sc.s.bc2;
    return dte::launch_adamw_forward(a, current_cus(), (hipStream_t)stream) == hipSuccess
               ? DTE_OK
               : DTE_ERR_HIP;
}

}  // extern "C"

namespace {

// dte_plan_create after its null-pointer check; host containers may throw
// (the caller turns that into DTE_ERR_HOST), and nothing is allocated on the
// device until every host table is built.
dte_status plan_create(const dte_segment* segs, int32_t nseg, const dte_op* ops, int32_t nop,
                       int32_t nranks, const int64_t* rank_numel, dte_plan** out)
{
    if (!segs || nseg < 1 || nop < 0 || (nop > 0 && !ops) || nranks < 1 ||
        nranks > DTE_MAX_RANKS || !rank_numel)
        return DTE_ERR_ARG;
    for (int32_t r = 0; r < nranks; ++r)
        if (rank_numel[r] < 0) return DTE_ERR_ARG;
    int64_t total = 0;
    int32_t max_rep = 0;
    const dte_status st = validate_plan(segs, nseg, ops, nop, nranks, rank_numel, &total,
                                        &max_rep);
    if (st != DTE_OK) return st;

    // host images of the device tables
    std::vector<int64_t> seg_begin(nseg + 1);
    std::vector<uint32_t> seg_shape((size_t)nseg * DTE_MAX_DIMS, 1u);
    std::vector<int32_t> seg_ndim(nseg), seg_ops(nseg + 1, 0);
    for (int32_t s = 0; s < nseg; ++s) {
        seg_begin[s] = segs[s].flat_begin;
        seg_ndim[s] = segs[s].ndim;
        for (int d = 0; d < segs[s].ndim; ++d)
            seg_shape[(size_t)s * DTE_MAX_DIMS + d] = (uint32_t)segs[s].shape[d];
    }
    seg_begin[nseg] = total;
    for (int32_t k = 0; k < nop; ++k) seg_ops[ops[k].segment + 1]++;
    for (int32_t s = 0; s < nseg; ++s) seg_ops[s + 1] += seg_ops[s];
    std::vector<dte::DevOp> dops(nop > 0 ? nop : 1);
    {
        std::vector<int32_t> fill(seg_ops.begin(), seg_ops.end() - 1);
        for (int32_t k = 0; k < nop; ++k) {   // stable: input order within a segment
            const dte_op& o = ops[k];
            dte::DevOp& d = dops[fill[o.segment]++];
            std::memset(&d, 0, sizeof d);
            d.dst_base = o.dst_base;
            d.rank = o.rank;
            d.ndim = segs[o.segment].ndim;
            for (int i = 0; i < DTE_MAX_DIMS; ++i) {
                const bool used = i < d.ndim;
                d.src_origin[i] = used ? (uint32_t)o.src_origin[i] : 0u;
                d.extent[i] = used ? (uint32_t)o.extent[i] : 1u;
                d.dst_origin[i] = used ? (uint32_t)o.dst_origin[i] : 0u;
                d.dst_shape[i] = used ? (uint32_t)o.dst_shape[i] : 1u;
            }
        }
    }
    // bucket table: at most 2^20 buckets
    int32_t shift = 0;
    while ((total >> shift) > (int64_t(1) << 20)) ++shift;
    const int64_t nbuckets = (total >> shift) + 1;
    std::vector<int32_t> lookup(nbuckets);
    {
        int32_t s = 0;
        for (int64_t b = 0; b < nbuckets; ++b) {
            const int64_t first = b << shift;
            while (s + 1 < nseg && seg_begin[s + 1] <= first) ++s;
            lookup[b] = s;
        }
    }

    const size_t o_begin = 0;
    const size_t o_shape = align_up(o_begin + seg_begin.size() * sizeof(int64_t));
    const size_t o_ndim = align_up(o_shape + seg_shape.size() * sizeof(uint32_t));
    const size_t o_sops = align_up(o_ndim + seg_ndim.size() * sizeof(int32_t));
    const size_t o_ops = align_up(o_sops + seg_ops.size() * sizeof(int32_t));
    const size_t o_look = align_up(o_ops + dops.size() * sizeof(dte::DevOp));
    const size_t bytes = align_up(o_look + lookup.size() * sizeof(int32_t));

    std::vector<unsigned char> img(bytes, 0);
    std::memcpy(img.data() + o_begin, seg_begin.data(), seg_begin.size() * sizeof(int64_t));
    std::memcpy(img.data() + o_shape, seg_shape.data(), seg_shape.size() * sizeof(uint32_t));
    std::memcpy(img.data() + o_ndim, seg_ndim.data(), seg_ndim.size() * sizeof(int32_t));
    std::memcpy(img.data() + o_sops, seg_ops.data(), seg_ops.size() * sizeof(int32_t));
    std::memcpy(img.data() + o_ops, dops.data(), dops.size() * sizeof(dte::DevOp));
    std::memcpy(img.data() + o_look, lookup.data(), lookup.size() * sizeof(int32_t));
    std::unique_ptr<dte_plan> plan(new dte_plan);
    plan->dev_mem = nullptr;
    plan->rank_numel.assign(rank_numel, rank_numel + nranks);
    if (hipGetDevice(&plan->device) != hipSuccess || hipMalloc(&plan->dev_mem, bytes) != hipSuccess)
        return DTE_ERR_HIP;
    if (hipMemcpy(plan->dev_mem, img.data(), bytes, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(plan->dev_mem);
        return DTE_ERR_HIP;
    }
    unsigned char* base = static_cast<unsigned char*>(plan->dev_mem);
    plan->view.seg_begin = reinterpret_cast<const int64_t*>(base + o_begin);
    plan->view.seg_shape = reinterpret_cast<const uint32_t*>(base + o_shape);
    plan->view.seg_ndim = reinterpret_cast<const int32_t*>(base + o_ndim);
    plan->view.seg_ops = reinterpret_cast<const int32_t*>(base + o_sops);
    plan->view.ops = reinterpret_cast<const dte::DevOp*>(base + o_ops);
    plan->view.lookup = reinterpret_cast<const int32_t*>(base + o_look);
    plan->view.total = total;
    plan->view.nbuckets = nbuckets;
    plan->view.nseg = nseg;
    plan->view.shift = shift;
    plan->nseg = nseg;
    plan->nop = nop;
    plan->nranks = nranks;
    plan->max_replication = max_rep;
    plan->total = total;
    *out = plan.release();
    return DTE_OK;
}

}  // namespace

extern "C" {

dte_status dte_plan_create(const dte_segment* segs, int32_t nseg, const dte_op* ops,
                           int32_t nop, int32_t nranks, const int64_t* rank_numel,
                           dte_plan** out)
{
    if (!out) return DTE_ERR_ARG;
    *out = nullptr;
    return dte::no_throw(
        [&] { return plan_create(segs, nseg, ops, nop, nranks, rank_numel, out); });
}

void dte_plan_destroy(dte_plan* plan)
{
    if (!plan) return;
    if (plan->dev_mem) (void)hipFree(plan->dev_mem);
    delete plan;
}

dte_status dte_plan_info(const dte_plan* plan, int64_t* total, int32_t* nranks,
                         int32_t* max_replication)
{
    if (!plan) return DTE_ERR_ARG;
    if (total) *total = plan->total;
    if (nranks) *nranks = plan->nranks;
    if (max_replication) *max_replication = plan->max_replication;
    return DTE_OK;
}

dte_status dte_remap(const dte_plan* plan, const int64_t* idx, const uint16_t* val,
                     const int64_t* count, int64_t in_capacity, int64_t* const* out_off,
                     uint16_t* const* out_val, const int64_t* rank_capacity,
                     int64_t* rank_count, void* stream)
{
    if (!plan || !count || !out_off || !out_val || !rank_capacity || !rank_count ||
        in_capacity < 0 || !on_plan_device(plan))
        return DTE_ERR_ARG;
    if (in_capacity > 0 && (!idx || !val)) return DTE_ERR_ARG;
    for (int32_t r = 0; r < plan->nranks; ++r) {
        if (rank_capacity[r] < 0) return DTE_ERR_ARG;
        if (rank_capacity[r] > 0 && (!out_off[r] || !out_val[r])) return DTE_ERR_ARG;
    }
    hipStream_t s = (hipStream_t)stream;
    if (dte::launch_zero_i64(rank_count, plan->nranks, s) != hipSuccess) return DTE_ERR_HIP;
    const int cus = cu_count(plan->device);
    for (int32_t first = 0; first < plan->nranks; first += dte::kRanksPerLaunch) {
        dte::RankSlice sl;
        std::memset(&sl, 0, sizeof sl);
        sl.first = first;
        sl.count = std::min<int32_t>(dte::kRanksPerLaunch, plan->nranks - first);
        for (int32_t r = 0; r < sl.count; ++r) {
            sl.off[r] = out_off[first + r];
            sl.val[r] = out_val[first + r];
            sl.cap[r] = rank_capacity[first + r];
        }
        if (dte::launch_remap(plan->view, idx, val, count, in_capacity, sl, rank_count, cus, s) !=
            hipSuccess)
            return DTE_ERR_HIP;
    }
    return DTE_OK;
}

dte_status dte_extract_remap(const float* p, const float* m, const float* v, int64_t n,
                             int64_t index_base, const dte_adamw_step* hp, const dte_plan* plan,
                             int64_t* const* out_off, uint16_t* const* out_val,
                             const int64_t* rank_capacity, int64_t* rank_count, int64_t* count,
                             void* stream)
{
    if (!plan || !out_off || !out_val || !rank_capacity || !rank_count ||
        plan->nranks > dte::kRanksPerLaunch || !on_plan_device(plan))
        return DTE_ERR_ARG;
    if (!extract_args_ok(p, m, v, n, index_base, hp, nullptr, nullptr, 0, count))
        return DTE_ERR_ARG;
    for (int32_t r = 0; r < plan->nranks; ++r) {
        if (rank_capacity[r] < 0) return DTE_ERR_ARG;
        if (rank_capacity[r] > 0 && (!out_off[r] || !out_val[r])) return DTE_ERR_ARG;
    }
    if (n == 0) return DTE_OK;
    dte::ExtractParams a = extract_params(p, m, v, n, index_base, hp, nullptr, nullptr, 0, count,
                                          nullptr);
    a.route = 1;
    a.plan = plan->view;
    std::memset(&a.out, 0, sizeof a.out);
    a.out.first = 0;
    a.out.count = plan->nranks;
    for (int32_t r = 0; r < plan->nranks; ++r) {
        a.out.off[r] = out_off[r];
        a.out.val[r] = out_val[r];
        a.out.cap[r] = rank_capacity[r];
    }
    a.rank_count = rank_count;
    return dte::launch_extract(a, cu_count(plan->device), (hipStream_t)stream) == hipSuccess
               ? DTE_OK
               : DTE_ERR_HIP;
}

dte_status dte_apply(const dte_plan* plan, uint16_t* const* shards, const int64_t* const* off,
                     const uint16_t* const* val, const int64_t* rank_count,
                     const int64_t* rank_capacity, void* stream)
{
    if (!plan || !shards || !off || !val || !rank_count || !rank_capacity || !on_plan_device(plan))
        return DTE_ERR_ARG;
    for (int32_t r = 0; r < plan->nranks; ++r) {
        if (rank_capacity[r] < 0) return DTE_ERR_ARG;
        if (rank_capacity[r] > 0 && (!off[r] || !val[r])) return DTE_ERR_ARG;
        if (plan->rank_numel[r] > 0 && !shards[r]) return DTE_ERR_ARG;
    }
    const int cus = cu_count(plan->device);
    for (int32_t first = 0; first < plan->nranks; first += dte::kRanksPerLaunch) {
        dte::ApplySlice sl;
        std::memset(&sl, 0, sizeof sl);
        sl.first = first;
        sl.count = std::min<int32_t>(dte::kRanksPerLaunch, plan->nranks - first);
        for (int32_t r = 0; r < sl.count; ++r) {
            sl.shard[r] = shards[first + r];
            sl.off[r] = off[first + r];
            sl.val[r] = val[first + r];
            sl.cap[r] = rank_capacity[first + r];
            sl.numel[r] = plan->rank_numel[first + r];
        }
        if (dte::launch_apply(sl, rank_count, cus, (hipStream_t)stream) != hipSuccess)
            return DTE_ERR_HIP;
    }
    return DTE_OK;
}

}  // extern "C"
