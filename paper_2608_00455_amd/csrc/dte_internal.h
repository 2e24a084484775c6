// Internal declarations shared by the host API (dte_api.hip) and the kernel
// translation units (extract.hip, remap.hip).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dte.h"

namespace dte {

// ---- transfer plan on the device ----------------------------------------

constexpr int kRanksPerLaunch = 16;   // per-rank pointers travel as kernel arguments

struct DevOp {
    int64_t dst_base;
    int32_t rank;
    int32_t ndim;
    uint32_t src_origin[DTE_MAX_DIMS];
    uint32_t extent[DTE_MAX_DIMS];
    uint32_t dst_origin[DTE_MAX_DIMS];
    uint32_t dst_shape[DTE_MAX_DIMS];
};

struct PlanView {
    const int64_t* seg_begin;   // nseg + 1 (last = total)
    const uint32_t* seg_shape;  // nseg * DTE_MAX_DIMS
    const int32_t* seg_ndim;    // nseg
    const int32_t* seg_ops;     // nseg + 1, CSR into ops (by segment)
    const DevOp* ops;           // nop
    const int32_t* lookup;      // nbuckets: segment holding element (b << shift)
    int64_t total;
    int64_t nbuckets;
    int32_t nseg;
    int32_t shift;
};

struct RankSlice {                 // ranks [first, first + count) of one launch
    int32_t first;
    int32_t count;
    int64_t* off[kRanksPerLaunch];
    uint16_t* val[kRanksPerLaunch];
    int64_t cap[kRanksPerLaunch];
};

// ---- extract (fused AdamW inverse + BF16 detection + compaction) --------

// One flush of one wave in ordered mode: `count` entries written at
// unordered position `src`, preceded in the wave's ascending output by
// `woff` entries of earlier flushes.
struct OrderRun {
    int64_t src;
    int64_t woff;
    int32_t count;
    int32_t wave;         // global wave number (launch order)
};

// Operation order of the step and its inverse (dte_scalars).
struct ExtractParams {
    const float* p;
    const float* m;
    const float* v;
    int64_t n;            // elements of this call
    int64_t index_base;   // flat trainer offset of element 0
    float lrb1, rbc2, eps, decay;
    float rd_lo, rd_hi;   // binary32 bracket of 1/decay: rd_lo <= 1/decay <= rd_hi
    int32_t literal;      // order: 0 folded, 1 literal
    float lr, bc1, bc2;   // literal order
    int32_t lit_filter;   // literal order: the "unchanged" proof may be used
    float floor;          // literal order: additive term of the proof's bound
    int64_t* out_idx;
    uint16_t* out_val;
    int64_t capacity;
    int64_t* cursor;
    float* out_prev;      // nullable
    // ordered mode (runs != nullptr): wave g writes its first flushes to its
    // own region [g region_size, (g+1) region_size) of region_idx/region_val
    // (no atomics) and the number of entries there to region_count[g]; the
    // flushes that no longer fit go to out_idx/out_val at positions from the
    // cursor and are recorded in runs; every wave writes its entry total to
    // wave_count[wave]
    OrderRun* runs;
    int64_t max_runs;
    int64_t* run_cursor;
    int64_t* wave_count;
    int64_t* region_idx;
    uint16_t* region_val;
    int64_t* region_count;
    int64_t region_size;      // entries per wave region
    int32_t wave0;        // global number of this launch's first wave
    // routing mode (route != 0): each flush sends its entries through the
    // plan into the receiver buckets (out, counts added to rank_count)
    // instead of writing (out_idx, out_val); the cursor still counts them
    int32_t route;
    PlanView plan;
    RankSlice out;
    int64_t* rank_count;
};

// Largest number of waves one extract call launches in ordered mode.
constexpr int kMaxOrderedWaves = 16384;
// Entries a wave stages before it flushes them: every flush but a wave's
// last holds exactly this many (the ordered workspace is sized with it).
constexpr int kWaveStage = 1536;

// Launches the extract kernels; *waves receives the number of waves
// launched (the global wave numbers are 0 .. *waves - 1).
hipError_t launch_extract(const ExtractParams& a, int cus, hipStream_t stream,
                          int32_t* waves = nullptr);

// The number of waves launch_extract(a, cus, ...) launches.
int64_t extract_waves(const ExtractParams& a, int cus);

// Ordered mode, after launch_extract: wave_base[g] = *cursor + entries of
// waves < g; copies every wave's region part to (out_idx, out_val) at
// wave_base[g] and every recorded run from the shared area at
// wave_base[run.wave] + run.woff (positions below capacity); then *cursor
// += the total of the wave counts.
struct OrderParams {
    const OrderRun* runs;
    const int64_t* run_cursor;
    int64_t max_runs;
    const int64_t* wave_count;
    int64_t* wave_base;
    int32_t waves;
    const int64_t* src_idx;
    const uint16_t* src_val;
    int64_t src_capacity;
    const int64_t* region_idx;
    const uint16_t* region_val;
    const int64_t* region_count;
    int64_t region_size;
    int64_t* out_idx;
    uint16_t* out_val;
    int64_t capacity;
    int64_t* cursor;
};

hipError_t launch_order(const OrderParams& o, int cus, hipStream_t stream);

struct ForwardParams {
    float* p;
    float* m;
    float* v;
    const float* g;
    int64_t n;
    float lrb1, rbc2, eps, decay, b1, b2, omb1, omb2;
    float lr, bc1, bc2;
    int32_t literal;
};

hipError_t launch_adamw_forward(const ForwardParams& a, int cus, hipStream_t stream);

hipError_t launch_zero_i64(int64_t* p, int64_t n, hipStream_t stream);

hipError_t launch_remap(const PlanView& plan, const int64_t* idx, const uint16_t* val,
                        const int64_t* count, int64_t in_capacity, const RankSlice& out,
                        int64_t* rank_count, int cus, hipStream_t stream);

struct ApplySlice {
    int32_t first;
    int32_t count;
    uint16_t* shard[kRanksPerLaunch];
    const int64_t* off[kRanksPerLaunch];
    const uint16_t* val[kRanksPerLaunch];
    int64_t cap[kRanksPerLaunch];
    int64_t numel[kRanksPerLaunch];
};

hipError_t launch_apply(const ApplySlice& s, const int64_t* rank_count, int cus,
                        hipStream_t stream);

}  // namespace dte
