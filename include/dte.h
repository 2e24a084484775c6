/*
 * dte.h -- C ABI of the snapshot-free delta-extraction hot path for
 * AMD Instinct MI355X (gfx950).
 *
 * The method (AReaL-DTE, "Delta Transfer Engine"): after an AdamW step,
 * rebuild the previous FP32 master weights from the live state instead of a
 * stored snapshot, find the elements whose BF16 (inference) bit pattern
 * changed, remap their trainer-side flat offsets into receiver-local shard
 * offsets, and write the new BF16 values into the receiver shards.
 *
 * Conventions for every call:
 *  - Plain C types only.  "device" pointers address GPU memory of the
 *    current HIP device; "host" pointers address CPU memory.  Every buffer
 *    is owned by the caller unless stated otherwise; the library keeps no
 *    pointer past the call except inside a dte_plan.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    The three hot calls only enqueue work: no allocation, no host
 *    synchronisation, no host<->device copies.
 *  - Return value: DTE_OK, or an error code; dte_status_string() names it.
 *    Argument errors are detected on the host before anything is enqueued.
 *    The library never aborts and never throws across this interface: a
 *    call that builds host tables or starts host threads returns
 *    DTE_ERR_HOST when host memory or a thread cannot be obtained.
 *  - Sizes are element counts (int64).  Zero-length inputs are legal and
 *    enqueue nothing.
 *  - Floating point: IEEE binary32, round-to-nearest-even, no fused
 *    multiply-add contraction, subnormals kept, correctly rounded divide and
 *    square root; the results are bit-reproducible.
 */
#ifndef DTE_H
#define DTE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dte_status;
#define DTE_OK 0
#define DTE_ERR_ARG 1      /* invalid argument (null pointer, bad size, bad hyperparameter) */
#define DTE_ERR_PLAN 2     /* transfer plan failed validation */
#define DTE_ERR_CAPACITY 3 /* a capacity beyond dte_ordered_noalloc_max_capacity(); overflow of
                             output buffers is reported through the counters instead */
#define DTE_ERR_HIP 4      /* a HIP runtime call failed */
#define DTE_ERR_IO 5       /* a file could not be read or written (dte_store.h) */
#define DTE_ERR_CORRUPT 6  /* stored data failed its checksum or format check */
#define DTE_ERR_CHAIN 7    /* a stored version does not extend the local base version */
#define DTE_ERR_UNSUPPORTED 8 /* the requested codec is not available on this host */
#define DTE_ERR_HOST 9     /* a host resource (memory, a thread) could not be obtained */

#define DTE_MAX_DIMS 4     /* tensor rank limit of segments and plan operations */
#define DTE_MAX_RANKS 64   /* receiver ranks per plan */

#define DTE_ORDER_FOLDED 0   /* bias corrections folded into two scalars */
#define DTE_ORDER_LITERAL 1  /* eq. adamw_inverse as printed: four divisions */

/* Hyperparameters of one AdamW step of one parameter group (paper sec. 4.1,
 * eq. adamw_moments and eq. adamw_inverse; appendix A): learning rate eta_t,
 * moment coefficients beta1, beta2, epsilon, the group's decoupled weight
 * decay lambda, and the step index t of the step just taken (t >= 1);
 * `order` selects the binary32 operation order of the step and its inverse
 * (DTE_ORDER_FOLDED or DTE_ORDER_LITERAL, see dte_scalars); `reserved` must
 * be 0.  Valid: lr >= 0 finite, 0 <= beta < 1, eps >= 0 finite,
 * 1 - lr*wd > 0. */
typedef struct {
    double lr;
    double beta1;
    double beta2;
    double eps;
    double weight_decay;
    int64_t step;
    int32_t order;
    int32_t reserved;
} dte_adamw_step;

/* The step scalars of the inverse, each computed in binary64 from
 * dte_adamw_step and rounded once to binary32:
 *   lrb1  = lr / (1 - beta1^t)      rbc2  = 1 / (1 - beta2^t)
 *   eps   = eps                     decay = 1 - lr * weight_decay
 *   lr    = lr                      bc1 = 1 - beta1^t,  bc2 = 1 - beta2^t
 * With them the inverse of sec. 4.1, eq. adamw_inverse, is evaluated per
 * element, left to right, as
 *   folded:  u = (lrb1 * m) / (sqrt(v * rbc2) + eps)
 *   literal: u = lr * ((m / bc1) / (sqrt(v / bc2) + eps))
 *   theta_hat = (theta + u) / decay
 * (folded: the bias corrections folded into two scalars, as a fused
 * optimizer folds them; literal: the printed expression, four divisions).
 * dte_adamw_forward uses the same u. */
typedef struct {
    float lrb1;
    float rbc2;
    float eps;
    float decay;
    float lr;
    float bc1;
    float bc2;
    int32_t order;
} dte_scalars;

/* Host-only.  Derive the scalars above.  Errors: DTE_ERR_ARG for a null
 * pointer or an invalid dte_adamw_step. */
dte_status dte_derive_scalars(const dte_adamw_step* hp, dte_scalars* out);

/* Extract the BF16-visible delta of one contiguous range of the flat
 * trainer shard (paper sec. 4.1 reconstruction; sec. 4.2.1 eq.
 * canonical_delta_detection).
 *
 * For each element i in [0, n):
 *   theta_hat = inverse(p[i], m[i], v[i])            (sec. 4.1, see dte_scalars;
 *                                                     in hp->order)
 *   b_old = BF16(theta_hat), b_new = BF16(p[i])     (round to nearest even on
 *           the binary32 pattern; overflow to +-inf; any NaN -> 0x7FC0)
 *   changed if b_old != b_new as 16-bit patterns     (+0 and -0 differ)
 * and every changed element appends one entry
 *   out_idx = index_base + i   (flat trainer offset)
 *   out_val = b_new            (target BF16 pattern, not a difference)
 *
 * p, m, v : device, n binary32 each: theta_t, m_t, v_t of the range,
 *           element-aligned (paper sec. 4.1: optimizer-native slices).
 *           16-byte alignment of p, m, v (equal modulo 16) enables vector loads.
 * index_base : flat trainer offset of p[0]; >= 0.
 * hp      : host; the step's hyperparameters (one parameter group per call;
 *           several groups = several calls on their sub-ranges).
 * out_idx : device int64[capacity]; out_val: device uint16[capacity].
 * cursor  : device int64, append semantics: on entry the fill level of
 *           out_idx/out_val (0 for a fresh delta, below 2^36), on completion
 *           the total number of entries including those that did not fit.
 *           Entries at positions >= capacity are dropped; after a stream
 *           synchronisation, *cursor > capacity means the delta is
 *           incomplete and must be recomputed with capacity >= *cursor.
 *           While the call runs, its bits from 36 up count the work units
 *           that blocks take (cleared by the call's last kernel).
 * out_prev: device binary32[n] receiving theta_hat, or NULL (no write).
 * Entry order is unspecified (the set of entries is exact; each wave of the
 * kernel writes its entries in ascending runs); offsets are unique within
 * one call; dte_extract_delta_ordered gives ascending order.  Errors: DTE_ERR_ARG (null pointer with n > 0,
 * n < 0, index_base < 0, capacity < 0, invalid hp), DTE_ERR_HIP. */
dte_status dte_extract_delta(const float* p, const float* m, const float* v, int64_t n,
                             int64_t index_base, const dte_adamw_step* hp, int64_t* out_idx,
                             uint16_t* out_val, int64_t capacity, int64_t* cursor,
                             float* out_prev, void* stream);

/* Bytes of device workspace that dte_extract_delta_ordered needs for a
 * given capacity (about 20 bytes per entry of capacity plus a fixed
 * 0.8 MB); -1 if capacity is negative or above 2^40. */
int64_t dte_ordered_workspace_bytes(int64_t capacity);

/* dte_extract_delta with the entries in ascending offset order (paper
 * sec. 4.2.2 asks for an ordered sparse payload per sender-receiver pair):
 * the same set of entries, written to out_idx / out_val at positions
 * *cursor, *cursor + 1, ... sorted by offset, and the same cursor
 * semantics.  The order does not depend on timing: repeated calls on the
 * same input write identical bytes.  Successive calls on ascending
 * sub-ranges (parameter groups) keep the whole delta ascending.
 * workspace: device memory of at least dte_ordered_workspace_bytes(capacity)
 *            bytes, 256-byte aligned, owned by the caller, not read by the
 *            caller afterwards; calls that overlap on one workspace race.
 * If the true total exceeds capacity the output holds an unspecified
 * subset (recompute with capacity >= *cursor - entry value).
 * Errors: as dte_extract_delta; DTE_ERR_ARG also for a missing, small or
 * misaligned workspace. */
dte_status dte_extract_delta_ordered(const float* p, const float* m, const float* v, int64_t n,
                                     int64_t index_base, const dte_adamw_step* hp,
                                     int64_t* out_idx, uint16_t* out_val, int64_t capacity,
                                     int64_t* cursor, void* workspace, int64_t workspace_bytes,
                                     float* out_prev, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * ordered call of dte_extract_delta_ordered with its workspace in a static
 * array of 64 MiB that the library holds on every device it runs on until
 * the process ends, so the call needs no workspace argument and allocates
 * nothing (no hipMalloc, no hipFree, no allocating library routine).
 * Arguments, results, order and cursor semantics are those of
 * dte_extract_delta_ordered.  The array is shared by every call on one
 * device and keeps the last call's contents; calls that overlap on one
 * device (several streams or host threads) race and must be serialised by
 * the caller.
 * capacity: at most dte_ordered_noalloc_max_capacity() (about 3.3 million
 *           entries), else DTE_ERR_CAPACITY and nothing is enqueued.
 * Errors: as dte_extract_delta; DTE_ERR_CAPACITY; DTE_ERR_HIP also when the
 * array's device address cannot be obtained. */
dte_status dte_extract_delta_ordered_noalloc(const float* p, const float* m, const float* v,
                                             int64_t n, int64_t index_base,
                                             const dte_adamw_step* hp, int64_t* out_idx,
                                             uint16_t* out_val, int64_t capacity,
                                             int64_t* cursor, float* out_prev, void* stream);

/* Host-only.  The largest capacity dte_extract_delta_ordered_noalloc
 * accepts. */
int64_t dte_ordered_noalloc_max_capacity(void);

/* One canonical parameter of the flat trainer shard (paper sec. 4.2.2:
 * sender-local converted tensor of shape n_s): flat_begin is its offset in
 * the shard, shape[0..ndim) its row-major extents (ndim in 1..4). */
typedef struct {
    int64_t flat_begin;
    int32_t ndim;
    int32_t reserved;
    int64_t shape[DTE_MAX_DIMS];
} dte_segment;

/* One operation o of the transfer plan T (paper sec. 4.2.2): the
 * hyperrectangular overlap between segment `segment` (shape n_s) and a
 * receiver-local view of shape dst_shape (n_r) that starts at flat offset
 * dst_base of receiver rank `rank`'s buffer.  Source origin a_s, extent e,
 * destination origin a_r; all with the segment's ndim.  A change at
 * coordinate u of the segment belongs to o when a_s <= u < a_s + e
 * component-wise (containment) and lands at
 *   dst_base + ravel(u - a_s + a_r, dst_shape)   (eq. receiver_local_remapping). */
typedef struct {
    int32_t segment;
    int32_t rank;
    int64_t dst_base;
    int64_t src_origin[DTE_MAX_DIMS];
    int64_t extent[DTE_MAX_DIMS];
    int64_t dst_origin[DTE_MAX_DIMS];
    int64_t dst_shape[DTE_MAX_DIMS];
} dte_op;

/* Opaque, immutable once created; owns device copies of the tables; may be
 * shared by concurrent calls on any streams of the device it was created on. */
typedef struct dte_plan dte_plan;

/* Validate and upload a transfer plan (paper sec. 4.2.2; Observation 3:
 * layouts and therefore T are fixed before synchronisation).
 *
 * segs : host, nseg segments sorted by flat_begin, contiguous from 0 (they
 *        tile [0, total)); each numel < 2^32 and each extent < 2^31.
 * ops  : host, nop operations, any order.
 * nranks, rank_numel: receiver count (1..DTE_MAX_RANKS) and each rank's
 *        buffer length in BF16 elements (host int64[nranks]).
 * Validation (DTE_ERR_PLAN on failure):
 *  - every box lies inside its segment and its destination view, and every
 *    view inside its rank's buffer;
 *  - views of one rank are identical (same dst_base and dst_shape) or have
 *    disjoint flat ranges, and boxes inside one view are disjoint, so every
 *    receiver element has at most one writer (apply is race-free);
 *  - the boxes of one segment sent to one rank are disjoint (one entry per
 *    element per rank), and together the segment's boxes cover every
 *    element (no change can be lost).
 * A canonical element may go to several ranks (replication).
 * *out receives the plan (NULL on error); the caller releases it with
 * dte_plan_destroy.  The plan belongs to the device current at creation:
 * dte_remap, dte_extract_remap and dte_apply return DTE_ERR_ARG when called
 * with another current device.
 * Errors: DTE_ERR_ARG, DTE_ERR_PLAN, DTE_ERR_HIP, DTE_ERR_HOST.  Allocates
 * device memory; not a hot-path call. */
dte_status dte_plan_create(const dte_segment* segs, int32_t nseg, const dte_op* ops,
                           int32_t nop, int32_t nranks, const int64_t* rank_numel,
                           dte_plan** out);

/* Release a plan (NULL is ignored).  The caller must ensure no enqueued
 * work still uses it (synchronise the streams first). */
void dte_plan_destroy(dte_plan* plan);

/* Host-only.  Total trainer elements covered by the plan, its receiver
 * count, and the largest number of receivers any element goes to (the
 * bound rank_capacity needs per input entry).  Any output may be NULL. */
dte_status dte_plan_info(const dte_plan* plan, int64_t* total, int32_t* nranks,
                         int32_t* max_replication);

/* Remap a delta into per-receiver buckets (paper sec. 4.2.2: unravel
 * eq. canonical_unravel, containment, ravel eq. receiver_local_remapping;
 * partition or replication per the plan).
 *
 * idx, val   : device, the entries of dte_extract_delta (flat trainer offset,
 *              target BF16 pattern).
 * count      : device int64, number of entries produced (the extract
 *              cursor); min(*count, in_capacity) entries are read.
 * out_off[r], out_val[r] : host array of nranks device pointers to int64 /
 *              uint16 buckets of rank_capacity[r] (host int64[nranks])
 *              entries: receiver-local flat offset and value.
 * rank_count : device int64[nranks], written: entries routed to each rank
 *              (the per-receiver sizes that the paper's first transfer round
 *              sends, zeros included, sec. 4.3).  rank_count[r] >
 *              rank_capacity[r] after synchronisation means bucket r is
 *              incomplete.  Offsets within a bucket are unique; order
 *              unspecified.  Entries whose idx lies outside the plan are
 *              ignored.
 * Errors: DTE_ERR_ARG, DTE_ERR_HIP. */
dte_status dte_remap(const dte_plan* plan, const int64_t* idx, const uint16_t* val,
                     const int64_t* count, int64_t in_capacity, int64_t* const* out_off,
                     uint16_t* const* out_val, const int64_t* rank_capacity,
                     int64_t* rank_count, void* stream);

/* dte_extract_delta and dte_remap in one pass (paper sec. 4.2.1: changed
 * indices are remapped as soon as they are detected): the changed entries
 * of [index_base, index_base + n) are routed through `plan` straight into
 * the receiver buckets, without the (I, V) arrays.  Arguments as in those
 * two calls; the plan has at most 16 ranks.  Unlike dte_remap, rank_count
 * is not cleared: each call adds its routed entries to it (and to *count,
 * device int64, the number of changed entries), so one step over several
 * parameter-group ranges clears both once, before its first call.  Entries
 * beyond rank_capacity[r] are dropped and counted; bucket order is
 * unspecified.  No theta_hat output.  Errors: DTE_ERR_ARG, DTE_ERR_HIP. */
dte_status dte_extract_remap(const float* p, const float* m, const float* v, int64_t n,
                             int64_t index_base, const dte_adamw_step* hp, const dte_plan* plan,
                             int64_t* const* out_off, uint16_t* const* out_val,
                             const int64_t* rank_capacity, int64_t* rank_count, int64_t* count,
                             void* stream);

/* Direct sparse apply (paper sec. 4.3, eq. direct_sparse_apply):
 * shards[r][off[r][k]] = val[r][k] for k < min(rank_count[r],
 * rank_capacity[r]), every rank r.  Because values are targets, applying a
 * delta twice equals applying it once.
 * shards : host array of nranks device pointers to BF16 (uint16) buffers of
 *          the plan's rank_numel[r] elements.
 * off, val, rank_count, rank_capacity: as produced/used by dte_remap.
 * Offsets outside a shard are ignored.  Errors: DTE_ERR_ARG, DTE_ERR_HIP. */
dte_status dte_apply(const dte_plan* plan, uint16_t* const* shards, const int64_t* const* off,
                     const uint16_t* const* val, const int64_t* rank_count,
                     const int64_t* rank_capacity, void* stream);

/* The trainer-side step that dte_extract_delta inverts (paper sec. 4.1,
 * eq. adamw_moments; appendix A, eq. appendix_adamw_forward), in place on
 * device buffers p, m, v (theta, m, v of step t-1 in, of step t out) with
 * gradient g, n elements each, in the same binary32 operation order:
 *   m = beta1*m + (1-beta1)*g;  v = beta2*v + (1-beta2)*(g*g);
 *   u as in dte_scalars for hp->order;  p = decay*p - u
 * (beta1, beta2, 1-beta1, 1-beta2 rounded once to binary32).  Provided so
 * a trainer (or a test) can produce states whose inverse is exact up to the
 * rounding of p.  Errors: DTE_ERR_ARG, DTE_ERR_HIP. */
dte_status dte_adamw_forward(float* p, float* m, float* v, const float* g, int64_t n,
                             const dte_adamw_step* hp, void* stream);

/* Static string naming a status code. */
const char* dte_status_string(dte_status status);

#ifdef __cplusplus
}
#endif

#endif /* DTE_H */
