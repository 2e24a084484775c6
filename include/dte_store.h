/*
 * dte_store.h -- storage-mediated publication of sparse BF16 deltas
 * (AReaL-DTE, paper sec. 4.4, cross-cluster transfer).
 *
 * Across clusters there is no communication group between trainer and
 * rollout workers, so a version's canonical sparse changes (the (I, V) of
 * sec. 4.2.1, one entry per changed canonical element) travel through a
 * shared filesystem: writer ranks serialise only the changed index-value
 * pairs of the partitions they own into compressed chunks, staged through
 * a bounded pinned-memory pipeline; a coordinator commits a version
 * manifest (version chain, chunk locations, lengths, checksums) after every
 * writer has reported, including writers without changes; a version with
 * no changed entry is not published.  The destination checks that a
 * committed version extends the version it last applied, verifies every
 * chunk and scatters the entries into its own layout (dte_remap and
 * dte_apply with its receiver plan).
 *
 * Directory layout under `dir`:
 *   v<version>/chunk-<writer>-<k>.dte   one compressed chunk
 *   v<version>/part-<writer>.json       a writer's chunk list
 *   v<version>/manifest.json            the committed version
 *   LATEST                              the newest committed version number
 * Files are written to a temporary name and renamed into place, manifest
 * before LATEST, so a reader never sees a partial version.
 *
 * Chunk file: a 40-byte header (magic "DTEC", format 1, segment, index
 * transform, first entry (ordinal among the writer's entries of the
 * segment), count, payload bytes), then the payload (count
 * uint32 segment-local indices, ascending, stored as gaps with transform 1
 * or as values with transform 0, then count uint16 BF16 patterns), either
 * verbatim (codec none) or as one Zstandard frame (codec zstd).  The
 * manifest records each file's XXH64 (seed 0) of its bytes as stored.
 *
 * Conventions of dte.h apply; these calls allocate, synchronise and do file
 * I/O (they are not hot-path calls).  Errors: DTE_ERR_ARG, DTE_ERR_IO,
 * DTE_ERR_CORRUPT, DTE_ERR_CHAIN, DTE_ERR_UNSUPPORTED, DTE_ERR_HIP,
 * DTE_ERR_HOST.
 */
#ifndef DTE_STORE_H
#define DTE_STORE_H

#include <stdint.h>

#include "dte.h"

#ifdef __cplusplus
extern "C" {
#endif

/* One canonical parameter of the flat index space: entries with
 * flat_begin <= idx < flat_begin + numel belong to it (numel < 2^32).
 * Segments are sorted by flat_begin and do not overlap. */
typedef struct {
    const char* name;   /* canonical parameter name, UTF-8 without quotes or
                           backslashes; NULL is stored as "" */
    int64_t flat_begin;
    int64_t numel;
} dte_store_segment;

/* A contiguous range [sender_begin, sender_end) of the writer's flat shard
 * that holds whole rows of a box of canonical segment `segment` (the
 * converter's map for a trainer layout such as Megatron-Core, sec. 4.2.1
 * and appendix B): shard element sender_begin + q, with q = row *
 * local_cols + col, is element (canon_row0 + row, canon_col0 + col) of the
 * segment viewed as rows of canon_cols, i.e. its canonical local index is
 * (canon_row0 + row) * canon_cols + canon_col0 + col.  segment = -1: the
 * range's entries are published by another writer (replicated tensors).
 * Pieces are sorted by sender_begin and disjoint; the pieces a writer
 * publishes for one segment cover ascending, disjoint canonical ranges. */
typedef struct {
    int64_t sender_begin;
    int64_t sender_end;
    int32_t segment;
    int32_t reserved;
    int64_t local_cols;
    int64_t canon_cols;
    int64_t canon_row0;
    int64_t canon_col0;
} dte_store_piece;

typedef struct {
    int32_t codec;           /* 0: none, 1: zstd (needs libzstd.so.1 at run time) */
    int32_t level;           /* zstd level 1..19 */
    int32_t threads;         /* host serialisation threads, 1..64 */
    int32_t index_transform; /* 0: indices as values, 1: as gaps (smaller after zstd) */
    int64_t chunk_entries;   /* entries per chunk at most, 1..2^26; bounds the pinned
                                staging (6 bytes per entry per slot, threads + 2 slots) */
} dte_store_options;

typedef struct {
    int64_t entries;          /* entries written or read */
    int64_t chunks;
    int64_t raw_bytes;        /* payload bytes before compression */
    int64_t stored_bytes;     /* chunk bytes on storage, headers included */
} dte_store_stats;

/* Writer rank `writer` (0..4095) stores its entries of version `version`
 * (>= 1): count entries with ascending, unique flat offsets idx (int64)
 * and BF16 patterns val, every offset inside one of the nseg segments.
 * Writes the chunks and part-<writer>.json (also when count == 0, so the
 * coordinator knows the writer reported).  Host arrays. */
dte_status dte_store_write_part_host(const char* dir, int64_t version, int32_t writer,
                                     const dte_store_segment* segs, int32_t nseg,
                                     const int64_t* idx, const uint16_t* val, int64_t count,
                                     const dte_store_options* opt, dte_store_stats* stats);

/* As dte_store_write_part_host, from device arrays: idx / val hold
 * min(*count, capacity) entries (the output of dte_extract_delta_ordered;
 * *count > capacity is DTE_ERR_ARG since the delta is incomplete).  On the
 * device the offsets become 32-bit segment-local indices; chunks then move
 * through the pinned staging ring to the host threads.  Work on `stream`
 * is waited for. */
dte_status dte_store_write_part_device(const char* dir, int64_t version, int32_t writer,
                                       const dte_store_segment* segs, int32_t nseg,
                                       const int64_t* idx, const uint16_t* val,
                                       const int64_t* count, int64_t capacity,
                                       const dte_store_options* opt, dte_store_stats* stats,
                                       void* stream);

/* Coordinator: once part-0 .. part-(nwriters-1) of `version` exist, commit
 * the version with parent `parent` (the previously committed version, 0
 * for the first): *committed = 1 and manifest.json then LATEST written.  If
 * the parts hold no entry at all, nothing is published (*committed = 0,
 * the version directory is removed, LATEST unchanged).  A missing part is
 * DTE_ERR_IO with nothing published.  Several writers may publish entries
 * of one segment (tensor-parallel trainer ranks); their entries must be
 * disjoint, which the writers' piece tables guarantee. */
dte_status dte_store_commit(const char* dir, int64_t version, int64_t parent, int32_t nwriters,
                            int32_t* committed);

/* Newest committed version (*version = 0 when none). */
dte_status dte_store_latest(const char* dir, int64_t* version);

/* Versions after `base` up to `latest`, oldest first, following parents
 * back from `latest`: out[0..*n).  DTE_ERR_CHAIN if the chain does not reach
 * `base`; DTE_ERR_ARG if more than max versions. */
dte_status dte_store_chain(const char* dir, int64_t base, int64_t latest, int64_t* out,
                           int32_t max, int32_t* n);

/* Entries of committed version `version`, whose parent must equal `base`
 * (the version the destination applied last; else DTE_ERR_CHAIN): every
 * chunk is checked against its manifest length and XXH64 and its own
 * header before use (DTE_ERR_CORRUPT).  Output: flat offsets (segment
 * flat_begin from the manifest + local index) and values, grouped by
 * segment, then writer, ascending within each (segment, writer) group
 * (ascending overall when every segment has a single writer);
 * *count = the version's entry total; entries beyond capacity are not
 * written (then call again with capacity >= *count). */
dte_status dte_store_read_host(const char* dir, int64_t version, int64_t base, int64_t* idx,
                               uint16_t* val, int64_t capacity, int64_t* count,
                               int32_t threads, dte_store_stats* stats);

/* As dte_store_read_host into device arrays: chunks are verified and
 * decoded by the host threads into pinned staging and copied to the
 * device; the offsets are widened on the device.  *count is host memory.
 * Work on `stream` is complete on return. */
dte_status dte_store_read_device(const char* dir, int64_t version, int64_t base, int64_t* idx,
                                 uint16_t* val, int64_t capacity, int64_t* count,
                                 int32_t threads, dte_store_stats* stats, void* stream);

/* As dte_store_write_part_host / _device for a writer whose shard is not
 * laid out as the canonical segments: idx are offsets in the writer's flat
 * shard, mapped to canonical segments by `pieces` (npiece entries). */
dte_status dte_store_write_part_host_mapped(const char* dir, int64_t version, int32_t writer,
                                            const dte_store_segment* segs, int32_t nseg,
                                            const dte_store_piece* pieces, int32_t npiece,
                                            const int64_t* idx, const uint16_t* val, int64_t count,
                                            const dte_store_options* opt, dte_store_stats* stats);

dte_status dte_store_write_part_device_mapped(const char* dir, int64_t version, int32_t writer,
                                              const dte_store_segment* segs, int32_t nseg,
                                              const dte_store_piece* pieces, int32_t npiece,
                                              const int64_t* idx, const uint16_t* val,
                                              const int64_t* count, int64_t capacity,
                                              const dte_store_options* opt, dte_store_stats* stats,
                                              void* stream);

/* XXH64 of n bytes with the given seed (the chunk checksum). */
uint64_t dte_store_xxh64(const void* data, int64_t n, uint64_t seed);

#ifdef __cplusplus
}
#endif

#endif /* DTE_STORE_H */
