/*
 * dit_migrate.h -- C ABI of layout-aware artifact migration.
 *
 * When two adjacent trajectory tasks run under different execution layouts
 * (for example sequence-parallel groups of different sizes), each artifact is
 * rebuilt under the consumer's layout (section 5.3, Layout-Aware Artifact
 * Migration).  dit_migration_plan derives the transfers from the producer and
 * consumer views of one field: for a sharded tensor, every non-empty
 * intersection of a source-owned slice with a destination-required slice is
 * one entry (source rank, destination rank, source range, destination range,
 * bytes); a replicated field sends the whole tensor to each destination (from
 * the source on the same rank if there is one, else from source j mod n_src to
 * the j-th destination); a metadata-only field sends nothing.  Entries come
 * destination by destination, and within one destination source by source, in
 * the order the slices are given.
 *
 * A slice is a half-open box [start, end) in the field's global coordinates
 * (1 to 4 dimensions), held densely and row-major on its rank.  Ranges in an
 * entry are offsets inside the source and destination slices plus a common
 * extent.
 *
 * dit_migration_execute applies a plan on one GPU, where device buffers stand
 * in for the ranks' slices; it is how the plan is checked and timed on one
 * GPU.  Across GPUs each entry would be one point-to-point transfer: the
 * source packs its range, the destination installs it.
 */
#ifndef DIT_MIGRATE_H
#define DIT_MIGRATE_H

#include <stdint.h>

#include "dit_block.h"

#ifdef __cplusplus
extern "C" {
#endif

#define DIT_MIG_MAX_DIMS 4

typedef enum { DIT_MIG_SHARDED = 0, DIT_MIG_REPLICATED = 1, DIT_MIG_METADATA = 2 } dit_mig_kind;

typedef struct {
  int32_t rank;
  int64_t start[DIT_MIG_MAX_DIMS]; /* first n_dims entries used */
  int64_t end[DIT_MIG_MAX_DIMS];
} dit_mig_slice;

typedef struct {
  dit_mig_kind kind;
  int n_dims;                        /* 1..4 */
  int64_t shape[DIT_MIG_MAX_DIMS];   /* global shape */
  int elem_bytes;                    /* 1, 2, 4, 8 or 16 */
  int n_src;                         /* >= 1 unless metadata-only */
  const dit_mig_slice *src;          /* host [n_src]: the producer's slices */
  int n_dst;                         /* >= 0 */
  const dit_mig_slice *dst;          /* host [n_dst]: the consumer's slices */
} dit_mig_field;

typedef struct {
  int32_t src_index, dst_index;      /* positions in f->src and f->dst */
  int32_t src_rank, dst_rank;
  int64_t src_off[DIT_MIG_MAX_DIMS];
  int64_t dst_off[DIT_MIG_MAX_DIMS];
  int64_t extent[DIT_MIG_MAX_DIMS];
  int64_t bytes;
} dit_mig_entry;

/* The plan of one field.  *n_entries receives the number of entries; they are
 * written to `entries` (host) when capacity allows, else DIT_ERR_WORKSPACE is
 * returned and nothing is written (call with entries NULL, capacity 0 to
 * size).  Every slice must lie inside the shape; a replicated field's slices
 * must cover the whole shape. */
dit_status dit_migration_plan(const dit_mig_field *f, dit_mig_entry *entries, int64_t capacity,
                              int64_t *n_entries);

/* Apply `n` entries of a plan of `f` on the current device: src_bufs[i] and
 * dst_bufs[j] (host arrays of device pointers, 16-byte aligned) hold source
 * slice i and destination slice j densely.  Asynchronous on `stream`;
 * destination bytes not covered by any entry are left as they are. */
dit_status dit_migration_execute(const dit_mig_field *f, const dit_mig_entry *entries, int64_t n,
                                 const void *const *src_bufs, void *const *dst_bufs, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DIT_MIGRATE_H */
