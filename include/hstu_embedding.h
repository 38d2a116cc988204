/*
 * hstu_embedding.h -- C ABI of the jagged multi-table embedding lookup
 * (paper Sec. 4.1.2, "Jagged Embedding Lookup Acceleration").
 *
 * Operation.  The paper looks sparse features up over explicit jagged
 * indices (offsets instead of per-sample lengths, so no padding ids and no
 * zero checks exist) and regroups a batch by table, spreading each table's
 * ids evenly over the compute units so that all of them work on the same
 * table at the same time (cache locality, no hot/cold-table imbalance).
 * This library computes the non-pooled lookup that sequence models use:
 *
 *   tables t = 0 .. F-1 are the row ranges [row_offsets[t], row_offsets[t+1])
 *   of one weight matrix W [total_rows][D];
 *   the ids of table t are ids[id_offsets[t] .. id_offsets[t+1]-1]
 *   (table-major: all ids of table 0, then table 1, ...);
 *   forward:  out(r) = W[row_offsets[t] + ids[r]]   for id position r of table t;
 *   backward: dW[g]  = sum of dout(r) over the positions r whose global row
 *             row_offsets[t] + ids[r] is g.
 *
 * An id outside [0, rows of its table) violates the contract: its forward
 * row is written as zeros and it adds no gradient (never an out-of-bounds
 * access).
 *
 * Output layouts (hstu_emb_layout):
 *   HSTU_EMB_FLAT:  out is [num_ids][D]; position r is row r.
 *   HSTU_EMB_TOKEN: every table holds the same number T = num_ids / F of
 *                   ids (id_offsets[t] = t*T is then required); out is
 *                   [T][F*D] and position j of table t is row j, columns
 *                   t*D .. t*D+D-1: the concatenated per-token embedding a
 *                   sequence model reads, written with no conversion pass.
 * dout has the layout of out.
 *
 * Schedule.  The forward walks the ids in table-major order, each
 * work-group a contiguous run of them, so at any time the device works on
 * one or two tables (the table-grouped partitioning).  The backward sorts
 * the global rows of all ids (stable radix sort), sums the output gradient
 * of each distinct row in ascending position order in fixed 32-position
 * chunks, then joins rows that span chunks in chunk order: the result is
 * bitwise reproducible from run to run (no floating-point atomics).
 *
 * Precision.  HSTU_F32: W, out, dout float32.  HSTU_BF16: W, out, dout
 * bfloat16.  Gradients are float32 either way, summed in float32.
 *
 * Pointers and streams.  Every tensor pointer is a DEVICE pointer on the
 * current HIP device; the caller owns all memory.  Calls never allocate and
 * never synchronise: each enqueues its kernels on `stream` (a hipStream_t;
 * NULL = the default stream) and returns.
 *
 * Return codes as in hstu_jagged.h (HSTU_OK, HSTU_EINVAL, HSTU_ENOTSUP,
 * HSTU_EWORKSPACE, HSTU_EHIP); hstu_last_error() describes a failure.
 */
#ifndef HSTU_EMBEDDING_H
#define HSTU_EMBEDDING_H

#include <stddef.h>
#include <stdint.h>

#include "hstu_jagged.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { HSTU_EMB_FLAT = 0, HSTU_EMB_TOKEN = 1 } hstu_emb_layout;

/* Shape of one lookup batch.  The two offset arrays are DEVICE pointers;
 * total_rows and num_ids are their last entries, given on the host so that
 * no call has to read device memory. */
typedef struct {
  hstu_dtype dtype;            /* HSTU_F32 or HSTU_BF16 (W, out, dout)          */
  int32_t num_tables;          /* F, 0 <= F <= 1024                              */
  int32_t dim;                 /* D, a multiple of 8, 8 <= D <= 4096             */
  const int64_t *row_offsets;  /* [F+1], row_offsets[0] = 0, non-decreasing      */
  const int64_t *id_offsets;   /* [F+1], id_offsets[0] = 0, non-decreasing       */
  int64_t total_rows;          /* row_offsets[F], < 2^40                         */
  int64_t num_ids;             /* id_offsets[F], < 2^31                          */
  hstu_emb_layout layout;
} hstu_emb_desc;

/* Forward lookup: out (layout of desc) <- rows of `weights` [total_rows][D]
 * picked by `ids` (int64 [num_ids]).  num_ids = 0 is a successful no-op. */
int hstu_jagged_embedding_fwd(const hstu_emb_desc *desc, const void *weights,
                              const int64_t *ids, void *out, void *stream);

/* Workspace bytes the backward needs for this batch (0 with
 * hstu_last_error set for an invalid descriptor). */
size_t hstu_jagged_embedding_bwd_workspace_bytes(const hstu_emb_desc *desc);

/* Backward: for every global row g that some valid id touches,
 *   grad_weights[g][0 .. D-1] (float32, [total_rows][D]) is OVERWRITTEN with
 *   dW[g]; rows no valid id touches are not written (the caller keeps or
 *   clears them);
 *   unique_rows (int64 [num_ids], may be NULL) receives the touched rows in
 *   ascending order in its first U entries, and *num_unique (int32, device,
 *   may be NULL) receives U.
 * The workspace (256-byte aligned) holds the sort keys and the chunk
 * partials and is clobbered.  num_ids = 0 writes U = 0 and nothing else. */
int hstu_jagged_embedding_bwd(const hstu_emb_desc *desc, const int64_t *ids,
                              const void *dout, float *grad_weights,
                              int64_t *unique_rows, int32_t *num_unique,
                              void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* HSTU_EMBEDDING_H */
