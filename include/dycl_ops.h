/*
 * dycl_ops.h - the routing primitives of the batched executor as standalone
 * calls: stream compaction of a flag array into two stable index lists, and
 * row gathers / scatters.  dycl_run uses the same kernels between a logic
 * node and the sub-network it selects (Sec. 5.3: a logic node decides, per
 * input, which sub-DNN runs next; on a batch the decision becomes a
 * partition of the rows).  These entry points exist for unit tests and
 * bandwidth measurements.
 *
 * All pointers are device pointers, caller-owned; work is queued on
 * `hip_stream` (a hipStream_t, NULL = default stream) and is complete after
 * the stream is synchronised.  Errors are reported as dycl_status codes with
 * dycl_last_error() (declared in dycl.h); validation happens before any
 * launch.
 */
#ifndef DYCL_OPS_H_
#define DYCL_OPS_H_

#include <stddef.h>
#include <stdint.h>

#include "dycl.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes dycl_op_compact needs for n flags. */
size_t dycl_op_compact_workspace(int64_t n);

/*
 * Stable two-way partition of rows 0..n-1 by flags[i] != 0.
 *   flags        [n] uint8, 16-byte aligned.
 *   orig         [n] int32 original ids of the rows, or NULL (id = row).
 *   idx1, org1   [n] int32 outputs: rows with a set flag, in increasing row
 *                order, and their ids (org1 may be NULL).
 *   idx0, org0   the same for the clear flags (org0 may be NULL).
 *   counts       [2] int32: number of set / clear flags.
 *   workspace    dycl_op_compact_workspace(n) bytes, 8-byte aligned (may be
 *                NULL when that is 0).
 * 0 <= n < 2^31; n == 0 writes counts = {0, 0}.
 */
int dycl_op_compact(const uint8_t* flags, const int32_t* orig, int64_t n, int32_t* idx1, int32_t* org1,
                    int32_t* idx0, int32_t* org0, int32_t* counts, void* workspace, size_t workspace_bytes,
                    void* hip_stream);

/*
 * Row move: for r < n, row (dst_idx ? dst_idx[r] : r) of dst receives row
 * (src_idx ? src_idx[r] : r) of src; rows are row_bytes long (a multiple of
 * 16; dst and src 16-byte aligned).  A gather passes src_idx, a scatter
 * dst_idx.  Indices must lie inside the respective arrays (not checked on
 * the device).
 */
int dycl_op_move_rows(void* dst, const int32_t* dst_idx, const void* src, const int32_t* src_idx, size_t row_bytes,
                      int64_t n, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* DYCL_OPS_H_ */
