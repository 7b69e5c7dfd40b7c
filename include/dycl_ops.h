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
 *   orig         [n] int32 original ids of the rows, 16-byte aligned, or NULL
 *                (id = row).
 *   idx1, org1   [n] int32 outputs: rows with a set flag, in increasing row
 *                order, and their ids (org1 may be NULL).
 *   idx0, org0   the same for the clear flags (org0 may be NULL).
 *   counts       [2] int32: number of set / clear flags.
 *   workspace    dycl_op_compact_workspace(n) bytes, 8-byte aligned (may be
 *                NULL when that is 0).
 * 0 <= n < 2^31; n == 0 writes counts = {0, 0}.
 * Above 16384 flags the partition is one chained pass over blocks of 16384
 * flags, 8192 with ids (each block waits, boundedly, for the counts of the
 * blocks before it); if that wait ever ran out, counts reads {-1, -1} and
 * the lists are incomplete.
 */
int dycl_op_compact(const uint8_t* flags, const int32_t* orig, int64_t n, int32_t* idx1, int32_t* org1,
                    int32_t* idx0, int32_t* org0, int32_t* counts, void* workspace, size_t workspace_bytes,
                    void* hip_stream);

/*
 * Allocation-free dycl_op_compact, for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, results and
 * errors as dycl_op_compact without the workspace pair; it calls no
 * allocating routine.  The block status words of the chained form (or the
 * ids of a small partition whose org1 / org0 is NULL) live in a
 * library-owned static device array of DYCL_OP_COMPACT_NOALLOC_SCRATCH
 * bytes, one per GPU the library runs on, held until the process ends; its
 * device address is resolved on the first call on each device.
 *   0 <= n <= DYCL_OP_COMPACT_NOALLOC_MAX_N (2^28); larger n returns
 *   DYCL_E_INVALID.  n == 0 writes counts = {0, 0} with a kernel.
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents (a call's first kernel clears what the chained form needs at
 * zero): calls that overlap on one GPU (concurrent streams, threads) race
 * and must be serialised by the caller.
 */
#define DYCL_OP_COMPACT_NOALLOC_MAX_N (1LL << 28)
#define DYCL_OP_COMPACT_NOALLOC_SCRATCH ((((1LL << 28) + 4095) / 4096) * 12 + 256)
int dycl_op_compact_noalloc(const uint8_t* flags, const int32_t* orig, int64_t n, int32_t* idx1, int32_t* org1,
                            int32_t* idx0, int32_t* org0, int32_t* counts, void* hip_stream);

/*
 * Row move: for r < n, row (dst_idx ? dst_idx[r] : r) of dst receives row
 * (src_idx ? src_idx[r] : r) of src; rows are row_bytes long (a multiple of
 * 16; dst and src 16-byte aligned).  A gather passes src_idx, a scatter
 * dst_idx.  Indices must lie inside the respective arrays (not checked on
 * the device).
 */
int dycl_op_move_rows(void* dst, const int32_t* dst_idx, const void* src, const int32_t* src_idx, size_t row_bytes,
                      int64_t n, void* hip_stream);

/*
 * A sub-network convolution on its own (Sec. 5.3: sub-DNN nodes are
 * conditional-free tensor code; here, one conv layer with its folded
 * BatchNorm, residual and activation), on the kernels dycl_run uses:
 *   y[i, oh, ow, co] = act(scale[co] * sum_{kh, kw, ci} x[i, oh*stride - pad + kh, ow*stride - pad + kw, ci]
 *                                                   * w[co, kh, kw, ci]
 *                          + shift[co] + res[i, oh, ow, co])
 * bf16 storage, float32 accumulation, one round-to-nearest-even to bf16 at
 * the end.  Ho = (H + 2 pad - k) / stride + 1, likewise Wo.
 *
 * dycl_op_conv_packed_bytes  size of the packed weight layout (0 if the
 *                            shape is invalid).
 * dycl_op_conv_pack          host to host: w [cout][k][k][cin] bf16 into the
 *                            packed layout (zero-padded rows and K); both
 *                            pointers are host memory.
 * dycl_op_conv_workspace_bytes  device workspace that lets a layer with a
 *                            deep K on few output pixels per image (Ho*Wo <=
 *                            64, K = k*k*cin >= 4608, cout >= 256) split each
 *                            output tile's K range over several workgroups;
 *                            0 for every other shape.  The split depends on
 *                            the shape alone, never on n.
 * dycl_op_conv               device pointers: x [n][H][W][cin] bf16,
 *                            packed (uploaded result of dycl_op_conv_pack),
 *                            scale / shift [cout] float32 or NULL (1 / 0),
 *                            res [n][Ho][Wo][cout] bf16 or NULL, y the same
 *                            shape as res.  act: 0 none, 1 ReLU, 2 exact GELU.
 *                            k in {1, 3, 7}; n >= 0 (0 does nothing); every
 *                            tensor below 2^31 elements.  workspace: NULL, or
 *                            workspace_bytes >= dycl_op_conv_workspace_bytes
 *                            of device memory, caller-owned, which the call
 *                            overwrites (calls sharing one must not overlap);
 *                            without it a split layer runs unsplit: the same
 *                            sums, added in another order.  dycl_run always
 *                            splits.  Work is queued on hip_stream.
 */
size_t dycl_op_conv_packed_bytes(int cout, int k, int cin);
int dycl_op_conv_pack(const uint16_t* w, int cout, int k, int cin, uint16_t* packed, size_t packed_bytes);
size_t dycl_op_conv_workspace_bytes(int n, int H, int W, int cin, int cout, int k, int stride, int pad);
int dycl_op_conv(const uint16_t* x, int n, int H, int W, int cin, const uint16_t* packed, int cout, int k, int stride,
                 int pad, const float* scale, const float* shift, const uint16_t* res, int act, uint16_t* y,
                 void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * A convolution and the 3x3 / stride-2 / pad-1 max-pool that follows it in
 * one launch (two tensor statements of one sub-DNN node, Sec. 5.3, fused):
 *   y[i, ph, pw, co] = max over oh in [2 ph - 1, 2 ph + 1] and ow in
 *                      [2 pw - 1, 2 pw + 1] inside [0, Ho) x [0, Wo) of
 *                      the dycl_op_conv output (no residual)
 * Hp = (Ho - 1) / 2 + 1, likewise Wp.  Only the pooled tensor is written.
 * Taken for the ImageNet stem: cin 3, cout 64, k 7, stride 2, pad <= 3,
 * W % 8 == 0, Wo <= 112, act 1 (ReLU); other arguments return
 * DYCL_E_INVALID.  x [n][H][W][3], packed as for dycl_op_conv, scale /
 * shift [64] float32 or NULL, y [n][Hp][Wp][64]; device pointers, 16-byte
 * aligned; n >= 0 (0 does nothing).  Work is queued on hip_stream.
 */
int dycl_op_conv_maxpool(const uint16_t* x, int n, int H, int W, int cin, const uint16_t* packed, int cout, int k,
                         int stride, int pad, const float* scale, const float* shift, int act, uint16_t* y,
                         void* hip_stream);

/*
 * A bottleneck block's last 1x1 convolution and the next block's first 1x1
 * convolution, which reads nothing but its output, in one launch (two
 * layers of one sub-DNN node in succession, Sec. 5.3; dycl_run runs such
 * pairs this way unless the spec says "pair_pointwise": false):
 *   y3 = dycl_op_conv(x, packed3, c3, k 1, stride 1, pad 0, scale3, shift3, res, act 1)
 *   y1 = dycl_op_conv(y3, packed1, c1, k 1, stride 1, pad 0, scale1, shift1, NULL, act 1)
 * bit for bit; each tile of y3 stays on chip for the second contraction, so
 * y3 is written once and never read back.  Taken for ReLU on both and
 * either c3 256, c1 64, cin % 64 == 0 with 64 <= cin <= 1024 (ResNet-50's
 * first stage) or c3 512, c1 128, cin 128 (its second stage, the first
 * layer's output channels taken 128 at a time); other shapes return
 * DYCL_E_INVALID.  x [n][H][W][cin], res [n][H][W][c3]
 * or NULL, y3 [n][H][W][c3], y1 [n][H][W][c1]; packed3 / packed1 from
 * dycl_op_conv_pack (k 1; cin and c3 input channels); scale / shift [cout]
 * float32, all four required; device pointers, 16-byte aligned; n >= 0 (0
 * does nothing).  Work is queued on hip_stream.
 */
int dycl_op_conv_pair(const uint16_t* x, int n, int H, int W, int cin, const uint16_t* packed3, const float* scale3,
                      const float* shift3, const uint16_t* res, int c3, uint16_t* y3, const uint16_t* packed1,
                      const float* scale1, const float* shift1, int c1, uint16_t* y1, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* DYCL_OPS_H_ */
