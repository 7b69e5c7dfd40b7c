/*
 * dycl.h - C ABI of the batched dynamic-routing executor for MI355X (gfx950).
 *
 * DyCL (ISSTA'23, arXiv 2307.04963) compiles a dynamic neural network into
 * conditional-free sub-networks plus a host program that keeps the
 * conditionals and calls the compiled pieces (Sec. 5, Fig. 5 steps 1-5).
 * The host program must be semantically identical to the dynamic network
 * for every input (Sec. 5, Eq. 2) and is called like a compiled module:
 * set the input, run, read the output (Listing 2; Sec. 5: "call the API
 * using a similar way").  This library executes that compiled form on a
 * BATCH: each sample follows the branch its own decision selects, the
 * samples of one branch are compacted into a packed buffer, and the host
 * code reads only the per-branch counts.
 *
 * The plan is built from a specification whose nodes are the two kinds of
 * node of the paper's heterogeneous control-flow graph (Sec. 5.3): runs of
 * tensor statements (sub-DNNs) and single logic statements.  Shapes are
 * propagated from the input in topological order, a logic node keeping its
 * predecessor's shape (Alg. 2).
 *
 * Threading: calls on different plans may run concurrently; one plan runs
 * one batch at a time.  No C++ exception crosses this interface; the
 * library never aborts the process.  Every function returns a dycl_status
 * (0 on success); the message of the calling thread's last failure is
 * available from dycl_last_error().
 */
#ifndef DYCL_H_
#define DYCL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dycl_plan dycl_plan; /* opaque; owns device weights + workspace */

typedef enum {
  DYCL_OK = 0,
  DYCL_E_INVALID = -1, /* null pointer, bad argument, misaligned buffer    */
  DYCL_E_SPEC = -2,    /* specification does not parse or is inconsistent */
  DYCL_E_WEIGHTS = -3, /* weight blob too small for what the spec reads   */
  DYCL_E_BATCH = -4,   /* batch < 0 or batch > max_batch                  */
  DYCL_E_OOM = -5,     /* device memory allocation failed                 */
  DYCL_E_HIP = -6      /* a HIP runtime call failed (message has details) */
} dycl_status;

/* Per-sample record of what the dynamic network did (16 bytes). */
typedef struct {
  int32_t exit_index;  /* 0-based exit head that produced the logits; -1 if none */
  int32_t iterations;  /* bounded-loop steps executed (1..max_steps); 0 if no loop */
  uint64_t skip_mask;  /* bit i set <=> gate i chose the identity / shortcut path */
} dycl_record;

/*
 * Build a plan (the paper's sub-DNN compilation, Alg. 2, for a fixed
 * maximum batch).
 *   spec_json     NUL-terminated JSON specification: the input shape and
 *                 dtype, and a list of nodes - "conv" (convolution or
 *                 linear layer with folded BatchNorm / bias, optional
 *                 residual, ReLU or GELU), "maxpool", "exit" (global
 *                 average pool, linear head, softmax, confidence test),
 *                 "gate" (pool, linear, sigmoid, run a sub-list of nodes
 *                 on the samples that execute), "halt" (halting unit of a
 *                 bounded loop, unrolled) and "output" (final linear on the
 *                 loop's parked states).  Optional "pair_pointwise": false
 *                 runs every layer in its own launch (by default a
 *                 bottleneck's last 1x1 convolution and the next 1x1
 *                 convolution share one; the results are the same bits
 *                 either way).  Copied, not retained.
 *   weights       host pointer to the weight blob the spec's offsets index;
 *                 copied to the device, not retained.
 *   weights_bytes size of that blob.
 *   max_batch     largest batch a later dycl_run may pass (>= 1); the
 *                 workspace is sized for it.
 *   device        HIP device ordinal.
 *   out           receives the plan; set to NULL on failure.
 * The spec and the blob size are validated before any HIP call.
 */
int dycl_plan_create(const char* spec_json, const void* weights, size_t weights_bytes, int max_batch,
                     int device, dycl_plan** out);

/*
 * Run one batch (asynchronously on `hip_stream`, a hipStream_t; NULL is the
 * default stream).
 *   x_dev       device pointer, [batch, per-sample input] in the spec's
 *               input dtype (bf16 NHWC images or vectors; fp32 for fp32
 *               specs), 16-byte aligned, caller-owned.
 *   batch       0 <= batch <= max_batch; 0 returns immediately.
 *   aux_dev     device fp32 [batch] per-sample scalars for specs that read
 *               them (a halting bias), else may be NULL.
 *   logits_dev  device fp32 [batch, n_out], written in the original sample
 *               order.
 *   records_dev device dycl_record [batch], original order.
 * In the default host mode (DYCL_HOST_SYNC) the host code waits only for the
 * per-decision branch counts; in the device modes it waits for nothing (see
 * dycl_plan_set_host_mode).  When the call returns, the remaining work may
 * still be queued on the stream.  Results are valid after the stream is
 * synchronised.
 */
int dycl_run(dycl_plan* plan, const void* x_dev, int batch, const float* aux_dev, float* logits_dev,
             dycl_record* records_dev, void* hip_stream);

/*
 * dycl_run for a plan whose network emits token sequences (a generative
 * network, Table 1's En-Decoder family: one token per step, read back as
 * the next step's input, until an end token or the spec's max_len; the
 * bounded loop of Sec. 2.2).  The same arguments, plus
 *   tokens_dev  device int32 [batch][max_len] (max_len from
 *               dycl_plan_info), 4-byte aligned, caller-owned: the emitted
 *               tokens in the original sample order, -1 after a sample's
 *               last token.
 * logits_dev must be 16-byte aligned here.
 * logits_dev receives each sample's last step logits [batch][n_out] and
 * records_dev its length as `iterations`.  dycl_run refuses such a plan and
 * dycl_run_seq any other (DYCL_E_INVALID).
 */
int dycl_run_seq(dycl_plan* plan, const void* x_dev, int batch, const float* aux_dev, float* logits_dev,
                 dycl_record* records_dev, int32_t* tokens_dev, void* hip_stream);

/*
 * How the host module learns the branch counts (Sec. 5: the host program
 * keeps the conditionals and calls the compiled sub-DNNs; Sec. 4, Challenge
 * 2 and Sec. 6.4, Table 4: host-device transfers that compute nothing are
 * overhead worth removing).
 *   DYCL_HOST_SYNC    after each decision point the host reads the two branch
 *                     counts back and launches the next kernels on exactly
 *                     that many rows (one wait per decision point).
 *   DYCL_HOST_DEVICE  the counts stay on the device: every later kernel is
 *                     launched for the largest possible row count (the rows
 *                     that reached the decision) and reads the live count
 *                     when it starts; surplus workgroups leave at once.  The
 *                     host never waits inside dycl_run.
 *   DYCL_HOST_GRAPH   DYCL_HOST_DEVICE with the whole run captured once into
 *                     a HIP graph and replayed by later runs with the same
 *                     batch size and the same x / aux / logits / records
 *                     pointers (any change re-captures).  While profiling is
 *                     enabled, runs are launched without the graph.
 *   DYCL_HOST_PERSISTENT  DYCL_HOST_DEVICE, except that the bounded loop of an
 *                     adaptive-computation-time network (Sec. 2.2) runs as one
 *                     cooperative launch: every step's layer, halting test and
 *                     compaction in one kernel, with grid-wide barriers between
 *                     the phases of a step (max_batch <= 4096).  Bit for bit the
 *                     same results; on MI355X the barriers across the 8 XCDs cost
 *                     more than the per-step launches they replace.
 * Results are identical in every mode.  Returns the previous mode, or
 * DYCL_E_INVALID for an unknown mode.  Not to be called while a run of the
 * plan is being enqueued.
 */
typedef enum { DYCL_HOST_SYNC = 0, DYCL_HOST_DEVICE = 1, DYCL_HOST_GRAPH = 2, DYCL_HOST_PERSISTENT = 3 } dycl_host_mode;
int dycl_plan_set_host_mode(dycl_plan* plan, int mode);

/*
 * Branch counts of the last dycl_run: for decision point d (in program
 * order, loop steps unrolled) counts[2d] = samples that took the "true"
 * branch (exit / execute / halt) and counts[2d+1] = the others; decisions
 * the batch never reached read 0.  Writes min(n, 2 * decisions) entries and
 * returns the number of decision points.  After a run in a device mode the
 * counts are read from the device, which first synchronises that run's
 * stream.
 */
int dycl_last_counts(const dycl_plan* plan, int32_t* counts, int n);

/*
 * Plan facts, info[0..n): 0 n_out, 1 input bytes per sample, 2 decision
 * points, 3 device workspace bytes, 4 device weight bytes, 5 max_batch,
 * 6 aux required (0/1), 7 number of nodes, 8 host mode, 9 graph captures
 * so far, 10 tokens per sample a run emits (max_len; 0: a plan for
 * dycl_run).  Returns the number written.
 */
int dycl_plan_info(const dycl_plan* plan, int64_t* info, int n);

/*
 * Per-kernel-class timing of later runs: when enabled, every kernel launch
 * of dycl_run is bracketed by HIP events on its stream and its algorithmic
 * work (FLOPs of the executed rows, bytes it must move) is accumulated.
 * dycl_profile_read fills up to `cap` rows of
 *   { launches, total_ms, flops, bytes }  (4 doubles per row)
 * for the classes named by dycl_profile_class(i) and returns the number of
 * classes.  Reading synchronises the plan's last stream.  In the device host
 * modes the host does not know the live row counts, and the work is counted
 * for the rows each kernel was launched for (an upper bound).
 */
int dycl_profile_enable(dycl_plan* plan, int on);
int dycl_profile_read(dycl_plan* plan, double* rows, int cap);
const char* dycl_profile_class(int i);

/*
 * Every launch of the last run made while profiling was enabled, in launch
 * order: up to `cap` rows of { class index, ms, flops, bytes } (4 doubles),
 * the same quantities dycl_profile_read sums.  Returns the number of
 * launches of that run (which may exceed cap); synchronises like
 * dycl_profile_read.
 */
int dycl_profile_launches(dycl_plan* plan, double* rows, int cap);

/*
 * Label of launch i of the rows dycl_profile_launches returned: the node it
 * belongs to - a layer by the tensor it writes (with the projection folded
 * into it, or the fused max-pool; "a + b" for two 1x1 layers in one
 * launch), a decision as "exit k", "gate k" or "halt k".  "" for an index out of range or an invalid plan.  The string
 * lives in the plan until its next profiled run.
 */
const char* dycl_profile_launch_label(const dycl_plan* plan, int i);

/*
 * Host-only validation of a spec against a blob size and a batch bound (no
 * HIP call): parses, checks every reference and weight range, propagates
 * shapes, and writes a one-line summary into `summary` (may be NULL).
 */
int dycl_spec_check(const char* spec_json, size_t weights_bytes, int max_batch, char* summary, size_t cap);

/* Releases the plan's device memory; NULL-safe. */
void dycl_plan_destroy(dycl_plan* plan);

/* Message of the calling thread's last failure ("" if none). */
const char* dycl_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DYCL_H_ */
