// Plan = the compiled form of a dynamic network for one maximum batch.
//
// The specification lists the nodes of the paper's heterogeneous control
// flow graph (Sec. 5.3): sub-DNN nodes (runs of tensor statements; here
// "conv", "maxpool", "output") and logic nodes, each a single conditional
// that reads an intermediate tensor ("exit", "gate", "halt").  Loops are
// already unrolled, as the paper's rewriting step does (Sec. 5.2).  Building
// the plan walks the nodes in program order and propagates each tensor's
// per-sample shape from its producer; a logic node passes its input's shape
// on unchanged (Alg. 2).  Then every tensor gets a device buffer sized for
// max_batch rows, with buffers reused once their tensor is dead.
#pragma once

#include <hip/hip_runtime.h>

#include <array>
#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "../../include/dycl.h"
#include "json.hpp"
#include "kernels.hpp"

namespace dycl {

enum class DType { BF16, F32 };

struct TensorInfo {
  std::string name;
  int H = 1, W = 1, C = 1;
  int space = 0;       // row space it lives in (changes at every compaction)
  bool external = false;   // the caller's input
  bool parked = false;     // full batch, original sample order
  int first = -1, last = -1;   // liveness (node sequence numbers)
  bool unused = false;     // never materialised (its readers go through a row list)
  bool f32 = false;        // float32 in a bf16 spec (an LSTM cell state)
  int buf = -1;
  size_t row_bytes(DType dt) const { return (size_t)H * W * C * (dt == DType::BF16 && !f32 ? 2 : 4); }
};

enum class NodeKind { Conv, MaxPool, Exit, Gate, Halt, Output, Decode };

struct Node {
  NodeKind kind = NodeKind::Conv;
  int seq_pre = 0, seq_post = 0;
  // tensors
  int src = -1, src2 = -1, dst = -1, res = -1;
  // conv / linear
  int k = 1, stride = 1, pad = 0, cin1 = 0, cin2 = 0, cout = 0;
  int H = 1, W = 1, Ho = 1, Wo = 1;
  int act = 0;
  int64_t w_off = -1, w_ldk = 0, w_k0 = 0;   // weight tensor byte offset, row length, first column
  int64_t scale_off = -1, shift_off = -1;    // fp32 [cout] byte offsets (or -1)
  int packed = -1;                           // index of packed bf16 weights
  bool pad_in = false;                       // reads the input padded to 8 channels
  bool pool = false;                         // a 3x3 / 2 max-pool fused in: dst is the pooled tensor
  // a 1x1 projection shortcut folded in as src2: the packed weights are
  // [W_c | W_p]; the kernel runs the projection's K steps first, rounds
  // s_p * acc + b_p to bf16 exactly as the unfused projection stores it,
  // and carries it into the block's own sum divided by the block's scale
  // (plan-owned vector fold_shift: [scale | shift | s_p | b_p | 1 / scale],
  // scale 1 and W_c zero for a channel whose scale is 0)
  int64_t scale2_off = -1, shift2_off = -1;
  int s2 = 1;            // src2 is read at this stride (a folded strided projection)
  // an LSTM step (act ACT_LSTM): the concatenated input is a row of the
  // embedding table in the blob (emb_off, emb_rows rows of cin2 values)
  // chosen by each row's previous token; cell_in / cell_out are the
  // float32 cell states (cell_in -1: zeros); the gate weight rows and the
  // bias are interleaved per cell at plan creation (lstm_shift vector)
  int64_t emb_off = -1;
  int emb_rows = 0;
  int cell_in = -1, cell_out = -1;
  int lstm_shift = -1;
  // decode (greedy token choice): eos token, step (index), max_len (max_steps)
  int eos = 0;
  bool fold = false;
  int fold_shift = -1;
  // fused gathers / scatters: which row list of the last decision maps this
  // layer's images to those of src, res, dst (0: none, 1: the rows that
  // stay (exit, halt), 2: the rows that take the true branch (gate body),
  // 3: the original sample ids of the current rows)
  int src_list = 0, src2_list = 0, res_list = 0, dst_list = 0;
  // heads: exit W [ncls][C], b [ncls], T [1]; gate u [C], v [1]; halt w [C]
  int64_t h_w = -1, h_b = -1, h_T = -1;
  int ncls = 0, hc = 0;
  int head_t = -1;      // index of the transposed fp32 weights (exit heads, fp32 linear layers), or -1
  bool fused = false;   // exit head small enough for the one-kernel path
  // a conv whose output an exit head pools, with the pooling's partial sums
  // taken in its epilogue (conv), or that exit head (Exit)
  bool gap_pool = false;
  // this conv and the next node (a 1x1 conv reading only its output) run as
  // one kernel (conv_pair) when the kernel takes them
  bool pair = false;
  float tau = 0.f;
  bool final_ = false;
  int index = 0;        // exit head / gate / loop step
  int max_steps = 0;
  int decision = -1;    // slot in the per-run counts
  std::vector<std::pair<int, int>> pairs;     // exit/halt carry (old, new); gate gather (outer, inner)
  std::vector<std::pair<int, int>> scatter;   // gate: (inner, outer)
  int park_src = -1, park_dst = -1;           // halt
  std::vector<Node> body;                     // gate
};

struct Packed {
  int64_t w_off, w_ldk, w_k0;
  int cout, K, cout_pad, Kp;
  bool interleave4 = false;   // packed row co = stored row (co % 4) * (cout / 4) + co / 4 (LSTM gates per cell)
  // taps x cin_src weights per output channel in the blob, stored as
  // taps x cin_pack (zero-filled) when the input channels are padded
  int taps = 1, cin_src = 0, cin_pack = 0;
  // a folded projection: a second 1x1 block of cin2 columns appended to K
  // (the projection's weights as stored); rows whose scale_1 is 0 keep only
  // that block
  int64_t w2_off = -1, w2_ldk = 0, w2_k0 = 0;
  int cin2 = 0;
  int64_t scale1_off = -1;
  uint16_t* dev = nullptr;
};

struct ProfileRow {
  double launches = 0, ms = 0, flops = 0, bytes = 0;
};

enum ProfileClass { P_CONV = 0, P_LINEAR32, P_HEAD, P_COMPACT, P_MOVE, P_POOL, P_MISC, P_COUNT };

struct Spec {
  DType dt = DType::BF16;
  int n_out = 0;
  bool aux = false;
  int input = -1;
  std::vector<TensorInfo> tensors;
  std::vector<Node> nodes;
  std::vector<Packed> packed;
  int decisions = 0;
  int seq = 0;
  bool any_halt = false;
  int max_head_c = 8, max_ncls = 8;
  int nodes_total = 0;
  int pad_input_c = 0;
  int fused_gathers = 0;   // exit carries read in place through the row list
  int fused_gates = 0;     // gates whose gathers and scatters are fused into the body convolutions
  int fused_pools = 0;     // max-pools fused into the stem convolution that feeds them
  int fused_projections = 0;   // 1x1 projection shortcuts folded into the block's last 1x1 convolution
  int fused_pairs = 0;         // 1x1 convolutions run in one kernel with the 1x1 convolution before them
  int n_fold_shift = 0;        // constant vectors of the folded projections
  int n_lstm_shift = 0;        // interleaved biases of the LSTM steps
  bool any_decode = false;     // a greedy decoding loop: runs emit tokens
  int max_len = 0, bos = 0;    // its length bound and start token
  int n_head_t = 0;      // fp32 weight matrices kept transposed on the device   // > 0: the input is zero-padded to this many channels for the stem
  std::string summary;
  const uint8_t* host_w = nullptr;   // the host weight blob during parse, when given

  // weights: the host blob when it is at hand (plan creation), or null
  // (validation only); the projection fold reads the batch-norm scales
  void parse(const std::string& json, size_t weights_bytes, int max_batch, const void* weights = nullptr);
  void fuse_original_order_reads();
  void fuse_exit_gathers();
  void fuse_gate_moves();
  void fuse_stem_pools();
  void fuse_projections();
  void pair_pointwise();
};

}  // namespace dycl

struct dycl_plan {
  uint32_t magic = 0x44594350u;  // "DYCP"
  dycl::Spec spec;
  int device = 0;
  int max_batch = 0;
  // device memory
  uint8_t* d_blob = nullptr;
  size_t blob_bytes = 0;
  std::vector<void*> buffers;
  std::vector<size_t> buffer_bytes;
  uint8_t* d_flags = nullptr;
  int32_t *d_idx1 = nullptr, *d_org1 = nullptr, *d_idx0 = nullptr, *d_org0 = nullptr;
  int32_t* d_orig[2] = {nullptr, nullptr};
  int32_t* d_iota = nullptr;      // 0..max_batch-1: original ids of a fresh batch
  int32_t* d_counts = nullptr;
  int32_t* h_counts = nullptr;   // pinned
  float* d_G = nullptr;          // [max_batch, max_head_c]
  float* d_Gpart = nullptr;      // [kGapMaxSplit, max_batch, max_head_c] split pooling partials, or null
  float* d_gapQ = nullptr;       // [ceil(max_batch * HW / 32), 2, C] pooling chunk sums from a conv epilogue, or null
  float* d_split = nullptr;      // K-split conv partial sums (largest layer at max_batch rows), or null
  size_t split_bytes = 0;
  float* d_Z = nullptr;          // [max_batch, max_ncls]
  float* d_headP = nullptr;      // K-slice partial sums of the wide exit heads, or null
  float* d_S = nullptr;          // [max_batch]
  void* d_cws = nullptr;         // workspace of the large-n compaction (max_batch > 16384)
  uint16_t* d_zeros = nullptr;   // 256 zero bytes: source of convolution padding taps
  uint16_t* d_xpad = nullptr;    // input padded to 8 channels (stems with Cin < 8)
  std::vector<float*> head_t;    // transposed fp32 weights: exit heads [C][ncls], fp32 linears [cin][cout]
  std::vector<float*> fold_shift;   // folded projections: [scale | shift | s_p | b_p | 1 / scale] of 5 x cout
  std::vector<float*> lstm_shift;   // LSTM steps: the gate bias, interleaved per cell
  int32_t* d_tok[2] = {nullptr, nullptr};   // decoding: [0] the current rows' previous tokens, [1] this step's
  // an adaptive-computation-time loop run as one persistent launch in the
  // device host mode: top-level nodes [begin, end) (the unrolled steps'
  // convolutions and halting tests), the Output node at `end`
  struct ActLoop {
    bool ok = false;
    size_t begin = 0, end = 0;
    int packed = -1, hidden = 0, d_in = 0, steps = 0, d0 = 0, park = -1, input = -1;
    int64_t b1 = -1, wh = -1;
    float tau = 0.f;
    uint16_t* h[2] = {nullptr, nullptr};
  } act;
  size_t workspace_bytes = 0, weight_bytes = 0;
  // profiling
  bool profile = false;
  std::vector<hipEvent_t> ev_free;
  struct Pending {
    int cls;
    hipEvent_t a, b;
    double flops, bytes;
    std::string label;   // the node the launch belongs to
  };
  std::vector<Pending> pending;
  dycl::ProfileRow prof[dycl::P_COUNT];
  // launches of the last profiled run: {class, ms, flops, bytes}
  std::vector<std::array<double, 4>> last_run;
  std::vector<std::string> last_run_labels;
  size_t last_run_begin = 0;
  hipStream_t last_stream = nullptr;
  // host mode (dycl_host_mode) and the last run's: whether its branch
  // counts are only in d_counts (device modes)
  int mode = DYCL_HOST_SYNC;
  bool counts_on_device = false;
  // graph mode: the captured run, replayed while its key is unchanged
  hipStream_t cap_stream = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t graph_exec = nullptr;
  struct GraphKey {
    const void* x = nullptr;
    int B = 0;
    const float* aux = nullptr;
    float* logits = nullptr;
    dycl_record* rec = nullptr;
    int32_t* tokens = nullptr;
  } graph_key;
  long graph_captures = 0;
  // device modes: the branch counts of an earlier run, copied back without a
  // wait, as the expected live rows that pick tile shapes (never the grid)
  std::vector<int32_t> hint;       // [2 * decisions]
  int hint_B = 0;                  // batch those counts came from (0: none yet)
  int32_t* h_hint_stage = nullptr; // pinned target of the asynchronous copy
  hipEvent_t hint_ev = nullptr;
  bool hint_pending = false;
  int hint_pending_B = 0;
};

namespace dycl {
int plan_build(dycl_plan* p, const std::string& json, const void* weights, size_t weights_bytes);
void plan_free(dycl_plan* p);
void plan_run(dycl_plan* p, const void* x, int B, const float* aux, float* logits, dycl_record* rec,
              int32_t* tokens, hipStream_t s);
void profile_flush(dycl_plan* p);
// host mode (a dycl_host_mode value, already validated); drops a captured graph
void plan_set_mode(dycl_plan* p, int mode);
// the first min(n, 2 * decisions) branch counts of the last run
void plan_read_counts(const dycl_plan* p, int32_t* out, int n);

struct HipError : std::runtime_error {
  explicit HipError(const std::string& m) : std::runtime_error(m) {}
};
struct OomError : std::runtime_error {
  explicit OomError(const std::string& m) : std::runtime_error(m) {}
};
struct WeightsError : std::runtime_error {
  explicit WeightsError(const std::string& m) : std::runtime_error(m) {}
};
}  // namespace dycl
