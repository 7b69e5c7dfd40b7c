// Plan construction (device side) and the host module that runs a batch.
//
// The host module plays the role of the paper's generated host program
// (Sec. 5.6): it keeps the conditionals and calls the compiled sub-networks.
// On a batch, every logic node is evaluated on the device for all active
// rows at once; a stable compaction splits the rows by branch, and the only
// value the host waits for is the pair of branch counts, which sizes the
// launches of the next sub-network.  Per-sample work never touches the host.
//
// Computation-free outputs stay off the device path (Sec. 5.4): a skipped
// residual block's output is its input (identity path) and is never copied;
// records and counts are plain stores of the decision kernels.
#include <algorithm>
#include <functional>
#include <cstring>

#include "plan.hpp"

namespace dycl {

namespace {

// bf16 <-> fp32 on the host, rounding to nearest even (finite values: the
// weights and their batch-norm scales)
float host_f32(uint16_t b) {
  const uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}
uint16_t host_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) throw HipError(std::string(what) + ": " + hipGetErrorString(e));
}

template <class T>
T* dev_alloc(dycl_plan* p, size_t count, const char* what) {
  void* ptr = nullptr;
  const size_t bytes = std::max<size_t>(count * sizeof(T), 256);
  hipError_t e = hipMalloc(&ptr, bytes);
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) {
    (void)hipGetLastError();   // leave no error behind for the next launch check
    throw OomError(std::string(what) + ": hipMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  hip_check(e, what);
  p->workspace_bytes += bytes;
  return static_cast<T*>(ptr);
}

void assign_buffers(dycl_plan* p, int max_batch) {
  Spec& sp = p->spec;
  std::vector<int> order;
  for (int i = 0; i < static_cast<int>(sp.tensors.size()); ++i)
    if (!sp.tensors[i].external && !sp.tensors[i].unused) order.push_back(i);
  std::sort(order.begin(), order.end(), [&](int a, int b) { return sp.tensors[a].first < sp.tensors[b].first; });
  std::vector<int> active;
  std::vector<bool> busy;
  for (int t : order) {
    TensorInfo& ti = sp.tensors[t];
    for (auto it = active.begin(); it != active.end();) {
      if (sp.tensors[*it].last < ti.first) {
        busy[sp.tensors[*it].buf] = false;
        it = active.erase(it);
      } else {
        ++it;
      }
    }
    const size_t need = static_cast<size_t>(max_batch) * ti.row_bytes(sp.dt);
    int best = -1;
    for (int b = 0; b < static_cast<int>(p->buffer_bytes.size()); ++b)
      if (!busy[b] && p->buffer_bytes[b] >= need && (best < 0 || p->buffer_bytes[b] < p->buffer_bytes[best]))
        best = b;
    if (best < 0) {
      // grow the largest free buffer that is too small instead of adding one
      for (int b = 0; b < static_cast<int>(p->buffer_bytes.size()); ++b)
        if (!busy[b] && (best < 0 || p->buffer_bytes[b] > p->buffer_bytes[best])) best = b;
      if (best >= 0) {
        p->buffer_bytes[best] = need;
      } else {
        p->buffer_bytes.push_back(need);
        busy.push_back(false);
        best = static_cast<int>(p->buffer_bytes.size()) - 1;
      }
    }
    busy[best] = true;
    ti.buf = best;
    active.push_back(t);
  }
  p->buffers.assign(p->buffer_bytes.size(), nullptr);
  for (size_t b = 0; b < p->buffers.size(); ++b) p->buffers[b] = dev_alloc<uint8_t>(p, p->buffer_bytes[b], "activation buffer");
}

// The unrolled loop of an adaptive-computation-time network: for t = 1..T a
// GELU linear layer h_t = GELU(W1 [h_{t-1}; x] + b1) (t = 1: the x columns
// of W1 alone) and its halting test, the states parked into one tensor,
// then the output layer.  Such a loop can run as one persistent launch.
void detect_act_loop(dycl_plan* p) {
  const Spec& sp = p->spec;
  auto& L = p->act;
  L = dycl_plan::ActLoop{};
  const auto& nd = sp.nodes;
  for (size_t i = 0; i + 2 < nd.size(); ++i) {
    const Node& c1 = nd[i];
    if (c1.kind != NodeKind::Conv || nd[i + 1].kind != NodeKind::Halt || c1.act != k::ACT_GELU || c1.src2 >= 0 ||
        !sp.tensors[c1.src].external || c1.H != 1 || c1.W != 1 || c1.res >= 0 || c1.scale_off >= 0 ||
        c1.src_list != 0)
      continue;
    const Node& h1 = nd[i + 1];
    const int T = h1.max_steps, Hd = c1.cout, D = c1.cin1;
    if (h1.index != 1 || T < 2 || i + 2 * static_cast<size_t>(T) >= nd.size() || c1.w_k0 != Hd ||
        c1.w_ldk != Hd + D || h1.src != c1.dst)
      continue;
    bool ok = true;
    int packed = -1;
    for (int t = 1; t <= T && ok; ++t) {
      const Node& c = nd[i + 2 * (t - 1)];
      const Node& h = nd[i + 2 * (t - 1) + 1];
      ok = c.kind == NodeKind::Conv && h.kind == NodeKind::Halt && c.act == k::ACT_GELU && c.cout == Hd &&
           c.w_off == c1.w_off && c.shift_off == c1.shift_off && c.scale_off < 0 && c.res < 0 && c.H == 1 &&
           c.W == 1 && !c.pad_in && c.dst_list == 0 && h.src == c.dst && h.index == t && h.max_steps == T &&
           h.h_w == h1.h_w && h.tau == h1.tau && h.park_dst == h1.park_dst && h.park_src == c.dst &&
           h.decision == h1.decision + t - 1 && h.hc == Hd;
      if (ok && t > 1)
        ok = c.src_list == 1 && c.cin1 == Hd && c.src2 == c1.src && c.src2_list == 3 && c.cin2 == D &&
             c.w_k0 == 0 && c.w_ldk == Hd + D && (packed < 0 || packed == c.packed);
      if (ok && t > 1) packed = c.packed;
    }
    const size_t end = i + 2 * static_cast<size_t>(T);
    if (!ok || packed < 0 || nd[end].kind != NodeKind::Output || nd[end].src != h1.park_dst) continue;
    if (!k::act_loop_fits(p->max_batch, Hd, D)) return;
    L.ok = true;
    L.begin = i;
    L.end = end;
    L.packed = packed;
    L.hidden = Hd;
    L.d_in = D;
    L.steps = T;
    L.d0 = h1.decision;
    L.park = h1.park_dst;
    L.input = c1.src;
    L.b1 = c1.shift_off;
    L.wh = h1.h_w;
    L.tau = h1.tau;
    return;
  }
}

}  // namespace

int plan_build(dycl_plan* p, const std::string& json, const void* weights, size_t weights_bytes) {
  Spec& sp = p->spec;
  sp.parse(json, weights_bytes, p->max_batch, weights);
  hip_check(hipSetDevice(p->device), "hipSetDevice");

  // weights: the blob as is (fp32 vectors, heads, fp32 linear layers) ...
  p->blob_bytes = weights_bytes;
  {
    void* ptr = nullptr;
    hipError_t e = hipMalloc(&ptr, std::max<size_t>(weights_bytes, 256));
    if (e != hipSuccess) throw OomError("weight blob: hipMalloc failed");
    p->d_blob = static_cast<uint8_t*>(ptr);
    p->weight_bytes += weights_bytes;
    hip_check(hipMemcpy(p->d_blob, weights, weights_bytes, hipMemcpyHostToDevice), "weights upload");
  }
  // ... and every bf16 contraction's weights packed to [cout_pad][Kp] with
  // zero rows / columns, so tile loads never leave the array
  const uint8_t* hb = static_cast<const uint8_t*>(weights);
  auto hf32 = [&](int64_t off, int i) {
    float v;
    std::memcpy(&v, hb + off + static_cast<size_t>(i) * 4, 4);
    return v;
  };
  for (Packed& q : sp.packed) {
    std::vector<uint16_t> h(static_cast<size_t>(q.cout_pad) * q.Kp, 0);
    for (int co = 0; co < q.cout; ++co) {
      // LSTM gates: packed row 4 j + k is gate k of cell j (stored in blocks of cout / 4)
      const int srow = q.interleave4 ? (co % 4) * (q.cout / 4) + co / 4 : co;
      const uint8_t* row = hb + q.w_off + (static_cast<size_t>(srow) * q.w_ldk + q.w_k0) * 2;
      if (q.w2_off >= 0) {
        // a folded projection: [W_c | W_p], both as stored; a channel whose
        // own scale is 0 keeps only the projection block
        const uint8_t* row2 = hb + q.w2_off + (static_cast<size_t>(co) * q.w2_ldk + q.w2_k0) * 2;
        const float s1 = q.scale1_off >= 0 ? hf32(q.scale1_off, co) : 1.0f;
        uint16_t* dst = &h[static_cast<size_t>(co) * q.Kp];
        const int k1 = q.K - q.cin2;
        if (s1 != 0.0f) std::memcpy(dst, row, static_cast<size_t>(k1) * 2);
        std::memcpy(dst + k1, row2, static_cast<size_t>(q.cin2) * 2);
        continue;
      }
      for (int t = 0; t < q.taps; ++t)
        std::memcpy(&h[static_cast<size_t>(co) * q.Kp + static_cast<size_t>(t) * q.cin_pack],
                    row + static_cast<size_t>(t) * q.cin_src * 2, static_cast<size_t>(q.cin_src) * 2);
    }
    void* ptr = nullptr;
    if (hipMalloc(&ptr, h.size() * 2) != hipSuccess) throw OomError("packed weights: hipMalloc failed");
    q.dev = static_cast<uint16_t*>(ptr);
    p->weight_bytes += h.size() * 2;
    hip_check(hipMemcpy(q.dev, h.data(), h.size() * 2, hipMemcpyHostToDevice), "packed weights upload");
  }

  // folded projections: [scale | shift | s_p | b_p | 1 / scale] of the
  // block's last convolution (scale 1 where it is 0) and the projection
  p->fold_shift.assign(sp.n_fold_shift, nullptr);
  for (const Node& nd : sp.nodes) {
    if (!nd.fold) continue;
    const size_t C = static_cast<size_t>(nd.cout);
    std::vector<float> ss(5 * C);
    for (size_t co = 0; co < C; ++co) {
      const float s1 = nd.scale_off >= 0 ? hf32(nd.scale_off, static_cast<int>(co)) : 1.0f;
      const float sc = s1 != 0.0f ? s1 : 1.0f;
      ss[co] = sc;
      ss[C + co] = nd.shift_off >= 0 ? hf32(nd.shift_off, static_cast<int>(co)) : 0.0f;
      ss[2 * C + co] = nd.scale2_off >= 0 ? hf32(nd.scale2_off, static_cast<int>(co)) : 1.0f;
      ss[3 * C + co] = nd.shift2_off >= 0 ? hf32(nd.shift2_off, static_cast<int>(co)) : 0.0f;
      ss[4 * C + co] = 1.0f / sc;
    }
    void* ptr = nullptr;
    if (hipMalloc(&ptr, ss.size() * 4) != hipSuccess) throw OomError("folded projection constants: hipMalloc failed");
    p->fold_shift[nd.fold_shift] = static_cast<float*>(ptr);
    p->weight_bytes += ss.size() * 4;
    hip_check(hipMemcpy(ptr, ss.data(), ss.size() * 4, hipMemcpyHostToDevice), "folded projection constants upload");
  }

  // LSTM steps: the gate bias in the interleaved order of the packed rows
  p->lstm_shift.assign(sp.n_lstm_shift, nullptr);
  std::function<void(const std::vector<Node>&)> lstm_walk = [&](const std::vector<Node>& nodes) {
    for (const Node& nd : nodes) {
      if (nd.lstm_shift >= 0) {
        const int H = nd.cout / 4;
        std::vector<float> b(static_cast<size_t>(nd.cout), 0.0f);
        for (int co = 0; co < nd.cout; ++co)
          if (nd.shift_off >= 0) b[co] = hf32(nd.shift_off, (co % 4) * H + co / 4);
        void* ptr = nullptr;
        if (hipMalloc(&ptr, b.size() * 4) != hipSuccess) throw OomError("LSTM bias: hipMalloc failed");
        p->lstm_shift[nd.lstm_shift] = static_cast<float*>(ptr);
        p->weight_bytes += b.size() * 4;
        hip_check(hipMemcpy(ptr, b.data(), b.size() * 4, hipMemcpyHostToDevice), "LSTM bias upload");
      }
      lstm_walk(nd.body);
    }
  };
  lstm_walk(sp.nodes);

  // fp32 weight matrices [rows][cols] kept transposed ([cols][rows]): exit
  // heads and fp32 linear layers
  p->head_t.assign(sp.n_head_t, nullptr);
  for (const Node& nd : sp.nodes) {
    if (nd.head_t < 0) continue;
    const bool ex = nd.kind == NodeKind::Exit;
    const int rows = ex ? nd.ncls : nd.cout, cols = ex ? nd.hc : nd.cin1;
    std::vector<float> wt(static_cast<size_t>(rows) * cols);
    const float* w = reinterpret_cast<const float*>(hb + (ex ? nd.h_w : nd.w_off));
    for (int j = 0; j < rows; ++j)
      for (int c = 0; c < cols; ++c) wt[static_cast<size_t>(c) * rows + j] = w[static_cast<size_t>(j) * cols + c];
    void* ptr = nullptr;
    if (hipMalloc(&ptr, wt.size() * 4) != hipSuccess) throw OomError("head weights: hipMalloc failed");
    p->head_t[nd.head_t] = static_cast<float*>(ptr);
    p->weight_bytes += wt.size() * 4;
    hip_check(hipMemcpy(ptr, wt.data(), wt.size() * 4, hipMemcpyHostToDevice), "head weights upload");
  }

  assign_buffers(p, p->max_batch);
  const int B = p->max_batch;
  detect_act_loop(p);
  if (p->act.ok) {
    p->act.h[0] = dev_alloc<uint16_t>(p, static_cast<size_t>(B) * p->act.hidden, "persistent loop state");
    p->act.h[1] = dev_alloc<uint16_t>(p, static_cast<size_t>(B) * p->act.hidden, "persistent loop state");
  }
  p->d_flags = dev_alloc<uint8_t>(p, B, "flags");
  p->d_idx1 = dev_alloc<int32_t>(p, B, "idx1");
  p->d_org1 = dev_alloc<int32_t>(p, B, "org1");
  p->d_idx0 = dev_alloc<int32_t>(p, B, "idx0");
  p->d_org0 = dev_alloc<int32_t>(p, B, "org0");
  p->d_orig[0] = dev_alloc<int32_t>(p, B, "orig0");
  p->d_orig[1] = dev_alloc<int32_t>(p, B, "orig1");
  p->d_iota = dev_alloc<int32_t>(p, B, "iota");
  p->d_counts = dev_alloc<int32_t>(p, 2 * std::max(1, sp.decisions), "counts");
  p->d_G = dev_alloc<float>(p, static_cast<size_t>(B) * sp.max_head_c, "pooled features");
  bool split_pool = false;   // a bf16 head pooled outside the fused kernel
  for (const Node& nd : sp.nodes)
    if (nd.kind == NodeKind::Exit && !nd.fused && sp.dt == DType::BF16) split_pool = true;
  if (split_pool)
    p->d_Gpart = dev_alloc<float>(p, static_cast<size_t>(k::kGapMaxSplit) * B * sp.max_head_c, "pooling partials");
  {
    // an exit head whose input a top-level conv has just written pools from
    // 32-row chunk sums taken in that conv's epilogue (when the conv's kernel
    // takes them; else the exit pools the tensor itself)
    size_t q = 0;
    std::vector<int> writer(sp.tensors.size(), -1);
    for (size_t i = 0; i < p->spec.nodes.size(); ++i) {
      Node& nd = p->spec.nodes[i];
      if (nd.kind == NodeKind::Exit && !nd.fused && sp.dt == DType::BF16 && nd.src >= 0 && writer[nd.src] >= 0 &&
          nd.H * nd.W >= 32) {
        Node& cv = p->spec.nodes[writer[nd.src]];
        if (cv.act != k::ACT_LSTM && !cv.pool && cv.dst_list == 0 && cv.cout == nd.hc) {
          cv.gap_pool = nd.gap_pool = true;
          q = std::max(q, (static_cast<size_t>(B) * nd.H * nd.W + 31) / 32 * 2 * nd.hc);
        }
      }
      // only a conv that directly precedes the exit, on the same rows, counts
      std::fill(writer.begin(), writer.end(), -1);
      if (nd.kind == NodeKind::Conv && nd.dst >= 0 && nd.body.empty()) writer[nd.dst] = static_cast<int>(i);
    }
    if (q) p->d_gapQ = dev_alloc<float>(p, q, "pooling chunk sums");
  }
  // K-split partial sums: the largest any bf16 conv layer needs at B rows
  size_t split_bytes = 0;
  std::function<void(const std::vector<Node>&)> walk = [&](const std::vector<Node>& nodes) {
    for (const Node& nd : nodes) {
      if (nd.kind == NodeKind::Conv && sp.dt == DType::BF16) {
        const int K = nd.k * nd.k * (nd.pad_in ? sp.pad_input_c : nd.cin1 + nd.cin2);
        split_bytes = std::max(split_bytes, k::conv_ksplit_bytes(B, nd.Ho, nd.Wo, nd.cout, K, false));
      }
      walk(nd.body);
    }
  };
  walk(sp.nodes);
  if (split_bytes) {
    p->d_split = dev_alloc<float>(p, split_bytes / sizeof(float), "K-split partials");
    p->split_bytes = split_bytes;
  }
  p->d_Z = dev_alloc<float>(p, static_cast<size_t>(B) * sp.max_ncls, "head logits");
  {
    size_t hp = 0;   // partial sums of the sliced exit heads
    for (const Node& nd : sp.nodes)
      if (nd.kind == NodeKind::Exit && !nd.fused && k::head_sliced_fits(nd.hc, nd.ncls))
        hp = std::max(hp, k::head_partials_floats(nd.hc, B, nd.ncls));
    if (hp) p->d_headP = dev_alloc<float>(p, hp, "exit head partial sums");
  }
  p->d_S = dev_alloc<float>(p, B, "halting sums");
  if (sp.any_decode) {
    p->d_tok[0] = dev_alloc<int32_t>(p, B, "previous tokens");
    p->d_tok[1] = dev_alloc<int32_t>(p, B, "step tokens");
  }
  p->d_zeros = dev_alloc<uint16_t>(p, 128, "zero page");
  if (B > 16384) p->d_cws = dev_alloc<uint8_t>(p, k::compact_workspace(B), "compaction workspace");
  if (sp.pad_input_c) {
    const TensorInfo& in = sp.tensors[sp.input];
    p->d_xpad = dev_alloc<uint16_t>(p, static_cast<size_t>(B) * in.H * in.W * sp.pad_input_c, "padded input");
  }
  hip_check(hipMemset(p->d_zeros, 0, 256), "zero page");
  {
    void* ptr = nullptr;
    hip_check(hipHostMalloc(&ptr, sizeof(int32_t) * 2 * std::max(1, sp.decisions), hipHostMallocDefault),
              "hipHostMalloc");
    p->h_counts = static_cast<int32_t*>(ptr);
    std::memset(p->h_counts, 0, sizeof(int32_t) * 2 * std::max(1, sp.decisions));
    ptr = nullptr;
    hip_check(hipHostMalloc(&ptr, sizeof(int32_t) * 2 * std::max(1, sp.decisions), hipHostMallocDefault),
              "hipHostMalloc");
    p->h_hint_stage = static_cast<int32_t*>(ptr);
    p->hint.assign(2 * std::max(1, sp.decisions), 0);
    hip_check(hipEventCreateWithFlags(&p->hint_ev, hipEventDisableTiming), "hipEventCreate");
  }
  k::iota_i32(p->d_iota, B, nullptr);
  hip_check(hipGetLastError(), "iota launch");
  hip_check(hipDeviceSynchronize(), "plan build");
  return DYCL_OK;
}

void plan_free(dycl_plan* p) {
  if (!p) return;
  if (p->d_blob || !p->buffers.empty()) hipSetDevice(p->device);
  if (!p->pending.empty()) {
    for (auto& e : p->pending) {
      hipEventSynchronize(e.b);
      hipEventDestroy(e.a);
      hipEventDestroy(e.b);
    }
    p->pending.clear();
  }
  for (hipEvent_t e : p->ev_free) hipEventDestroy(e);
  p->ev_free.clear();
  if (p->graph_exec) hipGraphExecDestroy(p->graph_exec);
  if (p->graph) hipGraphDestroy(p->graph);
  if (p->cap_stream) hipStreamDestroy(p->cap_stream);
  p->graph_exec = nullptr;
  p->graph = nullptr;
  p->cap_stream = nullptr;
  for (Packed& q : p->spec.packed)
    if (q.dev) hipFree(q.dev);
  for (float* h : p->head_t)
    if (h) hipFree(h);
  for (float* h : p->fold_shift)
    if (h) hipFree(h);
  for (float* h : p->lstm_shift)
    if (h) hipFree(h);
  for (void* b : p->buffers)
    if (b) hipFree(b);
  void* singles[] = {p->d_blob, p->d_flags, p->d_idx1, p->d_org1, p->d_idx0, p->d_org0, p->d_orig[0],
                     p->d_orig[1], p->d_iota, p->d_counts, p->d_G, p->d_Z, p->d_headP, p->d_S, p->d_zeros,
                     p->d_xpad, p->d_cws, p->d_Gpart, p->d_gapQ, p->d_split, p->d_tok[0], p->d_tok[1], p->act.h[0],
                     p->act.h[1]};
  for (void* s : singles)
    if (s) hipFree(s);
  if (p->h_counts) hipHostFree(p->h_counts);
  if (p->hint_ev) hipEventSynchronize(p->hint_ev);
  if (p->h_hint_stage) hipHostFree(p->h_hint_stage);
  if (p->hint_ev) hipEventDestroy(p->hint_ev);
  p->h_counts = nullptr;
  p->h_hint_stage = nullptr;
  p->hint_ev = nullptr;
}

// ------------------------------------------------------------------ run ---

namespace {

// The rows a node runs on: n rows exactly (nc null, sync mode), or at most n
// rows whose live count the kernels read from nc (device modes); `hint` is
// the live count expected (tile shapes only).
struct Rows {
  int n;
  const int32_t* nc;
  int hint;
};

struct Run {
  dycl_plan* p;
  hipStream_t s;
  const float* aux;
  float* logits;
  dycl_record* rec;
  int32_t* tokens;           // decoding: [B][max_len] emitted tokens, or null
  int B;
  bool device;               // counts stay on the device
  std::vector<void*> tp;     // tensor pointers
  std::string label;         // the node being enqueued (profiling labels)
  const int32_t* orig;       // original ids of the current rows
  int orig_next = 0;         // which d_orig buffer the next compaction fills
  int gap_tensor = -1;       // tensor whose pooling chunk sums the last conv left in d_gapQ
  int conv_launches = 0;     // alternates the implicit GEMM's tile order from one layer to the next

  hipEvent_t event() {
    if (p->ev_free.empty()) {
      hipEvent_t e;
      hip_check(hipEventCreate(&e), "hipEventCreate");
      return e;
    }
    hipEvent_t e = p->ev_free.back();
    p->ev_free.pop_back();
    return e;
  }

  template <class F>
  void launch(int cls, double flops, double bytes, F&& f) {
    if (!p->profile) {
      f();
      hip_check(hipGetLastError(), "kernel launch");
      return;
    }
    hipEvent_t a = event(), b = event();
    hip_check(hipEventRecord(a, s), "hipEventRecord");
    f();
    hip_check(hipGetLastError(), "kernel launch");
    hip_check(hipEventRecord(b, s), "hipEventRecord");
    p->pending.push_back({cls, a, b, flops, bytes, label});
  }

  const float* f32(int64_t off) const { return off < 0 ? nullptr : reinterpret_cast<const float*>(p->d_blob + off); }

  // Partition the rows by flag at decision d.  Sync mode waits for the two
  // counts (the only device->host read); device mode leaves them in
  // d_counts and returns the rows of each branch as bounded by `r`.
  void compact(Rows r, int d, int32_t* org0, Rows& ones, Rows& zeros) {
    int32_t* cnt = p->d_counts + 2 * d;
    launch(P_COMPACT, 0, r.n * (1.0 + 4.0 + 16.0), [&] {
      if (r.n <= 16384)
        k::compact(p->d_flags, orig, r.n, p->d_idx1, p->d_org1, p->d_idx0, org0, cnt, s, r.nc);
      else
        k::compact_large(p->d_flags, orig, r.n, p->d_idx1, p->d_org1, p->d_idx0, org0, cnt, p->d_cws, s, r.nc);
    });
    if (device) {
      ones = {r.n, cnt, expected(2 * d, r.n)};
      zeros = {r.n, cnt + 1, expected(2 * d + 1, r.n)};
      return;
    }
    hip_check(hipMemcpyAsync(p->h_counts + 2 * d, cnt, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, s),
              "count readback");
    hip_check(hipStreamSynchronize(s), "count readback sync");
    ones = {p->h_counts[2 * d], nullptr, p->h_counts[2 * d]};
    zeros = {p->h_counts[2 * d + 1], nullptr, p->h_counts[2 * d + 1]};
  }

  // expected count of branch i: an earlier run's, scaled to this batch,
  // within [1, bound]; the bound when there is none
  int expected(int i, int bound) const {
    if (!p->hint_B) return bound;
    const long e = (static_cast<long>(p->hint[i]) * B + p->hint_B - 1) / p->hint_B;
    return static_cast<int>(std::max(1L, std::min<long>(e, bound)));
  }

  void move(int cls, void* dst, const int32_t* didx, const void* src, const int32_t* sidx, size_t rb, Rows r) {
    if (r.n <= 0) return;
    launch(cls, 0, 2.0 * rb * r.n + 4.0 * r.n, [&] { k::move_rows(dst, didx, src, sidx, rb, r.n, s, r.nc); });
  }

  // every (from, to) tensor pair moved with the same index lists (row r of
  // `to` at didx[r] <- row sidx[r] of `from`; null = identity), four per launch
  void move_pairs(const std::vector<std::pair<int, int>>& pairs, const int32_t* didx, const int32_t* sidx, Rows r) {
    if (r.n <= 0 || pairs.empty()) return;
    const Spec& sp = p->spec;
    for (size_t i = 0; i < pairs.size(); i += 4) {
      k::MoveSet set{};
      double bytes = 0;
      for (size_t j = i; j < pairs.size() && j < i + 4; ++j) {
        const int from = pairs[j].first, to = pairs[j].second;
        const size_t rb = sp.tensors[from].row_bytes(sp.dt);
        set.src[set.count] = tp[from];
        set.dst[set.count] = tp[to];
        set.vpr[set.count] = rb / 16;
        ++set.count;
        bytes += 2.0 * rb * r.n + 4.0 * r.n;
      }
      launch(P_MOVE, 0, bytes, [&] { k::move_rows_multi(set, didx, sidx, r.n, s, r.nc); });
    }
  }

  void conv(const Node& nd, Rows r) {
    const Spec& sp = p->spec;
    const int n = r.n;
    const Packed* q = nd.packed >= 0 ? &sp.packed[nd.packed] : nullptr;
    const int cin = nd.cin1 + nd.cin2;
    const double M = static_cast<double>(n) * nd.Ho * nd.Wo;
    const double flops = 2.0 * M * nd.cout * nd.k * nd.k * cin;
    if (sp.dt == DType::F32) {
      const double bytes = 4.0 * (static_cast<double>(n) * (cin + nd.cout) + static_cast<double>(nd.cout) * cin);
      launch(P_LINEAR32, flops, bytes, [&] {
        k::linear_t_f32(static_cast<const float*>(tp[nd.src]), n, cin, p->head_t[nd.head_t], f32(nd.shift_off),
                        nd.cout, nd.act, static_cast<float*>(tp[nd.dst]), s, r.nc, r.hint);
      });
      return;
    }
    k::ConvArgs a;
    a.src = nd.pad_in ? p->d_xpad : static_cast<const uint16_t*>(tp[nd.src]);
    a.src2 = nd.src2 >= 0 ? static_cast<const uint16_t*>(tp[nd.src2]) : nullptr;
    if (nd.src2 >= 0) {
      a.src2_H = sp.tensors[nd.src2].H;
      a.src2_W = sp.tensors[nd.src2].W;
      a.src2_stride = nd.s2;
    }
    a.cin1 = nd.pad_in ? sp.pad_input_c : nd.cin1;
    a.cin2 = nd.cin2;
    a.n = n;
    a.H = nd.H;
    a.W = nd.W;
    a.cin = nd.pad_in ? sp.pad_input_c : cin;
    a.Ho = nd.Ho;
    a.Wo = nd.Wo;
    a.cout = nd.cout;
    a.k = nd.k;
    a.stride = nd.stride;
    a.pad = nd.pad;
    a.w = q->dev;
    a.Kp = q->Kp;
    a.scale = nd.fold ? p->fold_shift[nd.fold_shift] : f32(nd.scale_off);
    a.shift = nd.fold ? p->fold_shift[nd.fold_shift] + nd.cout : f32(nd.shift_off);
    if (nd.fold) {
      a.kfold = nd.cin2 / k::kBK;
      a.fold_sp = p->fold_shift[nd.fold_shift] + 2 * nd.cout;
      a.fold_bp = p->fold_shift[nd.fold_shift] + 3 * nd.cout;
      a.fold_inv = p->fold_shift[nd.fold_shift] + 4 * nd.cout;
    }
    a.res = nd.res >= 0 ? static_cast<const uint16_t*>(tp[nd.res]) : nullptr;
    a.act = nd.act;
    if (nd.act == k::ACT_LSTM) {
      // the concatenated input is the embedding row of each row's previous token
      a.src2 = reinterpret_cast<const uint16_t*>(p->d_blob + nd.emb_off);
      a.src2_H = a.src2_W = 1;
      a.src2_stride = 1;
      a.src2_rows = p->d_tok[0];
      a.cell_in = nd.cell_in >= 0 ? static_cast<const float*>(tp[nd.cell_in]) : nullptr;
      a.cell_out = static_cast<float*>(tp[nd.cell_out]);
      a.shift = p->lstm_shift[nd.lstm_shift];
    }
    a.dst = tp[nd.dst];
    a.out_f32 = 0;
    a.zeros = p->d_zeros;
    a.ncount = r.nc;
    a.nhint = r.hint;
    auto list = [&](int which) -> const int32_t* {
      return which == 1 ? p->d_idx0 : which == 2 ? p->d_idx1 : which == 3 ? orig : nullptr;
    };
    a.src_rows = list(nd.src_list);
    if (nd.act != k::ACT_LSTM) a.src2_rows = list(nd.src2_list);
    a.res_rows = list(nd.res_list);
    a.dst_rows = list(nd.dst_list);
    if (a.src_rows || a.res_rows || a.dst_rows) a.list_rows = p->max_batch;
    a.splitws = p->d_split;
    a.splitws_bytes = p->split_bytes;
    if (nd.pool) {
      // stem with the max-pool fused in: the pooled tensor is all it writes
      a.pool = 1;
      const TensorInfo& d = sp.tensors[nd.dst];
      const double bytes = 2.0 * (static_cast<double>(n) * (nd.H * nd.W * cin + d.H * d.W * d.C) +
                                  static_cast<double>(nd.cout) * nd.k * nd.k * cin);
      launch(P_CONV, flops, bytes, [&] {
        if (!k::conv_rgb_stem(a, s)) throw HipError("stem with fused max-pool: arguments the kernel does not take");
      });
      return;
    }
    if (nd.act == k::ACT_LSTM) {
      // h and the embedding row in, bf16 h' and float32 c (in, out) per cell
      const double H = nd.cout / 4.0;
      const double bytes = static_cast<double>(n) * (2.0 * cin + 2.0 * H + 4.0 * H * (nd.cell_in >= 0 ? 2 : 1)) +
                           2.0 * nd.cout * cin;
      launch(P_CONV, flops, bytes, [&] { k::conv_bf16(a, s); });
      return;
    }
    const double bytes = 2.0 * (static_cast<double>(n) * (nd.H * nd.W * cin + M / n * nd.cout * (nd.res >= 0 ? 2 : 1)) +
                                static_cast<double>(nd.cout) * nd.k * nd.k * cin);
    if (nd.gap_pool) a.gap_part = p->d_gapQ;
    a.rev = conv_launches++ & 1;
    launch(P_CONV, flops, bytes, [&] { gap_tensor = k::conv_bf16(a, s) ? nd.dst : -1; });
  }

  // a conv and the 1x1 conv after it in one launch (Spec::pair_pointwise);
  // false: the kernel does not take this argument set and nothing ran
  bool pair(const Node& c, const Node& d, Rows r) {
    const Spec& sp = p->spec;
    if (d.kind != NodeKind::Conv || d.gap_pool || c.gap_pool) return false;
    const int n = r.n;
    const Packed& q3 = sp.packed[c.packed];
    const Packed& q1 = sp.packed[d.packed];
    k::PairArgs a;
    a.x = static_cast<const uint16_t*>(tp[c.src]);
    a.K3 = c.cin1;
    if (c.fold) {
      const float* fs = p->fold_shift[c.fold_shift];
      a.x2 = static_cast<const uint16_t*>(tp[c.src2]);
      a.K2 = c.cin2;
      a.H2 = sp.tensors[c.src2].H;
      a.W2 = sp.tensors[c.src2].W;
      a.s2 = c.s2;
      // the pair kernel indexes the projection input's pixels in 32 bits
      if (static_cast<long>(r.n) * a.H2 * a.W2 > 0x7fffffffL) return false;
      a.scale3 = fs;
      a.shift3 = fs + c.cout;
      a.fold_sp = fs + 2 * c.cout;
      a.fold_bp = fs + 3 * c.cout;
      a.fold_inv = fs + 4 * c.cout;
    } else {
      a.scale3 = f32(c.scale_off);
      a.shift3 = f32(c.shift_off);
      a.res = c.res >= 0 ? static_cast<const uint16_t*>(tp[c.res]) : nullptr;
    }
    a.w3 = q3.dev;
    a.Kp3 = q3.Kp;
    a.y3 = static_cast<uint16_t*>(tp[c.dst]);
    a.C3 = c.cout;
    a.w1 = q1.dev;
    a.Kp1 = q1.Kp;
    a.scale1 = f32(d.scale_off);
    a.shift1 = f32(d.shift_off);
    a.y1 = static_cast<uint16_t*>(tp[d.dst]);
    a.C1 = d.cout;
    a.act3 = c.act;
    a.act1 = d.act;
    a.n = n;
    a.H = c.Ho;
    a.W = c.Wo;
    a.ncount = r.nc;
    a.zeros = p->d_zeros;
    a.rev = conv_launches & 1;
    if (!k::conv_pair_takes(a)) return false;
    const double M = static_cast<double>(n) * c.Ho * c.Wo;
    const double x2 = c.fold ? static_cast<double>(n) * c.Ho * c.Wo * c.cin2 : 0.0;   // read at the output pixels
    const double flops = 2.0 * M * (static_cast<double>(c.cout) * (c.cin1 + c.cin2) + static_cast<double>(d.cout) * d.cin1);
    const double bytes = 2.0 * (M * (c.cin1 + c.cout * (c.res >= 0 ? 2.0 : 1.0) + d.cout) + x2 +
                                static_cast<double>(c.cout) * (c.cin1 + c.cin2) + static_cast<double>(d.cout) * d.cin1);
    if (p->profile) label = node_label(c) + " + " + node_label(d);
    launch(P_CONV, flops, bytes, [&] {
      if (!k::conv_pair(a, s)) throw HipError("conv pair: arguments the kernel does not take");
    });
    ++conv_launches;
    gap_tensor = -1;
    return true;
  }

  // what a profiled launch belongs to: a layer by the tensor it writes (a
  // folded projection named with it), a decision by its kind and index
  std::string node_label(const Node& nd) const {
    const Spec& sp = p->spec;
    switch (nd.kind) {
      case NodeKind::Conv:
        return sp.tensors[nd.dst].name + (nd.fold ? " (+ projection of " + sp.tensors[nd.src2].name + ")" : "") +
               (nd.pool ? " (+ max-pool)" : "");
      case NodeKind::MaxPool: return "maxpool " + sp.tensors[nd.dst].name;
      case NodeKind::Exit: return "exit " + std::to_string(nd.index);
      case NodeKind::Gate: return "gate " + std::to_string(nd.index);
      case NodeKind::Halt: return "halt " + std::to_string(nd.index);
      case NodeKind::Output: return "output";
      case NodeKind::Decode: return "decode " + std::to_string(nd.index);
    }
    return "";
  }

  void exec(const std::vector<Node>& nodes, Rows& rows) { exec_range(nodes, 0, nodes.size(), rows); }

  // the persistent launch of an adaptive-computation-time loop (device
  // host mode): every step of nodes [act.begin, act.end) in one kernel
  void act_loop() {
    const Spec& sp = p->spec;
    const auto& L = p->act;
    const Packed& q = sp.packed[L.packed];
    k::ActLoopArgs a;
    a.x = static_cast<const uint16_t*>(tp[L.input]);
    a.w = q.dev;
    a.Kp = q.Kp;
    a.b1 = f32(L.b1);
    a.wh = f32(L.wh);
    a.aux = aux;
    a.h0 = L.h[0];
    a.h1 = L.h[1];
    a.park = static_cast<uint16_t*>(tp[L.park]);
    a.S = p->d_S;
    a.flags = p->d_flags;
    a.counts = p->d_counts;
    a.d0 = L.d0;
    a.rec = rec;
    a.zeros = p->d_zeros;
    a.B = B;
    a.H = L.hidden;
    a.D = L.d_in;
    a.steps = L.steps;
    a.tau = L.tau;
    // work bound: every row for every step (the live rows are on the device)
    const double flops = 2.0 * B * L.hidden * (L.d_in + (L.steps - 1.0) * (L.hidden + L.d_in));
    const double bytes = 2.0 * B * (L.d_in + 2.0 * L.steps * L.hidden) + 2.0 * L.hidden * (L.hidden + L.d_in);
    launch(P_CONV, flops, bytes, [&] { k::act_loop(a, s); });
  }

  void exec_range(const std::vector<Node>& nodes, size_t first, size_t last, Rows& rows) {
    Spec& sp = p->spec;
    for (size_t ni = first; ni < last; ++ni) {
      const Node& nd = nodes[ni];
      // the persistent host mode runs the loop in one launch; the others
      // launch its steps one by one
      if (&nodes == &sp.nodes && p->act.ok && p->mode == DYCL_HOST_PERSISTENT && ni == p->act.begin) {
        if (p->profile) label = "act loop (persistent)";
        act_loop();
        rows = {0, nullptr, 0};   // every row halted
        ni = p->act.end - 1;
        continue;
      }
      const int n = rows.n;
      if (p->profile) label = node_label(nd);
      switch (nd.kind) {
        case NodeKind::Conv:
          if (n > 0) {
            if (nd.pair && ni + 1 < last && pair(nd, nodes[ni + 1], rows)) {
              ++ni;   // the second conv ran in the same launch
              break;
            }
            conv(nd, rows);
          }
          break;
        case NodeKind::MaxPool:
          if (n > 0) {
            const TensorInfo& t = sp.tensors[nd.src];
            launch(P_POOL, 0, 2.0 * n * (t.H * t.W + nd.Ho * nd.Wo) * t.C, [&] {
              k::maxpool3s2_bf16(static_cast<const uint16_t*>(tp[nd.src]), n, t.H, t.W, t.C,
                                 static_cast<uint16_t*>(tp[nd.dst]), s, rows.nc);
            });
          }
          break;
        case NodeKind::Exit: {
          if (n <= 0) break;
          const int HW = nd.H * nd.W;
          const float* G = static_cast<const float*>(tp[nd.src]);
          const double esz = sp.dt == DType::BF16 ? 2.0 : 4.0;
          if (nd.fused) {
            launch(P_HEAD, 2.0 * n * nd.hc * nd.ncls, esz * n * HW * nd.hc + 4.0 * nd.ncls * (nd.hc + 1), [&] {
              k::exit_head(tp[nd.src], sp.dt == DType::BF16, n, HW, nd.hc, f32(nd.h_w), f32(nd.h_b),
                           nd.ncls, f32(nd.h_T), nd.tau, nd.final_ ? 1 : 0, nd.index, orig, p->d_flags, logits,
                           sp.n_out, rec, s, rows.nc, rows.hint);
            });
          } else if (sp.dt == DType::BF16 && nd.gap_pool && gap_tensor == nd.src) {
            // the producing conv left 32-row chunk sums of this tensor
            launch(P_HEAD, 0, 4.0 * n * (HW / 32.0 + 2) * nd.hc, [&] {
              k::gap_chunks(p->d_gapQ, n, HW, nd.hc, p->d_G, s, rows.nc);
            });
            G = p->d_G;
          } else if (sp.dt == DType::BF16) {
            launch(P_HEAD, 0, 2.0 * n * HW * nd.hc + 4.0 * n * nd.hc, [&] {
              k::gap_bf16(static_cast<const uint16_t*>(tp[nd.src]), n, HW, nd.hc, p->d_G, p->d_Gpart, s, rows.nc);
            });
            G = p->d_G;
          }
          if (!nd.fused && k::head_sliced_fits(nd.hc, nd.ncls)) {
            // the head linear in K slices, then the slices' sum and the decision
            launch(P_HEAD, 2.0 * n * nd.hc * nd.ncls, 4.0 * (n * (nd.hc + nd.ncls) + nd.ncls * nd.hc), [&] {
              k::exit_head_sliced(G, n, nd.hc, p->head_t[nd.head_t], f32(nd.h_b), nd.ncls, f32(nd.h_T), nd.tau,
                                  nd.final_ ? 1 : 0, nd.index, orig, p->d_flags, logits, sp.n_out, rec, p->d_headP,
                                  s, rows.nc);
            });
          } else if (!nd.fused) {
            launch(P_HEAD, 2.0 * n * nd.hc * nd.ncls, 4.0 * (n * (nd.hc + nd.ncls) + nd.ncls * nd.hc), [&] {
              k::linear_t_f32(G, n, nd.hc, p->head_t[nd.head_t], f32(nd.h_b), nd.ncls, k::ACT_NONE, p->d_Z, s,
                              rows.nc, rows.hint);
            });
            launch(P_HEAD, 0, 4.0 * n * nd.ncls * 2, [&] {
              k::exit_decide(p->d_Z, n, nd.ncls, f32(nd.h_T), nd.tau, nd.final_ ? 1 : 0, nd.index, orig, p->d_flags,
                             logits, sp.n_out, rec, s, rows.nc);
            });
          }
          if (nd.final_) {
            if (device) {
              launch(P_MISC, 0, 8.0, [&] { k::final_counts(rows.nc, n, p->d_counts + 2 * nd.decision, s); });
            } else {
              p->h_counts[2 * nd.decision] = n;
              p->h_counts[2 * nd.decision + 1] = 0;
            }
            rows = {0, nullptr, 0};
            break;
          }
          int32_t* next = p->d_orig[orig_next];
          Rows gone, stay;
          compact(rows, nd.decision, next, gone, stay);
          move_pairs(nd.pairs, nullptr, p->d_idx0, stay);
          orig = next;
          orig_next ^= 1;
          rows = stay;
          break;
        }
        case NodeKind::Gate: {
          if (n <= 0) break;
          const int HW = nd.H * nd.W;
          launch(P_HEAD, 2.0 * n * nd.hc, 2.0 * n * HW * nd.hc, [&] {
            k::gate_head(static_cast<const uint16_t*>(tp[nd.src]), n, HW, nd.hc, f32(nd.h_w), f32(nd.h_b), nd.tau,
                         nd.index, orig, p->d_flags, rec, s, rows.nc);
          });
          Rows run, skip;
          compact(rows, nd.decision, p->d_org0, run, skip);
          if (run.n > 0) {
            move_pairs(nd.pairs, nullptr, p->d_idx1, run);     // gather the executing rows
            Rows body = run;
            exec(nd.body, body);
            if (p->profile) label = node_label(nd);
            move_pairs(nd.scatter, p->d_idx1, nullptr, run);   // scatter the block outputs back
          }
          break;
        }
        case NodeKind::Halt: {
          if (n <= 0) break;
          launch(P_HEAD, 2.0 * n * nd.hc, 2.0 * n * nd.hc, [&] {
            k::halt_head(static_cast<const uint16_t*>(tp[nd.src]), n, nd.hc, f32(nd.h_w), aux, orig, p->d_S, nd.index,
                         nd.max_steps, nd.tau, p->d_flags, rec, s, rows.nc);
          });
          int32_t* next = p->d_orig[orig_next];
          Rows halted, stay;
          compact(rows, nd.decision, next, halted, stay);
          move(P_MOVE, tp[nd.park_dst], p->d_org1, tp[nd.park_src], p->d_idx1,
               sp.tensors[nd.park_src].row_bytes(sp.dt), halted);
          move_pairs(nd.pairs, nullptr, p->d_idx0, stay);
          orig = next;
          orig_next ^= 1;
          rows = stay;
          break;
        }
        case NodeKind::Decode: {
          if (n <= 0) break;
          // the step's logits (output layer, float32) ...
          const Packed& q = sp.packed[nd.packed];
          k::ConvArgs a{};
          a.src = static_cast<const uint16_t*>(tp[nd.src]);
          a.cin1 = a.cin = nd.cin1;
          a.n = n;
          a.H = a.W = a.Ho = a.Wo = 1;
          a.cout = nd.cout;
          a.k = a.stride = 1;
          a.w = q.dev;
          a.Kp = q.Kp;
          a.shift = f32(nd.shift_off);
          a.act = k::ACT_NONE;
          a.dst = p->d_Z;
          a.out_f32 = 1;
          a.zeros = p->d_zeros;
          a.ncount = rows.nc;
          a.nhint = rows.hint;
          launch(P_CONV, 2.0 * n * nd.cout * nd.cin1,
                 2.0 * n * nd.cin1 + 4.0 * n * nd.cout + 2.0 * nd.cout * nd.cin1, [&] { k::conv_bf16(a, s); });
          // ... then the token choice, the end test and the records
          launch(P_HEAD, 0, 4.0 * n * nd.ncls + 16.0 * n, [&] {
            k::decode_step(p->d_Z, n, nd.ncls, nd.eos, nd.index, nd.max_steps, orig, p->d_flags, p->d_tok[1], tokens,
                           logits, rec, s, rows.nc);
          });
          if (nd.final_) {
            if (device) {
              launch(P_MISC, 0, 8.0, [&] { k::final_counts(rows.nc, n, p->d_counts + 2 * nd.decision, s); });
            } else {
              p->h_counts[2 * nd.decision] = n;
              p->h_counts[2 * nd.decision + 1] = 0;
            }
            rows = {0, nullptr, 0};
            break;
          }
          int32_t* next = p->d_orig[orig_next];
          Rows done, stay;
          compact(rows, nd.decision, next, done, stay);
          if (stay.n > 0) {
            // the continuing rows' tokens, in their new order, for the next step's embedding rows
            launch(P_MOVE, 0, 12.0 * stay.n,
                   [&] { k::gather_i32(p->d_tok[0], p->d_tok[1], p->d_idx0, stay.n, s, stay.nc); });
            move_pairs(nd.pairs, nullptr, p->d_idx0, stay);
          }
          orig = next;
          orig_next ^= 1;
          rows = stay;
          break;
        }
        case NodeKind::Output: {
          const Packed& q = sp.packed[nd.packed];
          k::ConvArgs a{};
          a.src = static_cast<const uint16_t*>(tp[nd.src]);
          a.src2 = nullptr;
          a.cin1 = nd.cin1;
          a.cin2 = 0;
          a.n = B;
          a.H = a.W = a.Ho = a.Wo = 1;
          a.cin = nd.cin1;
          a.cout = nd.cout;
          a.k = 1;
          a.stride = 1;
          a.pad = 0;
          a.w = q.dev;
          a.Kp = q.Kp;
          a.scale = nullptr;
          a.shift = f32(nd.shift_off);
          a.res = nullptr;
          a.act = k::ACT_NONE;
          a.dst = logits;
          a.out_f32 = 1;
          a.zeros = p->d_zeros;
          a.ncount = nullptr;
          const double flops = 2.0 * B * nd.cout * nd.cin1;
          launch(P_CONV, flops, 2.0 * B * nd.cin1 + 4.0 * B * nd.cout + 2.0 * nd.cout * nd.cin1,
                 [&] { k::conv_bf16(a, s); });
          break;
        }
      }
    }
  }

  // the whole run, enqueued on s
  void all(const void* x) {
    Spec& sp = p->spec;
    tp.resize(sp.tensors.size());
    for (size_t t = 0; t < sp.tensors.size(); ++t)
      tp[t] = sp.tensors[t].external ? const_cast<void*>(x)
              : sp.tensors[t].unused ? nullptr : p->buffers[sp.tensors[t].buf];
    orig = p->d_iota;
    launch(P_MISC, 0, 16.0 * B, [&] { k::init_records(rec, B, s); });
    if (sp.any_halt) launch(P_MISC, 0, 4.0 * B, [&] { k::fill_f32(p->d_S, 0.f, B, s); });
    if (sp.any_decode) {
      launch(P_MISC, 0, 4.0 * B * sp.max_len,
             [&] { k::fill_i32(tokens, -1, static_cast<size_t>(B) * sp.max_len, s); });
      launch(P_MISC, 0, 4.0 * B, [&] { k::fill_i32(p->d_tok[0], sp.bos, static_cast<size_t>(B), s); });
    }
    if (sp.pad_input_c) {
      const TensorInfo& in = sp.tensors[sp.input];
      const size_t pix = static_cast<size_t>(B) * in.H * in.W;
      launch(P_MISC, 0, pix * 2.0 * (in.C + sp.pad_input_c), [&] {
        k::pad_channels_bf16(static_cast<const uint16_t*>(x), pix, in.C, sp.pad_input_c, p->d_xpad, s);
      });
    }
    Rows rows{B, nullptr, B};
    exec(sp.nodes, rows);
  }
};

void graph_reset(dycl_plan* p) {
  if (p->graph_exec) hipGraphExecDestroy(p->graph_exec);
  if (p->graph) hipGraphDestroy(p->graph);
  p->graph_exec = nullptr;
  p->graph = nullptr;
  p->graph_key = dycl_plan::GraphKey{};
}

}  // namespace

void plan_run(dycl_plan* p, const void* x, int B, const float* aux, float* logits, dycl_record* rec,
              int32_t* tokens, hipStream_t s) {
  Spec& sp = p->spec;
  hip_check(hipSetDevice(p->device), "hipSetDevice");
  p->last_stream = s;
  if (p->pending.size() > 8192) profile_flush(p);
  if (p->profile) {
    p->last_run.clear();
    p->last_run_labels.clear();
    p->last_run_begin = p->pending.size();
  }
  Run r;
  r.p = p;
  r.aux = aux;
  r.logits = logits;
  r.rec = rec;
  r.tokens = tokens;
  r.B = B;
  r.device = p->mode != DYCL_HOST_SYNC;
  p->counts_on_device = r.device;
  const size_t cbytes = sizeof(int32_t) * 2 * std::max(1, sp.decisions);
  if (!r.device) {
    std::memset(p->h_counts, 0, cbytes);
    r.s = s;
    r.all(x);
    std::copy(p->h_counts, p->h_counts + 2 * std::max(1, sp.decisions), p->hint.begin());
    p->hint_B = B;
    return;
  }
  // the counts of an earlier device-mode run, if their copy has landed
  if (p->hint_pending) {
    const hipError_t q = hipEventQuery(p->hint_ev);
    if (q == hipSuccess) {
      std::copy(p->h_hint_stage, p->h_hint_stage + 2 * std::max(1, sp.decisions), p->hint.begin());
      p->hint_B = p->hint_pending_B;
      p->hint_pending = false;
    } else if (q == hipErrorNotReady) {
      hipGetLastError();   // not an error: the copy is still queued
    } else {
      hip_check(q, "hipEventQuery");
    }
  }
  if (p->mode != DYCL_HOST_GRAPH || p->profile) {
    r.s = s;
    r.all(x);
    if (!p->hint_pending) {
      hip_check(hipMemcpyAsync(p->h_hint_stage, p->d_counts, cbytes, hipMemcpyDeviceToHost, s), "count copy");
      hip_check(hipEventRecord(p->hint_ev, s), "hipEventRecord");
      p->hint_pending = true;
      p->hint_pending_B = B;
    }
    return;
  }
  const dycl_plan::GraphKey key{x, B, aux, logits, rec, tokens};
  const dycl_plan::GraphKey& k0 = p->graph_key;
  if (!p->graph_exec || k0.x != key.x || k0.B != key.B || k0.aux != key.aux || k0.logits != key.logits ||
      k0.rec != key.rec || k0.tokens != key.tokens) {
    graph_reset(p);
    if (!p->cap_stream) hip_check(hipStreamCreateWithFlags(&p->cap_stream, hipStreamNonBlocking), "hipStreamCreate");
    // the capture stream only records: nothing runs on it
    r.s = p->cap_stream;
    hip_check(hipStreamBeginCapture(p->cap_stream, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
    try {
      r.all(x);
    } catch (...) {
      hipGraph_t g = nullptr;
      hipStreamEndCapture(p->cap_stream, &g);
      if (g) hipGraphDestroy(g);
      hipGetLastError();
      throw;
    }
    hip_check(hipStreamEndCapture(p->cap_stream, &p->graph), "hipStreamEndCapture");
    hip_check(hipGraphInstantiate(&p->graph_exec, p->graph, nullptr, nullptr, 0), "hipGraphInstantiate");
    p->graph_key = key;
    ++p->graph_captures;
  }
  hip_check(hipGraphLaunch(p->graph_exec, s), "hipGraphLaunch");
}

void plan_set_mode(dycl_plan* p, int mode) {
  if (mode != p->mode) {
    hip_check(hipSetDevice(p->device), "hipSetDevice");
    graph_reset(p);
  }
  p->mode = mode;
}

void plan_read_counts(const dycl_plan* p, int32_t* out, int n) {
  const int total = 2 * p->spec.decisions;
  const int m = std::min(n, total);
  if (m <= 0) return;
  if (!p->counts_on_device) {
    std::copy(p->h_counts, p->h_counts + m, out);
    return;
  }
  hip_check(hipSetDevice(p->device), "hipSetDevice");
  hip_check(hipStreamSynchronize(p->last_stream), "hipStreamSynchronize");
  hip_check(hipMemcpy(out, p->d_counts, m * sizeof(int32_t), hipMemcpyDeviceToHost), "count read");
}

void profile_flush(dycl_plan* p) {
  for (size_t i = 0; i < p->pending.size(); ++i) {
    auto& e = p->pending[i];
    hip_check(hipEventSynchronize(e.b), "hipEventSynchronize");
    float ms = 0.f;
    hip_check(hipEventElapsedTime(&ms, e.a, e.b), "hipEventElapsedTime");
    ProfileRow& row = p->prof[e.cls];
    row.launches += 1;
    row.ms += ms;
    row.flops += e.flops;
    row.bytes += e.bytes;
    if (i >= p->last_run_begin) {
      p->last_run.push_back({static_cast<double>(e.cls), ms, e.flops, e.bytes});
      p->last_run_labels.push_back(e.label);
    }
    p->ev_free.push_back(e.a);
    p->ev_free.push_back(e.b);
  }
  p->pending.clear();
  p->last_run_begin = 0;
}

}  // namespace dycl
