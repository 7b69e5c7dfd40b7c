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
#include <cstring>

#include "plan.hpp"

namespace dycl {

namespace {

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) throw HipError(std::string(what) + ": " + hipGetErrorString(e));
}

template <class T>
T* dev_alloc(dycl_plan* p, size_t count, const char* what) {
  void* ptr = nullptr;
  const size_t bytes = std::max<size_t>(count * sizeof(T), 256);
  hipError_t e = hipMalloc(&ptr, bytes);
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
    throw OomError(std::string(what) + ": hipMalloc of " + std::to_string(bytes) + " bytes failed");
  hip_check(e, what);
  p->workspace_bytes += bytes;
  return static_cast<T*>(ptr);
}

void assign_buffers(dycl_plan* p, int max_batch) {
  Spec& sp = p->spec;
  std::vector<int> order;
  for (int i = 0; i < static_cast<int>(sp.tensors.size()); ++i)
    if (!sp.tensors[i].external) order.push_back(i);
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

}  // namespace

int plan_build(dycl_plan* p, const std::string& json, const void* weights, size_t weights_bytes) {
  Spec& sp = p->spec;
  sp.parse(json, weights_bytes, p->max_batch);
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
  for (Packed& q : sp.packed) {
    std::vector<uint16_t> h(static_cast<size_t>(q.cout_pad) * q.Kp, 0);
    for (int co = 0; co < q.cout; ++co) {
      const uint8_t* row = hb + q.w_off + (static_cast<size_t>(co) * q.w_ldk + q.w_k0) * 2;
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
  p->d_Z = dev_alloc<float>(p, static_cast<size_t>(B) * sp.max_ncls, "head logits");
  p->d_S = dev_alloc<float>(p, B, "halting sums");
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
  for (Packed& q : p->spec.packed)
    if (q.dev) hipFree(q.dev);
  for (float* h : p->head_t)
    if (h) hipFree(h);
  for (void* b : p->buffers)
    if (b) hipFree(b);
  void* singles[] = {p->d_blob, p->d_flags, p->d_idx1, p->d_org1, p->d_idx0, p->d_org0, p->d_orig[0],
                     p->d_orig[1], p->d_iota, p->d_counts, p->d_G, p->d_Z, p->d_S, p->d_zeros,
                     p->d_xpad, p->d_cws, p->d_Gpart};
  for (void* s : singles)
    if (s) hipFree(s);
  if (p->h_counts) hipHostFree(p->h_counts);
}

// ------------------------------------------------------------------ run ---

namespace {

struct Run {
  dycl_plan* p;
  hipStream_t s;
  const float* aux;
  float* logits;
  dycl_record* rec;
  int B;
  std::vector<void*> tp;     // tensor pointers
  const int32_t* orig;       // original ids of the current rows
  int orig_next = 0;         // which d_orig buffer the next compaction fills

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
    p->pending.push_back({cls, a, b, flops, bytes});
  }

  const float* f32(int64_t off) const { return off < 0 ? nullptr : reinterpret_cast<const float*>(p->d_blob + off); }

  // wait for the branch counts of decision d (the only device->host read)
  void read_counts(int d) {
    hip_check(hipMemcpyAsync(p->h_counts + 2 * d, p->d_counts + 2 * d, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, s),
              "count readback");
    hip_check(hipStreamSynchronize(s), "count readback sync");
  }

  void compact(int n, int d, int32_t* org0) {
    const Spec& sp = p->spec;
    (void)sp;
    launch(P_COMPACT, 0, n * (1.0 + 4.0 + 16.0), [&] {
      if (n <= 16384)
        k::compact(p->d_flags, orig, n, p->d_idx1, p->d_org1, p->d_idx0, org0, p->d_counts + 2 * d, s);
      else
        k::compact_large(p->d_flags, orig, n, p->d_idx1, p->d_org1, p->d_idx0, org0, p->d_counts + 2 * d, p->d_cws, s);
    });
    read_counts(d);
  }

  void move(int cls, void* dst, const int32_t* didx, const void* src, const int32_t* sidx, size_t rb, int n) {
    if (n <= 0) return;
    launch(cls, 0, 2.0 * rb * n + 4.0 * n, [&] { k::move_rows(dst, didx, src, sidx, rb, n, s); });
  }

  // every (from, to) tensor pair moved with the same index lists (row r of
  // `to` at didx[r] <- row sidx[r] of `from`; null = identity), four per launch
  void move_pairs(const std::vector<std::pair<int, int>>& pairs, const int32_t* didx, const int32_t* sidx, int n) {
    if (n <= 0 || pairs.empty()) return;
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
        bytes += 2.0 * rb * n + 4.0 * n;
      }
      launch(P_MOVE, 0, bytes, [&] { k::move_rows_multi(set, didx, sidx, n, s); });
    }
  }

  void conv(const Node& nd, int n) {
    const Spec& sp = p->spec;
    const Packed* q = nd.packed >= 0 ? &sp.packed[nd.packed] : nullptr;
    const int cin = nd.cin1 + nd.cin2;
    const double M = static_cast<double>(n) * nd.Ho * nd.Wo;
    const double flops = 2.0 * M * nd.cout * nd.k * nd.k * cin;
    if (sp.dt == DType::F32) {
      const double bytes = 4.0 * (static_cast<double>(n) * (cin + nd.cout) + static_cast<double>(nd.cout) * cin);
      launch(P_LINEAR32, flops, bytes, [&] {
        k::linear_t_f32(static_cast<const float*>(tp[nd.src]), n, cin, p->head_t[nd.head_t], f32(nd.shift_off),
                        nd.cout, nd.act, static_cast<float*>(tp[nd.dst]), s);
      });
      return;
    }
    k::ConvArgs a;
    a.src = nd.pad_in ? p->d_xpad : static_cast<const uint16_t*>(tp[nd.src]);
    a.src2 = nd.src2 >= 0 ? static_cast<const uint16_t*>(tp[nd.src2]) : nullptr;
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
    a.scale = f32(nd.scale_off);
    a.shift = f32(nd.shift_off);
    a.res = nd.res >= 0 ? static_cast<const uint16_t*>(tp[nd.res]) : nullptr;
    a.act = nd.act;
    a.dst = tp[nd.dst];
    a.out_f32 = 0;
    a.zeros = p->d_zeros;
    const double bytes = 2.0 * (static_cast<double>(n) * (nd.H * nd.W * cin + M / n * nd.cout * (nd.res >= 0 ? 2 : 1)) +
                                static_cast<double>(nd.cout) * nd.k * nd.k * cin);
    launch(P_CONV, flops, bytes, [&] { k::conv_bf16(a, s); });
  }

  void exec(const std::vector<Node>& nodes, int& n) {
    Spec& sp = p->spec;
    for (const Node& nd : nodes) {
      switch (nd.kind) {
        case NodeKind::Conv:
          if (n > 0) conv(nd, n);
          break;
        case NodeKind::MaxPool:
          if (n > 0) {
            const TensorInfo& t = sp.tensors[nd.src];
            launch(P_POOL, 0, 2.0 * n * (t.H * t.W + nd.Ho * nd.Wo) * t.C, [&] {
              k::maxpool3s2_bf16(static_cast<const uint16_t*>(tp[nd.src]), n, t.H, t.W, t.C,
                                 static_cast<uint16_t*>(tp[nd.dst]), s);
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
                           sp.n_out, rec, s);
            });
          } else if (sp.dt == DType::BF16) {
            launch(P_HEAD, 0, 2.0 * n * HW * nd.hc + 4.0 * n * nd.hc, [&] {
              k::gap_bf16(static_cast<const uint16_t*>(tp[nd.src]), n, HW, nd.hc, p->d_G, p->d_Gpart, s);
            });
            G = p->d_G;
          }
          if (!nd.fused) {
            launch(P_HEAD, 2.0 * n * nd.hc * nd.ncls, 4.0 * (n * (nd.hc + nd.ncls) + nd.ncls * nd.hc), [&] {
              k::linear_t_f32(G, n, nd.hc, p->head_t[nd.head_t], f32(nd.h_b), nd.ncls, k::ACT_NONE, p->d_Z, s);
            });
            launch(P_HEAD, 0, 4.0 * n * nd.ncls * 2, [&] {
              k::exit_decide(p->d_Z, n, nd.ncls, f32(nd.h_T), nd.tau, nd.final_ ? 1 : 0, nd.index, orig, p->d_flags,
                             logits, sp.n_out, rec, s);
            });
          }
          if (nd.final_) {
            p->h_counts[2 * nd.decision] = n;
            p->h_counts[2 * nd.decision + 1] = 0;
            n = 0;
            break;
          }
          int32_t* next = p->d_orig[orig_next];
          compact(n, nd.decision, next);
          const int stay = p->h_counts[2 * nd.decision + 1];
          move_pairs(nd.pairs, nullptr, p->d_idx0, stay);
          orig = next;
          orig_next ^= 1;
          n = stay;
          break;
        }
        case NodeKind::Gate: {
          if (n <= 0) break;
          const int HW = nd.H * nd.W;
          launch(P_HEAD, 2.0 * n * nd.hc, 2.0 * n * HW * nd.hc, [&] {
            k::gate_head(static_cast<const uint16_t*>(tp[nd.src]), n, HW, nd.hc, f32(nd.h_w), f32(nd.h_b), nd.tau,
                         nd.index, orig, p->d_flags, rec, s);
          });
          compact(n, nd.decision, p->d_org0);
          int ne = p->h_counts[2 * nd.decision];
          if (ne > 0) {
            move_pairs(nd.pairs, nullptr, p->d_idx1, ne);     // gather the executing rows
            int nb = ne;
            exec(nd.body, nb);
            move_pairs(nd.scatter, p->d_idx1, nullptr, ne);   // scatter the block outputs back
          }
          break;
        }
        case NodeKind::Halt: {
          if (n <= 0) break;
          launch(P_HEAD, 2.0 * n * nd.hc, 2.0 * n * nd.hc, [&] {
            k::halt_head(static_cast<const uint16_t*>(tp[nd.src]), n, nd.hc, f32(nd.h_w), aux, orig, p->d_S, nd.index,
                         nd.max_steps, nd.tau, p->d_flags, rec, s);
          });
          int32_t* next = p->d_orig[orig_next];
          compact(n, nd.decision, next);
          const int nh = p->h_counts[2 * nd.decision], stay = p->h_counts[2 * nd.decision + 1];
          move(P_MOVE, tp[nd.park_dst], p->d_org1, tp[nd.park_src], p->d_idx1,
               sp.tensors[nd.park_src].row_bytes(sp.dt), nh);
          move_pairs(nd.pairs, nullptr, p->d_idx0, stay);
          orig = next;
          orig_next ^= 1;
          n = stay;
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
          const double flops = 2.0 * B * nd.cout * nd.cin1;
          launch(P_CONV, flops, 2.0 * B * nd.cin1 + 4.0 * B * nd.cout + 2.0 * nd.cout * nd.cin1,
                 [&] { k::conv_bf16(a, s); });
          break;
        }
      }
    }
  }
};

}  // namespace

void plan_run(dycl_plan* p, const void* x, int B, const float* aux, float* logits, dycl_record* rec,
              hipStream_t s) {
  Spec& sp = p->spec;
  hip_check(hipSetDevice(p->device), "hipSetDevice");
  p->last_stream = s;
  std::memset(p->h_counts, 0, sizeof(int32_t) * 2 * std::max(1, sp.decisions));
  if (p->pending.size() > 8192) profile_flush(p);
  Run r;
  r.p = p;
  r.s = s;
  r.aux = aux;
  r.logits = logits;
  r.rec = rec;
  r.B = B;
  r.tp.resize(sp.tensors.size());
  for (size_t t = 0; t < sp.tensors.size(); ++t)
    r.tp[t] = sp.tensors[t].external ? const_cast<void*>(x) : p->buffers[sp.tensors[t].buf];
  r.orig = p->d_iota;
  r.launch(P_MISC, 0, 16.0 * B, [&] { k::init_records(rec, B, s); });
  if (sp.any_halt) r.launch(P_MISC, 0, 4.0 * B, [&] { k::fill_f32(p->d_S, 0.f, B, s); });
  if (sp.pad_input_c) {
    const TensorInfo& in = sp.tensors[sp.input];
    const size_t pix = static_cast<size_t>(B) * in.H * in.W;
    r.launch(P_MISC, 0, pix * 2.0 * (in.C + sp.pad_input_c), [&] {
      k::pad_channels_bf16(static_cast<const uint16_t*>(x), pix, in.C, sp.pad_input_c, p->d_xpad, s);
    });
  }
  int n = B;
  r.exec(sp.nodes, n);
}

void profile_flush(dycl_plan* p) {
  for (auto& e : p->pending) {
    hip_check(hipEventSynchronize(e.b), "hipEventSynchronize");
    float ms = 0.f;
    hip_check(hipEventElapsedTime(&ms, e.a, e.b), "hipEventElapsedTime");
    ProfileRow& row = p->prof[e.cls];
    row.launches += 1;
    row.ms += ms;
    row.flops += e.flops;
    row.bytes += e.bytes;
    p->ev_free.push_back(e.a);
    p->ev_free.push_back(e.b);
  }
  p->pending.clear();
}

}  // namespace dycl
