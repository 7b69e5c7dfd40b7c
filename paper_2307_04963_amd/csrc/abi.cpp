// C ABI: argument checks, error mapping, and the thread-local message.
// Nothing thrown inside the library crosses this boundary.
#include <algorithm>
#include <cstring>
#include <new>
#include <string>

#include "plan.hpp"

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

bool valid(const dycl_plan* p) { return p != nullptr && p->magic == 0x44594350u; }

const char* kClassNames[dycl::P_COUNT] = {"conv_bf16_mfma", "linear_f32", "decision_heads", "compaction",
                                          "gather_scatter", "maxpool", "misc"};

template <class F>
int guarded(F&& f) {
  try {
    return f();
  } catch (const dycl::WeightsError& e) {
    return fail(DYCL_E_WEIGHTS, e.what());
  } catch (const dycl::SpecError& e) {
    return fail(DYCL_E_SPEC, e.what());
  } catch (const dycl::OomError& e) {
    return fail(DYCL_E_OOM, e.what());
  } catch (const dycl::HipError& e) {
    return fail(DYCL_E_HIP, e.what());
  } catch (const std::bad_alloc&) {
    return fail(DYCL_E_OOM, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(DYCL_E_INVALID, e.what());
  } catch (...) {
    return fail(DYCL_E_INVALID, "unknown failure");
  }
}

}  // namespace

extern "C" {

int dycl_plan_create(const char* spec_json, const void* weights, size_t weights_bytes, int max_batch, int device,
                     dycl_plan** out) {
  if (out) *out = nullptr;
  if (!spec_json || !out) return fail(DYCL_E_INVALID, "dycl_plan_create: null spec or out pointer");
  if (!weights && weights_bytes) return fail(DYCL_E_INVALID, "dycl_plan_create: null weights");
  if (max_batch < 1) return fail(DYCL_E_BATCH, "dycl_plan_create: max_batch must be >= 1");
  if (device < 0) return fail(DYCL_E_INVALID, "dycl_plan_create: negative device");
  dycl_plan* p = new (std::nothrow) dycl_plan();
  if (!p) return fail(DYCL_E_OOM, "host allocation failed");
  p->device = device;
  p->max_batch = max_batch;
  int rc = guarded([&] { return dycl::plan_build(p, spec_json, weights, weights_bytes); });
  if (rc != DYCL_OK) {
    dycl::plan_free(p);
    p->magic = 0;
    delete p;
    return rc;
  }
  *out = p;
  g_err.clear();
  return DYCL_OK;
}

namespace {

int run_checked(const char* fn, dycl_plan* plan, const void* x_dev, int batch, const float* aux_dev,
                float* logits_dev, dycl_record* records_dev, int32_t* tokens_dev, void* hip_stream) {
  const std::string f(fn);
  if (!valid(plan)) return fail(DYCL_E_INVALID, f + ": invalid plan handle");
  if (batch < 0 || batch > plan->max_batch)
    return fail(DYCL_E_BATCH, f + ": batch " + std::to_string(batch) + " outside [0, " +
                                  std::to_string(plan->max_batch) + "]");
  if (batch == 0) return DYCL_OK;
  if (!x_dev || !logits_dev || !records_dev) return fail(DYCL_E_INVALID, f + ": null input or output pointer");
  if (plan->spec.aux && !aux_dev) return fail(DYCL_E_INVALID, f + ": this plan reads per-sample aux inputs");
  // a decoding run copies logits rows as 16-byte vectors
  const uintptr_t la = tokens_dev ? 15 : 3;
  if ((reinterpret_cast<uintptr_t>(x_dev) & 15) || (reinterpret_cast<uintptr_t>(logits_dev) & la) ||
      (reinterpret_cast<uintptr_t>(records_dev) & 7) || (reinterpret_cast<uintptr_t>(tokens_dev) & 3))
    return fail(DYCL_E_INVALID, f + ": x must be 16-byte aligned, logits 4 (16 for dycl_run_seq), records 8, "
                                    "tokens 4");
  return guarded([&] {
    dycl::plan_run(plan, x_dev, batch, aux_dev, logits_dev, records_dev, tokens_dev,
                   static_cast<hipStream_t>(hip_stream));
    return DYCL_OK;
  });
}

}  // namespace

int dycl_run(dycl_plan* plan, const void* x_dev, int batch, const float* aux_dev, float* logits_dev,
             dycl_record* records_dev, void* hip_stream) {
  if (valid(plan) && plan->spec.any_decode)
    return fail(DYCL_E_INVALID, "dycl_run: this plan emits token sequences; call dycl_run_seq");
  return run_checked("dycl_run", plan, x_dev, batch, aux_dev, logits_dev, records_dev, nullptr, hip_stream);
}

int dycl_run_seq(dycl_plan* plan, const void* x_dev, int batch, const float* aux_dev, float* logits_dev,
                 dycl_record* records_dev, int32_t* tokens_dev, void* hip_stream) {
  if (valid(plan) && !plan->spec.any_decode)
    return fail(DYCL_E_INVALID, "dycl_run_seq: this plan emits no tokens; call dycl_run");
  if (batch > 0 && !tokens_dev) return fail(DYCL_E_INVALID, "dycl_run_seq: null tokens");
  return run_checked("dycl_run_seq", plan, x_dev, batch, aux_dev, logits_dev, records_dev, tokens_dev, hip_stream);
}

int dycl_plan_set_host_mode(dycl_plan* plan, int mode) {
  if (!valid(plan)) return fail(DYCL_E_INVALID, "dycl_plan_set_host_mode: invalid plan handle");
  if (mode != DYCL_HOST_SYNC && mode != DYCL_HOST_DEVICE && mode != DYCL_HOST_GRAPH && mode != DYCL_HOST_PERSISTENT)
    return fail(DYCL_E_INVALID, "dycl_plan_set_host_mode: unknown mode " + std::to_string(mode));
  const int prev = plan->mode;
  const int rc = guarded([&] {
    dycl::plan_set_mode(plan, mode);
    return DYCL_OK;
  });
  return rc == DYCL_OK ? prev : rc;
}

int dycl_last_counts(const dycl_plan* plan, int32_t* counts, int n) {
  if (!valid(plan)) return fail(DYCL_E_INVALID, "dycl_last_counts: invalid plan handle");
  if (n < 0 || (n > 0 && !counts)) return fail(DYCL_E_INVALID, "dycl_last_counts: bad buffer");
  const int rc = guarded([&] {
    dycl::plan_read_counts(plan, counts, n);
    return DYCL_OK;
  });
  return rc == DYCL_OK ? plan->spec.decisions : rc;
}

int dycl_plan_info(const dycl_plan* plan, int64_t* info, int n) {
  if (!valid(plan)) return fail(DYCL_E_INVALID, "dycl_plan_info: invalid plan handle");
  if (n < 0 || (n > 0 && !info)) return fail(DYCL_E_INVALID, "dycl_plan_info: bad buffer");
  const dycl::Spec& sp = plan->spec;
  const dycl::TensorInfo& in = sp.tensors[sp.input];
  const int64_t v[11] = {sp.n_out,
                         static_cast<int64_t>(in.row_bytes(sp.dt)),
                         sp.decisions,
                         static_cast<int64_t>(plan->workspace_bytes),
                         static_cast<int64_t>(plan->weight_bytes),
                         plan->max_batch,
                         sp.aux ? 1 : 0,
                         sp.nodes_total,
                         plan->mode,
                         plan->graph_captures,
                         sp.any_decode ? sp.max_len : 0};
  int w = 0;
  for (; w < n && w < 11; ++w) info[w] = v[w];
  return w;
}

int dycl_profile_enable(dycl_plan* plan, int on) {
  if (!valid(plan)) return fail(DYCL_E_INVALID, "dycl_profile_enable: invalid plan handle");
  return guarded([&] {
    dycl::profile_flush(plan);
    for (auto& r : plan->prof) r = dycl::ProfileRow();
    plan->profile = on != 0;
    return DYCL_OK;
  });
}

int dycl_profile_read(dycl_plan* plan, double* rows, int cap) {
  if (!valid(plan)) return fail(DYCL_E_INVALID, "dycl_profile_read: invalid plan handle");
  if (cap < 0 || (cap > 0 && !rows)) return fail(DYCL_E_INVALID, "dycl_profile_read: bad buffer");
  int rc = guarded([&] {
    hipSetDevice(plan->device);
    dycl::profile_flush(plan);
    return DYCL_OK;
  });
  if (rc != DYCL_OK) return rc;
  for (int c = 0; c < dycl::P_COUNT && c < cap; ++c) {
    rows[4 * c + 0] = plan->prof[c].launches;
    rows[4 * c + 1] = plan->prof[c].ms;
    rows[4 * c + 2] = plan->prof[c].flops;
    rows[4 * c + 3] = plan->prof[c].bytes;
  }
  return dycl::P_COUNT;
}

int dycl_profile_launches(dycl_plan* plan, double* rows, int cap) {
  if (!valid(plan)) return fail(DYCL_E_INVALID, "dycl_profile_launches: invalid plan handle");
  if (cap < 0 || (cap > 0 && !rows)) return fail(DYCL_E_INVALID, "dycl_profile_launches: bad buffer");
  int rc = guarded([&] {
    hipSetDevice(plan->device);
    dycl::profile_flush(plan);
    return DYCL_OK;
  });
  if (rc != DYCL_OK) return rc;
  const size_t n = plan->last_run.size();
  for (size_t i = 0; i < n && i < static_cast<size_t>(cap); ++i)
    for (int j = 0; j < 4; ++j) rows[4 * i + j] = plan->last_run[i][j];
  return static_cast<int>(n);
}

const char* dycl_profile_launch_label(const dycl_plan* plan, int i) {
  if (!valid(plan) || i < 0 || static_cast<size_t>(i) >= plan->last_run_labels.size()) return "";
  return plan->last_run_labels[static_cast<size_t>(i)].c_str();
}

const char* dycl_profile_class(int i) {
  if (i < 0 || i >= dycl::P_COUNT) return "";
  return kClassNames[i];
}

int dycl_spec_check(const char* spec_json, size_t weights_bytes, int max_batch, char* summary, size_t cap) {
  if (!spec_json) return fail(DYCL_E_INVALID, "dycl_spec_check: null spec");
  if (max_batch < 1) return fail(DYCL_E_BATCH, "dycl_spec_check: max_batch must be >= 1");
  return guarded([&] {
    dycl::Spec sp;
    sp.parse(spec_json, weights_bytes, max_batch);
    if (summary && cap) {
      std::strncpy(summary, sp.summary.c_str(), cap - 1);
      summary[cap - 1] = '\0';
    }
    return DYCL_OK;
  });
}

void dycl_plan_destroy(dycl_plan* plan) {
  if (!valid(plan)) return;
  dycl::plan_free(plan);
  plan->magic = 0;
  delete plan;
}

const char* dycl_last_error(void) { return g_err.c_str(); }

}  // extern "C"

// ------------------------------------------------------------ routing ops ---

#include "../../include/dycl_ops.h"

static_assert(DYCL_OP_COMPACT_NOALLOC_MAX_N == static_cast<long long>(dycl::k::kScratchCompactMaxN),
              "header and library disagree on the no-alloc compaction's limit");
static_assert(DYCL_OP_COMPACT_NOALLOC_SCRATCH == static_cast<long long>(dycl::k::kScratchBytes),
              "header and library disagree on the static scratch size");

extern "C" {

size_t dycl_op_compact_workspace(int64_t n) {
  if (n <= 0) return 0;
  return n <= 16384 ? 0 : dycl::k::compact_workspace(static_cast<size_t>(n));
}

int dycl_op_compact(const uint8_t* flags, const int32_t* orig, int64_t n, int32_t* idx1, int32_t* org1,
                    int32_t* idx0, int32_t* org0, int32_t* counts, void* workspace, size_t workspace_bytes,
                    void* hip_stream) {
  if (n < 0 || n >= (int64_t(1) << 31)) return fail(DYCL_E_INVALID, "dycl_op_compact: n outside [0, 2^31)");
  if (!counts) return fail(DYCL_E_INVALID, "dycl_op_compact: null counts");
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (n == 0) {
    return guarded([&] {
      const int32_t z[2] = {0, 0};
      if (hipMemcpyAsync(counts, z, sizeof(z), hipMemcpyHostToDevice, s) != hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess)
        throw dycl::HipError("dycl_op_compact: clearing counts failed");
      return DYCL_OK;
    });
  }
  if (!flags || !idx1 || !idx0) return fail(DYCL_E_INVALID, "dycl_op_compact: null flags or index output");
  if (reinterpret_cast<uintptr_t>(flags) & 15) return fail(DYCL_E_INVALID, "dycl_op_compact: flags must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(orig) & 15) return fail(DYCL_E_INVALID, "dycl_op_compact: orig must be 16-byte aligned");
  const size_t need = dycl_op_compact_workspace(n);
  if (need && (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 7)))
    return fail(DYCL_E_INVALID, "dycl_op_compact: workspace missing, too small or misaligned (need " +
                                    std::to_string(need) + " bytes)");
  return guarded([&] {
    if (n <= 16384) {
      // single workgroup; it always writes both id lists
      if (!org1 || !org0) {
        if (!workspace || workspace_bytes < 8 * static_cast<size_t>(n))
          throw std::invalid_argument(
              "dycl_op_compact: for n <= 16384 pass org1 and org0, or 8*n bytes of workspace to receive them");
        int32_t* w = static_cast<int32_t*>(workspace);
        dycl::k::compact(flags, orig, static_cast<int>(n), idx1, org1 ? org1 : w, idx0, org0 ? org0 : w + n, counts,
                         s);
      } else {
        dycl::k::compact(flags, orig, static_cast<int>(n), idx1, org1, idx0, org0, counts, s);
      }
    } else {
      dycl::k::compact_large(flags, orig, static_cast<size_t>(n), idx1, org1, idx0, org0, counts, workspace, s);
    }
    if (hipGetLastError() != hipSuccess) throw dycl::HipError("dycl_op_compact: launch failed");
    return DYCL_OK;
  });
}

int dycl_op_compact_noalloc(const uint8_t* flags, const int32_t* orig, int64_t n, int32_t* idx1, int32_t* org1,
                            int32_t* idx0, int32_t* org0, int32_t* counts, void* hip_stream) {
  if (n < 0 || static_cast<uint64_t>(n) > dycl::k::kScratchCompactMaxN)
    return fail(DYCL_E_INVALID, "dycl_op_compact_noalloc: n outside [0, " +
                                    std::to_string(dycl::k::kScratchCompactMaxN) + "] (the static scratch's limit)");
  if (!counts) return fail(DYCL_E_INVALID, "dycl_op_compact_noalloc: null counts");
  if (n > 0 && (!flags || !idx1 || !idx0))
    return fail(DYCL_E_INVALID, "dycl_op_compact_noalloc: null flags or index output");
  if (reinterpret_cast<uintptr_t>(flags) & 15)
    return fail(DYCL_E_INVALID, "dycl_op_compact_noalloc: flags must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(orig) & 15)
    return fail(DYCL_E_INVALID, "dycl_op_compact_noalloc: orig must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  return guarded([&] {
    // resolved once per device, with the device current; never the symbol itself
    uint8_t* ws = static_cast<uint8_t*>(dycl::k::compact_scratch());
    if (!ws) throw dycl::HipError("dycl_op_compact_noalloc: the static scratch's device address is unavailable");
    if (n == 0) {
      dycl::k::final_counts(nullptr, 0, counts, s);   // counts = {0, 0}, written by a kernel
    } else if (n <= 16384) {
      // single workgroup, no block offsets; ids the caller does not want land in the scratch
      int32_t* w = reinterpret_cast<int32_t*>(ws);
      dycl::k::compact(flags, orig, static_cast<int>(n), idx1, org1 ? org1 : w, idx0, org0 ? org0 : w + n, counts, s);
    } else {
      // block status words in the scratch, cleared by the
      // call's first kernel (not by a memset, so the call can be captured)
      dycl::k::compact_large(flags, orig, static_cast<size_t>(n), idx1, org1, idx0, org0, counts, ws, s);
    }
    if (hipGetLastError() != hipSuccess) throw dycl::HipError("dycl_op_compact_noalloc: launch failed");
    return DYCL_OK;
  });
}

int dycl_op_move_rows(void* dst, const int32_t* dst_idx, const void* src, const int32_t* src_idx, size_t row_bytes,
                      int64_t n, void* hip_stream) {
  if (n < 0 || n >= (int64_t(1) << 31)) return fail(DYCL_E_INVALID, "dycl_op_move_rows: n outside [0, 2^31)");
  if (n == 0) return DYCL_OK;
  if (!dst || !src) return fail(DYCL_E_INVALID, "dycl_op_move_rows: null dst or src");
  if (row_bytes == 0 || row_bytes % 16 || (reinterpret_cast<uintptr_t>(dst) & 15) ||
      (reinterpret_cast<uintptr_t>(src) & 15))
    return fail(DYCL_E_INVALID, "dycl_op_move_rows: row_bytes must be a positive multiple of 16, buffers 16-byte aligned");
  if (row_bytes / 16 > (size_t(65535) * 1024))
    return fail(DYCL_E_INVALID, "dycl_op_move_rows: rows longer than 1 GiB are not supported");
  return guarded([&] {
    dycl::k::move_rows(dst, dst_idx, src, src_idx, row_bytes, static_cast<int>(n), static_cast<hipStream_t>(hip_stream));
    if (hipGetLastError() != hipSuccess) throw dycl::HipError("dycl_op_move_rows: launch failed");
    return DYCL_OK;
  });
}

size_t dycl_op_conv_packed_bytes(int cout, int k, int cin) {
  if (cout < 1 || cin < 1 || (k != 1 && k != 3 && k != 7) || cout > (1 << 20) || cin > (1 << 20)) return 0;
  const size_t K = static_cast<size_t>(k) * k * cin;
  const size_t Kp = (K + dycl::k::kBK - 1) / dycl::k::kBK * dycl::k::kBK;
  return static_cast<size_t>(dycl::k::conv_cout_pad(cout)) * Kp * 2;
}

int dycl_op_conv_pack(const uint16_t* w, int cout, int k, int cin, uint16_t* packed, size_t packed_bytes) {
  const size_t need = dycl_op_conv_packed_bytes(cout, k, cin);
  if (!need) return fail(DYCL_E_INVALID, "dycl_op_conv_pack: need cout, cin >= 1 and k in {1, 3, 7}");
  if (!w || !packed) return fail(DYCL_E_INVALID, "dycl_op_conv_pack: null weights or output");
  if (packed_bytes < need)
    return fail(DYCL_E_INVALID, "dycl_op_conv_pack: output too small (need " + std::to_string(need) + " bytes)");
  const size_t K = static_cast<size_t>(k) * k * cin;
  const size_t Kp = need / 2 / dycl::k::conv_cout_pad(cout);
  std::memset(packed, 0, need);
  for (int co = 0; co < cout; ++co) std::memcpy(packed + co * Kp, w + co * K, K * 2);
  return DYCL_OK;
}

size_t dycl_op_conv_workspace_bytes(int n, int H, int W, int cin, int cout, int k, int stride, int pad) {
  if (n < 1 || H < 1 || W < 1 || stride < 1 || pad < 0 || !dycl_op_conv_packed_bytes(cout, k, cin)) return 0;
  if (H + 2 * pad < k || W + 2 * pad < k) return 0;
  const int Ho = (H + 2 * pad - k) / stride + 1, Wo = (W + 2 * pad - k) / stride + 1;
  return dycl::k::conv_ksplit_bytes(n, Ho, Wo, cout, k * k * cin, false);
}

int dycl_op_conv(const uint16_t* x, int n, int H, int W, int cin, const uint16_t* packed, int cout, int k, int stride,
                 int pad, const float* scale, const float* shift, const uint16_t* res, int act, uint16_t* y,
                 void* workspace, size_t workspace_bytes, void* hip_stream) {
  if (n < 0) return fail(DYCL_E_INVALID, "dycl_op_conv: n < 0");
  if (!dycl_op_conv_packed_bytes(cout, k, cin))
    return fail(DYCL_E_INVALID, "dycl_op_conv: need cout, cin >= 1 and k in {1, 3, 7}");
  if (H < 1 || W < 1 || stride < 1 || pad < 0 || pad >= k || act < 0 || act > 2)
    return fail(DYCL_E_INVALID, "dycl_op_conv: need H, W, stride >= 1, 0 <= pad < k, act in {0, 1, 2}");
  const long Ho = (static_cast<long>(H) + 2 * pad - k) / stride + 1, Wo = (static_cast<long>(W) + 2 * pad - k) / stride + 1;
  if (H + 2 * pad < k || W + 2 * pad < k) return fail(DYCL_E_INVALID, "dycl_op_conv: kernel larger than the padded input");
  const long lim = 1L << 31;
  if (static_cast<long>(n) * H * W * cin >= lim || static_cast<long>(n) * Ho * Wo * cout >= lim)
    return fail(DYCL_E_INVALID, "dycl_op_conv: a tensor reaches 2^31 elements");
  if (n == 0) return DYCL_OK;
  if (!x || !packed || !y) return fail(DYCL_E_INVALID, "dycl_op_conv: null x, packed weights or y");
  if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(packed) | reinterpret_cast<uintptr_t>(y) |
       reinterpret_cast<uintptr_t>(res) | reinterpret_cast<uintptr_t>(workspace)) & 15)
    return fail(DYCL_E_INVALID, "dycl_op_conv: x, packed, y, res and workspace must be 16-byte aligned");
  return guarded([&] {
    const uint16_t* zeros = dycl::k::zero_page();
    if (!zeros) throw dycl::HipError("dycl_op_conv: zero page unavailable");
    dycl::k::ConvArgs a;
    a.src = x;
    a.src2 = nullptr;
    a.cin1 = cin;
    a.cin2 = 0;
    a.n = n;
    a.H = H;
    a.W = W;
    a.cin = cin;
    a.Ho = static_cast<int>(Ho);
    a.Wo = static_cast<int>(Wo);
    a.cout = cout;
    a.k = k;
    a.stride = stride;
    a.pad = pad;
    a.w = packed;
    a.Kp = static_cast<int>(dycl_op_conv_packed_bytes(cout, k, cin) / 2 / dycl::k::conv_cout_pad(cout));
    a.scale = scale;
    a.shift = shift;
    a.res = res;
    a.act = act;
    a.dst = y;
    a.out_f32 = 0;
    a.zeros = zeros;
    a.splitws = static_cast<float*>(workspace);
    a.splitws_bytes = workspace ? workspace_bytes : 0;
    dycl::k::conv_bf16(a, static_cast<hipStream_t>(hip_stream));
    if (hipGetLastError() != hipSuccess) throw dycl::HipError("dycl_op_conv: launch failed");
    return DYCL_OK;
  });
}

int dycl_op_conv_maxpool(const uint16_t* x, int n, int H, int W, int cin, const uint16_t* packed, int cout, int k,
                         int stride, int pad, const float* scale, const float* shift, int act, uint16_t* y,
                         void* hip_stream) {
  if (n < 0) return fail(DYCL_E_INVALID, "dycl_op_conv_maxpool: n < 0");
  if (act != 1 || H < 1 || W < 1 || !dycl::k::conv_rgb_stem_fits(H, W, cin, cout, k, stride, pad))
    return fail(DYCL_E_INVALID,
                "dycl_op_conv_maxpool: needs cin 3, cout 64, k 7, stride 2, pad <= 3, W % 8 == 0, Wo <= 112, ReLU");
  const long Ho = (static_cast<long>(H) + 2 * pad - k) / stride + 1, Wo = (static_cast<long>(W) + 2 * pad - k) / stride + 1;
  const long lim = 1L << 31;
  if (static_cast<long>(n) * H * W * cin >= lim || static_cast<long>(n) * Ho * Wo * cout >= lim)
    return fail(DYCL_E_INVALID, "dycl_op_conv_maxpool: a tensor reaches 2^31 elements");
  if (n == 0) return DYCL_OK;
  if (!x || !packed || !y) return fail(DYCL_E_INVALID, "dycl_op_conv_maxpool: null x, packed weights or y");
  if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(packed) | reinterpret_cast<uintptr_t>(y)) & 15)
    return fail(DYCL_E_INVALID, "dycl_op_conv_maxpool: x, packed and y must be 16-byte aligned");
  return guarded([&] {
    dycl::k::ConvArgs a;
    a.src = x;
    a.src2 = nullptr;
    a.cin1 = cin;
    a.cin2 = 0;
    a.n = n;
    a.H = H;
    a.W = W;
    a.cin = cin;
    a.Ho = static_cast<int>(Ho);
    a.Wo = static_cast<int>(Wo);
    a.cout = cout;
    a.k = k;
    a.stride = stride;
    a.pad = pad;
    a.w = packed;
    a.Kp = static_cast<int>(dycl_op_conv_packed_bytes(cout, k, cin) / 2 / dycl::k::conv_cout_pad(cout));
    a.scale = scale;
    a.shift = shift;
    a.res = nullptr;
    a.act = act;
    a.dst = y;
    a.out_f32 = 0;
    a.zeros = nullptr;
    a.pool = 1;
    if (!dycl::k::conv_rgb_stem(a, static_cast<hipStream_t>(hip_stream)))
      throw dycl::HipError("dycl_op_conv_maxpool: the fused kernel declined the arguments");
    if (hipGetLastError() != hipSuccess) throw dycl::HipError("dycl_op_conv_maxpool: launch failed");
    return DYCL_OK;
  });
}

}  // extern "C"

int dycl_op_conv_pair(const uint16_t* x, int n, int H, int W, int cin, const uint16_t* packed3, const float* scale3,
                      const float* shift3, const uint16_t* res, int c3, uint16_t* y3, const uint16_t* packed1,
                      const float* scale1, const float* shift1, int c1, uint16_t* y1, void* hip_stream) {
  if (n < 0) return fail(DYCL_E_INVALID, "dycl_op_conv_pair: n < 0");
  if (H < 1 || W < 1 || !dycl::k::conv_pair_fits(cin, 0, c3, c1, dycl::k::ACT_RELU, dycl::k::ACT_RELU))
    return fail(DYCL_E_INVALID,
                "dycl_op_conv_pair: needs H, W >= 1 and c3 256, c1 64, cin % 64 == 0 in [64, 1024] or c3 512, c1 128, "
                "cin 128");
  const long lim = 1L << 31;
  if (static_cast<long>(n) * H * W * std::max(cin, c3) >= lim)
    return fail(DYCL_E_INVALID, "dycl_op_conv_pair: a tensor reaches 2^31 elements");
  if (n == 0) return DYCL_OK;
  if (!x || !packed3 || !y3 || !packed1 || !y1 || !scale3 || !shift3 || !scale1 || !shift1)
    return fail(DYCL_E_INVALID, "dycl_op_conv_pair: null tensor, weights or scale / shift vector");
  const void* ptrs[] = {x, packed3, scale3, shift3, res, y3, packed1, scale1, shift1, y1};
  for (const void* q : ptrs)
    if (reinterpret_cast<uintptr_t>(q) & 15)
      return fail(DYCL_E_INVALID, "dycl_op_conv_pair: every pointer must be 16-byte aligned");
  return guarded([&] {
    const uint16_t* zeros = dycl::k::zero_page();
    if (!zeros) throw dycl::HipError("dycl_op_conv_pair: zero page unavailable");
    dycl::k::PairArgs a;
    a.x = x;
    a.K3 = cin;
    a.w3 = packed3;
    a.Kp3 = static_cast<int>(dycl_op_conv_packed_bytes(c3, 1, cin) / 2 / dycl::k::conv_cout_pad(c3));
    a.scale3 = scale3;
    a.shift3 = shift3;
    a.res = res;
    a.y3 = y3;
    a.C3 = c3;
    a.w1 = packed1;
    a.Kp1 = static_cast<int>(dycl_op_conv_packed_bytes(c1, 1, c3) / 2 / dycl::k::conv_cout_pad(c1));
    a.scale1 = scale1;
    a.shift1 = shift1;
    a.y1 = y1;
    a.C1 = c1;
    a.act3 = dycl::k::ACT_RELU;
    a.act1 = dycl::k::ACT_RELU;
    a.n = n;
    a.H = H;
    a.W = W;
    a.zeros = zeros;
    if (!dycl::k::conv_pair(a, static_cast<hipStream_t>(hip_stream)))
      throw dycl::HipError("dycl_op_conv_pair: the fused kernel declined the arguments");
    if (hipGetLastError() != hipSuccess) throw dycl::HipError("dycl_op_conv_pair: launch failed");
    return DYCL_OK;
  });
}
