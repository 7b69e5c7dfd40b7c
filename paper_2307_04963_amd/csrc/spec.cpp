// Specification parsing, validation and shape propagation (host only; no
// HIP call happens here, so every check runs without a GPU).
#include <cmath>
#include <cstring>
#include <algorithm>
#include <map>
#include <sstream>

#include "plan.hpp"

namespace dycl {

namespace {

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

struct Builder {
  Spec& sp;
  size_t blob;
  std::map<std::string, int> names;
  int space = 0;
  int next_space = 1;
  bool in_body = false;

  Builder(Spec& s, size_t b) : sp(s), blob(b) {}

  [[noreturn]] void fail(const std::string& m) { throw SpecError(m); }

  void need_bytes(int64_t off, int64_t bytes, int64_t align, const char* what) {
    if (off < 0) fail(std::string(what) + ": negative offset");
    if (off % align != 0) fail(std::string(what) + ": offset not aligned to " + std::to_string(align));
    if (bytes < 0 || static_cast<uint64_t>(off) + static_cast<uint64_t>(bytes) > blob)
      throw WeightsError(std::string(what) + ": weight range [" + std::to_string(off) + ", +" +
                         std::to_string(bytes) + ") exceeds the blob of " + std::to_string(blob) + " bytes");
  }

  int lookup(const Json& j, const char* what) {
    const std::string& n = j.as_str(what);
    auto it = names.find(n);
    if (it == names.end()) fail(std::string(what) + ": unknown tensor '" + n + "'");
    return it->second;
  }

  int use(const Json& j, const char* what, int seq) {
    int t = lookup(j, what);
    TensorInfo& ti = sp.tensors[t];
    if (!ti.parked && ti.space != space)
      fail(std::string(what) + ": tensor '" + ti.name +
           "' belongs to rows that were regrouped by a decision; carry it through that decision");
    touch(t, seq);
    return t;
  }

  void touch(int t, int seq) {
    TensorInfo& ti = sp.tensors[t];
    if (ti.first < 0 || seq < ti.first) ti.first = seq;
    ti.last = std::max(ti.last, seq);
  }

  int define(const Json& j, int H, int W, int C, int seq, const char* what) {
    const std::string& n = j.as_str(what);
    if (names.count(n)) fail(std::string(what) + ": tensor '" + n + "' is defined twice");
    if (H < 1 || W < 1 || C < 1) fail(std::string(what) + ": empty shape for '" + n + "'");
    TensorInfo ti;
    ti.name = n;
    ti.H = H;
    ti.W = W;
    ti.C = C;
    ti.space = space;
    sp.tensors.push_back(ti);
    int id = static_cast<int>(sp.tensors.size()) - 1;
    names[n] = id;
    touch(id, seq);
    return id;
  }

  int act_of(const std::string& a) {
    if (a == "none") return k::ACT_NONE;
    if (a == "relu") return k::ACT_RELU;
    if (a == "gelu") return k::ACT_GELU;
    if (a == "tanh") return k::ACT_TANH;
    if (a == "lstm") return k::ACT_LSTM;
    fail("unknown activation '" + a + "'");
  }

  int64_t f32_vec(const Json& n, const char* key, int64_t count) {
    if (!n.has(key) || n.at(key).is_null()) return -1;
    int64_t off = n.at(key).as_int(key);
    need_bytes(off, count * 4, 4, key);
    return off;
  }

  int pack_index(int64_t off, int64_t ldk, int64_t k0, int cout, int K, int taps = 1, int cin_src = 0,
                 int cin_pack = 0, bool interleave4 = false) {
    if (cin_src == 0) cin_src = cin_pack = K;   // one run of K values
    for (size_t i = 0; i < sp.packed.size(); ++i) {
      const Packed& q = sp.packed[i];
      if (q.w_off == off && q.w_ldk == ldk && q.w_k0 == k0 && q.cout == cout && q.K == taps * cin_pack &&
          q.cin_src == cin_src && q.cin_pack == cin_pack && q.interleave4 == interleave4)
        return static_cast<int>(i);
    }
    Packed q;
    q.w_off = off;
    q.w_ldk = ldk;
    q.w_k0 = k0;
    q.cout = cout;
    q.K = taps * cin_pack;
    q.taps = taps;
    q.cin_src = cin_src;
    q.cin_pack = cin_pack;
    q.cout_pad = k::conv_cout_pad(cout);
    q.Kp = (q.K + k::kBK - 1) / k::kBK * k::kBK;
    q.interleave4 = interleave4;
    sp.packed.push_back(q);
    return static_cast<int>(sp.packed.size()) - 1;
  }

  // An LSTM step: h' and the float32 cell state c' from h, c and the
  // embedding of each row's previous token (Table 1's En-Decoder cell).
  Node lstm_conv(const Json& n) {
    Node nd;
    nd.kind = NodeKind::Conv;
    nd.seq_pre = nd.seq_post = sp.seq++;
    if (sp.dt != DType::BF16 || !sp.any_decode) fail("an lstm step needs a bf16 spec with a decode section");
    if (in_body) fail("an lstm step inside a gate body is not supported");
    nd.src = use(n.at("src"), "lstm.src", nd.seq_pre);
    const TensorInfo src = sp.tensors[nd.src];
    if (src.H != 1 || src.W != 1 || src.f32) fail("lstm.src must be a bf16 1x1 row");
    nd.cin1 = src.C;
    nd.cout = static_cast<int>(n.at("cout").as_int("cout"));
    if (nd.cout != 4 * src.C || src.C % 8) fail("lstm.cout must be 4 x the hidden size, a multiple of 8");
    const Json& e = n.at("emb");
    nd.emb_off = e.at("off").as_int("emb.off");
    nd.emb_rows = static_cast<int>(e.at("rows").as_int("emb.rows"));
    nd.cin2 = static_cast<int>(e.at("dim").as_int("emb.dim"));
    if (nd.emb_rows < 1 || nd.cin2 < 8 || nd.cin2 % 8) fail("lstm.emb: rows >= 1, dim a multiple of 8");
    if (nd.emb_rows < sp.n_out) fail("lstm.emb: every token of the vocabulary needs a row");
    need_bytes(nd.emb_off, static_cast<int64_t>(nd.emb_rows) * nd.cin2 * 2, 16, "lstm.emb");
    nd.act = k::ACT_LSTM;
    nd.H = nd.W = nd.Ho = nd.Wo = 1;
    const int K = nd.cin1 + nd.cin2;
    const Json& w = n.at("w");
    nd.w_off = w.at("off").as_int("w.off");
    nd.w_ldk = w.get_int("ldk", K);
    nd.w_k0 = w.get_int("k0", 0);
    if (nd.w_k0 < 0 || nd.w_k0 + K > nd.w_ldk) fail("lstm.w: column range [k0, k0+K) exceeds ldk");
    need_bytes(nd.w_off, ((int64_t)(nd.cout - 1) * nd.w_ldk + nd.w_k0 + K) * 2, 2, "lstm.w");
    nd.shift_off = f32_vec(n, "shift", nd.cout);
    nd.lstm_shift = sp.n_lstm_shift++;
    nd.packed = pack_index(nd.w_off, nd.w_ldk, nd.w_k0, nd.cout, K, 1, 0, 0, true);
    if (n.has("cell_in") && !n.at("cell_in").is_null()) {
      nd.cell_in = use(n.at("cell_in"), "lstm.cell_in", nd.seq_pre);
      const TensorInfo& ci = sp.tensors[nd.cell_in];
      if (!ci.f32 || ci.C != src.C) fail("lstm.cell_in must be a float32 cell state of the hidden size");
    }
    nd.dst = define(n.at("dst"), 1, 1, src.C, nd.seq_pre, "lstm.dst");
    nd.cell_out = define(n.at("cell_out"), 1, 1, src.C, nd.seq_pre, "lstm.cell_out");
    sp.tensors[nd.cell_out].f32 = true;
    return nd;
  }

  // Greedy token choice (a logic node): the output layer's float32 logits,
  // argmax, and the end-token / length test that partitions the rows.
  Node decode_node(const Json& n) {
    Node nd;
    nd.kind = NodeKind::Decode;
    nd.seq_pre = nd.seq_post = sp.seq++;
    if (in_body) fail("decode inside a gate body is not supported");
    if (sp.dt != DType::BF16 || !sp.any_decode) fail("decode needs a bf16 spec with a decode section");
    nd.src = use(n.at("src"), "decode.src", nd.seq_pre);
    const TensorInfo s = sp.tensors[nd.src];
    if (s.H != 1 || s.W != 1 || s.f32 || s.C % 8) fail("decode.src must be a bf16 1x1 row of channels divisible by 8");
    nd.cin1 = s.C;
    nd.cout = nd.ncls = sp.n_out;
    if (nd.ncls % 4) fail("decode: the vocabulary (n_out) must be a multiple of 4");
    const Json& w = n.at("w");
    nd.w_off = w.at("off").as_int("w.off");
    nd.w_ldk = w.get_int("ldk", s.C);
    nd.w_k0 = w.get_int("k0", 0);
    if (nd.w_k0 < 0 || nd.w_k0 + s.C > nd.w_ldk) fail("decode.w: column range exceeds ldk");
    need_bytes(nd.w_off, ((int64_t)(nd.cout - 1) * nd.w_ldk + nd.w_k0 + s.C) * 2, 2, "decode.w");
    nd.shift_off = f32_vec(n, "b", nd.cout);
    nd.packed = pack_index(nd.w_off, nd.w_ldk, nd.w_k0, nd.cout, s.C);
    nd.eos = static_cast<int>(n.at("eos").as_int("eos"));
    if (nd.eos < 0 || nd.eos >= sp.n_out) fail("decode.eos must be a token of the vocabulary");
    nd.index = static_cast<int>(n.at("step").as_int("step"));
    nd.max_steps = sp.max_len;
    if (nd.index < 1 || nd.index > sp.max_len) fail("decode.step must be in [1, max_len]");
    nd.final_ = nd.index == sp.max_len;
    nd.decision = sp.decisions++;
    sp.max_ncls = std::max(sp.max_ncls, nd.ncls);
    if (!nd.final_) {
      int old = space;
      space = next_space++;
      carry(n, "carry", nd, old);
      space = next_space - 1;
    } else {
      if (n.has("carry") && n.at("carry").size()) fail("the last decoding step carries nothing");
      space = next_space++;   // no rows remain
    }
    return nd;
  }

  Node conv(const Json& n, int max_batch) {
    if (n.get_str("act", "none") == "lstm") return lstm_conv(n);
    Node nd;
    nd.kind = NodeKind::Conv;
    nd.seq_pre = nd.seq_post = sp.seq++;
    nd.src = use(n.at("src"), "conv.src", nd.seq_pre);
    const TensorInfo src = sp.tensors[nd.src];
    nd.H = src.H;
    nd.W = src.W;
    nd.cin1 = src.C;
    if (n.has("src2") && !n.at("src2").is_null()) {
      nd.src2 = use(n.at("src2"), "conv.src2", nd.seq_pre);
      const TensorInfo& s2 = sp.tensors[nd.src2];
      if (s2.H != src.H || s2.W != src.W) fail("conv.src2: spatial shape differs from src");
      nd.cin2 = s2.C;
    }
    nd.k = static_cast<int>(n.get_int("k", 1));
    nd.stride = static_cast<int>(n.get_int("stride", 1));
    nd.pad = static_cast<int>(n.get_int("pad", 0));
    nd.cout = static_cast<int>(n.at("cout").as_int("cout"));
    if (nd.k != 1 && nd.k != 3 && nd.k != 7) fail("conv.k must be 1, 3 or 7");
    if (nd.stride < 1 || nd.stride > 4 || nd.pad < 0 || nd.pad >= nd.k + 1) fail("conv: bad stride / pad");
    if (nd.cout < 1 || nd.cout > 65536) fail("conv.cout out of range");
    if (nd.src2 >= 0 && (nd.k != 1 || nd.cin1 % 8 || nd.cin2 % 8))
      fail("conv.src2 (channel concat) needs k == 1 and channel counts divisible by 8");
    nd.Ho = (nd.H + 2 * nd.pad - nd.k) / nd.stride + 1;
    nd.Wo = (nd.W + 2 * nd.pad - nd.k) / nd.stride + 1;
    if (nd.Ho < 1 || nd.Wo < 1) fail("conv: output would be empty");
    nd.act = act_of(n.get_str("act", "none"));
    const int cin = nd.cin1 + nd.cin2;
    const int K = nd.k * nd.k * cin;
    const Json& w = n.at("w");
    nd.w_off = w.at("off").as_int("w.off");
    nd.w_ldk = w.get_int("ldk", K);
    nd.w_k0 = w.get_int("k0", 0);
    if (nd.w_k0 < 0 || nd.w_k0 + K > nd.w_ldk) fail("conv.w: column range [k0, k0+K) exceeds ldk");
    const int esz = sp.dt == DType::BF16 ? 2 : 4;
    need_bytes(nd.w_off, ((int64_t)(nd.cout - 1) * nd.w_ldk + nd.w_k0 + K) * esz, esz, "conv.w");
    nd.scale_off = f32_vec(n, "scale", nd.cout);
    nd.shift_off = f32_vec(n, "shift", nd.cout);
    if (n.has("res") && !n.at("res").is_null()) {
      nd.res = use(n.at("res"), "conv.res", nd.seq_pre);
      const TensorInfo& r = sp.tensors[nd.res];
      if (r.H != nd.Ho || r.W != nd.Wo || r.C != nd.cout) fail("conv.res: shape differs from the output");
    }
    if (nd.act == k::ACT_TANH && (nd.k != 1 || nd.H != 1 || nd.W != 1 || nd.res >= 0 || nd.cout % 8 ||
                                  sp.dt != DType::BF16))
      fail("tanh is taken by bf16 linear layers on 1x1 rows (cout a multiple of 8, no residual)");
    if (sp.tensors[nd.src].f32 || (nd.src2 >= 0 && sp.tensors[nd.src2].f32))
      fail("conv: a float32 cell state is read only by an lstm step");
    if (sp.dt == DType::F32) {
      if (nd.k != 1 || nd.H != 1 || nd.W != 1 || nd.src2 >= 0 || nd.res >= 0 || nd.scale_off >= 0 ||
          nd.act == k::ACT_GELU || nd.act == k::ACT_TANH)
        fail("fp32 specs support only linear layers (k 1 on 1x1 rows, bias, ReLU)");
      if (nd.w_k0 != 0 || nd.w_ldk != K) fail("fp32 linear weights must be dense [cout][cin]");
      nd.head_t = sp.n_head_t++;   // kept transposed on the device
    } else if (sp.tensors[nd.src].external && nd.src2 < 0 && nd.cin1 < 8 &&
               (nd.res >= 0 || !k::conv_rgb_stem_fits(nd.H, nd.W, nd.cin1, nd.cout, nd.k, nd.stride, nd.pad))) {
      // a stem on a narrow input: the input is zero-padded to 8 channels once
      // per run and the weights likewise, so the stem runs on 16-byte
      // vectors (the padded products are exact zeros)
      nd.pad_in = true;
      sp.pad_input_c = 8;
      nd.packed = pack_index(nd.w_off, nd.w_ldk, nd.w_k0, nd.cout, K, nd.k * nd.k, nd.cin1, 8);
    } else {
      nd.packed = pack_index(nd.w_off, nd.w_ldk, nd.w_k0, nd.cout, K);
    }
    nd.dst = define(n.at("dst"), nd.Ho, nd.Wo, nd.cout, nd.seq_pre, "conv.dst");
    return nd;
  }

  Node maxpool(const Json& n) {
    Node nd;
    nd.kind = NodeKind::MaxPool;
    nd.seq_pre = nd.seq_post = sp.seq++;
    if (sp.dt != DType::BF16) fail("maxpool needs a bf16 spec");
    nd.src = use(n.at("src"), "maxpool.src", nd.seq_pre);
    const TensorInfo s = sp.tensors[nd.src];
    if (s.C % 8) fail("maxpool: channels must be a multiple of 8");
    nd.H = s.H;
    nd.W = s.W;
    nd.Ho = (s.H + 2 - 3) / 2 + 1;
    nd.Wo = (s.W + 2 - 3) / 2 + 1;
    nd.dst = define(n.at("dst"), nd.Ho, nd.Wo, s.C, nd.seq_pre, "maxpool.dst");
    return nd;
  }

  void head_channels(const TensorInfo& s, const char* what) {
    if (sp.dt == DType::BF16) {
      if (!is_pow2(s.C) || s.C < 8 || s.C > 2048)
        fail(std::string(what) + ": pooled channels must be a power of two in [8, 2048]");
    } else if (s.H * s.W != 1) {
      fail(std::string(what) + ": fp32 heads read 1x1 rows");
    }
  }

  void carry(const Json& n, const char* key, Node& nd, int old_space) {
    if (!n.has(key)) return;
    const Json& c = n.at(key);
    for (size_t i = 0; i < c.size(); ++i) {
      const Json& pr = c.at(i);
      if (pr.size() != 2) fail(std::string(key) + ": entries are [old, new] pairs");
      space = old_space;
      int o = use(pr.at(0), key, nd.seq_pre);
      space = next_space - 1;   // the new row space of the surviving rows
      const TensorInfo ot = sp.tensors[o];
      int nw = define(pr.at(1), ot.H, ot.W, ot.C, nd.seq_pre, key);
      sp.tensors[nw].f32 = ot.f32;
      nd.pairs.push_back({o, nw});
    }
  }

  Node exit_node(const Json& n) {
    Node nd;
    nd.kind = NodeKind::Exit;
    nd.seq_pre = nd.seq_post = sp.seq++;
    if (in_body) fail("exit inside a gate body is not supported");
    nd.src = use(n.at("src"), "exit.src", nd.seq_pre);
    const TensorInfo s = sp.tensors[nd.src];
    head_channels(s, "exit");
    nd.H = s.H;
    nd.W = s.W;
    nd.hc = s.C;
    nd.ncls = static_cast<int>(n.at("ncls").as_int("ncls"));
    if (nd.ncls != sp.n_out) fail("exit.ncls must equal n_out");
    nd.h_w = f32_vec(n, "w", (int64_t)nd.ncls * s.C);
    nd.h_b = f32_vec(n, "b", nd.ncls);
    nd.h_T = f32_vec(n, "T", 1);
    nd.final_ = n.get_bool("final", false);
    if (nd.h_w < 0 || nd.h_b < 0) fail("exit: w and b are required");
    if (!nd.final_ && nd.h_T < 0) fail("exit: a non-final exit needs its temperature T");
    nd.tau = static_cast<float>(n.get_num("tau", 0.0));
    nd.index = static_cast<int>(n.get_int("index", 0));   // -1: a classifier that records no exit
    if (nd.index < -1) fail("exit.index must be >= -1");
    nd.decision = sp.decisions++;
    sp.max_head_c = std::max(sp.max_head_c, s.C);
    sp.max_ncls = std::max(sp.max_ncls, nd.ncls);
    // small heads run as one fused kernel (pooling, linear on the weights
    // as stored [ncls][C], decision); the others pool, then multiply by a
    // transposed copy of the weights
    nd.head_t = sp.n_head_t++;
    nd.fused = nd.ncls <= 1024 && s.C <= 2048 && s.C % 4 == 0 &&
               static_cast<int64_t>(s.C) * nd.ncls <= (int64_t(1) << 16);
    if (!nd.final_) {
      int old = space;
      space = next_space++;
      carry(n, "carry", nd, old);
      space = next_space - 1;
    } else {
      if (n.has("carry") && n.at("carry").size()) fail("a final exit carries nothing");
      space = next_space++;   // no rows remain
    }
    return nd;
  }

  Node gate_node(const Json& n, int max_batch) {
    Node nd;
    nd.kind = NodeKind::Gate;
    nd.seq_pre = sp.seq++;
    if (in_body) fail("nested gates are not supported");
    if (sp.dt != DType::BF16) fail("gates need a bf16 spec");
    nd.src = use(n.at("src"), "gate.src", nd.seq_pre);
    const TensorInfo s = sp.tensors[nd.src];
    head_channels(s, "gate");
    nd.H = s.H;
    nd.W = s.W;
    nd.hc = s.C;
    nd.h_w = f32_vec(n, "u", s.C);
    nd.h_b = f32_vec(n, "v", 1);
    if (nd.h_w < 0 || nd.h_b < 0) fail("gate: u and v are required");
    nd.tau = static_cast<float>(n.get_num("threshold", 0.5));
    nd.index = static_cast<int>(n.at("index").as_int("index"));
    if (nd.index < 0 || nd.index > 63) fail("gate.index must be in [0, 63]");
    nd.decision = sp.decisions++;
    const int outer = space;
    const int inner = next_space++;
    const Json& g = n.at("gather");
    for (size_t i = 0; i < g.size(); ++i) {
      const Json& pr = g.at(i);
      if (pr.size() != 2) fail("gate.gather entries are [outer, inner] pairs");
      space = outer;
      int o = use(pr.at(0), "gate.gather", nd.seq_pre);
      space = inner;
      const TensorInfo ot = sp.tensors[o];
      nd.pairs.push_back({o, define(pr.at(1), ot.H, ot.W, ot.C, nd.seq_pre, "gate.gather")});
    }
    space = inner;
    in_body = true;
    const Json& body = n.at("body");
    for (size_t i = 0; i < body.size(); ++i) nd.body.push_back(node(body.at(i), max_batch));
    in_body = false;
    nd.seq_post = sp.seq++;
    const Json& sc = n.at("scatter");
    for (size_t i = 0; i < sc.size(); ++i) {
      const Json& pr = sc.at(i);
      if (pr.size() != 2) fail("gate.scatter entries are [inner, outer] pairs");
      space = inner;
      int in = use(pr.at(0), "gate.scatter", nd.seq_post);
      space = outer;
      int out = use(pr.at(1), "gate.scatter", nd.seq_post);
      const TensorInfo &a = sp.tensors[in], &b = sp.tensors[out];
      if (a.H != b.H || a.W != b.W || a.C != b.C) fail("gate.scatter: shapes differ");
      if (b.external) fail("gate.scatter: cannot write the caller's input");
      nd.scatter.push_back({in, out});
    }
    space = outer;
    return nd;
  }

  Node halt_node(const Json& n) {
    Node nd;
    nd.kind = NodeKind::Halt;
    nd.seq_pre = nd.seq_post = sp.seq++;
    if (in_body) fail("halt inside a gate body is not supported");
    if (sp.dt != DType::BF16 || !sp.aux) fail("halt needs a bf16 spec with per-sample aux inputs");
    nd.src = use(n.at("src"), "halt.src", nd.seq_pre);
    const TensorInfo s = sp.tensors[nd.src];
    if (s.H != 1 || s.W != 1 || s.C % 8) fail("halt.src must be a 1x1 row with channels divisible by 8");
    nd.hc = s.C;
    nd.h_w = f32_vec(n, "w", s.C);
    if (nd.h_w < 0) fail("halt.w is required");
    nd.tau = static_cast<float>(n.at("tau").as_num("tau"));
    nd.index = static_cast<int>(n.at("step").as_int("step"));
    nd.max_steps = static_cast<int>(n.at("max_steps").as_int("max_steps"));
    if (nd.index < 1 || nd.index > nd.max_steps) fail("halt.step must be in [1, max_steps]");
    nd.decision = sp.decisions++;
    sp.any_halt = true;
    const Json& pk = n.at("park");
    if (pk.size() != 2) fail("halt.park is [src, parked]");
    nd.park_src = use(pk.at(0), "halt.park", nd.seq_pre);
    const std::string& pn = pk.at(1).as_str("halt.park");
    if (names.count(pn)) {
      nd.park_dst = names[pn];
      const TensorInfo& pt = sp.tensors[nd.park_dst];
      if (!pt.parked || pt.C != s.C) fail("halt.park: '" + pn + "' is not a parked tensor of this shape");
      touch(nd.park_dst, nd.seq_pre);
    } else {
      nd.park_dst = define(pk.at(1), 1, 1, s.C, nd.seq_pre, "halt.park");
      sp.tensors[nd.park_dst].parked = true;
    }
    int old = space;
    space = next_space++;
    carry(n, "carry", nd, old);
    space = next_space - 1;
    return nd;
  }

  Node output_node(const Json& n) {
    Node nd;
    nd.kind = NodeKind::Output;
    nd.seq_pre = nd.seq_post = sp.seq++;
    if (in_body) fail("output inside a gate body is not supported");
    int t = lookup(n.at("src"), "output.src");
    if (!sp.tensors[t].parked) fail("output.src must be a parked tensor");
    touch(t, nd.seq_pre);
    nd.src = t;
    const TensorInfo s = sp.tensors[t];
    nd.cin1 = s.C;
    nd.cout = static_cast<int>(n.at("cout").as_int("cout"));
    if (nd.cout != sp.n_out) fail("output.cout must equal n_out");
    const Json& w = n.at("w");
    nd.w_off = w.at("off").as_int("w.off");
    nd.w_ldk = w.get_int("ldk", s.C);
    nd.w_k0 = w.get_int("k0", 0);
    if (nd.w_k0 < 0 || nd.w_k0 + s.C > nd.w_ldk) fail("output.w: column range exceeds ldk");
    need_bytes(nd.w_off, ((int64_t)(nd.cout - 1) * nd.w_ldk + nd.w_k0 + s.C) * 2, 2, "output.w");
    nd.shift_off = f32_vec(n, "bias", nd.cout);
    nd.packed = pack_index(nd.w_off, nd.w_ldk, nd.w_k0, nd.cout, s.C);
    return nd;
  }

  Node node(const Json& n, int max_batch) {
    const std::string& op = n.at("op").as_str("op");
    ++sp.nodes_total;
    if (op == "conv") return conv(n, max_batch);
    if (op == "maxpool") return maxpool(n);
    if (op == "exit") return exit_node(n);
    if (op == "gate") return gate_node(n, max_batch);
    if (op == "halt") return halt_node(n);
    if (op == "output") return output_node(n);
    if (op == "decode") return decode_node(n);
    fail("unknown node op '" + op + "'");
  }
};

}  // namespace

namespace {

// Every read of tensor t: the reading node, whether it is a conv's main
// input, and the node's index among the top-level nodes (-1 inside a body).
struct Use {
  Node* node;
  bool conv_src;
  long top;
};

void uses_of(std::vector<Node>& nodes, int t, long top, std::vector<Use>& out) {
  for (size_t i = 0; i < nodes.size(); ++i) {
    Node& nd = nodes[i];
    const long at = top < 0 ? static_cast<long>(i) : -1;
    bool other = nd.src2 == t || nd.res == t || nd.park_src == t || nd.cell_in == t;
    for (auto& pr : nd.pairs) other = other || pr.first == t;
    for (auto& pr : nd.scatter) other = other || pr.first == t;
    if (nd.src == t) out.push_back({&nd, nd.kind == NodeKind::Conv, at});
    if (other) out.push_back({&nd, false, at});
    uses_of(nd.body, t, 0, out);
  }
}

bool is_decision(const Node& nd) {
  return nd.kind == NodeKind::Exit || nd.kind == NodeKind::Gate || nd.kind == NodeKind::Halt ||
         nd.kind == NodeKind::Decode;
}

}  // namespace

// A stem convolution on the 3-channel input whose output only the 3x3 /
// stride-2 max-pool right after it reads: the pooling runs in the stem
// kernel's epilogue (ReLU outputs, whose maxima are exact on bf16 bits) and
// the full-resolution output is never stored.
void Spec::fuse_stem_pools() {
  if (dt != DType::BF16) return;
  for (size_t i = 0; i + 1 < nodes.size(); ++i) {
    Node& c = nodes[i];
    const Node& mp = nodes[i + 1];
    if (c.kind != NodeKind::Conv || mp.kind != NodeKind::MaxPool || mp.src != c.dst) continue;
    if (c.pad_in || c.pool || c.src2 >= 0 || c.res >= 0 || c.act != k::ACT_RELU || !tensors[c.src].external ||
        c.src_list || c.src2_list || c.res_list || c.dst_list ||
        !k::conv_rgb_stem_fits(c.H, c.W, c.cin1, c.cout, c.k, c.stride, c.pad))
      continue;
    std::vector<Use> us;
    uses_of(nodes, c.dst, -1, us);
    if (us.size() != 1) continue;   // another node reads the stem output
    tensors[c.dst].unused = true;
    c.dst = mp.dst;
    c.pool = true;
    TensorInfo& d = tensors[c.dst];
    d.first = std::min(d.first, c.seq_pre);
    nodes.erase(nodes.begin() + static_cast<long>(i) + 1);
    ++fused_pools;
  }
}

// A 1x1 projection shortcut P = scale_p * (W_p x) + shift_p (any stride s) whose
// only reader is the block's last 1x1 convolution, as its residual:
//   y = act(scale_c * (W_c h) + shift_c + P)
//     = act(scale_c * ([W_c | (scale_p / scale_c) W_p] [h; x]) + (shift_c + shift_p)),
// one contraction over the channel concatenation of h and x (src2, read at
// stride s: output pixel (i, j) takes x at (s i, s j)); the
// block's own weights stay as they are and the projection's rows carry the
// ratio of the scales (one bf16 rounding, in place of the rounding of P).
// The projection's output is never written nor read back.  Top-level nodes
// only, with no decision between the two (the rows of x and h then match).
void Spec::fuse_projections() {
  if (dt != DType::BF16) return;
  for (size_t i = 0; i < nodes.size(); ++i) {
    Node& c = nodes[i];
    // both K blocks whole 64-wide K steps, so the kernel can finish the
    // projection's sum before the block's own starts; 8-channel output vectors
    if (c.kind != NodeKind::Conv || c.k != 1 || c.stride != 1 || c.pad != 0 || c.src2 >= 0 || c.res < 0 ||
        c.pad_in || c.pool || c.cin1 % k::kBK || c.cout % 8 || c.src_list || c.res_list || c.dst_list)
      continue;
    long j = -1;
    bool between = false;   // a decision between the projection and c
    for (long t = static_cast<long>(i) - 1; t >= 0; --t) {
      if (nodes[t].kind == NodeKind::Conv && nodes[t].dst == c.res) {
        j = t;
        break;
      }
      between = between || is_decision(nodes[t]);
    }
    if (j < 0 || between) continue;
    const Node& pn = nodes[j];
    if (pn.k != 1 || pn.pad != 0 || pn.src2 >= 0 || pn.res >= 0 || pn.act != k::ACT_NONE ||
        pn.pad_in || pn.pool || pn.cout != c.cout || pn.Ho != c.H || pn.Wo != c.W || pn.cin1 % k::kBK ||
        pn.src_list || pn.dst_list || tensors[pn.dst].external)
      continue;
    // the rounded projection is carried into the block's sum divided by the
    // block's scale: every nonzero scale must have a finite, moderate inverse
    // (weights unknown here, as in a validation-only parse: assumed so)
    if (host_w && c.scale_off >= 0) {
      bool fine = true;
      for (int co = 0; co < c.cout && fine; ++co) {
        float sc;
        std::memcpy(&sc, host_w + c.scale_off + static_cast<size_t>(co) * 4, 4);
        fine = sc == 0.0f || (std::isfinite(sc) && std::fabs(sc) >= 0x1p-64f && std::fabs(sc) <= 0x1p64f);
      }
      if (!fine) continue;
    }
    std::vector<Use> us;
    uses_of(nodes, pn.dst, -1, us);
    if (us.size() != 1 || us[0].node != &c) continue;
    const Packed& q1 = packed[c.packed];
    Packed q = q1;
    q.w2_off = pn.w_off;
    q.w2_ldk = pn.w_ldk;
    q.w2_k0 = pn.w_k0;
    q.cin2 = pn.cin1;
    q.scale1_off = c.scale_off;
    q.K = c.cin1 + pn.cin1;
    q.Kp = (q.K + k::kBK - 1) / k::kBK * k::kBK;
    q.dev = nullptr;
    packed.push_back(q);
    c.packed = static_cast<int>(packed.size()) - 1;
    c.src2 = pn.src;
    c.cin2 = pn.cin1;
    c.s2 = pn.stride;
    c.res = -1;
    c.fold = true;
    c.scale2_off = pn.scale_off;
    c.shift2_off = pn.shift_off;
    c.fold_shift = n_fold_shift++;
    tensors[pn.dst].unused = true;
    TensorInfo& x = tensors[pn.src];
    x.last = std::max(x.last, c.seq_pre);
    nodes.erase(nodes.begin() + j);
    --i;
    ++fused_projections;
  }
}

// A bottleneck block's last 1x1 convolution and the next block's first 1x1
// convolution, which reads nothing but its output, in one kernel that keeps
// each tile of the first output on chip for the second contraction
// (conv_pair): the second layer no longer reads that output back.  Top-level
// nodes in direct succession on the same rows, no row lists.  The inputs of
// the first stay live through the second, since one launch reads them while
// it writes the second's output.
void Spec::pair_pointwise() {
  if (dt != DType::BF16) return;
  auto plain = [&](const Node& n) {
    return n.kind == NodeKind::Conv && n.body.empty() && n.k == 1 && n.stride == 1 && n.pad == 0 && !n.pad_in &&
           !n.pool && n.act != k::ACT_LSTM && n.packed >= 0 && !n.src_list && !n.src2_list && !n.res_list &&
           !n.dst_list;
  };
  for (size_t i = 0; i + 1 < nodes.size(); ++i) {
    Node& c = nodes[i];
    const Node& d = nodes[i + 1];
    if (!plain(c) || !plain(d) || c.pair) continue;
    if (c.fold ? (c.src2 < 0 || c.res >= 0) : (c.src2 >= 0 || c.scale_off < 0 || c.shift_off < 0)) continue;
    if (d.src != c.dst || d.src2 >= 0 || d.res >= 0 || d.fold || d.scale_off < 0 || d.shift_off < 0 ||
        d.cin1 != c.cout || d.H != c.Ho || d.W != c.Wo || tensors[c.dst].external || tensors[c.dst].unused)
      continue;
    if (!k::conv_pair_fits(c.cin1, c.fold ? c.cin2 : 0, c.cout, d.cout, c.act, d.act)) continue;
    c.pair = true;
    for (int t : {c.src, c.src2, c.res})
      if (t >= 0) tensors[t].last = std::max(tensors[t].last, d.seq_pre);
    ++fused_pairs;
    ++i;   // the second conv is taken
  }
}

// The gather of an exit's carried tensor fused into its readers (a row
// gather is a copy that computes nothing): when every reader of the carried
// copy is a bf16 convolution that takes it as its main input before the next
// decision, the readers take the surviving rows of the original tensor
// through the exit's stay list and the copy is never made.
void Spec::fuse_exit_gathers() {
  if (dt != DType::BF16) return;
  for (size_t i = 0; i < nodes.size(); ++i) {
    Node& ex = nodes[i];
    if (!((ex.kind == NodeKind::Exit && !ex.final_) || ex.kind == NodeKind::Halt ||
          (ex.kind == NodeKind::Decode && !ex.final_)))
      continue;
    size_t next = i + 1;
    while (next < nodes.size() && !is_decision(nodes[next])) ++next;
    for (size_t q = 0; q < ex.pairs.size();) {
      const int from = ex.pairs[q].first, to = ex.pairs[q].second;
      std::vector<Use> us;
      uses_of(nodes, to, -1, us);
      // a reader is a convolution taking the copy as its main input, or as
      // the concatenated input of a folded projection (src2 with no list)
      auto src2_read = [&](const Use& u) {
        const Node& nd = *u.node;
        return !u.conv_src && nd.kind == NodeKind::Conv && nd.src2 == to && nd.src2_list == 0 && nd.src != to &&
               nd.res != to && nd.park_src != to;
      };
      bool ok = !us.empty();
      for (const Use& u : us)
        ok = ok && u.top > static_cast<long>(i) && u.top < static_cast<long>(next) && !u.node->pad_in &&
             ((u.conv_src && (u.node->src2 < 0 || u.node->src2_list == 3 || u.node->src2_list == 1)) || src2_read(u));
      if (!ok) {
        ++q;
        continue;
      }
      for (const Use& u : us) {
        if (u.conv_src) {
          u.node->src = from;
          u.node->src_list = 1;
        } else {
          u.node->src2 = from;
          u.node->src2_list = 1;
        }
        TensorInfo& f = tensors[from];
        f.last = std::max(f.last, u.node->seq_pre);
      }
      tensors[to].unused = true;
      ex.pairs.erase(ex.pairs.begin() + q);
      ++fused_gathers;
    }
  }
}

// Reads of a tensor that is still in sample order, through copies carried
// across decisions: a convolution reads the original through the original
// ids of its rows (the list every run keeps), and carries that nothing reads
// any more are dropped (the bounded loop's input is never copied).
void Spec::fuse_original_order_reads() {
  if (dt != DType::BF16) return;
  std::map<int, int> root;   // carried copy -> the sample-order tensor it copies
  for (const Node& nd : nodes) {
    if (nd.kind != NodeKind::Exit && nd.kind != NodeKind::Halt) continue;
    for (auto& pr : nd.pairs) {
      const int from = pr.first;
      if (root.count(from))
        root[pr.second] = root[from];
      else if (tensors[from].space == 0 && !tensors[from].parked)
        root[pr.second] = from;
    }
  }
  if (root.empty()) return;
  for (Node& nd : nodes) {
    if (nd.kind != NodeKind::Conv || nd.pad_in) continue;
    if (nd.src2 >= 0 && root.count(nd.src2)) {
      nd.src2 = root[nd.src2];
      nd.src2_list = 3;
      tensors[nd.src2].last = std::max(tensors[nd.src2].last, nd.seq_pre);
    }
  }
  // drop carries whose copies nothing reads, until none is left
  for (bool changed = true; changed;) {
    changed = false;
    for (Node& nd : nodes) {
      if (nd.kind != NodeKind::Exit && nd.kind != NodeKind::Halt) continue;
      for (size_t q = 0; q < nd.pairs.size();) {
        std::vector<Use> us;
        uses_of(nodes, nd.pairs[q].second, -1, us);
        if (!us.empty()) {
          ++q;
          continue;
        }
        tensors[nd.pairs[q].second].unused = true;
        nd.pairs.erase(nd.pairs.begin() + q);
        ++fused_gathers;
        changed = true;
      }
    }
  }
}

// A gate's gathers and scatters fused into its body (Sec. 5.4: copies that
// compute nothing stay out of the sub-DNN): the body convolutions read the
// outer tensors through the gate's list of executing rows, and the layer that
// produces a scattered value writes it straight into the outer tensor's rows.
// Only for bodies of convolutions that run on the implicit GEMM anyway (the
// halo kernels stage contiguous images), whose gathered copies are read only
// as main input or residual, and whose scattered values are each written by
// one convolution that reads its target at most as its residual (an element
// read and then written by the same thread).
void Spec::fuse_gate_moves() {
  if (dt != DType::BF16) return;
  // bodies on the streamed-weight halo kernel cannot take row lists; the
  // register-weight one (64 -> 64 channels) can on whole-image tiles
  auto halo_kind = [](const Node& nd, const TensorInfo& src) {
    const bool wres_images = nd.cin1 == 64 && nd.cout == 64 && src.H * src.W <= 128;
    return nd.k == 3 && nd.stride == 1 && nd.pad == 1 && nd.src2 < 0 && nd.cin1 % 64 == 0 && nd.cout % 64 == 0 &&
           !(src.H * src.W <= 128 && 2 * src.H * src.W < (src.H + 2) * (src.W + 2)) && !wres_images;
  };
  for (Node& g : nodes) {
    if (g.kind != NodeKind::Gate) continue;
    bool ok = !g.body.empty();
    for (const Node& b : g.body) ok = ok && b.kind == NodeKind::Conv && !halo_kind(b, tensors[b.src]);
    if (!ok) continue;
    std::map<int, int> outer_of;   // gathered copy -> outer tensor
    for (auto& pr : g.pairs) outer_of[pr.second] = pr.first;
    for (const Node& b : g.body) {
      if (b.src2 >= 0 && outer_of.count(b.src2)) ok = false;
      if (b.dst >= 0 && outer_of.count(b.dst)) ok = false;
    }
    std::map<int, int> writer;     // scattered value -> index of the body conv that writes it
    for (auto& pr : g.scatter) {
      int w = -1, readers = 0;
      for (size_t j = 0; j < g.body.size(); ++j) {
        const Node& b = g.body[j];
        if (b.dst == pr.first) w = static_cast<int>(j);
        if (b.src == pr.first || b.src2 == pr.first || b.res == pr.first) ++readers;
      }
      if (w < 0 || readers) ok = false;
      for (auto& q : g.scatter)
        if (&q != &pr && q.first == pr.first) ok = false;
      writer[pr.first] = w;
    }
    if (!ok) continue;
    // the writer must not read its own target but as the residual, and no
    // body conv after it may read the target at all
    for (auto& pr : g.scatter) {
      const int w = writer[pr.first];
      const int target = pr.second;
      for (size_t j = 0; j < g.body.size(); ++j) {
        const Node& b = g.body[j];
        auto is_target = [&](int t) { return t >= 0 && (t == target || (outer_of.count(t) && outer_of[t] == target)); };
        if (static_cast<int>(j) == w && (is_target(b.src) || is_target(b.src2))) ok = false;
        if (static_cast<int>(j) > w && (is_target(b.src) || is_target(b.src2) || is_target(b.res))) ok = false;
      }
    }
    if (!ok) continue;
    for (Node& b : g.body) {
      if (outer_of.count(b.src)) {
        b.src = outer_of[b.src];
        b.src_list = 2;
        tensors[b.src].last = std::max(tensors[b.src].last, b.seq_pre);
      }
      if (b.res >= 0 && outer_of.count(b.res)) {
        b.res = outer_of[b.res];
        b.res_list = 2;
        tensors[b.res].last = std::max(tensors[b.res].last, b.seq_pre);
      }
    }
    for (auto& pr : g.scatter) {
      Node& b = g.body[writer[pr.first]];
      tensors[pr.first].unused = true;
      b.dst = pr.second;
      b.dst_list = 2;
    }
    for (auto& pr : g.pairs) tensors[pr.second].unused = true;
    g.pairs.clear();
    g.scatter.clear();
    ++fused_gates;
  }
}

void Spec::parse(const std::string& json, size_t weights_bytes, int max_batch, const void* weights) {
  *this = Spec();
  host_w = static_cast<const uint8_t*>(weights);
  Json j = Json::parse(json);
  if (j.kind != Json::Object) throw SpecError("the spec must be a JSON object");
  if (j.get_int("version", 1) != 1) throw SpecError("unsupported spec version");
  const std::string dts = j.at("dtype").as_str("dtype");
  if (dts == "bf16")
    dt = DType::BF16;
  else if (dts == "f32")
    dt = DType::F32;
  else
    throw SpecError("dtype must be bf16 or f32");
  n_out = static_cast<int>(j.at("n_out").as_int("n_out"));
  if (n_out < 1 || n_out > 65536) throw SpecError("n_out out of range");
  aux = j.get_bool("aux", false);
  if (max_batch < 1 || max_batch > (1 << 24)) throw SpecError("max_batch must be in [1, 2^24]");

  if (j.has("decode") && !j.at("decode").is_null()) {
    // a greedy decoding loop: runs emit up to max_len tokens per sample,
    // the first step reading the start token bos
    const Json& dj = j.at("decode");
    any_decode = true;
    max_len = static_cast<int>(dj.at("max_len").as_int("decode.max_len"));
    bos = static_cast<int>(dj.at("bos").as_int("decode.bos"));
    if (max_len < 1 || max_len > 4096) throw SpecError("decode.max_len must be in [1, 4096]");
    if (bos < 0 || bos >= n_out) throw SpecError("decode.bos must be a token of the vocabulary (n_out)");
    if (dt != DType::BF16) throw SpecError("decoding needs a bf16 spec");
  }
  Builder b(*this, weights_bytes);
  const Json& in = j.at("input");
  const Json& shp = in.at("shape");
  int H = 1, W = 1, C = 1;
  if (shp.size() == 3) {
    H = static_cast<int>(shp.at(0).as_int("shape"));
    W = static_cast<int>(shp.at(1).as_int("shape"));
    C = static_cast<int>(shp.at(2).as_int("shape"));
  } else if (shp.size() == 1) {
    C = static_cast<int>(shp.at(0).as_int("shape"));
  } else {
    throw SpecError("input.shape is [H, W, C] or [D]");
  }
  input = b.define(in.at("name"), H, W, C, seq++, "input");
  tensors[input].external = true;
  if (tensors[input].row_bytes(dt) % 16 != 0 && (dt == DType::F32 || C % 8 == 0))
    ;  // rows are moved only for non-input tensors; nothing to check here
  const Json& ns = j.at("nodes");
  if (ns.kind != Json::Array || ns.size() == 0) throw SpecError("nodes must be a non-empty array");
  for (size_t i = 0; i < ns.size(); ++i) nodes.push_back(b.node(ns.at(i), max_batch));
  fuse_stem_pools();
  fuse_projections();
  fuse_original_order_reads();
  fuse_exit_gathers();
  fuse_gate_moves();
  if (j.get_bool("pair_pointwise", true)) pair_pointwise();

  // every tensor that is moved between row groups must be a whole number of
  // 16-byte vectors, and a whole batch of it must be indexable with 32-bit
  // pixel offsets
  for (const TensorInfo& t : tensors) {
    if (!t.external && t.row_bytes(dt) % 16 != 0)
      throw SpecError("tensor '" + t.name + "': per-sample bytes must be a multiple of 16");
    if (static_cast<int64_t>(max_batch) * t.H * t.W * t.C >= (int64_t(1) << 31))
      throw SpecError("tensor '" + t.name + "': max_batch rows exceed 2^31 elements");
  }

  std::ostringstream os;
  os << "nodes=" << nodes_total << " decisions=" << decisions << " tensors=" << tensors.size()
     << " packed_weights=" << packed.size() << " fused_gathers=" << fused_gathers
     << " fused_gates=" << fused_gates << " fused_pools=" << fused_pools
     << " fused_projections=" << fused_projections << " fused_pairs=" << fused_pairs << " n_out=" << n_out
     << " dtype=" << dts;
  summary = os.str();
  host_w = nullptr;   // the caller's blob is not kept
}

}  // namespace dycl
