// Host-side launchers of the gfx950 kernels.  Every launcher checks nothing
// about shapes: the plan builder validates them before any launch, and each
// launcher is called only with n >= 1 rows.
//
// Row counts on the device: the launchers whose work scales with the row
// count take `nc`, a device pointer to the live count.  With nc null the
// kernels process n rows; otherwise the launch is sized for n rows (an
// upper bound the host knows) and the kernels read the count when they
// start and process min(*nc, n) rows (possibly none), so the host never has
// to wait for a count to launch the next kernel.  `nhint`, where taken, is
// the live count the host expects (0: n): it only picks the tile shape or
// rows per workgroup, which change no result.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/dycl.h"

namespace dycl {
namespace k {

// ACT_TANH and ACT_LSTM run on the implicit-GEMM kernel only (linear
// layers on 1x1 rows).  ACT_LSTM: the layer's cout = 4 H outputs are the
// gates of H cells interleaved (channel 4 j + k = gate k of cell j: input,
// forget, cell, output); the epilogue is the cell itself, reading the old
// cell state (cell_in, float32 [rows][H], through res_rows; null: zeros)
// and writing the new one (cell_out) and h = o tanh(c) in bf16 to dst
// [rows][H].
enum Act { ACT_NONE = 0, ACT_RELU = 1, ACT_GELU = 2, ACT_TANH = 3, ACT_LSTM = 4 };

// The implicit-GEMM convolution picks its tile at launch from the active
// row count.  Packed weights are [conv_cout_pad(cout)][Kp] with Kp a
// multiple of kBK, zero-filled, so that every tile width divides the rows.
constexpr int kBK = 64;
int conv_cout_pad(int cout);

struct ConvArgs {
  const uint16_t* src;   // [n, H, W, cin1] bf16 NHWC
  const uint16_t* src2;  // [n, H2, W2, cin2] channel concat (k == 1, pad 0 only), read at output pixel
                         // (oh, ow) from (oh * src2_stride, ow * src2_stride), or null
  int src2_H = 0, src2_W = 0, src2_stride = 1;   // 0: src2 has the spatial shape of src
  int cin1, cin2;        // cin = cin1 + cin2
  int n, H, W, cin, Ho, Wo, cout, k, stride, pad;
  const uint16_t* w;     // packed [cout_pad][Kp] bf16, K order (kh, kw, ci)
  int Kp;
  const float* scale;    // [cout] or null (1)
  const float* shift;    // [cout] or null (0)
  const uint16_t* res;   // [n, Ho, Wo, cout] bf16 or null
  int act;
  void* dst;             // [n, Ho, Wo, cout] bf16, or fp32 when out_f32
  int out_f32;
  const uint16_t* zeros; // >= 16 zero bytes on the device (padding taps)
  const int32_t* ncount = nullptr;  // device count of live images (<= n) or null
  int nhint = 0;                    // expected live images for the tile choice (0: n)
  // fused gathers / scatters: image i of the layer reads image src_rows[i]
  // of src and res_rows[i] of res and writes image dst_rows[i] of dst (null: i)
  const int32_t* src_rows = nullptr;
  const int32_t* src2_rows = nullptr;
  const int32_t* res_rows = nullptr;
  const int32_t* dst_rows = nullptr;
  int list_rows = 0;     // rows of the tensors read or written through a list (0: no list)
  float* splitws = nullptr;         // K-split partial sums (conv_ksplit_bytes), or null: no split
  size_t splitws_bytes = 0;
  const float* cell_in = nullptr;   // ACT_LSTM: old cell state, or null (zeros)
  float* cell_out = nullptr;        // ACT_LSTM: new cell state
  // a folded projection shortcut (src2 holds its input, its weights are
  // the last cin2 K columns, cin1 and cin2 multiples of kBK): the kfold K
  // steps of src2 run first and their sum becomes bf16(fold_sp * acc +
  // fold_bp) * fold_inv before the block's own steps add to it (0: none)
  int kfold = 0;
  const float* fold_sp = nullptr;
  const float* fold_bp = nullptr;
  const float* fold_inv = nullptr;
  // 1: a 3x3 / stride-2 / pad-1 max-pool of the output is fused in and dst
  // holds the pooled tensor [n, (Ho - 1) / 2 + 1, (Wo - 1) / 2 + 1, cout]
  // (conv_rgb_stem with ReLU only)
  int pool = 0;
  // global average pooling of the output taken in the epilogue: when set,
  // Ho * Wo >= 32, the output is bf16 without a dst list and the layer runs
  // on the implicit-GEMM kernel without a K split, each output column's sum
  // over each 32-row chunk of layer rows (image * Ho * Wo + pixel; the bf16
  // values as stored, added in row order) goes to gap_part[chunk][0][cout],
  // split at an image boundary inside the chunk: the rows of the next image
  // to gap_part[chunk][1][cout]; conv_bf16 then returns true
  float* gap_part = nullptr;
  // 1: the implicit GEMM walks each XCD's tiles last to first (the results
  // do not depend on the order); alternating it from one layer to the next
  // lets a layer start on the rows its producer wrote last, which the
  // memory-side cache still holds
  int rev = 0;
};
bool conv_bf16(const ConvArgs& a, hipStream_t s);

// A bottleneck block's last 1x1 layer and the next block's first 1x1 layer
// in one kernel (both stride 1, no row lists; 256 -> 64 channels, or 512 ->
// 128 without a fold):
//   y3 = act3(scale3 * (x W3^T) + shift3 + res)   [n * H * W][C3]
//   y1 = act1(scale1 * (y3 W1^T) + shift1)        [n * H * W][C1]
// with packed weights w3 [>= C3][Kp3] and w1 [>= C1][Kp1] (C3 used).  The
// first layer may carry a folded projection shortcut instead of a residual
// (x2 set; ConvArgs::kfold and its vectors): x2 [n][H2][W2][K2] read at
// stride s2, whose K steps are the last K2 / 64 of w3.  Both outputs are bit
// for bit those of the two layers launched one by one through conv_bf16.
// Every pointer 16-byte aligned; ncount, when set, is the device count of
// live images (<= n).  conv_pair_fits says whether the kernel takes a shape,
// conv_pair_takes whether it takes an argument set; conv_pair returns false
// (launching nothing) when the arguments do not qualify.
struct PairArgs {
  const uint16_t* x = nullptr;
  int K3 = 0;                          // channels of x
  const uint16_t* x2 = nullptr;        // a folded projection's input, or null
  int K2 = 0, H2 = 0, W2 = 0, s2 = 1;
  const float* fold_sp = nullptr;
  const float* fold_bp = nullptr;
  const float* fold_inv = nullptr;
  const uint16_t* w3 = nullptr;
  int Kp3 = 0;
  const float* scale3 = nullptr;
  const float* shift3 = nullptr;
  const uint16_t* res = nullptr;       // or null
  uint16_t* y3 = nullptr;
  int C3 = 0;
  const uint16_t* w1 = nullptr;
  int Kp1 = 0;
  const float* scale1 = nullptr;
  const float* shift1 = nullptr;
  uint16_t* y1 = nullptr;
  int C1 = 0;
  int act3 = 0, act1 = 0;
  int n = 0, H = 0, W = 0;
  const int32_t* ncount = nullptr;
  const uint16_t* zeros = nullptr;
  int rev = 0;   // as ConvArgs::rev
};
bool conv_pair_fits(int K3, int K2, int C3, int C1, int act3, int act1);
bool conv_pair_takes(const PairArgs& a);
bool conv_pair(const PairArgs& a, hipStream_t s);

// the pooled features of n images from those chunk sums: G[r][c] = (sum of
// image r's parts of the chunks it overlaps, in chunk order) / HW
void gap_chunks(const float* Q, int n, int HW, int C, float* G, hipStream_t s, const int32_t* nc = nullptr);

// 7x7 stride-2 stems on 3-channel (RGB) input with 64 output channels,
// W % 8 == 0, output rows of at most 112 pixels: a dedicated kernel reads
// the 3-channel input directly (no channel padding).
// conv_rgb_stem_fits says whether a shape qualifies; conv_rgb_stem launches
// it for a conv_bf16 argument set with plain packed weights and returns
// false (launching nothing) when the arguments do not qualify (row lists, a
// residual, a device count, fp32 output, misaligned pointers, a fused
// max-pool without ReLU).
bool conv_rgb_stem_fits(int H, int W, int cin, int cout, int k, int stride, int pad);
bool conv_rgb_stem(const ConvArgs& a, hipStream_t s);

// 3x3 / stride-1 / pad-1 layers with 16 -> 16 or 32 -> 32 channels on 16- or
// 32-pixel-wide images (row lists and device counts allowed): a halo kernel
// with all weights in registers.  Returns false (launching nothing) for
// other arguments.
bool conv3_narrow(const ConvArgs& a, hipStream_t s);

// K ranges per output tile for the layer shape (1: none).  A split layer
// needs conv_ksplit_bytes of workspace; without it the layer runs unsplit
// (the same sums in another order).  Depends on the shape only, so every
// row count takes the same rounding.
int conv_ksplit(int Ho, int Wo, int cout, int K, bool out_f32);
inline size_t conv_ksplit_bytes(int n, int Ho, int Wo, int cout, int K, bool out_f32) {
  const int S = conv_ksplit(Ho, Wo, cout, K, out_f32);
  return S > 1 ? static_cast<size_t>(S) * n * Ho * Wo * cout * sizeof(float) : 0;
}

// 128 zero bytes in device memory of the current device (the source of the
// convolutions' padding taps), or null if the symbol cannot be resolved
const uint16_t* zero_page();

// Y[m, j] = act(sum_k X[m, k] Wt[k, j] + bias[j]), fp32, weights transposed;
// for few rows (MLP layers, exit heads)
void linear_t_f32(const float* X, int n, int K, const float* Wt, const float* bias, int N, int act, float* Y,
                  hipStream_t s, const int32_t* nc = nullptr, int nhint = 0);

// Y[m, j] = act(sum_k X[m, k] W[j, k] + bias[j]), fp32
void linear_f32(const float* X, int n, int K, const float* W, const float* bias, int N, int act, float* Y,
                hipStream_t s);

// G[r, c] = sum_{hw} x[r, hw, c] / HW.  With a workspace P of
// kGapMaxSplit * n * C floats, long rows are split over several workgroups
// (partial sums, then a fixed-order merge; the split depends on HW only);
// P may be null.
constexpr int kGapMaxSplit = 16;
void gap_bf16(const uint16_t* x, int n, int HW, int C, float* G, float* P, hipStream_t s,
              const int32_t* nc = nullptr);

// Exit decision from head logits Z [n, ncls]: p = max softmax(Z / T); rows
// with p >= tau (or all rows when final) write their logits and exit index at
// their original position.
void exit_decide(const float* Z, int n, int ncls, const float* T, float tau, int final_, int head,
                 const int32_t* orig, uint8_t* flags, float* logits, int n_out, dycl_record* rec, hipStream_t s,
                 const int32_t* nc = nullptr);

// Exit head over pooled features G [n][K] float32 with transposed weights
// Wt [K][ncls] (ncls <= 1024): the linear cut into head_slices(K) K-slices
// whose partial sums (P, head_partials_floats(K, n, ncls) floats) are added
// in slice order with the bias, then the decision as exit_decide takes it.
int head_slices(int K);
bool head_sliced_fits(int K, int ncls);   // K <= 2048 (16 slices), ncls <= 1024
size_t head_partials_floats(int K, int n, int ncls);
void exit_head_sliced(const float* G, int n, int K, const float* Wt, const float* bias, int ncls, const float* T,
                      float tau, int final_, int head, const int32_t* orig, uint8_t* flags, float* logits, int n_out,
                      dycl_record* rec, float* P, hipStream_t s, const int32_t* nc = nullptr);

// Fused exit head for small heads (C <= 2048 and a multiple of 4, ncls <=
// 1024): pooling, head linear on the weights as stored W [ncls][C] (16-byte
// aligned rows), and the exit decision, up to 8 rows per workgroup.  Same
// outputs as gap_bf16 + linear_t_f32 + exit_decide.
void exit_head(const void* x, bool bf16, int n, int HW, int C, const float* W, const float* bias, int ncls,
               const float* T, float tau, int final_, int head, const int32_t* orig, uint8_t* flags, float* logits,
               int n_out, dycl_record* rec, hipStream_t s, const int32_t* nc = nullptr, int nhint = 0);

// Gate: q = sigmoid(u . GAP(x) + v); flag = q > thr (execute); skipped rows set
// bit `gate` of their record.
void gate_head(const uint16_t* x, int n, int HW, int C, const float* u, const float* v, float thr, int gate,
               const int32_t* orig, uint8_t* flags, dycl_record* rec, hipStream_t s, const int32_t* nc = nullptr);

// Halting unit of step `step`: p = sigmoid(w . h + aux[orig]); S[orig] += p;
// flag = S >= tau or step == max_steps (halt); halted rows record step.
void halt_head(const uint16_t* h, int n, int C, const float* w, const float* aux, const int32_t* orig, float* S,
               int step, int max_steps, float tau, uint8_t* flags, dycl_record* rec, hipStream_t s,
               const int32_t* nc = nullptr);

// Stable two-way partition of rows 0..n-1 by flag: idx1/org1 list the rows
// (and their original ids) with flag != 0, idx0/org0 the others, in order;
// counts[0] = |flag != 0|, counts[1] = the rest.
void compact(const uint8_t* flags, const int32_t* orig, int n, int32_t* idx1, int32_t* org1, int32_t* idx0,
             int32_t* org0, int32_t* counts, hipStream_t s, const int32_t* nc = nullptr);

// The same partition for large n (one chained pass over 4096-flag blocks:
// a clearing kernel, then the pass); org1 / org0 may be null.  workspace:
// compact_workspace(n) bytes, 8-byte aligned.  n < 2^31.
size_t compact_workspace(size_t n);
void compact_large(const uint8_t* flags, const int32_t* orig, size_t n, int32_t* idx1, int32_t* org1, int32_t* idx0,
                   int32_t* org0, int32_t* counts, void* workspace, hipStream_t s, const int32_t* nc = nullptr);

// Device address, on the current device, of the library's static compaction
// scratch (kScratchBytes, 256-byte aligned), resolved on the first call per
// device; null if it cannot be resolved.  Enough for compact_large of up to
// kScratchCompactMaxN flags, or 8 * n bytes of ids for n <= 16384.  Every
// call on one device shares it: calls that overlap there race.
constexpr size_t kScratchCompactMaxN = size_t(1) << 28;
constexpr size_t kScratchBytes = ((kScratchCompactMaxN + 4095) / 4096) * (sizeof(int32_t) + sizeof(int64_t)) + 256;
constexpr int kMaxDevices = 64;
void* compact_scratch();

// dst row (dst_idx ? dst_idx[r] : r) = src row (src_idx ? src_idx[r] : r),
// r < n; row_bytes is a multiple of 16.
void move_rows(void* dst, const int32_t* dst_idx, const void* src, const int32_t* src_idx, size_t row_bytes, int n,
               hipStream_t s, const int32_t* nc = nullptr);

// y[p, c] = c < cin ? x[p, c] : 0 for every pixel p, c < cout (cout == 8)
void pad_channels_bf16(const uint16_t* x, size_t pixels, int cin, int cout, uint16_t* y, hipStream_t s);

// up to 4 tensors moved with one index list in one launch
struct MoveSet {
  int count;
  void* dst[4];
  const void* src[4];
  size_t vpr[4];   // 16-byte vectors per row
};
void move_rows_multi(const MoveSet& set, const int32_t* dst_idx, const int32_t* src_idx, int n, hipStream_t s,
                     const int32_t* nc = nullptr);

void maxpool3s2_bf16(const uint16_t* x, int n, int H, int W, int C, uint16_t* y, hipStream_t s,
                     const int32_t* nc = nullptr);
// counts[0] = *nc (or n when nc is null), counts[1] = 0: the branch counts of
// a final exit, which every row takes
void final_counts(const int32_t* nc, int n, int32_t* counts, hipStream_t s);
void init_records(dycl_record* rec, int n, hipStream_t s);
void fill_f32(float* p, float v, int n, hipStream_t s);
void fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t s);
// dst[i] = src[idx[i]] for i < min(*nc, n) (nc null: n)
void gather_i32(int32_t* dst, const int32_t* src, const int32_t* idx, int n, hipStream_t s,
                const int32_t* nc = nullptr);

// One step of greedy decoding on the step's logits Z [n][V] (float32): the
// token of row r is the argmax of its logits (the lowest index among equal
// maxima); tok_next[r] = token; tokens[orig[r] * max_len + step - 1] =
// token; the row finishes (flag 1) when the token is `eos` or step ==
// max_len, and then records `step` as its iteration count and copies its
// logits to logits[orig[r]] (row length V).  V % 4 == 0.
void decode_step(const float* Z, int n, int V, int eos, int step, int max_len, const int32_t* orig,
                 uint8_t* flags, int32_t* tok_next, int32_t* tokens, float* logits, dycl_record* rec, hipStream_t s,
                 const int32_t* nc = nullptr);
void iota_i32(int32_t* p, int n, hipStream_t s);

// The bounded loop of an adaptive-computation-time network, every step in
// one cooperative launch (one workgroup per CU, grid barriers between the
// phases of a step): step t computes h_t = bf16(GELU(W1 [h_{t-1}; x] + b1))
// for the running rows (step 1: the x columns only, h_0 = 0), the halting
// unit (S += sigmoid(wh . h_t + aux), halt at S >= tau or t == steps),
// parks the halted rows' h_t in sample order and compacts the running
// rows.  Bit for bit what the per-step kernels compute.  Rows start in
// sample order; B <= act_loop_max_rows().
struct ActLoopArgs {
  const uint16_t* x;   // [B][D] bf16
  const uint16_t* w;   // packed W1 [>= H][Kp] bf16, K = [h | x] (H + D)
  int Kp;
  const float* b1;     // [H]
  const float* wh;     // [H]
  const float* aux;    // [B]
  uint16_t* h0;        // two [B][H] bf16 state buffers
  uint16_t* h1;
  uint16_t* park;      // [B][H] bf16, sample order
  float* S;            // [B], zero
  uint8_t* flags;      // [B]
  int32_t* counts;     // branch counts, decision d0 + t - 1 for step t
  int d0;
  dycl_record* rec;
  const uint16_t* zeros;
  int B, H, D, steps;
  float tau;
};
size_t act_loop_max_rows();
bool act_loop_fits(int B, int H, int D);
void act_loop(const ActLoopArgs& a, hipStream_t s);

}  // namespace k
}  // namespace dycl
