// Two consecutive 1x1 convolutions of a bottleneck network in one kernel:
// a block's last 1x1 layer (folded BatchNorm, residual, activation) and the
// first 1x1 layer of the next block, whose only input is that output.
//   y3 = act3(s3 * (x W3^T) + b3 + r)      [M][C3]
//   y1 = act1(s1 * (y3 W1^T) + b1)         [M][C1]
// Run as two layers, y3 goes to HBM and the second layer reads all of it
// back (2 * C3 bytes per row: 512 at ResNet-50's first stage, where the
// pair moves 1 280 bytes per row fused against 1 792 unfused).  Here a
// workgroup keeps its 64 rows of y3, rounded to bf16 exactly as they are
// stored, in LDS: it writes them out once and runs the second contraction
// on them.
//
// Both contractions are the implicit GEMM of the single layers with the
// MFMA operands swapped: the weights are the A operand (rows = output
// channels) and the pixels the B operand, so a lane's accumulators hold 4
// consecutive channels of one pixel and the epilogues work on 8-byte pieces
// of NHWC rows.  Each output is the same sum of the same products, taken
// in the same K order with the same v_mfma_f32_32x32x16_bf16 steps, as in
// the single-layer kernel, and the epilogue arithmetic is the same, so the
// two outputs are bit for bit those of the two layers run one by one.
//
// A tile's course (512 threads, eight waves):
//  1. the scale / shift vectors, the tile's x rows and W3 (one 64-wide K
//     step), and the residual rows are requested straight into LDS (the
//     residual into the y3 buffer), W1 into registers;
//  2. MFMAs of the first contraction (wave: 64 channels x 32 pixels);
//  3. epilogue in place: each lane reads the residual of its 4 channels of
//     one pixel, finishes them and writes the bf16 result over it; W1 goes
//     to the space of W3 and x;
//  4. waves 0-3 run the second contraction (32 x 32 each) from the y3
//     buffer and stage its bf16 output; waves 4-7 meanwhile store y3;
//  5. all waves store y1.
// LDS 74.5 KB: two workgroups per CU.
#include <stdexcept>

#include "kernels.hpp"

namespace dycl {
namespace k {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void* lds_ptr;

struct PairP {
  const uint16_t* x;     // [M][cin1]
  const uint16_t* x2;    // a folded projection's input [n][H2][W2][cin2], or null
  const uint16_t* w3;    // [>= C3][Kp3] packed; a fold's K steps are the last kfold
  const float* v3[5];    // s3, b3 (and the fold's s_p, b_p, 1 / s3)
  const uint16_t* res;   // [M][C3], or null
  uint16_t* y3;          // [M][C3]
  const uint16_t* w1;    // [>= C1][Kp1] packed (Kp1 >= C3)
  const float* sc1;
  const float* sh1;
  uint16_t* y1;          // [M][C1]
  const uint16_t* zeros; // >= 16 zero bytes: the source of rows past M
  const int32_t* nc;     // device count of live images (<= nmax) or null
  int nmax, H, W, cin1, cin2, H2, W2, s2, Kp3, Kp1, rev;
};

constexpr int kRowsT = 64;    // rows per tile
constexpr int kThr = 512;     // threads per workgroup

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

template <int ACT>
__device__ __forceinline__ float act_of(float v) {
  if (ACT == ACT_RELU) return v > 0.f ? v : 0.f;
  if (ACT == ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  return v;
}

// wait until at most N of this wave's vector-memory operations are in
// flight (they complete in order), then barrier
template <int N>
__device__ __forceinline__ void vm_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// this wave's LDS operations done, then barrier (global loads and stores
// may stay in flight)
__device__ __forceinline__ void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ void to_lds(const void* g, char* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr)(lds_wave_base), 16, 0, 0);
}

template <int C3, int C1, int ACT3, int ACT1, bool RES, bool FOLD>
__global__ __launch_bounds__(kThr) __attribute__((amdgpu_waves_per_eu(4))) void conv_pair_kernel(PairP p) {
  static_assert(C3 == 256 && C1 == 64, "tile roles are laid out for 256 -> 64 channels");
  constexpr int W3_BYTES = C3 * 128;            // one 64-wide K step of W3
  constexpr int X_BYTES = kRowsT * 128;         // one K step of the tile's x rows
  constexpr int S_BYTES = W3_BYTES + X_BYTES;
  constexpr int ROW3 = C3 * 2;                  // bytes of a y3 row
  constexpr int CPR = ROW3 / 16;                // 16-byte chunks of a y3 row
  constexpr int A_BYTES = kRowsT * ROW3;
  constexpr int NV3 = (FOLD ? 5 : 2) * C3;      // [s3 | b3 (| s_p | b_p | 1 / s3)]
  constexpr int NV = NV3 + 2 * C1;              // then [s1 | b1]
  constexpr int JW3 = W3_BYTES / 16 / kThr;     // loads per thread: W3, residual, W1
  constexpr int JR = A_BYTES / 16 / kThr;
  constexpr int JW1 = C1 * ROW3 / 16 / kThr;
  static_assert(C1 * ROW3 <= W3_BYTES, "W1 takes the place of W3");
  static_assert(kRowsT * C1 * 2 <= X_BYTES, "the y1 staging takes the place of x");
  static_assert(X_BYTES == 16 * kThr && CPR == 32, "one x load per thread; 32 chunks per y3 row");
  static_assert(NV / 4 <= kThr, "one vector load per thread at most");
  // separate LDS objects, so that the compiler can tell a direct-to-LDS
  // load into one from a read of another (and does not wait for the loads
  // in flight before reading the vectors)
  __shared__ __align__(16) char sw[W3_BYTES];   // W3, then W1
  __shared__ __align__(16) char sx[X_BYTES];    // x, then the y1 staging
  __shared__ __align__(16) char sa[A_BYTES];    // the residual, then y3
  __shared__ __align__(16) float sv[NV];

  const int HW = p.H * p.W;
  const int M = (p.nc ? min(*p.nc, p.nmax) : p.nmax) * HW;
  const int T = (M + kRowsT - 1) / kRowsT;
  const int wg = blockIdx.x;
  if (wg >= T) return;
  // consecutive tiles on one XCD; every other layer walks them backwards
  const int T8 = (T >> 3) << 3;
  const int t = wg < T8 ? (wg & 7) * (T8 >> 3) + (p.rev ? (T8 >> 3) - 1 - (wg >> 3) : (wg >> 3)) : wg;
  const int m0 = t * kRowsT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // 1. requests, oldest first: vectors, x and W3, then the residual
  if (tid < NV / 4) {
    const int q = tid * 4;   // float index in [v3 ... | s1 | b1]
    const float* g = q < NV3 ? p.v3[q / C3] + q % C3 : q < NV3 + C1 ? p.sc1 + (q - NV3) : p.sh1 + (q - NV3 - C1);
    to_lds(g, reinterpret_cast<char*>(sv) + wave * 1024);
  }
  // rows of 128 bytes (x, W3): chunk c of row r at physical chunk c ^ ((r >> 1) & 7)
  const int lc128 = (tid & 7) ^ ((tid >> 4) & 7);
  const int xm = m0 + (tid >> 3);   // this thread's x row
  int xpix2 = 0;                    // its pixel in a folded projection's input
  if (FOLD && xm < M) {
    const int img = xm / HW, rem = xm - img * HW, oh = rem / p.W, ow = rem - oh * p.W;
    xpix2 = (img * p.H2 + oh * p.s2) * p.W2 + ow * p.s2;
  }
  const int kfold = FOLD ? p.cin2 / 64 : 0;
  const int nk3 = (p.cin1 + (FOLD ? p.cin2 : 0)) / 64;
  // K step kt: a fold's projection steps first (its input, the last kfold
  // steps of W3), then the block's own
  auto issue_xw = [&](int kt) __attribute__((always_inline)) {
    const bool proj = FOLD && kt < kfold;
    const int kw = proj ? kt + (p.Kp3 / 64 - kfold) : kt - kfold;
    to_lds(xm >= M ? p.zeros
           : proj  ? p.x2 + static_cast<size_t>(xpix2) * p.cin2 + kt * 64 + lc128 * 8
                   : p.x + static_cast<size_t>(xm) * p.cin1 + (kt - kfold) * 64 + lc128 * 8,
           sx + wave * 1024);
#pragma unroll
    for (int j = 0; j < JW3; ++j) {
      const int row = (j * kThr + tid) >> 3;
      to_lds(p.w3 + static_cast<size_t>(row) * p.Kp3 + kw * 64 + lc128 * 8, sw + (j * kThr + wave * 64) * 16);
    }
  };
  // rows of ROW3 bytes (y3, W1): chunk c of row r at physical chunk c ^ (r & 15)
  issue_xw(0);
  if (RES) {
#pragma unroll
    for (int j = 0; j < JR; ++j) {
      const int q = j * kThr + tid, row = q / CPR, lc = (q % CPR) ^ (row & 15);
      const int m = m0 + row;
      to_lds(m < M ? p.res + static_cast<size_t>(m) * C3 + lc * 8 : p.zeros, sa + (j * kThr + wave * 64) * 16);
    }
  }

  // W1 into registers (it goes to LDS after the epilogue).  Everything is
  // requested at once and awaited at once: with direct-to-LDS loads and
  // register loads both in flight, the compiler waits for all of them
  // before any LDS read anyway.  (Four named vectors, not an array: an
  // array would be kept in scratch memory across the barriers' memory
  // clobbers.)
  static_assert(JW1 == 4, "four W1 vectors per thread");
  auto w1_at = [&](int j) __attribute__((always_inline)) {
    const int q = j * kThr + tid;
    return *reinterpret_cast<const uint4*>(p.w1 + static_cast<size_t>(q / CPR) * p.Kp1 + (q % CPR) * 8);
  };
  const uint4 w1a = w1_at(0), w1b = w1_at(1), w1c = w1_at(2), w1d = w1_at(3);

  // 2. first contraction: wave (wc, wp) = 64 channels x 32 pixels
  const int wc = wave & 3, wp = wave >> 2;
  f32x16 acc3[2];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc3[b][r] = 0.f;
  // the projection's sums become its output as the unfused layer stores it
  // (scale, shift, bf16), divided by the block's scale: done while the
  // block's first K step is in flight
  auto fold_round = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c0 = 64 * wc + 32 * b + 8 * g + 4 * (lane >> 5);
        const float4 sp = *reinterpret_cast<const float4*>(sv + 2 * C3 + c0);
        const float4 bp = *reinterpret_cast<const float4*>(sv + 3 * C3 + c0);
        const float4 iv = *reinterpret_cast<const float4*>(sv + 4 * C3 + c0);
        const float spv[4] = {sp.x, sp.y, sp.z, sp.w}, bpv[4] = {bp.x, bp.y, bp.z, bp.w},
                    ivv[4] = {iv.x, iv.y, iv.z, iv.w};
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc3[b][4 * g + i] =
              __uint_as_float(static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(
                                  fmaf(acc3[b][4 * g + i], spv[i], bpv[i]))))
                              << 16) *
              ivv[i];
      }
  };
  for (int kt = 0; kt < nk3; ++kt) {
    if (kt) {
      lds_sync();   // every wave is done reading the previous step
      issue_xw(kt);
      if (FOLD && kt == kfold) fold_round();
    }
    vm_barrier<0>();
    const int lsw = (lane >> 1) & 7;
    const char* pa = sw + (64 * wc + (lane & 31)) * 128;
    const char* pb = sx + (32 * wp + (lane & 31)) * 128;
    bf16x8 af[2][2], bx[2];
    auto fetch = [&](int s, int slot) __attribute__((always_inline)) {
      const int phys = ((2 * s + (lane >> 5)) ^ lsw) * 16;
      af[slot][0] = *reinterpret_cast<const bf16x8*>(pa + phys);
      af[slot][1] = *reinterpret_cast<const bf16x8*>(pa + 32 * 128 + phys);
      bx[slot] = *reinterpret_cast<const bf16x8*>(pb + phys);
    };
    fetch(0, 0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s + 1 < 4) fetch(s + 1, (s + 1) & 1);
#pragma unroll
      for (int b = 0; b < 2; ++b)
        acc3[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1][b], bx[s & 1], acc3[b], 0, 0, 0);
    }
  }
  lds_sync();   // every wave is done reading W3 and x

  // 3. epilogue of the first contraction, in place over the residual
  {
    const int row = 32 * wp + (lane & 31);
    char* const arow = sa + row * ROW3 + (lane >> 5) * 8;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c0 = 64 * wc + 32 * b + 8 * g + 4 * (lane >> 5);
        uint2* const e = reinterpret_cast<uint2*>(arow + (((c0 >> 3) ^ (row & 15)) * 16));
        const float4 s = *reinterpret_cast<const float4*>(sv + c0);
        const float4 h = *reinterpret_cast<const float4*>(sv + C3 + c0);
        float v0 = fmaf(acc3[b][4 * g + 0], s.x, h.x);
        float v1 = fmaf(acc3[b][4 * g + 1], s.y, h.y);
        float v2 = fmaf(acc3[b][4 * g + 2], s.z, h.z);
        float v3 = fmaf(acc3[b][4 * g + 3], s.w, h.w);
        if (RES) {
          const uint2 r = *e;
          v0 += __uint_as_float(r.x << 16);
          v1 += __uint_as_float(r.x & 0xffff0000u);
          v2 += __uint_as_float(r.y << 16);
          v3 += __uint_as_float(r.y & 0xffff0000u);
        }
        *e = make_uint2(pack2(act_of<ACT3>(v0), act_of<ACT3>(v1)), pack2(act_of<ACT3>(v2), act_of<ACT3>(v3)));
      }
  }
  // W1 into the space of W3 and x, which every wave has finished reading
  auto w1_put = [&](int j, const uint4& v) __attribute__((always_inline)) {
    const int q = j * kThr + tid, row = q / CPR;
    *reinterpret_cast<uint4*>(sw + row * ROW3 + (((q % CPR) ^ (row & 15)) * 16)) = v;
  };
  w1_put(0, w1a);
  w1_put(1, w1b);
  w1_put(2, w1c);
  w1_put(3, w1d);
  lds_sync();   // W1 and y3 complete

  // 4. second contraction (waves 0-3) while waves 4-7 store y3
  if (wave < 4) {
    const int bch = wave & 1, bpx = wave >> 1;
    f32x16 acc1;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc1[r] = 0.f;
    const char* pa = sw + (32 * bch + (lane & 31)) * ROW3;
    const char* pb = sa + (32 * bpx + (lane & 31)) * ROW3;
    const int lsw = lane & 15;
    bf16x8 af[2], bx[2];
    auto fetch = [&](int s, int slot) __attribute__((always_inline)) {
      const int phys = ((2 * s + (lane >> 5)) ^ lsw) * 16;
      af[slot] = *reinterpret_cast<const bf16x8*>(pa + phys);
      bx[slot] = *reinterpret_cast<const bf16x8*>(pb + phys);
    };
    fetch(0, 0);
#pragma unroll
    for (int s = 0; s < C3 / 16; ++s) {
      if (s + 1 < C3 / 16) fetch(s + 1, (s + 1) & 1);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1], bx[s & 1], acc1, 0, 0, 0);
    }
    const int px = 32 * bpx + (lane & 31);
    char* const yrow = sx + px * (C1 * 2) + (lane >> 5) * 8;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c0 = 32 * bch + 8 * g + 4 * (lane >> 5);
      const float4 s = *reinterpret_cast<const float4*>(sv + NV3 + c0);
      const float4 h = *reinterpret_cast<const float4*>(sv + NV3 + C1 + c0);
      const float v0 = act_of<ACT1>(fmaf(acc1[4 * g + 0], s.x, h.x));
      const float v1 = act_of<ACT1>(fmaf(acc1[4 * g + 1], s.y, h.y));
      const float v2 = act_of<ACT1>(fmaf(acc1[4 * g + 2], s.z, h.z));
      const float v3 = act_of<ACT1>(fmaf(acc1[4 * g + 3], s.w, h.w));
      *reinterpret_cast<uint2*>(yrow + (((c0 >> 3) ^ (px & 7)) * 16)) = make_uint2(pack2(v0, v1), pack2(v2, v3));
    }
  } else {
    const int t2 = tid - 256;
#pragma unroll
    for (int j = 0; j < A_BYTES / 16 / 256; ++j) {
      const int q = j * 256 + t2, row = q / CPR, lc = q % CPR;
      if (m0 + row < M)
        *reinterpret_cast<uint4*>(p.y3 + static_cast<size_t>(m0 + row) * C3 + lc * 8) =
            *reinterpret_cast<const uint4*>(sa + row * ROW3 + ((lc ^ (row & 15)) * 16));
    }
  }
  lds_sync();   // the y1 staging is written

  // 5. y1 rows: one 16-byte piece per thread
  {
    const int row = tid / (C1 / 8), lc = tid % (C1 / 8);
    if (m0 + row < M)
      *reinterpret_cast<uint4*>(p.y1 + static_cast<size_t>(m0 + row) * C1 + lc * 8) =
          *reinterpret_cast<const uint4*>(sx + row * (C1 * 2) + ((lc ^ (row & 7)) * 16));
  }
}

// Wider blocks (C3 = 512: ResNet-50's second stage) do not fit W3, the
// tile's y3 rows and W1 side by side in LDS.  Here the first layer's
// output channels are taken in chunks of 128: per chunk its W3 rows (all of
// K, 32 KB) and residual columns come in, the chunk's y3 columns are
// finished in place and stored, W1's matching 128 K columns (requested
// with the rest) take the place of W3, and the second contraction adds that
// K range to its sums: one round of requests per chunk.  The second layer
// runs over K in chunk order, 16 at a time, as the single layer does, so
// the bits are again those of the two layers run one by one.  The tile's x
// rows (both K steps) stay in LDS for all chunks.  LDS 69 KB: two
// workgroups per CU.
//   wave (wl & 3, wl >> 2) = 32 channels x 32 pixels, in both contractions
template <int C3, int C1, int K3, int ACT3, int ACT1, bool RES>
__global__ __launch_bounds__(kThr) __attribute__((amdgpu_waves_per_eu(4))) void conv_pair_chunked_kernel(PairP p) {
  constexpr int CW = 128;                     // y3 channels per chunk
  constexpr int NCH = C3 / CW;
  constexpr int XROW = K3 * 2;                // bytes of an x row (all K steps)
  constexpr int X_BYTES = kRowsT * XROW;
  constexpr int WROW = 256;                   // bytes of a W3 chunk row (K3 = 128) and of a W1 chunk row (CW = 128)
  constexpr int W_BYTES = 128 * WROW;         // 128 rows: CW rows of W3, or the C1 rows of W1
  constexpr int AROW = CW * 2;                // bytes of a y3 chunk row
  constexpr int A_BYTES = kRowsT * AROW;
  constexpr int NV = 2 * C3 + 2 * C1;         // [s3 | b3 | s1 | b1]
  static_assert(C3 % CW == 0 && C1 == 128 && K3 == 128, "laid out for 128 -> 512 -> 128 channels");
  static_assert(XROW == WROW && AROW == WROW, "all LDS rows 256 bytes: 16 chunks, swizzled by row & 15");
  static_assert(kRowsT * C1 * 2 <= X_BYTES, "the y1 staging takes the place of x");
  static_assert(NV / 4 <= kThr, "one vector load per thread at most");
  constexpr int JX = X_BYTES / 16 / kThr, JW = W_BYTES / 16 / kThr, JA = A_BYTES / 16 / kThr;
  static_assert(JW == 4, "four W1 vectors per thread");
  __shared__ __align__(16) char smem[X_BYTES + W_BYTES + A_BYTES + NV * 4];
  char* const sx = smem;                              // x rows, then the y1 staging
  char* const sw = smem + X_BYTES;                    // a W3 chunk, then a W1 chunk
  char* const sa = smem + X_BYTES + W_BYTES;          // a residual chunk, then a y3 chunk
  float* const sv = reinterpret_cast<float*>(smem + X_BYTES + W_BYTES + A_BYTES);

  const int HW = p.H * p.W;
  const int M = (p.nc ? min(*p.nc, p.nmax) : p.nmax) * HW;
  const int T = (M + kRowsT - 1) / kRowsT;
  const int wg = blockIdx.x;
  if (wg >= T) return;
  const int T8 = (T >> 3) << 3;
  const int t = wg < T8 ? (wg & 7) * (T8 >> 3) + (p.rev ? (T8 >> 3) - 1 - (wg >> 3) : (wg >> 3)) : wg;
  const int m0 = t * kRowsT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // slot q of a region of 256-byte rows: row q / 16, physical chunk q % 16
  // holding logical chunk (q % 16) ^ (row & 15)
  auto lchunk = [](int q) { return (q & 15) ^ ((q >> 4) & 15); };
  if (tid < NV / 4) {
    const int q = tid * 4;
    const float* g = q < C3 ? p.v3[0] + q : q < 2 * C3 ? p.v3[1] + (q - C3) : q < 2 * C3 + C1 ? p.sc1 + (q - 2 * C3)
                                                                                             : p.sh1 + (q - 2 * C3 - C1);
    to_lds(g, reinterpret_cast<char*>(sv) + wave * 1024);
  }
#pragma unroll
  for (int j = 0; j < JX; ++j) {
    const int q = j * kThr + tid, m = m0 + (q >> 4);
    to_lds(m < M ? p.x + static_cast<size_t>(m) * K3 + lchunk(q) * 8 : p.zeros, sx + (j * kThr + wave * 64) * 16);
  }

  const int wc = wave & 3, wp = wave >> 2;
  const int lsw = lane & 15;
  f32x16 acc1;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc1[r] = 0.f;
  // 16 MFMA steps of K = 16 over 256-byte rows: A rows at pa, B rows at pb
  auto mma16 = [&](f32x16& acc, const char* pa, const char* pb) __attribute__((always_inline)) {
    bf16x8 af[2], bx[2];
    auto fetch = [&](int s, int slot) __attribute__((always_inline)) {
      const int phys = ((2 * s + (lane >> 5)) ^ lsw) * 16;
      af[slot] = *reinterpret_cast<const bf16x8*>(pa + phys);
      bx[slot] = *reinterpret_cast<const bf16x8*>(pb + phys);
    };
    fetch(0, 0);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if (s + 1 < 8) fetch(s + 1, (s + 1) & 1);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1], bx[s & 1], acc, 0, 0, 0);
    }
  };

  for (int c = 0; c < NCH; ++c) {
    if (c) lds_sync();   // the previous chunk's W1 and y3 are no longer read
    // W3 rows c CW .. + CW (all of K) and the residual's chunk columns
#pragma unroll
    for (int j = 0; j < JW; ++j) {
      const int q = j * kThr + tid;
      to_lds(p.w3 + static_cast<size_t>(c * CW + (q >> 4)) * p.Kp3 + lchunk(q) * 8, sw + (j * kThr + wave * 64) * 16);
    }
    if (RES) {
#pragma unroll
      for (int j = 0; j < JA; ++j) {
        const int q = j * kThr + tid, m = m0 + (q >> 4);
        to_lds(m < M ? p.res + static_cast<size_t>(m) * C3 + c * CW + lchunk(q) * 8 : p.zeros,
               sa + (j * kThr + wave * 64) * 16);
      }
    }
    // W1 columns c CW .. + CW of all C1 rows into registers (they go to the
    // space of W3 after the epilogue), requested and awaited with the rest:
    // with direct-to-LDS loads and register loads in flight, the compiler
    // waits for all of them before any LDS read anyway
    auto w1_at = [&](int j) __attribute__((always_inline)) {
      const int q = j * kThr + tid;
      return *reinterpret_cast<const uint4*>(p.w1 + static_cast<size_t>(q >> 4) * p.Kp1 + c * CW + lchunk(q) * 8);
    };
    const uint4 w1a = w1_at(0), w1b = w1_at(1), w1c = w1_at(2), w1d = w1_at(3);
    vm_barrier<0>();
    f32x16 acc3;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc3[r] = 0.f;
    mma16(acc3, sw + (32 * wc + (lane & 31)) * WROW, sx + (32 * wp + (lane & 31)) * XROW);
    lds_sync();   // every wave is done reading W3
    {
      const int row = 32 * wp + (lane & 31);
      char* const arow = sa + row * AROW + (lane >> 5) * 8;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int cl = 32 * wc + 8 * g + 4 * (lane >> 5), c0 = c * CW + cl;
        uint2* const e = reinterpret_cast<uint2*>(arow + (((cl >> 3) ^ (row & 15)) * 16));
        const float4 sc = *reinterpret_cast<const float4*>(sv + c0);
        const float4 sh = *reinterpret_cast<const float4*>(sv + C3 + c0);
        float v0 = fmaf(acc3[4 * g + 0], sc.x, sh.x);
        float v1 = fmaf(acc3[4 * g + 1], sc.y, sh.y);
        float v2 = fmaf(acc3[4 * g + 2], sc.z, sh.z);
        float v3 = fmaf(acc3[4 * g + 3], sc.w, sh.w);
        if (RES) {
          const uint2 r = *e;
          v0 += __uint_as_float(r.x << 16);
          v1 += __uint_as_float(r.x & 0xffff0000u);
          v2 += __uint_as_float(r.y << 16);
          v3 += __uint_as_float(r.y & 0xffff0000u);
        }
        *e = make_uint2(pack2(act_of<ACT3>(v0), act_of<ACT3>(v1)), pack2(act_of<ACT3>(v2), act_of<ACT3>(v3)));
      }
    }
    auto w1_put = [&](int j, const uint4& v) __attribute__((always_inline)) {
      const int q = j * kThr + tid;
      *reinterpret_cast<uint4*>(sw + q * 16) = v;   // slot q: row q / 16, physical chunk q % 16
    };
    w1_put(0, w1a);
    w1_put(1, w1b);
    w1_put(2, w1c);
    w1_put(3, w1d);
    lds_sync();   // the chunk's y3 columns and W1 columns are complete
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int q = j * kThr + tid, row = q >> 4, lc = lchunk(q);
      if (m0 + row < M)
        *reinterpret_cast<uint4*>(p.y3 + static_cast<size_t>(m0 + row) * C3 + c * CW + lc * 8) =
            *reinterpret_cast<const uint4*>(sa + q * 16);
    }
    mma16(acc1, sw + (32 * wc + (lane & 31)) * WROW, sa + (32 * wp + (lane & 31)) * AROW);
  }
  lds_sync();   // x is no longer read: its space takes the y1 staging
  {
    const int px = 32 * wp + (lane & 31);
    char* const yrow = sx + px * (C1 * 2) + (lane >> 5) * 8;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c0 = 32 * wc + 8 * g + 4 * (lane >> 5);
      const float4 sc = *reinterpret_cast<const float4*>(sv + 2 * C3 + c0);
      const float4 sh = *reinterpret_cast<const float4*>(sv + 2 * C3 + C1 + c0);
      const float v0 = act_of<ACT1>(fmaf(acc1[4 * g + 0], sc.x, sh.x));
      const float v1 = act_of<ACT1>(fmaf(acc1[4 * g + 1], sc.y, sh.y));
      const float v2 = act_of<ACT1>(fmaf(acc1[4 * g + 2], sc.z, sh.z));
      const float v3 = act_of<ACT1>(fmaf(acc1[4 * g + 3], sc.w, sh.w));
      *reinterpret_cast<uint2*>(yrow + (((c0 >> 3) ^ (px & 15)) * 16)) = make_uint2(pack2(v0, v1), pack2(v2, v3));
    }
  }
  lds_sync();
#pragma unroll
  for (int j = 0; j < kRowsT * C1 * 2 / 16 / kThr; ++j) {
    const int q = j * kThr + tid, row = q >> 4;
    if (m0 + row < M)
      *reinterpret_cast<uint4*>(p.y1 + static_cast<size_t>(m0 + row) * C1 + lchunk(q) * 8) =
          *reinterpret_cast<const uint4*>(sx + q * 16);
  }
}

bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; }

}  // namespace

bool conv_pair_fits(int K3, int K2, int C3, int C1, int act3, int act1) {
  if (act3 != ACT_RELU || act1 != ACT_RELU) return false;
  if (C3 == 512) return C1 == 128 && K3 == 128 && K2 == 0;   // the chunked kernel: no fold
  return C3 == 256 && C1 == 64 && K3 >= 64 && K3 % 64 == 0 && K2 >= 0 && K2 % 64 == 0 && K3 + K2 <= 1024;
}

bool conv_pair_takes(const PairArgs& a) {
  const bool fold = a.x2 != nullptr;
  if (!conv_pair_fits(a.K3, fold ? a.K2 : 0, a.C3, a.C1, a.act3, a.act1)) return false;
  if (a.n <= 0 || a.H <= 0 || a.W <= 0 || !a.x || !a.w3 || !a.y3 || !a.w1 || !a.y1 || !a.zeros || !a.scale3 ||
      !a.shift3 || !a.scale1 || !a.shift1)
    return false;
  // a fold and a residual never come together (the fold is the residual)
  if (fold && (a.res || a.K2 <= 0 || !a.fold_sp || !a.fold_bp || !a.fold_inv || a.H2 <= 0 || a.W2 <= 0 ||
               a.s2 <= 0 || (a.H - 1) * a.s2 >= a.H2 || (a.W - 1) * a.s2 >= a.W2))
    return false;
  const void* ptrs[] = {a.x, a.x2, a.w3, a.res, a.y3, a.w1, a.y1, a.scale3, a.shift3, a.scale1, a.shift1,
                        a.fold_sp, a.fold_bp, a.fold_inv};
  for (const void* q : ptrs)
    if (!aligned16(q)) return false;
  if (a.Kp3 < a.K3 + (fold ? a.K2 : 0) || a.Kp3 % 64 || a.Kp1 < a.C3 || a.Kp1 % 8) return false;
  return static_cast<long>(a.n) * a.H * a.W <= 0x7fffffffL - kRowsT;
}

bool conv_pair(const PairArgs& a, hipStream_t s) {
  if (!conv_pair_takes(a)) return false;
  const bool fold = a.x2 != nullptr;
  const long M = static_cast<long>(a.n) * a.H * a.W;
  PairP p;
  p.x = a.x;
  p.x2 = fold ? a.x2 : nullptr;
  p.w3 = a.w3;
  p.v3[0] = a.scale3;
  p.v3[1] = a.shift3;
  p.v3[2] = a.fold_sp;
  p.v3[3] = a.fold_bp;
  p.v3[4] = a.fold_inv;
  p.res = a.res;
  p.y3 = a.y3;
  p.w1 = a.w1;
  p.sc1 = a.scale1;
  p.sh1 = a.shift1;
  p.y1 = a.y1;
  p.zeros = a.zeros;
  p.nc = a.ncount;
  p.nmax = a.n;
  p.H = a.H;
  p.W = a.W;
  p.cin1 = a.K3;
  p.cin2 = fold ? a.K2 : 0;
  p.H2 = a.H2;
  p.W2 = a.W2;
  p.s2 = a.s2;
  p.Kp3 = a.Kp3;
  p.Kp1 = a.Kp1;
  p.rev = a.rev;
  const dim3 grid(static_cast<unsigned>((M + kRowsT - 1) / kRowsT));
  if (a.C3 == 512 && a.res)
    hipLaunchKernelGGL((conv_pair_chunked_kernel<512, 128, 128, ACT_RELU, ACT_RELU, true>), grid, dim3(kThr), 0, s, p);
  else if (a.C3 == 512)
    hipLaunchKernelGGL((conv_pair_chunked_kernel<512, 128, 128, ACT_RELU, ACT_RELU, false>), grid, dim3(kThr), 0, s, p);
  else if (fold)
    hipLaunchKernelGGL((conv_pair_kernel<256, 64, ACT_RELU, ACT_RELU, false, true>), grid, dim3(kThr), 0, s, p);
  else if (a.res)
    hipLaunchKernelGGL((conv_pair_kernel<256, 64, ACT_RELU, ACT_RELU, true, false>), grid, dim3(kThr), 0, s, p);
  else
    hipLaunchKernelGGL((conv_pair_kernel<256, 64, ACT_RELU, ACT_RELU, false, false>), grid, dim3(kThr), 0, s, p);
  return true;
}

}  // namespace k
}  // namespace dycl
