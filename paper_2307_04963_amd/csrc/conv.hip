// bf16 implicit-GEMM convolution / linear layer for gfx950 (CDNA4).
//
// A sub-network of the compiled dynamic network is conditional-free tensor
// code (Sec. 5.3); its convolutions and linear layers are dense
// contractions:
//   y[m, co] = sum_{kh, kw, ci} x[img, oh*s - p + kh, ow*s - p + kw, ci] * w[co, kh, kw, ci]
// with m = (img, oh, ow) running over the rows active in this branch.
// As a GEMM: M = rows * Ho * Wo, N = Cout, K = kh * kw * Cin.  NHWC keeps
// the Cin run of one tap contiguous, so A is gathered in 16-byte vectors
// straight from the activation tensor (no im2col buffer).
//
// Workgroup: 64*WM*WN threads computing a BM x BN tile; wave (wm, wn)
// accumulates a (BM/WM) x (BN/WN) block with v_mfma_f32_32x32x16_bf16
// (fp32 accumulate).  K advances 64 per step: the next step's A/B vectors
// are loaded into registers while the current step's MFMAs run from LDS
// (rows padded by 16 bytes: the lanes of each ds_read_b128 phase hit
// distinct banks).  LDS use (<= 55 KB) and registers leave room for two
// workgroups per CU, whose barrier phases interleave.
//
// Tiles are visited in an XCD-aware order: the dispatcher deals workgroups
// round-robin over the 8 XCDs, so consecutive tile indices (the N tiles of
// one M tile, which share their A rows) are given to workgroups of the same
// XCD and its L2.
//
// Epilogue: folded BatchNorm scale/shift (or bias), residual, ReLU or exact
// GELU, then round-to-nearest-even bf16 or an fp32 store.
#include <stdexcept>
#include <type_traits>

#include "kernels.hpp"

namespace dycl {
namespace k {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct ConvP {
  const uint16_t* src;
  const uint16_t* src2;
  int cin1, cin2;
  int H, W, cin, Ho, Wo, cout, stride, pad;
  int M, K, Kp, cin_log2;
  int mt, nt;
  const int32_t* nc;       // device count of live images (<= nmax) or null
  int nmax;                // images the grid is sized for
  // fused gathers / scatters: image i of the layer reads input image
  // srows[i] and residual image rrows[i] and writes output image drows[i]
  // (null: i)
  const int32_t* srows;
  const int32_t* s2rows;   // image list of src2 (the concatenated input)
  int H2, W2, s2;          // src2: spatial shape and the stride it is read at
  const int32_t* rrows;
  const int32_t* drows;
  // a folded projection (conv_lds_kernel, no K split): its kfold K steps
  // (the last ones of the packed layout) run first; then every sum becomes
  // bf16(fsp * acc + fbp) * finv, the rounded projection output in the
  // units of the block's own sum, which the remaining steps add to
  const float* cell_in;    // ACT_LSTM: old cell state [rows][cout / 4] (through rrows), or null
  float* cell_out;         // ACT_LSTM: new cell state [rows][cout / 4] (through drows)
  int kfold;
  const float* fsp;
  const float* fbp;
  const float* finv;
  int ksplit;              // K ranges per tile (conv_lds_kernel); > 1: fp32 partials to `part`
  float* part;             // [ksplit][M][cout] partial sums (rows of the nmax images)
  const uint16_t* w;
  const float* scale;
  const float* shift;
  const uint16_t* res;
  void* dst;
  int act, out_f32;
  const uint16_t* zeros;   // >= 16 zero bytes: the source of padding taps
  float* gap;              // conv_lds_kernel: 32-row chunk column sums of the bf16 output, or null
  int rev;                 // conv_lds_kernel: each XCD walks its tiles last to first
};

// round to nearest even (v_cvt_pk_bf16_f32; NaN stays NaN), as every
// kernel's epilogue
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// the element row (image * HoWo + pixel) that layer row `row` maps to
// through an image list (null: itself)
__device__ __forceinline__ size_t row_at(const int32_t* rows, int row, int HoWo) {
  if (!rows) return static_cast<size_t>(row);
  const int img = row / HoWo;
  return static_cast<size_t>(rows[img]) * HoWo + (row - img * HoWo);
}

template <int ACT>
__device__ __forceinline__ float act_t(float v) {
  if (ACT == ACT_RELU) return v > 0.f ? v : 0.f;
  if (ACT == ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  if (ACT == ACT_TANH) return tanhf(v);
  return v;
}

__device__ __forceinline__ float apply_act(float v, int act) {
  if (act == ACT_RELU) return v > 0.f ? v : 0.f;
  if (act == ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  if (act == ACT_TANH) return tanhf(v);
  return v;
}

__device__ __forceinline__ float sigmoidf(float v) { return 1.0f / (1.0f + expf(-v)); }

template <int BM, int BN, int WM, int WN, int KS, bool SCALAR, int BK = 64, int STAGES = 1>
__global__ __launch_bounds__(64 * WM* WN) void conv_kernel(ConvP p) {
  constexpr int NT = 64 * WM * WN;
  constexpr int LDK = BK + 8;
  constexpr int VPR = BK / 8;        // 16-byte vectors per tile row
  constexpr int RPP = NT / VPR;      // tile rows per load pass
  constexpr int PA = (BM + RPP - 1) / RPP;
  constexpr int PB = (BN + RPP - 1) / RPP;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be 32x32 blocks");

  __shared__ __align__(16) uint16_t As[STAGES][BM * LDK];
  __shared__ __align__(16) uint16_t Bs[STAGES][BN * LDK];

  // XCD-aware tile order (bijective on [0, mt*nt))
  // with a device count, only the tiles of the live images exist: the
  // grid was sized for nmax images and the surplus workgroups leave
  const int M = p.nc ? min(*p.nc, p.nmax) * p.Ho * p.Wo : p.M;
  const int T = (p.nc ? (M + BM - 1) / BM : p.mt) * p.nt;
  const int T8 = (T >> 3) << 3;
  const int wg = blockIdx.x;
  if (wg >= T) return;
  const int t = wg < T8 ? (wg & 7) * (T8 >> 3) + (wg >> 3) : wg;
  const int mtile = t / p.nt;
  const int m0 = mtile * BM, n0 = (t - mtile * p.nt) * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int chunk = tid % VPR, rsub = tid / VPR;
  const int HoWo = p.Ho * p.Wo;

  // per A row: pixel index of the window origin and its (ih0, iw0); rows
  // past M get an origin far outside the image, so every tap reads zero
  int a_pix[PA], a_pix2[PA], a_ih[PA], a_iw[PA];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int m = m0 + rsub + i * RPP;
    if (m < M) {
      const int img = m / HoWo;
      const int rem = m - img * HoWo;
      const int oh = rem / p.Wo, ow = rem - (rem / p.Wo) * p.Wo;
      const int simg = p.srows ? p.srows[img] : img;
      const int s2img = p.s2rows ? p.s2rows[img] : img;
      a_ih[i] = oh * p.stride - p.pad;
      a_iw[i] = ow * p.stride - p.pad;
      a_pix[i] = (simg * p.H + a_ih[i]) * p.W + a_iw[i];
      a_pix2[i] = (s2img * p.H2 + a_ih[i] * p.s2) * p.W2 + a_iw[i] * p.s2;
    } else {
      a_ih[i] = -0x4000;
      a_iw[i] = -0x4000;
      a_pix[i] = 0;
      a_pix2[i] = 0;
    }
  }

  uint4 ra[PA], rb[PB];
  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;


  auto load_tile = [&](int kt) __attribute__((always_inline)) {
    const int kidx = kt * BK + chunk * 8;
    if constexpr (!SCALAR) {
      int tap = 0, ci = kidx;
      if constexpr (KS != 1) {
        tap = kidx >> p.cin_log2;
        ci = kidx & (p.cin - 1);
      }
      const int kh = tap / KS, kw = tap - (tap / KS) * KS;
      const bool kok = kidx < p.K;
      const uint16_t* sp = p.src;
      int cs = p.cin1, co = ci;
      if (ci >= p.cin1) {
        sp = p.src2;
        cs = p.cin2;
        co = ci - p.cin1;
      }
      const int doff = kh * p.W + kw;
#pragma unroll
      for (int i = 0; i < PA; ++i) {
        uint4 v = make_uint4(0, 0, 0, 0);
        const int ih = a_ih[i] + kh, iw = a_iw[i] + kw;
        if (kok && (unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W && rsub + i * RPP < BM)
          v = *reinterpret_cast<const uint4*>(sp + (size_t)((ci >= p.cin1 ? a_pix2[i] : a_pix[i]) + doff) * cs + co);
        ra[i] = v;
      }
    } else {
#pragma unroll
      for (int i = 0; i < PA; ++i) {
        uint16_t e[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          e[j] = 0;
          const int kk = kidx + j;
          if (kk < p.K && rsub + i * RPP < BM) {
            const int tap = kk / p.cin;
            const int ci = kk - tap * p.cin;
            const int kh = tap / KS, kw = tap - (tap / KS) * KS;
            const int ih = a_ih[i] + kh, iw = a_iw[i] + kw;
            if ((unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W)
              e[j] = p.src[(size_t)(a_pix[i] + kh * p.W + kw) * p.cin + ci];
          }
        }
        ra[i].x = e[0] | (uint32_t(e[1]) << 16);
        ra[i].y = e[2] | (uint32_t(e[3]) << 16);
        ra[i].z = e[4] | (uint32_t(e[5]) << 16);
        ra[i].w = e[6] | (uint32_t(e[7]) << 16);
      }
    }
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      // written on every path: a register array assigned only under a
      // divergent branch is kept in scratch memory by the compiler
      const int row = rsub + i * RPP;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (BN % RPP == 0 || row < BN) v = *reinterpret_cast<const uint4*>(p.w + (size_t)(n0 + row) * p.Kp + kidx);
      rb[i] = v;
    }
  };

  auto store_tile = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < PA; ++i) {
      const int row = rsub + i * RPP;
      if (row < BM) *reinterpret_cast<uint4*>(&As[buf][row * LDK + chunk * 8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      const int row = rsub + i * RPP;
      if (row < BN) *reinterpret_cast<uint4*>(&Bs[buf][row * LDK + chunk * 8]) = rb[i];
    }
  };

  auto compute = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      bf16x8 af[TM], bfr[TN];
      const int koff = s * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = *reinterpret_cast<const bf16x8*>(&As[buf][(wm * WTM + a * 32 + (lane & 31)) * LDK + koff]);
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bfr[b] = *reinterpret_cast<const bf16x8*>(&Bs[buf][(wn * WTN + b * 32 + (lane & 31)) * LDK + koff]);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
  };

  const int nk = p.Kp / BK;
  load_tile(0);
  if constexpr (STAGES == 1) {
    // one LDS buffer: store, barrier, prefetch the next step, compute, barrier
    for (int kt = 0; kt < nk; ++kt) {
      if (kt > 0) __syncthreads();    // every wave is done reading the previous step
      store_tile(0);
      __syncthreads();
      if (kt + 1 < nk) load_tile(kt + 1);
      compute(0);
    }
  } else {
    // two LDS buffers: one barrier per step
    store_tile(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) load_tile(kt + 1);
      compute(kt & 1);
      if (kt + 1 < nk) store_tile((kt + 1) & 1);
      __syncthreads();
    }
  }

  // epilogue: lane owns column (lane & 31) of each 32x32 block, rows
  // 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
  for (int b = 0; b < TN; ++b) {
    const int col = n0 + wn * WTN + b * 32 + (lane & 31);
    if (col >= p.cout) continue;
    const float sc = p.scale ? p.scale[col] : 1.0f;
    const float sh = p.shift ? p.shift[col] : 0.0f;
#pragma unroll
    for (int a = 0; a < TM; ++a) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * WTM + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row >= M) continue;
        const size_t o = row_at(p.drows, row, HoWo) * p.cout + col;
        float v = fmaf(acc[a][b][r], sc, sh);
        if (p.res) v += bf2f(p.res[row_at(p.rrows, row, HoWo) * p.cout + col]);
        v = apply_act(v, p.act);
        if (p.out_f32)
          static_cast<float*>(p.dst)[o] = v;
        else
          static_cast<uint16_t*>(p.dst)[o] = f2bf(v);
      }
    }
  }
}


// ------------------------------------------------- direct-to-LDS kernel ----
// Same contraction, with gfx950's global_load_lds_dwordx4: each lane's 16
// bytes go straight from global memory to LDS at (wave base + 16 * lane), so
// tiles need no staging registers and no ds_write.  The LDS row of a tile is
// 128 bytes (64 bf16 of K); its eight 16-byte chunks are stored XOR-swizzled
// (physical chunk = logical ^ ((row >> 1) & 7)), which makes the 16 lanes of
// every ds_read_b128 phase of the MFMA operand reads hit 16 distinct bank
// groups.  The swizzle is applied on the global side: each lane picks the
// global chunk that belongs at its fixed LDS slot.  Padding taps and rows
// past M read a zero buffer.  Two LDS stages, one barrier per K step: the
// loads of step k+1 are in flight while step k's MFMAs run.
typedef __attribute__((address_space(3))) void* lds_void_ptr;

// Wait until at most N vector-memory operations of this thread are still in
// flight (loads complete in order, so every older one - the tile about to be
// read - has landed), then barrier.  Inline asm with a memory clobber keeps
// the compiler from moving LDS reads across it and from widening the wait.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// One K step (NS 1) is the memory-bound 1x1 case, whose speed follows the
// number of workgroups in flight: its registers are capped for five waves
// per SIMD (128 x 64 tiles: 85 VGPRs, the accumulators out of AGPRs, no
// spill), where unconstrained it takes 85 + 32 AGPRs and runs four; a cap
// for six spills.
template <int BM, int BN, int WM, int WN, int KS, int NS = 2>
__global__ __launch_bounds__(64 * WM* WN) __attribute__((amdgpu_waves_per_eu(NS == 1 ? 5 : 1))) void conv_lds_kernel(
    ConvP p) {
  constexpr int NT = 64 * WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * 128, B_BYTES = BN * 128, STAGE = A_BYTES + B_BYTES;
  constexpr int JA = BM * 8 / NT, JB = BN * 8 / NT;
  constexpr int EPW = WTN + 4;                        // epilogue row stride (floats)
  constexpr int EPI = (NT / 64) * 32 * EPW * 4;
  constexpr int SMEM = NS * STAGE > EPI ? NS * STAGE : EPI;
  static_assert(NS >= 1 && NS <= 4, "1 to 4 LDS stages (1: a single K step only)");
  static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0 && JB >= 1, "tile rows must fill whole load passes");
  static_assert(NT % 128 == 0, "swizzle assumes NT a multiple of 128");
  static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be 32x32 blocks");

  __shared__ __align__(16) char smem[SMEM];

  // with a device count, only the tiles of the live images exist: the
  // grid was sized for nmax images and the surplus workgroups leave.  With
  // a K split, workgroup wg takes K range wg / T of tile wg % T.
  const int M = p.nc ? min(*p.nc, p.nmax) * p.Ho * p.Wo : p.M;
  const int T = (p.nc ? (M + BM - 1) / BM : p.mt) * p.nt;
  const int T8 = (T >> 3) << 3;
  if (static_cast<int>(blockIdx.x) >= T * p.ksplit) return;
  const int split = blockIdx.x / T;
  const int wg = blockIdx.x - split * T;
  const int t = wg < T8 ? (wg & 7) * (T8 >> 3) + (p.rev ? (T8 >> 3) - 1 - (wg >> 3) : (wg >> 3)) : wg;
  const int mtile = t / p.nt;
  const int m0 = mtile * BM, n0 = (t - mtile * p.nt) * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lchunk = (tid & 7) ^ ((tid >> 4) & 7);   // logical K chunk this thread loads
  const int rbase = tid >> 3;                        // + j * NT / 8
  const int HoWo = p.Ho * p.Wo;

  int a_pix[JA], a_pix2[JA], a_ih[JA], a_iw[JA];
#pragma unroll
  for (int j = 0; j < JA; ++j) {
    const int m = m0 + rbase + j * (NT / 8);
    if (m < M) {
      const int img = m / HoWo;
      const int rem = m - img * HoWo;
      const int oh = rem / p.Wo, ow = rem - (rem / p.Wo) * p.Wo;
      const int simg = p.srows ? p.srows[img] : img;
      const int s2img = p.s2rows ? p.s2rows[img] : img;
      a_ih[j] = oh * p.stride - p.pad;
      a_iw[j] = ow * p.stride - p.pad;
      a_pix[j] = (simg * p.H + a_ih[j]) * p.W + a_iw[j];
      a_pix2[j] = (s2img * p.H2 + a_ih[j] * p.s2) * p.W2 + a_iw[j] * p.s2;
    } else {
      a_ih[j] = -0x4000;
      a_iw[j] = -0x4000;
      a_pix[j] = 0;
      a_pix2[j] = 0;
    }
  }
  const uint16_t* wrow = p.w + (size_t)(n0 + rbase) * p.Kp + lchunk * 8;

  // this workgroup's K steps: [kb, kb + nk) of the layer's Kp / 64
  const int nk_all = p.Kp / 64;
  const int kb = split * nk_all / p.ksplit;
  const int nk = (split + 1) * nk_all / p.ksplit - kb;

  auto issue = [&](int kt, int stage) __attribute__((always_inline)) {
    char* sb = smem + stage * STAGE;
    kt += kb;
    // a folded projection's steps (the last kfold of the layout) come first
    if (p.kfold) kt = kt < p.kfold ? kt + (nk_all - p.kfold) : kt - p.kfold;
    const int kidx = kt * 64 + lchunk * 8;
    int tap = 0, ci = kidx;
    if constexpr (KS != 1) {
      tap = kidx >> p.cin_log2;
      ci = kidx & (p.cin - 1);
    }
    const int kh = tap / KS, kw = tap - (tap / KS) * KS;
    const bool kok = kidx < p.K;
    const uint16_t* sp = p.src;
    int cs = p.cin1, co = ci;
    if (ci >= p.cin1) {
      sp = p.src2;
      cs = p.cin2;
      co = ci - p.cin1;
    }
    const int doff = kh * p.W + kw;
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int ih = a_ih[j] + kh, iw = a_iw[j] + kw;
      const bool ok = kok && (unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W;
      const uint16_t* g = ok ? sp + (size_t)((ci >= p.cin1 ? a_pix2[j] : a_pix[j]) + doff) * cs + co : p.zeros;
      __builtin_amdgcn_global_load_lds((const void*)g, (lds_void_ptr)(sb + (j * NT + wave * 64) * 16), 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const uint16_t* g = wrow + (size_t)j * (NT / 8) * p.Kp + kt * 64;
      __builtin_amdgcn_global_load_lds((const void*)g, (lds_void_ptr)(sb + A_BYTES + (j * NT + wave * 64) * 16), 16,
                                       0, 0);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const int lsw = (lane >> 1) & 7;
  // operands of K sub-step s+1 are read from LDS while sub-step s's MFMAs run
  auto compute = [&](int stage) __attribute__((always_inline)) {
    const char* sa = smem + stage * STAGE + (wm * WTM + (lane & 31)) * 128;
    const char* sbp = smem + stage * STAGE + A_BYTES + (wn * WTN + (lane & 31)) * 128;
    bf16x8 af[2][TM], bfr[2][TN];
    auto fetch = [&](int s, int slot) __attribute__((always_inline)) {
      const int phys = ((2 * s + (lane >> 5)) ^ lsw) * 16;
#pragma unroll
      for (int a = 0; a < TM; ++a) af[slot][a] = *reinterpret_cast<const bf16x8*>(sa + a * 32 * 128 + phys);
#pragma unroll
      for (int b = 0; b < TN; ++b) bfr[slot][b] = *reinterpret_cast<const bf16x8*>(sbp + b * 32 * 128 + phys);
    };
    fetch(0, 0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s + 1 < 4) fetch(s + 1, (s + 1) & 1);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1][a], bfr[s & 1][b], acc[a][b], 0, 0, 0);
    }
  };

  // a folded projection: once its K steps are summed, each sum becomes the
  // projection's output as the unfused layer stores it (scale, shift, bf16
  // rounding), divided by the block's scale, so the block's own steps add
  // to it and the epilogue's scale / shift finish the residual sum
  float fsp[TN], fbp[TN], finv[TN];
  {
    if (p.kfold) {
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int col = n0 + wn * WTN + b * 32 + (lane & 31);
        const bool in = col < p.cout;
        fsp[b] = in ? p.fsp[col] : 0.f;
        fbp[b] = in ? p.fbp[col] : 0.f;
        finv[b] = in ? p.finv[col] : 0.f;
      }
    }
  }
  auto fold_round = [&]() __attribute__((always_inline)) {
    {
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            acc[a][b][r] = bf2f(f2bf(fmaf(acc[a][b][r], fsp[b], fbp[b]))) * finv[b];
    }
  };

  const bool partial = p.ksplit > 1;   // raw sums; the split reduction finishes them
  // residual vectors of the rows and 8-channel groups this lane finishes in
  // the epilogue (below)
  constexpr int G = WTN / 8;           // 8-channel groups per row
  constexpr int VI = 32 * G / 64;      // groups per lane in a 32-row block
  uint4 rv[TM][VI];
  auto load_res = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int v = 0; v < VI; ++v) {
        const int idx = v * 64 + lane;
        const int rl = idx / G, g = idx - (idx / G) * G;
        const int row = m0 + wm * WTM + a * 32 + rl;
        const int col = n0 + wn * WTN + g * 8;
        rv[a][v] = (row < M && col < p.cout)
                       ? *reinterpret_cast<const uint4*>(p.res + row_at(p.rrows, row, HoWo) * p.cout + col)
                       : make_uint4(0, 0, 0, 0);
      }
  };

  // NS-stage pipeline: the loads of step kt+NS-1 are issued while step kt
  // is computed; the stage they fill was read in step kt-1, which every wave
  // finished before the barrier of step kt
#pragma unroll
  for (int i = 0; i < NS - 1; ++i)
    if (i < nk) issue(i, i);
  if constexpr (NS == 1) {
    // one stage, the K steps one after another (one step, or a few on a
    // memory-bound layer): a small LDS footprint, more workgroups per CU,
    // whose number (not the bytes in flight per workgroup) sets the speed
    // of these layers
    for (int kt = 0; kt < nk; ++kt) {
      if (kt) __syncthreads();   // every wave is done reading the stage
      issue(kt, 0);
      wait_vm_barrier<0>();
      compute(0);
      if (kt + 1 == p.kfold) fold_round();
    }
  } else if (NS == 2) {
    // rounds of two K steps requested together: the second step's latency
    // overlaps the first's, and a layer of nk steps waits on ceil(nk / 2)
    // round trips (measured 5-25 % faster than keeping one step in flight
    // behind the MFMAs, on every layer shape tried, and ahead of four
    // pipelined stages on 64 x 64 tiles)
    for (int kt = 0; kt < nk; kt += 2) {
      if (kt) {
        __syncthreads();   // every wave is done reading both stages
        issue(kt, 0);
      }
      if (kt + 1 < nk) {
        issue(kt + 1, 1);
        wait_vm_barrier<JA + JB>();   // step kt has landed; kt + 1 may be in flight
      } else {
        wait_vm_barrier<0>();
      }
      compute(0);
      if (kt + 1 == p.kfold) fold_round();
      if (kt + 1 < nk) {
        wait_vm_barrier<0>();
        compute(1);
        if (kt + 2 == p.kfold) fold_round();
      }
    }
  } else {
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + NS - 2 < nk)
        wait_vm_barrier<(NS - 2) * (JA + JB)>();   // steps kt+1 .. kt+NS-2 may stay in flight
      else
        wait_vm_barrier<0>();
      if (kt + NS - 1 < nk) issue(kt + NS - 1, (kt + NS - 1) % NS);
      compute(kt % NS);
      if (kt + 1 == p.kfold) fold_round();
    }
  }

  // epilogue through LDS: each wave stages 32 x WTN fp32 values (scale and
  // shift applied) in its own region, then every lane finishes 8
  // consecutive channels of a row (residual, activation, rounding) and
  // writes them with one 16-byte store.  The residual vectors of all the
  // wave's rows are requested first, so their latency overlaps the staging.
  __syncthreads();   // the main loop's last tiles are no longer read
  float* ep = reinterpret_cast<float*>(smem) + wave * 32 * EPW;
  float sc[TN], sh[TN];
#pragma unroll
  for (int b = 0; b < TN; ++b) {
    const int col = n0 + wn * WTN + b * 32 + (lane & 31);
    sc[b] = (!partial && p.scale && col < p.cout) ? p.scale[col] : 1.0f;
    sh[b] = (!partial && p.shift && col < p.cout) ? p.shift[col] : 0.0f;
  }
  if (p.res && !partial) load_res();
  // the activation is chosen once, outside the epilogue's loops
  auto epilogue = [&](auto act_c) __attribute__((always_inline)) {
    constexpr int ACT = decltype(act_c)::value;
#pragma unroll
    for (int a = 0; a < TM; ++a) {
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          ep[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * EPW + b * 32 + (lane & 31)] = fmaf(acc[a][b][r], sc[b], sh[b]);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's own staging region: in-order LDS
#pragma unroll
      for (int v = 0; v < VI; ++v) {
        const int idx = v * 64 + lane;
        const int rl = idx / G, g = idx - (idx / G) * G;
        const int row = m0 + wm * WTM + a * 32 + rl;
        const int col = n0 + wn * WTN + g * 8;
        if (row < M && col < p.cout) {
          const float4 lo = *reinterpret_cast<const float4*>(ep + rl * EPW + g * 8);
          const float4 hi = *reinterpret_cast<const float4*>(ep + rl * EPW + g * 8 + 4);
          float vv[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
          if (partial) {
            float* d = p.part + (size_t)split * p.M * p.cout + (size_t)row * p.cout + col;
            *reinterpret_cast<float4*>(d) = lo;
            *reinterpret_cast<float4*>(d + 4) = hi;
            continue;
          }
          if constexpr (ACT == ACT_LSTM) {
            // the 8 values are the gates of cells u and u + 1 (input,
            // forget, cell, output each); cell state float32, h bf16
            const int H = p.cout >> 2, u = col >> 2;
            float2 cp = make_float2(0.f, 0.f);
            if (p.cell_in) cp = *reinterpret_cast<const float2*>(p.cell_in + row_at(p.rrows, row, HoWo) * H + u);
            const float c0 = sigmoidf(vv[1]) * cp.x + sigmoidf(vv[0]) * tanhf(vv[2]);
            const float c1 = sigmoidf(vv[5]) * cp.y + sigmoidf(vv[4]) * tanhf(vv[6]);
            const float h0 = sigmoidf(vv[3]) * tanhf(c0), h1 = sigmoidf(vv[7]) * tanhf(c1);
            const size_t oc = row_at(p.drows, row, HoWo) * H + u;
            *reinterpret_cast<float2*>(p.cell_out + oc) = make_float2(c0, c1);
            *reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(p.dst) + oc) = pack_bf16(h0, h1);
            continue;
          }
          const size_t o = row_at(p.drows, row, HoWo) * p.cout + col;
          if (p.res) {
            const uint32_t rw[4] = {rv[a][v].x, rv[a][v].y, rv[a][v].z, rv[a][v].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              vv[2 * q] += __uint_as_float(rw[q] << 16);
              vv[2 * q + 1] += __uint_as_float(rw[q] & 0xffff0000u);
            }
          }
#pragma unroll
          for (int q = 0; q < 8; ++q) vv[q] = act_t<ACT>(vv[q]);
          if (p.out_f32) {
            float* d = static_cast<float*>(p.dst) + o;
            *reinterpret_cast<float4*>(d) = make_float4(vv[0], vv[1], vv[2], vv[3]);
            *reinterpret_cast<float4*>(d + 4) = make_float4(vv[4], vv[5], vv[6], vv[7]);
          } else {
            uint4 ov;
            ov.x = pack_bf16(vv[0], vv[1]);
            ov.y = pack_bf16(vv[2], vv[3]);
            ov.z = pack_bf16(vv[4], vv[5]);
            ov.w = pack_bf16(vv[6], vv[7]);
            *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p.dst) + o) = ov;
            if (p.gap) {
              // the stored values back into the staging rows, for the
              // chunk's column sums below
              const uint32_t ow[4] = {ov.x, ov.y, ov.z, ov.w};
              float* e8 = ep + rl * EPW + g * 8;
              *reinterpret_cast<float4*>(e8) = make_float4(__uint_as_float(ow[0] << 16), __uint_as_float(ow[0] & 0xffff0000u),
                                                           __uint_as_float(ow[1] << 16), __uint_as_float(ow[1] & 0xffff0000u));
              *reinterpret_cast<float4*>(e8 + 4) = make_float4(__uint_as_float(ow[2] << 16), __uint_as_float(ow[2] & 0xffff0000u),
                                                               __uint_as_float(ow[3] << 16), __uint_as_float(ow[3] & 0xffff0000u));
            }
          }
        }
      }
      if constexpr (ACT != ACT_LSTM) {
        const int row0 = m0 + wm * WTM + a * 32;   // a 32-row chunk of layer rows
        if (p.gap && !partial && row0 < M) {
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's own rows: in-order LDS
          // rows before `bnd` belong to the chunk's first image, the rest to
          // the next one (an image has at least 32 rows; rows past M land in
          // the second sum of the last image's chunk, which is never read)
          const int bnd = min(32, (row0 / HoWo + 1) * HoWo - row0);
#pragma unroll
          for (int c0 = 0; c0 < WTN; c0 += 64) {
            const int c = c0 + lane, col = n0 + wn * WTN + c;
            if (c < WTN && col < p.cout) {
              float t0 = 0.f, t1 = 0.f;
              if (bnd == 32) {
#pragma unroll 8
                for (int r = 0; r < 32; ++r) t0 += ep[r * EPW + c];
              } else {
                for (int r = 0; r < bnd; ++r) t0 += ep[r * EPW + c];
                for (int r = bnd; r < 32; ++r) t1 += ep[r * EPW + c];
              }
              float* q = p.gap + static_cast<size_t>(row0 / 32) * 2 * p.cout + col;
              q[0] = t0;
              if (bnd < 32) q[p.cout] = t1;   // read only for a chunk that crosses into the next image
            }
          }
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // reads done before the next block's staging
    }
  };
  if (p.act == ACT_RELU)
    epilogue(std::integral_constant<int, ACT_RELU>{});
  else if (p.act == ACT_GELU)
    epilogue(std::integral_constant<int, ACT_GELU>{});
  else if (p.act == ACT_TANH)
    epilogue(std::integral_constant<int, ACT_TANH>{});
  else if (p.act == ACT_LSTM)
    epilogue(std::integral_constant<int, ACT_LSTM>{});
  else
    epilogue(std::integral_constant<int, ACT_NONE>{});
}

// 16 bytes per lane from a raw buffer straight into LDS at `lds` + 16 * lane:
// the buffer spans `bytes` from `base`, and a load at or past its end (an
// offset of 2^31 or more included) writes zeros instead of reading memory.
__device__ __forceinline__ void buffer_load_lds16(const void* base, uint32_t bytes, uint32_t offset, lds_void_ptr lds) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, offset, 0, 0, 0);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16 bytes per lane to a raw buffer of `bytes` from `base`; a store at or
// past its end is dropped.
__device__ __forceinline__ void buffer_store16(void* base, uint32_t bytes, uint32_t offset, u32x4 v) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(base, 0, bytes, 0x00020000);
  __builtin_amdgcn_raw_buffer_store_b128(v, r, offset, 0, 0);
}

// --------------------------------- 3x3 conv, halo tiles, resident weights ----
// For 3x3 / stride 1 / pad 1 layers with 64 input and 64 output channels,
// and for stems with 8 (padded) input channels and 64 output channels.
// A persistent workgroup walks a contiguous range of 128 x 64 output tiles;
// a tile is R whole output rows of one image (or G whole images when an
// image is smaller than the tile).  The tile's input patch - its rows plus
// one halo row above and below, one zero column left and right - is staged
// in LDS once and the nine taps read shifted windows of it, so each input
// pixel crosses L2 -> LDS about (R + 2) / R times instead of nine.
//
// Eight waves in three roles, one barrier per tile:
//  * four compute waves (2 x 2 over the tile, 64 x 32 each) hold their
//    weights in registers for the whole kernel (36 B fragments per lane:
//    9 taps x 4 K sub-steps of one output column), run the 36 MFMA K steps
//    on the current patch and write the finished bf16 tile (scale / shift,
//    residual, activation, rounding) to an LDS staging buffer;
//  * two loader waves copy the next tile's patch and residual rows from
//    global memory straight into LDS and, before the barrier, wait for them;
//  * two store waves copy the previous tile's staging buffer to global
//    memory with 16-byte stores and never wait for them.
// The memory counter of gfx9 counts loads and stores together; with loads
// and stores in different waves, the one wait per tile covers loads issued
// a whole tile earlier and nothing else.
//
// Patch pixels are stored 144 bytes apart (eight 16-byte K chunks and one
// unused slot): the 16 lanes of a ds_read_b128 phase, 16 consecutive
// pixels, fall on 16 distinct bank groups, and a tap's window is a constant
// byte offset from the lane's base address.  With 8 input channels a pixel
// is one 16-byte K chunk (stored densely), a K sub-step of 16 spans two
// taps - tap 2s in lanes 0-31, 2s + 1 in lanes 32-63 - and nine taps take
// five sub-steps (the tenth tap's weights are zero).
struct Conv3P {
  const uint16_t* src;
  const uint16_t* w;      // [64][Kp] packed, K = tap * cin + ci (Kp = 576, or 128 for 8 channels)
  const float* scale;
  const float* shift;
  const uint16_t* res;
  uint16_t* dst;
  const uint16_t* zeros;
  int n, H, W, cout, act;
  int RS, segs, PW, NP;    // rows per patch segment, segments, patch width, patch pixels
  int tiles, tpi;          // tiles; tiles per image (row mode) or 0 (image mode)
  const int32_t* nc;       // device count of live images (<= n) or null
  // image mode only: image i of the layer is image srows[i] of src, rrows[i]
  // of res, drows[i] of dst (null: i); listed tensors are addressed from
  // their first byte, so their size stays below 2^31 bytes (host check)
  const int32_t* srows;
  const int32_t* rrows;
  const int32_t* drows;
};

constexpr int kW3Patch = 256;                      // patch pixels per buffer (= kHP)
constexpr int kW3RB = 128 * 128;                   // 16384 B: a tile of residual / output rows
// patch bytes per pixel and per buffer, by input channels
constexpr int w3_pxb(int cin) { return cin == 8 ? 16 : 144; }
constexpr int w3_pb(int cin) { return kW3Patch * w3_pxb(cin); }

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void all_barrier() { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int CIN, int ACT, bool RES>
__global__ __launch_bounds__(512) void conv3_wres_kernel(Conv3P p) {
  constexpr int NL = 128;                          // loader / store threads
  constexpr int PXB = w3_pxb(CIN), kW3PB = w3_pb(CIN);
  constexpr int SLOTS = PXB / 16;                  // 16-byte slots per patch pixel (9 or 1)
  constexpr int JP = kW3Patch * SLOTS / NL;        // patch loads per loader thread (18 or 2)
  constexpr int KP = CIN == 8 ? 128 : 576;         // packed row length
  constexpr int NS = CIN == 8 ? 5 : 36;            // K sub-steps of 16
  __shared__ __align__(16) char smem[2 * kW3PB + 4 * kW3RB + 512];
  char* const pbuf = smem;                         // [2][256 px][144 B]
  char* const rbuf = smem + 2 * kW3PB;             // [2][128 rows][128 B] residual
  char* const sbuf = rbuf + 2 * kW3RB;             // [2][128 rows][128 B] finished bf16 tile

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int HW = p.H * p.W;
  // with a device count the live tiles are dealt over the grid (sized for
  // n images); workgroups left without a tile leave
  const int n = p.nc ? min(*p.nc, p.n) : p.n;
  const int tiles = p.nc ? (p.tpi ? n * p.tpi : (n + p.segs - 1) / p.segs) : p.tiles;
  const int t_begin = static_cast<int>((static_cast<long>(tiles) * blockIdx.x) / gridDim.x);
  const int t_end = static_cast<int>((static_cast<long>(tiles) * (blockIdx.x + 1)) / gridDim.x);
  if (t_begin >= t_end) return;

  auto tile_geom = [&](int t, int& img, int& oh0, int& m0, int& lim) __attribute__((always_inline)) {
    if (p.tpi) {
      img = t / p.tpi;
      oh0 = (t - img * p.tpi) * p.RS;
      m0 = img * HW + oh0 * p.W;
      lim = min(p.RS, p.H - oh0) * p.W;
    } else {
      img = t * p.segs;
      oh0 = 0;
      m0 = img * HW;
      lim = min(p.segs, n - img) * HW;
    }
  };
  // 16-byte chunk position of (row, logical chunk) in a residual / staging
  // row of 128 bytes: XOR with (row >> 1) & 7, so that 16 consecutive rows
  // at one logical chunk fall on 16 distinct bank groups
  auto rsw = [](int row, int c) { return c ^ ((row >> 1) & 7); };

  const int wv = __builtin_amdgcn_readfirstlane(wave);   // the same, known wave-uniform
  if (wv >= 6) {
    // ---------------- store waves: tile t - 1 while tile t is computed ----
    // buffer stores: the tile's rows from m0, at most lim of them (stores
    // to later rows fall outside the buffer and are dropped)
    const int st = tid - 6 * 64;
    for (int t = t_begin; t <= t_end; ++t) {
      lds_barrier();
      if (t == t_begin) continue;
      int img, oh0, m0, lim;
      tile_geom(t - 1, img, oh0, m0, lim);
      const char* sb = sbuf + ((t - 1 - t_begin) & 1) * kW3RB;
      if (p.drows) {
        // listed output: a row's image through drows, offsets from dst's start
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int u = k * NL + st, row = u >> 3, pos = u & 7;
          const int sg = row / HW, px = row - sg * HW;
          const uint32_t o = row < lim ? static_cast<uint32_t>((p.drows[img + sg] * HW + px) * 128 + rsw(row, pos) * 16)
                                       : 0xC0000000u;
          const u32x4 v = *reinterpret_cast<const u32x4*>(sb + u * 16);
          buffer_store16(p.dst, 0x7fffffffu, o, v);
        }
        continue;
      }
      uint16_t* const dbase = p.dst + (size_t)m0 * 64;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int u = k * NL + st, row = u >> 3, pos = u & 7;
        const u32x4 v = *reinterpret_cast<const u32x4*>(sb + u * 16);
        buffer_store16(dbase, static_cast<uint32_t>(lim) * 128, row * 128 + rsw(row, pos) * 16, v);
      }
    }
    return;
  }

  if (wv >= 4) {
    // ---------------- loader waves: tile t + 1 while tile t is computed ----
    // Buffer loads straight into LDS.  The patch's buffer spans the tile's
    // image(s); a slot's byte offset is relative to the tile's first output
    // row (row mode: plus oh0 rows, so the halo row above image row 0 wraps
    // to a huge offset and rows past the image exceed the buffer), and
    // slots that never hold data (zero columns, the unused ninth slot, past
    // the patch, image-mode halo rows) get an offset above 2^31: all read as
    // zeros, the convolution's padding.
    const int ld = tid - 4 * 64, lw = wv - 4;
    const int rowb = p.W * CIN * 2, imgb = p.H * rowb;
    uint32_t vofs[JP];
    // listed input (image mode): a slot's segment and its offset inside the
    // image (vseg -1: a slot that never holds data); the row ids of a tile's
    // segments are requested with the previous tile's loads
    int vseg[JP], rid[JP];
#pragma unroll
    for (int j = 0; j < JP; ++j) {
      const int u = j * NL + ld, q = u / SLOTS, ch = u - (u / SLOTS) * SLOTS;
      const int segpix = (p.RS + 2) * p.PW;
      const int sg = q / segpix, rem = q - sg * segpix;
      const int pr = rem / p.PW, pc = rem - (rem / p.PW) * p.PW;
      bool data = q < p.NP && ch < 8 && pc >= 1 && pc <= p.W;
      if (!p.tpi) data = data && pr >= 1 && pr <= p.H;
      vofs[j] = data ? static_cast<uint32_t>(sg * imgb + (pr - 1) * rowb + (pc - 1) * CIN * 2 + ch * 16) : 0xC0000000u;
      vseg[j] = data ? sg : -1;
      if (data) vofs[j] -= static_cast<uint32_t>(sg * imgb);
      if (!p.srows) vofs[j] += data ? static_cast<uint32_t>(sg * imgb) : 0u;
      rid[j] = 0;
    }
    // residual slots (listed residual): segment and pixel of each row
    auto fetch_rids = [&](int t) __attribute__((always_inline)) {
      int img, oh0, m0, lim;
      tile_geom(t, img, oh0, m0, lim);
#pragma unroll
      for (int j = 0; j < JP; ++j) rid[j] = vseg[j] >= 0 && img + vseg[j] < n ? p.srows[img + vseg[j]] : -1;
    };
    if (p.srows) fetch_rids(t_begin);
    for (int t = t_begin; t <= t_end; ++t) {
      if (t < t_end) {
        const int buf = (t - t_begin) & 1;
        int img, oh0, m0, lim;
        tile_geom(t, img, oh0, m0, lim);
        const int nimg = p.tpi ? 1 : min(p.segs, n - img);
        char* pb = pbuf + buf * kW3PB;
        if (p.srows) {
#pragma unroll
          for (int j = 0; j < JP; ++j) {
            const uint32_t o = rid[j] >= 0 ? static_cast<uint32_t>(rid[j]) * imgb + vofs[j] : 0xC0000000u;
            buffer_load_lds16(p.src, 0x7fffffffu, o, (lds_void_ptr)(pb + (j * NL + lw * 64) * 16));
          }
        } else {
          const uint16_t* pbase = p.src + (size_t)img * p.H * p.W * CIN;
          const uint32_t pbytes = static_cast<uint32_t>(nimg) * imgb, tofs = static_cast<uint32_t>(oh0) * rowb;
#pragma unroll
          for (int j = 0; j < JP; ++j)
            buffer_load_lds16(pbase, pbytes, vofs[j] + tofs, (lds_void_ptr)(pb + (j * NL + lw * 64) * 16));
        }
        if (RES) {
          char* rb = rbuf + buf * kW3RB;
          if (p.rrows) {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
              const int u = k * NL + ld, row = u >> 3, pos = u & 7;
              const int sg = row / HW, px = row - sg * HW;
              const uint32_t o = row < lim ? static_cast<uint32_t>((p.rrows[img + sg] * HW + px) * 128 + rsw(row, pos) * 16)
                                           : 0xC0000000u;
              buffer_load_lds16(p.res, 0x7fffffffu, o, (lds_void_ptr)(rb + (k * NL + lw * 64) * 16));
            }
          } else {
            const uint16_t* rbase = p.res + (size_t)m0 * 64;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
              const int u = k * NL + ld, row = u >> 3, pos = u & 7;
              buffer_load_lds16(rbase, static_cast<uint32_t>(lim) * 128, row * 128 + rsw(row, pos) * 16,
                                (lds_void_ptr)(rb + (k * NL + lw * 64) * 16));
            }
          }
        }
        if (p.srows && t + 1 < t_end) fetch_rids(t + 1);
      }
      all_barrier();                      // tile t is in LDS for the compute waves
    }
    return;
  }

  // ---------------- compute waves: tile t ----------------
  // MFMA operands: A = weights (32 output channels of this wave), B = patch
  // pixels, so a lane's results are 4 consecutive channels of one pixel per
  // group: channels wn*32 + 8q + 4*hi .. +3, q = 0..3, of pixel (lane & 31)
  const int wm = wave >> 1, wn = wave & 1, hi = lane >> 5;
  const int co_l = wn * 32 + (lane & 31);
  // B fragments: sub-step k covers K 16k .. 16k + 15 (64 channels: tap k/4,
  // channels 16 (k%4) ..; 8 channels: taps 2k, 2k + 1); this lane's half
  bf16x8 bw[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k)
    bw[k] = *reinterpret_cast<const bf16x8*>(p.w + (size_t)co_l * KP + 16 * k + 8 * hi);
  // scale / shift of the 64 channels, in LDS after the staging buffers
  float* const ssl = reinterpret_cast<float*>(sbuf + 2 * kW3RB);
  if (tid < 64) ssl[tid] = p.scale ? p.scale[tid] : 1.0f;
  else if (tid < 128) ssl[tid] = p.shift ? p.shift[tid - 64] : 0.0f;
  int pix0[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int i = wm * 64 + a * 32 + (lane & 31);
    const int sg = i / (p.RS * p.W), r = (i / p.W) - sg * p.RS, c = i - (i / p.W) * p.W;
    pix0[a] = sg < p.segs ? (sg * (p.RS + 2) + r) * p.PW + c : 0;
  }
  // a compiler-visible wait: the fragments are resident before the loop,
  // so no memory wait is placed inside it
  __builtin_amdgcn_s_waitcnt(0);

  lds_barrier();                          // the loaders' first tile
  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    f32x16 acc[2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][r] = 0.f;
    if constexpr (CIN == 8) {
      // sub-step k: this lane's tap 2k + hi (the tenth tap has zero weights)
      const char* pcur = pbuf + buf * kW3PB;
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        const int tap = 2 * k + hi < 9 ? 2 * k + hi : 0;
        const int toff = (tap / 3) * p.PW + (tap % 3);
        bf16x8 af[2];
#pragma unroll
        for (int a = 0; a < 2; ++a) af[a] = *reinterpret_cast<const bf16x8*>(pcur + (pix0[a] + toff) * 16);
#pragma unroll
        for (int a = 0; a < 2; ++a) acc[a] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bw[k], af[a], acc[a], 0, 0, 0);
      }
    } else {
      // lane base addresses of the three tap rows; the tap column and the K
      // chunk are constant offsets
      const char* ab[2][3];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int dy = 0; dy < 3; ++dy) ab[a][dy] = pbuf + buf * kW3PB + (pix0[a] + dy * p.PW) * 144 + hi * 16;
      bf16x8 af[2][2][2];                   // [slot][step of the pair][a]
      auto fetch = [&](int g, int slot) __attribute__((always_inline)) {
        const int tap = g >> 1, dy = tap / 3, dx = tap % 3;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            af[slot][j][a] = *reinterpret_cast<const bf16x8*>(ab[a][dy] + dx * 144 + (2 * (2 * (g & 1) + j)) * 16);
      };
      fetch(0, 0);
#pragma unroll
      for (int g = 0; g < 18; ++g) {
        if (g + 1 < 18) fetch(g + 1, (g + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int a = 0; a < 2; ++a)
            acc[a] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bw[2 * g + j], af[g & 1][j][a], acc[a], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // epilogue into this tile's staging buffer (the store waves finished its
    // previous contents, tile t - 2, before the last barrier): 8 bytes =
    // 4 channels per group.  All LDS reads of a step are issued before any
    // is used, so their latencies overlap.
    const char* rb = rbuf + buf * kW3RB;
    char* sb = sbuf + buf * kW3RB;
    float4 sc[4], sh[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      sc[q] = *reinterpret_cast<const float4*>(ssl + wn * 32 + 8 * q + 4 * hi);
      sh[q] = *reinterpret_cast<const float4*>(ssl + 64 + wn * 32 + 8 * q + 4 * hi);
    }
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int px = wm * 64 + a * 32 + (lane & 31);
      int off[4];
      uint2 rr[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        off[q] = px * 128 + (rsw(px, wn * 4 + q) << 4) + hi * 8;
        if (RES) rr[q] = *reinterpret_cast<const uint2*>(rb + off[q]);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4] = {fmaf(acc[a][4 * q], sc[q].x, sh[q].x), fmaf(acc[a][4 * q + 1], sc[q].y, sh[q].y),
                      fmaf(acc[a][4 * q + 2], sc[q].z, sh[q].z), fmaf(acc[a][4 * q + 3], sc[q].w, sh[q].w)};
        if (RES) {
          v[0] += __uint_as_float(rr[q].x << 16);
          v[1] += __uint_as_float(rr[q].x & 0xffff0000u);
          v[2] += __uint_as_float(rr[q].y << 16);
          v[3] += __uint_as_float(rr[q].y & 0xffff0000u);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = apply_act(v[e], ACT);
        bf16x2 lo = {(__bf16)v[0], (__bf16)v[1]}, hv = {(__bf16)v[2], (__bf16)v[3]};
        *reinterpret_cast<uint2*>(sb + off[q]) =
            make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hv));
      }
    }
    lds_barrier();                        // staging written; the next tile has landed
  }
}

// ------------------------------ 3x3 conv, halo tiles, streamed weights ----
// For 3x3 / stride 1 / pad 1 layers with Cin and Cout multiples of 64.  A
// persistent workgroup walks a contiguous range of work units, a unit being
// one BM-pixel output tile (128 as launched; the row / image geometry of the
// kernel above) times BN output channels.  The K loop runs over 64-channel chunks and,
// inside a chunk, the nine taps: one step = one tap of one chunk = 64 of K.
//  * the input patch of a chunk (the tile's pixels plus the one-pixel halo,
//    144 bytes per pixel) is staged in LDS once and read by all nine taps;
//    it is double-buffered, and the next chunk's patch is requested at the
//    first step of the current chunk, nine steps before it is needed;
//  * the weights of a step (BN rows x 128 bytes, XOR-swizzled) stream
//    through NS LDS stages, NS - 1 steps ahead of the MFMAs.
// Eight waves, one barrier per step: four compute waves (2 x 2, each
// BM/2 pixels x BN/2 channels: 4 or 2 MFMA blocks of 32 pixels by BN/64
// blocks of 32 channels) touch global memory only in the epilogue;
// two weight loader waves and two patch loader waves issue every load
// straight into LDS.  Each loader role waits only for its own loads (the memory counter
// completes in order, so one role's slow loads never hold up the other's):
// the weight loaders for step g's weights, issued NS - 1 steps earlier; the
// patch loaders, at a chunk start, for that chunk's patch.
//
// MFMA operands: A = weights (32 output channels), B = patch pixels, so a
// lane's results are 4 consecutive channels of one pixel per group and the
// epilogue writes 8-byte pieces of NHWC rows directly; scale and shift of
// every output channel are kept in LDS.
struct Conv3HP {
  const uint16_t* src;
  const uint16_t* w;       // [cout_pad][Kp] packed, K = tap * cin + ci
  const float* scale;
  const float* shift;
  const uint16_t* res;
  uint16_t* dst;
  const uint16_t* zeros;
  int n, H, W, cin, cout, Kp;
  int RS, segs, PW, NP, tpi;
  int ntiles, units, nch;  // output channel tiles, units, 64-channel chunks
  const int32_t* nc;       // device count of live images (<= n) or null
};

constexpr int kHP = 256;                           // patch pixels per buffer of 128-pixel tiles
constexpr int kHMaxC = 512;                        // output channels whose scale / shift fit LDS
// patch loads per patch-loader thread and chunk (128 threads x 16 bytes),
// and patch capacity in pixels, by tile height
constexpr int halo_jp(int bm) { return bm == 128 ? 18 : 24; }
constexpr int halo_cap(int bm) { return halo_jp(bm) * 128 / 9; }

template <int BM, int BN, int WA, int ACT, bool RES, int kHNS>
__global__ __launch_bounds__(64 * (BM / (16 * WA) + 4)) void conv3h_kernel(Conv3HP p) {
  constexpr int CW = BM / (16 * WA);               // compute waves (BM / (32 WA) x 2)
  constexpr int JW = BN / 16;                      // weight loads per weight-loader thread and step
  constexpr int JP = halo_jp(BM);                  // patch loads per patch-loader thread and chunk
  constexpr int kHPB = JP * 128 * 16;              // patch buffer bytes
  constexpr int WSTAGE = BN * 128;
  constexpr int TB = BN / 64;                      // 32-channel blocks per compute wave
  static_assert(kHNS >= 3 && (kHNS - 3) * JW < 64, "stage count");
  __shared__ __align__(16) char smem[kHNS * WSTAGE + 2 * kHPB + 2 * kHMaxC * 4];
  char* const wbuf = smem;
  char* const pbuf = smem + kHNS * WSTAGE;
  float* const ssl = reinterpret_cast<float*>(pbuf + 2 * kHPB);   // [scale | shift]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = __builtin_amdgcn_readfirstlane(wave);   // the same, known wave-uniform
  const int HW = p.H * p.W;
  const int n = p.nc ? min(*p.nc, p.n) : p.n;
  const int units = p.nc ? (p.tpi ? n * p.tpi : (n + p.segs - 1) / p.segs) * p.ntiles : p.units;
  const int u_begin = static_cast<int>((static_cast<long>(units) * blockIdx.x) / gridDim.x);
  const int u_end = static_cast<int>((static_cast<long>(units) * (blockIdx.x + 1)) / gridDim.x);
  if (u_begin >= u_end) return;
  const int S = 9 * p.nch;                         // steps per unit
  const int T = (u_end - u_begin) * S;             // steps of this workgroup

  // unit -> (pixel tile, channel tile); consecutive units share the pixel tile
  auto unit_geom = [&](int u, int& img, int& oh0, int& m0, int& lim, int& n0) __attribute__((always_inline)) {
    const int mt = u / p.ntiles;
    n0 = (u - mt * p.ntiles) * BN;
    if (p.tpi) {
      img = mt / p.tpi;
      oh0 = (mt - img * p.tpi) * p.RS;
      m0 = img * HW + oh0 * p.W;
      lim = min(p.RS, p.H - oh0) * p.W;
    } else {
      img = mt * p.segs;
      oh0 = 0;
      m0 = img * HW;
      lim = min(p.segs, n - img) * HW;
    }
  };

  if (wv >= CW + 2) {
    // ---------------- patch loader waves ----------------
    // Buffer loads straight into LDS.  A chunk's loads use one buffer
    // resource spanning the tile's image(s) from the chunk's first channel;
    // a load outside it returns zeros, which is the convolution's padding:
    // a slot's byte offset is taken relative to the tile's first output row
    // (row mode: plus oh0 rows, so the halo row above image row 0 wraps to
    // a huge offset, and rows past the image exceed the resource), and slots
    // that can never hold data (zero columns, the unused ninth slot, past
    // the patch, the halo rows of image mode) get an offset above 2^31.
    const int lt = tid - (CW + 2) * 64, lw = wv - (CW + 2);
    const int rowb = p.W * p.cin * 2, imgb = p.H * rowb;
    uint32_t vofs[JP];
#pragma unroll
    for (int i = 0; i < JP; ++i) {
      const int u = i * 128 + lt, q = u / 9, ch = u - (u / 9) * 9;
      const int segpix = (p.RS + 2) * p.PW;
      const int sg = q / segpix, rem = q - sg * segpix;
      const int pr = rem / p.PW, pc = rem - (rem / p.PW) * p.PW;
      bool data = q < p.NP && ch < 8 && pc >= 1 && pc <= p.W;
      if (!p.tpi) data = data && pr >= 1 && pr <= p.H;
      vofs[i] = data ? static_cast<uint32_t>(sg * imgb + (pr - 1) * rowb + (pc - 1) * p.cin * 2 + ch * 16) : 0xC0000000u;
    }
    // chunk iterator: (unit, chunk) of the next patch to request
    int pu = u_begin, pc_ = 0;
    const uint16_t* rbase = p.src;                 // the chunk's buffer: base and size
    uint32_t rbytes = 0;
    uint32_t tofs = 0;                             // row mode: oh0 rows, in bytes
    auto set_chunk = [&]() __attribute__((always_inline)) {
      int img = 0, oh0 = 0, nimg = 0;
      if (pu < u_end) {
        int m0, lim, n0;
        unit_geom(pu, img, oh0, m0, lim, n0);
        nimg = p.tpi ? 1 : min(p.segs, n - img);
      }
      rbase = p.src + (size_t)img * p.H * p.W * p.cin + pc_ * 64;
      rbytes = nimg ? nimg * imgb - pc_ * 128 : 0;
      tofs = static_cast<uint32_t>(oh0) * rowb;
    };
    set_chunk();
    // loads k0 .. k1-1 of the patch of chunk sequence number cs
    auto issue_patch = [&](int cs, int k0, int k1) __attribute__((always_inline)) {
      char* pb = pbuf + (cs & 1) * kHPB;
#pragma unroll
      for (int i = 0; i < JP; ++i) {
        if (i < k0 || i >= k1) continue;
        buffer_load_lds16(rbase, rbytes, vofs[i] + tofs, (lds_void_ptr)(pb + (i * 128 + lw * 64) * 16));
      }
    };
    auto next_chunk = [&]() __attribute__((always_inline)) {
      if (++pc_ == p.nch) {
        pc_ = 0;
        ++pu;
      }
      set_chunk();
    };
    issue_patch(0, 0, JP);
    next_chunk();
    // chunk q + 1 is requested in six pieces over the first six steps of
    // chunk q and must have landed before the barrier of step 9q + 8 (whose
    // compute waves prefetch the first operands of step 9(q + 1)).
    // Iteration k precedes the barrier that starts compute step k, k = 0..T.
    int r = 0;
    for (int k = 0; k <= T; ++k) {
      if (k == 0 || r == 8)
        wait_vm_barrier<0>();
      else
        asm volatile("s_barrier" ::: "memory");
      if (r < 6) {
        const int cs = k / 9 + 1;
        if (r == 0) issue_patch(cs, 0, JP / 6);
        else if (r == 1) issue_patch(cs, JP / 6, 2 * JP / 6);
        else if (r == 2) issue_patch(cs, 2 * JP / 6, 3 * JP / 6);
        else if (r == 3) issue_patch(cs, 3 * JP / 6, 4 * JP / 6);
        else if (r == 4) issue_patch(cs, 4 * JP / 6, 5 * JP / 6);
        else {
          issue_patch(cs, 5 * JP / 6, JP);
          next_chunk();
        }
      }
      if (++r == 9) r = 0;
    }
    wait_vm_barrier<0>();                          // the last (placeholder) chunk, before the workgroup ends
    return;
  }

  if (wv >= CW) {
    // ---------------- weight loader waves ----------------
    // one buffer resource per step (its weights: BN rows from the step's K
    // offset); each thread's slots are constant byte offsets from it
    const int lt = tid - CW * 64, lw = wv - CW;
    uint32_t wofs[JW];
#pragma unroll
    for (int k = 0; k < JW; ++k) {
      const int u = k * 128 + lt, row = u >> 3, pos = u & 7;
      wofs[k] = static_cast<uint32_t>(row * p.Kp + ((pos ^ ((row >> 1) & 7)) * 8)) * 2;
    }
    const uint32_t wbytes = static_cast<uint32_t>(p.ntiles * BN) * p.Kp * 2;
    // step iterator of the next weights to request: unit, its channel
    // tile, chunk and tap (K offset tap * cin + chunk * 64)
    int wu = u_begin, wnt = u_begin % p.ntiles, wc = 0, wt = 0, ws_i = 0;
    auto issue_weights = [&]() __attribute__((always_inline)) {
      const uint32_t e0 = static_cast<uint32_t>(wnt * BN) * p.Kp + wt * p.cin + wc * 64;
      const uint32_t wb = wu < u_end ? wbytes - e0 * 2 : 0;
      char* ws = wbuf + ws_i * WSTAGE;
#pragma unroll
      for (int k = 0; k < JW; ++k)
        buffer_load_lds16(p.w + e0, wb, wofs[k], (lds_void_ptr)(ws + (k * 128 + lw * 64) * 16));
      if (++ws_i == kHNS) ws_i = 0;
      if (++wt == 9) {
        wt = 0;
        if (++wc == p.nch) {
          wc = 0;
          ++wu;
          if (++wnt == p.ntiles) wnt = 0;
        }
      }
    };
    for (int k = 0; k < kHNS - 1; ++k) issue_weights();
    // iteration k precedes the barrier that starts compute step k: steps k
    // and k + 1 must be resident (step k + 1's first operands are read
    // during step k), i.e. everything up to step k + 1's weights, issued
    // NS - 2 iterations ago
    for (int k = 0; k <= T; ++k) {
      wait_vm_barrier<(kHNS - 3) * JW>();
      issue_weights();                             // step k + NS - 1, into the stage of step k - 1
    }
    wait_vm_barrier<0>();
    return;
  }

  // ---------------- compute waves ----------------
  for (int c = tid; c < p.cout; c += CW * 64) {
    ssl[c] = p.scale ? p.scale[c] : 1.0f;
    ssl[kHMaxC + c] = p.shift ? p.shift[c] : 0.0f;
  }
  const int wm = wave >> 1, wn = wave & 1, hi = lane >> 5;
  int pix0[WA];
#pragma unroll
  for (int a = 0; a < WA; ++a) {
    const int i = wm * (32 * WA) + a * 32 + (lane & 31);
    const int sg = i / (p.RS * p.W), r = (i / p.W) - sg * p.RS, c = i - (i / p.W) * p.W;
    pix0[a] = sg < p.segs ? (sg * (p.RS + 2) + r) * p.PW + c : 0;
  }
  int wrow[TB];
#pragma unroll
  for (int b = 0; b < TB; ++b) wrow[b] = wn * (BN / 2) + b * 32 + (lane & 31);

  f32x16 acc[TB][WA];
#pragma unroll
  for (int b = 0; b < TB; ++b)
#pragma unroll
    for (int a = 0; a < WA; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[b][a][r] = 0.f;

  // fragment addresses of a step: weight stage and patch window
  auto step_ptrs = [&](int st_, int pbi_, int tap_, const char*& ws_, const char*& pb_) __attribute__((always_inline)) {
    const int dy = tap_ / 3, dx = tap_ - (tap_ / 3) * 3;
    ws_ = wbuf + st_ * WSTAGE;
    pb_ = pbuf + pbi_ * kHPB + (dy * p.PW + dx) * 144 + hi * 16;
  };
  bf16x8 wf[2][TB], pf[2][WA];
  auto fetch = [&](const char* ws_, const char* pb_, int s, int slot) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < TB; ++b)
      wf[slot][b] = *reinterpret_cast<const bf16x8*>(ws_ + wrow[b] * 128 + (((2 * s + hi) ^ ((wrow[b] >> 1) & 7)) << 4));
#pragma unroll
    for (int a = 0; a < WA; ++a) pf[slot][a] = *reinterpret_cast<const bf16x8*>(pb_ + pix0[a] * 144 + s * 32);
  };
  int tap = 0, jc = 0, cu = u_begin, st = 0, pbi = 0;   // tap, step in unit, unit, stage, patch buffer
  // the barrier of step g also guarantees step g + 1's data, so the first
  // operands of step g + 1 are read before it
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");   // scale / shift; steps 0 and 1
  const char* ws;
  const char* pb;
  step_ptrs(0, 0, 0, ws, pb);
  fetch(ws, pb, 0, 0);
  for (int g = 0; g < T; ++g) {
    const bool unit_end = jc == S - 1;
    // the next step's stage / patch buffer / tap
    int st1 = st + 1 == kHNS ? 0 : st + 1, tap1 = tap + 1, pbi1 = pbi;
    if (tap1 == 9) {
      tap1 = 0;
      pbi1 ^= 1;
    }
    const char* ws1;
    const char* pb1;
    step_ptrs(st1, pbi1, tap1, ws1, pb1);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s + 1 < 4)
        fetch(ws, pb, s + 1, (s + 1) & 1);
      else if (g + 1 < T)
        fetch(ws1, pb1, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int b = 0; b < TB; ++b)
#pragma unroll
        for (int a = 0; a < WA; ++a)
          acc[b][a] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[s & 1][b], pf[s & 1][a], acc[b][a], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    st = st1;
    tap = tap1;
    pbi = pbi1;
    ws = ws1;
    pb = pb1;
    if (++jc == S) jc = 0;

    if (unit_end) {
      // unit done: epilogue straight to global memory, 8 bytes per group
      int img, oh0, m0, lim, n0;
      unit_geom(cu++, img, oh0, m0, lim, n0);
#pragma unroll
      for (int a = 0; a < WA; ++a) {
        const int px = wm * (32 * WA) + a * 32 + (lane & 31);
        const bool live = px < lim;
        const size_t rowo = (size_t)(m0 + (live ? px : 0)) * p.cout;
        uint2 rr[TB][4];
        if (RES && live) {
#pragma unroll
          for (int b = 0; b < TB; ++b)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              rr[b][q] = *reinterpret_cast<const uint2*>(p.res + rowo + n0 + wn * (BN / 2) + b * 32 + 8 * q + 4 * hi);
        }
#pragma unroll
        for (int b = 0; b < TB; ++b)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int c0 = n0 + wn * (BN / 2) + b * 32 + 8 * q + 4 * hi;
            const float4 sc = *reinterpret_cast<const float4*>(ssl + c0);
            const float4 sh = *reinterpret_cast<const float4*>(ssl + kHMaxC + c0);
            float v[4] = {fmaf(acc[b][a][4 * q], sc.x, sh.x), fmaf(acc[b][a][4 * q + 1], sc.y, sh.y),
                          fmaf(acc[b][a][4 * q + 2], sc.z, sh.z), fmaf(acc[b][a][4 * q + 3], sc.w, sh.w)};
            if (RES) {
              v[0] += __uint_as_float(rr[b][q].x << 16);
              v[1] += __uint_as_float(rr[b][q].x & 0xffff0000u);
              v[2] += __uint_as_float(rr[b][q].y << 16);
              v[3] += __uint_as_float(rr[b][q].y & 0xffff0000u);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = apply_act(v[e], ACT);
            bf16x2 lo = {(__bf16)v[0], (__bf16)v[1]}, hv = {(__bf16)v[2], (__bf16)v[3]};
            if (live)
              *reinterpret_cast<uint2*>(p.dst + rowo + c0) =
                  make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hv));
          }
      }
#pragma unroll
      for (int b = 0; b < TB; ++b)
#pragma unroll
        for (int a = 0; a < WA; ++a)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[b][a][r] = 0.f;
    }
    // this step's LDS reads are done; step g + 2's data is ready after it
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  }
}

// ------------------------------------------------------- K-split sums ----
// y[m, c..c+7] = finish(sum_s part[s][m][c..c+7]) with the splits added in
// order s = 0, 1, ...: scale / shift, residual, activation, bf16 rounding,
// as the single-range epilogue does.
template <int ACT>
__global__ __launch_bounds__(256) void ksplit_finish_kernel(const float* __restrict__ part, int S, int Mb, int cout,
                                                            const int32_t* nc, int nmax, int HoWo,
                                                            const float* __restrict__ scale,
                                                            const float* __restrict__ shift,
                                                            const uint16_t* __restrict__ res,
                                                            uint16_t* __restrict__ dst) {
  const int M = (nc ? min(*nc, nmax) : nmax) * HoWo;
  const int C8 = cout >> 3;
  const size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<size_t>(M) * C8) return;
  const size_t row = i / C8;
  const int c = static_cast<int>(i - row * C8) * 8;
  const size_t o = row * cout + c;
  const size_t stride = static_cast<size_t>(Mb) * cout;
  float4 lo = *reinterpret_cast<const float4*>(part + o), hi = *reinterpret_cast<const float4*>(part + o + 4);
  for (int sp = 1; sp < S; ++sp) {
    const float4 a = *reinterpret_cast<const float4*>(part + sp * stride + o);
    const float4 b = *reinterpret_cast<const float4*>(part + sp * stride + o + 4);
    lo.x += a.x; lo.y += a.y; lo.z += a.z; lo.w += a.w;
    hi.x += b.x; hi.y += b.y; hi.z += b.z; hi.w += b.w;
  }
  float vv[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
  for (int q = 0; q < 8; ++q) vv[q] = fmaf(vv[q], scale ? scale[c + q] : 1.0f, shift ? shift[c + q] : 0.0f);
  if (res) {
    const uint4 rv = *reinterpret_cast<const uint4*>(res + o);
    const uint32_t rw[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      vv[2 * q] += __uint_as_float(rw[q] << 16);
      vv[2 * q + 1] += __uint_as_float(rw[q] & 0xffff0000u);
    }
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) vv[q] = act_t<ACT>(vv[q]);
  uint4 ov;
  ov.x = pack_bf16(vv[0], vv[1]);
  ov.y = pack_bf16(vv[2], vv[3]);
  ov.z = pack_bf16(vv[4], vv[5]);
  ov.w = pack_bf16(vv[6], vv[7]);
  *reinterpret_cast<uint4*>(dst + o) = ov;
}

// ------------------------------------------------------------- launch ----

namespace {

struct TileCfg {
  int bm, bn, wm, wn;
};

// register-staged kernel (element-gathering stems, unaligned outputs)
constexpr TileCfg kWide[] = {{128, 128, 2, 2}, {128, 64, 2, 2}, {64, 64, 2, 2}};
constexpr TileCfg kMid[] = {{128, 64, 2, 2}, {64, 64, 2, 2}};
constexpr TileCfg kNarrow[] = {{128, 32, 4, 1}, {64, 32, 2, 1}};

long tiles_of(const TileCfg& c, int M, int cout) {
  return (long)((M + c.bm - 1) / c.bm) * ((cout + c.bn - 1) / c.bn);
}

template <size_t N>
TileCfg choose(const TileCfg (&cs)[N], int M, int cout) {
  for (size_t i = 0; i < N; ++i)
    if (tiles_of(cs[i], M, cout) >= 512) return cs[i];
  return cs[N - 1];
}

template <int BM, int BN, int WM, int WN, int KS, bool SC>
void go(const ConvP& p, hipStream_t s) {
  hipLaunchKernelGGL((conv_kernel<BM, BN, WM, WN, KS, SC, 64, 1>), dim3(p.mt * p.nt), dim3(64 * WM * WN), 0, s, p);
}

template <int KS>
void dispatch_staged(const TileCfg& c, const ConvP& p, hipStream_t s) {
  switch (c.bm * 1000 + c.bn) {
    case 128128: go<128, 128, 2, 2, KS, false>(p, s); break;
    case 128064: go<128, 64, 2, 2, KS, false>(p, s); break;
    case 64064: go<64, 64, 2, 2, KS, false>(p, s); break;
    case 128032: go<128, 32, 4, 1, KS, false>(p, s); break;
    default: go<64, 32, 2, 1, KS, false>(p, s); break;
  }
}

// direct-to-LDS kernel.  A workgroup's LDS (two stages) sets how many fit
// on a CU: two of 128 x 128 (64 KB), three of 128 x 64 (48 KB); a grid runs
// in ceil(tiles / resident) rounds.  Tiles are compared by rounds times tile
// area, the time of the slowest CU (measured on the layer shapes of the
// workloads; 256 x 256 tiles lost on every one of them)
TileCfg choose_lds(int M, int cout, int Kp) {
  const TileCfg c128{128, 128, 2, 2}, c12864{128, 64, 2, 2}, c64{64, 64, 2, 2}, c64128{64, 128, 2, 2},
      c32{128, 32, 4, 1};
  if (cout < 64) return c32;
  // one K step: memory-bound; 128 x 64 tiles (24 KB of LDS, five
  // workgroups per CU by registers) keep the most rows in flight (measured
  // against 128 x 128, 64 x 128, 64 x 64 and 256 x 64 on the ResNet-50 1x1
  // layers)
  if (Kp <= 64) return c12864;
  constexpr long kCUs = 256;
  const long r128 = (tiles_of(c128, M, cout) + 2 * kCUs - 1) / (2 * kCUs);
  const long t12864 = tiles_of(c12864, M, cout), r12864 = (t12864 + 3 * kCUs - 1) / (3 * kCUs);
  // few tiles (a layer bound by its chains of K rounds): 64 x 64 below ~1.5
  // tiles of 128 x 64 per CU, 64 x 128 below four (measured with rounds of
  // two K steps: ResNet-50's strided stage-3 3x3 49 -> 42 us, its stage-3/4
  // reductions and stage-4 expansions 4-10 % faster than 128 x 64)
  if (t12864 < 400) return c64;
  if (t12864 < 1024 && cout % 128 == 0) return c64128;
  // 128 x 128 when its rounds of double-area tiles take no longer, or when
  // one tile column spans a short-K layer's channels, so that each input
  // pixel (the bulk of its traffic) is fetched by one workgroup
  if (cout >= 128 && (2 * r128 <= r12864 || (cout == 128 && Kp <= 256))) return c128;
  return c12864;
}

// stages: one (`one`, 128 x 64 or 128 x 256 tiles only: the K steps taken
// in turn) where the workgroups a CU holds bound the layer, five with one
// 24 KB stage against three with two: measured 2-20 % faster on the
// ResNet-50 1x1 shapes with many tiles and 8-16 % on its strided 3x3
// layers with 2.5 or more tiles per CU (slower with fewer); else two,
// filled in rounds of two K steps
template <int BM, int BN, int WM, int WN, int KS>
void go_lds(const ConvP& p, hipStream_t s, int S, bool one) {
  const dim3 grid(p.mt * p.nt * S);
  if (one && S == 1) {
    if constexpr (BM == 128 && (BN == 64 || BN == 256))
      hipLaunchKernelGGL((conv_lds_kernel<BM, BN, WM, WN, KS, 1>), grid, dim3(64 * WM * WN), 0, s, p);
    else
      throw std::invalid_argument("conv_bf16: the one-stage implicit GEMM takes 128 x 64 or 128 x 256 tiles only");
  } else if constexpr (BN == 256) {
    throw std::invalid_argument("conv_bf16: 128 x 256 tiles are one-stage only");
  } else {
    hipLaunchKernelGGL((conv_lds_kernel<BM, BN, WM, WN, KS, 2>), grid, dim3(64 * WM * WN), 0, s, p);
  }
}

template <int KS>
void dispatch_lds(const TileCfg& c, const ConvP& p, hipStream_t s, int S = 1, bool one = false) {
  switch (c.bm * 1000 + c.bn) {
    case 128128: go_lds<128, 128, 2, 2, KS>(p, s, S, one); break;
    case 128064: go_lds<128, 64, 2, 2, KS>(p, s, S, one); break;
    case 128256: go_lds<128, 256, 2, 4, KS>(p, s, S, one); break;
    case 64064: go_lds<64, 64, 2, 2, KS>(p, s, S, one); break;
    case 64128: go_lds<64, 128, 2, 2, KS>(p, s, S, one); break;
    default: go_lds<128, 32, 4, 1, KS>(p, s, S, one); break;
  }
}

// Tile geometry of the halo kernels: BM-pixel tiles of R whole rows of one
// image, or of G whole images; the patch (tile rows + halo) must fit `cap`
// pixels.
struct HaloGeom {
  int RS, segs, tpi, PW, NP, mtiles;
};

bool halo_geom(int n, int H, int W, int bm, int cap, HaloGeom& g) {
  if (W > bm || n <= 0) return false;
  const int HW = H * W;
  if (HW > bm) {
    g.RS = bm / W;
    g.segs = 1;
    g.tpi = (H + g.RS - 1) / g.RS;
    g.mtiles = n * g.tpi;
  } else {
    g.RS = H;
    g.segs = bm / HW;
    while (g.segs > 1 && g.segs * (H + 2) * (W + 2) > cap) --g.segs;
    g.tpi = 0;
    g.mtiles = (n + g.segs - 1) / g.segs;
  }
  g.PW = W + 2;
  g.NP = g.segs * (g.RS + 2) * g.PW;
  return g.NP <= cap;
}

int cu_count() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (!cus[dev] && hipDeviceGetAttribute(&cus[dev], hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus[dev] = 0;
  return cus[dev];
}

bool is_halo_layer(const ConvArgs& a) {
  return a.k == 3 && a.stride == 1 && a.pad == 1 && !a.src2 && !a.out_f32 && a.Ho == a.H && a.Wo == a.W &&
         a.cin % 64 == 0 && a.cout % 64 == 0 && a.Kp == 9 * a.cin &&
         !((reinterpret_cast<uintptr_t>(a.scale) | reinterpret_cast<uintptr_t>(a.shift)) & 15);
}

// the weights-resident 3x3 kernel (64 -> 64 channels)
bool conv3_wres(const ConvArgs& a, hipStream_t s) {
  HaloGeom g;
  const bool stem = a.cin == 8 && a.Kp == 128 && a.k == 3 && a.stride == 1 && a.pad == 1 && !a.src2 && !a.out_f32 &&
                    a.Ho == a.H && a.Wo == a.W &&
                    !((reinterpret_cast<uintptr_t>(a.scale) | reinterpret_cast<uintptr_t>(a.shift)) & 15);
  if (!(stem || (is_halo_layer(a) && a.cin == 64)) || a.cout != 64 || !halo_geom(a.n, a.H, a.W, 128, kHP, g))
    return false;
  const int cus = cu_count();
  if (!cus) return false;
  Conv3P p;
  p.src = a.src;
  p.w = a.w;
  p.scale = a.scale;
  p.shift = a.shift;
  p.res = a.res;
  p.dst = static_cast<uint16_t*>(a.dst);
  p.zeros = a.zeros;
  p.n = a.n;
  p.H = a.H;
  p.W = a.W;
  p.cout = a.cout;
  p.act = a.act;
  p.RS = g.RS;
  p.segs = g.segs;
  p.tpi = g.tpi;
  p.PW = g.PW;
  p.NP = g.NP;
  p.tiles = g.mtiles;
  p.nc = a.ncount;
  // row lists: image mode only, no concatenated input, and every listed
  // tensor small enough for 31-bit byte offsets from its start
  const bool listed = a.src_rows || a.res_rows || a.dst_rows;
  if (listed && (stem || g.tpi != 0 || a.src2_rows || a.list_rows <= 0 ||
                 static_cast<long>(a.list_rows) * a.H * a.W * 128 > 0x7ffffff0L))
    return false;
  p.srows = a.src_rows;
  p.rrows = a.res_rows;
  p.drows = a.dst_rows;
  const int grid = p.tiles < cus ? p.tiles : cus;
  auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(grid), dim3(512), 0, s, p); };
#define DYCL_W(CIN)                                                     \
  if (p.res) {                                                          \
    if (p.act == ACT_RELU) go(conv3_wres_kernel<CIN, ACT_RELU, true>);  \
    else if (p.act == ACT_GELU) go(conv3_wres_kernel<CIN, ACT_GELU, true>); \
    else go(conv3_wres_kernel<CIN, ACT_NONE, true>);                    \
  } else {                                                              \
    if (p.act == ACT_RELU) go(conv3_wres_kernel<CIN, ACT_RELU, false>); \
    else if (p.act == ACT_GELU) go(conv3_wres_kernel<CIN, ACT_GELU, false>); \
    else go(conv3_wres_kernel<CIN, ACT_NONE, false>);                   \
  }
  if (stem) {
    DYCL_W(8)
  } else {
    DYCL_W(64)
  }
#undef DYCL_W
  return true;
}

// the streamed-weights 3x3 kernel (Cin, Cout multiples of 64) on 128-pixel
// tiles: measured 2-5 % faster than 256-pixel tiles on the ResNet-50
// stage-2 / 3 and ResNet-18 stage-2 layers (interleaved runs, best of four
// each), and a shape whose 128-pixel patch does not fit LDS fits no
// 256-pixel patch either, once the smallest images (taken by the implicit
// GEMM, below) are set aside
bool conv3_halo(const ConvArgs& a, hipStream_t s) {
  if (!is_halo_layer(a) || a.cout > kHMaxC) return false;
  // images so small that the halo more than doubles the patch (4 x 4: 36
  // pixels for 16) go to the implicit GEMM, which is faster there
  if (a.H * a.W <= 128 && 2 * a.H * a.W < (a.H + 2) * (a.W + 2)) return false;
  const int cus = cu_count();
  if (!cus) return false;
  // the tile shape follows the expected live images; the geometry (and the
  // grid) is then laid out for all n
  const int nh = a.nhint > 0 && a.nhint < a.n ? a.nhint : a.n;
  HaloGeom g;
  constexpr int bm = 128;
  if (!halo_geom(nh, a.H, a.W, bm, halo_cap(bm), g)) return false;
  const int bn = (a.cout % 128 == 0 && conv_cout_pad(a.cout) % 128 == 0 && (long)g.mtiles * (a.cout / 128) >= cus)
                     ? 128 : 64;
  if (!halo_geom(a.n, a.H, a.W, bm, halo_cap(bm), g)) return false;
  Conv3HP p;
  p.src = a.src;
  p.w = a.w;
  p.scale = a.scale;
  p.shift = a.shift;
  p.res = a.res;
  p.dst = static_cast<uint16_t*>(a.dst);
  p.zeros = a.zeros;
  p.n = a.n;
  p.H = a.H;
  p.W = a.W;
  p.cin = a.cin;
  p.cout = a.cout;
  p.Kp = a.Kp;
  p.RS = g.RS;
  p.segs = g.segs;
  p.tpi = g.tpi;
  p.PW = g.PW;
  p.NP = g.NP;
  p.ntiles = a.cout / bn;
  p.units = g.mtiles * p.ntiles;
  p.nch = a.cin / 64;
  p.nc = a.ncount;
  const int grid = p.units < cus ? p.units : cus;
  // four compute waves of 64 x BN/2 (pixels x channels), four loader waves
  auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(grid), dim3(512), 0, s, p); };
#define DYCL_H(BM, BN, NS)                                                              \
  if (p.res) {                                                                          \
    if (a.act == ACT_RELU) go(conv3h_kernel<BM, BN, BM / 64, ACT_RELU, true, NS>);      \
    else if (a.act == ACT_GELU) go(conv3h_kernel<BM, BN, BM / 64, ACT_GELU, true, NS>); \
    else go(conv3h_kernel<BM, BN, BM / 64, ACT_NONE, true, NS>);                        \
  } else {                                                                              \
    if (a.act == ACT_RELU) go(conv3h_kernel<BM, BN, BM / 64, ACT_RELU, false, NS>);     \
    else if (a.act == ACT_GELU) go(conv3h_kernel<BM, BN, BM / 64, ACT_GELU, false, NS>); \
    else go(conv3h_kernel<BM, BN, BM / 64, ACT_NONE, false, NS>);                       \
  }
  if (bn == 128) {
    DYCL_H(128, 128, 5)
  } else {
    DYCL_H(128, 64, 8)
  }
#undef DYCL_H
  return true;
}

}  // namespace

__device__ __align__(16) uint16_t g_zero_page[64];   // zero-initialised device memory

const uint16_t* zero_page() {
  static const uint16_t* addr[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  if (!addr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(g_zero_page)) != hipSuccess) return nullptr;
    addr[dev] = static_cast<const uint16_t*>(ptr);
  }
  return addr[dev];
}

int conv_ksplit(int Ho, int Wo, int cout, int K, bool out_f32) {
  // measured: K = 4608 on 4x4 and 7x7 outputs gains from four ranges
  // (ResNet-50 stage 4, 51 images: 42 -> 34 us; ResNet-18 stage 4, 255
  // images: its step 1.218 -> 1.201 ms, same box, interleaved runs), K =
  // 2304 loses from two (the partial sums cost more than the idle CUs)
  if (out_f32 || Ho * Wo > 64 || K < 4608 || cout < 256 || cout % 64) return 1;
  return 4;
}

int conv_cout_pad(int cout) {
  if (cout >= 256) return (cout + 255) / 256 * 256;
  if (cout >= 128) return (cout + 127) / 128 * 128;
  if (cout >= 64) return (cout + 63) / 64 * 64;
  return (cout + 31) / 32 * 32;
}

bool conv_bf16(const ConvArgs& a, hipStream_t s) {
  if (a.pool) return false;   // only conv_rgb_stem fuses a max-pool (its dst is the pooled tensor)
  if (a.cin == 3 && conv_rgb_stem(a, s)) return false;
  ConvP p;
  p.src = a.src;
  p.src2 = a.src2;
  p.H2 = a.src2_H > 0 ? a.src2_H : a.H;
  p.W2 = a.src2_W > 0 ? a.src2_W : a.W;
  p.s2 = a.src2_stride > 0 ? a.src2_stride : 1;
  p.cin1 = a.cin1;
  p.cin2 = a.cin2;
  p.H = a.H;
  p.W = a.W;
  p.cin = a.cin;
  p.Ho = a.Ho;
  p.Wo = a.Wo;
  p.cout = a.cout;
  p.stride = a.stride;
  p.pad = a.pad;
  p.M = a.n * a.Ho * a.Wo;
  p.K = a.k * a.k * a.cin;
  p.Kp = a.Kp;
  int lg = 0;
  while ((1 << lg) < a.cin) ++lg;
  p.cin_log2 = lg;
  p.w = a.w;
  p.scale = a.scale;
  p.shift = a.shift;
  p.res = a.res;
  p.dst = a.dst;
  p.act = a.act;
  p.out_f32 = a.out_f32;
  p.zeros = a.zeros;
  p.nc = a.ncount;
  p.nmax = a.n;
  p.ksplit = 1;
  p.part = nullptr;
  p.cell_in = a.cell_in;
  p.cell_out = a.cell_out;
  p.gap = nullptr;
  p.rev = a.rev;
  p.kfold = a.kfold;
  p.fsp = a.fold_sp;
  p.fbp = a.fold_bp;
  p.finv = a.fold_inv;
  if (a.kfold && (!a.src2 || a.cin1 % kBK || a.cin2 != a.kfold * kBK || a.k != 1 || a.res || a.out_f32 ||
                  !a.fold_sp || !a.fold_bp || !a.fold_inv || a.cout % 8 || (reinterpret_cast<uintptr_t>(a.dst) & 15) ||
                  !a.zeros))
    throw std::invalid_argument("folded projection: arguments the implicit-GEMM kernel does not take");
  // tanh and the LSTM cell exist only in the implicit GEMM's epilogue: a
  // linear layer on 1x1 rows with 16-byte output vectors, never split
  const bool special = a.act == ACT_TANH || a.act == ACT_LSTM;
  if (special && (a.k != 1 || a.H != 1 || a.W != 1 || a.cin % 8 || a.cout % 8 || a.res || a.out_f32 || !a.zeros ||
                  (reinterpret_cast<uintptr_t>(a.dst) & 15) ||
                  (a.act == ACT_LSTM && (!a.cell_out || (reinterpret_cast<uintptr_t>(a.cell_out) & 7) ||
                                         (reinterpret_cast<uintptr_t>(a.cell_in) & 7)))))
    throw std::invalid_argument("tanh / LSTM-cell epilogue: arguments the implicit-GEMM kernel does not take");
  p.srows = a.src_rows;
  p.s2rows = a.src2_rows;
  p.rrows = a.res_rows;
  p.drows = a.dst_rows;

  // 16-byte A vectors need Cin % 8 == 0, and a power-of-two Cin when the tap
  // index is split off with a shift; anything else gathers element by element
  const bool pow2 = (a.cin & (a.cin - 1)) == 0;
  const bool scalar = (a.cin % 8) != 0 || (a.k != 1 && !pow2);
  if (scalar) {
    const TileCfg c = a.cout >= 64 ? TileCfg{128, 64, 2, 2} : TileCfg{128, 32, 4, 1};
    p.mt = (p.M + c.bm - 1) / c.bm;
    p.nt = (a.cout + c.bn - 1) / c.bn;
    if (c.bn == 64) {
      if (a.k == 7) go<128, 64, 2, 2, 7, true>(p, s);
      else if (a.k == 3) go<128, 64, 2, 2, 3, true>(p, s);
      else go<128, 64, 2, 2, 1, true>(p, s);
    } else {
      if (a.k == 7) go<128, 32, 4, 1, 7, true>(p, s);
      else if (a.k == 3) go<128, 32, 4, 1, 3, true>(p, s);
      else go<128, 32, 4, 1, 1, true>(p, s);
    }
    return false;
  }
  // tile shapes follow the expected live rows (the grid covers all n)
  const int Mh = (a.nhint > 0 && a.nhint < a.n ? a.nhint : a.n) * a.Ho * a.Wo;
  // the direct-to-LDS kernel stores 8 channels per 16-byte vector
  const bool vec_out = a.cout % 8 == 0 && (reinterpret_cast<uintptr_t>(a.dst) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.res) & 15) == 0 && a.zeros != nullptr;
  // the streamed-weight halo kernel stages whole images from contiguous
  // rows: a layer with row lists takes the register-weight halo kernel
  // (image mode) or the implicit GEMM
  const bool listed = a.src_rows || a.src2_rows || a.res_rows || a.dst_rows;
  if (conv3_narrow(a, s)) return false;   // 16 / 32 channels: row lists allowed
  if (vec_out && (listed ? conv3_wres(a, s) : (conv3_wres(a, s) || conv3_halo(a, s)))) return false;
  if (vec_out) {
    // deep K on few pixels per image: K ranges of one tile on several
    // workgroups, fp32 partials summed in a fixed order by a second kernel
    // (the split depends on the layer's shape only, never on n)
    const int S = conv_ksplit(a.Ho, a.Wo, a.cout, p.K, a.out_f32 != 0);
    const bool split = S > 1 && a.splitws && !a.res_rows && !a.dst_rows && !a.kfold && !special &&
                       a.splitws_bytes >= static_cast<size_t>(S) * p.M * a.cout * sizeof(float);
    // one LDS stage on 128 x 64 tiles: a spatial layer with at least 1024
    // such tiles (and K <= 1024 for a 1x1 layer); fewer tiles wait on fewer
    // round trips in rounds of two K steps (the ResNet-50 stage-3/4 layers
    // 4-15 % faster); on 128 x 256
    // tiles (eight waves, whole 512-byte row pieces per workgroup: the
    // output-heavy layers' stores were the limit) when Cout is a multiple of
    // 256 and there are at least 512 of them (measured 4-15 % faster on the
    // ResNet-50 expansions and folded projections with 2.5 or more such
    // tiles per CU, slower with fewer)
    const long t12864 = (static_cast<long>(Mh) + 127) / 128 * ((a.cout + 63) / 64);
    const long t128256 = (static_cast<long>(Mh) + 127) / 128 * ((a.cout + 255) / 256);
    const bool one = !split && a.cout >= 64 && a.Ho * a.Wo > 1 && t12864 >= 1024 && (a.k != 1 || p.Kp <= 1024);
    const bool wide = one && a.cout % 256 == 0 && t128256 >= 512;
    const TileCfg c = split ? (a.cout % 128 == 0 ? TileCfg{128, 128, 2, 2} : TileCfg{128, 64, 2, 2})
                      : wide ? TileCfg{128, 256, 2, 4}
                      : one ? TileCfg{128, 64, 2, 2}
                            : choose_lds(Mh, a.cout, p.Kp);
    p.mt = (p.M + c.bm - 1) / c.bm;
    p.nt = (a.cout + c.bn - 1) / c.bn;
    if (split) {
      p.ksplit = S;
      p.part = a.splitws;
      if (a.k == 1)
        dispatch_lds<1>(c, p, s, S);
      else if (a.k == 3)
        dispatch_lds<3>(c, p, s, S);
      else
        dispatch_lds<7>(c, p, s, S);
      const size_t items = static_cast<size_t>(p.M) * (a.cout / 8);
      const dim3 fgrid(static_cast<unsigned>((items + 255) / 256));
      auto finish = [&](auto k) {
        hipLaunchKernelGGL(k, fgrid, dim3(256), 0, s, a.splitws, S, p.M, a.cout, a.ncount, a.n, a.Ho * a.Wo, a.scale,
                           a.shift, a.res, static_cast<uint16_t*>(a.dst));
      };
      if (a.act == ACT_RELU)
        finish(ksplit_finish_kernel<ACT_RELU>);
      else if (a.act == ACT_GELU)
        finish(ksplit_finish_kernel<ACT_GELU>);
      else
        finish(ksplit_finish_kernel<ACT_NONE>);
      return false;
    }
    if (a.gap_part && !a.out_f32 && !a.dst_rows && a.act != ACT_LSTM && a.Ho * a.Wo >= 32) p.gap = a.gap_part;
    if (a.k == 1)
      dispatch_lds<1>(c, p, s, 1, one);
    else if (a.k == 3)
      dispatch_lds<3>(c, p, s, 1, one);
    else
      dispatch_lds<7>(c, p, s, 1, one);
    return p.gap != nullptr;
  }
  const TileCfg c = a.cout >= 128 ? choose(kWide, Mh, a.cout)
                    : a.cout >= 64 ? choose(kMid, Mh, a.cout)
                                   : choose(kNarrow, Mh, a.cout);
  p.mt = (p.M + c.bm - 1) / c.bm;
  p.nt = (a.cout + c.bn - 1) / c.bn;
  if (a.k == 1)
    dispatch_staged<1>(c, p, s);
  else if (a.k == 3)
    dispatch_staged<3>(c, p, s);
  else
    dispatch_staged<7>(c, p, s);
}

}  // namespace k
}  // namespace dycl
