// bf16 implicit-GEMM convolution / linear layer for gfx950 (CDNA4).
//
// A sub-network of the compiled dynamic network is conditional-free tensor
// code (Sec. 5.3); its convolutions and linear layers are dense
// contractions:
//   y[m, co] = sum_{kh, kw, ci} x[img, oh*s - p + kh, ow*s - p + kw, ci] * w[co, kh, kw, ci]
// with m = (img, oh, ow) over the rows that are active in this branch.
// As a GEMM: M = rows * Ho * Wo, N = Cout, K = kh * kw * Cin; NHWC keeps
// the Cin run of one tap contiguous, so A is gathered in 16-byte vectors.
//
// Each 256-thread workgroup computes a BM x BN tile with four wave64s in a
// WM x WN grid, each wave accumulating 32x32 blocks with
// v_mfma_f32_32x32x16_bf16 (fp32 accumulate).  K advances 32 at a time
// through double-buffered LDS (rows padded by 16 bytes so the 16 lanes of
// a ds_read_b128 phase hit distinct banks).  The epilogue applies the
// folded BatchNorm scale / shift (or bias), the residual, ReLU or exact
// GELU, and rounds to bf16 (nearest even) or stores fp32.
#include "kernels.hpp"

namespace dycl {
namespace k {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct ConvP {
  const uint16_t* src;
  const uint16_t* src2;
  int cin1, cin2;
  int H, W, cin, Ho, Wo, cout, stride, pad;
  int M, K, Kp, cin_log2;
  const uint16_t* w;
  const float* scale;
  const float* shift;
  const uint16_t* res;
  void* dst;
  int act, out_f32;
};

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);                    // nearest, ties to even
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

__device__ __forceinline__ float apply_act(float v, int act) {
  if (act == ACT_RELU) return v > 0.f ? v : 0.f;
  if (act == ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  return v;
}

template <int BM, int BN, int WM, int WN, int KS, bool SCALAR>
__global__ __launch_bounds__(256) void conv_igemm_kernel(ConvP p) {
  constexpr int BK = kBK, LDK = BK + 8;
  constexpr int VPR = BK / 8;       // 16-byte vectors per tile row
  constexpr int RPP = 256 / VPR;    // tile rows covered by one load pass
  constexpr int PA = (BM + RPP - 1) / RPP;
  constexpr int PB = (BN + RPP - 1) / RPP;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(TM >= 1 && TN >= 1, "wave tile below 32x32");

  __shared__ __align__(16) uint16_t As[2][BM * LDK];
  __shared__ __align__(16) uint16_t Bs[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int chunk = tid % VPR, rsub = tid / VPR;
  const int HoWo = p.Ho * p.Wo;

  int a_img[PA], a_ih0[PA], a_iw0[PA];
  bool a_ok[PA];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int row = rsub + i * RPP;
    const int m = m0 + row;
    a_ok[i] = row < BM && m < p.M;
    int img = 0, oh = 0, ow = 0;
    if (a_ok[i]) {
      img = m / HoWo;
      const int rem = m - img * HoWo;
      oh = rem / p.Wo;
      ow = rem - oh * p.Wo;
    }
    a_img[i] = img;
    a_ih0[i] = oh * p.stride - p.pad;
    a_iw0[i] = ow * p.stride - p.pad;
  }

  uint4 ra[PA], rb[PB];

  auto load_tile = [&](int kt) {
    const int kidx = kt * BK + chunk * 8;
#pragma unroll
    for (int i = 0; i < PA; ++i) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (a_ok[i]) {
        if constexpr (!SCALAR) {
          if (kidx < p.K) {
            int tap = 0, ci = kidx;
            if constexpr (KS != 1) {
              tap = kidx >> p.cin_log2;
              ci = kidx & (p.cin - 1);
            }
            const int kh = tap / KS, kw = tap - (tap / KS) * KS;
            const int ih = a_ih0[i] + kh, iw = a_iw0[i] + kw;
            if ((unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W) {
              const size_t pix = ((size_t)a_img[i] * p.H + ih) * p.W + iw;
              const uint16_t* ptr =
                  ci < p.cin1 ? p.src + pix * p.cin1 + ci : p.src2 + pix * p.cin2 + (ci - p.cin1);
              v = *reinterpret_cast<const uint4*>(ptr);
            }
          }
        } else {
          uint16_t e[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            e[j] = 0;
            const int kk = kidx + j;
            if (kk < p.K) {
              const int tap = kk / p.cin;
              const int ci = kk - tap * p.cin;
              const int kh = tap / KS, kw = tap - (tap / KS) * KS;
              const int ih = a_ih0[i] + kh, iw = a_iw0[i] + kw;
              if ((unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W)
                e[j] = p.src[(((size_t)a_img[i] * p.H + ih) * p.W + iw) * p.cin + ci];
            }
          }
          v.x = e[0] | (uint32_t(e[1]) << 16);
          v.y = e[2] | (uint32_t(e[3]) << 16);
          v.z = e[4] | (uint32_t(e[5]) << 16);
          v.w = e[6] | (uint32_t(e[7]) << 16);
        }
      }
      ra[i] = v;
    }
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      const int row = rsub + i * RPP;
      if (row < BN) rb[i] = *reinterpret_cast<const uint4*>(p.w + (size_t)(n0 + row) * p.Kp + kidx);
    }
  };

  auto store_tile = [&](int buf) {
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

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const int nk = p.Kp / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile(kt + 1);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      bf16x8 af[TM], bfr[TN];
      const int koff = s * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = *reinterpret_cast<const bf16x8*>(&As[cur][(wm * WTM + a * 32 + (lane & 31)) * LDK + koff]);
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bfr[b] = *reinterpret_cast<const bf16x8*>(&Bs[cur][(wn * WTN + b * 32 + (lane & 31)) * LDK + koff]);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tile(cur ^ 1);
    __syncthreads();
  }

  // epilogue: lane owns column (lane & 31) of each 32x32 block, rows
  // 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
  for (int a = 0; a < TM; ++a) {
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int col = n0 + wn * WTN + b * 32 + (lane & 31);
      if (col >= p.cout) continue;
      const float sc = p.scale ? p.scale[col] : 1.0f;
      const float sh = p.shift ? p.shift[col] : 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * WTM + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row >= p.M) continue;
        const size_t o = (size_t)row * p.cout + col;
        float v = fmaf(acc[a][b][r], sc, sh);
        if (p.res) v += bf2f(p.res[o]);
        v = apply_act(v, p.act);
        if (p.out_f32)
          static_cast<float*>(p.dst)[o] = v;
        else
          static_cast<uint16_t*>(p.dst)[o] = f2bf(v);
      }
    }
  }
}

ConvTile conv_pick_tile(int /*M*/, int cout) {
  if (cout >= 128) return {128, 128};
  if (cout >= 64) return {128, 64};
  return {128, 32};
}

template <int BM, int BN, int WM, int WN, int KS>
static void launch_sc(dim3 grid, bool scalar, const ConvP& p, hipStream_t s) {
  if (scalar)
    hipLaunchKernelGGL((conv_igemm_kernel<BM, BN, WM, WN, KS, true>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((conv_igemm_kernel<BM, BN, WM, WN, KS, false>), grid, dim3(256), 0, s, p);
}

template <int BM, int BN, int WM, int WN>
static void launch_ks(const ConvArgs& a, const ConvP& p, hipStream_t s) {
  dim3 grid((p.M + BM - 1) / BM, (a.cout + BN - 1) / BN);
  // 16-byte A vectors need Cin % 8 == 0, and a power-of-two Cin when the
  // tap index is split off with a shift; anything else gathers by element
  const bool pow2 = (a.cin & (a.cin - 1)) == 0;
  const bool scalar = (a.cin % 8) != 0 || (a.k != 1 && !pow2);
  if (a.k == 1)
    launch_sc<BM, BN, WM, WN, 1>(grid, scalar, p, s);
  else if (a.k == 3)
    launch_sc<BM, BN, WM, WN, 3>(grid, scalar, p, s);
  else
    launch_sc<BM, BN, WM, WN, 7>(grid, scalar, p, s);
}

void conv_bf16(const ConvArgs& a, hipStream_t s) {
  ConvP p;
  p.src = a.src;
  p.src2 = a.src2;
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
  if (a.tile.bn == 128)
    launch_ks<128, 128, 2, 2>(a, p, s);
  else if (a.tile.bn == 64)
    launch_ks<128, 64, 2, 2>(a, p, s);
  else
    launch_ks<128, 32, 4, 1>(a, p, s);
}

}  // namespace k
}  // namespace dycl
