// 3x3 / stride-1 / pad-1 convolution with few channels: 16 -> 16 and 32 -> 32
// (the narrow CIFAR ResNets, e.g. SkipNet's first two stages) and the
// 8-channel (padded RGB) CIFAR stem to 16 channels.  (An 8 -> 64 stem is
// faster on the register-weight halo kernel, whose 64-channel output tile
// amortises the staged rows over four times the MFMA work.)
//
// With so few channels a layer is a stream of bytes (about 70 FLOP per
// byte): the implicit GEMM's per-tap gathers (each input pixel fetched nine
// times from L2) and its 32-wide channel tiles (half of them padding at 16
// channels) left these layers near 1.4 TB/s.  Here a workgroup walks units
// of RT output rows of one image: the unit's input rows plus a one-pixel halo
// are staged in LDS once (pixels padded to 48 or 80 bytes, so the 16 lanes
// of a read phase hit distinct banks), and every tap reads a shifted window
// of them.  All the weights live in registers (12 to 72 VGPRs per lane).
// v_mfma_f32_16x16x32_bf16 with the weights as A and pixels as B: a 32-wide
// K step is four taps of 8 channels, two of 16 or one of 32, and a lane's
// result is 4 consecutive output channels of one pixel, stored (after scale
// / shift, residual, activation, rounding) as 8-byte pieces of contiguous
// pixel rows.
// Persistent: the next unit's input rows are loaded into registers while the
// current one computes.  Images are addressed through the row lists (fused
// gate gathers / scatters) and the live count of the device host modes.
#include "kernels.hpp"

namespace dycl {
namespace k {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kNL = 3;   // 16-byte input chunks per thread and unit, at most

template <int CI, int CO, int W>
struct NarrowGeom {
  static constexpr int WB = W / 16;              // 16-pixel blocks per row
  static constexpr int RPW = 2 / WB;             // rows per wave
  static constexpr int RT = 4 * RPW;             // output rows per unit
  static constexpr int PR = RT + 2;              // staged rows
  static constexpr int PWX = W + 2;              // staged pixels per row
  // bytes per staged pixel: 16 consecutive pixels of one read phase hit
  // distinct banks (16 B pixels are contiguous; 48 and 80 B pixels are
  // 12 and 20 words apart)
  static constexpr int PS = CI == 8 ? 16 : CI == 16 ? 48 : 80;
  static constexpr int CB = CO / 16;             // 16-channel output blocks
  static constexpr int CH = CI / 8;              // 16-byte chunks per input pixel
  static constexpr int TPS = 32 / CI;            // taps per 32-wide K step
  static constexpr int KSTEPS = (9 * CI + 31) / 32;
  static constexpr int CHUNKS = PR * W * CH;     // chunks per unit
  static constexpr int BYTES = PR * PWX * PS;
  static_assert(CHUNKS <= 256 * kNL, "input chunks per unit");
};

struct NarrowP {
  const uint16_t* x;
  const uint16_t* w;   // [cout_pad][Kp], K = tap * CI + ci
  int Kp;
  const float* scale;
  const float* shift;
  const uint16_t* res;
  uint16_t* y;
  int n, H;
  const int32_t* nc;
  const int32_t* srows;   // image lists (null: identity)
  const int32_t* rrows;
  const int32_t* drows;
  int act;
};

template <int ACT>
__device__ __forceinline__ float narrow_act(float v) {
  if (ACT == ACT_RELU) return v > 0.f ? v : 0.f;
  if (ACT == ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  return v;
}

template <int CI, int CO, int W, int ACT, bool RES>
__global__ __launch_bounds__(256) void conv3n_kernel(NarrowP p) {
  using G = NarrowGeom<CI, CO, W>;
  __shared__ __align__(16) char pl[G::BYTES];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int n = p.nc ? min(*p.nc, p.n) : p.n;
  const int RG = (p.H + G::RT - 1) / G::RT;
  const int units = n * RG;
  if (static_cast<int>(blockIdx.x) >= units) return;   // uniform over the workgroup

  // weights: lane holds output channel 16 cb + l16 at K 32 s + 8 g .. + 7
  bf16x8 wr[G::CB][G::KSTEPS];
#pragma unroll
  for (int cb = 0; cb < G::CB; ++cb)
#pragma unroll
    for (int s = 0; s < G::KSTEPS; ++s)
      wr[cb][s] = *reinterpret_cast<const bf16x8*>(p.w + static_cast<size_t>(cb * 16 + l16) * p.Kp + s * 32 + g * 8);
  float4 sc[G::CB], sh[G::CB];   // channels 16 cb + 4 g .. + 3
#pragma unroll
  for (int cb = 0; cb < G::CB; ++cb) {
    const int c0 = cb * 16 + 4 * g;
    sc[cb] = p.scale ? *reinterpret_cast<const float4*>(p.scale + c0) : make_float4(1.f, 1.f, 1.f, 1.f);
    sh[cb] = p.shift ? *reinterpret_cast<const float4*>(p.shift + c0) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  // the halo columns are zero for every unit (data never lands there)
  for (int r = tid; r < G::PR * 2; r += 256) {
    char* px = pl + ((r >> 1) * G::PWX + ((r & 1) ? W + 1 : 0)) * G::PS;
#pragma unroll
    for (int c = 0; c < G::CH; ++c) *reinterpret_cast<uint4*>(px + c * 16) = make_uint4(0, 0, 0, 0);
  }

  // B operand offsets (bytes in the staged rows) of this lane's taps: step
  // s, lane group g: tap TPS s + g / CH, channels 8 (g % CH) .. + 7 (K is
  // tap-major, so these are the lane's K values 32 s + 8 g ..); a tap past
  // the ninth reads a halo pixel, which is zero
  int toff[G::KSTEPS];
#pragma unroll
  for (int s = 0; s < G::KSTEPS; ++s) {
    const int tap = G::TPS * s + g / G::CH, ch = g % G::CH;
    toff[s] = tap < 9 ? ((tap / 3) * G::PWX + (tap % 3)) * G::PS + ch * 16 : -1;
  }

  // staging: chunk q = tid + 256 i of the unit's rows (16 bytes of channels
  // of one pixel); its source offset within the image and its LDS offset
  int crow[kNL], csrc[kNL], clds[kNL];
#pragma unroll
  for (int i = 0; i < kNL; ++i) {
    const int q = tid + 256 * i, pr = q / (W * G::CH), rem = q - pr * (W * G::CH);
    const int px = rem / G::CH, c = rem - px * G::CH;
    crow[i] = q < G::CHUNKS ? pr : -0x40000000;
    csrc[i] = (pr * W + px) * CI + c * 8;
    clds[i] = (pr * G::PWX + px + 1) * G::PS + c * 16;
  }
  uint4 raw[kNL];
  bool inside[kNL];
  auto load = [&](int t) {
    const int img = t / RG, oh0 = (t - img * RG) * G::RT;
    const int simg = p.srows ? p.srows[img] : img;
    const int64_t base = (static_cast<int64_t>(simg) * p.H + oh0 - 1) * W * CI;
#pragma unroll
    for (int i = 0; i < kNL; ++i) {
      const int ih = oh0 - 1 + crow[i];
      inside[i] = ih >= 0 && ih < p.H;
      raw[i] = *reinterpret_cast<const uint4*>(p.x + (inside[i] ? base + csrc[i] : 0));
    }
  };
  int t = blockIdx.x;
  load(t);

  while (true) {
    __syncthreads();   // the previous unit's MFMAs are done with the staged rows
#pragma unroll
    for (int i = 0; i < kNL; ++i)
      if (crow[i] >= 0) *reinterpret_cast<uint4*>(pl + clds[i]) = inside[i] ? raw[i] : make_uint4(0, 0, 0, 0);
    __syncthreads();
    const int tn = t + gridDim.x;
    if (tn < units) load(tn);   // lands while this unit computes

    const int img = t / RG, oh0 = (t - img * RG) * G::RT;
    const int rimg = p.rrows ? p.rrows[img] : img, dimg = p.drows ? p.drows[img] : img;
#pragma unroll
    for (int rr = 0; rr < G::RPW; ++rr) {
      const int lr = wave * G::RPW + rr, oh = oh0 + lr;
      f32x4 acc[G::WB][G::CB];
#pragma unroll
      for (int b = 0; b < G::WB; ++b)
#pragma unroll
        for (int cb = 0; cb < G::CB; ++cb) acc[b][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < G::KSTEPS; ++s) {
#pragma unroll
        for (int b = 0; b < G::WB; ++b) {
          const int o = toff[s] >= 0 ? (lr * G::PWX + b * 16 + l16) * G::PS + toff[s] : 0;
          const bf16x8 xf = *reinterpret_cast<const bf16x8*>(pl + o);
#pragma unroll
          for (int cb = 0; cb < G::CB; ++cb)
            acc[b][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wr[cb][s], xf, acc[b][cb], 0, 0, 0);
        }
      }
      if (oh < p.H) {
#pragma unroll
        for (int b = 0; b < G::WB; ++b) {
          const size_t pix = static_cast<size_t>(oh) * W + b * 16 + l16;
#pragma unroll
          for (int cb = 0; cb < G::CB; ++cb) {
            const int c0 = cb * 16 + 4 * g;
            float v[4] = {fmaf(acc[b][cb][0], sc[cb].x, sh[cb].x), fmaf(acc[b][cb][1], sc[cb].y, sh[cb].y),
                          fmaf(acc[b][cb][2], sc[cb].z, sh[cb].z), fmaf(acc[b][cb][3], sc[cb].w, sh[cb].w)};
            if (RES) {
              const uint2 rv = *reinterpret_cast<const uint2*>(p.res + (static_cast<size_t>(rimg) * p.H * W + pix) * CO + c0);
              v[0] += __uint_as_float(rv.x << 16);
              v[1] += __uint_as_float(rv.x & 0xffff0000u);
              v[2] += __uint_as_float(rv.y << 16);
              v[3] += __uint_as_float(rv.y & 0xffff0000u);
            }
            // v_cvt_pk_bf16_f32: round to nearest even, as the other kernels' epilogues
            const bf16x2 lo = {static_cast<__bf16>(narrow_act<ACT>(v[0])), static_cast<__bf16>(narrow_act<ACT>(v[1]))};
            const bf16x2 hi = {static_cast<__bf16>(narrow_act<ACT>(v[2])), static_cast<__bf16>(narrow_act<ACT>(v[3]))};
            *reinterpret_cast<uint2*>(p.y + (static_cast<size_t>(dimg) * p.H * W + pix) * CO + c0) =
                make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
          }
        }
      }
    }
    if (tn >= units) break;
    t = tn;
  }
}

template <int CI, int CO, int W>
void go(const NarrowP& p, hipStream_t s) {
  const int RG = (p.H + NarrowGeom<CI, CO, W>::RT - 1) / NarrowGeom<CI, CO, W>::RT;
  const long units = static_cast<long>(p.n) * RG;
  // the workgroups the CUs hold at once (registers: five per CU with the
  // small weight sets, three with 32 -> 32)
  const long resident = (CI * CO <= 256 ? 5 : 3) * 256;
  const int grid = static_cast<int>(units < resident ? units : resident);
  auto launch = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, s, p); };
  const bool res = p.res != nullptr;
  if (p.act == ACT_RELU)
    res ? launch(conv3n_kernel<CI, CO, W, ACT_RELU, true>) : launch(conv3n_kernel<CI, CO, W, ACT_RELU, false>);
  else if (p.act == ACT_GELU)
    res ? launch(conv3n_kernel<CI, CO, W, ACT_GELU, true>) : launch(conv3n_kernel<CI, CO, W, ACT_GELU, false>);
  else
    res ? launch(conv3n_kernel<CI, CO, W, ACT_NONE, true>) : launch(conv3n_kernel<CI, CO, W, ACT_NONE, false>);
}

}  // namespace

bool conv3_narrow(const ConvArgs& a, hipStream_t s) {
  const int CI = a.cin, CO = a.cout;
  const bool pair = (CI == 16 && CO == 16) || (CI == 32 && CO == 32) || (CI == 8 && CO == 16);
  if (a.k != 3 || a.stride != 1 || a.pad != 1 || a.src2 || a.out_f32 || a.pool || !pair || (a.W != 16 && a.W != 32) ||
      a.Ho != a.H || a.Wo != a.W || a.H < 1 || a.Kp < ((9 * CI + 31) / 32) * 32)
    return false;
  if ((reinterpret_cast<uintptr_t>(a.src) | reinterpret_cast<uintptr_t>(a.dst) | reinterpret_cast<uintptr_t>(a.res) |
       reinterpret_cast<uintptr_t>(a.w) | reinterpret_cast<uintptr_t>(a.scale) | reinterpret_cast<uintptr_t>(a.shift)) &
      15)
    return false;
  NarrowP p;
  p.x = a.src;
  p.w = a.w;
  p.Kp = a.Kp;
  p.scale = a.scale;
  p.shift = a.shift;
  p.res = a.res;
  p.y = static_cast<uint16_t*>(a.dst);
  p.n = a.n;
  p.H = a.H;
  p.nc = a.ncount;
  p.srows = a.src_rows;
  p.rrows = a.res_rows;
  p.drows = a.dst_rows;
  p.act = a.act;
  if (CI == 16)
    a.W == 32 ? go<16, 16, 32>(p, s) : go<16, 16, 16>(p, s);
  else if (CI == 32)
    a.W == 32 ? go<32, 32, 32>(p, s) : go<32, 32, 16>(p, s);
  else
    a.W == 32 ? go<8, 16, 32>(p, s) : go<8, 16, 16>(p, s);
  return true;
}

}  // namespace k
}  // namespace dycl
