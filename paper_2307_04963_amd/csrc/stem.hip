// 7x7 stride-2 convolution of a 3-channel (RGB) image batch: the stem of
// the ImageNet ResNets.
//
// The generic implicit GEMM gathers A in 16-byte vectors of one tap's input
// channels, which a 3-channel input cannot supply; padding the input to 8
// channels costs an extra pass over it and makes 5 of every 8 K values
// zeros.  Here K is arranged per kernel row instead: one row of the window
// is 7 pixels of 3 channels, stored in LDS as 8-byte pixels (the fourth
// channel zero), so a 32-wide K step of v_mfma_f32_16x16x32_bf16 is one
// kernel row (8 pixel slots, the last reading zeros), and each lane's 8 K
// values are two adjacent pixels.  The 7x7 window takes 7 such steps (K 224
// for the 147 real values, against 448 with 8 padded channels).
//
// Work unit: 4 output rows of one image, one row per wave.  The workgroup
// stages the input rows those outputs read (with zero padding around them)
// in LDS, converting 3 to 4 channels on the way, and keeps the layer's
// weights in LDS, rearranged once per workgroup from the common packed
// [cout_pad][Kp] layout into MFMA fragments.  The kernel is persistent:
// the input rows of the next unit are loaded into registers while the
// current unit computes.  Units are dealt XCD by XCD, so that neighbouring
// units, which share input rows, run under one L2.
//
// The weights are the MFMA's A operand and the pixels its B operand, so that
// each lane's accumulator holds 4 consecutive output channels of one pixel:
// the epilogue (folded BatchNorm, ReLU / GELU, round to bf16 with
// v_cvt_pk_bf16_f32) writes them as 8-byte vectors to a per-wave staging
// block, and each output row leaves in 2 KB runs of whole pixels.
//
// Measured on the ResNet-50 stem at batch 256 (224 x 224 -> 112 x 112): the
// epilogue (conversion and 411 MB of stores) takes about half the time, the
// MFMA loop and the staging of the input rows the other half.
#include "kernels.hpp"

namespace dycl {
namespace k {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

constexpr int kRows = 4;       // output rows per unit (one per wave)
constexpr int kCout = 64;      // output channels: four 16-wide MFMA blocks
constexpr int kEStride = 72;   // staging row (one pixel): 64 channels + 8, in u16
constexpr int kPairsPerThread = 6;   // input pixel pairs each thread stages per unit

struct alignas(4) U3 {
  uint32_t a, b, c;   // two pixels of 3 bf16 channels
};

template <int KS, int S, int MB, bool POOL>
struct StemGeom {
  static constexpr int PR = (kRows - 1) * S + KS;   // input rows of a unit
  static constexpr int PW = 16 * MB * S + 16;       // staged pixels per row (8 bytes each)
  static constexpr int W_BYTES = KS * 4 * 64 * 16;  // [kh][channel block][lane] 16-byte fragments
  static constexpr int S_BYTES = 2 * kCout * 4;       // scale, shift
  // pooled: the unit's four row maxima over pixel triples ([row][pooled
  // pixel][64 channels] bf16) take the staged input rows' place once the
  // MFMAs are done; the carried row (the previous unit's last) has its own
  static constexpr int WP = 8 * MB;                  // pooled pixels per row, at most
  static constexpr int HP_BYTES = POOL ? kRows * WP * kCout * 2 : 0;
  static constexpr int C_BYTES = POOL ? WP * kCout * 2 : 0;
  static constexpr int P_BYTES = PR * PW * 8 > HP_BYTES ? PR * PW * 8 : HP_BYTES;
  // staging blocks per wave: two (alternating) when stored, one when pooled
  static constexpr int E_BYTES = kRows * (POOL ? 1 : 2) * 16 * kEStride * 2;
  static constexpr int BYTES = W_BYTES + P_BYTES + E_BYTES + C_BYTES + S_BYTES;
};

struct StemP {
  const uint16_t* x;   // [n][H][W][3]
  const uint16_t* w;   // [cout_pad][Kp], K order (kh, kw, c)
  int Kp;
  const float* scale;
  const float* shift;
  uint16_t* y;         // [n][Ho][Wo][64], or pooled: [n][Hp][Wp][64]
  int n, H, W, Ho, Wo, pad, off, act;
  int units, per_xcd; // units = n * ceil(Ho / 4); per_xcd = ceil(units / 8)
  int Hp, Wp;          // pooled output (3x3 / stride 2 / pad 1 max-pool)
  int parts, ranges;   // pooled: each image's units in `parts` consecutive ranges
};

// the larger of two non-negative bf16 values is the one with the larger
// bits: element-wise maxima of 8 bf16 by 16-bit integer maxima.  The pooled
// path works on vector types throughout: with the struct type uint4, a
// choice between a loaded value and a constant became a choice between
// addresses, i.e. a generic (flat) load, whose wait also waited for the
// next unit's input loads in flight
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4 max_bf16x8(u32x4 a, u32x4 b) {
  return __builtin_bit_cast(u32x4, __builtin_elementwise_max(__builtin_bit_cast(u16x8, a), __builtin_bit_cast(u16x8, b)));
}

template <int ACT>
__device__ __forceinline__ float act_of(float v) {
  if (ACT == ACT_RELU) return v > 0.f ? v : 0.f;
  if (ACT == ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  return v;
}

// the u-th unit slot of the dispatch order: slot u runs on XCD u % 8 and
// takes the (u / 8)-th unit of that XCD's contiguous range (or none)
__device__ __forceinline__ int unit_of(int u, const StemP& p) {
  const int t = (u & 7) * p.per_xcd + (u >> 3);
  return (u >> 3) < p.per_xcd && t < p.units ? t : -1;
}

// The units a workgroup computes, in order.  Stored output: the unit slots
// of unit_of.  Pooled output: ranges r = blockIdx.x, + gridDim.x, ... of
// consecutive units of one image, walked in order so that a unit's last
// stem row (the first pooled row of the next unit needs it) stays in LDS; a
// range that starts inside an image first recomputes the unit before it,
// only to fill that carried row.
struct StemWork {
  int t;          // unit (image * units per image + row group)
  int slot;       // stored output: dispatch slot
  int r, j, j1;   // pooled output: range, row group, end of the range's row groups
  bool pre;       // pooled output: computed only for the carried row
};

template <bool POOL>
__device__ __forceinline__ bool stem_first(int start, const StemP& p, int RG, StemWork& w) {
  if constexpr (POOL) {
    if (start >= p.ranges) return false;
    const int img = start / p.parts, part = start - img * p.parts;
    const int j0 = part * RG / p.parts;
    w.r = start;
    w.j1 = (part + 1) * RG / p.parts;
    w.pre = j0 > 0;
    w.j = j0 > 0 ? j0 - 1 : j0;
    w.t = img * RG + w.j;
    return true;
  } else {
    const int slots = 8 * p.per_xcd;
    for (int u = start; u < slots; u += gridDim.x) {
      const int t = unit_of(u, p);
      if (t >= 0) {
        w.slot = u;
        w.t = t;
        return true;
      }
    }
    return false;
  }
}

template <bool POOL>
__device__ __forceinline__ bool stem_next(const StemWork& cur, const StemP& p, int RG, StemWork& w) {
  if constexpr (POOL) {
    if (cur.j + 1 < cur.j1) {
      w = cur;
      w.pre = false;
      ++w.j;
      ++w.t;
      return true;
    }
    return stem_first<true>(cur.r + gridDim.x, p, RG, w);
  } else {
    return stem_first<false>(cur.slot + gridDim.x, p, RG, w);
  }
}

template <int KS, int S, int MB, int ACT, bool POOL>
__global__ __launch_bounds__(256, 2) void stem_rgb_kernel(StemP p) {
  constexpr int NP = kPairsPerThread;
  using G = StemGeom<KS, S, MB, POOL>;
  static_assert(!POOL || ACT == ACT_RELU, "pooled maxima are taken on the bits of non-negative bf16 values");
  __shared__ __align__(16) char smem[G::BYTES];
  char* const wl = smem;
  char* const pl = smem + G::W_BYTES;
  uint16_t* const el = reinterpret_cast<uint16_t*>(smem + G::W_BYTES + G::P_BYTES);
  uint16_t* const cl = reinterpret_cast<uint16_t*>(smem + G::W_BYTES + G::P_BYTES + G::E_BYTES);   // carried row
  float* const ss = reinterpret_cast<float*>(smem + G::W_BYTES + G::P_BYTES + G::E_BYTES + G::C_BYTES);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int RG = (p.Ho + kRows - 1) / kRows;

  StemWork cur;
  if (!stem_first<POOL>(blockIdx.x, p, RG, cur)) return;   // uniform over the workgroup

  // weights: fragment (kh, channel block cb, lane) holds output channel
  // 16 cb + l16 at K values (kw, c) = (2 g + j / 4, j % 4), j < 8 (zero
  // where kw >= KS or c == 3)
  for (int e = tid; e < KS * 4 * 64; e += 256) {
    const int kh = e >> 8, cb = (e >> 6) & 3, l = e & 63;
    const uint16_t* wr = p.w + static_cast<size_t>(cb * 16 + (l & 15)) * p.Kp + kh * KS * 3;
    uint16_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kw = 2 * (l >> 4) + (j >> 2), c = j & 3;
      v[j] = (kw < KS && c < 3) ? wr[kw * 3 + c] : uint16_t(0);
    }
    uint4 q;
    q.x = v[0] | (uint32_t(v[1]) << 16);
    q.y = v[2] | (uint32_t(v[3]) << 16);
    q.z = v[4] | (uint32_t(v[5]) << 16);
    q.w = v[6] | (uint32_t(v[7]) << 16);
    *reinterpret_cast<uint4*>(wl + e * 16) = q;
  }
  // staged pixels outside [off, off + W) are the zero padding of every unit
  for (int e = tid; e < G::PR * G::PW; e += 256) {
    const int pc = e % G::PW;
    if (pc < p.off || pc >= p.off + p.W) *reinterpret_cast<uint2*>(pl + e * 8) = make_uint2(0, 0);
  }
  if (tid < kCout)
    ss[tid] = p.scale ? p.scale[tid] : 1.0f;
  else if (tid < 2 * kCout)
    ss[tid] = p.shift ? p.shift[tid - kCout] : 0.0f;

  // staging: thread tid takes pixel pairs q = tid + 256 i of the unit's input
  // rows (row pr = q / (W / 2)): 12 bytes in, one 16-byte LDS write out, so
  // a wave reads 768 contiguous bytes and writes 1 KB with no bank conflict.
  // The pairs' offsets are the same for every unit: packed per pair as
  // row (5 bits; 31: no pair), first pixel within the unit's rows (12 bits)
  // and LDS position in 16-byte units (11 bits).
  static_assert(G::PR < 31 && G::PR * G::PW / 2 < 2048, "pair fields");
  const int pairs = G::PR * (p.W >> 1);
  uint32_t pinfo[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int q = tid + 256 * i, pr = q / (p.W >> 1), cp = q - pr * (p.W >> 1);
    pinfo[i] = q < pairs ? pr | (pr * p.W + 2 * cp) << 5 | ((pr * G::PW + p.off + 2 * cp) / 2) << 17 : 31u;
  }
  // B fragment addresses (LDS bytes from the staged rows, kernel row 0): pixel
  // 16 mb + l16 of this wave's output row, taps kw = 2 g and 2 g + 1; a tap
  // past the window reads the last staged pixel of the row, which is always
  // padding (zero), so no input value enters through a zero weight
  int alo[MB], ahi[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int row0 = wave * S * G::PW;
    const int pc = (mb * 16 + l16) * S - p.pad + p.off + 2 * g;
    alo[mb] = (row0 + (2 * g < KS ? pc : G::PW - 1)) * 8;
    ahi[mb] = (row0 + (2 * g + 1 < KS ? pc + 1 : G::PW - 1)) * 8;
  }

  // every thread loads unconditionally (a pair outside the image reads the
  // batch's first pair instead and is staged as zeros), so the loads land
  // straight in the registers the next unit stages from
  U3 raw[NP];
  bool inside[NP];
  auto load = [&](int t) {
    const int img = t / RG, ih0 = (t - img * RG) * kRows * S - p.pad;
    const int64_t base = (static_cast<int64_t>(img) * p.H + ih0) * p.W * 3;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int pr = pinfo[i] & 31, ih = ih0 + pr;
      inside[i] = pr != 31 && ih >= 0 && ih < p.H;
      raw[i] = *reinterpret_cast<const U3*>(p.x + (inside[i] ? base + 3 * ((pinfo[i] >> 5) & 4095) : 0));
    }
  };
  load(cur.t);

  while (true) {
    __syncthreads();   // the previous unit's MFMAs are done with the staged rows
    // 2 pixels of 3 channels (3 words) -> 2 pixels of 4 channels (4 words)
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      if ((pinfo[i] & 31) != 31) {
        uint4 o;
        o.x = raw[i].a;
        o.y = raw[i].b & 0xffffu;
        o.z = (raw[i].b >> 16) | (raw[i].c << 16);
        o.w = raw[i].c >> 16;
        *reinterpret_cast<uint4*>(pl + (pinfo[i] >> 17) * 16) = inside[i] ? o : make_uint4(0, 0, 0, 0);
      }
    }
    if constexpr (POOL) {   // the previous unit's pooled rows overwrote the padding
      const int npad = G::PW - p.W;
      for (int e = tid; e < G::PR * npad; e += 256) {
        const int pr = e / npad, k = e - pr * npad;
        *reinterpret_cast<uint2*>(pl + (pr * G::PW + (k < p.off ? k : p.W + k)) * 8) = make_uint2(0, 0);
      }
    }
    __syncthreads();

    StemWork nxt;
    const bool more = stem_next<POOL>(cur, p, RG, nxt);
    if (more) load(nxt.t);   // lands while this unit computes

    f32x4 acc[MB][4];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) acc[mb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
    for (int kh = 0; kh < KS; ++kh) {
      bf16x8 wf[4];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) wf[cb] = *reinterpret_cast<const bf16x8*>(wl + ((kh * 4 + cb) * 64 + lane) * 16);
      const char* const row = pl + kh * G::PW * 8;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const uint2 lo = *reinterpret_cast<const uint2*>(row + alo[mb]);
        const uint2 hi = *reinterpret_cast<const uint2*>(row + ahi[mb]);
        uint4 v;
        v.x = lo.x;
        v.y = lo.y;
        v.z = hi.x;
        v.w = hi.y;
        const bf16x8 xf = __builtin_bit_cast(bf16x8, v);
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
          acc[mb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[cb], xf, acc[mb][cb], 0, 0, 0);
      }
    }

    // epilogue: lane holds channels 16 cb + 4 g + i of pixel 16 mb + l16.
    // Stored: each 16-pixel block goes through one of two per-wave staging
    // buffers (alternating, so a block's writes never wait for the previous
    // block's reads) and leaves as 2 KB of whole pixels.  Pooled: through
    // the wave's one staging buffer into the maxima over pixel triples.
    const int img = cur.t / RG, oh = (cur.t - img * RG) * kRows + wave;
    float4 sc[4], sh[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      sc[cb] = *reinterpret_cast<const float4*>(ss + cb * 16 + 4 * g);
      sh[cb] = *reinterpret_cast<const float4*>(ss + kCout + cb * 16 + 4 * g);
    }
    if constexpr (POOL) {
      // maxima over pixel triples: lane (t8, q) takes pooled pixel 8 mb + t8
      // (output columns 16 mb + 2 t8 - 1 .. + 1) and channels 8 q .. 8 q + 7;
      // columns outside the output, and rows past it, enter as 0, the
      // identity of a maximum of ReLU outputs
      uint16_t* const ew = el + wave * 16 * kEStride;
      uint16_t* const hp = reinterpret_cast<uint16_t*>(pl);   // [kRows][WP][64]
      const int t8 = lane >> 3, q = lane & 7;
      const u32x4 zero = {0u, 0u, 0u, 0u};
      u32x4 prev = zero;   // the previous block's pixel 15
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          const float a0 = act_of<ACT>(fmaf(acc[mb][cb][0], sc[cb].x, sh[cb].x));
          const float a1 = act_of<ACT>(fmaf(acc[mb][cb][1], sc[cb].y, sh[cb].y));
          const float a2 = act_of<ACT>(fmaf(acc[mb][cb][2], sc[cb].z, sh[cb].z));
          const float a3 = act_of<ACT>(fmaf(acc[mb][cb][3], sc[cb].w, sh[cb].w));
          const bf16x2 lo = {static_cast<__bf16>(a0), static_cast<__bf16>(a1)};
          const bf16x2 hi = {static_cast<__bf16>(a2), static_cast<__bf16>(a3)};
          *reinterpret_cast<uint2*>(ew + l16 * kEStride + cb * 16 + 4 * g) =
              make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        const int c1 = 2 * t8;
        const u32x4 center = *reinterpret_cast<const u32x4*>(ew + c1 * kEStride + q * 8);
        const u32x4 right = *reinterpret_cast<const u32x4*>(ew + (c1 + 1) * kEStride + q * 8);
        const u32x4 lft = *reinterpret_cast<const u32x4*>(ew + (t8 > 0 ? c1 - 1 : 0) * kEStride + q * 8);
        const u32x4 left = t8 > 0 ? lft : prev;
        const u32x4 last = *reinterpret_cast<const u32x4*>(ew + 15 * kEStride + q * 8);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // reads done before the next block's staging
        const int ow = mb * 16 + c1;
        u32x4 m = ow < p.Wo ? center : zero;
        if (ow + 1 < p.Wo) m = max_bf16x8(m, right);
        if (ow >= 1 && ow - 1 < p.Wo) m = max_bf16x8(m, left);
        if (oh >= p.Ho) m = zero;
        *reinterpret_cast<u32x4*>(hp + (wave * G::WP + mb * 8 + t8) * kCout + q * 8) = m;
        prev = last;
      }
      __syncthreads();   // every row's maxima are in LDS
      // pooled rows 2 j (stem rows 4 j - 1 .. 4 j + 1: the carried row and
      // the unit's first two) and 2 j + 1 (stem rows 4 j + 1 .. 4 j + 3)
      const int j = cur.j, WP8 = p.Wp * 8;
      if (!cur.pre) {
        for (int e = tid; e < 2 * WP8; e += 256) {
          const int pr = e >= WP8 ? 1 : 0, rem = e - pr * WP8, pw = rem >> 3, qq = rem & 7;
          const int po = 2 * j + pr;
          if (po >= p.Hp) continue;
          const int o = pw * kCout + qq * 8;
          const u32x4 r1 = *reinterpret_cast<const u32x4*>(hp + (pr * 2) * G::WP * kCout + o);
          const u32x4 r2 = *reinterpret_cast<const u32x4*>(hp + (pr * 2 + 1) * G::WP * kCout + o);
          const u32x4 ra = *reinterpret_cast<const u32x4*>(hp + G::WP * kCout + o);
          const u32x4 rc = *reinterpret_cast<const u32x4*>(cl + o);
          const u32x4 r0 = pr ? ra : (j > 0 ? rc : zero);
          *reinterpret_cast<u32x4*>(p.y + ((static_cast<size_t>(img) * p.Hp + po) * p.Wp + pw) * kCout + qq * 8) =
              max_bf16x8(max_bf16x8(r0, r1), r2);
        }
      }
      __syncthreads();   // the carried row is read
      for (int e = tid; e < WP8; e += 256)   // the unit's last stem row is carried
        *reinterpret_cast<u32x4*>(cl + e * 8) = *reinterpret_cast<const u32x4*>(hp + 3 * G::WP * kCout + e * 8);
    } else {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        uint16_t* const ew = el + (wave * 2 + (mb & 1)) * 16 * kEStride;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          const float a0 = act_of<ACT>(fmaf(acc[mb][cb][0], sc[cb].x, sh[cb].x));
          const float a1 = act_of<ACT>(fmaf(acc[mb][cb][1], sc[cb].y, sh[cb].y));
          const float a2 = act_of<ACT>(fmaf(acc[mb][cb][2], sc[cb].z, sh[cb].z));
          const float a3 = act_of<ACT>(fmaf(acc[mb][cb][3], sc[cb].w, sh[cb].w));
          // v_cvt_pk_bf16_f32: round to nearest even, as the other kernels' epilogues
          const bf16x2 lo = {static_cast<__bf16>(a0), static_cast<__bf16>(a1)};
          const bf16x2 hi = {static_cast<__bf16>(a2), static_cast<__bf16>(a3)};
          *reinterpret_cast<uint2*>(ew + l16 * kEStride + cb * 16 + 4 * g) =
              make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        // lanes 16 apart take the four quarters of one pixel, so that each
        // 16-lane phase of the read covers the 64 banks once
        const int px = lane & 15, ow = mb * 16 + px;
        const uint4* sp = reinterpret_cast<const uint4*>(ew + px * kEStride + (lane >> 4) * 16);
        const uint4 v0 = sp[0], v1 = sp[1];
        if (oh < p.Ho && ow < p.Wo) {
          uint4* d = reinterpret_cast<uint4*>(p.y + ((static_cast<size_t>(img) * p.Ho + oh) * p.Wo + ow) * kCout +
                                              (lane >> 4) * 16);
          d[0] = v0;
          d[1] = v1;
        }
      }
    }
    if (!more) break;
    cur = nxt;
  }
}

template <int KS, int S, int MB>
bool go(const StemP& p, hipStream_t s) {
  using G = StemGeom<KS, S, MB, false>;
  if (p.off + p.W >= G::PW || G::PR * (p.W / 2) > 256 * kPairsPerThread) return false;
  if (p.Hp) {   // pooled: ReLU only (maxima on the bits of non-negative values)
    if (p.act != ACT_RELU) return false;
    const int grid = p.ranges < 2 * 256 ? p.ranges : 2 * 256;
    hipLaunchKernelGGL((stem_rgb_kernel<KS, S, MB, ACT_RELU, true>), dim3(grid), dim3(256), 0, s, p);
    return true;
  }
  int grid = 2 * 256;   // two workgroups per CU (about 62 KB of LDS each at 7x7)
  const int need = (p.units + 7) / 8 * 8;
  if (need < grid) grid = need;
  if (p.act == ACT_RELU)
    hipLaunchKernelGGL((stem_rgb_kernel<KS, S, MB, ACT_RELU, false>), dim3(grid), dim3(256), 0, s, p);
  else if (p.act == ACT_GELU)
    hipLaunchKernelGGL((stem_rgb_kernel<KS, S, MB, ACT_GELU, false>), dim3(grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((stem_rgb_kernel<KS, S, MB, ACT_NONE, false>), dim3(grid), dim3(256), 0, s, p);
  return true;
}

}  // namespace

// 3x3 stride-1 stems (CIFAR) are left to the 8-channel path: with a third of
// each K step used they measured slower than it, padding pass included
bool conv_rgb_stem_fits(int H, int W, int cin, int cout, int k, int stride, int pad) {
  if (cin != 3 || cout != kCout || W % 8 != 0 || pad < 0 || pad > k / 2) return false;
  if (k != 7 || stride != 2) return false;
  const int Ho = (H + 2 * pad - k) / stride + 1, Wo = (W + 2 * pad - k) / stride + 1;
  if (Ho < 1 || Wo < 1 || Wo > 112) return false;
  const int MB = Wo <= 32 ? 2 : Wo <= 64 ? 4 : 7;
  const int PR = (kRows - 1) * stride + k, PW = 16 * MB * stride + 16;
  // the last staged pixel of each row stays padding
  return (pad + (pad & 1)) + W < PW && PR * (W / 2) <= 256 * kPairsPerThread;
}

bool conv_rgb_stem(const ConvArgs& a, hipStream_t s) {
  const bool aligned = (reinterpret_cast<uintptr_t>(a.src) | reinterpret_cast<uintptr_t>(a.dst)) % 16 == 0;
  if (!aligned || a.src2 || a.cin1 != 3 || a.res || a.out_f32 || a.ncount || a.src_rows || a.res_rows || a.dst_rows ||
      !conv_rgb_stem_fits(a.H, a.W, a.cin, a.cout, a.k, a.stride, a.pad) || (a.pool && a.act != ACT_RELU))
    return false;
  StemP p;
  p.x = a.src;
  p.w = a.w;
  p.Kp = a.Kp;
  p.scale = a.scale;
  p.shift = a.shift;
  p.y = static_cast<uint16_t*>(a.dst);
  p.n = a.n;
  p.H = a.H;
  p.W = a.W;
  p.Ho = a.Ho;
  p.Wo = a.Wo;
  p.pad = a.pad;
  p.off = a.pad + (a.pad & 1);   // even: every 8-pixel run lands on a 16-byte boundary
  p.act = a.act;
  p.units = a.n * ((a.Ho + kRows - 1) / kRows);
  p.per_xcd = (p.units + 7) / 8;
  p.Hp = p.Wp = p.parts = p.ranges = 0;
  if (a.pool) {
    // pooled output: each image's row groups in consecutive ranges, enough
    // ranges for two workgroups per CU (a range inside an image recomputes
    // one row group)
    const int RG = (a.Ho + kRows - 1) / kRows;
    p.Hp = (a.Ho - 1) / 2 + 1;
    p.Wp = (a.Wo - 1) / 2 + 1;
    p.parts = (2 * 256 + a.n - 1) / a.n;
    if (p.parts > RG) p.parts = RG;
    p.ranges = a.n * p.parts;
  }
  const int MB = a.Wo <= 32 ? 2 : a.Wo <= 64 ? 4 : 7;
  return MB == 2 ? go<7, 2, 2>(p, s) : MB == 4 ? go<7, 2, 4>(p, s) : go<7, 2, 7>(p, s);
}

}  // namespace k
}  // namespace dycl
