// Persistent bounded loop of an adaptive-computation-time network: every
// step of the loop in one cooperative launch (Sec. 2.2: a loop with a
// constant maximum step count; the host program keeps no per-step work,
// cf. the host-device overhead of Sec. 6.4 / Table 4).
//
// Step t of the loop, for the rows still running:
//   h_t = bf16(GELU(W1 [h_{t-1}; x] + b1))     (step 1: h_0 = 0, the x columns only)
//   p_t = sigmoid(w . h_t + aux), S += p_t, halt when S >= tau or t = max_steps
// then the halted rows' h_t are parked in sample order and the running rows
// are compacted (stable) for step t + 1.
//
// One workgroup per CU, all resident (cooperative launch); three phases per
// step, separated by grid barriers:
//   A  128 x 64 output tiles of the step's GEMM dealt over the workgroups:
//      K in 64-wide steps through two LDS stages, v_mfma_f32_32x32x16_bf16
//      over each 16-wide K block in increasing order, the epilogue staged
//      through LDS (bias, GELU, round to bf16) - per output element the same
//      instruction sequence as the implicit-GEMM kernel that runs one step
//      per launch, so both give the same bits;
//   B  one wave per row: the halting unit (the same device function as the
//      per-step halting kernel);
//   C  every workgroup partitions the step's flags itself (ballots and a
//      prefix over its four waves) into its own LDS copy of the next step's
//      row lists, so no barrier is needed after it; workgroup 0 writes the
//      branch counts, and the halted rows are parked by the workgroups in
//      turn.
// Every workgroup runs the same number of steps and barriers (the live row
// count is computed identically everywhere), so every wave reaches every
// barrier and the launch drains.
#include <hip/hip_cooperative_groups.h>

#include <stdexcept>
#include <string>

#include "halt_row.hpp"
#include "kernels.hpp"

namespace dycl {
namespace k {

namespace {

namespace cg = cooperative_groups;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void* lds_ptr;

constexpr int kBM = 128, kBN = 64, kNT = 256;
constexpr int kWTM = 64, kWTN = 32, kTM = 2, kTN = 1;        // 2 x 2 waves of 64 x 32
constexpr int kA = kBM * 128, kB = kBN * 128, kStage = kA + kB;
constexpr int kNS = 4;                                       // LDS stages: loads run three K steps ahead
constexpr int kJA = kBM * 8 / kNT, kJB = kBN * 8 / kNT;
constexpr int kEPW = kWTN + 4;
constexpr int kLoopMaxRows = 4096;                          // row lists held in LDS (16-bit entries)
constexpr int kRowsPerThread = kLoopMaxRows / kNT;          // flags each thread partitions
static_assert(4 * 32 * kEPW * 4 <= kNS * kStage, "epilogue staging fits the stages");
static_assert(kLoopMaxRows * 2 <= kNS * kStage, "the halted list fits the stages");
static_assert(kRowsPerThread == 16, "one 16-byte flag load per thread");

struct ActLoopP {
  const uint16_t* x;        // [B][D] loop input, sample order
  const uint16_t* w;        // packed W1 [H][Kp], K = [h | x]
  int Kp;
  const float* b1;          // [H]
  const float* wh;          // [H] halting weights
  const float* aux;         // [B] halting bias per sample
  uint16_t* h0;             // step states, ping-pong, [B][H] each, row order of the step
  uint16_t* h1;
  uint16_t* park;           // [B][H] final states, sample order
  float* S;                 // [B] running sums, sample order (zeroed)
  uint8_t* flags;           // [B]
  int32_t* counts;          // decision d0 + t - 1 at [2 (d0 + t - 1)]
  int d0;
  dycl_record* rec;
  const uint16_t* zeros;    // >= 16 zero bytes
  int B, H, D, steps;
  float tau;
};

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float gelu(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }

__global__ __launch_bounds__(kNT) void act_loop_kernel(ActLoopP p) {
  __shared__ __align__(16) char smem[kNS * kStage];
  __shared__ uint16_t lorig[2][kLoopMaxRows];   // original id of each row of the step
  __shared__ uint16_t lsrc[2][kLoopMaxRows];    // row of the previous step each row continues
  __shared__ int wcnt[4][2];

  cg::grid_group grid = cg::this_grid();
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = gridDim.x;
  for (int i = tid; i < p.B; i += kNT) lorig[0][i] = i;
  __syncthreads();

  int n = p.B, cur = 0;
  const int wm = wave >> 1, wn = wave & 1;
  const int lchunk = (tid & 7) ^ ((tid >> 4) & 7);
  const int rbase = tid >> 3;
  const int lsw = (lane >> 1) & 7;
  const int nt = p.H / kBN;

  for (int t = 1; t <= p.steps && n > 0; ++t) {
    const uint16_t* hprev = (t & 1) ? p.h1 : p.h0;   // state of step t - 1 (unused at t = 1)
    uint16_t* hcur = (t & 1) ? p.h0 : p.h1;
    const uint16_t* orow = lorig[cur];
    const uint16_t* srow = lsrc[cur];

    // ---- phase A: h_t = bf16(GELU(W1 [h; x] + b1)) for the n rows
    const int kbase = t == 1 ? p.H : 0;
    const int nk = (p.H + p.D - kbase) / 64;
    const int T = (n + kBM - 1) / kBM * nt;
    for (int tile = blockIdx.x; tile < T; tile += G) {
      const int m0 = tile / nt * kBM, n0 = (tile % nt) * kBN;
      const uint16_t* arow_h[kJA];
      const uint16_t* arow_x[kJA];
#pragma unroll
      for (int j = 0; j < kJA; ++j) {
        const int m = m0 + rbase + j * (kNT / 8);
        arow_h[j] = m < n ? hprev + static_cast<size_t>(t > 1 ? srow[m] : 0) * p.H : nullptr;
        arow_x[j] = m < n ? p.x + static_cast<size_t>(orow[m]) * p.D : nullptr;
      }
      const uint16_t* wrow = p.w + static_cast<size_t>(n0 + rbase) * p.Kp + lchunk * 8;
      auto issue = [&](int kt, int stage) __attribute__((always_inline)) {
        char* sb = smem + stage * kStage;
        const int kidx = kbase + kt * 64 + lchunk * 8;
#pragma unroll
        for (int j = 0; j < kJA; ++j) {
          const uint16_t* g = !arow_x[j] ? p.zeros : kidx < p.H ? arow_h[j] + kidx : arow_x[j] + (kidx - p.H);
          __builtin_amdgcn_global_load_lds((const void*)g, (lds_ptr)(sb + (j * kNT + wave * 64) * 16), 16, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kJB; ++j) {
          const uint16_t* g = wrow + static_cast<size_t>(j) * (kNT / 8) * p.Kp + (kbase + kt * 64);
          __builtin_amdgcn_global_load_lds((const void*)g, (lds_ptr)(sb + kA + (j * kNT + wave * 64) * 16), 16, 0,
                                           0);
        }
      };
      f32x16 acc[kTM][kTN];
#pragma unroll
      for (int a = 0; a < kTM; ++a)
#pragma unroll
        for (int b = 0; b < kTN; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
      auto compute = [&](int stage) __attribute__((always_inline)) {
        const char* sa = smem + stage * kStage + (wm * kWTM + (lane & 31)) * 128;
        const char* sbp = smem + stage * kStage + kA + (wn * kWTN + (lane & 31)) * 128;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int phys = ((2 * s + (lane >> 5)) ^ lsw) * 16;
          bf16x8 af[kTM], bfr[kTN];
#pragma unroll
          for (int a = 0; a < kTM; ++a) af[a] = *reinterpret_cast<const bf16x8*>(sa + a * 32 * 128 + phys);
#pragma unroll
          for (int b = 0; b < kTN; ++b) bfr[b] = *reinterpret_cast<const bf16x8*>(sbp + b * 32 * 128 + phys);
#pragma unroll
          for (int a = 0; a < kTM; ++a)
#pragma unroll
            for (int b = 0; b < kTN; ++b)
              acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
        }
      };
      __syncthreads();   // the stages are free (previous tile or phase done)
      // four stages: the loads of step kt + 3 are issued while step kt is
      // computed; the stage they fill was read in step kt - 1, which every
      // wave finished before the barrier of step kt
#pragma unroll
      for (int i = 0; i < kNS - 1; ++i)
        if (i < nk) issue(i, i);
      for (int kt = 0; kt < nk; ++kt) {
        if (kt + 2 < nk)
          asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(2 * (kJA + kJB)) : "memory");
        else if (kt + 1 < nk)
          asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(kJA + kJB) : "memory");
        else
          asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        if (kt + kNS - 1 < nk) issue(kt + kNS - 1, (kt + kNS - 1) % kNS);
        compute(kt % kNS);
      }
      __syncthreads();   // every wave's last MFMA operands are read
      // epilogue: bias, GELU, bf16, one 16-byte store per lane and row
      float* ep = reinterpret_cast<float*>(smem) + wave * 32 * kEPW;
      const int col_l = n0 + wn * kWTN + (lane & 31);
      const float sh = p.b1[col_l];
#pragma unroll
      for (int a = 0; a < kTM; ++a) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          ep[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * kEPW + (lane & 31)] = fmaf(acc[a][0][r], 1.0f, sh);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int v = 0; v < 2; ++v) {
          const int idx = v * 64 + lane;
          const int rl = idx >> 2, g = idx & 3;
          const int row = m0 + wm * kWTM + a * 32 + rl;
          if (row < n) {
            const float4 lo = *reinterpret_cast<const float4*>(ep + rl * kEPW + g * 8);
            const float4 hi = *reinterpret_cast<const float4*>(ep + rl * kEPW + g * 8 + 4);
            uint4 ov;
            ov.x = pack2(gelu(lo.x), gelu(lo.y));
            ov.y = pack2(gelu(lo.z), gelu(lo.w));
            ov.z = pack2(gelu(hi.x), gelu(hi.y));
            ov.w = pack2(gelu(hi.z), gelu(hi.w));
            *reinterpret_cast<uint4*>(hcur + static_cast<size_t>(row) * p.H + n0 + wn * kWTN + g * 8) = ov;
          }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
    }
    grid.sync();

    // ---- phase B: the halting unit, one wave per row
    for (int r = blockIdx.x * 4 + wave; r < n; r += G * 4) {
      const int o = orow[r];
      const bool stop = halt_row(hcur + static_cast<size_t>(r) * p.H, p.H, p.wh, p.aux[o], p.S, o, t, p.steps,
                                 p.tau, p.rec, lane);
      if (lane == 0) p.flags[r] = stop ? 1 : 0;
    }
    grid.sync();

    // ---- phase C: stable partition of the flags, in every workgroup: each
    // thread takes 16 consecutive rows (one 16-byte load), the threads'
    // counts are prefix-summed (shuffles in a wave, LDS across the waves)
    int16_t* halted = reinterpret_cast<int16_t*>(smem);   // the stages are free until the next tile
    const int nxt = cur ^ 1;
    const int i0 = tid * kRowsPerThread;
    uint32_t fw[4] = {0, 0, 0, 0};
    if (i0 + kRowsPerThread <= n) {
      const uint4 q = *reinterpret_cast<const uint4*>(p.flags + i0);
      fw[0] = q.x;
      fw[1] = q.y;
      fw[2] = q.z;
      fw[3] = q.w;
    } else {
      for (int j = 0; j < kRowsPerThread; ++j)
        if (i0 + j < n) fw[j >> 2] |= static_cast<uint32_t>(p.flags[i0 + j] != 0) << (8 * (j & 3));
    }
    const int nv = max(0, min(kRowsPerThread, n - i0));
    int c1 = 0;
#pragma unroll
    for (int j = 0; j < kRowsPerThread; ++j) c1 += (j < nv && ((fw[j >> 2] >> (8 * (j & 3))) & 0xff) != 0);
    const int c0 = nv - c1;
    int s0 = c0, s1 = c1;   // inclusive scans over the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int u0 = __shfl_up(s0, o, 64), u1 = __shfl_up(s1, o, 64);
      if (lane >= o) {
        s0 += u0;
        s1 += u1;
      }
    }
    if (lane == 63) {
      wcnt[wave][0] = s0;
      wcnt[wave][1] = s1;
    }
    __syncthreads();
    int o0 = s0 - c0, o1 = s1 - c1, run0 = 0, run1 = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (w < wave) {
        o0 += wcnt[w][0];
        o1 += wcnt[w][1];
      }
      run0 += wcnt[w][0];
      run1 += wcnt[w][1];
    }
    for (int j = 0; j < nv; ++j) {
      const int i = i0 + j;
      if (((fw[j >> 2] >> (8 * (j & 3))) & 0xff) != 0) {
        halted[o1++] = static_cast<int16_t>(i);
      } else {
        lsrc[nxt][o0] = static_cast<uint16_t>(i);
        lorig[nxt][o0] = orow[i];
        ++o0;
      }
    }
    __syncthreads();
    if (blockIdx.x == 0 && tid == 0) {
      p.counts[2 * (p.d0 + t - 1)] = run1;
      p.counts[2 * (p.d0 + t - 1) + 1] = run0;
    }
    // park the halted rows' states in sample order, rows dealt over the workgroups
    for (int j = blockIdx.x; j < run1; j += G) {
      const int r = halted[j];
      const uint4* src = reinterpret_cast<const uint4*>(hcur + static_cast<size_t>(r) * p.H);
      uint4* dst = reinterpret_cast<uint4*>(p.park + static_cast<size_t>(orow[r]) * p.H);
      for (int v = tid; v < p.H / 8; v += kNT) dst[v] = src[v];
    }
    n = run0;
    cur = nxt;
    __syncthreads();   // lists and the halted list settled before the next step
  }
}

}  // namespace

size_t act_loop_max_rows() { return kLoopMaxRows; }

bool act_loop_fits(int B, int H, int D) {
  return B >= 1 && B <= kLoopMaxRows && H % kBN == 0 && H % 64 == 0 && D % 64 == 0 && H >= 64;
}

void act_loop(const ActLoopArgs& a, hipStream_t s) {
  if (!act_loop_fits(a.B, a.H, a.D)) throw std::invalid_argument("persistent loop: shape it does not take");
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess)
    throw std::runtime_error("persistent loop: device attributes unavailable");
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, act_loop_kernel, kNT, 0) != hipSuccess || per_cu < 1)
    throw std::runtime_error("persistent loop: the kernel does not fit a CU");
  ActLoopP p;
  p.x = a.x;
  p.w = a.w;
  p.Kp = a.Kp;
  p.b1 = a.b1;
  p.wh = a.wh;
  p.aux = a.aux;
  p.h0 = a.h0;
  p.h1 = a.h1;
  p.park = a.park;
  p.S = a.S;
  p.flags = a.flags;
  p.counts = a.counts;
  p.d0 = a.d0;
  p.rec = a.rec;
  p.zeros = a.zeros;
  p.B = a.B;
  p.H = a.H;
  p.D = a.D;
  p.steps = a.steps;
  p.tau = a.tau;
  void* args[] = {&p};
  const hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(act_loop_kernel), dim3(cus), dim3(kNT),
                                                  args, 0, s);
  if (e != hipSuccess) throw std::runtime_error(std::string("persistent loop launch: ") + hipGetErrorString(e));
}

}  // namespace k
}  // namespace dycl
