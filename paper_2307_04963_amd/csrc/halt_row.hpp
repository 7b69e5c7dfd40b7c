// The halting unit of an adaptive-computation-time loop for one row, shared
// by the per-step kernel and the persistent loop kernel so that both take
// every decision with the same arithmetic: p = sigmoid(w . h + aux[orig]),
// S[orig] += p, halt when S >= tau or at the last step.  One wave per row;
// h is bf16 [C], C a multiple of 8.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/dycl.h"

namespace dycl {
namespace k {

__device__ __forceinline__ float halt_wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Returns the halt flag (the same in every lane); lane 0 updates S and the
// record.
__device__ __forceinline__ bool halt_row(const uint16_t* __restrict__ row, int C, const float* __restrict__ w,
                                         float aux_o, float* S, int o, int step, int max_steps, float tau,
                                         dycl_record* rec, int lane) {
  float d = 0.f;
  for (int c = lane * 8; c < C; c += 64 * 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(row + c);
    d = fmaf(__uint_as_float(v.x << 16), w[c + 0], d);
    d = fmaf(__uint_as_float(v.x & 0xffff0000u), w[c + 1], d);
    d = fmaf(__uint_as_float(v.y << 16), w[c + 2], d);
    d = fmaf(__uint_as_float(v.y & 0xffff0000u), w[c + 3], d);
    d = fmaf(__uint_as_float(v.z << 16), w[c + 4], d);
    d = fmaf(__uint_as_float(v.z & 0xffff0000u), w[c + 5], d);
    d = fmaf(__uint_as_float(v.w << 16), w[c + 6], d);
    d = fmaf(__uint_as_float(v.w & 0xffff0000u), w[c + 7], d);
  }
  d = halt_wave_sum(d);
  const float p = 1.0f / (1.0f + expf(-(d + aux_o)));
  const float Sn = S[o] + p;
  const bool stop = (Sn >= tau) || (step == max_steps);
  if (lane == 0) {
    S[o] = Sn;
    if (stop) rec[o].iterations = step;
  }
  return stop;
}

}  // namespace k
}  // namespace dycl
