// Decision heads, stream compaction, row movement and small kernels for
// gfx950.  The logic nodes of the compiled network (Sec. 5.3: a node that
// holds a single conditional reading an intermediate tensor, Sec. 2.2) are
// evaluated here per sample, on the device, for a whole batch at once; the
// branch each sample takes is then materialised by a stable compaction and
// row gathers, so the next sub-network runs on a packed subset.
#include "kernels.hpp"
#include "halt_row.hpp"

#include <mutex>
#include <stdexcept>

namespace dycl {
namespace k {

namespace {

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// live rows: the device count when there is one (never above the n the
// launch was sized for), else n
__device__ __forceinline__ int live(const int32_t* nc, int n) { return nc ? min(*nc, n) : n; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum over HW of one row [HW, C] (bf16) into per-channel floats in `red`
// (shared, C floats).  256 threads; C is a power of two >= 8 and <= 2048.
// Channel sums of positions [p0, p1) of one NHWC bf16 row: red[c], fp32.
// 256 threads: each takes 16-byte vectors of one channel group at every
// PG-th position, four positions in flight; partial sums meet in `part`.
__device__ void row_channel_sums(const uint16_t* __restrict__ x, int p0, int p1, int C, float* red, float* part) {
  const int tid = threadIdx.x;
  const int C8 = C >> 3;              // 16-byte vectors per position
  const int PG = 256 / C8 > 0 ? 256 / C8 : 1;
  const int cv = tid % C8, pg = tid / C8;
  float s[4][8] = {};
  if (pg < PG) {
    int pos = p0 + pg;
    for (; pos + 3 * PG < p1; pos += 4 * PG) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const uint4*>(x + (size_t)(pos + u * PG) * C + cv * 8);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        s[u][0] += __uint_as_float(v[u].x << 16);
        s[u][1] += __uint_as_float(v[u].x & 0xffff0000u);
        s[u][2] += __uint_as_float(v[u].y << 16);
        s[u][3] += __uint_as_float(v[u].y & 0xffff0000u);
        s[u][4] += __uint_as_float(v[u].z << 16);
        s[u][5] += __uint_as_float(v[u].z & 0xffff0000u);
        s[u][6] += __uint_as_float(v[u].w << 16);
        s[u][7] += __uint_as_float(v[u].w & 0xffff0000u);
      }
    }
    for (; pos < p1; pos += PG) {
      const uint4 v = *reinterpret_cast<const uint4*>(x + (size_t)pos * C + cv * 8);
      s[0][0] += __uint_as_float(v.x << 16);
      s[0][1] += __uint_as_float(v.x & 0xffff0000u);
      s[0][2] += __uint_as_float(v.y << 16);
      s[0][3] += __uint_as_float(v.y & 0xffff0000u);
      s[0][4] += __uint_as_float(v.z << 16);
      s[0][5] += __uint_as_float(v.z & 0xffff0000u);
      s[0][6] += __uint_as_float(v.w << 16);
      s[0][7] += __uint_as_float(v.w & 0xffff0000u);
    }
  }
  // part: [PG][C]
  if (pg < PG) {
#pragma unroll
    for (int j = 0; j < 8; ++j) part[pg * C + cv * 8 + j] = (s[0][j] + s[1][j]) + (s[2][j] + s[3][j]);
  }
  __syncthreads();
  for (int c = tid; c < C; c += 256) {
    float t = 0.f;
    for (int g = 0; g < PG; ++g) t += part[g * C + c];
    red[c] = t;
  }
  __syncthreads();
}

}  // namespace

// ----------------------------------------------------------------- GAP ----

__global__ __launch_bounds__(256) void gap_kernel(const uint16_t* __restrict__ x, int HW, int C, float* G,
                                                  const int32_t* nc, int n) {
  __shared__ float part[2048];
  __shared__ float red[2048];
  const int r = blockIdx.x;
  if (r >= live(nc, n)) return;
  row_channel_sums(x + (size_t)r * HW * C, 0, HW, C, red, part);
  const float inv = 1.0f / static_cast<float>(HW);
  for (int c = threadIdx.x; c < C; c += 256) G[(size_t)r * C + c] = red[c] * inv;
}

// a large row's positions split over S workgroups: partial sums
// P[split][row][C], then a fixed-order sum per (row, channel)
__global__ __launch_bounds__(256) void gap_split_kernel(const uint16_t* __restrict__ x, int n, int HW, int C, int S,
                                                        float* __restrict__ P, const int32_t* nc) {
  __shared__ float part[2048];
  __shared__ float red[2048];
  const int r = blockIdx.x / S, sp = blockIdx.x - (blockIdx.x / S) * S;
  if (r >= live(nc, n)) return;
  const int p0 = static_cast<int>(static_cast<long>(HW) * sp / S), p1 = static_cast<int>(static_cast<long>(HW) * (sp + 1) / S);
  row_channel_sums(x + (size_t)r * HW * C, p0, p1, C, red, part);
  for (int c = threadIdx.x; c < C; c += 256) P[((size_t)sp * n + r) * C + c] = red[c];
}

__global__ void gap_merge_kernel(const float* __restrict__ P, int n, int HW, int C, int S, float* __restrict__ G,
                                 const int32_t* nc) {
  // P is laid out for n rows; only the live ones are summed
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<size_t>(live(nc, n)) * C) return;
  float t = 0.f;
  for (int sp = 0; sp < S; ++sp) t += P[(size_t)sp * n * C + i];
  G[i] = t * (1.0f / static_cast<float>(HW));
}

// pooled features from the 32-row chunk sums a conv epilogue left: one
// thread per (image, channel); the chunks image r overlaps, in order, each
// contributing its first part when the chunk starts in image r and its
// second part when it starts in the image before (up to 32 loads in flight),
// then divided by HW as gap_merge_kernel does
__global__ __launch_bounds__(256) void gap_chunks_kernel(const float* __restrict__ Q, int n, int HW, int C,
                                                         float* __restrict__ G, const int32_t* nc) {
  const size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<size_t>(live(nc, n)) * C) return;
  const size_t r = i / C, c = i - r * C;
  const size_t j0 = r * HW / 32, j1 = ((r + 1) * HW - 1) / 32;
  // only the first chunk can start in the image before (HW >= 32)
  float t = Q[(2 * j0 + ((r * HW) % 32 ? 1 : 0)) * C + c];
  size_t j = j0 + 1;
  for (; j + 32 <= j1 + 1; j += 32) {
    float v[32];
#pragma unroll
    for (int u = 0; u < 32; ++u) v[u] = Q[2 * (j + u) * C + c];
#pragma unroll
    for (int u = 0; u < 32; ++u) t += v[u];
  }
  for (; j + 8 <= j1 + 1; j += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = Q[2 * (j + u) * C + c];
#pragma unroll
    for (int u = 0; u < 8; ++u) t += v[u];
  }
  for (; j <= j1; ++j) t += Q[2 * j * C + c];
  G[i] = t * (1.0f / static_cast<float>(HW));
}

void gap_chunks(const float* Q, int n, int HW, int C, float* G, hipStream_t s, const int32_t* nc) {
  if (n <= 0) return;
  if (HW < 32) throw std::invalid_argument("gap_chunks: an image needs at least 32 rows");
  const size_t total = static_cast<size_t>(n) * C;
  hipLaunchKernelGGL(gap_chunks_kernel, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, s, Q, n, HW,
                     C, G, nc);
}

// splits of a row: a function of HW alone (about 256 positions each), so a
// row's sum has the same rounding whatever the row count of the launch
int gap_splits(int HW) {
  const int S = HW / 256;
  return S < 1 ? 1 : (S > kGapMaxSplit ? kGapMaxSplit : S);
}

void gap_bf16(const uint16_t* x, int n, int HW, int C, float* G, float* P, hipStream_t s, const int32_t* nc) {
  const int S = P ? gap_splits(HW) : 1;
  if (S == 1) {
    hipLaunchKernelGGL(gap_kernel, dim3(n), dim3(256), 0, s, x, HW, C, G, nc, n);
    return;
  }
  hipLaunchKernelGGL(gap_split_kernel, dim3(n * S), dim3(256), 0, s, x, n, HW, C, S, P, nc);
  const size_t total = static_cast<size_t>(n) * C;
  hipLaunchKernelGGL(gap_merge_kernel, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, s, P, n, HW, C, S,
                     G, nc);
}

// -------------------------------------------------------------- linear ----

__global__ __launch_bounds__(256) void linear_f32_kernel(const float* __restrict__ X, int n, int K,
                                                         const float* __restrict__ W, const float* __restrict__ bias,
                                                         int N, int act, float* __restrict__ Y) {
  __shared__ float Xs[16][68];
  __shared__ float Ws[16][68];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = threadIdx.x + i * 256;
      const int rr = e >> 4, kk = e & 15;
      Xs[kk][rr] = (m0 + rr < n && k0 + kk < K) ? X[(size_t)(m0 + rr) * K + k0 + kk] : 0.f;
      Ws[kk][rr] = (n0 + rr < N && k0 + kk < K) ? W[(size_t)(n0 + rr) * K + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = Xs[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Ws[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= n) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = n0 + tx * 4 + j;
      if (c >= N) continue;
      float v = acc[i][j] + (bias ? bias[c] : 0.f);
      if (act == ACT_RELU) v = v > 0.f ? v : 0.f;
      Y[(size_t)m * N + c] = v;
    }
  }
}

void linear_f32(const float* X, int n, int K, const float* W, const float* bias, int N, int act, float* Y,
                hipStream_t s) {
  dim3 grid((n + 63) / 64, (N + 63) / 64);
  hipLaunchKernelGGL(linear_f32_kernel, grid, dim3(256), 0, s, X, n, K, W, bias, N, act, Y);
}

// ------------------------------------------------------- skinny linear ----
// Y[m, j] = act(b[j] + sum_k X[m, k] Wt[k, j]) with the weights transposed
// (Wt [K][N]): a workgroup owns R rows x 64 columns; its NW waves take the
// K range interleaved (wave w: k = w, w + NW, ...) so that every lane keeps
// many independent loads in flight, and the partial sums meet in LDS.  The
// weight reads are coalesced over columns and shared by the R rows.

template <int R, int NW>
__global__ __launch_bounds__(64 * NW) void linear_t_kernel(const float* __restrict__ X, int n, int K,
                                                           const float* __restrict__ Wt,
                                                           const float* __restrict__ bias, int N, int act,
                                                           float* __restrict__ Y, const int32_t* nc) {
  __shared__ float red[NW][R][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // workgroup = row group * gy + column block: the workgroups of live rows
  // are dispatched first and the surplus ones (device counts) last
  const int gy = (N + 63) / 64;
  const int rg = blockIdx.x / gy;
  const int col = (blockIdx.x - rg * gy) * 64 + lane, m0 = rg * R;
  n = live(nc, n);
  if (m0 >= n) return;
  const int cc = col < N ? col : N - 1;
  const float* xr[R];
#pragma unroll
  for (int r = 0; r < R; ++r) xr[r] = X + (size_t)(m0 + r < n ? m0 + r : n - 1) * K;
  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;
#pragma unroll 4
  for (int k = w; k < K; k += NW) {
    const float wv = Wt[(size_t)k * N + cc];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = fmaf(xr[r][k], wv, acc[r]);
  }
#pragma unroll
  for (int r = 0; r < R; ++r) red[w][r][lane] = acc[r];
  __syncthreads();
  if (w == 0 && col < N) {
    const float b = bias ? bias[col] : 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (m0 + r >= n) break;
      float v = 0.f;
#pragma unroll
      for (int q = 0; q < NW; ++q) v += red[q][r][lane];
      v += b;
      if (act == ACT_RELU) v = v > 0.f ? v : 0.f;
      Y[(size_t)(m0 + r) * N + col] = v;
    }
  }
}

void linear_t_f32(const float* X, int n, int K, const float* Wt, const float* bias, int N, int act, float* Y,
                  hipStream_t s, const int32_t* nc, int nhint) {
  const int gy = (N + 63) / 64;
  const int nh = nhint > 0 && nhint < n ? nhint : n;
  // rows per workgroup: as many as keep >= 256 workgroups in flight
  if ((long)((nh + 7) / 8) * gy >= 256)
    hipLaunchKernelGGL((linear_t_kernel<8, 8>), dim3(gy * ((n + 7) / 8)), dim3(512), 0, s, X, n, K, Wt, bias, N, act, Y, nc);
  else if ((long)((nh + 3) / 4) * gy >= 128)
    hipLaunchKernelGGL((linear_t_kernel<4, 8>), dim3(gy * ((n + 3) / 4)), dim3(512), 0, s, X, n, K, Wt, bias, N, act, Y, nc);
  else
    hipLaunchKernelGGL((linear_t_kernel<1, 8>), dim3(gy * (n)), dim3(512), 0, s, X, n, K, Wt, bias, N, act, Y, nc);
}

// --------------------------------------------------------- exit decide ----

__global__ __launch_bounds__(64) void exit_decide_kernel(const float* __restrict__ Z, int ncls,
                                                         const float* __restrict__ Tp, float tau, int final_, int head,
                                                         const int32_t* __restrict__ orig, uint8_t* flags,
                                                         float* __restrict__ logits, int n_out, dycl_record* rec,
                                                         const int32_t* nc, int n) {
  const int r = blockIdx.x, lane = threadIdx.x;
  if (r >= live(nc, n)) return;
  const float* z = Z + (size_t)r * ncls;
  bool ex = final_ != 0;
  if (!ex) {
    const float T = *Tp;
    float m = -INFINITY;
    for (int j = lane; j < ncls; j += 64) m = fmaxf(m, z[j]);
    m = wave_max(m);
    float s = 0.f;
    for (int j = lane; j < ncls; j += 64) s += expf((z[j] - m) / T);
    s = wave_sum(s);
    ex = (1.0f / s) >= tau;
  }
  if (ex) {
    const int o = orig ? orig[r] : r;
    for (int j = lane; j < ncls; j += 64) logits[(size_t)o * n_out + j] = z[j];
    if (lane == 0 && head >= 0) rec[o].exit_index = head;
  }
  if (lane == 0) flags[r] = ex ? 1 : 0;
}

void exit_decide(const float* Z, int n, int ncls, const float* T, float tau, int final_, int head, const int32_t* orig,
                 uint8_t* flags, float* logits, int n_out, dycl_record* rec, hipStream_t s, const int32_t* nc) {
  hipLaunchKernelGGL(exit_decide_kernel, dim3(n), dim3(64), 0, s, Z, ncls, T, tau, final_, head, orig, flags,
                     logits, n_out, rec, nc, n);
}

// ------------------------------------------------- sliced exit head ----
// Wide exit heads (C x ncls beyond the fused kernel): the head linear
// z = W g + b over K = C is cut into slices of about 128 so that a launch has
// many short sums instead of a few long ones (the long chains left the
// linear waiting on its loads).  head_partial_kernel: workgroup (row group of
// 8, 64 classes, slice s) sums its slice, its four waves taking interleaved
// k and meeting in LDS in wave order; head_decide_kernel: one workgroup per
// row adds the slices in order, the bias, and takes the exit decision.  The
// slices depend on C alone, so every row count sums in the same order.  Both
// kernels issue all their loads before the first wait: a few long dependent
// load rounds, not the arithmetic, were what bounded these launches.

int head_slices(int K) { return K <= 128 ? 1 : (K + 127) / 128; }
bool head_sliced_fits(int K, int ncls) { return K >= 1 && K <= 2048 && ncls >= 1 && ncls <= 1024; }

__global__ __launch_bounds__(256) void head_partial_kernel(const float* __restrict__ G, int n, int K,
                                                           const float* __restrict__ Wt, int N, int S,
                                                           float* __restrict__ P, int nP, const int32_t* nc) {
  constexpr int R = 8, KSMAX = 132;
  __shared__ __align__(16) float xs[KSMAX][R];   // k-major: a k's 8 rows in two 16-byte reads
  __shared__ float red[4][R][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gy = (N + 63) / 64;
  const int s = blockIdx.x % S, rest = blockIdx.x / S;
  const int cb = rest % gy, rg = rest / gy;
  n = live(nc, n);
  const int m0 = rg * R;
  if (m0 >= n) return;
  const int k0 = static_cast<int>(static_cast<long>(K) * s / S), k1 = static_cast<int>(static_cast<long>(K) * (s + 1) / S);
  const int ks = k1 - k0;   // at most 128: S = ceil(K / 128)
  const int col = cb * 64 + lane, cc = col < N ? col : N - 1;
  // every load of the workgroup is issued before the first wait: the wave's
  // weights (k = w + 4 i of the slice, addresses clamped into the slice) and
  // the rows' features (clamped into the live rows)
  constexpr int KI = (KSMAX + 3) / 4;
  float wv[KI];
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const int kk = min(w + 4 * i, ks - 1);
    wv[i] = Wt[static_cast<size_t>(k0 + kk) * N + cc];
  }
  constexpr int XI = (R * KSMAX + 255) / 256;
  float xv[XI];
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int e = min(static_cast<int>(threadIdx.x) + 256 * i, R * ks - 1);
    const int r = e / ks, kk = e - r * ks;
    xv[i] = G[static_cast<size_t>(min(m0 + r, n - 1)) * K + k0 + kk];
  }
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int e = threadIdx.x + 256 * i;
    if (e < R * ks) {
      const int r = e / ks, kk = e - r * ks;
      xs[kk][r] = m0 + r < n ? xv[i] : 0.f;
    }
  }
  __syncthreads();
  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const int kk = w + 4 * i;
    if (kk < ks) {
      const float4 x0 = *reinterpret_cast<const float4*>(&xs[kk][0]);
      const float4 x1 = *reinterpret_cast<const float4*>(&xs[kk][4]);
      const float xr[R] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int r = 0; r < R; ++r) acc[r] = fmaf(xr[r], wv[i], acc[r]);
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) red[w][r][lane] = acc[r];
  __syncthreads();
  // 256 threads finish 8 rows x 64 columns: thread -> (row w + 4 q, column lane)
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int r = w + 4 * q;
    if (m0 + r < n && col < N)
      P[(static_cast<size_t>(s) * nP + m0 + r) * N + col] =
          ((red[0][r][lane] + red[1][r][lane]) + red[2][r][lane]) + red[3][r][lane];
  }
}

// One workgroup per row: thread t holds classes t + 256 q (q < 4); it loads
// every slice of all of them before adding (SP >= S slices, addresses
// clamped), adds the slices in order and the bias, and the four waves meet
// in LDS, in wave order, for the row's maximum and exponential sum.
template <int SP>
__global__ __launch_bounds__(256) void head_decide_kernel(const float* __restrict__ P, int nP, int S, int ncls,
                                                          const float* __restrict__ bias, const float* __restrict__ Tp,
                                                          float tau, int final_, int head,
                                                          const int32_t* __restrict__ orig, uint8_t* flags,
                                                          float* __restrict__ logits, int n_out, dycl_record* rec,
                                                          const int32_t* nc, int n) {
  constexpr int JQ = 4;   // ncls <= 1024
  __shared__ float wred[2][4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r = blockIdx.x;
  if (r >= live(nc, n)) return;
  float pv[JQ][SP];
#pragma unroll
  for (int q = 0; q < JQ; ++q) {
    const int j = min(tid + 256 * q, ncls - 1);
#pragma unroll
    for (int sl = 0; sl < SP; ++sl)
      pv[q][sl] = P[(static_cast<size_t>(min(sl, S - 1)) * nP + r) * ncls + j];
  }
  float z[JQ];
#pragma unroll
  for (int q = 0; q < JQ; ++q) {
    const int j = tid + 256 * q;
    float v = pv[q][0];
#pragma unroll
    for (int sl = 1; sl < SP; ++sl)
      if (sl < S) v += pv[q][sl];
    z[q] = j < ncls ? v + (bias ? bias[j] : 0.f) : 0.f;
  }
  bool ex = final_ != 0;
  if (!ex) {
    const float T = *Tp;
    float m = -INFINITY;
#pragma unroll
    for (int q = 0; q < JQ; ++q)
      if (tid + 256 * q < ncls) m = fmaxf(m, z[q]);
    m = wave_max(m);
    if (lane == 0) wred[0][w] = m;
    __syncthreads();
    m = fmaxf(fmaxf(wred[0][0], wred[0][1]), fmaxf(wred[0][2], wred[0][3]));
    float sm = 0.f;
#pragma unroll
    for (int q = 0; q < JQ; ++q)
      if (tid + 256 * q < ncls) sm += expf((z[q] - m) / T);
    sm = wave_sum(sm);
    if (lane == 0) wred[1][w] = sm;
    __syncthreads();
    sm = ((wred[1][0] + wred[1][1]) + wred[1][2]) + wred[1][3];
    ex = (1.0f / sm) >= tau;
  }
  if (ex) {
    const int o = orig ? orig[r] : r;
#pragma unroll
    for (int q = 0; q < JQ; ++q)
      if (tid + 256 * q < ncls) logits[static_cast<size_t>(o) * n_out + tid + 256 * q] = z[q];
    if (tid == 0 && head >= 0) rec[o].exit_index = head;
  }
  if (tid == 0) flags[r] = ex ? 1 : 0;
}

size_t head_partials_floats(int K, int n, int ncls) {
  return static_cast<size_t>(head_slices(K)) * n * ncls;
}

void exit_head_sliced(const float* G, int n, int K, const float* Wt, const float* bias, int ncls, const float* T,
                      float tau, int final_, int head, const int32_t* orig, uint8_t* flags, float* logits, int n_out,
                      dycl_record* rec, float* P, hipStream_t s, const int32_t* nc) {
  if (!head_sliced_fits(K, ncls)) throw std::invalid_argument("exit_head_sliced: K or class count out of range");
  if (n <= 0) return;
  const int S = head_slices(K), gy = (ncls + 63) / 64;
  hipLaunchKernelGGL(head_partial_kernel, dim3(((n + 7) / 8) * gy * S), dim3(256), 0, s, G, n, K, Wt, ncls, S, P, n,
                     nc);
  const dim3 g(n), b(256);
  if (S <= 1)
    hipLaunchKernelGGL(head_decide_kernel<1>, g, b, 0, s, P, n, S, ncls, bias, T, tau, final_, head, orig, flags,
                       logits, n_out, rec, nc, n);
  else if (S <= 2)
    hipLaunchKernelGGL(head_decide_kernel<2>, g, b, 0, s, P, n, S, ncls, bias, T, tau, final_, head, orig, flags,
                       logits, n_out, rec, nc, n);
  else if (S <= 4)
    hipLaunchKernelGGL(head_decide_kernel<4>, g, b, 0, s, P, n, S, ncls, bias, T, tau, final_, head, orig, flags,
                       logits, n_out, rec, nc, n);
  else if (S <= 8)
    hipLaunchKernelGGL(head_decide_kernel<8>, g, b, 0, s, P, n, S, ncls, bias, T, tau, final_, head, orig, flags,
                       logits, n_out, rec, nc, n);
  else
    hipLaunchKernelGGL(head_decide_kernel<16>, g, b, 0, s, P, n, S, ncls, bias, T, tau, final_, head, orig, flags,
                       logits, n_out, rec, nc, n);
}

// ----------------------------------------------------- fused exit head ----
// One workgroup per row: pooled features g (GAP of a bf16 [HW, C] row, or
// the fp32 row itself), head logits z = W g + b from the transposed head
// weights Wt [C][ncls] (coalesced over classes), then the decision of the
// exit: p = max softmax(z / T), leave when p >= tau (or always when final).

template <bool BF16>
__global__ __launch_bounds__(256) void exit_head_kernel(const void* __restrict__ x, int n, int R, int HW, int C,
                                                        const float* __restrict__ W, const float* __restrict__ bias,
                                                        int ncls, const float* __restrict__ Tp, float tau,
                                                        int final_, int head, const int32_t* __restrict__ orig,
                                                        uint8_t* flags, float* __restrict__ logits, int n_out,
                                                        dycl_record* rec, const int32_t* nc) {
  // R rows per workgroup: pooled features g [R][C] and logits z [R][ncls]
  // in LDS; the head weights W [ncls][C] are read once per workgroup
  constexpr int RMAX = 8;
  extern __shared__ float dyn[];   // part [2048] | g [R][C] | z [R][ncls]
  float* const part = dyn;
  float* const g = dyn + 2048;
  float* const z = g + R * C;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  n = live(nc, n);
  const int r0 = blockIdx.x * R, nr = min(R, n - r0);
  if (nr <= 0) return;
  for (int i = 0; i < nr; ++i) {
    float* gi = g + i * C;
    if constexpr (BF16) {
      row_channel_sums(static_cast<const uint16_t*>(x) + (size_t)(r0 + i) * HW * C, 0, HW, C, gi, part);
      const float inv = 1.0f / static_cast<float>(HW);
      for (int c = tid; c < C; c += 256) gi[c] *= inv;
    } else {
      for (int c = tid; c < C; c += 256) gi[c] = static_cast<const float*>(x)[(size_t)(r0 + i) * C + c];
    }
  }
  __syncthreads();

  // z[i][j] = bias[j] + sum_c W[j][c] g[i][c]: four lanes per class, each
  // taking every fourth 16-byte piece of the weight row (independent loads),
  // combined by lane shuffles
  const int q = tid & 3, jl = tid >> 2, C4 = C >> 2;
  for (int j0 = 0; j0 < ncls; j0 += 64) {
    const int j = j0 + jl;
    float acc[RMAX];
#pragma unroll
    for (int i = 0; i < RMAX; ++i) acc[i] = 0.f;
    if (j < ncls) {
      const float4* wr = reinterpret_cast<const float4*>(W + (size_t)j * C);
#pragma unroll 4
      for (int f = q; f < C4; f += 4) {
        const float4 w = wr[f];
#pragma unroll
        for (int i = 0; i < RMAX; ++i) {
          if (i < nr) {
            const float4 gv = *reinterpret_cast<const float4*>(g + i * C + 4 * f);
            acc[i] = fmaf(w.x, gv.x, fmaf(w.y, gv.y, fmaf(w.z, gv.z, fmaf(w.w, gv.w, acc[i]))));
          }
        }
      }
    }
#pragma unroll
    for (int i = 0; i < RMAX; ++i) {
      acc[i] += __shfl_xor(acc[i], 1);
      acc[i] += __shfl_xor(acc[i], 2);
    }
    if (q == 0 && j < ncls) {
      const float bj = bias[j];
#pragma unroll
      for (int i = 0; i < RMAX; ++i)
        if (i < nr) z[i * ncls + j] = acc[i] + bj;
    }
  }
  __syncthreads();

  // decision per row, one wave each: max softmax probability 1 / sum exp((z - max) / T)
  for (int i = wave; i < nr; i += 4) {
    const int r = r0 + i;
    const float* zi = z + i * ncls;
    bool ex = final_ != 0;
    if (!ex) {
      float m = -INFINITY;
      for (int j = lane; j < ncls; j += 64) m = fmaxf(m, zi[j]);
      m = wave_max(m);
      const float T = *Tp;
      float sum = 0.f;
      for (int j = lane; j < ncls; j += 64) sum += expf((zi[j] - m) / T);
      sum = wave_sum(sum);
      ex = (1.0f / sum) >= tau;
    }
    if (ex) {
      const int o = orig ? orig[r] : r;
      for (int j = lane; j < ncls; j += 64) logits[(size_t)o * n_out + j] = zi[j];
      if (lane == 0 && head >= 0) rec[o].exit_index = head;
    }
    if (lane == 0) flags[r] = ex ? 1 : 0;
  }
}

void exit_head(const void* x, bool bf16, int n, int HW, int C, const float* W, const float* bias, int ncls,
               const float* T, float tau, int final_, int head, const int32_t* orig, uint8_t* flags, float* logits,
               int n_out, dycl_record* rec, hipStream_t s, const int32_t* nc, int nhint) {
  // rows per workgroup: one where pooling dominates (a row's pooling reads
  // HW * C elements, its linear C * ncls weights); else enough rows to share
  // the weights, keeping a workgroup for every CU, at most 8, within LDS
  const int nh = nhint > 0 && nhint < n ? nhint : n;
  int R = HW >= ncls ? 1 : nh / 256;
  R = R < 1 ? 1 : (R > 8 ? 8 : R);
  while (R > 1 && (R * C > 8 * 2048 || R * ncls > 8 * 1024)) --R;
  const int grid = (n + R - 1) / R;
  const size_t lds = (2048 + static_cast<size_t>(R) * (C + ncls)) * sizeof(float);
  if (bf16)
    hipLaunchKernelGGL(exit_head_kernel<true>, dim3(grid), dim3(256), lds, s, x, n, R, HW, C, W, bias, ncls, T, tau,
                       final_, head, orig, flags, logits, n_out, rec, nc);
  else
    hipLaunchKernelGGL(exit_head_kernel<false>, dim3(grid), dim3(256), lds, s, x, n, R, HW, C, W, bias, ncls, T, tau,
                       final_, head, orig, flags, logits, n_out, rec, nc);
}

// ---------------------------------------------------------------- gate ----

__global__ __launch_bounds__(256) void gate_kernel(const uint16_t* __restrict__ x, int HW, int C,
                                                   const float* __restrict__ u, const float* __restrict__ v,
                                                   float thr, int gate, const int32_t* __restrict__ orig,
                                                   uint8_t* flags, dycl_record* rec, const int32_t* nc, int n) {
  __shared__ float part[2048];
  __shared__ float red[2048];
  __shared__ float wsum[4];
  const int r = blockIdx.x;
  if (r >= live(nc, n)) return;
  row_channel_sums(x + (size_t)r * HW * C, 0, HW, C, red, part);
  const float inv = 1.0f / static_cast<float>(HW);
  float d = 0.f;
  for (int c = threadIdx.x; c < C; c += 256) d = fmaf(u[c], red[c] * inv, d);
  d = wave_sum(d);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = d;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float pre = wsum[0] + wsum[1] + wsum[2] + wsum[3] + *v;
    const float q = 1.0f / (1.0f + expf(-pre));
    const bool run = q > thr;
    flags[r] = run ? 1 : 0;
    if (!run) {
      const int o = orig ? orig[r] : r;
      rec[o].skip_mask |= (1ull << gate);
    }
  }
}

void gate_head(const uint16_t* x, int n, int HW, int C, const float* u, const float* v, float thr, int gate,
               const int32_t* orig, uint8_t* flags, dycl_record* rec, hipStream_t s, const int32_t* nc) {
  hipLaunchKernelGGL(gate_kernel, dim3(n), dim3(256), 0, s, x, HW, C, u, v, thr, gate, orig, flags, rec, nc, n);
}

// ---------------------------------------------------------------- halt ----

__global__ __launch_bounds__(64) void halt_kernel(const uint16_t* __restrict__ h, int C, const float* __restrict__ w,
                                                  const float* __restrict__ aux, const int32_t* __restrict__ orig,
                                                  float* S, int step, int max_steps, float tau, uint8_t* flags,
                                                  dycl_record* rec, const int32_t* nc, int n) {
  const int r = blockIdx.x, lane = threadIdx.x;
  if (r >= live(nc, n)) return;
  const int o = orig ? orig[r] : r;
  const bool stop = halt_row(h + (size_t)r * C, C, w, aux[o], S, o, step, max_steps, tau, rec, lane);
  if (lane == 0) flags[r] = stop ? 1 : 0;
}

void halt_head(const uint16_t* h, int n, int C, const float* w, const float* aux, const int32_t* orig, float* S,
               int step, int max_steps, float tau, uint8_t* flags, dycl_record* rec, hipStream_t s,
               const int32_t* nc) {
  hipLaunchKernelGGL(halt_kernel, dim3(n), dim3(64), 0, s, h, C, w, aux, orig, S, step, max_steps, tau, flags, rec,
                     nc, n);
}

// ---------------------------------------------------------- compaction ----
// One workgroup of 16 wave64s walks the flags 1024 at a time.  Within a wave
// the rank of a row among the rows of its branch is the popcount of the
// 64-bit ballot below its lane (mbcnt); the waves' totals are prefix-summed
// through LDS.  Rows keep their order in both lists (stable partition).

__global__ __launch_bounds__(1024) void compact_kernel(const uint8_t* __restrict__ flags,
                                                       const int32_t* __restrict__ orig, int n, int32_t* idx1,
                                                       int32_t* org1, int32_t* idx0, int32_t* org0, int32_t* counts,
                                                       const int32_t* nc) {
  __shared__ int wc1[16], wc0[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  n = live(nc, n);
  int base1 = 0, base0 = 0;
  for (int start = 0; start < n; start += 1024) {
    const int i = start + tid;
    const bool valid = i < n;
    // the row's id requested with its flag: one memory round trip, not two
    const int32_t id = valid && orig ? orig[i] : i;
    const uint8_t fl = valid ? flags[i] : 0;
    const bool f = valid && fl != 0;
    const bool g = valid && fl == 0;
    const uint64_t b1 = __ballot(f);
    const uint64_t b0 = __ballot(g);
    const int r1 = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(b1 >> 32),
                                             __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(b1), 0));
    const int r0 = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(b0 >> 32),
                                             __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(b0), 0));
    if (lane == 0) {
      wc1[wave] = __popcll(b1);
      wc0[wave] = __popcll(b0);
    }
    __syncthreads();
    int off1 = base1, off0 = base0, t1 = 0, t0 = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      const int c1 = wc1[w], c0 = wc0[w];
      if (w < wave) {
        off1 += c1;
        off0 += c0;
      }
      t1 += c1;
      t0 += c0;
    }
    if (f) {
      idx1[off1 + r1] = i;
      org1[off1 + r1] = id;
    }
    if (g) {
      idx0[off0 + r0] = i;
      org0[off0 + r0] = id;
    }
    base1 += t1;
    base0 += t0;
    __syncthreads();
  }
  if (tid == 0) {
    counts[0] = base1;
    counts[1] = base0;
  }
}

void compact(const uint8_t* flags, const int32_t* orig, int n, int32_t* idx1, int32_t* org1, int32_t* idx0,
             int32_t* org0, int32_t* counts, hipStream_t s, const int32_t* nc) {
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, s, flags, orig, n, idx1, org1, idx0, org0, counts, nc);
}

// ------------------------------------------------- large-n compaction ----
// One pass, chained over blocks of 16384 flags (8192 when ids are carried).
// A workgroup reads its block's flags (and ids) once, counts the ones,
// publishes that count in the block's status word, ranks its elements and
// stages the block's partition in LDS (block positions, and the ids); wave 0
// then learns how many ones all earlier blocks hold by reading their status
// words backwards, 64 a round, to the nearest one that already carries an
// inclusive prefix, publishes the block's own inclusive prefix, and the
// workgroup writes both runs with coalesced stores.  Order is preserved
// (stable partition).  Flags cross HBM once and every index once; blocks are
// large because each one's prefix costs a round trip through the chain.
//
// Status word: the top two bits say what it holds (0 nothing yet, 1 the
// block's count, 2 the ones of blocks 0..b), the rest the value.  The words
// and the counts are cleared by the call's first kernel.  The wait is
// bounded (kSpinLimit polls in all): it cannot run out unless a predecessor
// never publishes, which in-order dispatch rules out; a workgroup that still
// runs out of polls writes counts {-1, -1} and nothing else instead of
// waiting for ever.

constexpr int kCompactEPT = 64;                       // flags per thread, without ids
constexpr int kCompactEPTI = 32;                      // with ids (their LDS staging halves the block)
constexpr int kCompactBlock = 256 * kCompactEPT;
constexpr int kCompactBlockI = 256 * kCompactEPTI;
static_assert(kCompactEPTI <= kCompactEPT && kCompactEPT <= 256 && kCompactEPTI % 16 == 0,
              "the workspace is sized by the smaller block; positions fit 16 bits");
constexpr uint64_t kStCount = 1ull << 62, kStPrefix = 2ull << 62, kStValue = (1ull << 62) - 1;
constexpr int kSpinLimit = 1 << 16;

__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

__device__ __forceinline__ long long wave_sum_ll(long long v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ void status_put(uint64_t* w, uint64_t v) {
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t status_get(uint64_t* w) {
  return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// a pause that grows with the polls already spent (1 to 16 sleeps of 64 clocks)
__device__ __forceinline__ void backoff(int spins) {
  const int k = spins < 4 ? 1 << spins : 16;
  for (int i = 0; i < k; ++i) __builtin_amdgcn_s_sleep(1);
}

__global__ __launch_bounds__(256) void compact_clear_kernel(uint64_t* __restrict__ st, int nb, int32_t* counts) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < nb) st[i] = 0;
  if (i == 0) {
    counts[0] = 0;
    counts[1] = 0;
  }
}

// Block b = workgroup b: workgroups of a grid are dispatched in index order,
// so the blocks a workgroup waits for have all been dispatched.
template <bool IDS>
__global__ __launch_bounds__(256) void compact_chain_kernel(const uint8_t* __restrict__ flags,
                                                            const int32_t* __restrict__ orig, size_t n,
                                                            uint64_t* st, int32_t* idx1, int32_t* org1,
                                                            int32_t* idx0, int32_t* org0, int32_t* counts,
                                                            const int32_t* nc) {
  constexpr int EPT = IDS ? kCompactEPTI : kCompactEPT, NB = 256 * EPT;
  __shared__ uint16_t spos[NB];              // block position of each staged element
  __shared__ int32_t sorg[IDS ? NB : 1];
  __shared__ int wsum[4];
  __shared__ int s_fail;
  __shared__ long long s_excl;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (nc) n = min(n, static_cast<size_t>(max(*nc, 0)));
  const int nbl = static_cast<int>((n + NB - 1) / NB);
  const int b = blockIdx.x;
  if (b >= nbl) return;
  const size_t blk0 = static_cast<size_t>(b) * NB;
  const int nblk = static_cast<int>(min(n - blk0, static_cast<size_t>(NB)));

  // EPT consecutive flags per thread (16-byte loads; the ids likewise)
  const int l0 = tid * EPT;
  const size_t e = blk0 + l0;
  const int nv = max(0, min(EPT, nblk - l0));
  uint8_t v[EPT];
  int32_t id[IDS ? EPT : 1];
  if (nv == EPT) {
#pragma unroll
    for (int h = 0; h < EPT / 16; ++h) {
      const uint4 q = *reinterpret_cast<const uint4*>(flags + e + 16 * h);
      const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int j = 0; j < 16; ++j) v[16 * h + j] = (w4[j >> 2] >> (8 * (j & 3))) & 0xff;
    }
    if constexpr (IDS) {
#pragma unroll
      for (int j = 0; j < EPT / 4; ++j) {
        const int4 o4 = *reinterpret_cast<const int4*>(orig + e + 4 * j);
        id[4 * j] = o4.x;
        id[4 * j + 1] = o4.y;
        id[4 * j + 2] = o4.z;
        id[4 * j + 3] = o4.w;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      v[j] = j < nv ? flags[e + j] : 0;
      if constexpr (IDS) id[j] = j < nv ? orig[e + j] : 0;
    }
  }
  int c = 0;
#pragma unroll
  for (int j = 0; j < EPT; ++j) c += (j < nv && v[j] != 0);

  // the block's count (waves in order), published before anything waits
  const int incl = wave_incl_scan(c);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int below = incl - c, agg = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (w < wave) below += wsum[w];
    agg += wsum[w];
  }
  if (tid == 0) status_put(st + b, (b == 0 ? kStPrefix : kStCount) | static_cast<uint64_t>(agg));

  // stage the partition: ones from the front, zeros from the back
  int r1 = below;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    if (j < nv) {
      const int slot = v[j] ? r1 : NB - 1 - (l0 + j - r1);
      spos[slot] = static_cast<uint16_t>(l0 + j);
      if constexpr (IDS) sorg[slot] = id[j];
      r1 += v[j] != 0;
    }
  }

  // ones of the earlier blocks: wave 0 first waits for the block just
  // before (one word, polled by one lane), then reads the status words
  // backwards, 64 a round, to the nearest inclusive prefix
  if (wave == 0) {
    long long excl = 0;
    int fail = 0, spins = 0;
    if (b > 0) {
      if (lane == 0)
        while ((status_get(st + b - 1) >> 62) == 0 && spins <= kSpinLimit) backoff(spins++);
      spins = __shfl(spins, 0, 64);
      int top = b - 1;
      while (true) {
        const int k = top - lane;
        // below block 0 reads as an empty prefix, so the walk always ends
        const uint64_t w = k >= 0 ? status_get(st + k) : kStPrefix;
        const uint64_t pre = __ballot((w >> 62) == 2);
        const uint64_t empty = __ballot((w >> 62) == 0);
        const int lim = pre ? __builtin_ctzll(pre) : 63;   // nearest word with a prefix
        const uint64_t upto = lim == 63 ? ~0ull : ((2ull << lim) - 1);
        if (empty & upto) {
          if (++spins > kSpinLimit) {
            fail = 1;
            break;
          }
          backoff(spins);
          continue;
        }
        excl += wave_sum_ll(lane <= lim ? static_cast<long long>(w & kStValue) : 0);
        if (pre) break;
        top -= 64;
      }
      if (lane == 0 && !fail) status_put(st + b, kStPrefix | static_cast<uint64_t>(excl + agg));
    }
    if (lane == 0) {
      s_excl = excl;
      s_fail = fail;
      if (fail) {
        counts[0] = -1;
        counts[1] = -1;
      } else if (b == nbl - 1) {
        counts[0] = static_cast<int32_t>(excl + agg);
        counts[1] = static_cast<int32_t>(static_cast<long long>(n) - (excl + agg));
      }
    }
  }
  __syncthreads();
  if (s_fail) return;
  const long long base1 = s_excl, base0 = static_cast<long long>(blk0) - base1;
  for (int k = tid; k < agg; k += 256) {
    const int32_t row = static_cast<int32_t>(blk0 + spos[k]);
    idx1[base1 + k] = row;
    if (org1) org1[base1 + k] = IDS ? sorg[k] : row;
  }
  const int zeros = nblk - agg;
  for (int k = tid; k < zeros; k += 256) {
    const int32_t row = static_cast<int32_t>(blk0 + spos[NB - 1 - k]);
    idx0[base0 + k] = row;
    if (org0) org0[base0 + k] = IDS ? sorg[NB - 1 - k] : row;
  }
}

size_t compact_workspace(size_t n) {
  const size_t nb = (n + kCompactBlockI - 1) / kCompactBlockI;
  return nb * sizeof(uint64_t) + 256;
}

void compact_large(const uint8_t* flags, const int32_t* orig, size_t n, int32_t* idx1, int32_t* org1, int32_t* idx0,
                   int32_t* org0, int32_t* counts, void* workspace, hipStream_t s, const int32_t* nc) {
  const int NB = orig ? kCompactBlockI : kCompactBlock;
  const int nb = static_cast<int>((n + NB - 1) / NB);
  uint64_t* st = static_cast<uint64_t*>(workspace);
  hipLaunchKernelGGL(compact_clear_kernel, dim3((nb + 255) / 256), dim3(256), 0, s, st, nb, counts);
  if (nb <= 0) return;
  if (orig)
    hipLaunchKernelGGL(compact_chain_kernel<true>, dim3(nb), dim3(256), 0, s, flags, orig, n, st, idx1, org1, idx0,
                       org0, counts, nc);
  else
    hipLaunchKernelGGL(compact_chain_kernel<false>, dim3(nb), dim3(256), 0, s, flags, orig, n, st, idx1, org1, idx0,
                       org0, counts, nc);
}

// Library-owned scratch of the allocation-free compaction entry point: the
// block status words of up to kScratchCompactMaxN flags (or the
// two id lists of a small partition whose caller passes none).  Each GPU the
// library runs on holds one copy until the process ends.  In host code the
// array's name is not a device address: compact_scratch() resolves it once
// per device and only that address is ever handed to a kernel.
__device__ __align__(256) uint8_t scratch[kScratchBytes];
static_assert(((kScratchCompactMaxN + kCompactBlockI - 1) / kCompactBlockI) * sizeof(uint64_t) + 256 <= kScratchBytes,
              "scratch too small for the largest chained partition it takes");
static_assert(8 * 16384 <= kScratchBytes, "scratch too small for the ids of a single-workgroup partition");

void* compact_scratch() {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    addr[dev] = ptr;
  }
  return addr[dev];
}

// ------------------------------------------------------------ row moves ---

// Work item w = row * chunks + chunk (chunk: 1024 16-byte vectors of a row),
// taken by workgroups in a grid-stride loop over the live rows' items: the
// first workgroups take the live rows, surplus ones (device counts) leave.
constexpr size_t kMoveMaxGrid = size_t(1) << 20;

__global__ __launch_bounds__(256) void move_rows_kernel(uint4* __restrict__ dst, const int32_t* __restrict__ dst_idx,
                                                        const uint4* __restrict__ src,
                                                        const int32_t* __restrict__ src_idx, size_t vpr,
                                                        const int32_t* nc, int n) {
  const size_t chunks = (vpr + 1023) / 1024;
  const size_t items = chunks * static_cast<size_t>(live(nc, n));
  for (size_t w = blockIdx.x; w < items; w += gridDim.x) {
    const size_t r = w / chunks;
    const size_t d = dst_idx ? static_cast<size_t>(dst_idx[r]) : r;
    const size_t sr = src_idx ? static_cast<size_t>(src_idx[r]) : r;
    const uint4* sp = src + sr * vpr;
    uint4* dp = dst + d * vpr;
    const size_t v0 = (w - r * chunks) * 1024 + threadIdx.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const size_t v = v0 + static_cast<size_t>(j) * 256;
      if (v < vpr) dp[v] = sp[v];
    }
  }
}

// several tensors moved with the same index lists in one launch: work item
// w = (row * count + tensor) * chunks + chunk
__global__ __launch_bounds__(256) void move_rows_multi_kernel(MoveSet set, const int32_t* __restrict__ dst_idx,
                                                              const int32_t* __restrict__ src_idx, int chunks,
                                                              const int32_t* nc, int n) {
  const size_t items = static_cast<size_t>(live(nc, n)) * set.count * chunks;
  for (size_t w = blockIdx.x; w < items; w += gridDim.x) {
    const size_t rt = w / chunks;
    const size_t r = rt / set.count;
    const int t = static_cast<int>(rt - r * set.count);
    const size_t vpr = set.vpr[t];
    const size_t v0 = (w - rt * chunks) * 1024 + threadIdx.x;
    if (v0 >= vpr) continue;
    const size_t d = dst_idx ? static_cast<size_t>(dst_idx[r]) : r;
    const size_t sr = src_idx ? static_cast<size_t>(src_idx[r]) : r;
    const uint4* sp = static_cast<const uint4*>(set.src[t]) + sr * vpr;
    uint4* dp = static_cast<uint4*>(set.dst[t]) + d * vpr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const size_t v = v0 + static_cast<size_t>(j) * 256;
      if (v < vpr) dp[v] = sp[v];
    }
  }
}

void move_rows_multi(const MoveSet& set, const int32_t* dst_idx, const int32_t* src_idx, int n, hipStream_t s,
                     const int32_t* nc) {
  size_t maxv = 0;
  for (int t = 0; t < set.count; ++t) maxv = set.vpr[t] > maxv ? set.vpr[t] : maxv;
  const int chunks = static_cast<int>((maxv + 1023) / 1024);
  const size_t items = static_cast<size_t>(n) * set.count * chunks;
  const dim3 grid(static_cast<unsigned>(items < kMoveMaxGrid ? items : kMoveMaxGrid));
  hipLaunchKernelGGL(move_rows_multi_kernel, grid, dim3(256), 0, s, set, dst_idx, src_idx, chunks, nc, n);
}

void move_rows(void* dst, const int32_t* dst_idx, const void* src, const int32_t* src_idx, size_t row_bytes, int n,
               hipStream_t s, const int32_t* nc) {
  const size_t vpr = row_bytes / 16;
  const size_t items = (vpr + 1023) / 1024 * static_cast<size_t>(n);
  const dim3 grid(static_cast<unsigned>(items < kMoveMaxGrid ? items : kMoveMaxGrid));
  hipLaunchKernelGGL(move_rows_kernel, grid, dim3(256), 0, s, static_cast<uint4*>(dst), dst_idx,
                     static_cast<const uint4*>(src), src_idx, vpr, nc, n);
}

// ------------------------------------------------------------- maxpool ----

__global__ __launch_bounds__(256) void maxpool_kernel(const uint16_t* __restrict__ x, int H, int W, int C, int Ho,
                                                      int Wo, uint16_t* __restrict__ y, size_t total,
                                                      const int32_t* nc, int n) {
  const size_t t = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;   // one 8-channel vector
  if (nc) total = total / n * live(nc, n);   // the vectors of the live images
  if (t >= total) return;
  const int C8 = C >> 3;
  const int cv = static_cast<int>(t % C8);
  size_t pix = t / C8;
  const int ow = static_cast<int>(pix % Wo);
  pix /= Wo;
  const int oh = static_cast<int>(pix % Ho);
  const size_t img = pix / Ho;
  float m[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) m[j] = -INFINITY;
  for (int i = 0; i < 3; ++i) {
    const int ih = 2 * oh - 1 + i;
    if ((unsigned)ih >= (unsigned)H) continue;
    for (int jw = 0; jw < 3; ++jw) {
      const int iw = 2 * ow - 1 + jw;
      if ((unsigned)iw >= (unsigned)W) continue;
      const uint4 v = *reinterpret_cast<const uint4*>(x + ((img * H + ih) * W + iw) * C + cv * 8);
      const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        m[2 * q] = fmaxf(m[2 * q], __uint_as_float(w4[q] << 16));
        m[2 * q + 1] = fmaxf(m[2 * q + 1], __uint_as_float(w4[q] & 0xffff0000u));
      }
    }
  }
  uint4 o;
  uint32_t* op = reinterpret_cast<uint32_t*>(&o);
#pragma unroll
  for (int q = 0; q < 4; ++q)   // maxima of bf16 values are bf16 values: exact
    op[q] = (__float_as_uint(m[2 * q]) >> 16) | (__float_as_uint(m[2 * q + 1]) & 0xffff0000u);
  *reinterpret_cast<uint4*>(y + t * 8) = o;
}

void maxpool3s2_bf16(const uint16_t* x, int n, int H, int W, int C, uint16_t* y, hipStream_t s, const int32_t* nc) {
  const int Ho = (H + 2 - 3) / 2 + 1, Wo = (W + 2 - 3) / 2 + 1;
  const size_t total = static_cast<size_t>(n) * Ho * Wo * (C / 8);
  hipLaunchKernelGGL(maxpool_kernel, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, s, x, H, W, C,
                     Ho, Wo, y, total, nc, n);
}

// ---------------------------------------------------- stem input padding ----

__global__ __launch_bounds__(256) void pad_channels_kernel(const uint16_t* __restrict__ x, size_t pixels, int cin,
                                                           uint16_t* __restrict__ y) {
  const size_t p = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (p >= pixels) return;
  uint16_t e[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int c = 0; c < cin && c < 8; ++c) e[c] = x[p * cin + c];
  uint4 o;
  o.x = e[0] | (uint32_t(e[1]) << 16);
  o.y = e[2] | (uint32_t(e[3]) << 16);
  o.z = e[4] | (uint32_t(e[5]) << 16);
  o.w = e[6] | (uint32_t(e[7]) << 16);
  *reinterpret_cast<uint4*>(y + p * 8) = o;
}

void pad_channels_bf16(const uint16_t* x, size_t pixels, int cin, int cout, uint16_t* y, hipStream_t s) {
  (void)cout;   // always 8
  hipLaunchKernelGGL(pad_channels_kernel, dim3(static_cast<unsigned>((pixels + 255) / 256)), dim3(256), 0, s, x,
                     pixels, cin, y);
}

// --------------------------------------------------------------- small ----

__global__ void final_counts_kernel(const int32_t* nc, int n, int32_t* counts) {
  if (threadIdx.x == 0) {
    counts[0] = live(nc, n);
    counts[1] = 0;
  }
}

void final_counts(const int32_t* nc, int n, int32_t* counts, hipStream_t s) {
  hipLaunchKernelGGL(final_counts_kernel, dim3(1), dim3(64), 0, s, nc, n, counts);
}

__global__ void init_records_kernel(dycl_record* rec, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) {
    rec[i].exit_index = -1;
    rec[i].iterations = 0;
    rec[i].skip_mask = 0;
  }
}

void init_records(dycl_record* rec, int n, hipStream_t s) {
  hipLaunchKernelGGL(init_records_kernel, dim3((n + 255) / 256), dim3(256), 0, s, rec, n);
}

__global__ void fill_f32_kernel(float* p, float v, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

void fill_f32(float* p, float v, int n, hipStream_t s) {
  hipLaunchKernelGGL(fill_f32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, v, n);
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, size_t n) {
  const size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

void fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t s) {
  if (n == 0) return;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s, p, v, n);
}

__global__ void gather_i32_kernel(int32_t* dst, const int32_t* __restrict__ src, const int32_t* __restrict__ idx,
                                  int n, const int32_t* nc) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < live(nc, n)) dst[i] = src[idx[i]];
}

void gather_i32(int32_t* dst, const int32_t* src, const int32_t* idx, int n, hipStream_t s, const int32_t* nc) {
  hipLaunchKernelGGL(gather_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, src, idx, n, nc);
}

// ------------------------------------------------------ greedy decoding ----
// One wave per row: each lane scans float4 pieces of the row (lanes on
// consecutive pieces), keeps its largest value and that value's lowest
// index, and the wave merges the lanes' pairs by shuffles with the same
// rule, so ties go to the lowest index whatever the scan order.

__device__ __forceinline__ void better(float v, int i, float& bv, int& bi) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

__global__ __launch_bounds__(256) void decode_step_kernel(const float* __restrict__ Z, int n, int V, int eos, int step,
                                                          int max_len, const int32_t* __restrict__ orig,
                                                          uint8_t* flags, int32_t* tok_next, int32_t* tokens,
                                                          float* logits, dycl_record* rec, const int32_t* nc) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= live(nc, n)) return;
  const float4* zr = reinterpret_cast<const float4*>(Z + static_cast<size_t>(r) * V);
  const int V4 = V / 4;
  float bv = -INFINITY;
  int bi = V;
  // sixteen 16-byte loads in flight per lane before the comparisons (the
  // winner, the largest value and the lowest index among equals, does not
  // depend on the order in which a lane visits its values)
  int j = lane;
  for (; j + 64 * 15 < V4; j += 64 * 16) {
    float4 q[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) q[u] = zr[j + 64 * u];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i0 = 4 * (j + 64 * u);
      better(q[u].x, i0, bv, bi);
      better(q[u].y, i0 + 1, bv, bi);
      better(q[u].z, i0 + 2, bv, bi);
      better(q[u].w, i0 + 3, bv, bi);
    }
  }
  for (; j < V4; j += 64) {
    const float4 q = zr[j];
    better(q.x, 4 * j, bv, bi);
    better(q.y, 4 * j + 1, bv, bi);
    better(q.z, 4 * j + 2, bv, bi);
    better(q.w, 4 * j + 3, bv, bi);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    better(ov, oi, bv, bi);
  }
  const int tok = bi < V ? bi : 0;   // every logit NaN: token 0
  const bool done = tok == eos || step == max_len;
  const int o = orig[r];
  if (lane == 0) {
    flags[r] = done ? 1 : 0;
    tok_next[r] = tok;
    tokens[static_cast<size_t>(o) * max_len + step - 1] = tok;
    if (done) rec[o].iterations = step;
  }
  if (done) {
    float4* lr = reinterpret_cast<float4*>(logits + static_cast<size_t>(o) * V);
    for (int jj = lane; jj < V4; jj += 64) lr[jj] = zr[jj];
  }
}

void decode_step(const float* Z, int n, int V, int eos, int step, int max_len, const int32_t* orig, uint8_t* flags,
                 int32_t* tok_next, int32_t* tokens, float* logits, dycl_record* rec, hipStream_t s,
                 const int32_t* nc) {
  hipLaunchKernelGGL(decode_step_kernel, dim3((n + 3) / 4), dim3(256), 0, s, Z, n, V, eos, step, max_len, orig, flags,
                     tok_next, tokens, logits, rec, nc);
}

__global__ void iota_kernel(int32_t* p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = i;
}

void iota_i32(int32_t* p, int n, hipStream_t s) {
  hipLaunchKernelGGL(iota_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, n);
}

}  // namespace k
}  // namespace dycl
