// Pair broadcast and segment reductions: HBM-streaming kernels that walk the
// packed rows of one sample per workgroup.
#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

// Pair broadcast (Eq. running-block, first line): one workgroup per pair row
// (sample i, row a) writes the N_i contiguous cells o_i + a N_i + b, each C
// channels wide, as 16-byte coalesced stores.  v's rows of the sample are
// re-read by every row of the sample and stay in L2.
template <typename T>
__global__ void __launch_bounds__(256)
pair_broadcast_kernel(const int32_t* __restrict__ row_sample, const int32_t* __restrict__ cu_seqlens,
                      const int32_t* __restrict__ cu_pairs, int C, const T* __restrict__ u, int64_t ld_u,
                      const T* __restrict__ v, int64_t ld_v, T* __restrict__ z, int64_t ld_z,
                      int accumulate) {
  constexpr int VE = Vec<T>::N;
  const int eta = blockIdx.x;
  const int i = row_sample[eta];
  const int s0 = cu_seqlens[i];
  const int n = cu_seqlens[i + 1] - s0;
  const int a = eta - s0;
  const int64_t cell0 = (int64_t)cu_pairs[i] + (int64_t)a * n;
  const int cv = C / VE;                       // vector chunks per cell
  const T* urow = u + (int64_t)eta * ld_u;
  const T* vblk = v + (int64_t)s0 * ld_v;
  if (256 % cv == 0) {
    // every thread owns one fixed chunk of channels; u is loaded once
    const int ch = (threadIdx.x % cv) * VE;
    const int b0 = threadIdx.x / cv, bstep = 256 / cv;
    Vec<T> uu;
    uu.load(urow + ch);
    for (int b = b0; b < n; b += bstep) {
      Vec<T> vv, out;
      vv.load(vblk + (int64_t)b * ld_v + ch);
      T* dst = z + (cell0 + b) * ld_z + ch;
      if (accumulate) out.load(dst);
#pragma unroll
      for (int j = 0; j < VE; ++j) out.v[j] = (accumulate ? out.v[j] : 0.f) + (uu.v[j] + vv.v[j]);
      out.store(dst);
    }
  } else {
    const int total = n * cv;
    for (int t = threadIdx.x; t < total; t += 256) {
      const int b = t / cv, ch = (t - b * cv) * VE;
      Vec<T> uu, vv, out;
      uu.load(urow + ch);
      vv.load(vblk + (int64_t)b * ld_v + ch);
      T* dst = z + (cell0 + b) * ld_z + ch;
      if (accumulate) out.load(dst);
#pragma unroll
      for (int j = 0; j < VE; ++j) out.v[j] = (accumulate ? out.v[j] : 0.f) + (uu.v[j] + vv.v[j]);
      out.store(dst);
    }
  }
}

// Segment reduction: workgroup (segment, channel block).  Segment = pair row
// (level pairs: the N_i contiguous cells o_i + a N_i + b of pair row a),
// first-axis group (level pairs-first: the cells o_i + a N_i + b of column b,
// N_i rows apart) or sample (level singles: N_i rows).  Threads split the
// segment's rows into 256/CPB groups; groups combine in LDS, so every output
// is written by exactly one thread (no atomics).
template <typename T>
__global__ void __launch_bounds__(256)
segment_reduce_kernel(int level, const int32_t* __restrict__ row_sample,
                      const int32_t* __restrict__ cu_seqlens, const int32_t* __restrict__ cu_pairs,
                      int C, const T* __restrict__ x, int64_t ld_x, float* __restrict__ y, int64_t ld_y,
                      int mean, int accumulate) {
  constexpr int VE = Vec<T>::N;
  constexpr int CPB = 16;                    // vector chunks per workgroup
  constexpr int G = 256 / CPB;               // row groups
  __shared__ float part[G][CPB * VE];
  const int seg = blockIdx.x;
  int64_t base, step = 1;
  int n;
  if (level != NT_LEVEL_SINGLES) {
    const int i = row_sample[seg];
    n = cu_seqlens[i + 1] - cu_seqlens[i];
    const int a = seg - cu_seqlens[i];
    if (level == NT_LEVEL_PAIRS) {
      base = (int64_t)cu_pairs[i] + (int64_t)a * n;
    } else {
      base = (int64_t)cu_pairs[i] + a;
      step = n;
    }
  } else {
    n = cu_seqlens[seg + 1] - cu_seqlens[seg];
    base = cu_seqlens[seg];
  }
  const int cl = threadIdx.x % CPB, g = threadIdx.x / CPB;
  const int chunk = blockIdx.y * CPB + cl;
  const bool active = chunk * VE < C;
  float acc[VE];
#pragma unroll
  for (int j = 0; j < VE; ++j) acc[j] = 0.f;
  if (active) {
    for (int r = g; r < n; r += G) {
      Vec<T> t;
      t.load(x + (base + (int64_t)r * step) * ld_x + chunk * VE);
#pragma unroll
      for (int j = 0; j < VE; ++j) acc[j] += t.v[j];
    }
  }
#pragma unroll
  for (int j = 0; j < VE; ++j) part[g][cl * VE + j] = acc[j];
  __syncthreads();
  for (int e = threadIdx.x; e < CPB * VE; e += 256) {
    const int c = blockIdx.y * CPB * VE + e;
    if (c >= C) continue;
    float s = 0.f;
    for (int gg = 0; gg < G; ++gg) s += part[gg][e];
    if (mean) s = n > 0 ? s / (float)n : __builtin_nanf("");
    const int64_t out_row = seg;
    if (accumulate) s += y[out_row * ld_y + c];
    y[out_row * ld_y + c] = s;
  }
}

// Backward of a segment reduction: every position of a group receives the
// group's gradient (divided by N_i for a mean), added to dx or stored.  One
// workgroup per pair row (levels pairs / pairs-first: the N_i cells of pair
// row a, from dy[eta_i + a] or dy[eta_i + b]) or per single row (level
// singles: dx[eta_i + t] from dy[i]).
template <typename T>
__global__ void __launch_bounds__(256)
segment_reduce_backward_kernel(int level, const int32_t* __restrict__ row_sample,
                               const int32_t* __restrict__ cu_seqlens, const int32_t* __restrict__ cu_pairs,
                               int C, const float* __restrict__ dy, int64_t ld_dy, T* __restrict__ dx,
                               int64_t ld_dx, int mean, int accumulate) {
  constexpr int VE = Vec<T>::N;
  const int eta = blockIdx.x;
  const int i = row_sample[eta];
  const int s0 = cu_seqlens[i];
  const int n = cu_seqlens[i + 1] - s0;
  const float scale = mean ? 1.f / (float)n : 1.f;
  const int cv = C / VE;
  if (level == NT_LEVEL_SINGLES) {
    for (int ch = threadIdx.x; ch < cv; ch += 256) {
      Vec<T> out;
      T* dst = dx + (int64_t)eta * ld_dx + ch * VE;
      if (accumulate) out.load(dst);
#pragma unroll
      for (int j = 0; j < VE; ++j)
        out.v[j] = (accumulate ? out.v[j] : 0.f) + dy[(int64_t)i * ld_dy + ch * VE + j] * scale;
      out.store(dst);
    }
    return;
  }
  const int a = eta - s0;
  const int64_t cell0 = (int64_t)cu_pairs[i] + (int64_t)a * n;
  const int total = n * cv;
  for (int t = threadIdx.x; t < total; t += 256) {
    const int b = t / cv, ch = (t - b * cv) * VE;
    const float* g = dy + (int64_t)(s0 + (level == NT_LEVEL_PAIRS ? a : b)) * ld_dy + ch;
    T* dst = dx + (cell0 + b) * ld_dx + ch;
    Vec<T> out;
    if (accumulate) out.load(dst);
#pragma unroll
    for (int j = 0; j < VE; ++j) out.v[j] = (accumulate ? out.v[j] : 0.f) + g[j] * scale;
    out.store(dst);
  }
}

}  // namespace

hipError_t launch_segment_reduce_backward(const nt_layout& L, nt_level level, int op, int C, const float* dy,
                                          int64_t ld_dy, void* dx, int64_t ld_dx, nt_dtype dtype, int accumulate,
                                          hipStream_t s) {
  if (L.sum_n == 0) return hipSuccess;
  const dim3 grid((unsigned)L.sum_n), block(256);
  if (dtype == NT_BF16)
    segment_reduce_backward_kernel<bf16><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_cu_seqlens,
                                                                L.d_cu_pairs, C, dy, ld_dy, (bf16*)dx, ld_dx, op,
                                                                accumulate);
  else
    segment_reduce_backward_kernel<float><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_cu_seqlens,
                                                                 L.d_cu_pairs, C, dy, ld_dy, (float*)dx, ld_dx, op,
                                                                 accumulate);
  return hipGetLastError();
}

hipError_t launch_pair_broadcast(const nt_layout& L, int C, const void* u, int64_t ld_u, const void* v,
                                 int64_t ld_v, void* z, int64_t ld_z, int accumulate, nt_dtype dtype,
                                 hipStream_t s) {
  if (L.sum_n == 0) return hipSuccess;
  const dim3 grid((unsigned)L.sum_n), block(256);
  if (dtype == NT_BF16)
    pair_broadcast_kernel<bf16><<<grid, block, 0, s>>>(L.d_row_sample, L.d_cu_seqlens, L.d_cu_pairs, C,
                                                       (const bf16*)u, ld_u, (const bf16*)v, ld_v, (bf16*)z,
                                                       ld_z, accumulate);
  else
    pair_broadcast_kernel<float><<<grid, block, 0, s>>>(L.d_row_sample, L.d_cu_seqlens, L.d_cu_pairs, C,
                                                        (const float*)u, ld_u, (const float*)v, ld_v,
                                                        (float*)z, ld_z, accumulate);
  return hipGetLastError();
}

hipError_t launch_segment_reduce(const nt_layout& L, nt_level level, int op, int C, const void* x,
                                 int64_t ld_x, nt_dtype x_dtype, float* y, int64_t ld_y, hipStream_t s, int accumulate) {
  const int64_t segs = level != NT_LEVEL_SINGLES ? L.sum_n : L.batch;
  if (segs == 0) return hipSuccess;
  const int ve = x_dtype == NT_BF16 ? 8 : 4;
  const int cblocks = (C / ve + 15) / 16;
  const dim3 grid((unsigned)segs, (unsigned)cblocks), block(256);
  if (x_dtype == NT_BF16)
    segment_reduce_kernel<bf16><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_cu_seqlens, L.d_cu_pairs, C,
                                                       (const bf16*)x, ld_x, y, ld_y, op, accumulate);
  else
    segment_reduce_kernel<float><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_cu_seqlens, L.d_cu_pairs, C,
                                                        (const float*)x, ld_x, y, ld_y, op, accumulate);
  return hipGetLastError();
}

}  // namespace nt
