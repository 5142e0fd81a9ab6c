// Pair broadcast and segment reductions: HBM-streaming kernels that walk the
// packed rows of one sample per workgroup.
#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

// Pair broadcast (Eq. running-block, first line): one workgroup per pair row
// (sample i, row a) writes the M_i contiguous cells o_i + a M_i + b (M_i = N_i
// for square pairs), each C channels wide, as 16-byte coalesced stores.  v's
// rows of the sample are re-read by every row of the sample and stay in L2.
template <typename T>
__global__ void __launch_bounds__(256)
pair_broadcast_kernel(const int32_t* __restrict__ row_sample, const int32_t* __restrict__ cu_seqlens,
                      const int32_t* __restrict__ cu_cols, const int32_t* __restrict__ cu_pairs, int C,
                      const T* __restrict__ u, int64_t ld_u, const T* __restrict__ v, int64_t ld_v,
                      T* __restrict__ z, int64_t ld_z, int accumulate) {
  constexpr int VE = Vec<T>::N;
  const int eta = blockIdx.x;
  const int i = row_sample[eta];
  const int s0 = cu_seqlens[i];
  const int k0 = cu_cols[i];
  const int n = cu_cols[i + 1] - k0;           // cells per pair row (M_i)
  const int a = eta - s0;
  const int64_t cell0 = (int64_t)cu_pairs[i] + (int64_t)a * n;
  const int cv = C / VE;                       // vector chunks per cell
  const T* urow = u + (int64_t)eta * ld_u;
  const T* vblk = v + (int64_t)k0 * ld_v;
  if (cv <= 256) {
    // every thread owns one fixed chunk of channels (the first 256 / cv * cv
    // threads take part); u is loaded once
    const int bstep = 256 / cv;
    if ((int)threadIdx.x >= bstep * cv) return;
    const int ch = (threadIdx.x % cv) * VE;
    const int b0 = threadIdx.x / cv;
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
template <typename T, typename TO>
__global__ void __launch_bounds__(256)
segment_reduce_kernel(int level, const int32_t* __restrict__ row_sample, const int32_t* __restrict__ col_sample,
                      const int32_t* __restrict__ cu_seqlens, const int32_t* __restrict__ cu_cols,
                      const int32_t* __restrict__ cu_pairs, int C, const T* __restrict__ x, int64_t ld_x,
                      TO* __restrict__ y, int64_t ld_y, int mean, int accumulate) {
  constexpr int VE = Vec<T>::N;
  constexpr int CPB = 16;                    // vector chunks per workgroup
  constexpr int G = 256 / CPB;               // row groups
  __shared__ float part[G][CPB * VE];
  const int seg = blockIdx.x;
  int64_t base, step = 1;
  int n;
  if (level == NT_LEVEL_PAIRS) {               // pair row a: its M_i contiguous cells
    const int i = row_sample[seg];
    n = cu_cols[i + 1] - cu_cols[i];
    base = (int64_t)cu_pairs[i] + (int64_t)(seg - cu_seqlens[i]) * n;
  } else if (level == NT_LEVEL_PAIRS_FIRST) {  // column b: N_i cells, M_i apart
    const int i = col_sample[seg];
    const int m = cu_cols[i + 1] - cu_cols[i];
    n = cu_seqlens[i + 1] - cu_seqlens[i];
    base = (int64_t)cu_pairs[i] + (seg - cu_cols[i]);
    step = m;
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
    if (accumulate) s += to_f32(y[out_row * ld_y + c]);
    y[out_row * ld_y + c] = from_f32<TO>(s);
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
                               const int32_t* __restrict__ cu_seqlens, const int32_t* __restrict__ cu_cols,
                               const int32_t* __restrict__ cu_pairs, int C, const float* __restrict__ dy,
                               int64_t ld_dy, T* __restrict__ dx, int64_t ld_dx, int mean, int accumulate) {
  constexpr int VE = Vec<T>::N;
  const int eta = blockIdx.x;
  const int i = row_sample[eta];
  const int s0 = cu_seqlens[i];
  const int nrow = cu_seqlens[i + 1] - s0;
  const int k0 = cu_cols[i];
  const int n = cu_cols[i + 1] - k0;              // cells per pair row (M_i)
  // group sizes: M_i for a pair row, N_i for a column or a sample's rows
  const float scale = mean ? 1.f / (float)(level == NT_LEVEL_PAIRS ? n : nrow) : 1.f;
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
  if (level == NT_LEVEL_PAIRS && cv <= 256) {
    // the whole pair row takes dy[eta]: every thread owns one fixed chunk of
    // channels (the first 256 / cv * cv threads), loaded once
    const int bstep = 256 / cv;
    if ((int)threadIdx.x >= bstep * cv) return;
    const int ch = (threadIdx.x % cv) * VE;
    float gv[VE];
#pragma unroll
    for (int j = 0; j < VE; ++j) gv[j] = dy[(int64_t)(s0 + a) * ld_dy + ch + j] * scale;
    for (int b = threadIdx.x / cv; b < n; b += bstep) {
      T* dst = dx + (cell0 + b) * ld_dx + ch;
      Vec<T> out;
      if (accumulate) out.load(dst);
#pragma unroll
      for (int j = 0; j < VE; ++j) out.v[j] = (accumulate ? out.v[j] : 0.f) + gv[j];
      out.store(dst);
    }
    return;
  }
  const int total = n * cv;
  for (int t = threadIdx.x; t < total; t += 256) {
    const int b = t / cv, ch = (t - b * cv) * VE;
    const float* g = dy + (int64_t)(level == NT_LEVEL_PAIRS ? s0 + a : k0 + b) * ld_dy + ch;
    T* dst = dx + (cell0 + b) * ld_dx + ch;
    Vec<T> out;
    if (accumulate) out.load(dst);
#pragma unroll
    for (int j = 0; j < VE; ++j) out.v[j] = (accumulate ? out.v[j] : 0.f) + g[j] * scale;
    out.store(dst);
  }
}

// Weighted squared norm of every sample's rows with its gradient (the
// diagnostic loss of the measured single-pair-single program):
//   part[i * CH + c] = sum over chunk c of sample i's rows of sum_ch x^2
//   dx[r] = 2 * scale * w[i] * x[r]
// Rows of sample i are [off[i], off[i+1]) (singles: eta, pairs: o).  Grid
// (B, CH): chunk c takes an equal share of the sample's rows; partial sums are
// reduced per sample in a fixed order by loss_finish_kernel.
constexpr int kLossChunks = 256;   // workgroups per sample: enough loads in flight on a batch of 8

template <typename T, typename TO>
__global__ void __launch_bounds__(256)
weighted_sq_kernel(const int32_t* __restrict__ off, int C, const T* __restrict__ x, int64_t ld_x,
                   const float* __restrict__ w, float scale, float* __restrict__ part, TO* __restrict__ dx,
                   int64_t ld_dx, int dx_vec) {
  constexpr int VE = Vec<T>::N;
  __shared__ float red[4];
  const int i = blockIdx.x, c = blockIdx.y;
  const int64_t r0 = off[i], rows = (int64_t)off[i + 1] - r0;
  const int64_t a = r0 + rows * c / kLossChunks, b = r0 + rows * (c + 1) / kLossChunks;
  const int cv = C / VE;
  const float g = 2.f * scale * w[i];
  float acc = 0.f;
  // one chunk of VE channels: its squares, and dx = g x (one vector store
  // when dx_vec: dx and its row stride 16-byte aligned)
  auto chunk = [&](int64_t r, int ch) {
    Vec<T> t;
    t.load(x + r * ld_x + ch);
#pragma unroll
    for (int j = 0; j < VE; ++j) acc = fmaf(t.v[j], t.v[j], acc);
    if (!dx) return;
    TO* o = dx + r * ld_dx + ch;
    if (dx_vec) {
      if constexpr (sizeof(TO) == 4) {
#pragma unroll
        for (int j = 0; j < VE; j += 4)
          *reinterpret_cast<float4*>(o + j) = make_float4(g * t.v[j], g * t.v[j + 1], g * t.v[j + 2], g * t.v[j + 3]);
      } else if constexpr (VE == 8) {
        bf16x8 v;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (bf16)(g * t.v[j]);
        *reinterpret_cast<bf16x8*>(o) = v;
      } else {
        bf16x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = (bf16)(g * t.v[j]);
        *reinterpret_cast<bf16x4*>(o) = v;
      }
    } else {
#pragma unroll
      for (int j = 0; j < VE; ++j) o[j] = from_f32<TO>(g * t.v[j]);
    }
  };
  for (int64_t e = threadIdx.x; e < (b - a) * cv; e += 256) chunk(a + e / cv, (int)(e % cv) * VE);
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[i * kLossChunks + c] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ void loss_finish_kernel(const float* __restrict__ part, int B, const float* __restrict__ w, float scale,
                                   float* __restrict__ loss) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  float s = 0.f;
  for (int c = 0; c < kLossChunks; ++c) s += part[i * kLossChunks + c];
  loss[i] = scale * w[i] * s;
}

}  // namespace

size_t loss_workspace_bytes(const nt_layout& L) { return (size_t)L.batch * kLossChunks * sizeof(float); }

hipError_t launch_weighted_square_loss(const nt_layout& L, nt_level level, int C, const void* x, int64_t ld_x,
                                       nt_dtype dtype, const float* w, float scale, float* loss, void* dx,
                                       int64_t ld_dx, nt_dtype dx_dtype, void* workspace, hipStream_t s) {
  const int32_t* off = level == NT_LEVEL_PAIRS ? L.d_cu_pairs : L.d_cu_seqlens;
  float* part = static_cast<float*>(workspace);
  const dim3 grid((unsigned)L.batch, kLossChunks);
  const size_t eo = dx_dtype == NT_BF16 ? 2 : 4;
  const int dx_vec = dx && (reinterpret_cast<uintptr_t>(dx) % 16 == 0) && ((size_t)ld_dx * eo) % 16 == 0;
#define NT_LOSS(T, TO) weighted_sq_kernel<T, TO><<<grid, dim3(256), 0, s>>>(off, C, (const T*)x, ld_x, w, scale, part, \
                                                                            (TO*)dx, ld_dx, dx_vec)
  if (dtype == NT_BF16) { if (dx_dtype == NT_BF16) NT_LOSS(bf16, bf16); else NT_LOSS(bf16, float); }
  else { if (dx_dtype == NT_BF16) NT_LOSS(float, bf16); else NT_LOSS(float, float); }
#undef NT_LOSS
  loss_finish_kernel<<<dim3((L.batch + 63) / 64), dim3(64), 0, s>>>(part, L.batch, w, scale, loss);
  return hipGetLastError();
}

hipError_t launch_segment_reduce_backward(const nt_layout& L, nt_level level, int op, int C, const float* dy,
                                          int64_t ld_dy, void* dx, int64_t ld_dx, nt_dtype dtype, int accumulate,
                                          hipStream_t s) {
  if (L.sum_n == 0) return hipSuccess;
  const dim3 grid((unsigned)L.sum_n), block(256);
  if (dtype == NT_BF16)
    segment_reduce_backward_kernel<bf16><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_cu_seqlens,
                                                                L.d_cu_cols, L.d_cu_pairs, C, dy, ld_dy, (bf16*)dx,
                                                                ld_dx, op, accumulate);
  else
    segment_reduce_backward_kernel<float><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_cu_seqlens,
                                                                 L.d_cu_cols, L.d_cu_pairs, C, dy, ld_dy, (float*)dx,
                                                                 ld_dx, op, accumulate);
  return hipGetLastError();
}

hipError_t launch_pair_broadcast(const nt_layout& L, int C, const void* u, int64_t ld_u, const void* v,
                                 int64_t ld_v, void* z, int64_t ld_z, int accumulate, nt_dtype dtype,
                                 hipStream_t s) {
  if (L.sum_n == 0) return hipSuccess;
  const dim3 grid((unsigned)L.sum_n), block(256);
  if (dtype == NT_BF16)
    pair_broadcast_kernel<bf16><<<grid, block, 0, s>>>(L.d_row_sample, L.d_cu_seqlens, L.d_cu_cols, L.d_cu_pairs, C,
                                                       (const bf16*)u, ld_u, (const bf16*)v, ld_v, (bf16*)z,
                                                       ld_z, accumulate);
  else
    pair_broadcast_kernel<float><<<grid, block, 0, s>>>(L.d_row_sample, L.d_cu_seqlens, L.d_cu_cols, L.d_cu_pairs, C,
                                                        (const float*)u, ld_u, (const float*)v, ld_v,
                                                        (float*)z, ld_z, accumulate);
  return hipGetLastError();
}

hipError_t launch_segment_reduce(const nt_layout& L, nt_level level, int op, int C, const void* x,
                                 int64_t ld_x, nt_dtype x_dtype, void* y, int64_t ld_y, hipStream_t s, int accumulate,
                                 nt_dtype y_dtype) {
  const int64_t segs = level == NT_LEVEL_PAIRS ? L.sum_n : (level == NT_LEVEL_PAIRS_FIRST ? L.sum_m : L.batch);
  if (segs == 0) return hipSuccess;
  const int ve = x_dtype == NT_BF16 ? 8 : 4;
  const int cblocks = (C / ve + 15) / 16;
  const dim3 grid((unsigned)segs, (unsigned)cblocks), block(256);
#define NT_RED(T, TO)                                                                                            \
  segment_reduce_kernel<T, TO><<<grid, block, 0, s>>>((int)level, L.d_row_sample, L.d_col_sample, L.d_cu_seqlens, \
                                                      L.d_cu_cols, L.d_cu_pairs, C, (const T*)x, ld_x, (TO*)y,     \
                                                      ld_y, op, accumulate)
  if (x_dtype == NT_BF16) { if (y_dtype == NT_BF16) NT_RED(bf16, bf16); else NT_RED(bf16, float); }
  else { if (y_dtype == NT_BF16) NT_RED(float, bf16); else NT_RED(float, float); }
#undef NT_RED
  return hipGetLastError();
}

}  // namespace nt
