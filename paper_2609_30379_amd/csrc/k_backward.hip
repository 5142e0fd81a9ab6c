// Backward of the packed LayerNorm + Linear (Sec. 3.3, V' = V W^T + b after a
// LayerNorm on each row's features) for a training step (Sec. 3.4).
//
// Pieces, each one launch over all rows:
//   * ln_rows_kernel          LN(x) in bf16 (what the forward product consumed)
//                             and each row's mean and 1/std;
//   * gemm_bf16_kernel        C (+)= op(A) op(B), bf16 operands from memory,
//                             fp32 accumulation on matrix cores, 64 x 64 tiles,
//                             optional split of the contraction into partial
//                             sums (the weight gradients reduce over all rows);
//   * gelu / swiglu backward  elementwise, on the recomputed pre-activations;
//   * ln_backward_kernel      dx from d(LN(x)), with per-workgroup partial sums
//                             of dgamma and dbeta;
//   * column_sum / partials   bias gradients and the reduction of partials.
// Partial sums are written per workgroup and reduced in a fixed order, so
// every gradient is deterministic.
#include <algorithm>

#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kBM = 64, kBN = 64, kBK = 32;
constexpr int kLdsK = kBK + 8;      // LDS row stride (bf16) of a staged tile

// C[M, N] (+)= alpha * op(A)[M, K] op(B)[K, N] over the contraction range of
// split z (blockIdx.z): rows k in [z * kchunk, min(K, (z + 1) * kchunk)).
//   op(A)[m, k] = TA ? A[k * lda + m] : A[m * lda + k]
//   op(B)[k, n] = TB ? B[n * ldb + k] : B[k * ldb + n]
// With splits > 1 the result of split z goes to C + z * split_stride (the
// caller reduces the partials).  Element loads are bounds-checked, so M, N
// and K are arbitrary; 16-byte loads are used where a whole 8-element piece
// is in range and aligned.
template <bool TA, bool TB>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(int M, int N, int K, const bf16* __restrict__ A,
                                                         int64_t lda, const bf16* __restrict__ B, int64_t ldb,
                                                         float* __restrict__ C, int64_t ldc, float alpha,
                                                         int accumulate, int kchunk, int64_t split_stride) {
  __shared__ __attribute__((aligned(16))) bf16 As[kBM * kLdsK];
  __shared__ __attribute__((aligned(16))) bf16 Bs[kBN * kLdsK];
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN;
  const int kbeg = blockIdx.z * kchunk, kend = min(K, kbeg + kchunk);
  C += (int64_t)blockIdx.z * split_stride;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l16 = lane & 15, g = lane >> 4;
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // staging: tile rows r (m or n) with their kBK contraction values contiguous
  auto stage_rowmajor = [&](bf16* S, const bf16* P, int64_t ld, int r0, int R, int k0) {
    // P[r * ld + k]: thread -> row tid / 4, 8-element piece tid % 4
    const int r = tid >> 2, kc = (tid & 3) * 8;
    const int gr = r0 + r, gk = k0 + kc;
    bf16x8 v;
    if (gr < R && gk + 8 <= kend && ((ld | gk) & 7) == 0) {
      v = *reinterpret_cast<const bf16x8*>(P + (int64_t)gr * ld + gk);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (gr < R && gk + e < kend) ? P[(int64_t)gr * ld + gk + e] : (bf16)0.f;
    }
    *reinterpret_cast<bf16x8*>(&S[r * kLdsK + kc]) = v;
  };
  auto stage_colmajor = [&](bf16* S, const bf16* P, int64_t ld, int r0, int R, int k0) {
    // P[k * ld + r]: thread -> contraction index tid / 8, 8 consecutive rows (tid % 8) * 8
    const int k = tid >> 3, rc = (tid & 7) * 8;
    const int gk = k0 + k, gr = r0 + rc;
    bf16x8 v;
    if (gk < kend && gr + 8 <= R && ((ld | gr) & 7) == 0) {
      v = *reinterpret_cast<const bf16x8*>(P + (int64_t)gk * ld + gr);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (gk < kend && gr + e < R) ? P[(int64_t)gk * ld + gr + e] : (bf16)0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) S[(rc + e) * kLdsK + k] = v[e];
  };

  for (int k0 = kbeg; k0 < kend; k0 += kBK) {
    if (TA) stage_colmajor(As, A, lda, m0, M, k0); else stage_rowmajor(As, A, lda, m0, M, k0);
    if (TB) stage_rowmajor(Bs, B, ldb, n0, N, k0); else stage_colmajor(Bs, B, ldb, n0, N, k0);
    __syncthreads();
    bf16x8 af[2], bfr[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) af[i] = *reinterpret_cast<const bf16x8*>(&As[(wm * 32 + i * 16 + l16) * kLdsK + g * 8]);
#pragma unroll
    for (int j = 0; j < 2; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(&Bs[(wn * 32 + j * 16 + l16) * kLdsK + g * 8]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma16(af[i], bfr[j], acc[i][j]);
    __syncthreads();
  }
  // lane l holds rows 4 (l / 16) + e of each 16 x 16 subtile, column l % 16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm * 32 + i * 16 + g * 4 + e, n = n0 + wn * 32 + j * 16 + l16;
        if (m < M && n < N) {
          float* c = C + (int64_t)m * ldc + n;
          const float v = alpha * acc[i][j][e];
          *c = accumulate ? *c + v : v;
        }
      }
}

// out[i] (+)= sum_s part[s * stride + i], i < n: fixed order over s.
__global__ void __launch_bounds__(256) reduce_partials_kernel(const float* __restrict__ part, int splits,
                                                              int64_t stride, int64_t n, float* __restrict__ out,
                                                              int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[(int64_t)z * stride + i];
  out[i] = accumulate ? out[i] + s : s;
}

// First level of a long partial sum: part2[y * n + i] = sum of part[z * stride
// + i] over z in [64 y, min(splits, 64 y + 64)).  A workgroup takes 64
// outputs and one slice; its four waves each add every fourth partial of
// the slice, and the four sums are combined in a fixed order.
__global__ void __launch_bounds__(256) reduce_level1_kernel(const float* __restrict__ part, int splits,
                                                            int64_t stride, int64_t n, float* __restrict__ part2) {
  __shared__ float s[4][64];
  const int col = threadIdx.x & 63, sub = threadIdx.x >> 6;
  const int64_t i = (int64_t)blockIdx.x * 64 + col;
  const int z0 = blockIdx.y * 64, z1 = min(splits, z0 + 64);
  float a = 0.f;
  if (i < n)
    for (int z = z0 + sub; z < z1; z += 4) a += part[(int64_t)z * stride + i];
  s[sub][col] = a;
  __syncthreads();
  if (sub == 0 && i < n) part2[(int64_t)blockIdx.y * n + i] = (s[0][col] + s[1][col]) + (s[2][col] + s[3][col]);
}

// Column sums of a bf16 matrix [R, N] (row stride ld, N and ld multiples of
// 8): workgroup b sums rows [b * rpb, ...) into part[b * N + n].  A thread
// reads 16-byte pieces (8 columns); when N / 8 < 256 the rows of the group
// are dealt to 256 / (N / 8) thread subsets, combined in a fixed order.
__global__ void __launch_bounds__(256) column_partials_vec_kernel(const bf16* __restrict__ X, int64_t ld, int R,
                                                                  int N, int rpb, float* __restrict__ part) {
  __shared__ float s[2048];
  const int chunks = N / 8, subsets = max(1, 256 / chunks);
  const int r0 = blockIdx.x * rpb, r1 = min(R, r0 + rpb);
  for (int ch0 = 0; ch0 < chunks; ch0 += 256 / subsets) {
    const int ch = ch0 + threadIdx.x % (256 / subsets), sub = threadIdx.x / (256 / subsets);
    float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (ch < chunks && sub < subsets)
      for (int r = r0 + sub; r < r1; r += subsets) {
        const uint4 v = *reinterpret_cast<const uint4*>(X + (int64_t)r * ld + ch * 8);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          a[2 * e] += __uint_as_float(w[e] << 16);
          a[2 * e + 1] += __uint_as_float(w[e] & 0xffff0000u);
        }
      }
    __syncthreads();
    if (ch < chunks && sub < subsets)
#pragma unroll
      for (int e = 0; e < 8; ++e) s[sub * (256 / subsets) * 8 + (ch - ch0) * 8 + e] = a[e];
    __syncthreads();
    for (int c = threadIdx.x; c < (256 / subsets) * 8; c += 256) {
      const int col = ch0 * 8 + c;
      if (col >= N) continue;
      float t = 0.f;
      for (int u = 0; u < subsets; ++u) t += s[u * (256 / subsets) * 8 + c];
      part[(int64_t)blockIdx.x * N + col] = t;
    }
  }
}

// Column sums of a bf16 or fp32 matrix [R, N] (row stride ld): workgroup b
// sums rows [b * rpb, ...) into part[b * N + n].
template <typename T>
__global__ void __launch_bounds__(256) column_partials_kernel(const T* __restrict__ X, int64_t ld, int R, int N,
                                                              int rpb, float* __restrict__ part) {
  const int r0 = blockIdx.x * rpb, r1 = min(R, r0 + rpb);
  for (int n = threadIdx.x; n < N; n += 256) {
    float s = 0.f;
    for (int r = r0; r < r1; ++r) s += to_f32(X[(int64_t)r * ld + n]);
    part[(int64_t)blockIdx.x * N + n] = s;
  }
}

// One wave per row: xn = LN(x) gamma + beta rounded to bf16 (the values the
// forward product consumed), and the row's mean and 1/std.
template <typename T>
__global__ void __launch_bounds__(256) ln_rows_kernel(const T* __restrict__ x, int64_t ldx, int R, int K,
                                                      const float* __restrict__ gamma,
                                                      const float* __restrict__ beta, float eps,
                                                      bf16* __restrict__ xn, float* __restrict__ mean,
                                                      float* __restrict__ rstd) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= R) return;
  const T* xr = x + (int64_t)row * ldx;
  float s = 0.f;
  for (int c = lane; c < K; c += 64) s += to_f32(xr[c]);
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  const float mu = s / (float)K;
  float v = 0.f;
  for (int c = lane; c < K; c += 64) {
    const float d = to_f32(xr[c]) - mu;
    v += d * d;
  }
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  const float rs = rsqrtf(v / (float)K + eps);
  for (int c = lane; c < K; c += 64)
    xn[(int64_t)row * K + c] = (bf16)((to_f32(xr[c]) - mu) * rs * gamma[c] + (beta ? beta[c] : 0.f));
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// LN(x) rows for bf16 x with K in {64, 128, 256, 512} (ldx a multiple of 8):
// K / 8 lanes per row, each with one 16-byte piece of 8 channels, 64 / (K/8)
// rows per wave.
template <int K>
__global__ void __launch_bounds__(256) ln_rows_vec_kernel(const bf16* __restrict__ x, int64_t ldx, int R,
                                                          const float* __restrict__ gamma,
                                                          const float* __restrict__ beta, float eps,
                                                          bf16* __restrict__ xn, float* __restrict__ mean,
                                                          float* __restrict__ rstd) {
  constexpr int LPR = K / 8, RPW = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LPR, rw = lane / LPR;
  const int row = (blockIdx.x * 4 + wave) * RPW + rw;
  const bool ok = row < R;
  float v[8];
  {
    const uint4 q = ok ? *reinterpret_cast<const uint4*>(x + (int64_t)row * ldx + sub * 8) : make_uint4(0, 0, 0, 0);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(w[e] << 16);
      v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) s += v[e];
  for (int m = LPR / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  const float mu = s / (float)K;
  float q2 = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) q2 += (v[e] - mu) * (v[e] - mu);
  for (int m = LPR / 2; m >= 1; m >>= 1) q2 += __shfl_xor(q2, m, 64);
  const float rs = rsqrtf(q2 / (float)K + eps);
  if (!ok) return;
  const float4 g0 = *reinterpret_cast<const float4*>(gamma + sub * 8), g1 = *reinterpret_cast<const float4*>(gamma + sub * 8 + 4);
  float4 b0 = make_float4(0.f, 0.f, 0.f, 0.f), b1 = b0;
  if (beta) {
    b0 = *reinterpret_cast<const float4*>(beta + sub * 8);
    b1 = *reinterpret_cast<const float4*>(beta + sub * 8 + 4);
  }
  const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const float bb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (bf16)((v[e] - mu) * rs * gg[e] + bb[e]);
  *reinterpret_cast<bf16x8*>(xn + (int64_t)row * K + sub * 8) = o;
  if (sub == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// LayerNorm backward for bf16 x with K in {64, 128, 256, 512}, the layout of
// ln_rows_vec_kernel (K / 8 lanes per row, 16-byte pieces): workgroup b takes
// rows [b * rpb, ...), its waves stepping 4 * (64 / (K/8)) rows at a time, and
// writes the group's partial sums of d(LN x) xhat and d(LN x), combined in a
// fixed order (over the rows of a lane, then the row slots of a wave, then
// the waves).
template <int K, typename TO>
__global__ void __launch_bounds__(256) ln_backward_vec_kernel(const float* __restrict__ dxn,
                                                              const bf16* __restrict__ x, int64_t ldx, int R,
                                                              const float* __restrict__ gamma,
                                                              const float* __restrict__ mean,
                                                              const float* __restrict__ rstd,
                                                              const TO* __restrict__ res, int64_t ld_res,
                                                              TO* __restrict__ dx, int64_t ld_dx, int accumulate,
                                                              int rpb, float* __restrict__ part_g,
                                                              float* __restrict__ part_b) {
  constexpr int LPR = K / 8, RPW = 64 / LPR;
  __shared__ float sg[4][K], sb[4][K];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LPR, rw = lane / LPR;
  float pg[8], pb[8], gm[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    pg[e] = pb[e] = 0.f;
    gm[e] = gamma[sub * 8 + e];
  }
  const int r0 = blockIdx.x * rpb, r1 = min(R, r0 + rpb);
  for (int rb = r0; rb < r1; rb += 4 * RPW) {
    const int row = rb + wave * RPW + rw;
    const bool ok = row < r1;
    float d[8], xh[8], gv[8];
    const float mu = ok ? mean[row] : 0.f, rs = ok ? rstd[row] : 0.f;
    {
      float4 d0 = make_float4(0.f, 0.f, 0.f, 0.f), d1 = d0;
      uint4 q = make_uint4(0, 0, 0, 0);
      if (ok) {
        d0 = *reinterpret_cast<const float4*>(dxn + (int64_t)row * K + sub * 8);
        d1 = *reinterpret_cast<const float4*>(dxn + (int64_t)row * K + sub * 8 + 4);
        q = *reinterpret_cast<const uint4*>(x + (int64_t)row * ldx + sub * 8);
      }
      const float dd[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
      const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        xh[2 * e] = (__uint_as_float(w[e] << 16) - mu) * rs;
        xh[2 * e + 1] = (__uint_as_float(w[e] & 0xffff0000u) - mu) * rs;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = dd[e];
    }
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      gv[e] = d[e] * gm[e];
      s1 += gv[e];
      s2 += gv[e] * xh[e];
      pg[e] += d[e] * xh[e];
      pb[e] += d[e];
    }
    for (int m = LPR / 2; m >= 1; m >>= 1) {
      s1 += __shfl_xor(s1, m, 64);
      s2 += __shfl_xor(s2, m, 64);
    }
    s1 /= (float)K;
    s2 /= (float)K;
    if (!ok) continue;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = rs * (gv[e] - s1 - xh[e] * s2);
    if (res) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += to_f32(res[(int64_t)row * ld_res + sub * 8 + e]);
    }
    TO* o = dx + (int64_t)row * ld_dx + sub * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = from_f32<TO>(accumulate ? to_f32(o[e]) + v[e] : v[e]);
  }
  // lanes sub, sub + LPR, ... of a wave hold the same channels: combine them
  for (int m = LPR; m < 64; m <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pg[e] += __shfl_xor(pg[e], m, 64);
      pb[e] += __shfl_xor(pb[e], m, 64);
    }
  if (rw == 0)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sg[wave][sub * 8 + e] = pg[e];
      sb[wave][sub * 8 + e] = pb[e];
    }
  __syncthreads();
  for (int c = threadIdx.x; c < K; c += 256) {
    part_g[(int64_t)blockIdx.x * K + c] = (sg[0][c] + sg[1][c]) + (sg[2][c] + sg[3][c]);
    part_b[(int64_t)blockIdx.x * K + c] = (sb[0][c] + sb[1][c]) + (sb[2][c] + sb[3][c]);
  }
}

// LayerNorm backward, one wave per row (4 rows per workgroup, rpb rows per
// partial group):  g = d(LN x) * gamma,  xhat = (x - mean) rstd,
//   dx = rstd (g - mean(g) - xhat mean(g xhat))  (+ res, + dx if accumulating)
// and the group's partial sums of d(LN x) xhat (dgamma) and d(LN x) (dbeta).
template <typename T, typename TO>
__global__ void __launch_bounds__(256) ln_backward_kernel(const float* __restrict__ dxn, const T* __restrict__ x,
                                                          int64_t ldx, int R, int K, const float* __restrict__ gamma,
                                                          const float* __restrict__ mean,
                                                          const float* __restrict__ rstd, const TO* __restrict__ res,
                                                          int64_t ld_res, TO* __restrict__ dx, int64_t ld_dx,
                                                          int accumulate, int rpb, float* __restrict__ part_g,
                                                          float* __restrict__ part_b) {
  constexpr int kMaxPer = 16;                   // K <= 1024
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ float sg[4][1024], sb[4][1024];
  float pg[kMaxPer], pb[kMaxPer];
#pragma unroll
  for (int j = 0; j < kMaxPer; ++j) pg[j] = pb[j] = 0.f;
  const int r0 = blockIdx.x * rpb, r1 = min(R, r0 + rpb);
  for (int row = r0 + wave; row < r1; row += 4) {
    const float mu = mean[row], rs = rstd[row];
    float gv[kMaxPer], xh[kMaxPer];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxPer; ++j) {
      const int c = lane + 64 * j;
      gv[j] = xh[j] = 0.f;
      if (c < K) {
        const float d = dxn[(int64_t)row * K + c];
        xh[j] = (to_f32(x[(int64_t)row * ldx + c]) - mu) * rs;
        gv[j] = d * gamma[c];
        s1 += gv[j];
        s2 += gv[j] * xh[j];
        pg[j] += d * xh[j];
        pb[j] += d;
      }
    }
    for (int m = 32; m >= 1; m >>= 1) {
      s1 += __shfl_xor(s1, m, 64);
      s2 += __shfl_xor(s2, m, 64);
    }
    s1 /= (float)K;
    s2 /= (float)K;
#pragma unroll
    for (int j = 0; j < kMaxPer; ++j) {
      const int c = lane + 64 * j;
      if (c < K) {
        float v = rs * (gv[j] - s1 - xh[j] * s2);
        if (res) v += to_f32(res[(int64_t)row * ld_res + c]);
        TO* o = dx + (int64_t)row * ld_dx + c;
        *o = from_f32<TO>(accumulate ? to_f32(*o) + v : v);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxPer; ++j) {
    const int c = lane + 64 * j;
    if (c < K) {
      sg[wave][c] = pg[j];
      sb[wave][c] = pb[j];
    }
  }
  __syncthreads();
  for (int c = threadIdx.x; c < K; c += 256) {
    part_g[(int64_t)blockIdx.x * K + c] = (sg[0][c] + sg[1][c]) + (sg[2][c] + sg[3][c]);
    part_b[(int64_t)blockIdx.x * K + c] = (sb[0][c] + sb[1][c]) + (sb[2][c] + sb[3][c]);
  }
}

// d(pre-activation) of the GELU epilogue: dp = dy * gelu'(pre + bias), stored bf16.
__global__ void __launch_bounds__(256) gelu_backward_kernel(const float* __restrict__ pre, const float* __restrict__ bias,
                                                            const bf16* __restrict__ dy, int64_t ld_dy, int R, int N,
                                                            bf16* __restrict__ dp) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)R * N) return;
  const int64_t r = e / N, n = e % N;
  const float x = pre[e] + (bias ? bias[n] : 0.f);
  const float cdf = 0.5f * (1.f + erff(x * 0.70710678f));
  const float pdf = 0.39894228f * __expf(-0.5f * x * x);
  dp[e] = (bf16)((float)dy[r * ld_dy + n] * (cdf + x * pdf));
}

// SwiGLU: from [g | u] (fp32 products, [R, 2F], plus the bias) and
// dh = dy W2 (fp32, [R, F]):
//   h = silu(g) u (bf16, for dW2),  dp = [dh u silu'(g) | dh silu(g)] (bf16)
// A thread takes 8 consecutive hidden units of a row (F a multiple of 8):
// 32-byte reads and 16-byte writes.
__global__ void __launch_bounds__(256) swiglu_backward_kernel(const float* __restrict__ gu,
                                                              const float* __restrict__ bias,
                                                              const float* __restrict__ dh, int R, int F,
                                                              bf16* __restrict__ h, bf16* __restrict__ dp) {
  const int64_t e8 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e8 >= (int64_t)R * F / 8) return;
  const int64_t r = e8 / (F / 8);
  const int f0 = (int)(e8 % (F / 8)) * 8;
  const float* gp = gu + r * 2 * F + f0;
  const float* up = gp + F;
  const float* dp_in = dh + r * F + f0;
  float gv[8], uv[8], dv[8];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const float4 a = *reinterpret_cast<const float4*>(gp + 4 * q), b = *reinterpret_cast<const float4*>(up + 4 * q);
    const float4 c = *reinterpret_cast<const float4*>(dp_in + 4 * q);
    gv[4 * q] = a.x; gv[4 * q + 1] = a.y; gv[4 * q + 2] = a.z; gv[4 * q + 3] = a.w;
    uv[4 * q] = b.x; uv[4 * q + 1] = b.y; uv[4 * q + 2] = b.z; uv[4 * q + 3] = b.w;
    dv[4 * q] = c.x; dv[4 * q + 1] = c.y; dv[4 * q + 2] = c.z; dv[4 * q + 3] = c.w;
  }
  if (bias) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float4 bg = *reinterpret_cast<const float4*>(bias + f0 + 4 * q);
      const float4 bu = *reinterpret_cast<const float4*>(bias + F + f0 + 4 * q);
      gv[4 * q] += bg.x; gv[4 * q + 1] += bg.y; gv[4 * q + 2] += bg.z; gv[4 * q + 3] += bg.w;
      uv[4 * q] += bu.x; uv[4 * q + 1] += bu.y; uv[4 * q + 2] += bu.z; uv[4 * q + 3] += bu.w;
    }
  }
  bf16x8 ho, go, uo;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float g = gv[j], u = uv[j], d = dv[j];
    const float sg = 1.f / (1.f + __expf(-g));
    const float silu = g * sg;
    ho[j] = (bf16)(silu * u);
    go[j] = (bf16)(d * u * sg * (1.f + g * (1.f - sg)));
    uo[j] = (bf16)(d * silu);
  }
  *reinterpret_cast<bf16x8*>(h + r * F + f0) = ho;
  *reinterpret_cast<bf16x8*>(dp + r * 2 * F + f0) = go;
  *reinterpret_cast<bf16x8*>(dp + r * 2 * F + F + f0) = uo;
}

// ---------------------------------------------------------------- fused SwiGLU backward
// h and d[g | u] straight from the rows, for K = N in {64, 128} and F a
// multiple of 64: workgroup (unit block ub, row block rb) owns hidden units
// [64 ub, 64 ub + 64) and row tiles [rb * kSgRT, ...).  The gate, up and
// W2^T rows of its units are copied once into LDS as fragment images (lane
// (l16, g) of image (t, kk) = row 16 t + l16, columns 32 kk + 8 g .. +7); each
// wave takes 16-row tiles, reads LN(x) and dy straight into B fragments and
// runs, per 16-unit tile t, the products
//   G = Wg LN(x)^T,  U = Wu LN(x)^T,  D = W2^T dy^T
// so lane (l16, g) holds units 16 t + 4 g + i of row l16; the SwiGLU
// derivative is applied in registers (the same fp32 formulas as the unfused
// path) and h, d g, d u are stored as 8-byte pieces.  The workgroups of one
// row block run on one XCD, so its rows are read from HBM once.
constexpr int kSgRT = 64;                     // row tiles (of 16) per workgroup

template <int K>
__global__ void __launch_bounds__(256, 4) swiglu_backward_fused_kernel(const bf16* __restrict__ xn, int64_t ld_xn,
                                                                    const bf16* __restrict__ dy, int64_t ld_dy,
                                                                    const bf16* __restrict__ W,
                                                                    const bf16* __restrict__ W2T,
                                                                    const float* __restrict__ bias, int R, int F,
                                                                    bf16* __restrict__ h, bf16* __restrict__ dp) {
  constexpr int KT = K / 32;
  __shared__ __attribute__((aligned(16))) bf16 img[3 * 4 * KT * 512];   // [which][t][kk] images
  const int nub = F / 64, nrb = (R + 16 * kSgRT - 1) / (16 * kSgRT);
  const int ub = (blockIdx.x / kXcds) % nub;
  const int rb = (blockIdx.x / (kXcds * nub)) * kXcds + blockIdx.x % kXcds;
  if (rb >= nrb) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int u0 = ub * 64;
  // weight images: which 0 = gate rows, 1 = up rows (of W), 2 = rows of W2^T
  for (int im = wave; im < 3 * 4 * KT; im += 4) {
    const int which = im / (4 * KT), t = (im / KT) % 4, kk = im % KT;
    const bf16* src = which == 2 ? W2T + (int64_t)(u0 + 16 * t + l16) * K + kk * 32 + g * 8
                                 : W + (int64_t)(which * F + u0 + 16 * t + l16) * K + kk * 32 + g * 8;
    __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(img + im * 512), 16, 0, 0);
  }
  float bg[4][4], bu[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int f = u0 + 16 * t + 4 * g;
    const float4 a = bias ? *reinterpret_cast<const float4*>(bias + f) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 b = bias ? *reinterpret_cast<const float4*>(bias + F + f) : make_float4(0.f, 0.f, 0.f, 0.f);
    bg[t][0] = a.x; bg[t][1] = a.y; bg[t][2] = a.z; bg[t][3] = a.w;
    bu[t][0] = b.x; bu[t][1] = b.y; bu[t][2] = b.z; bu[t][3] = b.w;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const int rt0 = rb * kSgRT, rt1 = min((R + 15) / 16, rt0 + kSgRT);
  // rows of tile rt as B fragments; the next tile's are loaded while the
  // current one is computed (rows past R repeat the last, never stored)
  auto load_rows = [&](int rt, bf16x8 (&xf)[KT], bf16x8 (&df)[KT]) {
    const int rr = min(rt * 16 + l16, R - 1);
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      xf[kk] = *reinterpret_cast<const bf16x8*>(xn + (int64_t)rr * ld_xn + kk * 32 + g * 8);
      df[kk] = *reinterpret_cast<const bf16x8*>(dy + (int64_t)rr * ld_dy + kk * 32 + g * 8);
    }
  };
  bf16x8 xn_n[KT], dy_n[KT];
  if (rt0 + wave < rt1) load_rows(rt0 + wave, xn_n, dy_n);
  for (int rt = rt0 + wave; rt < rt1; rt += 4) {
    const int row = rt * 16 + l16;
    bf16x8 xf[KT], df[KT];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      xf[kk] = xn_n[kk];
      df[kk] = dy_n[kk];
    }
    if (rt + 4 < rt1) load_rows(rt + 4, xn_n, dy_n);
    // the weight fragments are read from LDS for every row tile: an opaque
    // lane offset keeps the compiler from holding all of them in registers
    int lo = lane * 8;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      f32x4 G = {0.f, 0.f, 0.f, 0.f}, U = G, D = G;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const bf16x8 ag = *reinterpret_cast<const bf16x8*>(img + ((0 * 4 + t) * KT + kk) * 512 + lo);
        const bf16x8 au = *reinterpret_cast<const bf16x8*>(img + ((1 * 4 + t) * KT + kk) * 512 + lo);
        const bf16x8 ad = *reinterpret_cast<const bf16x8*>(img + ((2 * 4 + t) * KT + kk) * 512 + lo);
        G = mfma16(ag, xf[kk], G);
        U = mfma16(au, xf[kk], U);
        D = mfma16(ad, df[kk], D);
      }
      bf16x4 ho, go, uo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float gv = G[i] + bg[t][i], uv = U[i] + bu[t][i], d = D[i];
        const float sg = 1.f / (1.f + __expf(-gv));
        const float silu = gv * sg;
        ho[i] = (bf16)(silu * uv);
        go[i] = (bf16)(d * uv * sg * (1.f + gv * (1.f - sg)));
        uo[i] = (bf16)(d * silu);
      }
      // a lane past R computed row R - 1 (its input row was clamped) and
      // stores those same values there: no divergent branch, so the waits
      // for the next tile's rows stay exact
      const int f = u0 + 16 * t + 4 * g;
      const int64_t ro = min(row, R - 1);
      *reinterpret_cast<bf16x4*>(h + ro * F + f) = ho;
      *reinterpret_cast<bf16x4*>(dp + ro * 2 * F + f) = go;
      *reinterpret_cast<bf16x4*>(dp + ro * 2 * F + F + f) = uo;
    }
  }
}

// W2 [N, F] -> W2^T [F, N] (bf16), one thread per element.
__global__ void __launch_bounds__(256) transpose_bf16_kernel(const bf16* __restrict__ a, int rows, int cols,
                                                             bf16* __restrict__ at) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)rows * cols) return;
  const int r = (int)(e / cols), c = (int)(e % cols);
  at[(int64_t)c * rows + r] = a[e];
}

// fp32 matrix [R, N] -> bf16 (row stride N).
__global__ void __launch_bounds__(256) to_bf16_kernel(const float* __restrict__ x, int64_t n, bf16* __restrict__ y) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n) y[e] = (bf16)x[e];
}

unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }

// Splits of a contraction of length K so the grid has about 1024 workgroups.
int splits_for(int64_t tiles, int64_t K) {
  const int64_t want = std::max<int64_t>(1, 1024 / std::max<int64_t>(1, tiles));
  return (int)std::min<int64_t>(want, std::max<int64_t>(1, K / 256));
}

// Workspace carve-out, 256-byte aligned pieces.
struct Carve {
  char* p;
  size_t used = 0;
  template <typename T> T* take(size_t n) {
    T* r = reinterpret_cast<T*>(p ? p + used : nullptr);
    used += (n * sizeof(T) + 255) / 256 * 256;
    return r;
  }
};

constexpr int kRowsPerGroup = 256;   // rows per partial group of the LayerNorm and column sums

// Plans (and, with launch, runs) the backward; with ws == nullptr it only
// counts the workspace bytes.
hipError_t run_linear_backward(const nt_linear_bwd_args& a, void* ws, size_t* bytes, hipStream_t s, bool launch) {
  const int R = (int)a.rows, K = a.c_in;
  const bool swiglu = a.epilogue == NT_EPI_SWIGLU_RESIDUAL, gelu = a.epilogue == NT_EPI_GELU;
  const int F = a.hidden;
  const int Nw = swiglu ? 2 * F : a.c_out;             // rows of W
  const bool ln = a.ln_gamma != nullptr;
  const bool xf = a.x_dtype == NT_F32;
  const bool dxf = a.dx_dtype == NT_F32;
  if (swiglu && F % 8 != 0) return hipErrorInvalidValue;
  // bf16 rows of K in {64, 128, 256, 512}: the LayerNorm passes read 16-byte
  // pieces, K / 8 lanes per row, and partial groups are 64 rows
  const bool vec_ln = !xf && (K == 64 || K == 128 || K == 256 || K == 512) && a.ldx % 8 == 0;
  const int rpg = vec_ln ? 64 : kRowsPerGroup;
  Carve c{static_cast<char*>(ws)};
  bf16* xn = (ln || xf) ? c.take<bf16>((size_t)R * K) : nullptr;       // LN(x), or x in bf16
  float* mean = ln ? c.take<float>(R) : nullptr;
  float* rstd = ln ? c.take<float>(R) : nullptr;
  // SwiGLU with K = N in {64, 128}: h and d[g | u] come from one fused
  // kernel, without the fp32 pre-activations and dh
  const bool sg_fused = swiglu && (K == 64 || K == 128) && a.c_out == K && F % 64 == 0 && a.ld_dy % 8 == 0 &&
                        (ln || xf || a.ldx % 8 == 0);
  float* pre = (gelu || (swiglu && !sg_fused)) ? c.take<float>((size_t)R * Nw) : nullptr;   // recomputed pre-activation
  float* dh = (swiglu && !sg_fused) ? c.take<float>((size_t)R * F) : nullptr;
  bf16* w2t = sg_fused ? c.take<bf16>((size_t)F * a.c_out) : nullptr;                       // W2^T [F, N]
  bf16* h = swiglu ? c.take<bf16>((size_t)R * F) : nullptr;
  bf16* dp = (gelu || swiglu) ? c.take<bf16>((size_t)R * Nw) : nullptr;        // d(pre-activation), bf16
  const bool direct_dx = !ln && dxf;                                      // the product writes dx itself
  float* dxn = direct_dx ? nullptr : c.take<float>((size_t)R * K);
  const int groups = (R + rpg - 1) / rpg;
  float* part_g = c.take<float>((size_t)groups * K);
  float* part_b = c.take<float>((size_t)groups * K);
  float* part_col = c.take<float>((size_t)groups * std::max(Nw, a.c_out));

  const int64_t tiles_w = (int64_t)((Nw + kBM - 1) / kBM) * ((K + kBN - 1) / kBN);
  const int sw = splits_for(tiles_w, R);
  float* part_w = c.take<float>((size_t)sw * Nw * K);
  const int64_t tiles_w2 = (int64_t)((a.c_out + kBM - 1) / kBM) * ((F + kBN - 1) / kBN);
  const int sw2 = swiglu ? splits_for(tiles_w2, R) : 0;
  float* part_w2 = swiglu ? c.take<float>((size_t)sw2 * a.c_out * F) : nullptr;
  // second level of the reductions with more than 64 partials
  auto slices = [](int64_t splits) -> size_t { return splits > 64 ? (size_t)((splits + 63) / 64) : 0; };
  const size_t n2 = std::max({slices(groups) * (size_t)std::max(std::max(Nw, a.c_out), K),
                              slices(sw) * (size_t)Nw * K, slices(sw2) * (size_t)a.c_out * F});
  float* part2 = c.take<float>(std::max<size_t>(n2, 1));
  *bytes = c.used;
  if (!launch) return hipSuccess;

  const bf16* W = (const bf16*)a.w;
  const bf16* dy = (const bf16*)a.dy;
  const int acc_w = a.overwrite_weights ? 0 : 1;
  const dim3 b256(256);
  // out (+)= sum over `splits` partials (stride apart) of n values, in a fixed
  // order: through part2 when there are more than 64 partials
  auto reduce_parts = [&](const float* part, int splits, int64_t stride, int64_t n, float* out) {
    if (splits > 64) {
      const int sl = (splits + 63) / 64;
      reduce_level1_kernel<<<dim3((unsigned)((n + 63) / 64), (unsigned)sl), b256, 0, s>>>(part, splits, stride, n, part2);
      reduce_partials_kernel<<<blocks_for(n), b256, 0, s>>>(part2, sl, n, n, out, acc_w);
    } else {
      reduce_partials_kernel<<<blocks_for(n), b256, 0, s>>>(part, splits, stride, n, out, acc_w);
    }
  };
  // column sums of a bf16 [R, N] matrix into part_col (groups of rpg rows)
  auto column_parts = [&](const bf16* X, int64_t ld, int N) {
    if (N % 8 == 0 && ld % 8 == 0 && N <= 2048)
      column_partials_vec_kernel<<<dim3(groups), b256, 0, s>>>(X, ld, R, N, rpg, part_col);
    else
      column_partials_kernel<bf16><<<dim3(groups), b256, 0, s>>>(X, ld, R, N, rpg, part_col);
  };
  // LN(x) (or x) in bf16 as the forward product consumed it, with the row statistics
  const bf16* xin = (const bf16*)a.x;
  int64_t ld_xin = a.ldx;
  if (ln) {
    if (vec_ln) {
#define NT_LNR(KK)                                                                                             \
      ln_rows_vec_kernel<KK><<<dim3((unsigned)((R + 4 * (512 / KK) - 1) / (4 * (512 / KK)))), b256, 0, s>>>( \
          (const bf16*)a.x, a.ldx, R, a.ln_gamma, a.ln_beta, a.ln_eps, xn, mean, rstd)
      if (K == 64) NT_LNR(64); else if (K == 128) NT_LNR(128); else if (K == 256) NT_LNR(256); else NT_LNR(512);
#undef NT_LNR
    } else if (xf)
      ln_rows_kernel<float><<<dim3((R + 3) / 4), b256, 0, s>>>((const float*)a.x, a.ldx, R, K, a.ln_gamma, a.ln_beta,
                                                              a.ln_eps, xn, mean, rstd);
    else
      ln_rows_kernel<bf16><<<dim3((R + 3) / 4), b256, 0, s>>>((const bf16*)a.x, a.ldx, R, K, a.ln_gamma, a.ln_beta,
                                                             a.ln_eps, xn, mean, rstd);
    xin = xn;
    ld_xin = K;
  } else if (xf) {
    if (a.ldx != K) return hipErrorInvalidValue;
    to_bf16_kernel<<<blocks_for((int64_t)R * K), b256, 0, s>>>((const float*)a.x, (int64_t)R * K, xn);
    xin = xn;
    ld_xin = K;
  }
  // d(pre-activation): dy itself, or through the GELU / SwiGLU epilogue
  const bf16* g = dy;
  int64_t ld_g = a.ld_dy;
  if (gelu || swiglu) {
    // pre = LN(x) W^T + b
    // (the bias is added where the pre-activation is read)
    if (!sg_fused)
      gemm_bf16_kernel<false, true><<<dim3((R + kBM - 1) / kBM, (Nw + kBN - 1) / kBN, 1), b256, 0, s>>>(
          R, Nw, K, xin, ld_xin, W, K, pre, Nw, 1.f, 0, K, 0);
    if (sg_fused) {
      transpose_bf16_kernel<<<blocks_for((int64_t)a.c_out * F), b256, 0, s>>>((const bf16*)a.w2, a.c_out, F, w2t);
      const int nrb = (R + 16 * kSgRT - 1) / (16 * kSgRT);
      const dim3 grid((unsigned)((nrb + kXcds - 1) / kXcds * kXcds * (F / 64)));
      if (K == 64)
        swiglu_backward_fused_kernel<64><<<grid, b256, 0, s>>>(xin, ld_xin, dy, a.ld_dy, W, w2t, a.bias, R, F, h, dp);
      else
        swiglu_backward_fused_kernel<128><<<grid, b256, 0, s>>>(xin, ld_xin, dy, a.ld_dy, W, w2t, a.bias, R, F, h, dp);
    } else if (gelu) {
      gelu_backward_kernel<<<blocks_for((int64_t)R * Nw), b256, 0, s>>>(pre, a.bias, dy, a.ld_dy, R, Nw, dp);
    } else {
      // dh = dy W2 (W2 [N, F]),  h = silu(g) u,  dp = d[g | u]
      gemm_bf16_kernel<false, false><<<dim3((R + kBM - 1) / kBM, (F + kBN - 1) / kBN, 1), b256, 0, s>>>(
          R, F, a.c_out, dy, a.ld_dy, (const bf16*)a.w2, F, dh, F, 1.f, 0, a.c_out, 0);
      swiglu_backward_kernel<<<blocks_for((int64_t)R * F / 8), b256, 0, s>>>(pre, a.bias, dh, R, F, h, dp);
    }
    if (swiglu) {
      // dW2 += dy^T h,  db2 += sum_rows dy
      if (a.dw2) {
        const int kc = (R + sw2 - 1) / sw2;
        gemm_bf16_kernel<true, false><<<dim3((a.c_out + kBM - 1) / kBM, (F + kBN - 1) / kBN, sw2), b256, 0, s>>>(
            a.c_out, F, R, dy, a.ld_dy, h, F, part_w2, F, 1.f, 0, kc, (int64_t)a.c_out * F);
        reduce_parts(part_w2, sw2, (int64_t)a.c_out * F, (int64_t)a.c_out * F, a.dw2);
      }
      if (a.db2) {
        column_parts(dy, a.ld_dy, a.c_out);
        reduce_parts(part_col, groups, a.c_out, a.c_out, a.db2);
      }
    }
    g = dp;
    ld_g = Nw;
  }
  // weight and bias gradients: dW += g^T LN(x),  db += sum_rows g
  if (a.dw) {
    const int kc = (R + sw - 1) / sw;
    gemm_bf16_kernel<true, false><<<dim3((Nw + kBM - 1) / kBM, (K + kBN - 1) / kBN, sw), b256, 0, s>>>(
        Nw, K, R, g, ld_g, xin, ld_xin, part_w, K, 1.f, 0, kc, (int64_t)Nw * K);
    reduce_parts(part_w, sw, (int64_t)Nw * K, (int64_t)Nw * K, a.dw);
  }
  if (a.db) {
    column_parts(g, ld_g, Nw);
    reduce_parts(part_col, groups, Nw, Nw, a.db);
  }
  const bf16* res = swiglu && a.residual_is_x ? dy : nullptr;
  if (direct_dx) {
    // no LayerNorm, fp32 dx: dx (+)= g W directly
    if (a.dx)
      gemm_bf16_kernel<false, false><<<dim3((R + kBM - 1) / kBM, (K + kBN - 1) / kBN, 1), b256, 0, s>>>(
          R, K, Nw, g, ld_g, W, K, (float*)a.dx, a.ld_dx, 1.f, a.accumulate_dx, Nw, 0);
    return hipGetLastError();
  }
  // d(LN x) = g W  (W stored [Nw, K])
  if (a.dx || a.dgamma || a.dbeta) {
    gemm_bf16_kernel<false, false><<<dim3((R + kBM - 1) / kBM, (K + kBN - 1) / kBN, 1), b256, 0, s>>>(
        R, K, Nw, g, ld_g, W, K, dxn, K, 1.f, 0, Nw, 0);
  }
  if (ln) {
#define NT_LNB(TX, TO)                                                                                          \
    ln_backward_kernel<TX, TO><<<dim3(groups), b256, 0, s>>>(dxn, (const TX*)a.x, a.ldx, R, K, a.ln_gamma, mean, \
                                                            rstd, (const TO*)res, a.ld_dy, (TO*)a.dx, a.ld_dx,  \
                                                            a.accumulate_dx, rpg, part_g, part_b)
#define NT_LNBV(KK, TO)                                                                                         \
    ln_backward_vec_kernel<KK, TO><<<dim3(groups), b256, 0, s>>>(dxn, (const bf16*)a.x, a.ldx, R, a.ln_gamma,    \
                                                                mean, rstd, (const TO*)res, a.ld_dy, (TO*)a.dx, \
                                                                a.ld_dx, a.accumulate_dx, rpg, part_g, part_b)
#define NT_LNBK(TO) do { if (K == 64) NT_LNBV(64, TO); else if (K == 128) NT_LNBV(128, TO);                     \
                         else if (K == 256) NT_LNBV(256, TO); else NT_LNBV(512, TO); } while (0)
    if (res && dxf) return hipErrorInvalidValue;     // the SwiGLU residual is bf16
    if (vec_ln) { if (dxf) NT_LNBK(float); else NT_LNBK(bf16); }
    else if (xf) { if (dxf) NT_LNB(float, float); else NT_LNB(float, bf16); }
    else { if (dxf) NT_LNB(bf16, float); else NT_LNB(bf16, bf16); }
#undef NT_LNBK
#undef NT_LNBV
#undef NT_LNB
    if (a.dgamma) reduce_parts(part_g, groups, K, K, a.dgamma);
    if (a.dbeta) reduce_parts(part_b, groups, K, K, a.dbeta);
  } else if (a.dx) {
    // no LayerNorm, bf16 dx = d(LN x)
    if (a.accumulate_dx || res) return hipErrorInvalidValue;
    to_bf16_kernel<<<blocks_for((int64_t)R * K), b256, 0, s>>>(dxn, (int64_t)R * K, (bf16*)a.dx);
  }
  return hipGetLastError();
}

}  // namespace

size_t linear_backward_workspace_bytes(const nt_linear_bwd_args& a) {
  size_t n = 0;
  run_linear_backward(a, nullptr, &n, nullptr, false);
  return n;
}

hipError_t launch_linear_backward(const nt_linear_bwd_args& a, void* ws, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  size_t n = 0;
  return run_linear_backward(a, ws, &n, s, true);
}

}  // namespace nt
