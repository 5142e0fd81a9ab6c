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

// d(pre-activation) of the GELU epilogue: dp = dy * gelu'(pre), stored bf16.
__global__ void __launch_bounds__(256) gelu_backward_kernel(const float* __restrict__ pre, const bf16* __restrict__ dy,
                                                            int64_t ld_dy, int R, int N, bf16* __restrict__ dp) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)R * N) return;
  const int64_t r = e / N, n = e % N;
  const float x = pre[e];
  const float cdf = 0.5f * (1.f + erff(x * 0.70710678f));
  const float pdf = 0.39894228f * __expf(-0.5f * x * x);
  dp[e] = (bf16)((float)dy[r * ld_dy + n] * (cdf + x * pdf));
}

// SwiGLU: from [g | u] (fp32, [R, 2F]) and dh = dy W2 (fp32, [R, F]):
//   h = silu(g) u (bf16, for dW2),  dp = [dh u silu'(g) | dh silu(g)] (bf16)
__global__ void __launch_bounds__(256) swiglu_backward_kernel(const float* __restrict__ gu, const float* __restrict__ dh,
                                                              int R, int F, bf16* __restrict__ h,
                                                              bf16* __restrict__ dp) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)R * F) return;
  const int64_t r = e / F, f = e % F;
  const float g = gu[r * 2 * F + f], u = gu[r * 2 * F + F + f], d = dh[e];
  const float sg = 1.f / (1.f + __expf(-g));
  const float silu = g * sg;
  h[e] = (bf16)(silu * u);
  dp[r * 2 * F + f] = (bf16)(d * u * sg * (1.f + g * (1.f - sg)));
  dp[r * 2 * F + F + f] = (bf16)(d * silu);
}

// Adds a bias row to an fp32 matrix [R, N] (row stride N).
__global__ void __launch_bounds__(256) add_bias_kernel(float* __restrict__ y, int R, int N,
                                                       const float* __restrict__ bias) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < (int64_t)R * N) y[e] += bias[e % N];
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
  Carve c{static_cast<char*>(ws)};
  bf16* xn = (ln || xf) ? c.take<bf16>((size_t)R * K) : nullptr;       // LN(x), or x in bf16
  float* mean = ln ? c.take<float>(R) : nullptr;
  float* rstd = ln ? c.take<float>(R) : nullptr;
  float* pre = (gelu || swiglu) ? c.take<float>((size_t)R * Nw) : nullptr;     // recomputed pre-activation
  float* dh = swiglu ? c.take<float>((size_t)R * F) : nullptr;
  bf16* h = swiglu ? c.take<bf16>((size_t)R * F) : nullptr;
  bf16* dp = (gelu || swiglu) ? c.take<bf16>((size_t)R * Nw) : nullptr;        // d(pre-activation), bf16
  const bool direct_dx = !ln && dxf;                                      // the product writes dx itself
  float* dxn = direct_dx ? nullptr : c.take<float>((size_t)R * K);
  const int groups = (R + kRowsPerGroup - 1) / kRowsPerGroup;
  float* part_g = c.take<float>((size_t)groups * K);
  float* part_b = c.take<float>((size_t)groups * K);
  float* part_col = c.take<float>((size_t)groups * std::max(Nw, a.c_out));
  const int64_t tiles_w = (int64_t)((Nw + kBM - 1) / kBM) * ((K + kBN - 1) / kBN);
  const int sw = splits_for(tiles_w, R);
  float* part_w = c.take<float>((size_t)sw * Nw * K);
  const int64_t tiles_w2 = (int64_t)((a.c_out + kBM - 1) / kBM) * ((F + kBN - 1) / kBN);
  const int sw2 = swiglu ? splits_for(tiles_w2, R) : 0;
  float* part_w2 = swiglu ? c.take<float>((size_t)sw2 * a.c_out * F) : nullptr;
  *bytes = c.used;
  if (!launch) return hipSuccess;

  const bf16* W = (const bf16*)a.w;
  const bf16* dy = (const bf16*)a.dy;
  const int acc_w = a.overwrite_weights ? 0 : 1;
  const dim3 b256(256);
  // LN(x) (or x) in bf16 as the forward product consumed it, with the row statistics
  const bf16* xin = (const bf16*)a.x;
  int64_t ld_xin = a.ldx;
  if (ln) {
    if (xf)
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
    gemm_bf16_kernel<false, true><<<dim3((R + kBM - 1) / kBM, (Nw + kBN - 1) / kBN, 1), b256, 0, s>>>(
        R, Nw, K, xin, ld_xin, W, K, pre, Nw, 1.f, 0, K, 0);
    if (a.bias) add_bias_kernel<<<blocks_for((int64_t)R * Nw), b256, 0, s>>>(pre, R, Nw, a.bias);
    if (gelu) {
      gelu_backward_kernel<<<blocks_for((int64_t)R * Nw), b256, 0, s>>>(pre, dy, a.ld_dy, R, Nw, dp);
    } else {
      // dh = dy W2 (W2 [N, F]),  h = silu(g) u,  dp = d[g | u]
      gemm_bf16_kernel<false, false><<<dim3((R + kBM - 1) / kBM, (F + kBN - 1) / kBN, 1), b256, 0, s>>>(
          R, F, a.c_out, dy, a.ld_dy, (const bf16*)a.w2, F, dh, F, 1.f, 0, a.c_out, 0);
      swiglu_backward_kernel<<<blocks_for((int64_t)R * F), b256, 0, s>>>(pre, dh, R, F, h, dp);
      // dW2 += dy^T h,  db2 += sum_rows dy
      if (a.dw2) {
        const int kc = (R + sw2 - 1) / sw2;
        gemm_bf16_kernel<true, false><<<dim3((a.c_out + kBM - 1) / kBM, (F + kBN - 1) / kBN, sw2), b256, 0, s>>>(
            a.c_out, F, R, dy, a.ld_dy, h, F, part_w2, F, 1.f, 0, kc, (int64_t)a.c_out * F);
        reduce_partials_kernel<<<blocks_for((int64_t)a.c_out * F), b256, 0, s>>>(part_w2, sw2, (int64_t)a.c_out * F,
                                                                                (int64_t)a.c_out * F, a.dw2, acc_w);
      }
      if (a.db2) {
        column_partials_kernel<bf16><<<dim3(groups), b256, 0, s>>>(dy, a.ld_dy, R, a.c_out, kRowsPerGroup, part_col);
        reduce_partials_kernel<<<blocks_for(a.c_out), b256, 0, s>>>(part_col, groups, a.c_out, a.c_out, a.db2, acc_w);
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
    reduce_partials_kernel<<<blocks_for((int64_t)Nw * K), b256, 0, s>>>(part_w, sw, (int64_t)Nw * K, (int64_t)Nw * K,
                                                                        a.dw, acc_w);
  }
  if (a.db) {
    column_partials_kernel<bf16><<<dim3(groups), b256, 0, s>>>(g, ld_g, R, Nw, kRowsPerGroup, part_col);
    reduce_partials_kernel<<<blocks_for(Nw), b256, 0, s>>>(part_col, groups, Nw, Nw, a.db, acc_w);
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
                                                            a.accumulate_dx, kRowsPerGroup, part_g, part_b)
    if (res && dxf) return hipErrorInvalidValue;     // the SwiGLU residual is bf16
    if (xf) { if (dxf) NT_LNB(float, float); else NT_LNB(float, bf16); }
    else { if (dxf) NT_LNB(bf16, float); else NT_LNB(bf16, bf16); }
#undef NT_LNB
    if (a.dgamma)
      reduce_partials_kernel<<<blocks_for(K), b256, 0, s>>>(part_g, groups, K, K, a.dgamma, acc_w);
    if (a.dbeta)
      reduce_partials_kernel<<<blocks_for(K), b256, 0, s>>>(part_b, groups, K, K, a.dbeta, acc_w);
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
