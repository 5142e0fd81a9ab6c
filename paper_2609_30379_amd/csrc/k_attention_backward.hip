// Backward of row / column attention with pair bias (the starting- and
// ending-node attention of the Pairformer cited in Sec. 4.3) for a training
// step (Sec. 3.4).  Per sample i, pair row r and head h (axis 1: the same on
// the sample's transpose), with S = scale Q K^T + B and P = softmax_k(S):
//   lse_j = log sum_k exp S_jk,  D_j = sum_k P_jk (dO_j . V_k)  (= dO_j . O_j),
//   dS_jk = P_jk (dO_j . V_k - D_j),
//   dQ_j = scale sum_k dS_jk K_k,  dK_k = scale sum_j dS_jk Q_j,
//   dV_k = sum_j P_jk dO_j,        dB_jk = sum_r dS_jk   (the bias is shared by all rows).
//
// attn_bwd_rows_kernel: one workgroup per (pair row, head).  The row's q, k,
// v and dO (N x 32 each) are staged in LDS; every thread first takes the
// softmax statistics of its queries, then the query gradients (a thread per
// query, keys broadcast from LDS), then the key and value gradients (a thread
// per key, queries broadcast), so no sum crosses threads.  lse and D go to
// the workspace for the bias gradient.
// attn_bwd_bias_kernel: one workgroup per (sample, 16-query block, head); a
// thread per key walks all pair rows and sums dS for its 16 queries, then
// writes its column of the bias gradient once (no atomics).
// Arithmetic is fp32 on the vector units.
#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kD = 32;                 // head_dim

struct AttnBwdArgs {
  int axis, H;
  const bf16* q;
  const bf16* k;
  const bf16* v;
  int64_t ld_qkv;
  const bf16* bias;                    // NULL: no bias
  int64_t ld_bias, ld_bias_head;
  const bf16* dout;
  int64_t ld_dout;
  float scale;
  bf16* dq;
  bf16* dk;
  bf16* dv;
  int64_t ld_dqkv;
  float* dbias;
  int64_t ld_dbias, ld_dbias_head;
  float* lse;                          // workspace: [sum N^2, H] per query element
  float* dsum;                         // workspace: D, same layout
  const int32_t* work;                 // (sample, row) pairs; -1 = idle
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  const int32_t* cu_qblk;              // prefix of ceil(N_i / 16)
  int batch;
};

__device__ __forceinline__ void load32(const bf16* p, float* out) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const uint4 t = *reinterpret_cast<const uint4*>(p + c * 8);
    const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[c * 8 + 2 * j] = __uint_as_float(w[j] << 16);
      out[c * 8 + 2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
}

__device__ __forceinline__ float dot32(const float* a, const bf16* b) {
  float t[kD];
  load32(b, t);
  float s = 0.f;
#pragma unroll
  for (int d = 0; d < kD; ++d) s = fmaf(a[d], t[d], s);
  return s;
}

__device__ __forceinline__ void store32(bf16* p, const float* x, float mul) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    bf16x8 t;
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = (bf16)(x[c * 8 + e] * mul);
    *reinterpret_cast<bf16x8*>(p + c * 8) = t;
  }
}

// head-h bias of (query j, key k) of sample i (axis 1: of cell (k, j))
__device__ __forceinline__ float bias_at(const AttnBwdArgs& p, int64_t cu, int n, int j, int k, int h) {
  if (!p.bias) return 0.f;
  const int64_t cell = cu + (p.axis == 0 ? (int64_t)j * n + k : (int64_t)k * n + j);
  return (float)p.bias[cell * p.ld_bias + (int64_t)h * p.ld_bias_head];
}

template <int NMAX>
__global__ void __launch_bounds__(256) attn_bwd_rows_kernel(AttnBwdArgs p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* Qs = reinterpret_cast<bf16*>(smem);
  bf16* Ks = Qs + NMAX * kD;
  bf16* Vs = Ks + NMAX * kD;
  bf16* Gs = Vs + NMAX * kD;
  float* lse_s = reinterpret_cast<float*>(Gs + NMAX * kD);
  float* d_s = lse_s + NMAX;
  const int i = p.work[2 * blockIdx.x], r = p.work[2 * blockIdx.x + 1];
  if (i < 0) return;
  const int h = blockIdx.y;
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int64_t cu = p.cu_pairs[i];
  // element t of this row: packed row base + t * step
  const int64_t base = p.axis == 0 ? cu + (int64_t)r * n : cu + r;
  const int64_t step = p.axis == 0 ? 1 : n;
  for (int e = threadIdx.x; e < n * 4; e += 256) {
    const int t = e >> 2, c = (e & 3) * 8;
    const int64_t row = base + (int64_t)t * step;
    *reinterpret_cast<uint4*>(&Qs[t * kD + c]) = *reinterpret_cast<const uint4*>(p.q + row * p.ld_qkv + h * kD + c);
    *reinterpret_cast<uint4*>(&Ks[t * kD + c]) = *reinterpret_cast<const uint4*>(p.k + row * p.ld_qkv + h * kD + c);
    *reinterpret_cast<uint4*>(&Vs[t * kD + c]) = *reinterpret_cast<const uint4*>(p.v + row * p.ld_qkv + h * kD + c);
    *reinterpret_cast<uint4*>(&Gs[t * kD + c]) =
        *reinterpret_cast<const uint4*>(p.dout + row * p.ld_dout + h * kD + c);
  }
  __syncthreads();
  // softmax statistics of every query, and D = sum_k P_jk (dO_j . V_k),
  // accumulated with the running maximum (fp32, from the recomputed softmax)
  for (int j = threadIdx.x; j < n; j += 256) {
    float qv[kD], gv[kD];
    load32(&Qs[j * kD], qv);
    load32(&Gs[j * kD], gv);
    float m = -INFINITY, l = 0.f, acc = 0.f;
    for (int k = 0; k < n; ++k) {
      const float sv = p.scale * dot32(qv, &Ks[k * kD]) + bias_at(p, cu, n, j, k, h);
      const float dp = dot32(gv, &Vs[k * kD]);
      if (sv > m) {
        const float c = __expf(m - sv);
        l = l * c + 1.f;
        acc = acc * c + dp;
        m = sv;
      } else {
        const float e = __expf(sv - m);
        l += e;
        acc = fmaf(e, dp, acc);
      }
    }
    const int64_t row = base + (int64_t)j * step;
    const float dsum = acc / l;
    const float ls = m + __logf(l);
    lse_s[j] = ls;
    d_s[j] = dsum;
    p.lse[row * p.H + h] = ls;
    p.dsum[row * p.H + h] = dsum;
  }
  __syncthreads();
  // dQ_j = scale sum_k P_jk (dO_j . V_k - D_j) K_k
  for (int j = threadIdx.x; j < n; j += 256) {
    float qv[kD], gv[kD], acc[kD];
    load32(&Qs[j * kD], qv);
    load32(&Gs[j * kD], gv);
#pragma unroll
    for (int d = 0; d < kD; ++d) acc[d] = 0.f;
    const float ls = lse_s[j], dsum = d_s[j];
    for (int k = 0; k < n; ++k) {
      float kv[kD];
      load32(&Ks[k * kD], kv);
      float sv = 0.f;
#pragma unroll
      for (int d = 0; d < kD; ++d) sv = fmaf(qv[d], kv[d], sv);
      const float pr = __expf(p.scale * sv + bias_at(p, cu, n, j, k, h) - ls);
      const float ds = pr * (dot32(gv, &Vs[k * kD]) - dsum);
#pragma unroll
      for (int d = 0; d < kD; ++d) acc[d] = fmaf(ds, kv[d], acc[d]);
    }
    store32(p.dq + (base + (int64_t)j * step) * p.ld_dqkv + h * kD, acc, p.scale);
  }
  // dK_k = scale sum_j dS_jk Q_j,  dV_k = sum_j P_jk dO_j
  for (int k = threadIdx.x; k < n; k += 256) {
    float kv[kD], vv[kD], ak[kD], av[kD];
    load32(&Ks[k * kD], kv);
    load32(&Vs[k * kD], vv);
#pragma unroll
    for (int d = 0; d < kD; ++d) ak[d] = av[d] = 0.f;
    for (int j = 0; j < n; ++j) {
      float qv[kD], gv[kD];
      load32(&Qs[j * kD], qv);
      load32(&Gs[j * kD], gv);
      float sv = 0.f, dp = 0.f;
#pragma unroll
      for (int d = 0; d < kD; ++d) {
        sv = fmaf(qv[d], kv[d], sv);
        dp = fmaf(gv[d], vv[d], dp);
      }
      const float pr = __expf(p.scale * sv + bias_at(p, cu, n, j, k, h) - lse_s[j]);
      const float ds = pr * (dp - d_s[j]);
#pragma unroll
      for (int d = 0; d < kD; ++d) {
        ak[d] = fmaf(ds, qv[d], ak[d]);
        av[d] = fmaf(pr, gv[d], av[d]);
      }
    }
    const int64_t row = base + (int64_t)k * step;
    store32(p.dk + row * p.ld_dqkv + h * kD, ak, p.scale);
    store32(p.dv + row * p.ld_dqkv + h * kD, av, 1.f);
  }
}

// Bias gradient: workgroup (sample, 16-query block, head); thread t owns keys
// t and t + 256 (N <= 512).
__global__ void __launch_bounds__(256) attn_bwd_bias_kernel(AttnBwdArgs p) {
  __shared__ __attribute__((aligned(16))) bf16 qs[16 * kD], gs[16 * kD];
  __shared__ float ls[16], dsm[16];
  const int blk = blockIdx.x, h = blockIdx.y;
  int lo = 0, hi = p.batch - 1;                   // sample: largest i with cu_qblk[i] <= blk
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.cu_qblk[mid] <= blk) lo = mid; else hi = mid - 1;
  }
  const int i = lo;
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int j0 = (blk - p.cu_qblk[i]) * 16;
  const int nj = min(16, n - j0);
  const int64_t cu = p.cu_pairs[i];
  const int64_t step = p.axis == 0 ? 1 : n;
  float acc[2][16];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) acc[u][jj] = 0.f;
  for (int r = 0; r < n; ++r) {
    const int64_t base = p.axis == 0 ? cu + (int64_t)r * n : cu + r;
    __syncthreads();                              // the previous row's staging is consumed
    if (threadIdx.x < nj * 4) {
      const int jj = threadIdx.x >> 2, c = (threadIdx.x & 3) * 8;
      const int64_t row = base + (int64_t)(j0 + jj) * step;
      *reinterpret_cast<uint4*>(&qs[jj * kD + c]) = *reinterpret_cast<const uint4*>(p.q + row * p.ld_qkv + h * kD + c);
      *reinterpret_cast<uint4*>(&gs[jj * kD + c]) =
          *reinterpret_cast<const uint4*>(p.dout + row * p.ld_dout + h * kD + c);
    }
    if (threadIdx.x < nj) {
      const int64_t row = base + (int64_t)(j0 + threadIdx.x) * step;
      ls[threadIdx.x] = p.lse[row * p.H + h];
      dsm[threadIdx.x] = p.dsum[row * p.H + h];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = threadIdx.x + 256 * u;
      if (k >= n) continue;
      const int64_t krow = base + (int64_t)k * step;
      float kv[kD], vv[kD];
      load32(p.k + krow * p.ld_qkv + h * kD, kv);
      load32(p.v + krow * p.ld_qkv + h * kD, vv);
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) {
        if (jj >= nj) break;
        float qv[kD], gv[kD];
        load32(&qs[jj * kD], qv);
        load32(&gs[jj * kD], gv);
        float sv = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < kD; ++d) {
          sv = fmaf(qv[d], kv[d], sv);
          dp = fmaf(gv[d], vv[d], dp);
        }
        const float pr = __expf(p.scale * sv + bias_at(p, cu, n, j0 + jj, k, h) - ls[jj]);
        acc[u][jj] += pr * (dp - dsm[jj]);
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int k = threadIdx.x + 256 * u;
    if (k >= n) continue;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      if (jj >= nj) break;
      const int j = j0 + jj;
      const int64_t cell = cu + (p.axis == 0 ? (int64_t)j * n + k : (int64_t)k * n + j);
      p.dbias[cell * p.ld_dbias + (int64_t)h * p.ld_dbias_head] = acc[u][jj];
    }
  }
}

}  // namespace

size_t attention_backward_workspace_bytes(const nt_layout& L, int H) {
  return 2 * (size_t)L.sum_n2 * (size_t)H * sizeof(float);
}

hipError_t launch_attention_backward(const nt_layout& L, int axis, int H, const void* q, const void* k,
                                     const void* v, int64_t ld_qkv, const void* bias, int64_t ld_bias,
                                     int64_t ld_bias_head, const void* dout,
                                     int64_t ld_dout, float scale, void* dq, void* dk, void* dv, int64_t ld_dqkv,
                                     float* dbias, int64_t ld_dbias, int64_t ld_dbias_head, void* workspace,
                                     hipStream_t s) {
  if (L.attn_items() == 0) return hipSuccess;
  float* lse = static_cast<float*>(workspace);
  AttnBwdArgs a{axis, H, (const bf16*)q, (const bf16*)k, (const bf16*)v, ld_qkv, (const bf16*)bias, ld_bias,
                ld_bias_head, (const bf16*)dout, ld_dout, scale, (bf16*)dq, (bf16*)dk,
                (bf16*)dv, ld_dqkv, dbias, ld_dbias, ld_dbias_head, lse, lse + L.sum_n2 * H, L.d_attn_work,
                L.d_cu_seqlens, L.d_cu_pairs, L.d_cu_qblk, L.batch};
  const dim3 grid((unsigned)L.attn_items(), (unsigned)H);
  if (L.max_len <= 256) {
    const size_t smem = (size_t)4 * 256 * kD * sizeof(bf16) + 2 * 256 * sizeof(float);
    hipFuncSetAttribute((const void*)attn_bwd_rows_kernel<256>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attn_bwd_rows_kernel<256><<<grid, dim3(256), smem, s>>>(a);
  } else {
    const size_t smem = (size_t)4 * 512 * kD * sizeof(bf16) + 2 * 512 * sizeof(float);
    hipFuncSetAttribute((const void*)attn_bwd_rows_kernel<512>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attn_bwd_rows_kernel<512><<<grid, dim3(256), smem, s>>>(a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !dbias) return e;
  const int64_t qblocks = L.cu_qblk.back();
  if (qblocks == 0) return hipSuccess;
  attn_bwd_bias_kernel<<<dim3((unsigned)qblocks, (unsigned)H), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace nt
