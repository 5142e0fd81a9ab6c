// Backward of the packed LayerNorm + Linear (Sec. 3.3, V' = V W^T + b after a
// LayerNorm on each row's features) for a training step (Sec. 3.4).
//
// Pieces, each one launch over all rows:
//   * ln_rows_kernel / ln_rows_vec_kernel
//                             LN(x) in bf16 (what the forward product consumed)
//                             and each row's mean and 1/std;
//   * swiglu_backward_fused_kernel
//                             (SwiGLU, K = N in {64, 128}) the recomputed gate
//                             and up products, d h = dy W2 and the SwiGLU
//                             derivative in one pass: h and d[g | u];
//   * wgrad_kernel            weight gradients g^T LN(x) and dy^T h, summed
//                             over row ranges (copy ring into LDS, transpose
//                             reads), with the bias gradient as the column sums
//                             of g from the same fragments;
//   * dgrad_ln_kernel         (LayerNorm, K in {64, 128}) d(LN x) = g W and the
//                             LayerNorm backward, with per-wave partial sums of
//                             dgamma and dbeta;
//   * gemm_bf16_kernel        the general product C (+)= op(A) op(B) (64 x 64
//                             tiles, split contraction) for the other shapes;
//   * gelu / swiglu backward  elementwise, on recomputed pre-activations
//                             (shapes the fused kernels do not take);
//   * ln_backward_kernel      dx from d(LN x) on the general path, with
//                             per-group partial sums of dgamma and dbeta;
//   * column partials         bias gradients the weight-gradient kernel does not
//                             give; the reductions of all partial sums.
// Partial sums are written per workgroup, wave or row range and reduced in a
// fixed order, so every gradient is deterministic.
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

// ---------------------------------------------------------------- weight gradients
// C[M, N] = sum over rows r of a range: A[r, m] B[r, n] (the weight gradient
// g^T x of a linear layer, the contraction running over all packed rows).
// Both operands are read row-major, as stored: per 32-row step a workgroup
// copies a 32 x 128 slice of each into LDS (global -> LDS, 256 contiguous
// bytes per row), and the fragments, which need 8 rows of one column, come
// from transpose reads.  Four stages of copies are in flight.  Inside a row
// of the LDS slice the 16-byte chunks are XOR-permuted by 2 (r % 8), so the
// four rows a 16-lane group reads land on different banks.
// Workgroup b runs on XCD b % 8: the column tiles of one row range are
// consecutive workgroups of one XCD, so an operand slice that several tiles
// read is fetched into that L2 once.
// Requires M and N multiples of 128, lda and ldb multiples of 8 and 16-byte
// aligned bases; row range z covers [z kchunk, min(R, (z + 1) kchunk)) with
// kchunk a multiple of 32, and its partial goes to C + z split_stride.
// With colsum, the column sums of A over the range (a bias gradient) go to
// colsum[z M + m]: the waves of the first column tile that hold no B columns
// past 64 add one more product per fragment, with a ones operand.
constexpr int kWgT = 128, kWgStages = 4;

__device__ __forceinline__ uint32_t lds_addr_wg(const bf16* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)p;
}
// Fragments of columns from row-major LDS slices with rows kWgT apart: per
// fragment two transpose reads 16 rows apart.  Lane (l16, grp) of a read at
// address a (its piece: row 4 grp + l16 / 4, columns 4 (l16 % 4) .. + 3 of a
// 16-column group) receives column l16 of rows 4 grp .. 4 grp + 3, and of
// rows 16 + 4 grp .. + 3 from the second read.  Written as one block with its
// own LDS wait: the compiler would otherwise make these reads wait for the
// global -> LDS copies still in flight into other stages.
__device__ __forceinline__ void tr_read_frags(const uint32_t (&a)[8], bf16x8 (&f)[8]) {
  uint2 r[16];
  asm volatile(
      "ds_read_b64_tr_b16 %0, %16\n"
      "ds_read_b64_tr_b16 %1, %16 offset:4096\n"
      "ds_read_b64_tr_b16 %2, %17\n"
      "ds_read_b64_tr_b16 %3, %17 offset:4096\n"
      "ds_read_b64_tr_b16 %4, %18\n"
      "ds_read_b64_tr_b16 %5, %18 offset:4096\n"
      "ds_read_b64_tr_b16 %6, %19\n"
      "ds_read_b64_tr_b16 %7, %19 offset:4096\n"
      "ds_read_b64_tr_b16 %8, %20\n"
      "ds_read_b64_tr_b16 %9, %20 offset:4096\n"
      "ds_read_b64_tr_b16 %10, %21\n"
      "ds_read_b64_tr_b16 %11, %21 offset:4096\n"
      "ds_read_b64_tr_b16 %12, %22\n"
      "ds_read_b64_tr_b16 %13, %22 offset:4096\n"
      "ds_read_b64_tr_b16 %14, %23\n"
      "ds_read_b64_tr_b16 %15, %23 offset:4096\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7]),
        "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11]), "=&v"(r[12]), "=&v"(r[13]), "=&v"(r[14]), "=&v"(r[15])
      : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
      : "memory");
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t w[4] = {r[2 * i].x, r[2 * i].y, r[2 * i + 1].x, r[2 * i + 1].y};
    f[i] = __builtin_bit_cast(bf16x8, w);
  }
}
static_assert(16 * 128 * 2 == 4096, "second transpose read: 16 rows of a 128-column slice further");
constexpr int kWgStage = 2 * 32 * kWgT;              // bf16 per stage (A and B slices)

__global__ void __launch_bounds__(256, 2) wgrad_kernel(int M, int N, int R, const bf16* __restrict__ A, int64_t lda,
                                                       const bf16* __restrict__ B, int64_t ldb, float* __restrict__ C,
                                                       int kchunk, int splits, int64_t split_stride,
                                                       float* __restrict__ colsum) {
  extern __shared__ __attribute__((aligned(16))) bf16 wg_lds[];
  const int mt = M / kWgT, T = mt * (N / kWgT);
  const int xcd = blockIdx.x % kXcds, q = blockIdx.x / kXcds;
  const int z = (q / T) * kXcds + xcd, t = q % T;
  if (z >= splits) return;
  const int m0 = (t % mt) * kWgT, n0 = (t / mt) * kWgT;
  const int rbeg = z * kchunk, rend = min(R, rbeg + kchunk);
  if (rbeg >= rend) return;
  const int nsteps = (rend - rbeg + 31) / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l16 = lane & 15, grp = lane >> 4;

  // copies of step s into stage s % kWgStages: wave w copies rows 8 w .. 8 w + 7
  // of both slices (two 1 KB instructions each); lane i of an instruction
  // writes LDS chunk i % 16 of row i / 16, which holds column chunk
  // (i % 16) ^ 2 (row % 8) of the operand row (clamped into the matrix)
  const int crow = lane >> 4, cpos = lane & 15;
  auto copy_step = [&](int s) {
    bf16* st = wg_lds + (s % kWgStages) * kWgStage;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = wave * 8 + h * 4 + crow;
      const int gr = min(rbeg + s * 32 + r, R - 1);
      const int ch = cpos ^ (2 * (r & 7));
      const bf16* sa = A + (int64_t)gr * lda + m0 + ch * 8;
      const bf16* sb = B + (int64_t)gr * ldb + n0 + ch * 8;
      bf16* da = st + (wave * 8 + h * 4) * kWgT;
      __builtin_amdgcn_global_load_lds((const void*)sa, (__attribute__((address_space(3))) void*)da, 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)sb, (__attribute__((address_space(3))) void*)(da + 32 * kWgT), 16, 0,
                                       0);
    }
  };
  // transpose-read byte offset of this lane inside a slice for the 16
  // columns at c0 (a multiple of 16): row 4 grp + l16 / 4 (the second read is
  // 16 rows further), columns c0 + 4 (l16 % 4) .. + 3
  const int trow = 4 * grp + (l16 >> 2);
  auto tr_off = [&](int c0) -> uint32_t {
    const int col = c0 + 4 * (l16 & 3);
    return (uint32_t)((trow * kWgT + (((col >> 3) ^ (2 * (trow & 7))) << 3) + (col & 7)) * 2);
  };
  uint32_t offa[4], offb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    offa[i] = tr_off(wm * 64 + 16 * i);
    offb[i] = tr_off(wn * 64 + 16 * i) + 32 * kWgT * 2;
  }
  f32x4 acc[4][4], accs[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    accs[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const bool do_cs = colsum != nullptr && n0 == 0 && wn == 0;     // uniform

#pragma unroll
  for (int s = 0; s < kWgStages - 1; ++s)
    if (s < nsteps) copy_step(s);
  for (int s = 0; s < nsteps; ++s) {
    // step s has landed once at most the newer stages' copies (4 per stage
    // per wave) are outstanding
    const int newer = min(kWgStages - 2, nsteps - 1 - s);
    if (newer >= 2) __builtin_amdgcn_s_waitcnt(0x3F70 | 8);        // vmcnt(8)
    else if (newer == 1) __builtin_amdgcn_s_waitcnt(0x3F70 | 4);   // vmcnt(4)
    else __builtin_amdgcn_s_waitcnt(0x3F70);                       // vmcnt(0)
    // every wave's copies of step s have landed and its reads of step s - 1
    // are done (they end in an LDS wait): the stage of step s - 1 is free
    __builtin_amdgcn_s_barrier();
    if (s + kWgStages - 1 < nsteps) copy_step(s + kWgStages - 1);
    const uint32_t base = lds_addr_wg(wg_lds + (s % kWgStages) * kWgStage);
    uint32_t ad[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ad[i] = base + offa[i];
      ad[4 + i] = base + offb[i];
    }
    bf16x8 fr[8];
    tr_read_frags(ad, fr);
    bf16x8 fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa[i] = fr[i];
      fb[i] = fr[4 + i];
    }
    // rows past the range (last step only) contribute zero
    if (rbeg + s * 32 + 32 > rend) {
      const int lim = rend - rbeg - s * 32;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int rr = (e < 4 ? 0 : 16) + 4 * grp + (e & 3);
        if (rr >= lim)
#pragma unroll
          for (int i = 0; i < 4; ++i) fa[i][e] = (bf16)0.f;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(fa[i], fb[j], acc[i][j]);
    if (do_cs) {
      const bf16x8 ones = {(bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f, (bf16)1.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) accs[i] = mfma16(fa[i], ones, accs[i]);
    }
  }
  // accs[i][e] (every column l16 alike) = sum of A column m0 + 64 wm + 16 i + 4 grp + e
  if (do_cs && l16 == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) colsum[(int64_t)z * M + m0 + 64 * wm + 16 * i + 4 * grp + e] = accs[i][e];
  }
  // acc[i][j][e] = C[m0 + 64 wm + 16 i + 4 grp + e][n0 + 64 wn + 16 j + l16]
  float* Cz = C + (int64_t)z * split_stride;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Cz[(int64_t)(m0 + 64 * wm + 16 * i + 4 * grp + e) * N + n0 + 64 * wn + 16 * j + l16] = acc[i][j][e];
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
    if (!ok || !dx) continue;                   // (dx == NULL: only dgamma / dbeta wanted)
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

// d(LN x) = g W and the LayerNorm backward in one pass (K = 64 or 128
// channels): g [R, Nw] bf16 (row stride ld_g), W given transposed, wt [K, Nw].
// A workgroup of eight waves owns 256 rows, a wave 32 of them, and computes
// d(LN x)^T = W^T g^T on matrix cores.  Per 64-wide step of the contraction
// it copies the g slice of its rows and the W^T slice into LDS (global ->
// LDS; each copy instruction covers whole 128-byte lines of 8 rows, the
// address unit being the limit with shorter pieces), three stages deep.  In
// a slice row r keeps its 16-byte chunk c at position c ^ ((r / 2) % 8), so
// the 16 rows a fragment read spans land on different banks.  A lane ends
// with K / 4 channels 16 j + 4 grp + e of row 16 i + l16 of each of its
// wave's two row tiles, so a row's sums are in-lane sums plus two lane-row
// swaps.  Then, as ln_backward_vec_kernel,
//   gv = d(LN x) gamma,  xhat = (x - mean) rstd,
//   dx = rstd (gv - mean(gv) - xhat mean(gv xhat))  (+ res, + dx if accumulating),
// and the wave's sums of d(LN x) xhat and d(LN x) go to part_g / part_b row
// (32-row group) blockIdx.x * 8 + wave.  Requires Nw a multiple of 64,
// ld_g, ldx and the bases 16-byte aligned.
constexpr int kDgStages = 3, kDgRT = 2, kDgWaves = 8;   // stages; row tiles per wave; waves
constexpr int kDgRows = kDgWaves * 16 * kDgRT;           // rows per workgroup
template <int K> constexpr int dg_stage_elems() { return kDgRows * 64 + K * 64; }   // g slice + W^T slice

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Sum over the 16 lanes of a DPP row (lanes 16 r .. 16 r + 15): four
// rotate-and-add steps within the row; lane 16 r holds the whole sum.
__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));   // row_ror:8
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false));   // row_ror:4
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x122, 0xf, 0xf, false));   // row_ror:2
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x121, 0xf, 0xf, false));   // row_ror:1
  return v;
}
// the fragments of one 32-wide half step: KT W^T fragments at aw + 2 KB j,
// two g fragments at ag, ag + 2 KB (16 slice rows of 128 bytes apart); one
// block with its own LDS wait (the compiler would make plain reads wait for
// the copies in flight into other stages)
template <int KT>
__device__ __forceinline__ void dg_read(uint32_t aw, uint32_t ag, bf16x8 (&wf)[KT], bf16x8 (&gf)[kDgRT]);
template <>
__device__ __forceinline__ void dg_read<8>(uint32_t aw, uint32_t ag, bf16x8 (&wf)[8], bf16x8 (&gf)[kDgRT]) {
  u32x4 r[10];
  asm volatile(
      "ds_read_b128 %0, %10\n"
      "ds_read_b128 %1, %10 offset:2048\n"
      "ds_read_b128 %2, %10 offset:4096\n"
      "ds_read_b128 %3, %10 offset:6144\n"
      "ds_read_b128 %4, %10 offset:8192\n"
      "ds_read_b128 %5, %10 offset:10240\n"
      "ds_read_b128 %6, %10 offset:12288\n"
      "ds_read_b128 %7, %10 offset:14336\n"
      "ds_read_b128 %8, %11\n"
      "ds_read_b128 %9, %11 offset:2048\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7]),
        "=&v"(r[8]), "=&v"(r[9])
      : "v"(aw), "v"(ag)
      : "memory");
#pragma unroll
  for (int j = 0; j < 8; ++j) wf[j] = __builtin_bit_cast(bf16x8, r[j]);
#pragma unroll
  for (int i = 0; i < kDgRT; ++i) gf[i] = __builtin_bit_cast(bf16x8, r[8 + i]);
}
template <>
__device__ __forceinline__ void dg_read<4>(uint32_t aw, uint32_t ag, bf16x8 (&wf)[4], bf16x8 (&gf)[kDgRT]) {
  u32x4 r[6];
  asm volatile(
      "ds_read_b128 %0, %6\n"
      "ds_read_b128 %1, %6 offset:2048\n"
      "ds_read_b128 %2, %6 offset:4096\n"
      "ds_read_b128 %3, %6 offset:6144\n"
      "ds_read_b128 %4, %7\n"
      "ds_read_b128 %5, %7 offset:2048\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5])
      : "v"(aw), "v"(ag)
      : "memory");
#pragma unroll
  for (int j = 0; j < 4; ++j) wf[j] = __builtin_bit_cast(bf16x8, r[j]);
#pragma unroll
  for (int i = 0; i < kDgRT; ++i) gf[i] = __builtin_bit_cast(bf16x8, r[4 + i]);
}
static_assert(kDgRT == 2, "dg_read reads two g fragments");

template <int K, typename TO>
__global__ void __launch_bounds__(64 * kDgWaves, 1) dgrad_ln_kernel(
    const bf16* __restrict__ g, int64_t ld_g, int Nw, const bf16* __restrict__ wt, const bf16* __restrict__ x,
    int64_t ldx, int R, const float* __restrict__ gamma, const float* __restrict__ mean,
    const float* __restrict__ rstd, const TO* __restrict__ res, int64_t ld_res, TO* __restrict__ dx, int64_t ld_dx,
    int accumulate, float* __restrict__ part_g, float* __restrict__ part_b) {
  constexpr int KT = K / 16;
  constexpr int SE = dg_stage_elems<K>();
  constexpr int GI = kDgRows / 8 / kDgWaves;    // g copy instructions per wave per step (8 rows each)
  constexpr int WI = K / 8 / kDgWaves;          // W^T copy instructions per wave per step
  constexpr int NOPS = GI + WI;
  static_assert(GI >= 1 && WI >= 1 && K / 8 == WI * kDgWaves, "copies cover the slices");
  extern __shared__ __attribute__((aligned(16))) bf16 dg_lds[];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, grp = lane >> 4;
  const int rb = blockIdx.x * kDgRows;
  const int wg = blockIdx.x * kDgWaves + wave;
  const int r0 = wg * 16 * kDgRT;
  const int nks = Nw / 64;

  // copies of step s: instruction u covers slice rows 8 u .. 8 u + 7; lane i
  // fetches row 8 u + i / 8, LDS position i % 8, which holds the row's chunk
  // (i % 8) ^ ((row / 2) % 8).  Rows past R are clamped (they only feed
  // their own discarded outputs).
  const int crow = lane >> 3, cpos = lane & 7;
  auto copy_step = [&](int s) {
    bf16* st = dg_lds + (s % kDgStages) * SE;
#pragma unroll
    for (int t = 0; t < GI; ++t) {
      const int u = GI * wave + t, r = 8 * u + crow;
      const int c = cpos ^ ((r >> 1) & 7);
      const bf16* src = g + (int64_t)min(rb + r, R - 1) * ld_g + 64 * s + 8 * c;
      __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(st + u * 512), 16,
                                       0, 0);
    }
#pragma unroll
    for (int t = 0; t < WI; ++t) {
      const int v = wave + kDgWaves * t, n = 8 * v + crow;
      const int c = cpos ^ ((n >> 1) & 7);
      const bf16* src = wt + (int64_t)n * Nw + 64 * s + 8 * c;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(st + kDgRows * 64 + v * 512), 16, 0, 0);
    }
  };
  // this lane's fragment offset in a slice for half step h: row (or channel)
  // l16 of a 16-row tile, chunk 4 h + grp, permuted as stored
  auto frag_off = [&](int h) -> uint32_t {
    return (uint32_t)(l16 * 128 + (((4 * h + grp) ^ ((l16 >> 1) & 7)) << 4));
  };
  f32x4 acc[KT][kDgRT];
#pragma unroll
  for (int j = 0; j < KT; ++j)
#pragma unroll
    for (int i = 0; i < kDgRT; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < kDgStages - 1; ++s)
    if (s < nks) copy_step(s);
  for (int ks = 0; ks < nks; ++ks) {
    // step ks has landed once at most the next step's copies are outstanding
    static_assert(kDgStages == 3 && NOPS < 16, "the wait below covers one later step");
    if (ks + 1 < nks) __builtin_amdgcn_s_waitcnt(0x3F70 | NOPS);
    else __builtin_amdgcn_s_waitcnt(0x3F70);
    __builtin_amdgcn_s_barrier();               // all copies of step ks; step ks - 1 read everywhere
    if (ks + kDgStages - 1 < nks) copy_step(ks + kDgStages - 1);
    const uint32_t base =
        (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)(dg_lds + (ks % kDgStages) * SE);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t off = frag_off(h);
      bf16x8 wf[KT], gf[kDgRT];
      dg_read<KT>(base + kDgRows * 128 + off, base + wave * 16 * kDgRT * 128 + off, wf, gf);
#pragma unroll
      for (int j = 0; j < KT; ++j)
#pragma unroll
        for (int i = 0; i < kDgRT; ++i) acc[j][i] = mfma16(wf[j], gf[i], acc[j][i]);
    }
  }
  // The ring is free once every wave is past its last read: it now takes
  // the workgroup's x rows and gamma, copied in one burst (global -> LDS).
  // x row r (of the workgroup) holds its 16-byte chunk c at slot
  // (r % RW) CR + (c ^ f(r)), CR = K / 8 chunks per row, RW = 256 / (2 K)
  // rows per 256 bytes, f(r) = (r / RW) % CR: the 16 consecutive rows a
  // read spans land on 16 different 16-byte slots of the banks.
  constexpr int CR = K / 8, RW = 256 / (2 * K);
  __builtin_amdgcn_s_waitcnt(0xC07F);           // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  {
    constexpr int XI = kDgRows * CR / 64 / kDgWaves;   // 1 KB copies of x per wave
#pragma unroll
    for (int t = 0; t < XI; ++t) {
      const int u = wave * XI + t;              // copy u: LDS bytes [1024 u, 1024 u + 1024)
      const int slot = u * 64 + lane;           // 16-byte slot of the x tile
      const int r = (slot / (RW * CR)) * RW + (slot % (RW * CR)) / CR;   // row owning the slot
      const int c = (slot % CR) ^ ((r / RW) % CR);
      const bf16* src = x + (int64_t)min(rb + r, R - 1) * ldx + 8 * c;
      __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(dg_lds + u * 512),
                                       16, 0, 0);
    }
    if (wave == 0) {                            // gamma after the x tile (lanes past K / 4 repeat its last piece)
      const float* src = gamma + 4 * min(lane, K / 4 - 1);
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(dg_lds + kDgRows * K), 16, 0, 0);
    }
  }
  static_assert(kDgRows * K * 2 + 1024 <= kDgStages * dg_stage_elems<K>() * 2, "x tile and gamma fit in the ring");
  __builtin_amdgcn_s_waitcnt(0x3F70);           // vmcnt(0)
  __builtin_amdgcn_s_barrier();
  if (r0 >= R) return;
  const bf16* xs = dg_lds;
  const float* gs = reinterpret_cast<const float*>(dg_lds + kDgRows * K);
  // acc[j][i][e] = d(LN x)[r0 + 16 i + l16][16 j + 4 grp + e].
  // First pass, channel tiles outer: the row sums of gv and gv xhat, and per
  // channel tile the wave's sums of d(LN x) xhat and d(LN x) over its rows
  // (lane sums over the row tiles, then over the 16 lanes of a row group),
  // written at once.  Second pass: dx.  x and gamma are read from LDS in
  // both passes rather than held in registers next to the accumulators.
  // Rows past R (their g rows were clamped, so their values are finite)
  // enter the channel sums with weight okf = 0.
  float mu[kDgRT], rs[kDgRT], s1[kDgRT], s2[kDgRT], okf[kDgRT];
#pragma unroll
  for (int i = 0; i < kDgRT; ++i) {
    const int row = r0 + 16 * i + l16;
    okf[i] = row < R ? 1.f : 0.f;
    const int rr = min(row, R - 1);
    mu[i] = mean[rr];
    rs[i] = rstd[rr];
    s1[i] = s2[i] = 0.f;
  }
  // this lane's x piece (channels 16 j + 4 grp ..) of row tile i, from LDS
  auto xhat4 = [&](int i, int j, float (&xh)[4]) {
    const int r = wave * 16 * kDgRT + 16 * i + l16;        // row of the workgroup
    const int c = 2 * j + (grp >> 1);
    const int slot = (r / RW) * RW * CR + (r % RW) * CR + (c ^ ((r / RW) % CR));
    const uint2 q = *reinterpret_cast<const uint2*>(xs + slot * 8 + (grp & 1) * 4);
    xh[0] = (__uint_as_float(q.x << 16) - mu[i]) * rs[i];
    xh[1] = (__uint_as_float(q.x & 0xffff0000u) - mu[i]) * rs[i];
    xh[2] = (__uint_as_float(q.y << 16) - mu[i]) * rs[i];
    xh[3] = (__uint_as_float(q.y & 0xffff0000u) - mu[i]) * rs[i];
  };
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    const float4 gm = *reinterpret_cast<const float4*>(gs + 16 * j + 4 * grp);
    const float gg[4] = {gm.x, gm.y, gm.z, gm.w};
    float pg[4] = {0.f, 0.f, 0.f, 0.f}, pb[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kDgRT; ++i) {
      float xh[4];
      xhat4(i, j, xh);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float d = acc[j][i][e];
        const float gv = d * gg[e];
        s1[i] += gv;
        s2[i] += gv * xh[e];
        const float dm = d * okf[i];
        pg[e] += dm * xh[e];
        pb[e] += dm;
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      pg[e] = row16_sum(pg[e]);
      pb[e] = row16_sum(pb[e]);
    }
    if (l16 == 0) {
      const int64_t c = (int64_t)wg * K + 16 * j + 4 * grp;
      *reinterpret_cast<float4*>(part_g + c) = make_float4(pg[0], pg[1], pg[2], pg[3]);
      *reinterpret_cast<float4*>(part_b + c) = make_float4(pb[0], pb[1], pb[2], pb[3]);
    }
    // keep each channel tile's loads inside its iteration: hoisted, they
    // would sit in registers next to the accumulators
    __builtin_amdgcn_sched_barrier(0);
  }
  if (!dx) return;                              // only dgamma / dbeta wanted
#pragma unroll
  for (int i = 0; i < kDgRT; ++i) {
    s1[i] = sum_over_kgroups(s1[i]) / (float)K;
    s2[i] = sum_over_kgroups(s2[i]) / (float)K;
  }
  // an offset the compiler cannot see through: the second pass reads x and
  // gamma from LDS again instead of keeping the first pass's values live
  int z0 = 0;
  asm volatile("" : "+v"(z0));
#pragma unroll
  for (int i = 0; i < kDgRT; ++i) {
    if (okf[i] == 0.f) continue;
    const int64_t row = r0 + 16 * i + l16;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const float4 gm = *reinterpret_cast<const float4*>(gs + z0 + 16 * j + 4 * grp);
      const float gg[4] = {gm.x, gm.y, gm.z, gm.w};
      float xh[4];
      xhat4(i, j + z0, xh);
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = rs[i] * (acc[j][i][e] * gg[e] - s1[i] - xh[e] * s2[i]);
      const int64_t c = 16 * j + 4 * grp;
      if (res) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] += to_f32(res[row * ld_res + c + e]);
      }
      TO* o = dx + row * ld_dx + c;
      if (accumulate) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] += to_f32(o[e]);
      }
      if constexpr (sizeof(TO) == 4) {
        *reinterpret_cast<float4*>(o) = make_float4(v[0], v[1], v[2], v[3]);
      } else {
        bf16x4 ov;
#pragma unroll
        for (int e = 0; e < 4; ++e) ov[e] = (bf16)v[e];
        *reinterpret_cast<bf16x4*>(o) = ov;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
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
    if (!dx) continue;                          // only dgamma / dbeta wanted
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
// path) and h, d g, d u are stored as 16-byte pieces after a lane-row swap.  The workgroups of one
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
    uint32_t ow[3][4][2];                       // [h, d g, d u][unit tile t] as packed bf16 pairs
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
      const uint2 a = __builtin_bit_cast(uint2, ho), b = __builtin_bit_cast(uint2, go),
                  c = __builtin_bit_cast(uint2, uo);
      ow[0][t][0] = a.x; ow[0][t][1] = a.y;
      ow[1][t][0] = b.x; ow[1][t][1] = b.y;
      ow[2][t][0] = c.x; ow[2][t][1] = c.y;
    }
    // lane (l16, g) holds units 16 t + 4 g .. + 3 of row l16.  Lane-row
    // groups g, g ^ 1 trade the pieces of tiles t, t + 1 (t even) so that an
    // even g holds units 16 t + 4 g .. + 7 and an odd g units
    // 16 (t + 1) + 4 (g - 1) .. + 7: one 16-byte store per lane and tile pair,
    // the four lane groups of a row writing 64 contiguous bytes (the address
    // unit is charged per line an instruction touches).
#pragma unroll
    for (int o = 0; o < 3; ++o)
#pragma unroll
      for (int t = 0; t < 4; t += 2)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const auto sw = __builtin_amdgcn_permlane16_swap(ow[o][t][e], ow[o][t + 1][e], false, false);
          ow[o][t][e] = sw[0];
          ow[o][t + 1][e] = sw[1];
        }
    // a lane past R computed row R - 1 (its input row was clamped) and
    // stores those same values there: no divergent branch, so the waits
    // for the next tile's rows stay exact
    const int64_t ro = min(row, R - 1);
#pragma unroll
    for (int t = 0; t < 4; t += 2) {
      const int f = u0 + 16 * t + ((g & 1) ? 16 + 4 * (g - 1) : 4 * g);
      *reinterpret_cast<uint4*>(h + ro * F + f) = make_uint4(ow[0][t][0], ow[0][t][1], ow[0][t + 1][0], ow[0][t + 1][1]);
      *reinterpret_cast<uint4*>(dp + ro * 2 * F + f) =
          make_uint4(ow[1][t][0], ow[1][t][1], ow[1][t + 1][0], ow[1][t + 1][1]);
      *reinterpret_cast<uint4*>(dp + ro * 2 * F + F + f) =
          make_uint4(ow[2][t][0], ow[2][t][1], ow[2][t + 1][0], ow[2][t + 1][1]);
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

// fp32 rows [R, K] (contiguous) -> bf16 rows ld apart, one thread per element.
__global__ void __launch_bounds__(256) to_bf16_rows_kernel(const float* __restrict__ x, int R, int K,
                                                           bf16* __restrict__ y, int64_t ld) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)R * K) return;
  const int64_t r = e / K, c = e % K;
  y[r * ld + c] = (bf16)x[e];
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

// Row ranges of a weight gradient C[M, N] = sum_r A[r, m] B[r, n] on
// wgrad_kernel: about two workgroups per CU in all, ranges a multiple of 32
// rows and at least 128.  splits == 0: the shape does not fit the kernel.
struct WgPlan {
  int splits = 0, kchunk = 0;
  unsigned grid = 0;
};
WgPlan wgrad_plan(int M, int N, int R, int64_t lda, int64_t ldb) {
  WgPlan w;
  if (M % kWgT || N % kWgT || lda % 8 || ldb % 8 || R <= 0 || M <= 0 || N <= 0) return w;
  const int T = (M / kWgT) * (N / kWgT);
  const int want = std::max(1, 512 / T);
  w.kchunk = std::max(128, ((R + want - 1) / want + 31) / 32 * 32);
  w.splits = (R + w.kchunk - 1) / w.kchunk;
  w.grid = (unsigned)((w.splits + kXcds - 1) / kXcds * kXcds * T);
  return w;
}
void launch_wgrad(const WgPlan& w, int M, int N, int R, const bf16* A, int64_t lda, const bf16* B, int64_t ldb,
                  float* part, float* colsum, hipStream_t s) {
  wgrad_kernel<<<dim3(w.grid), dim3(256), kWgStages * kWgStage * sizeof(bf16), s>>>(
      M, N, R, A, lda, B, ldb, part, w.kchunk, w.splits, (int64_t)M * N, colsum);
}

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
  // LayerNorm on bf16 rows of 64 or 128: d(LN x) = g W and the LayerNorm
  // backward in one kernel (no fp32 d(LN x) in memory)
  const int64_t ld_g_dx = (gelu || swiglu) ? Nw : a.ld_dy;
  const bool dgrad_fused = ln && vec_ln && (K == 64 || K == 128) && Nw % 64 == 0 && ld_g_dx % 8 == 0 &&
                           (a.dx || a.dgamma || a.dbeta);
  bf16* wt1 = dgrad_fused ? c.take<bf16>((size_t)K * Nw) : nullptr;         // W^T [K, Nw]
  float* dxn = (direct_dx || dgrad_fused) ? nullptr : c.take<float>((size_t)R * K);
  // rows per partial group of the LayerNorm and column sums: one wave's rows
  // in the fused kernel, 64 on the 16-byte LayerNorm passes, else 256
  const int rpg = dgrad_fused ? 16 * kDgRT : (vec_ln ? 64 : kRowsPerGroup);
  const int groups = (R + rpg - 1) / rpg;
  float* part_g = c.take<float>((size_t)groups * K);
  float* part_b = c.take<float>((size_t)groups * K);

  // weight gradients: dW = g^T LN(x) [Nw, K] and (SwiGLU) dW2 = dy^T h [N, F],
  // on wgrad_kernel where the shape allows, else on the general product
  const int64_t ld_g_plan = (gelu || swiglu) ? Nw : a.ld_dy;
  const int64_t ld_x_plan = (ln || xf) ? K : a.ldx;
  const WgPlan wp = wgrad_plan(Nw, K, R, ld_g_plan, ld_x_plan);
  const int64_t tiles_w = (int64_t)((Nw + kBM - 1) / kBM) * ((K + kBN - 1) / kBN);
  const int sw = wp.splits ? wp.splits : splits_for(tiles_w, R);
  float* part_w = c.take<float>((size_t)sw * Nw * K);
  const WgPlan wp2 = swiglu ? wgrad_plan(a.c_out, F, R, a.ld_dy, F) : WgPlan{};
  const int64_t tiles_w2 = (int64_t)((a.c_out + kBM - 1) / kBM) * ((F + kBN - 1) / kBN);
  const int sw2 = swiglu ? (wp2.splits ? wp2.splits : splits_for(tiles_w2, R)) : 0;
  float* part_w2 = swiglu ? c.take<float>((size_t)sw2 * a.c_out * F) : nullptr;
  // bias gradients as column sums inside the weight-gradient kernel (per row range)
  const bool cs_fused = wp.splits && a.dw && a.db;
  const bool cs2_fused = wp2.splits && a.dw2 && a.db2;
  float* part_cs = cs_fused ? c.take<float>((size_t)wp.splits * Nw) : nullptr;
  float* part_cs2 = cs2_fused ? c.take<float>((size_t)wp2.splits * a.c_out) : nullptr;
  // column sums of the bias gradients that the weight-gradient kernel does not give
  const bool need_col = (a.db && !cs_fused) || (swiglu && a.db2 && !cs2_fused);
  float* part_col = need_col ? c.take<float>((size_t)groups * std::max(Nw, a.c_out)) : nullptr;
  // second level of the reductions with more than 64 partials
  auto slices = [](int64_t splits) -> size_t { return splits > 64 ? (size_t)((splits + 63) / 64) : 0; };
  const size_t n2 = std::max({slices(groups) * (size_t)std::max(std::max(Nw, a.c_out), K),
                              slices(sw) * (size_t)Nw * K, slices(sw2) * (size_t)a.c_out * F});
  float* part2 = c.take<float>(std::max<size_t>(n2, 1));
  // third level and beyond (ping-pong with part2): at most 1/64 of part2
  auto slices2 = [&](int64_t splits) -> size_t { return slices((int64_t)slices(splits)); };
  const size_t n3 = std::max({slices2(groups) * (size_t)std::max(std::max(Nw, a.c_out), K),
                              slices2(sw) * (size_t)Nw * K, slices2(sw2) * (size_t)a.c_out * F});
  float* part3 = c.take<float>(std::max<size_t>(n3, 1));
  *bytes = c.used;
  if (!launch) return hipSuccess;

  const bf16* W = (const bf16*)a.w;
  const bf16* dy = (const bf16*)a.dy;
  const int acc_w = a.overwrite_weights ? 0 : 1;
  const dim3 b256(256);
  // out (+)= sum over `splits` partials (stride apart) of n values, in a fixed
  // order: while more than 64 remain, each 64 of them are summed into one
  // (reduce_level1_kernel, alternately into part2 and part3), then the rest
  auto reduce_parts = [&](const float* part, int splits, int64_t stride, int64_t n, float* out) {
    float* bufs[2] = {part2, part3};
    int b = 0;
    while (splits > 64) {
      const int sl = (splits + 63) / 64;
      reduce_level1_kernel<<<dim3((unsigned)((n + 63) / 64), (unsigned)sl), b256, 0, s>>>(part, splits, stride, n,
                                                                                         bufs[b]);
      part = bufs[b];
      stride = n;
      splits = sl;
      b ^= 1;
    }
    reduce_partials_kernel<<<blocks_for(n), b256, 0, s>>>(part, splits, stride, n, out, acc_w);
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
        if (wp2.splits)
          launch_wgrad(wp2, a.c_out, F, R, dy, a.ld_dy, h, F, part_w2, part_cs2, s);
        else
          gemm_bf16_kernel<true, false><<<dim3((a.c_out + kBM - 1) / kBM, (F + kBN - 1) / kBN, sw2), b256, 0, s>>>(
              a.c_out, F, R, dy, a.ld_dy, h, F, part_w2, F, 1.f, 0, kc, (int64_t)a.c_out * F);
        reduce_parts(part_w2, sw2, (int64_t)a.c_out * F, (int64_t)a.c_out * F, a.dw2);
      }
      if (cs2_fused) {
        reduce_parts(part_cs2, wp2.splits, a.c_out, a.c_out, a.db2);
      } else if (a.db2) {
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
    if (ld_g != ld_g_plan || ld_xin != ld_x_plan) return hipErrorInvalidValue;   // the plan saw these strides
    if (wp.splits)
      launch_wgrad(wp, Nw, K, R, g, ld_g, xin, ld_xin, part_w, part_cs, s);
    else
      gemm_bf16_kernel<true, false><<<dim3((Nw + kBM - 1) / kBM, (K + kBN - 1) / kBN, sw), b256, 0, s>>>(
          Nw, K, R, g, ld_g, xin, ld_xin, part_w, K, 1.f, 0, kc, (int64_t)Nw * K);
    reduce_parts(part_w, sw, (int64_t)Nw * K, (int64_t)Nw * K, a.dw);
  }
  if (cs_fused) {
    reduce_parts(part_cs, wp.splits, Nw, Nw, a.db);
  } else if (a.db) {
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
  if (dgrad_fused) {
    if (ld_g != ld_g_dx) return hipErrorInvalidValue;                       // the plan saw this stride
    if (res && dxf) return hipErrorInvalidValue;                            // the SwiGLU residual is bf16
    transpose_bf16_kernel<<<blocks_for((int64_t)Nw * K), b256, 0, s>>>(W, Nw, K, wt1);
    const dim3 grid((unsigned)((R + kDgRows - 1) / kDgRows)), bdg(64 * kDgWaves);
#define NT_DGLN(KK, TO)                                                                                        \
  do {                                                                                                         \
    (void)hipFuncSetAttribute((const void*)dgrad_ln_kernel<KK, TO>, hipFuncAttributeMaxDynamicSharedMemorySize,   \
                              (int)(kDgStages * dg_stage_elems<KK>() * sizeof(bf16)));                           \
    dgrad_ln_kernel<KK, TO><<<grid, bdg, kDgStages * dg_stage_elems<KK>() * sizeof(bf16), s>>>(g, ld_g, Nw, wt1, (const bf16*)a.x, a.ldx, R, a.ln_gamma, mean, \
                                                  rstd, (const TO*)res, a.ld_dy, (TO*)a.dx, a.ld_dx,            \
                                                  a.accumulate_dx, part_g, part_b);                                     \
  } while (0)
    if (K == 64) { if (dxf) NT_DGLN(64, float); else NT_DGLN(64, bf16); }
    else { if (dxf) NT_DGLN(128, float); else NT_DGLN(128, bf16); }
#undef NT_DGLN
    if (a.dgamma) reduce_parts(part_g, groups, K, K, a.dgamma);
    if (a.dbeta) reduce_parts(part_b, groups, K, K, a.dbeta);
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
    // no LayerNorm, bf16 dx = d(LN x), rows ld_dx apart
    if (a.accumulate_dx || res) return hipErrorInvalidValue;
    to_bf16_rows_kernel<<<blocks_for((int64_t)R * K), b256, 0, s>>>(dxn, R, K, (bf16*)a.dx, a.ld_dx);
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
