// Large-K projection (the packed-token encoder path, Sec. 3.3: V' = V W^T + b
// on packed rows, with the pre-normalisation of the encoder layer): a tiled
// bf16 GEMM on the matrix cores for K a multiple of 32, computed transposed as
// D^T = W X^T so that a lane ends up with four consecutive output channels of
// one row.
//
// A workgroup of 8 waves owns a 256-row x 256-channel output tile; wave w
// computes 128 channels (w & 1) x 64 rows (w >> 1), i.e. 8 x 4 products per
// 32-wide k-step, with every weight fragment used 4 times and every row
// fragment 8 times.  Operand tiles (256 x 32 of W and of X per k-step) are
// copied global -> LDS with global_load_lds into a ring of four stages, three
// k-steps ahead, so one barrier per k-step covers both "the copy has landed"
// and "the slot is free again".  Each 64-byte row of a staged tile holds its
// four 16-byte pieces in the order piece ^ ((row >> 2) & 3): the 16 rows of a
// fragment read then fall on 16 different bank groups.  With a LayerNorm the
// rows are first normalised (two-pass statistics in fp32, result rounded to
// bf16 as the product consumes it) into the library's device workspace by a
// one-wave-per-row pass, and the product reads that copy: one extra write and
// read of the rows instead of every channel tile re-reducing them.
#include <algorithm>

#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kGT = 256;                  // tile rows = tile channels
constexpr int kGBK = 32;                  // k per stage
constexpr int kGStages = 4;
constexpr int kGThreads = 512;
constexpr int kGStageElems = 2 * kGT * kGBK;          // W tile then X tile (bf16)
constexpr int kGStageBytes = kGStageElems * 2;        // 32 KB
constexpr int kGEpiStride = 68;                       // fp32 epilogue stage row stride (64 channels + 4)
constexpr int kGEpiBytes = 8 * 64 * kGEpiStride * 4;  // 8 waves x 64 rows
constexpr int kGRingBytes = kGStages * kGStageBytes;

__device__ __forceinline__ int swz(int row, int piece) { return piece ^ ((row >> 2) & 3); }

__device__ __forceinline__ float gelu_exact(float v) { return 0.5f * v * (1.f + erff(v * 0.70710678118654752f)); }

typedef uint32_t g_u32x4 __attribute__((ext_vector_type(4)));
// The fragments of one k-step: eight weight fragments at aw + 1 KB i and four
// row fragments at ax + 1 KB j (16 staged rows of 64 bytes apart), in one
// block with its own LDS wait: as plain loads the compiler would make them
// wait for the copies still in flight into the other stages.
__device__ __forceinline__ void gemm_frags(uint32_t aw, uint32_t ax, bf16x8 (&w)[8], bf16x8 (&x)[4]) {
  g_u32x4 r[12];
  asm volatile(
      "ds_read_b128 %0, %12\n"
      "ds_read_b128 %1, %12 offset:1024\n"
      "ds_read_b128 %2, %12 offset:2048\n"
      "ds_read_b128 %3, %12 offset:3072\n"
      "ds_read_b128 %4, %12 offset:4096\n"
      "ds_read_b128 %5, %12 offset:5120\n"
      "ds_read_b128 %6, %12 offset:6144\n"
      "ds_read_b128 %7, %12 offset:7168\n"
      "ds_read_b128 %8, %13\n"
      "ds_read_b128 %9, %13 offset:1024\n"
      "ds_read_b128 %10, %13 offset:2048\n"
      "ds_read_b128 %11, %13 offset:3072\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7]),
        "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11])
      : "v"(aw), "v"(ax)
      : "memory");
#pragma unroll
  for (int i = 0; i < 8; ++i) w[i] = __builtin_bit_cast(bf16x8, r[i]);
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = __builtin_bit_cast(bf16x8, r[8 + j]);
}

__global__ void __launch_bounds__(kGThreads, 1) gemm_kernel(GemmArgs p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* ring = reinterpret_cast<bf16*>(smem);

  // ---- tile of this workgroup: XCD x = id % 8 takes row tiles x, x + 8, ...
  // and walks their channel tiles in order, so a row tile is read into one L2
  const int id = blockIdx.x;
  const int xcd = id % kXcds, kq = id / kXcds;
  const int rt = (kq / p.ntn) * kXcds + xcd, nt = kq % p.ntn;
  if (rt >= p.ntm) return;
  const int m0 = rt * kGT, n0 = nt * kGT;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  const int wc = wave & 1, wr = wave >> 1;
  const int nk = p.K / kGBK;

  // ---- stage copies: instruction c (0..31) of a stage copies 16 rows of the
  // W tile (c < 16) or of the X tile; lane l -> row 16 c' + l/4, piece l % 4
  // at its swizzled place.  Rows past the matrix repeat its last row (their
  // outputs are never stored).
  auto copy_stage = [&](int kt, int slot) {
    bf16* st = ring + slot * kGStageElems;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = wave + 8 * u;
      const bool isx = c >= 16;
      const int cr = (c & 15) * 16 + (lane >> 2);               // row within the tile
      const int piece = swz(cr, lane & 3);                      // global piece landing at lane & 3
      const bf16* src = isx ? p.x + (int64_t)min(m0 + cr, p.rows - 1) * p.ldx
                            : p.w + (int64_t)min(n0 + cr, p.N - 1) * p.K;
      src += kt * kGBK + piece * 8;
      bf16* dst = st + (isx ? kGT * kGBK : 0) + (c & 15) * 16 * kGBK;
      __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
    }
  };
  for (int s = 0; s < kGStages - 1; ++s)
    if (s < nk) copy_stage(s, s);

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // this lane's byte offset inside a 16-row fragment block: row l16, piece g
  // at its swizzled place (the swizzle depends only on l16, since fragment
  // blocks start at multiples of 16 rows)
  const uint32_t lofs = (uint32_t)(l16 * kGBK * 2 + (swz(l16, g) << 4));
  for (int kt = 0; kt < nk; ++kt) {
    // stage kt has landed for this wave (later stages may still be in flight)
    if (kt + 2 < nk) __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | 8);   // vmcnt(8)
    else if (kt + 1 < nk) __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | 4);  // vmcnt(4)
    else __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | 0);
    // stage kt complete everywhere and slot (kt - 1) % 4 free (every wave's
    // reads of it ended in an LDS wait).  The plain barrier: __syncthreads
    // would also wait for the copies still in flight, leaving no lookahead.
    __builtin_amdgcn_s_barrier();
    if (kt + kGStages - 1 < nk) copy_stage(kt + kGStages - 1, (kt + kGStages - 1) % kGStages);
    const uint32_t st = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)(ring + (kt % kGStages) * kGStageElems);
    // fragments: weight rows wc*128 + 16 i + l16, tile rows wr*64 + 16 j + l16,
    // k = 8 g .. 8 g + 7 of the stage
    bf16x8 aw[8], bx[4];
    gemm_frags(st + wc * 128 * kGBK * 2 + lofs, st + (kGT + wr * 64) * kGBK * 2 + lofs, aw, bx);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(aw[i], bx[j], acc[i][j]);
  }

  // ---- epilogue, two rounds of 64 channels per wave through LDS: acc[i][j][ii]
  // is channel n0 + wc*128 + 16 i + 4 g + ii of row m0 + wr*64 + 16 j + l16
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();                                // the ring is free for the epilogue stage
  float* es = reinterpret_cast<float*>(smem) + wave * 64 * kGEpiStride;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int ii = half * 4 + i;
        *reinterpret_cast<float4*>(&es[(j * 16 + l16) * kGEpiStride + i * 16 + 4 * g]) =
            make_float4(acc[ii][j][0], acc[ii][j][1], acc[ii][j][2], acc[ii][j][3]);
      }
    // the wave's own stage: its LDS writes complete before its reads
    const int cc = lane & 7, n = n0 + wc * 128 + half * 64 + cc * 8;
    float bv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) bv[e] = (p.bias && n + e < p.N) ? p.bias[n + e] : 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int rl = q * 8 + (lane >> 3), m = m0 + wr * 64 + rl;
      if (m >= p.rows || n >= p.N) continue;      // N % 8 == 0: a piece is all in or all out
      const float4 a0 = *reinterpret_cast<const float4*>(&es[rl * kGEpiStride + cc * 8]);
      const float4 a1 = *reinterpret_cast<const float4*>(&es[rl * kGEpiStride + cc * 8 + 4]);
      float v[8] = {a0.x + bv[0], a0.y + bv[1], a0.z + bv[2], a0.w + bv[3], a1.x + bv[4], a1.y + bv[5], a1.z + bv[6], a1.w + bv[7]};
      if (p.epi == NT_EPI_GELU) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = gelu_exact(v[e]);
      } else if (p.epi == NT_EPI_RESIDUAL) {
        const uint4 rr = *reinterpret_cast<const uint4*>(p.res + (int64_t)m * p.ld_res + n);
        const uint32_t w4[4] = {rr.x, rr.y, rr.z, rr.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[2 * e] += __uint_as_float(w4[e] << 16);
          v[2 * e + 1] += __uint_as_float(w4[e] & 0xffff0000u);
        }
      }
      bf16x8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (bf16)v[e];
      *reinterpret_cast<bf16x8*>(p.y + (int64_t)m * p.ldy + n) = o;
    }
  }
}

// LayerNorm of every row into xn [rows, K] (row stride K), one wave per row:
// lane c of the row holds 16-byte pieces c, c + 64, ... in registers.
template <int CPL>
__global__ void __launch_bounds__(256) layernorm_rows_kernel(const bf16* x, int64_t ldx, int rows, int K,
                                                             const float* gamma, const float* beta, float eps,
                                                             bf16* xn) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int nc = K / 8;
  const bf16* xr = x + (int64_t)row * ldx;
  float v[CPL][8];
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const int c = lane + 64 * u;
    const uint4 r = c < nc ? *reinterpret_cast<const uint4*>(xr + c * 8) : make_uint4(0u, 0u, 0u, 0u);
    const uint32_t w4[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[u][2 * e] = __uint_as_float(w4[e] << 16);
      v[u][2 * e + 1] = __uint_as_float(w4[e] & 0xffff0000u);
    }
  }
  float s1 = 0.f;
#pragma unroll
  for (int u = 0; u < CPL; ++u)
#pragma unroll
    for (int e = 0; e < 8; ++e) s1 += v[u][e];
  const float mean = group_sum<64>(s1) / (float)K;
  float s2 = 0.f;
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    if (lane + 64 * u >= nc) break;
#pragma unroll
    for (int e = 0; e < 8; ++e) { const float d = v[u][e] - mean; s2 += d * d; }
  }
  const float rstd = rsqrtf(group_sum<64>(s2) / (float)K + eps);
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const int c = lane + 64 * u;
    if (c >= nc) break;
    const float4 g0 = *reinterpret_cast<const float4*>(gamma + c * 8), g1 = *reinterpret_cast<const float4*>(gamma + c * 8 + 4);
    const float4 b0 = beta ? *reinterpret_cast<const float4*>(beta + c * 8) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 b1 = beta ? *reinterpret_cast<const float4*>(beta + c * 8 + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
    const float bb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (bf16)((v[u][e] - mean) * rstd * gg[e] + bb[e]);
    *reinterpret_cast<bf16x8*>(xn + (int64_t)row * K + c * 8) = o;
  }
}

}  // namespace

bool gemm_fits(int K) { return K % kGBK == 0 && K >= 4 * kGBK && K <= 64 * 8 * 8; }

hipError_t launch_gemm(GemmArgs p, hipStream_t s) {
  if (p.rows == 0) return hipSuccess;
  if (p.gamma) {
    if (!p.ln_ws) return hipErrorInvalidValue;
    hipError_t e;
    bf16* xn = p.ln_ws;
    const dim3 grid((unsigned)((p.rows + 3) / 4));
    const int cpl = (p.K / 8 + 63) / 64;          // 16-byte pieces per lane
    if (cpl <= 2) layernorm_rows_kernel<2><<<grid, dim3(256), 0, s>>>(p.x, p.ldx, p.rows, p.K, p.gamma, p.beta, p.eps, xn);
    else if (cpl <= 4) layernorm_rows_kernel<4><<<grid, dim3(256), 0, s>>>(p.x, p.ldx, p.rows, p.K, p.gamma, p.beta, p.eps, xn);
    else layernorm_rows_kernel<8><<<grid, dim3(256), 0, s>>>(p.x, p.ldx, p.rows, p.K, p.gamma, p.beta, p.eps, xn);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    p.x = xn;
    p.ldx = p.K;
    p.gamma = p.beta = nullptr;
  }
  p.ntm = (p.rows + kGT - 1) / kGT;
  p.ntn = (p.N + kGT - 1) / kGT;
  const size_t smem = (size_t)std::max(kGRingBytes, kGEpiBytes);
  (void)hipFuncSetAttribute((const void*)gemm_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  const int grid = (p.ntm + kXcds - 1) / kXcds * kXcds * p.ntn;
  gemm_kernel<<<dim3((unsigned)grid), dim3(kGThreads), smem, s>>>(p);
  return hipGetLastError();
}

}  // namespace nt
