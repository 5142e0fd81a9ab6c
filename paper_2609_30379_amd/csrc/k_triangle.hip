// Triangle multiplicative update as one ragged grouped GEMM over the batch:
// for every sample i and channel c, T_c = A_c B_c^T with A_c, B_c the
// sample's N_i x N_i channel planes, then z[cell(x,y), c] += T_c[x, y].
//
// Operands arrive pair-padded channel-major (rows start 16-byte aligned), so
// every matrix-core fragment is one 16-byte load.  A workgroup owns a 32x32
// cell tile of one sample and a block of 16 channels (4 per wave).  Workgroup
// ids interleave the channel blocks of each tile, so with 8 blocks (C = 128)
// XCD x (ids = x mod 8) always works on channel block x: it walks the tile
// list sample by sample and keeps the current sample's 16 channel planes
// (2 x 16 x N^2 x 2 bytes, about 3 MB at N = 216) in its own L2, where the
// operand re-reads of neighbouring tiles hit.  The next k-step's fragments
// are loaded while the current one is on the matrix cores; with 64
// accumulator registers per lane two waves fit on each SIMD.
#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kTriCB = 16;    // channels per workgroup
constexpr int kTriCW = 4;     // channels per wave

struct TriArgs {
  int C, nblk;
  const bf16* a;
  const bf16* b;
  int64_t ld_ab;
  bf16* z;
  int64_t ld_z;
  const int32_t* work;   // quads (sample, x-tile, y-tile, 0)
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  const int32_t* cu_pad;
};

// Fragment of rows row..row+15 (lane row = l16) and k..k+7 of one plane;
// rows past the sample and k past N read as zero.
__device__ __forceinline__ bf16x8 load_frag(const bf16* plane, int row, int k, int n, int n8, bool tail) {
  if (row >= n || k >= n) return bf16x8{};
  bf16x8 f = *reinterpret_cast<const bf16x8*>(plane + (int64_t)row * n8 + k);
  if (tail) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (k + j >= n) f[j] = (bf16)0.f;
  }
  return f;
}

__global__ void __launch_bounds__(256, 2) triangle_mfma_kernel(TriArgs p) {
  const int id = blockIdx.x;
  const int item = id / p.nblk, cb = id % p.nblk;
  const int i = p.work[4 * item];
  if (i < 0) return;
  const int xt = p.work[4 * item + 1], yt = p.work[4 * item + 2];
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int n8 = (n + 7) & ~7;
  const int64_t P = p.cu_pad[i], cu = p.cu_pairs[i];
  const int x0 = xt * kTriTile, y0 = yt * kTriTile;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int c0 = cb * kTriCB + wave * kTriCW;

  const bf16* ap[kTriCW];
  const bf16* bp[kTriCW];
#pragma unroll
  for (int ch = 0; ch < kTriCW; ++ch) {
    ap[ch] = p.a + (int64_t)(c0 + ch) * p.ld_ab + P;
    bp[ch] = p.b + (int64_t)(c0 + ch) * p.ld_ab + P;
  }
  f32x4 acc[kTriCW][2][2];
#pragma unroll
  for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
    for (int xs = 0; xs < 2; ++xs)
#pragma unroll
      for (int ys = 0; ys < 2; ++ys) acc[ch][xs][ys] = f32x4{0.f, 0.f, 0.f, 0.f};

  bf16x8 fa[kTriCW][2], fb[kTriCW][2];
  auto load_step = [&](int k0, bf16x8 (&ra)[kTriCW][2], bf16x8 (&rb)[kTriCW][2]) {
    const int k = k0 + 8 * g;
    const bool tail = k0 + 32 > n;
#pragma unroll
    for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        ra[ch][h] = load_frag(ap[ch], x0 + 16 * h + l16, k, n, n8, tail);
        rb[ch][h] = load_frag(bp[ch], y0 + 16 * h + l16, k, n, n8, tail);
      }
  };
  load_step(0, fa, fb);
  for (int k0 = 0; k0 < n; k0 += 32) {
    bf16x8 na[kTriCW][2], nb[kTriCW][2];
    load_step(k0 + 32, na, nb);              // all-zero without a load past the last step
#pragma unroll
    for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
      for (int xs = 0; xs < 2; ++xs)
#pragma unroll
        for (int ys = 0; ys < 2; ++ys) acc[ch][xs][ys] = mfma16(fa[ch][xs], fb[ch][ys], acc[ch][xs][ys]);
#pragma unroll
    for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
      for (int h = 0; h < 2; ++h) { fa[ch][h] = na[ch][h]; fb[ch][h] = nb[ch][h]; }
  }

  // acc[ch][xs][ys][r] = T_{c0+ch}[x0 + 16xs + 4g + r][y0 + 16ys + l16]
#pragma unroll
  for (int xs = 0; xs < 2; ++xs)
#pragma unroll
    for (int ys = 0; ys < 2; ++ys)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int x = x0 + 16 * xs + 4 * g + r, y = y0 + 16 * ys + l16;
        if (x >= n || y >= n) continue;
        bf16x4* zp = reinterpret_cast<bf16x4*>(p.z + (cu + (int64_t)x * n + y) * p.ld_z + c0);
        bf16x4 zz = *zp;
#pragma unroll
        for (int ch = 0; ch < kTriCW; ++ch) zz[ch] = (bf16)((float)zz[ch] + acc[ch][xs][ys][r]);
        *zp = zz;
      }
}

// ---------------------------------------------------------------- fp32 path
struct TriF32Args {
  int C;
  const float* a;
  const float* b;
  int64_t ld_ab;
  float* z;
  int64_t ld_z;
  const int32_t* work;
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  const int32_t* cu_pad;
};

// One thread per (cell, channel) of the tile; exact fp32 dot over k.
__global__ void __launch_bounds__(256) triangle_f32_kernel(TriF32Args p) {
  const int item = blockIdx.x;
  const int i = p.work[4 * item];
  if (i < 0) return;
  const int xt = p.work[4 * item + 1], yt = p.work[4 * item + 2];
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int n8 = (n + 7) & ~7;
  const int64_t P = p.cu_pad[i], cu = p.cu_pairs[i];
  const int total = kTriTile * kTriTile * p.C;
  for (int e = threadIdx.x; e < total; e += 256) {
    const int c = e % p.C, cell = e / p.C;
    const int x = xt * kTriTile + cell / kTriTile, y = yt * kTriTile + cell % kTriTile;
    if (x >= n || y >= n) continue;
    const float* ar = p.a + (int64_t)c * p.ld_ab + P + (int64_t)x * n8;
    const float* br = p.b + (int64_t)c * p.ld_ab + P + (int64_t)y * n8;
    float s = 0.f;
    for (int k = 0; k < n; ++k) s = fmaf(ar[k], br[k], s);
    p.z[(cu + (int64_t)x * n + y) * p.ld_z + c] += s;
  }
}

}  // namespace

hipError_t launch_triangle(const nt_layout& L, int C, const void* a, const void* b, int64_t ld_ab, void* z,
                           int64_t ld_z, nt_dtype dtype, hipStream_t s) {
  const int64_t items = L.tri_items();
  if (items == 0) return hipSuccess;
  if (dtype == NT_F32) {
    TriF32Args t{C, (const float*)a, (const float*)b, ld_ab, (float*)z, ld_z, L.d_tri_work, L.d_cu_seqlens,
                 L.d_cu_pairs, L.d_cu_pad};
    triangle_f32_kernel<<<dim3((unsigned)items), dim3(256), 0, s>>>(t);
    return hipGetLastError();
  }
  const int nblk = C / kTriCB;
  TriArgs t{C, nblk, (const bf16*)a, (const bf16*)b, ld_ab, (bf16*)z, ld_z, L.d_tri_work, L.d_cu_seqlens,
            L.d_cu_pairs, L.d_cu_pad};
  triangle_mfma_kernel<<<dim3((unsigned)(items * nblk)), dim3(256), 0, s>>>(t);
  return hipGetLastError();
}

}  // namespace nt
