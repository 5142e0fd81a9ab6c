// Triangle multiplicative update as one ragged grouped GEMM over the batch:
// for every sample i and channel c, T_c = A_c B_c^T with A_c, B_c the
// sample's N_i x N_i channel planes, then z[cell(x,y), c] += T_c[x, y].
//
// Operands arrive pair-tiled (every 16 x 32 fragment stored in lane order),
// so each matrix-core fragment is one contiguous 1 KB wave load.  A workgroup
// owns a 32x32 cell tile of one sample and a block of 16 channels (4 per
// wave).  Workgroup ids interleave the channel blocks of each tile, so with 8
// blocks (C = 128) XCD x (ids = x mod 8) always works on channel block x: it
// walks the tile list sample by sample and keeps the current sample's 16
// channel planes (about 3 MB at N = 216) in its own L2, where the operand
// re-reads of neighbouring tiles hit.  The next k-step's fragments load while
// the current one is on the matrix cores.  The finished tile goes through LDS
// so that z is updated in 32-byte pieces (16 channels of one cell) instead of
// the 8-byte pieces a single wave holds.
#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kTriCB = 16;    // channels per workgroup
constexpr int kTriCW = 4;     // channels per wave
constexpr int kTriSC = 20;    // LDS floats per staged cell (16 channels + 4: conflict-free 16-byte writes)

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

__global__ void __launch_bounds__(256, 2) triangle_mfma_kernel(TriArgs p) {
  __shared__ __attribute__((aligned(16))) float stage[kTriTile * kTriTile * kTriSC];
  const int id = blockIdx.x;
  const int item = id / p.nblk, cb = id % p.nblk;
  const int i = p.work[4 * item];
  if (i < 0) return;
  const int xt = p.work[4 * item + 1], yt = p.work[4 * item + 2];
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int nkt = (n + 31) >> 5;
  const int64_t P = p.cu_pad[i], cu = p.cu_pairs[i];
  const int x0 = xt * kTriTile, y0 = yt * kTriTile;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int c0 = cb * kTriCB + wave * kTriCW;

  // row tiles of the output tile that hold rows of the sample (uniform)
  const bool xv[2] = {x0 < n, x0 + 16 < n};
  const bool yv[2] = {y0 < n, y0 + 16 < n};
  const bf16* ap[kTriCW];
  const bf16* bp[kTriCW];
#pragma unroll
  for (int ch = 0; ch < kTriCW; ++ch) {
    ap[ch] = p.a + (int64_t)(c0 + ch) * p.ld_ab + P + lane * 8;
    bp[ch] = p.b + (int64_t)(c0 + ch) * p.ld_ab + P + lane * 8;
  }
  f32x4 acc[kTriCW][2][2];
#pragma unroll
  for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
    for (int xs = 0; xs < 2; ++xs)
#pragma unroll
      for (int ys = 0; ys < 2; ++ys) acc[ch][xs][ys] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Fragments of k-step kt: tile (row tile, kt) of each channel plane.  Row
  // tiles past the sample read as zero without a load; k past N is zeroed in
  // the last step (rows past N inside a row tile only reach discarded cells).
  bf16x8 fa[kTriCW][2], fb[kTriCW][2];
  auto load_step = [&](int kt, bf16x8 (&ra)[kTriCW][2], bf16x8 (&rb)[kTriCW][2]) {
    const bool any = kt < nkt;
    const int kbase = kt * 32 + 8 * g;
#pragma unroll
    for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int64_t ta = ((int64_t)((x0 >> 4) + h) * nkt + kt) << 9;
        const int64_t tb = ((int64_t)((y0 >> 4) + h) * nkt + kt) << 9;
        ra[ch][h] = (any && xv[h]) ? *reinterpret_cast<const bf16x8*>(ap[ch] + ta) : bf16x8{};
        rb[ch][h] = (any && yv[h]) ? *reinterpret_cast<const bf16x8*>(bp[ch] + tb) : bf16x8{};
      }
    if (any && kbase + 8 > n) {
#pragma unroll
      for (int ch = 0; ch < kTriCW; ++ch)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (kbase + j >= n) { ra[ch][h][j] = (bf16)0.f; rb[ch][h][j] = (bf16)0.f; }
    }
  };
  load_step(0, fa, fb);
  for (int kt = 0; kt < nkt; ++kt) {
    bf16x8 na[kTriCW][2], nb[kTriCW][2];
    load_step(kt + 1, na, nb);              // all-zero without a load past the last step
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

  // acc[ch][xs][ys][r] = T_{c0+ch}[x0 + 16xs + 4g + r][y0 + 16ys + l16]; stage
  // the tile as [cell][16 channels] fp32
#pragma unroll
  for (int xs = 0; xs < 2; ++xs)
#pragma unroll
    for (int ys = 0; ys < 2; ++ys)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int cell = (16 * xs + 4 * g + r) * kTriTile + 16 * ys + l16;
        *reinterpret_cast<float4*>(&stage[cell * kTriSC + wave * kTriCW]) =
            make_float4(acc[0][xs][ys][r], acc[1][xs][ys][r], acc[2][xs][ys][r], acc[3][xs][ys][r]);
      }
  __syncthreads();
  // z += T: two threads per cell, 8 channels (16 bytes) each
#pragma unroll
  for (int it = 0; it < kTriTile * kTriTile * 2 / 256; ++it) {
    const int u = it * 256 + tid, cell = u >> 1, half = u & 1;
    const int x = x0 + cell / kTriTile, y = y0 + cell % kTriTile;
    if (x >= n || y >= n) continue;
    const float4 t0 = *reinterpret_cast<const float4*>(&stage[cell * kTriSC + half * 8]);
    const float4 t1 = *reinterpret_cast<const float4*>(&stage[cell * kTriSC + half * 8 + 4]);
    bf16* zp = p.z + (cu + (int64_t)x * n + y) * p.ld_z + cb * kTriCB + half * 8;
    Vec<bf16> zz;
    zz.load(zp);
    zz.v[0] += t0.x; zz.v[1] += t0.y; zz.v[2] += t0.z; zz.v[3] += t0.w;
    zz.v[4] += t1.x; zz.v[5] += t1.y; zz.v[6] += t1.z; zz.v[7] += t1.w;
    zz.store(zp);
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
  const int nkt = (n + 31) >> 5;
  const int64_t P = p.cu_pad[i], cu = p.cu_pairs[i];
  const int total = kTriTile * kTriTile * p.C;
  for (int e = threadIdx.x; e < total; e += 256) {
    const int c = e % p.C, cell = e / p.C;
    const int x = xt * kTriTile + cell / kTriTile, y = yt * kTriTile + cell % kTriTile;
    if (x >= n || y >= n) continue;
    const float* ap = p.a + (int64_t)c * p.ld_ab + P;
    const float* bp = p.b + (int64_t)c * p.ld_ab + P;
    float s = 0.f;
    for (int k = 0; k < n; ++k) s = fmaf(ap[tiled_offset(x, k, nkt)], bp[tiled_offset(y, k, nkt)], s);
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
