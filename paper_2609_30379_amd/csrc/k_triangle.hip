// Triangle multiplicative update as one ragged grouped GEMM over the batch:
// for every sample i and channel c, T_c = A_c B_c^T with A_c, B_c the
// sample's N_i x N_i channel planes, then z[cell(x,y), c] += T_c[x, y].
//
// Operands arrive pair-tiled (every 16 x 32 fragment stored in lane order),
// so each matrix-core fragment is one contiguous 1 KB wave load.  The kernel
// is bound by the vector-memory path that carries those loads, so a wave
// keeps a whole 64 x 64 cell tile of one channel in registers: each k-step
// loads 4 + 4 fragments for 16 products (half a load per product).  A
// workgroup of 16 waves owns the tile for a block of 16 channels, and the
// finished tile goes through LDS in four bands of 16 rows so that z is
// updated in 32-byte pieces (16 channels of a cell).  The four channel blocks
// that share one 128-byte line of z (64 channels) run back to back on the
// same XCD, so each z line is fetched into one L2 once instead of into four;
// this outweighs keeping a sample's operand planes in one L2 (re-reads of
// neighbouring tiles then come from the memory-side cache).
#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kTriCB = 16;         // channels per workgroup (one per wave)
constexpr int kTriThreads = 64 * kTriCB;
constexpr int kTriSC = 20;         // LDS floats per staged cell (16 channels + 4)
constexpr int kTriRS = kTriTile + 1;  // staged cells per band row: the 4 lane groups of a write hit different banks

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
  int items, groups;     // tiles, and line groups of four channel blocks
  int accumulate;        // 1: z += t;  0: z = t (z is not read)
  const int32_t* split;  // [9] item ranges of the XCDs
};

__global__ void __launch_bounds__(kTriThreads, 1) triangle_mfma_kernel(TriArgs p) {
  __shared__ __attribute__((aligned(16))) float stage[16 * kTriRS * kTriSC];
  __shared__ __attribute__((aligned(16))) bf16 zbuf[2][16 * kTriTile * kTriCB];   // z of two bands, [row][col][16]
  // Workgroup id runs on XCD x = id % 8, which takes the contiguous range
  // [4 G split[x], 4 G split[x + 1]) of the sequence u = 4 v + j, where v runs
  // over (sample, line group, tile) with the sample's tiles innermost, j is
  // the channel block inside the line group and G the line groups; the item
  // cuts split[] balance the k-steps over the XCDs.  The 32 workgroups an XCD
  // holds at once then cover 8 tiles x 4 channel blocks of one sample and
  // line group: an operand row block is fetched into that L2 for all tiles
  // that use it, and each z line by the four blocks that share it.
  const int id = blockIdx.x, xcd = id % kXcds;
  const int u = 4 * p.groups * p.split[xcd] + id / kXcds;
  if (u >= 4 * p.groups * p.split[xcd + 1]) return;
  const int v = u >> 2;
  const int e = v / p.groups;                         // an item of the same sample
  if (e >= p.items) return;
  const int i = p.work[4 * e];
  if (i < 0) return;
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int first = p.work[4 * e + 3], ntile = (n + kTriTile - 1) / kTriTile;
  const int r = v - p.groups * first;                 // in [0, groups * ntile^2)
  const int item = first + r % (ntile * ntile), cb = (r / (ntile * ntile)) * 4 + (u & 3);
  if (cb >= p.nblk) return;
  const int xt = p.work[4 * item + 1], yt = p.work[4 * item + 2];
  const int nkt = (n + 31) >> 5;
  const int64_t P = p.cu_pad[i], cu = p.cu_pairs[i];
  const int x0 = xt * kTriTile, y0 = yt * kTriTile;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  const int c = cb * kTriCB + wave;

  // z of band xs (16 rows x 64 cells x 16 channels) copied global -> LDS into
  // zbuf[slot] as [row][cell][16]: copy instruction u of the band covers row
  // u / 2, cells 32 (u % 2) .. +31, two lanes per cell.  Cells past N read the
  // sample's last cell (never written back).  Bands 0 and 1 are copied before
  // the contraction, band xs + 2 while band xs is written.
  auto z_copy = [&](int xs, int slot) {
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int u = wave + kTriCB * v;                // 0 .. 31
      const int r = u >> 1, cell = (u & 1) * 32 + (lane >> 1), half = lane & 1;
      const int x = min(x0 + 16 * xs + r, n - 1), y = min(y0 + cell, n - 1);
      const bf16* src = p.z + (cu + (int64_t)x * n + y) * p.ld_z + cb * kTriCB + half * 8;
      bf16* dst = &zbuf[slot][(r * kTriTile + (u & 1) * 32) * kTriCB];
      __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
    }
  };
  if (p.accumulate) {
    z_copy(0, 0);
    if (x0 + 16 < n) z_copy(1, 1);
  }

  // row tiles of the output tile that hold rows of the sample (uniform)
  bool xv[4], yv[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) { xv[s] = x0 + 16 * s < n; yv[s] = y0 + 16 * s < n; }
  const bf16* ap = p.a + (int64_t)c * p.ld_ab + P + lane * 8;
  const bf16* bp = p.b + (int64_t)c * p.ld_ab + P + lane * 8;
  f32x4 acc[4][4];
#pragma unroll
  for (int xs = 0; xs < 4; ++xs)
#pragma unroll
    for (int ys = 0; ys < 4; ++ys) acc[xs][ys] = f32x4{0.f, 0.f, 0.f, 0.f};

  // k-step kt: fragment (row tile, kt) of each plane.  Row tiles past the
  // sample read as zero without a load; k past N is zeroed in the last step
  // (rows past N inside a row tile only reach discarded cells).
  for (int kt = 0; kt < nkt; ++kt) {
    bf16x8 fa[4], fb[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int64_t ta = ((int64_t)((x0 >> 4) + s) * nkt + kt) << 9;
      const int64_t tb = ((int64_t)((y0 >> 4) + s) * nkt + kt) << 9;
      fa[s] = xv[s] ? *reinterpret_cast<const bf16x8*>(ap + ta) : bf16x8{};
      fb[s] = yv[s] ? *reinterpret_cast<const bf16x8*>(bp + tb) : bf16x8{};
    }
    const int kbase = kt * 32 + 8 * g;
    if (kbase + 8 > n) {
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (kbase + j >= n) { fa[s][j] = (bf16)0.f; fb[s][j] = (bf16)0.f; }
    }
#pragma unroll
    for (int xs = 0; xs < 4; ++xs)
#pragma unroll
      for (int ys = 0; ys < 4; ++ys) acc[xs][ys] = mfma16(fa[xs], fb[ys], acc[xs][ys]);
  }

  // acc[xs][ys][r] = T_c[x0 + 16xs + 4g + r][y0 + 16ys + l16].  Band xs:
  // stage its 16 x 64 cells as [cell][16 channels] fp32, then two threads
  // per cell add 8 channels (16 bytes) to the band's z copy and store them.
#pragma unroll
  for (int xs = 0; xs < 4; ++xs) {
    if (!xv[xs]) break;                               // uniform
#pragma unroll
    for (int ys = 0; ys < 4; ++ys)
#pragma unroll
      for (int r = 0; r < 4; ++r) stage[((4 * g + r) * kTriRS + 16 * ys + l16) * kTriSC + wave] = acc[xs][ys][r];
    __builtin_amdgcn_s_waitcnt(0);                    // this wave's z copies (and earlier stores) are done
    __syncthreads();
#pragma unroll
    for (int it = 0; it < 16 * kTriTile * 2 / kTriThreads; ++it) {
      const int u = it * kTriThreads + tid, cell = u >> 1, half = u & 1;
      const int row = cell / kTriTile, col = cell % kTriTile;
      const int x = x0 + 16 * xs + row, y = y0 + col;
      if (x >= n || y >= n) continue;
      const float* st = &stage[(row * kTriRS + col) * kTriSC + half * 8];
      const float4 t0 = *reinterpret_cast<const float4*>(st);
      const float4 t1 = *reinterpret_cast<const float4*>(st + 4);
      float v[8];
      if (p.accumulate) {
        const uint4 zq = *reinterpret_cast<const uint4*>(&zbuf[xs & 1][(row * kTriTile + col) * kTriCB + half * 8]);
        const uint32_t w4[4] = {zq.x, zq.y, zq.z, zq.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[2 * j] = __uint_as_float(w4[j] << 16);
          v[2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = 0.f;
      }
      v[0] += t0.x; v[1] += t0.y; v[2] += t0.z; v[3] += t0.w;
      v[4] += t1.x; v[5] += t1.y; v[6] += t1.z; v[7] += t1.w;
      bf16x8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (bf16)v[e];
      *reinterpret_cast<bf16x8*>(p.z + (cu + (int64_t)x * n + y) * p.ld_z + cb * kTriCB + half * 8) = o;
    }
    __syncthreads();                                  // stage and this band's z copy are free
    if (p.accumulate && xs + 2 < 4 && xv[xs + 2]) z_copy(xs + 2, xs & 1);
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
  int accumulate;
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
    float* zc = p.z + (cu + (int64_t)x * n + y) * p.ld_z + c;
    *zc = p.accumulate ? *zc + s : s;
  }
}

// ---------------------------------------------------------------- packed operands
// Re-tiling of a packed pair tensor [sum N^2, C] (row stride ld_src) into
// pair-tiled channel-major planes (channel stride ld_dst): plane element
// (r, k) of sample i holds cell (r, k) (plain) or cell (k, r) (transposed);
// positions outside the N x N matrix hold 0.  One workgroup per 16 x 32 tile
// (512 positions in fragment order, two per thread); channels are taken 16
// bytes at a time: each thread loads that piece of its two source cells,
// parks it in LDS, and the workgroup writes the chunk's channel slices of the
// tile as contiguous 16-byte pieces.  GATED: each source row holds the
// projection in channels [0, C) and the gate logits in [C, 2C), and the
// plane receives sigmoid(gate) * projection (the gated operands of the
// AlphaFold 3 form of the update), computed in fp32 and rounded once.
template <typename T, bool TRANS, bool GATED = false>
__global__ void __launch_bounds__(256) pack_tiled_kernel(const T* __restrict__ src, int64_t ld_src, int C,
                                                         T* __restrict__ dst, int64_t ld_dst, int batch,
                                                         const int32_t* __restrict__ cu_seqlens,
                                                         const int32_t* __restrict__ cu_pairs,
                                                         const int32_t* __restrict__ cu_pad) {
  constexpr int V = 16 / sizeof(T);                 // channels per 16-byte piece
  __shared__ __attribute__((aligned(16))) T park[V * 512];
  const int64_t tile_pos = (int64_t)blockIdx.x * 512;
  int lo = 0, hi = batch - 1;                       // sample: largest i with cu_pad[i] <= tile_pos
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_pad[mid] <= tile_pos) lo = mid; else hi = mid - 1;
  }
  const int i = lo;
  const int n = cu_seqlens[i + 1] - cu_seqlens[i];
  const int nkt = (n + 31) >> 5;
  const int lt = (int)((tile_pos - cu_pad[i]) >> 9);
  const int rt = lt / nkt, kt = lt % nkt;
  const int64_t cu = cu_pairs[i];
  int64_t row[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int q = threadIdx.x + 256 * h;
    const int r = rt * 16 + ((q >> 3) & 15), k = kt * 32 + (q >> 7) * 8 + (q & 7);
    const int a = TRANS ? k : r, b = TRANS ? r : k;
    row[h] = (r < n && k < n) ? cu + (int64_t)a * n + b : -1;
  }
  for (int c0 = 0; c0 < C; c0 += V) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = threadIdx.x + 256 * h;
      uint4 piece = make_uint4(0u, 0u, 0u, 0u);
      if (row[h] >= 0) piece = *reinterpret_cast<const uint4*>(src + row[h] * ld_src + c0);
      const T* e = reinterpret_cast<const T*>(&piece);
      if constexpr (GATED) {
        uint4 gp = make_uint4(0u, 0u, 0u, 0u);
        if (row[h] >= 0) gp = *reinterpret_cast<const uint4*>(src + row[h] * ld_src + C + c0);
        const T* ge = reinterpret_cast<const T*>(&gp);
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const float gl = (float)ge[j];
          park[j * 512 + q] = (T)((float)e[j] * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-gl * 1.4426950408889634f)));
        }
      } else {
#pragma unroll
        for (int j = 0; j < V; ++j) park[j * 512 + q] = e[j];
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int u = threadIdx.x + 256 * h;          // piece u: channel u / (512 / V), positions V * (u % (512 / V))
      const int ch = u / (512 / V), pos = (u % (512 / V)) * V;
      if (c0 + ch < C)
        *reinterpret_cast<uint4*>(dst + (int64_t)(c0 + ch) * ld_dst + tile_pos + pos) =
            *reinterpret_cast<const uint4*>(&park[ch * 512 + pos]);
    }
    __syncthreads();
  }
}

}  // namespace

size_t triangle_workspace_bytes(const nt_layout& L, int C, nt_tri_operands operands, nt_dtype dtype) {
  if (operands != NT_TRI_PACKED) return 0;
  const size_t ldp = (size_t)((L.sum_pad + 7) / 8 * 8);
  return 2 * (size_t)C * ldp * (dtype == NT_BF16 ? 2 : 4);
}

namespace {

// Re-tiles one packed operand (row stride ld_src) into planes at dst; gated:
// sigmoid(src[:, C:2C]) * src[:, 0:C].
hipError_t pack_planes(const nt_layout& L, const void* src, int64_t ld_src, bool trans, int C, void* dst,
                       int64_t ldp, nt_dtype dtype, hipStream_t s, bool gated = false) {
  const dim3 grid((unsigned)(L.sum_pad / 512));
  if (grid.x == 0) return hipSuccess;
#define NT_PACK(T, TR, G) pack_tiled_kernel<T, TR, G><<<grid, dim3(256), 0, s>>>((const T*)src, ld_src, C, (T*)dst, \
                                                                        ldp, L.batch, L.d_cu_seqlens, L.d_cu_pairs, L.d_cu_pad)
#define NT_PACK_G(T, TR) do { if (gated) NT_PACK(T, TR, true); else NT_PACK(T, TR, false); } while (0)
  if (dtype == NT_BF16) { if (trans) NT_PACK_G(bf16, true); else NT_PACK_G(bf16, false); }
  else { if (trans) NT_PACK_G(float, true); else NT_PACK_G(float, false); }
#undef NT_PACK_G
#undef NT_PACK
  return hipGetLastError();
}

// z[cell(x, y)] (+)= sum_k PA[x, k] PB[y, k] over pair-tiled planes (channel stride ld_ab).
hipError_t contract(const nt_layout& L, int C, const void* a, const void* b, int64_t ld_ab, void* z, int64_t ld_z,
                    nt_dtype dtype, hipStream_t s, int accumulate = 1) {
  const int64_t items = L.tri_items();
  if (items == 0) return hipSuccess;
  if (dtype == NT_F32) {
    TriF32Args t{C, (const float*)a, (const float*)b, ld_ab, (float*)z, ld_z, L.d_tri_work, L.d_cu_seqlens,
                 L.d_cu_pairs, L.d_cu_pad, accumulate};
    triangle_f32_kernel<<<dim3((unsigned)items), dim3(256), 0, s>>>(t);
    return hipGetLastError();
  }
  const int nblk = C / kTriCB, groups = (nblk + 3) / 4;
  TriArgs t{C, nblk, (const bf16*)a, (const bf16*)b, ld_ab, (bf16*)z, ld_z, L.d_tri_work, L.d_cu_seqlens,
            L.d_cu_pairs, L.d_cu_pad, (int)items, groups, accumulate, L.d_tri_split};
  // every XCD gets as many workgroups as the widest of the item ranges needs
  triangle_mfma_kernel<<<dim3((unsigned)((int64_t)L.tri_xcd_items * groups * 4 * kXcds)), dim3(kTriThreads), 0,
                         s>>>(t);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_triangle(const nt_layout& L, int direction, int C, const void* a, const void* b, int64_t ld_ab,
                           nt_tri_operands operands, void* z, int64_t ld_z, nt_dtype dtype, void* workspace,
                           hipStream_t s) {
  if (L.tri_items() == 0) return hipSuccess;
  if (operands == NT_TRI_PACKED) {
    // re-tile a and b into the workspace in the variant the direction needs
    const int64_t ldp = (L.sum_pad + 7) / 8 * 8;
    char* wa = static_cast<char*>(workspace);
    char* wb = wa + (size_t)C * ldp * (dtype == NT_BF16 ? 2 : 4);
    hipError_t e = pack_planes(L, a, ld_ab, direction == 1, C, wa, ldp, dtype, s);
    if (e == hipSuccess) e = pack_planes(L, b, ld_ab, direction == 1, C, wb, ldp, dtype, s);
    if (e != hipSuccess) return e;
    return contract(L, C, wa, wb, ldp, z, ld_z, dtype, s);
  }
  return contract(L, C, a, b, ld_ab, z, ld_z, dtype, s);
}

hipError_t launch_triangle_gated(const nt_layout& L, int direction, int C, const void* a, const void* b,
                                 int64_t ld_ab, nt_tri_operands operands, void* t, int64_t ld_t, nt_dtype dtype,
                                 void* workspace, hipStream_t s) {
  if (L.tri_items() == 0) return hipSuccess;
  if (operands != NT_TRI_PACKED) return contract(L, C, a, b, ld_ab, t, ld_t, dtype, s, 0);
  // gated operands re-tiled into the workspace in the direction's variant,
  // then contracted into t (overwritten)
  const int64_t ldp = (L.sum_pad + 7) / 8 * 8;
  char* wa = static_cast<char*>(workspace);
  char* wb = wa + (size_t)C * ldp * (dtype == NT_BF16 ? 2 : 4);
  hipError_t e = pack_planes(L, a, ld_ab, direction == 1, C, wa, ldp, dtype, s, true);
  if (e == hipSuccess) e = pack_planes(L, b, ld_ab, direction == 1, C, wb, ldp, dtype, s, true);
  if (e != hipSuccess) return e;
  return contract(L, C, wa, wb, ldp, t, ld_t, dtype, s, 0);
}

// Backward, per sample and channel c (T = A B^T outgoing, T = A^T B incoming):
//   outgoing  dA = dT B      = contraction of (dT, B^T) rows;  dB = dT^T A = (dT^T, A^T)
//   incoming  dA = B dT^T    = contraction of (B, dT);         dB = A dT   = (A, dT^T)
// where the contraction computes out[x, y] = sum_k PA[x, k] PB[y, k] and a
// transposed operand is re-tiled in the transposed variant.  Each pair of
// operands is re-tiled into the workspace, then contracted into da or db.
hipError_t launch_triangle_backward(const nt_layout& L, int direction, int C, const void* a, const void* b,
                                    int64_t ld_ab, const void* dt, int64_t ld_dt, void* da, void* db,
                                    int64_t ld_dab, nt_dtype dtype, void* workspace, hipStream_t s) {
  if (L.tri_items() == 0) return hipSuccess;
  const int64_t ldp = (L.sum_pad + 7) / 8 * 8;
  char* wa = static_cast<char*>(workspace);
  char* wb = wa + (size_t)C * ldp * (dtype == NT_BF16 ? 2 : 4);
  struct Pass { const void* pa; int64_t lda; bool ta; const void* pb; int64_t ldb; bool tb; void* out; };
  const Pass first = direction == 0 ? Pass{dt, ld_dt, false, b, ld_ab, true, da}
                                    : Pass{b, ld_ab, false, dt, ld_dt, false, da};
  const Pass second = direction == 0 ? Pass{dt, ld_dt, true, a, ld_ab, true, db}
                                     : Pass{a, ld_ab, false, dt, ld_dt, true, db};
  for (const Pass& p : {first, second}) {
    if (!p.out) continue;
    hipError_t e = pack_planes(L, p.pa, p.lda, p.ta, C, wa, ldp, dtype, s);
    if (e == hipSuccess) e = pack_planes(L, p.pb, p.ldb, p.tb, C, wb, ldp, dtype, s);
    if (e == hipSuccess) e = contract(L, C, wa, wb, ldp, p.out, ld_dab, dtype, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace nt
