// SwiGLU transition on packed pair rows (Eq. running-block, line 2; the
// transition of the Pairformer-style block of Sec. 4.3, expansion 4 as in
// App. A.1):
//
//   y = r + (silu(x^ W_g^T + b_g) * (x^ W_u^T + b_u)) W_d^T + b_d,   x^ = LN(x)
//
// with the residual r = x.  Rows are independent, so one launch covers the
// whole ragged batch as a dense [R, K] problem.
//
// Design (gfx950, one 8-wave workgroup per CU, two waves per SIMD):
//   * A pass covers 256 rows: each wave owns 32 of them as two 16-row
//     subtiles, held as matrix-core B fragments (the normalised rows) and as
//     fp32 accumulators of all K outputs.
//   * The hidden width is walked in chunks of 32 units.  A chunk's gate/up
//     weights and its down-projection columns are copied global -> LDS as
//     fragment images (global_load_lds, 1 KB per wave instruction) into a ring
//     of three slots, two chunks ahead of use, so a copy has two chunk times to
//     land.  All eight waves share the ring: the weights cross L2 -> LDS once
//     per 256 rows.  One workgroup barrier per chunk recycles the slots.
//   * Chunk c runs its gate/up products, then the down products subtile by
//     subtile; SiLU starts during the last product step on the finished halves
//     and continues beside the down products, so exp and reciprocal run under
//     the matrix-core work, and the other wave of the SIMD fills the gaps.
//   * The pass's raw rows are copied into a wave-private LDS region one pass
//     ahead.  They are read twice: for LayerNorm, and to seed the output
//     accumulators with residual + b_d, so the epilogue is a convert and a
//     store.
//   * Hidden units are permuted inside a chunk (see transition_image_kernel)
//     so the gate/up accumulators of a lane are the down product's B operand.
// Measured alternative: one 4-wave workgroup per CU with 64 rows per wave
// (weight fragments reused four times) was slower (219 vs 177 us on a
// 364k-row, 128 -> 512 -> 128 transition): one wave per SIMD leaves every
// LDS and barrier latency exposed.
#include <algorithm>

#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int kTwThreads = 512;                   // 8 waves, two per SIMD
constexpr int kTwWaves = kTwThreads / 64;
constexpr int kTwMT = 2;                          // 16-row subtiles per wave
constexpr int kTwRows = kTwWaves * kTwMT * 16;    // rows per pass
constexpr int kTwSlots = 3;                       // slots of each weight ring
constexpr int kTwMaxHidden = kTransitionMaxHidden;

template <int K> constexpr int tw_gu_frags() { return 4 * (K / 32); }   // gate + up images of a chunk
template <int K> constexpr int tw_d_frags() { return K / 16; }          // down-projection images of a chunk
template <int K> constexpr int tw_chunk_frags() { return tw_gu_frags<K>() + tw_d_frags<K>(); }
template <int K> constexpr size_t tw_smem_bytes() {
  return 1024 * ((size_t)kTwSlots * tw_chunk_frags<K>() + (size_t)kTwWaves * kTwMT * (K / 32));
}

// Weights in the order the chunks consume them: chunk f (32 hidden units) is
// CF consecutive fragment images of 64 lanes x 8 bf16.
//   gate/up image im = (which * 2 + ft) * KT + kk, lane (l16, g): row
//     which * F + hid of w, hid = 32 f + 8 (l16 / 4) + 4 ft + l16 % 4, columns
//     32 kk + 8 g .. +7.  The permutation puts hidden units 8 g .. 8 g + 7 of
//     the chunk in the accumulators of lane group g.
//   down image GU + a, lane (l16, g): row 16 a + l16 of w2, columns 32 f + 8 g ..
// One thread per 16-byte lane piece.
template <int K>
__global__ void __launch_bounds__(256) transition_image_kernel(const bf16* w, const bf16* w2, int F, bf16* img) {
  constexpr int KT = K / 32;
  constexpr int GU = tw_gu_frags<K>(), CF = tw_chunk_frags<K>();
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)(F / 32) * CF * 64;
  if (u >= total) return;
  const int lane = (int)(u % 64), im = (int)((u / 64) % CF), f = (int)(u / (64 * CF));
  const int l16 = lane & 15, g = lane >> 4;
  const bf16* src;
  if (im < GU) {
    const int which = im / (2 * KT), ft = (im / KT) & 1, kk = im % KT;
    const int hid = f * 32 + 8 * (l16 >> 2) + 4 * ft + (l16 & 3);
    src = w + (int64_t)(which * F + hid) * K + kk * 32 + g * 8;
  } else {
    const int a = im - GU;
    src = w2 + (int64_t)(a * 16 + l16) * F + f * 32 + g * 8;
  }
  *reinterpret_cast<uint4*>(img + u * 8) = *reinterpret_cast<const uint4*>(src);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt low bits [3:0], high bits [15:14]; expcnt and lgkmcnt at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void lds_copy16(const bf16* src, bf16* dst) {
  __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}

template <int K>
__global__ void __launch_bounds__(kTwThreads, 1) transition_wide_kernel(TransArgs p) {
  constexpr int KT = K / 32, NT = K / 16, MT = kTwMT;
  constexpr int GU = tw_gu_frags<K>(), DF = tw_d_frags<K>(), CF = GU + DF;
  // copies per wave and chunk; when the images do not split evenly the
  // last image is copied by several waves (identical bytes to one place), so
  // every wave issues the same count and the vmcnt waits below hold per wave
  constexpr int WC = (CF + kTwWaves - 1) / kTwWaves;
  constexpr int XC = MT * KT;                              // row copies per wave and pass

  static_assert(WC + XC < 64, "vmcnt range");
  constexpr int NSTEP = 2 * KT;                            // gate/up product steps per chunk

  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  __shared__ __attribute__((aligned(16))) float s_tab[2 * kTwMaxHidden + 3 * K];
  bf16* Wr = smem;                                         // kTwSlots x CF images (gate/up, then down)
  float* s_b = s_tab;                                      // [2F] gate/up bias
  float* s_b2 = s_b + 2 * p.F;                             // [K] down bias
  float* s_g = s_b2 + K;                                   // [K] LayerNorm gamma, then beta
  float* s_be = s_g + K;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  const int nch = p.F / 32;
  const int npass = (p.rows + kTwRows - 1) / kTwRows;
  int pass = blockIdx.x;
  if (pass >= npass) return;
  bf16* Xw = Wr + kTwSlots * CF * 512 + wave * XC * 512;   // this wave's raw rows
  for (int j = tid; j < 2 * p.F; j += kTwThreads) s_b[j] = p.bias ? p.bias[j] : 0.f;
  for (int j = tid; j < K; j += kTwThreads) {
    s_b2[j] = p.bias2 ? p.bias2[j] : 0.f;
    s_g[j] = p.gamma ? p.gamma[j] : 1.f;
    s_be[j] = p.beta ? p.beta[j] : 0.f;
  }

  // ---- copies ---------------------------------------------------------------
  auto copy_chunk = [&](int f, int slot) __attribute__((always_inline)) {
    const bf16* src = p.wimg + (int64_t)f * CF * 512 + lane * 8;
#pragma unroll
    for (int j = 0; j < WC; ++j) {
      const int im = min(wave + kTwWaves * j, CF - 1);
      lds_copy16(src + im * 512, Wr + (slot * CF + im) * 512);
    }
  };
  // rows of subtile (wave, mt) of a pass, as B-fragment images: image
  // (mt, kk), lane (l16, g) = row l16, columns 32 kk + 8 g .. +7.  Rows past
  // the end repeat the last row (computed, never stored).
  // row of lane l16 in subtile (wave, mt) of pass ps, clamped to the last row
  auto row_of = [&](int ps, int mt) -> int64_t __attribute__((always_inline)) {
    return min((int64_t)ps * kTwRows + (wave * MT + mt) * 16 + l16, (int64_t)p.rows - 1);
  };
  auto copy_x = [&](int ps) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int64_t m = row_of(ps, mt);
      const bf16* src = p.x + m * p.ldx + g * 8;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) lds_copy16(src + kk * 32, Xw + (mt * KT + kk) * 512);
    }
  };

  bf16x8 xf[MT][KT];                                       // normalised rows (B fragments)
  f32x4 accY[NT][MT];                                      // outputs: channels 16a + 4g + i, row l16
  auto layer_norm = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      uint4 raw[KT];
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) raw[kk] = *reinterpret_cast<const uint4*>(Xw + (mt * KT + kk) * 512 + lane * 8);
      float s = 0.f;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const uint32_t w4[4] = {raw[kk].x, raw[kk].y, raw[kk].z, raw[kk].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) s += __uint_as_float(w4[j] << 16) + __uint_as_float(w4[j] & 0xffff0000u);
      }
      const float mean = sum_over_kgroups(s) * (1.f / K);
      float qv = 0.f;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const uint32_t w4[4] = {raw[kk].x, raw[kk].y, raw[kk].z, raw[kk].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float d0 = __uint_as_float(w4[j] << 16) - mean, d1 = __uint_as_float(w4[j] & 0xffff0000u) - mean;
          qv += d0 * d0 + d1 * d1;
        }
      }
      const float rstd = rsqrtf(sum_over_kgroups(qv) * (1.f / K) + p.eps);
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int k0 = kk * 32 + g * 8;
        const float4 g0 = *reinterpret_cast<const float4*>(&s_g[k0]), g1 = *reinterpret_cast<const float4*>(&s_g[k0 + 4]);
        const float4 b0 = *reinterpret_cast<const float4*>(&s_be[k0]), b1 = *reinterpret_cast<const float4*>(&s_be[k0 + 4]);
        const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        const float bb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
        const uint32_t w4[4] = {raw[kk].x, raw[kk].y, raw[kk].z, raw[kk].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          xf[mt][kk][2 * j] = (bf16)((__uint_as_float(w4[j] << 16) - mean) * rstd * gg[2 * j] + bb[2 * j]);
          xf[mt][kk][2 * j + 1] = (bf16)((__uint_as_float(w4[j] & 0xffff0000u) - mean) * rstd * gg[2 * j + 1] + bb[2 * j + 1]);
        }
      }
    }
  };
  // output accumulators seeded with residual + b_d.  The residual of lane
  // (l16, g) for tile a is channels 16a + 4g .. +3 of row l16: the 8-byte half
  // (g & 1) of lane l16 + 16 ((a & 1) * 2 + g / 2) of row image (mt, a / 2).
  auto seed_out = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int a = 0; a < NT; ++a) {
        const char* base = reinterpret_cast<const char*>(Xw + (mt * KT + a / 2) * 512);
        const uint2 rr = *reinterpret_cast<const uint2*>(base + 16 * (l16 + 16 * ((a & 1) * 2 + (g >> 1))) + 8 * (g & 1));
        const float4 b2 = *reinterpret_cast<const float4*>(&s_b2[a * 16 + 4 * g]);
        accY[a][mt] = f32x4{b2.x + __uint_as_float(rr.x << 16), b2.y + __uint_as_float(rr.x & 0xffff0000u),
                            b2.z + __uint_as_float(rr.y << 16), b2.w + __uint_as_float(rr.y & 0xffff0000u)};
      }
  };
  // Lane (l16, g) holds channels 16 a + 4 g .. + 3 of row l16.  Lane-row
  // groups g, g ^ 1 trade the pieces of tiles a, a + 1 (a even), so that an
  // even g holds channels 16 a + 4 g .. + 7 and an odd g 16 (a + 1) +
  // 4 (g - 1) .. + 7: one 16-byte store per lane and tile pair, the four lane
  // groups of a row writing 64 contiguous bytes (the address unit is charged
  // per line a store instruction touches).
  auto store_out = [&](int ps) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int64_t m = (int64_t)ps * kTwRows + (wave * MT + mt) * 16 + l16;
      uint32_t ow[NT][2];
#pragma unroll
      for (int a = 0; a < NT; ++a) {
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (bf16)accY[a][mt][i];
        const uint2 u = __builtin_bit_cast(uint2, o);
        ow[a][0] = u.x;
        ow[a][1] = u.y;
      }
#pragma unroll
      for (int a = 0; a < NT; a += 2)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const auto sw = __builtin_amdgcn_permlane16_swap(ow[a][e], ow[a + 1][e], false, false);
          ow[a][e] = sw[0];
          ow[a + 1][e] = sw[1];
        }
      if (m >= p.rows) continue;
#pragma unroll
      for (int a = 0; a < NT; a += 2) {
        const int c = 16 * a + ((g & 1) ? 16 + 4 * (g - 1) : 4 * g);
        *reinterpret_cast<uint4*>(p.y + m * p.ldy + c) = make_uint4(ow[a][0], ow[a][1], ow[a + 1][0], ow[a + 1][1]);
      }
    }
  };
  static_assert(NT % 2 == 0, "tiles pair up for the 16-byte stores");

  // gate and up biases of the chunk at hidden offset f0: slot j = 4 ft + i of
  // lane group g is hidden unit f0 + 8g + j.  Read with inline assembly and
  // its own wait, so the compiler does not first wait for copies in flight.
  auto read_bias = [&](int f0, float (&bg)[8], float (&bu)[8]) __attribute__((always_inline)) {
    float4 bg0, bg1, bu0, bu1;
    const uint32_t ag = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)(&s_b[f0 + 8 * g]);
    const uint32_t au = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)(&s_b[p.F + f0 + 8 * g]);
    asm volatile(
        "ds_read_b128 %0, %4\n"
        "ds_read_b128 %1, %4 offset:16\n"
        "ds_read_b128 %2, %5\n"
        "ds_read_b128 %3, %5 offset:16\n"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(bg0), "=&v"(bg1), "=&v"(bu0), "=&v"(bu1)
        : "v"(ag), "v"(au)
        : "memory");
    bg[0] = bg0.x; bg[1] = bg0.y; bg[2] = bg0.z; bg[3] = bg0.w; bg[4] = bg1.x; bg[5] = bg1.y; bg[6] = bg1.z; bg[7] = bg1.w;
    bu[0] = bu0.x; bu[1] = bu0.y; bu[2] = bu0.z; bu[3] = bu0.w; bu[4] = bu1.x; bu[5] = bu1.y; bu[6] = bu1.z; bu[7] = bu1.w;
  };
  auto seed_gu = [&](int f0, f32x4 (&aG)[2][MT], f32x4 (&aU)[2][MT]) __attribute__((always_inline)) {
    float bg[8], bu[8];
    read_bias(f0, bg, bu);
#pragma unroll
    for (int ft = 0; ft < 2; ++ft)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        aG[ft][mt] = f32x4{bg[4 * ft], bg[4 * ft + 1], bg[4 * ft + 2], bg[4 * ft + 3]};
        aU[ft][mt] = f32x4{bu[4 * ft], bu[4 * ft + 1], bu[4 * ft + 2], bu[4 * ft + 3]};
      }
  };
  // gate/up fragments of product step st = 2 kk + ft from ring slot W
  auto gu_frags = [&](const bf16* W, int st, bf16x8& ag, bf16x8& au) __attribute__((always_inline)) {
    const int kk = st >> 1, ft = st & 1;
    ag = *reinterpret_cast<const bf16x8*>(&W[(ft * KT + kk) * 512 + lane * 8]);
    au = *reinterpret_cast<const bf16x8*>(&W[((2 + ft) * KT + kk) * 512 + lane * 8]);
  };
  auto gu_step = [&](int st, const bf16x8& ag, const bf16x8& au, f32x4 (&aG)[2][MT], f32x4 (&aU)[2][MT])
      __attribute__((always_inline)) {
    const int kk = st >> 1, ft = st & 1;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      aG[ft][mt] = mfma16(ag, xf[mt][kk], aG[ft][mt]);
      aU[ft][mt] = mfma16(au, xf[mt][kk], aU[ft][mt]);
    }
  };

  // SiLU-gated values of unit (mt, ft): hidden units 8 g + 4 ft + i of row
  // l16 of subtile mt, the B operand of the down product.
  bf16x8 hv[MT];
  auto silu_unit = [&](int mt, int ft, const f32x4 (&G)[2][MT], const f32x4 (&U)[2][MT]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float gv = G[ft][mt][i], uv = U[ft][mt][i];
      hv[mt][4 * ft + i] = (bf16)(gv * __builtin_amdgcn_rcpf(1.f + __expf(-gv)) * uv);
    }
  };

  // ---- prologue ---------------------------------------------------------------
  copy_x(pass);
  copy_chunk(0, 0);
  copy_chunk(1, 1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();                                         // tables and first weights visible
  layer_norm();
  seed_out();
  __builtin_amdgcn_s_waitcnt(0);                           // row reads done before the region is refilled
  copy_x(pass + (int)gridDim.x);

  // ---- chunks -----------------------------------------------------------------
  // Chunk c (ring slot q % kTwSlots, q = chunks so far):
  //   gate/up products in 8 steps (k-block kk, half ft), weight fragments read
  //   one step ahead; during the last step SiLU starts on the finished halves;
  //   then the down products subtile by subtile, each beside the SiLU of the
  //   next units, so exp and reciprocal run under the matrix-core work.
  f32x4 G[2][MT], U[2][MT];
  int q = 0;
  for (; pass < npass; pass += (int)gridDim.x) {
    const bool more = pass + (int)gridDim.x < npass;
    for (int c = 0; c < nch; ++c, ++q) {
      copy_chunk((c + 2) % nch, (q + 2) % kTwSlots);
      const bf16* W = Wr + (q % kTwSlots) * CF * 512;
      seed_gu(c * 32, G, U);
      bf16x8 ag, au;
      gu_frags(W, 0, ag, au);
      bf16x8 ad[NT];
#pragma unroll
      for (int st = 0; st < NSTEP; ++st) {
        bf16x8 agn, aun;
        if (st + 1 < NSTEP) gu_frags(W, st + 1, agn, aun);
        else {
#pragma unroll
          for (int a = 0; a < NT; ++a) ad[a] = *reinterpret_cast<const bf16x8*>(&W[(GU + a) * 512 + lane * 8]);
        }
        gu_step(st, ag, au, G, U);
        if (st == NSTEP - 1) {                             // first halves (ft = 0) are final
          silu_unit(0, 0, G, U);
          if (MT > 1) silu_unit(1, 0, G, U);
        }
        if (st + 1 < NSTEP) { ag = agn; au = aun; }
        __builtin_amdgcn_sched_barrier(0);
      }
      silu_unit(0, 1, G, U);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int a = 0; a < NT; ++a) accY[a][mt] = mfma16(ad[a], hv[mt], accY[a][mt]);
        // units still to gate, in order (1,1) (2,0) (2,1) (3,0) (3,1) ...
        if (mt + 1 < MT) silu_unit(mt + 1, 1, G, U);
        if (mt + 2 < MT) silu_unit(mt + 2, 0, G, U);
        __builtin_amdgcn_sched_barrier(0);
      }
      // The slot read at the next chunk was copied at the previous one; what
      // was issued since may stay in flight.  The barrier frees this chunk's
      // slot for the copy issued at the next chunk.
      // (A plain s_barrier: __syncthreads would also wait for every copy in
      // flight.  Each wave's LDS reads of the slot were consumed by its
      // products before the barrier.)
      if (c == 0) wait_vmcnt<WC + XC>();
      else wait_vmcnt<WC>();
      __builtin_amdgcn_s_barrier();
    }
    store_out(pass);
    if (more) {
      layer_norm();                                        // next pass's rows (landed: see the waits above)
      seed_out();
      __builtin_amdgcn_s_waitcnt(0);                       // row reads done before the region is refilled
      copy_x(pass + 2 * (int)gridDim.x);
    }
  }
  __builtin_amdgcn_s_waitcnt(0);                           // no copy outstanding at exit
}

}  // namespace

bool transition_supported(int K, int N, int F) {
  return (K == 64 || K == 128) && N == K && F >= 64 && F % 64 == 0 && F <= kTwMaxHidden;
}

hipError_t launch_transition(TransArgs p, void* wimg_workspace, hipStream_t s) {
  if (p.rows == 0) return hipSuccess;
  const int nch = p.F / 32;
  const size_t img_elems = (size_t)nch * (p.K == 64 ? tw_chunk_frags<64>() : tw_chunk_frags<128>()) * 512;
  (void)img_elems;
  p.wimg = static_cast<const bf16*>(wimg_workspace);
  const unsigned ig = (unsigned)((img_elems / 8 + 255) / 256);
  if (p.K == 64) transition_image_kernel<64><<<dim3(ig), dim3(256), 0, s>>>(p.w, p.w2, p.F, (bf16*)wimg_workspace);
  else transition_image_kernel<128><<<dim3(ig), dim3(256), 0, s>>>(p.w, p.w2, p.F, (bf16*)wimg_workspace);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int npass = (p.rows + kTwRows - 1) / kTwRows;
  const int grid = std::min(npass, compute_units());
  if (p.K == 64) {
    const size_t smem = tw_smem_bytes<64>();
    (void)hipFuncSetAttribute((const void*)transition_wide_kernel<64>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    transition_wide_kernel<64><<<dim3((unsigned)grid), dim3(kTwThreads), smem, s>>>(p);
  } else {
    const size_t smem = tw_smem_bytes<128>();
    (void)hipFuncSetAttribute((const void*)transition_wide_kernel<128>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    transition_wide_kernel<128><<<dim3((unsigned)grid), dim3(kTwThreads), smem, s>>>(p);
  }
  return hipGetLastError();
}

size_t transition_image_bytes(int K, int F) {
  return (size_t)(F / 32) * (K == 64 ? tw_chunk_frags<64>() : tw_chunk_frags<128>()) * 1024;
}

}  // namespace nt
