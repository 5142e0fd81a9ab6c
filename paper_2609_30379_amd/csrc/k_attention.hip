// Segmented softmax attention over packed buffers, one launch for the batch.
//
// A segment is one pair row (axis 0: cells (i, r, *)), one pair column
// (axis 1: cells (i, *, r)) or one sample's tokens (axis 2).  The workgroup
// for (segment, head) stages the segment's keys and transposed values in LDS
// once; each wave then runs 16-query tiles through an online softmax over
// 64-key chunks on matrix cores:
//   S^T = K Q^T       lane (g, q) holds scores of keys 16t + 4g + i for query q,
//                     so the running max/sum of a query live in one lane column
//   O^T += V^T P^T    P is taken from the S^T registers as the B operand
//                     (keys {4g..4g+3} of two 16-key tiles), no shuffles.
#include <algorithm>

#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

struct AttnArgs {
  int axis, H;
  const bf16* q;
  const bf16* k;
  const bf16* v;
  int64_t ld_qkv;
  const bf16* bias;
  int64_t ld_bias;
  float scale_log2;      // softmax scale * log2(e)
  bf16* o;
  int64_t ld_o;
  const int32_t* work;   // (sample, row) or (sample, query block) pairs
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  int vstride;           // LDS row stride of V^T (elements)
};

struct Seg {
  int n;                 // keys in the segment
  int64_t base, step;    // packed row of element t: base + t * step
  int q_begin, q_end;
  int64_t cu;            // pair offset of the sample (bias addressing)
};

template <typename A>
__device__ __forceinline__ bool segment_of(const A& p, Seg& s) {
  const int i = p.work[2 * blockIdx.x], r = p.work[2 * blockIdx.x + 1];
  if (i < 0) return false;
  if (p.axis == 2) {
    s.n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
    s.base = p.cu_seqlens[i];
    s.step = 1;
    s.q_begin = r * kSeqQBlock;
    s.q_end = min(s.n, s.q_begin + kSeqQBlock);
    s.cu = 0;
  } else {
    s.n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
    s.cu = p.cu_pairs[i];
    s.base = p.axis == 0 ? s.cu + (int64_t)r * s.n : s.cu + r;
    s.step = p.axis == 0 ? 1 : s.n;
    s.q_begin = 0;
    s.q_end = s.n;
  }
  return true;
}

template <int D>
__global__ void __launch_bounds__(256) attention_mfma_kernel(AttnArgs p) {
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  constexpr int KS = D + 8;                    // LDS stride of K rows (bf16)
  constexpr int DV = D / 8;                    // 16-byte vectors per head row
  Seg sg;
  if (!segment_of(p, sg)) return;
  const int h = blockIdx.y;
  const int n = sg.n;
  const int npad = (n + 63) & ~63;
  bf16* Ks = lds;                              // [npad][KS]
  bf16* Vt = lds + (size_t)npad * KS;          // [D][vstride]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;

  // ---- stage keys (row-major) and values (transposed) of this head -------
  for (int c = tid; c < npad * DV; c += 256) {
    const int key = c / DV, dc = (c % DV) * 8;
    uint4 kk = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (key < n) {
      const int64_t row = sg.base + (int64_t)key * sg.step;
      kk = *reinterpret_cast<const uint4*>(p.k + row * p.ld_qkv + h * D + dc);
      vv = *reinterpret_cast<const uint4*>(p.v + row * p.ld_qkv + h * D + dc);
    }
    *reinterpret_cast<uint4*>(&Ks[key * KS + dc]) = kk;
    const bf16x8 vb = *reinterpret_cast<const bf16x8*>(&vv);
#pragma unroll
    for (int j = 0; j < 8; ++j) Vt[(dc + j) * p.vstride + key] = vb[j];
  }
  __syncthreads();

  for (int qt = sg.q_begin / 16 + wave; qt * 16 < sg.q_end; qt += 4) {
    const int qi = qt * 16 + l16;
    const bool qvalid = qi < sg.q_end;
    const int64_t qrow = sg.base + (int64_t)qi * sg.step;
    bf16x8 qf[D / 32];
#pragma unroll
    for (int dd = 0; dd < D / 32; ++dd) {
      if (qvalid) qf[dd] = *reinterpret_cast<const bf16x8*>(p.q + qrow * p.ld_qkv + h * D + dd * 32 + g * 8);
      else qf[dd] = bf16x8{};
    }
    float m_run = -INFINITY, l_run = 0.f;
    f32x4 O[D / 16];
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) O[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16* brow = nullptr;                // bias row of this query (axis 0)
    if (p.bias && qvalid) brow = p.bias + (int64_t)h * p.ld_bias + sg.cu + (p.axis == 0 ? (int64_t)qi * n : qi);
    const int64_t bstep = p.axis == 0 ? 1 : n;

    for (int kc = 0; kc < npad; kc += 64) {
      f32x4 s[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        s[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dd = 0; dd < D / 32; ++dd) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[(kc + kt * 16 + l16) * KS + dd * 32 + g * 8]);
          s[kt] = mfma16(kf, qf[dd], s[kt]);
        }
      }
      float x[4][4];
      float mloc = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kc + kt * 16 + 4 * g + i;
          float t = s[kt][i] * p.scale_log2;
          if (brow && key < n) t += (float)brow[(int64_t)key * bstep] * kLog2e;
          t = key < n ? t : -INFINITY;
          x[kt][i] = t;
          mloc = fmaxf(mloc, t);
        }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
      const float m_new = fmaxf(m_run, mloc);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) O[dt] *= alpha;
      bf16x8 pf[2];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = __builtin_amdgcn_exp2f(x[kt][i] - m_new);
          l_run += e;
          pf[kt >> 1][(kt & 1) * 4 + i] = (bf16)e;
        }
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          const bf16* vr = &Vt[(dt * 16 + l16) * p.vstride + kc + pp * 32 + 4 * g];
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vr);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vr + 16);
          const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          O[dt] = mfma16(vf, pf[pp], O[dt]);
        }
    }
    l_run += __shfl_xor(l_run, 16, 64);
    l_run += __shfl_xor(l_run, 32, 64);
    if (qvalid) {
      const float inv = 1.f / l_run;
      bf16* orow = p.o + qrow * p.ld_o + h * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        bf16x4 ov;
#pragma unroll
        for (int i = 0; i < 4; ++i) ov[i] = (bf16)(O[dt][i] * inv);
        *reinterpret_cast<bf16x4*>(orow + dt * 16 + 4 * g) = ov;
      }
    }
  }
}

// ---------------------------------------------------------------- pair attention arguments
struct PairAttnArgs {
  int axis;
  const bf16* q;
  const bf16* k;
  const bf16* v;
  int64_t ld_qkv;
  const bf16* bias;
  int64_t ld_bias;
  float scale_log2;
  bf16* o;
  int64_t ld_o;
  const int32_t* work;   // quads (sample, first 16-query tile, row group, tile count)
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  int bstride;           // LDS stride (elements) of the staged bias slice
  float inv_scale;       // 1 / softmax scale
  int H;                 // heads (interleaved in the grid)
};

// ---------------------------------------------------------------- pair attention, head_dim 32
// Pair attention for head_dim 32 and N_i <= kAttnLongLen, organised so that
// the exponentials are nearly the only vector work.  A workgroup of 8 waves
// takes (sample, block of up to 128 queries, group of 16 pair rows, head):
//   * the bias of (query, key) does not depend on the pair row, so each lane
//     keeps the bias of its query for its 4-key groups of every key tile in
//     registers for the whole group of rows -- staged once through LDS and
//     divided by the softmax scale (one bf16 rounding) -- and it seeds the
//     score accumulators: the matrix cores produce bias/scale + q.k directly;
//   * keys and values of a row are copied straight into LDS (keys as fragment
//     images: 64 lanes x 16 bytes, read as one contiguous 1 KB per wave) in
//     two buffers that alias the bias staging area, the next row's copies in
//     flight while the current row runs: one barrier per row;
//   * the softmax denominator comes from one more matrix-core product with a
//     ones operand, on the same bf16 probabilities as the numerator.
// Scores are kept transposed (S^T = K Q^T), so a lane holds 16 keys of one
// query per 64-key chunk and the running max is mostly lane-local.
// Two instances: N <= 256 (64 KB of LDS, two workgroups per CU) and N <= 512
// (128 KB, one workgroup per CU, twice the bias registers).
template <int NMAX>
__global__ void __launch_bounds__(512, NMAX <= 256 ? 4 : 2) attention_pair_kernel(PairAttnArgs p) {
  constexpr int D = 32;
  constexpr int KT16 = NMAX / 16;               // key tiles
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  // Work position pos runs on XCD pos % 8; the H heads of one position are
  // launched as consecutive workgroups of that XCD (ids 8 (H k + h) + x), so
  // they read the same q|k|v cache lines at about the same time.
  const int x = blockIdx.x % kXcds, t = blockIdx.x / kXcds;
  const int h = t % p.H, pos = (t / p.H) * kXcds + x;
  const int4 w4 = reinterpret_cast<const int4*>(p.work)[pos];
  const int i = w4.x;
  if (i < 0) return;
  const int qt0 = w4.y, rg = w4.z, nqt = w4.w;       // first 16-query tile, row group, tile count
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int npad = (n + 63) & ~63;
  const int64_t cu = p.cu_pairs[i];
  const int64_t sr = p.axis == 0 ? n : 1, st = p.axis == 0 ? 1 : n;   // cell(r, t) = cu + r*sr + t*st
  bf16* Bs = lds;                                          // [kAttnQB][bstride], start-up only
  bf16* Kb0 = lds;                                         // key images: tile of 16 keys -> 512 elements
  bf16* Kb1 = Kb0 + NMAX * D;
  bf16* Vb0 = Kb1 + NMAX * D;                              // values, row-major [key][D]
  bf16* Vb1 = Vb0 + NMAX * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int j0 = qt0 * 16;

  // ---- bias slice / scale: Bs[q][k] = bias(j0 + q, k) / scale, 0 past N --
  {
    const bf16* bh = p.bias ? p.bias + (int64_t)h * p.ld_bias + cu : nullptr;
    const float inv_scale = p.inv_scale;
    if (p.axis == 0) {
      for (int e = tid; e < kAttnQB * (npad / 8); e += 512) {
        const int q = e / (npad / 8), k0 = (e % (npad / 8)) * 8, j = j0 + q;
        bf16x4 o0, o1;                            // rows are 8-byte aligned (stride 4 mod 8 elements)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          o0[u] = (bf16)((bh && j < n && k0 + u < n) ? (float)bh[(int64_t)j * n + k0 + u] * inv_scale : 0.f);
          o1[u] = (bf16)((bh && j < n && k0 + 4 + u < n) ? (float)bh[(int64_t)j * n + k0 + 4 + u] * inv_scale : 0.f);
        }
        *reinterpret_cast<bf16x4*>(&Bs[q * p.bstride + k0]) = o0;
        *reinterpret_cast<bf16x4*>(&Bs[q * p.bstride + k0 + 4]) = o1;
      }
    } else {
      for (int e = tid; e < kAttnQB * npad; e += 512) {
        const int q = e % kAttnQB, k = e / kAttnQB, j = j0 + q;
        Bs[q * p.bstride + k] = (bf16)((bh && j < n && k < n) ? (float)bh[(int64_t)k * n + j] * inv_scale : 0.f);
      }
    }
  }

  // ---- per-row staging: straight global -> LDS copies ---------------------
  // Each wave copies its key tiles (wave, wave + 8, ...; 16 keys each) with
  // global_load_lds, lane l's 16 bytes landing at byte 16 l of the tile:
  //   keys as fragment images: lane l = (key l%16, dims 8 (l/16) ..),
  //   values row-major [key][32]: lane l = (key l/4, dims 8 (l%4) ..).
  // Every tile below the 64-key padded length is written (the last chunk
  // reads up to there): keys past N repeat key N-1, so the padding holds
  // finite values whose probabilities are masked to zero.
  auto dma_kv = [&](int r, bf16* Kb, bf16* Vr) {
#pragma unroll
    for (int kt = wave; kt < KT16; kt += 8) {
      if (kt * 16 >= npad) break;
      // values: the 16-byte chunk at column c of key row kv holds dim group
      // c ^ ((kv >> 2) & 3), so the four key groups of a transpose read fall
      // on different banks
      const int kv = kt * 16 + (lane >> 2);
      const int key_k = min(kt * 16 + l16, n - 1), key_v = min(kv, n - 1);
      const int dgv = (lane & 3) ^ ((kv >> 2) & 3);
      const bf16* sk = p.k + (cu + (int64_t)r * sr + (int64_t)key_k * st) * p.ld_qkv + h * D + g * 8;
      const bf16* sv = p.v + (cu + (int64_t)r * sr + (int64_t)key_v * st) * p.ld_qkv + h * D + dgv * 8;
      __builtin_amdgcn_global_load_lds((const void*)sk, (__attribute__((address_space(3))) void*)(Kb + kt * 512), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)sv, (__attribute__((address_space(3))) void*)(Vr + kt * 512), 16, 0, 0);
    }
  };
  // Value fragments for O^T += V^T P^T: lane (dim 16 dt + l16, k-group g)
  // needs keys 32 kb + {4g..4g+3, 16+4g..16+4g+3}.  ds_read_b64_tr_b16 hands
  // lane 4q+m of each 16-lane group element m of the 8-byte pieces addressed
  // by lanes q, q+4, q+8, q+12; pointing lane i at key base + i/4, dims
  // 16 dt + 4 (i%4) therefore delivers 4 consecutive keys of dim l16.  The
  // four reads of a key block are issued together from inline assembly with
  // their own wait: the compiler cannot tell them apart from the copies into
  // the other buffer and would otherwise wait for those first.  The row-end
  // wait and barrier make the buffer being read complete.
  auto v_frags = [&](const bf16* Vr, int kb, bf16x8& f0, bf16x8& f1) {
    // key kk and kk + 16 share (kk >> 2) & 3 = g, hence the same swizzle
    const int kk = kb * 32 + 4 * g + (l16 >> 2), q = l16 & 3;
    const int off0 = ((q >> 1) ^ g) * 8 + (q & 1) * 4;         // dims 4q .. 4q+3 (dim group q/2)
    const int off1 = (((q >> 1) + 2) ^ g) * 8 + (q & 1) * 4;   // dims 16 + 4q ..
    const uint32_t a0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)(Vr + kk * D + off0);
    const uint32_t a1 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)(Vr + kk * D + off1);
    uint2 lo0, hi0, lo1, hi1;                     // dims 0-15 (keys +0, +16), dims 16-31
    asm volatile(
        "ds_read_b64_tr_b16 %0, %4\n"
        "ds_read_b64_tr_b16 %1, %4 offset:1024\n"
        "ds_read_b64_tr_b16 %2, %5\n"
        "ds_read_b64_tr_b16 %3, %5 offset:1024\n"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(lo0), "=&v"(hi0), "=&v"(lo1), "=&v"(hi1)
        : "v"(a0), "v"(a1)
        : "memory");
    const uint32_t w0[4] = {lo0.x, lo0.y, hi0.x, hi0.y}, w1[4] = {lo1.x, lo1.y, hi1.x, hi1.y};
    f0 = __builtin_bit_cast(bf16x8, w0);
    f1 = __builtin_bit_cast(bf16x8, w1);
  };

  const int jw = j0 + 16 * wave + l16;          // this lane's query
  const bool wave_has_queries = wave < nqt && j0 + 16 * wave < n;
  const bool qvalid = jw < n;
  const int r0 = rg * kAttnRG, r1 = min(n, r0 + kAttnRG);
  bf16x8 qf = qvalid ? *reinterpret_cast<const bf16x8*>(p.q + (cu + (int64_t)r0 * sr + (int64_t)jw * st) * p.ld_qkv + h * D + g * 8)
                     : bf16x8{};
  __syncthreads();                              // bias slice staged
  // lane's bias: query 16*wave + l16, keys 16*kt + 4g .. +3 of every key tile
  uint2 bias_r[KT16];
#pragma unroll
  for (int kt = 0; kt < KT16; ++kt)
    bias_r[kt] = kt * 16 < npad ? *reinterpret_cast<const uint2*>(&Bs[(16 * wave + l16) * p.bstride + kt * 16 + 4 * g])
                                : make_uint2(0u, 0u);
  __syncthreads();                              // staging area free for keys and values
  dma_kv(r0, Kb0, Vb0);
  __builtin_amdgcn_s_waitcnt(0);                // this wave's copies have landed
  __syncthreads();

  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (bf16)1.f;
  const float c = p.scale_log2;                 // scale * log2(e)
  for (int r = r0; r < r1; ++r) {
    const bool odd = (r - r0) & 1;
    const bf16* Kb = odd ? Kb1 : Kb0;
    const bf16* Vb = odd ? Vb1 : Vb0;
    const bool more = r + 1 < r1;
    bf16x8 qn = qf;
    if (more) {
      dma_kv(r + 1, odd ? Kb0 : Kb1, odd ? Vb0 : Vb1);
      if (qvalid) qn = *reinterpret_cast<const bf16x8*>(p.q + (cu + (int64_t)(r + 1) * sr + (int64_t)jw * st) * p.ld_qkv + h * D + g * 8);
    }
    // keep the bias packed: converting it once outside the row loop would
    // double its registers
#pragma unroll
    for (int kt = 0; kt < KT16; ++kt) asm volatile("" : "+v"(bias_r[kt].x), "+v"(bias_r[kt].y));
    if (wave_has_queries) {
      float m_s = -INFINITY;                      // running max of bias/scale + q.k
      f32x4 O[3];                                 // dims 0-15, 16-31, row sum
#pragma unroll
      for (int u = 0; u < 3; ++u) O[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ci = 0; ci < NMAX / 64; ++ci) {
        const int kc = ci * 64;
        if (kc >= n) break;
        const bool tail = kc + 64 > n;
        const int ntile = (tail && n - kc <= 32) ? 2 : 4;   // a short tail takes half a chunk
        f32x4 sacc[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          if (kt >= ntile) break;
          const uint2 bb = bias_r[ci * 4 + kt];
          sacc[kt] = f32x4{__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xffff0000u),
                           __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xffff0000u)};
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Kb[(ci * 4 + kt) * 512 + lane * 8]);
          sacc[kt] = mfma16(kf, qf, sacc[kt]);
        }
        if (tail) {
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii)
              if (kt >= ntile || kc + kt * 16 + 4 * g + ii >= n) sacc[kt][ii] = -INFINITY;
        }
        float mloc = fmaxf(fmaxf(sacc[0][0], sacc[0][1]), fmaxf(sacc[0][2], sacc[0][3]));
#pragma unroll
        for (int kt = 1; kt < 4; ++kt) {
          if (kt >= ntile) break;
          mloc = fmaxf(mloc, fmaxf(fmaxf(sacc[kt][0], sacc[kt][1]), fmaxf(sacc[kt][2], sacc[kt][3])));
        }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
        // the reference max moves only when some query's max grew by more
        // than 8 (log2 units): probabilities then stay below 2^8, and most
        // chunks skip rescaling the accumulators
        if (__any((mloc - m_s) * c > 8.f)) {
          const float m_new = fmaxf(m_s, mloc);
          const float alpha = __builtin_amdgcn_exp2f((m_s - m_new) * c);
          m_s = m_new;
#pragma unroll
          for (int u = 0; u < 3; ++u) O[u] *= alpha;
        }
        const float nm = -m_s * c;
        bf16x8 pf[2];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          if (kt >= ntile) break;
#pragma unroll
          for (int ii = 0; ii < 4; ++ii)
            pf[kt >> 1][(kt & 1) * 4 + ii] = (bf16)__builtin_amdgcn_exp2f(fmaf(sacc[kt][ii], c, nm));
        }
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          if (2 * pp >= ntile) break;
          const int kb = ci * 2 + pp;
          bf16x8 vf0, vf1;
          v_frags(Vb, kb, vf0, vf1);
          O[0] = mfma16(vf0, pf[pp], O[0]);
          O[1] = mfma16(vf1, pf[pp], O[1]);
          O[2] = mfma16(ones, pf[pp], O[2]);
        }
      }
      if (qvalid) {
        const float inv = 1.f / O[2][0];
        bf16* orow = p.o + (cu + (int64_t)r * sr + (int64_t)jw * st) * p.ld_o + h * D;
#pragma unroll
        for (int dt = 0; dt < 2; ++dt) {
          bf16x4 ov;
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) ov[ii] = (bf16)(O[dt][ii] * inv);
          *reinterpret_cast<bf16x4*>(orow + dt * 16 + 4 * g) = ov;
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);              // copies for the next row have landed
    __syncthreads();
    qf = qn;
  }
}

// ---------------------------------------------------------------- fp32 path
struct AttnF32Args {
  int axis, H;
  const float* q;
  const float* k;
  const float* v;
  int64_t ld_qkv;
  const float* bias;
  int64_t ld_bias;
  float scale;
  float* o;
  int64_t ld_o;
  const int32_t* work;
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
};

// Exact two-pass softmax per query in fp32: one thread per query.
template <int D>
__global__ void __launch_bounds__(256) attention_f32_kernel(AttnF32Args p) {
  Seg sg;
  if (!segment_of(p, sg)) return;
  const int h = blockIdx.y, n = sg.n;
  for (int qi = sg.q_begin + (int)threadIdx.x; qi < sg.q_end; qi += 256) {
    const int64_t qrow = sg.base + (int64_t)qi * sg.step;
    float qv[D];
#pragma unroll
    for (int d = 0; d < D; ++d) qv[d] = p.q[qrow * p.ld_qkv + h * D + d];
    const float* brow = p.bias ? p.bias + (int64_t)h * p.ld_bias + sg.cu + (p.axis == 0 ? (int64_t)qi * n : qi) : nullptr;
    auto logit = [&](int key) {
      const int64_t krow = sg.base + (int64_t)key * sg.step;
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) s = fmaf(qv[d], p.k[krow * p.ld_qkv + h * D + d], s);
      s *= p.scale;
      if (brow) s += brow[p.axis == 0 ? (int64_t)key : (int64_t)key * n];
      return s;
    };
    float mx = -INFINITY;
    for (int key = 0; key < n; ++key) mx = fmaxf(mx, logit(key));
    float sum = 0.f, acc[D];
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] = 0.f;
    for (int key = 0; key < n; ++key) {
      const float e = expf(logit(key) - mx);
      sum += e;
      const int64_t krow = sg.base + (int64_t)key * sg.step;
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] = fmaf(e, p.v[krow * p.ld_qkv + h * D + d], acc[d]);
    }
#pragma unroll
    for (int d = 0; d < D; ++d) p.o[qrow * p.ld_o + h * D + d] = acc[d] / sum;
  }
}

}  // namespace

hipError_t launch_attention(const nt_layout& L, int axis, int H, int D, const void* q, const void* k,
                            const void* v, int64_t ld_qkv, const void* bias, int64_t ld_bias, float scale,
                            void* o, int64_t ld_o, nt_dtype dtype, hipStream_t s) {
  const int32_t* work = axis == 2 ? L.d_seq_work : L.d_attn_work;
  const int64_t items = axis == 2 ? L.seq_items() : L.attn_items();
  if (items == 0) return hipSuccess;
  const dim3 grid((unsigned)items, (unsigned)H), block(256);
  if (dtype == NT_F32) {
    AttnF32Args a{axis, H, (const float*)q, (const float*)k, (const float*)v, ld_qkv, (const float*)bias,
                  ld_bias, scale, (float*)o, ld_o, work, L.d_cu_seqlens, L.d_cu_pairs};
    switch (D) {
      case 8: attention_f32_kernel<8><<<grid, block, 0, s>>>(a); break;
      case 16: attention_f32_kernel<16><<<grid, block, 0, s>>>(a); break;
      case 32: attention_f32_kernel<32><<<grid, block, 0, s>>>(a); break;
      case 64: attention_f32_kernel<64><<<grid, block, 0, s>>>(a); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int npad = (L.max_len + 63) & ~63;
  if (D == 32 && axis != 2 && L.max_len <= kAttnLongLen) {
    if (L.pattn_items() == 0) return hipSuccess;
    const int nmax = L.max_len <= kAttnShortLen ? kAttnShortLen : kAttnLongLen;
    // bias rows: 8-byte fragment reads are conflict-free with a row stride of 2 (mod 4) dwords
    const int bstride = nmax + 4;
    PairAttnArgs a{axis, (const bf16*)q, (const bf16*)k, (const bf16*)v, ld_qkv, (const bf16*)bias, ld_bias,
                   scale * kLog2e, (bf16*)o, ld_o, L.d_pattn_work, L.d_cu_seqlens, L.d_cu_pairs, bstride,
                   1.f / scale, H};
    const size_t smem = sizeof(bf16) * std::max((size_t)kAttnQB * bstride, 4 * (size_t)nmax * 32);
    const dim3 grid((unsigned)(L.pattn_items() * H));
    const void* fn = nmax == kAttnShortLen ? (const void*)attention_pair_kernel<kAttnShortLen>
                                          : (const void*)attention_pair_kernel<kAttnLongLen>;
    hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (nmax == kAttnShortLen)
      attention_pair_kernel<kAttnShortLen><<<grid, dim3(512), smem, s>>>(a);
    else
      attention_pair_kernel<kAttnLongLen><<<grid, dim3(512), smem, s>>>(a);
    return hipGetLastError();
  }
  const int vstride = (npad + 127) / 128 * 128 + 4;
  AttnArgs a{axis, H, (const bf16*)q, (const bf16*)k, (const bf16*)v, ld_qkv, (const bf16*)bias, ld_bias,
             scale * kLog2e, (bf16*)o, ld_o, work, L.d_cu_seqlens, L.d_cu_pairs, vstride};
  const size_t smem = sizeof(bf16) * ((size_t)npad * (D + 8) + (size_t)D * vstride);
  if (D == 32) {
    if (smem > 65536) hipFuncSetAttribute((const void*)attention_mfma_kernel<32>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attention_mfma_kernel<32><<<grid, block, smem, s>>>(a);
  } else if (D == 64) {
    if (smem > 65536) hipFuncSetAttribute((const void*)attention_mfma_kernel<64>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attention_mfma_kernel<64><<<grid, block, smem, s>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace nt
