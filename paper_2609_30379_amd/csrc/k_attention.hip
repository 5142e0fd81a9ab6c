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
#include <type_traits>

#include <mutex>

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
  int64_t ld_bias, ld_bias_head;  // element (cell c, head h) at c * ld_bias + h * ld_bias_head
  float scale_log2;      // softmax scale * log2(e)
  bf16* o;
  int64_t ld_o;
  const int32_t* work;   // (sample, row) or (sample, query block) pairs
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  int vstride;           // LDS row stride of V^T (elements)
  const bf16* gate;      // NULL, or o = sigmoid(gate) * attention (gate row stride ld_gate)
  int64_t ld_gate;
};

struct Seg {
  int n;                 // keys in the segment
  int64_t base, step;    // packed row of element t: base + t * step
  int q_begin, q_end;
  int64_t cu;            // pair offset of the sample (bias addressing)
  int sample;
};

template <typename A>
__device__ __forceinline__ bool segment_of(const A& p, Seg& s) {
  const int i = p.work[2 * blockIdx.x], r = p.work[2 * blockIdx.x + 1];
  if (i < 0) return false;
  s.sample = i;
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
    if (p.bias && qvalid)
      brow = p.bias + (int64_t)h * p.ld_bias_head + (sg.cu + (p.axis == 0 ? (int64_t)qi * n : qi)) * p.ld_bias;
    const int64_t bstep = (p.axis == 0 ? 1 : n) * p.ld_bias;

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
        for (int i = 0; i < 4; ++i) {
          float val = O[dt][i] * inv;
          if (p.gate) {
            const float gl = (float)p.gate[qrow * p.ld_gate + h * D + dt * 16 + 4 * g + i];
            val *= __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-gl * kLog2e));
          }
          ov[i] = (bf16)val;
        }
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
  int64_t ld_bias, ld_bias_head;
  float scale_log2;
  bf16* o;
  int64_t ld_o;
  const int32_t* work;   // quads (sample, first 16-query tile, row group, tile count)
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  int H;                 // heads (interleaved in the grid)
  const uint2* bias_img; // bias image (see bias_image_kernel) or NULL for no bias
  int64_t img_head;      // uint2 entries per head of the image
  const int32_t* bias_tiles;
  int batch;             // samples (persistent instance: rows are found from cu_seqlens)
  int64_t total_rows;    // sum of N_i (persistent instance)
  const bf16* gate;      // gated output: o = sigmoid(gate) * attention, gate [rows, >= H*D] (GATE instances)
  int64_t ld_gate;
};

// Pair bias image: for head h, sample i, 16-query tile qt and 16-key tile kt
// (kt < round_up(N_i,64)/16), lane l = l16 + 16 g of tile
// ((h * T + bias_tiles[i] + qt * KT_i + kt) holds the four values
// bias(j, k) / scale, j = 16 qt + l16, k = 16 kt + 4 g .. +3, each rounded to
// bf16 -- exactly the register image the attention lanes keep.  Keys past N
// hold -inf (for queries inside N), so the scores they seed are masked
// without further work; queries past N hold 0.
// bias(j, k) is the head-h bias of cell(j, k) for axis 0 and of cell(k, j)
// for axis 1, read at cell * ld_bias + h * ld_bias_head.  One wave per tile,
// the sample found by bisection.
struct BiasImgArgs {
  int axis, batch;
  const bf16* bias;
  int64_t ld_bias, ld_bias_head;
  float inv_scale;
  uint2* img;
  int64_t tiles;          // tiles per head
  const int32_t* bias_tiles;
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
};

__global__ void __launch_bounds__(256) bias_image_kernel(BiasImgArgs p) {
  const int64_t tile = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tile >= p.tiles) return;
  const int h = blockIdx.y, lane = threadIdx.x & 63, l16 = lane & 15, g = lane >> 4;
  int lo = 0, hi = p.batch - 1;                 // sample: largest i with bias_tiles[i] <= tile
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.bias_tiles[mid] <= tile) lo = mid; else hi = mid - 1;
  }
  const int i = lo;
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  const int kti = ((n + 63) >> 6) * 4;
  const int t = (int)(tile - p.bias_tiles[i]);
  const int j = (t / kti) * 16 + l16, k0 = (t % kti) * 16 + 4 * g;
  const bf16* bh = p.bias + (int64_t)h * p.ld_bias_head + (int64_t)p.cu_pairs[i] * p.ld_bias;
  bf16x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int k = k0 + e;
    float b = j < n ? -INFINITY : 0.f;
    if (j < n && k < n) b = (float)bh[(p.axis != 1 ? (int64_t)j * n + k : (int64_t)k * n + j) * p.ld_bias] * p.inv_scale;
    o[e] = (bf16)b;
  }
  *reinterpret_cast<bf16x4*>(&p.img[(int64_t)h * p.tiles * 64 + tile * 64 + lane]) = o;
}

// ---------------------------------------------------------------- shared pieces
// Value rows of 32 dims (64 bytes) staged row-major, the 16-byte piece at
// column c of key row kv holding dim group c ^ ((kv >> 2) & 3) (so the four
// key groups of a transposed read fall on different banks).  Fragments for
// O^T += V^T P^T: lane (dim 16 dt + l16, k-group g) needs keys 32 kb +
// {4g..4g+3, 16+4g..16+4g+3}.  ds_read_b64_tr_b16 hands lane 4q+m of each
// 16-lane group element m of the 8-byte pieces addressed by lanes q, q+4,
// q+8, q+12; pointing lane i at key base + i/4, dims 16 dt + 4 (i%4)
// therefore delivers 4 consecutive keys of dim l16.  Key blocks are 2 KB
// apart and keys kk, kk + 16 share (kk >> 2) & 3 = g, so every read of a lane
// uses the same swizzled column.  The reads of one or two key blocks are
// issued together from inline assembly with their own wait: the compiler
// cannot tell them apart from global->LDS copies in flight into other
// buffers and would otherwise wait for those first.
struct VtLane {
  uint32_t a0, a1;       // byte offsets in a value buffer, key block 0: dims 4q.., 16 + 4q..
};
__device__ __forceinline__ VtLane vt_lane(int l16, int g) {
  const int kk = 4 * g + (l16 >> 2), q = l16 & 3;
  return VtLane{(uint32_t)((kk * 32 + ((q >> 1) ^ g) * 8 + (q & 1) * 4) * 2),
                (uint32_t)((kk * 32 + (((q >> 1) + 2) ^ g) * 8 + (q & 1) * 4) * 2)};
}
__device__ __forceinline__ uint32_t lds_addr(const bf16* ptr) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)ptr;
}
// bf16 ones as an MFMA operand, materialised where it is used: kept live
// across the row loop it is one of the first values the register allocator
// spills, and its reload waits for every copy in flight.
__device__ __forceinline__ bf16x8 ones_bf16x8() {
  uint32_t w;
  asm volatile("v_mov_b32 %0, 0x3f803f80" : "=v"(w));
  const uint32_t q[4] = {w, w, w, w};
  return __builtin_bit_cast(bf16x8, q);
}
// an opaque copy of a lane-dependent value: what is derived from it is
// recomputed at each use instead of being hoisted out of the row loop and
// kept live (or spilled) across it
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ bf16x8 pack_u2(uint2 lo, uint2 hi) {
  const uint32_t w[4] = {lo.x, lo.y, hi.x, hi.y};
  return __builtin_bit_cast(bf16x8, w);
}
// one key block: f[0] dims 0-15, f[1] dims 16-31
__device__ __forceinline__ void vt_frags1(const bf16* Vr, int kb, const VtLane& vl, bf16x8 (&f)[2]) {
  const uint32_t base = lds_addr(Vr + kb * 32 * 32), a0 = base + vl.a0, a1 = base + vl.a1;
  uint2 r[4];
  asm volatile(
      "ds_read_b64_tr_b16 %0, %4\n"
      "ds_read_b64_tr_b16 %1, %4 offset:1024\n"
      "ds_read_b64_tr_b16 %2, %5\n"
      "ds_read_b64_tr_b16 %3, %5 offset:1024\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
      : "v"(a0), "v"(a1)
      : "memory");
  f[0] = pack_u2(r[0], r[1]);
  f[1] = pack_u2(r[2], r[3]);
}
// two key blocks kb, kb + 1: f[0..1] as above for kb, f[2..3] for kb + 1
__device__ __forceinline__ void vt_frags2(const bf16* Vr, int kb, const VtLane& vl, bf16x8 (&f)[4]) {
  const uint32_t base = lds_addr(Vr + kb * 32 * 32), a0 = base + vl.a0, a1 = base + vl.a1;
  uint2 r[8];
  asm volatile(
      "ds_read_b64_tr_b16 %0, %8\n"
      "ds_read_b64_tr_b16 %1, %8 offset:1024\n"
      "ds_read_b64_tr_b16 %2, %9\n"
      "ds_read_b64_tr_b16 %3, %9 offset:1024\n"
      "ds_read_b64_tr_b16 %4, %8 offset:2048\n"
      "ds_read_b64_tr_b16 %5, %8 offset:3072\n"
      "ds_read_b64_tr_b16 %6, %9 offset:2048\n"
      "ds_read_b64_tr_b16 %7, %9 offset:3072\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
      : "v"(a0), "v"(a1)
      : "memory");
  f[0] = pack_u2(r[0], r[1]);
  f[1] = pack_u2(r[2], r[3]);
  f[2] = pack_u2(r[4], r[5]);
  f[3] = pack_u2(r[6], r[7]);
}
// maximum over the four lanes l16 + 16 g holding one query: the swaps pair
// lane l with l ^ 16, then with l ^ 32, and leave both values in place
__device__ __forceinline__ float query_max(float v) {
  const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
  const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
}

// key-split hand-over: 10 floats per lane of 8 query slots
constexpr int kAttnHandBytes = 10 * 8 * 64 * 4;
constexpr int kAttnGateBytes = 16 * 1024;        // gate slots: 16 waves x 1 KB (8 when the keys are split)

// ---------------------------------------------------------------- pair attention, head_dim 32
// Pair attention for head_dim 32 and N_i <= kAttnLongLen, organised so that
// the exponentials are nearly the only vector work.  A workgroup of NW waves
// runs a stretch of pair rows of one head, a block of up to 16 NW queries:
//   * the bias of (query, key) does not depend on the pair row, so each lane
//     keeps the bias of its query for its 4-key groups of every key tile in
//     registers while the rows belong to one sample -- read from the bias
//     image, already divided by the softmax scale (one bf16 rounding) -- and
//     it seeds the score accumulators: the matrix cores produce
//     bias/scale + q.k directly;
//   * keys and values of a row are copied straight into LDS (keys as fragment
//     images: 64 lanes x 16 bytes, read as one contiguous 1 KB per wave) in
//     two buffers, the next row's copies in flight while the current row
//     runs: one barrier per row;
//   * the softmax denominator comes from one more matrix-core product with a
//     ones operand, on the same bf16 probabilities as the numerator.
// Scores are kept transposed (S^T = K Q^T), so a lane holds 16 keys of one
// query per 64-key chunk and the running max is mostly lane-local.
// Instances:
//   * N <= 256, persistent, with 16 waves (all queries of a row in one
//     workgroup, so a row's keys and values are copied once per CU; 64 KB of
//     LDS, four waves per SIMD, one workgroup per CU with an equal share of
//     the rows);
//   * N <= 512, key split (KS): 16 waves from a work list of (sample, query
//     block, group of 16 rows) items.  A sample longer than 256 splits its
//     keys between wave pairs: waves w and w + 8 hold the same 16 queries,
//     one the keys below the cut (half the row rounded up to 32 keys) and
//     the other the rest, each with the bias registers of at most 16 key
//     tiles (as the N <= 256 instance), and the second
//     hands its running maximum and accumulators to the first through LDS,
//     which merges them (rescaled to the larger maximum) and stores the row;
//     a block then holds 8 query tiles.  Shorter samples use all 16 waves as
//     query tiles.  128 KB of key/value buffers and 20 KB for the hand-over
//     (the gated instance adds 8 KB of gate rows) keep one workgroup per CU
//     at four waves per SIMD;
//   * N <= 512, 8 waves, each wave all keys (the single attention of axis 3,
//     one row per sample).
template <int NMAX, int NW, bool PERSIST, bool GATE = false, bool KS = false>
__global__ void __launch_bounds__(64 * NW, (NMAX <= 256 || KS) ? 4 : 2) attention_pair_kernel(PairAttnArgs p) {
  constexpr int D = 32;
  constexpr int KT16 = NMAX / 16;               // key tiles
  constexpr int BT = KS ? 16 : KT16;            // key tiles of bias kept per lane
  static_assert(!PERSIST || NW * 16 >= NMAX, "the persistent instance covers all queries of a row");
  static_assert(!KS || (NMAX == 512 && NW == 16 && !PERSIST), "the key-split instance: 16 waves, N <= 512");
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  bf16* Kb0 = lds;                                         // key images: tile of 16 keys -> 512 elements
  bf16* Kb1 = Kb0 + NMAX * D;
  bf16* Vb0 = Kb1 + NMAX * D;                              // values, row-major [key][D]
  bf16* Vb1 = Vb0 + NMAX * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;

  // ---- rows of this workgroup: packed rows [row, row_end) of one head, a
  // query block starting at tile qt0.
  //   * work-list instance: workgroup 8 (H k + h) + x runs on XCD x and takes
  //     work position pos = 8 k + x, head h: the H heads of a position are
  //     consecutive workgroups of one XCD, so they read the same q|k|v cache
  //     lines at about the same time; rows of one sample only.
  //   * persistent instance (one workgroup per CU): XCD x takes the x-th
  //     eighth of all packed rows, and its workgroups split that range among
  //     the heads, workgroup k taking head k % H and the (k / H)-th of the
  //     equal slices of that head, so every CU gets the same number of rows
  //     (crossing sample boundaries) and the heads of a row still run on one
  //     XCD together.
  int h, i, qt0, nqt_w = 0;
  int64_t row, row_end;
  bool split = false;                           // key split between wave pairs (KS, N > 256)
  if constexpr (PERSIST) {
    const int x = blockIdx.x % kXcds, k = blockIdx.x / kXcds, per = (int)(gridDim.x / kXcds);
    h = k % p.H;
    const int m = k / p.H, M = (per - h + p.H - 1) / p.H;
    const int64_t xa = p.total_rows * x / kXcds, xb = p.total_rows * (x + 1) / kXcds;
    row = xa + (xb - xa) * m / M;
    row_end = xa + (xb - xa) * (m + 1) / M;
    if (row >= row_end) return;
    int lo = 0, hi = p.batch;                   // cu_seqlens[lo] <= row < cu_seqlens[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.cu_seqlens[mid] <= row) lo = mid;
      else hi = mid;
    }
    i = __builtin_amdgcn_readfirstlane(lo);
    qt0 = 0;
  } else {
    const int x = blockIdx.x % kXcds, t = blockIdx.x / kXcds;
    h = t % p.H;
    const int pos = (t / p.H) * kXcds + x;
    const int4 w4 = reinterpret_cast<const int4*>(p.work)[pos];
    i = w4.x;
    if (i < 0) return;
    qt0 = w4.y;
    const int nn = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
    const int r0 = w4.z * kAttnRG;
    row = p.cu_seqlens[i] + r0;
    row_end = p.axis == 3 ? row + 1 : p.cu_seqlens[i] + min(nn, r0 + kAttnRG);   // axis 3: one row per sample
    nqt_w = w4.w;
    if constexpr (KS) split = nn > 256;
  }
  // query slot and key half of this wave (key split: waves w, w + 8 share slot w % 8)
  const int qs = __builtin_amdgcn_readfirstlane(KS && split ? wave & 7 : wave);
  const int kh = __builtin_amdgcn_readfirstlane(KS && split ? wave >> 3 : 0);
  const int j0 = qt0 * 16;
  const int jw = j0 + 16 * qs + l16;            // this lane's query
  // gate rows of this wave (gated key-split instance): 1 KB slots after the
  // key/value buffers, past the hand-over when the keys are split
  bf16* gslot = lds + 4 * NMAX * D + (split ? kAttnHandBytes / 2 : 0) + qs * 512;

  // ---- per-row staging: straight global -> LDS copies ---------------------
  // Each wave copies its key tiles (wave, wave + NW, ...; 16 keys each) with
  // global_load_lds, lane l's 16 bytes landing at byte 16 l of the tile:
  //   keys as fragment images: lane l = (key l%16, dims 8 (l/16) ..),
  //   values row-major [key][32]: lane l = (key l/4, dims 8 (l%4) ..).
  // Every tile below the 64-key padded length is written (the last chunk
  // reads up to there): keys past N repeat key N-1, so the padding holds
  // finite values whose probabilities are masked to zero.
  // this head's queries, keys, values, outputs (and gates): the head offset
  // as a scalar, so the bases stay in scalar registers (global pointers)
  const int hD = __builtin_amdgcn_readfirstlane(h * D);
  const bf16* kbase = p.k + hD;
  const bf16* vbase = p.v + hD;
  const bf16* qbase = p.q + hD;
  bf16* obase = p.o + hD;
  const bf16* gbase = GATE ? p.gate + hD : nullptr;
  auto dma_kv = [&](int sn, int64_t scu, int r, bf16* Kb, bf16* Vr) {
    const int snpad = (sn + 63) & ~63;
    const int64_t ssr = p.axis == 0 ? sn : (p.axis == 1 ? 1 : 0), sst = p.axis == 1 ? sn : 1;
    const int ln = opaque(lane);
#pragma unroll
    for (int kt = wave; kt < KT16; kt += NW) {
      if (kt * 16 >= snpad) break;
      // values: the 16-byte chunk at column c of key row kv holds dim group
      // c ^ ((kv >> 2) & 3), so the four key groups of a transpose read fall
      // on different banks
      const int kv = kt * 16 + (ln >> 2);
      const int key_k = min(kt * 16 + (ln & 15), sn - 1), key_v = min(kv, sn - 1);
      const int dgv = (ln & 3) ^ ((kv >> 2) & 3);
      const bf16* sk = kbase + (scu + (int64_t)r * ssr + (int64_t)key_k * sst) * p.ld_qkv + (ln >> 4) * 8;
      const bf16* sv = vbase + (scu + (int64_t)r * ssr + (int64_t)key_v * sst) * p.ld_qkv + dgv * 8;
      __builtin_amdgcn_global_load_lds((const void*)sk, (__attribute__((address_space(3))) void*)(Kb + kt * 512), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)sv, (__attribute__((address_space(3))) void*)(Vr + kt * 512), 16, 0, 0);
    }
  };
  // query fragment of this lane for row r of a sample with sn elements at
  // pair offset scu (zero past N)
  auto load_q = [&](int sn, int64_t scu, int r) -> bf16x8 {
    if (jw >= sn) return bf16x8{};
    const int64_t ssr = p.axis == 0 ? sn : (p.axis == 1 ? 1 : 0), sst = p.axis == 1 ? sn : 1;
    return *reinterpret_cast<const bf16x8*>(qbase + (scu + (int64_t)r * ssr + (int64_t)jw * sst) * p.ld_qkv + g * 8);
  };
  const VtLane vl = vt_lane(l16, g);
  auto v_frags1 = [&](const bf16* Vr, int kb, bf16x8 (&f)[2]) { vt_frags1(Vr, kb, vl, f); };
  auto v_frags2 = [&](const bf16* Vr, int kb, bf16x8 (&f)[4]) { vt_frags2(Vr, kb, vl, f); };

  // ---- per-sample state ------------------------------------------------------
  int n = 0;
  int64_t cu = 0, sr = 0, st = 0;               // cell(r, t) = cu + r*sr + t*st
  bool wave_has_queries = false, qvalid = false;
  // keys of this wave: [16 kto, kend).  A split row is cut at half its
  // length rounded up to 32 keys (at most 256 on either side), so both waves
  // of a pair run about the same number of key tiles.
  int kto = 0, kend = 0;
  // lane's bias: query 16*wave + l16, keys 16*kt + 4g .. +3 of every key
  // tile, read from the bias image (one contiguous 512 bytes per wave and tile)
  uint2 bias_r[BT];
  auto set_sample = [&](int si, int sn, int64_t scu) {
    n = sn;
    cu = scu;
    sr = p.axis == 0 ? n : (p.axis == 1 ? 1 : 0);
    st = p.axis == 1 ? n : 1;
    wave_has_queries = qs < (PERSIST ? (n + 15) / 16 : nqt_w) && j0 + 16 * qs < n;
    qvalid = jw < n;
    if (KS && split) {
      const int cut = __builtin_amdgcn_readfirstlane(min(n, ((n + 1) / 2 + 31) & ~31));
      kto = kh ? cut / 16 : 0;
      kend = kh ? n : cut;
    } else {
      kto = 0;
      kend = n;
    }
    const int kti = ((n + 63) & ~63) / 16;
    const uint2* img = p.bias_img && wave_has_queries
                           ? p.bias_img + h * p.img_head + ((int64_t)p.bias_tiles[si] + (int64_t)(qt0 + qs) * kti) * 64 + lane
                           : nullptr;
#pragma unroll
    for (int kt = 0; kt < BT; ++kt) {
      const int kk = kto + kt;                  // key tile of this wave's half
      bias_r[kt] = img && kk < kti ? img[kk * 64] : make_uint2(0u, 0u);
    }
  };
  // first cell of the sample: pair offset, or for axis 3 its first token
  set_sample(i, __builtin_amdgcn_readfirstlane(p.cu_seqlens[i + 1] - p.cu_seqlens[i]),
             p.axis == 3 ? p.cu_seqlens[i] : p.cu_pairs[i]);
  int r = __builtin_amdgcn_readfirstlane((int)(row - p.cu_seqlens[i]));
  bf16x8 qf = load_q(n, cu, r);
  dma_kv(n, cu, r, Kb0, Vb0);
  __builtin_amdgcn_s_waitcnt(0);                // this wave's copies have landed
  __syncthreads();

  const float c = p.scale_log2;                 // scale * log2(e)
  bool odd = false;
  for (; row < row_end; ++row) {
    const bf16* Kb = odd ? Kb1 : Kb0;
    const bf16* Vb = odd ? Vb1 : Vb0;
    const bool more = row + 1 < row_end;
    // the next row: same sample, or the first row of the next non-empty one
    // (sample extents are read only when the sample changes: a global load
    // here would make the wave wait for every copy and store in flight)
    int i2 = i, r2 = r + 1, n2 = n;
    int64_t cu2 = cu;
    if (more && r2 >= n) {
      i2 = i + 1;
      while (p.cu_seqlens[i2 + 1] <= row + 1) ++i2;
      r2 = 0;
      n2 = p.cu_seqlens[i2 + 1] - p.cu_seqlens[i2];
      cu2 = p.axis == 3 ? p.cu_seqlens[i2] : p.cu_pairs[i2];
    }
    i2 = __builtin_amdgcn_readfirstlane(i2);
    r2 = __builtin_amdgcn_readfirstlane(r2);
    n2 = __builtin_amdgcn_readfirstlane(n2);
    cu2 = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(cu2 >> 32)) << 32) |
                    (uint32_t)__builtin_amdgcn_readfirstlane((int)cu2));
    // gate of this lane's outputs (GATE): issued before the next row's
    // copies, so waiting for it leaves those in flight; the query index is
    // clamped into the row, so the load is unconditional
    // (key-split instance: the wave's 16 gate rows are copied into its LDS
    // slot, lane l taking dims 8 (l % 4) .. +7 of query l / 4; held in
    // registers across the row they were spilled, and each reload waited for
    // the copies in flight mid-row)
    uint2 gt[2];
    if constexpr (GATE && KS) {
      if (wave_has_queries && kh == 0) {
        const int lq = opaque(lane);
        const int jq = min(j0 + 16 * qs + (lq >> 2), n - 1);
        const bf16* gr = gbase + (cu + (int64_t)r * sr + (int64_t)jq * st) * p.ld_gate + 8 * (lq & 3);
        __builtin_amdgcn_global_load_lds((const void*)gr, (__attribute__((address_space(3))) void*)gslot, 16, 0, 0);
      }
    } else if constexpr (GATE) {
      if (wave_has_queries && kh == 0) {
        const bf16* gr = gbase + (cu + (int64_t)r * sr + (int64_t)min(jw, n - 1) * st) * p.ld_gate + 4 * g;
        gt[0] = *reinterpret_cast<const uint2*>(gr);
        gt[1] = *reinterpret_cast<const uint2*>(gr + 16);
      }
    }
    bf16x8 qn = qf;
    if (more) {
      dma_kv(n2, cu2, r2, odd ? Kb0 : Kb1, odd ? Vb0 : Vb1);
      qn = load_q(n2, cu2, r2);
    }
    // keep the bias packed: converting it once outside the row loop would
    // double its registers
#pragma unroll
    for (int kt = 0; kt < BT; ++kt) asm volatile("" : "+v"(bias_r[kt].x), "+v"(bias_r[kt].y));
    float m_s = -INFINITY;                        // running max of bias/scale + q.k
    f32x4 O[3];                                   // dims 0-15, 16-31, row sum
#pragma unroll
    for (int u = 0; u < 3; ++u) O[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (wave_has_queries) {
      // Keys in super-chunks of 128 (8 key tiles), the last one cut to the
      // 2, 4 or 6 tiles that hold keys: all score products of a super-chunk
      // are issued together, one maximum per query, then the exponentials
      // and the value products.  Tiles read stay below the staged length.
      // first key tile of this wave's half (key split), uniform
      const bf16* Kh = Kb + kto * 512;
      const bf16* Vh = Vb + kto * 512;
      auto super_chunk = [&](auto sc_c, auto nt_c) {
        constexpr int SC = decltype(sc_c)::value, NT = decltype(nt_c)::value;
        constexpr int T0 = SC * 8;                // first key tile (of this wave's half)
        const int kc = kto * 16 + SC * 128;
        f32x4 S[NT];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
          const uint2 bb = bias_r[T0 + kt];
          S[kt] = f32x4{__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xffff0000u),
                        __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xffff0000u)};
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Kh[(T0 + kt) * 512 + lane * 8]);
          S[kt] = mfma16(kf, qf, S[kt]);
          // at most four key fragments in flight (registers)
          if (kt % 4 == 3) __builtin_amdgcn_sched_barrier(0);
        }
        if (!p.bias_img && kc + NT * 16 > n) {    // keys past N (with a bias the image masks them)
#pragma unroll
          for (int kt = 0; kt < NT; ++kt)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii)
              if (kc + kt * 16 + 4 * g + ii >= n) S[kt][ii] = -INFINITY;
        }
        float mloc = S[0][0];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) mloc = fmaxf(mloc, S[kt][ii]);
        mloc = query_max(mloc);
        // the reference max moves only when some query's max grew by more
        // than 8 (log2 units): probabilities then stay below 2^8, and most
        // super-chunks skip rescaling the accumulators
        if (__any((mloc - m_s) * c > 8.f)) {
          const float m_new = fmaxf(m_s, mloc);
          const float alpha = __builtin_amdgcn_exp2f((m_s - m_new) * c);
          m_s = m_new;
#pragma unroll
          for (int u = 0; u < 3; ++u) O[u] *= alpha;
        }
        const float nm = -m_s * c;
        bf16x8 P[NT / 2];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int ii = 0; ii < 4; ++ii)
            P[kt >> 1][(kt & 1) * 4 + ii] = (bf16)__builtin_amdgcn_exp2f(fmaf(S[kt][ii], c, nm));
        const bf16x8 ones = ones_bf16x8();
#pragma unroll
        for (int pp = 0; pp + 1 < NT / 2; pp += 2) {
          bf16x8 vf[4];
          v_frags2(Vh, SC * 4 + pp, vf);
          O[0] = mfma16(vf[0], P[pp], O[0]);
          O[1] = mfma16(vf[1], P[pp], O[1]);
          O[2] = mfma16(ones, P[pp], O[2]);
          O[0] = mfma16(vf[2], P[pp + 1], O[0]);
          O[1] = mfma16(vf[3], P[pp + 1], O[1]);
          O[2] = mfma16(ones, P[pp + 1], O[2]);
        }
        if constexpr ((NT / 2) % 2 == 1) {
          bf16x8 vf[2];
          v_frags1(Vh, SC * 4 + NT / 2 - 1, vf);
          O[0] = mfma16(vf[0], P[NT / 2 - 1], O[0]);
          O[1] = mfma16(vf[1], P[NT / 2 - 1], O[1]);
          O[2] = mfma16(ones, P[NT / 2 - 1], O[2]);
        }
      };
      // keys left at super-chunk SC: more than 96 take all 8 tiles (the
      // staged length, a multiple of 64, then reaches 128 past kc)
      auto run_sc = [&](auto sc_c) {
        constexpr int SC = decltype(sc_c)::value;
        const int rem = kend - kto * 16 - SC * 128;
        if (rem <= 0) return;
        if (rem > 96) super_chunk(sc_c, std::integral_constant<int, 8>{});
        else if (rem > 64) super_chunk(sc_c, std::integral_constant<int, 6>{});
        else if (rem > 32) super_chunk(sc_c, std::integral_constant<int, 4>{});
        else super_chunk(sc_c, std::integral_constant<int, 2>{});
      };
      run_sc(std::integral_constant<int, 0>{});
      run_sc(std::integral_constant<int, 1>{});
      if constexpr (NMAX > 256 && !KS) {
        run_sc(std::integral_constant<int, 2>{});
        run_sc(std::integral_constant<int, 3>{});
      }
    }
    if constexpr (KS) {
      if (split) {
        // the upper key half hands (max, accumulators) to its partner, which
        // merges the two partial softmax sums rescaled to the larger maximum
        // [10][8 slots][64 lanes]: the maximum, dims 4g .. +3 and 16 + 4g .. +3,
        // and the denominator (the ones product gives it in all four elements)
        float* xf = reinterpret_cast<float*>(lds + 4 * NMAX * D);
        if (kh == 1 && wave_has_queries) {
          xf[(0 * 8 + qs) * 64 + lane] = m_s;
#pragma unroll
          for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) xf[((1 + 4 * u + ii) * 8 + qs) * 64 + lane] = O[u][ii];
          xf[(9 * 8 + qs) * 64 + lane] = O[2][0];
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);     // lgkmcnt(0): the hand-over is written (copies stay in flight)
        __builtin_amdgcn_s_barrier();
        if (kh == 0 && wave_has_queries) {
          const float m1 = xf[(0 * 8 + qs) * 64 + lane];
          const float mm = fmaxf(m_s, m1);
          const float a0 = __builtin_amdgcn_exp2f((m_s - mm) * c), a1 = __builtin_amdgcn_exp2f((m1 - mm) * c);
#pragma unroll
          for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) O[u][ii] = O[u][ii] * a0 + xf[((1 + 4 * u + ii) * 8 + qs) * 64 + lane] * a1;
          O[2][0] = O[2][0] * a0 + xf[(9 * 8 + qs) * 64 + lane] * a1;
        }
      }
    }
    if (wave_has_queries && kh == 0) {
      // lane (l16, g) holds dims 4g .. 4g+3 and 16 + 4g .. +3 of its query;
      // the rows g, g ^ 1 trade halves so that an even row holds dims
      // 4g .. 4g+7 and an odd one 16 + 4(g-1) .. +7: one 16-byte store per
      // lane instead of two 8-byte ones (each store instruction gathers 16
      // cells and holds the texture-address unit the copies also need)
      if constexpr (GATE && KS) {
        // the gate copy has landed (so have the next row's copies, which the
        // row end waits for anyway); lane (l16, g): dims 4g .. +3, 16 + 4g .. +3
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        const bf16* gl = gslot + l16 * 32 + 4 * g;
        gt[0] = *reinterpret_cast<const uint2*>(gl);
        gt[1] = *reinterpret_cast<const uint2*>(gl + 16);
      }
      const float inv = 1.f / O[2][0];
      uint32_t ow[2][2];
#pragma unroll
      for (int dt = 0; dt < 2; ++dt) {
        float gs[4] = {1.f, 1.f, 1.f, 1.f};
        if constexpr (GATE) {
          const float gl[4] = {__uint_as_float(gt[dt].x << 16), __uint_as_float(gt[dt].x & 0xffff0000u),
                               __uint_as_float(gt[dt].y << 16), __uint_as_float(gt[dt].y & 0xffff0000u)};
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) gs[ii] = __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-gl[ii] * kLog2e));
        }
        bf16x4 ov;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) ov[ii] = (bf16)(O[dt][ii] * inv * gs[ii]);
        const uint2 u = __builtin_bit_cast(uint2, ov);
        ow[dt][0] = u.x;
        ow[dt][1] = u.y;
      }
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        // odd rows of the first operand trade with even rows of the second
        const auto sw = __builtin_amdgcn_permlane16_swap(ow[0][e], ow[1][e], false, false);
        ow[0][e] = sw[0];
        ow[1][e] = sw[1];
      }
      if (qvalid) {
        bf16* orow = obase + (cu + (int64_t)r * sr + (int64_t)jw * st) * p.ld_o;
        const int d0 = (g & 1) ? 16 + 4 * (g - 1) : 4 * g;
        *reinterpret_cast<uint4*>(orow + d0) = make_uint4(ow[0][0], ow[0][1], ow[1][0], ow[1][1]);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);              // copies for the next row have landed
    __syncthreads();
    if (i2 != i) {                              // bias of the next sample
      set_sample(i2, n2, cu2);
      // landed before the back edge, so the loop head has no load pending
      // and waits for none of the next row's copies
      __builtin_amdgcn_s_waitcnt(0);
    }
    i = i2;
    r = r2;
    qf = qn;
    odd = !odd;
  }
}

// ---------------------------------------------------------------- 1-D attention, head_dim 32 / 64
// Variable-length attention over each sample's tokens (Sec. 3.3 "Attention
// through packed blocks"), head_dim D in {32, 64}, at most NMAX keys per
// sample.  Queries of sample i are rows cu_q[i] .. cu_q[i+1] and its keys and
// values rows cu_kv[i] .. cu_kv[i+1]: self-attention passes the same offsets
// twice; cross-attention passes the key structure separately, and the output
// takes the query structure (a query whose sample has no keys gets the empty
// sum, 0).  A workgroup of 8 waves takes (sample, block of up to 128 queries,
// head): all keys and values of the sample are copied global -> LDS once
// (32-dim halves: keys as fragment images, values row-major with the swizzle
// of the value reads), then each wave runs its 16 queries over 128-key
// super-chunks -- score products, one maximum per query, the exponentials and
// the value products -- with the lazily rescaled running maximum of the pair
// kernel.  Keys past the key count repeat the last key in LDS and get
// probability zero.
struct SeqAttnArgs {
  const bf16* q;
  int64_t ld_q;
  const bf16* k;
  const bf16* v;
  int64_t ld_kv;
  float scale_log2;
  bf16* o;
  int64_t ld_o;
  const int32_t* work;   // quads (sample, first 16-query tile, 0, tile count) over the query layout
  const int32_t* cu_q;   // query offsets
  const int32_t* cu_kv;  // key / value offsets (= cu_q for self-attention)
  int H;
};

template <int NMAX, int D>
__global__ void __launch_bounds__(512, NMAX <= 256 ? 4 : 2) attention_seq_kernel(SeqAttnArgs p) {
  static_assert(D == 32 || D == 64, "head_dim 32 or 64");
  constexpr int HV = D / 32;                      // 32-dim halves
  constexpr int KT16 = NMAX / 16;
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  const int x = blockIdx.x % kXcds, t = blockIdx.x / kXcds;
  const int h = t % p.H, pos = (t / p.H) * kXcds + x;
  const int4 w4 = reinterpret_cast<const int4*>(p.work)[pos];
  const int i = w4.x;
  if (i < 0) return;
  const int qt0 = w4.y, nqt = w4.w;
  const int64_t qbase = p.cu_q[i];
  const int n = p.cu_q[i + 1] - (int)qbase;       // queries of the sample
  const int64_t kbase = p.cu_kv[i];
  const int m = p.cu_kv[i + 1] - (int)kbase;      // keys of the sample
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  const int j0 = qt0 * 16;
  const int jw = j0 + 16 * wave + l16;            // this lane's query
  const bool wave_has_queries = wave < nqt && j0 + 16 * wave < n;
  const bool qvalid = jw < n;
  if (m == 0) {
    // no keys: the empty sum
    if (wave_has_queries && qvalid) {
      bf16* orow = p.o + (qbase + jw) * p.ld_o + h * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<bf16x4*>(orow + dt * 16 + 4 * g) = bf16x4{};
    }
    return;
  }
  const int npad = (m + 63) & ~63;
  bf16* Kh[2] = {lds, lds + NMAX * 32};           // key images per 32-dim half: tile of 16 keys -> 512 elements
  bf16* Vh[2] = {lds + HV * NMAX * 32, lds + (HV + 1) * NMAX * 32};   // values, row-major [key][32] per half

  // ---- stage keys and values of the whole sample (tiles below npad)
  for (int kt = wave; kt < KT16; kt += 8) {
    if (kt * 16 >= npad) break;
    const int key_k = min(kt * 16 + l16, m - 1);
    const int kv = kt * 16 + (lane >> 2), key_v = min(kv, m - 1);
    const int dgv = (lane & 3) ^ ((kv >> 2) & 3);
    const bf16* sk = p.k + (kbase + key_k) * p.ld_kv + h * D + g * 8;
    const bf16* sv = p.v + (kbase + key_v) * p.ld_kv + h * D + dgv * 8;
#pragma unroll
    for (int hv = 0; hv < HV; ++hv) {
      __builtin_amdgcn_global_load_lds((const void*)(sk + 32 * hv), (__attribute__((address_space(3))) void*)(Kh[hv] + kt * 512), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(sv + 32 * hv), (__attribute__((address_space(3))) void*)(Vh[hv] + kt * 512), 16, 0, 0);
    }
  }
  bf16x8 qf[HV];
#pragma unroll
  for (int hv = 0; hv < HV; ++hv) qf[hv] = bf16x8{};
  if (qvalid) {
    const bf16* qr = p.q + (qbase + jw) * p.ld_q + h * D + g * 8;
#pragma unroll
    for (int hv = 0; hv < HV; ++hv) qf[hv] = *reinterpret_cast<const bf16x8*>(qr + 32 * hv);
  }
  __builtin_amdgcn_s_waitcnt(0);                  // this wave's copies have landed
  __syncthreads();
  if (!wave_has_queries) return;

  const VtLane vl = vt_lane(l16, g);
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (bf16)1.f;
  const float c = p.scale_log2;
  float m_s = -INFINITY;
  constexpr int NO = D / 16;                      // output accumulators; O[NO] is the row sum
  f32x4 O[NO + 1];
#pragma unroll
  for (int u = 0; u <= NO; ++u) O[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto super_chunk = [&](auto sc_c, auto nt_c) {
    constexpr int SC = decltype(sc_c)::value, NT = decltype(nt_c)::value;
    constexpr int T0 = SC * 8;
    const int kc = SC * 128;
    f32x4 S[NT];
#pragma unroll
    for (int kt = 0; kt < NT; ++kt) {
      S[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int hv = 0; hv < HV; ++hv) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Kh[hv][(T0 + kt) * 512 + lane * 8]);
        S[kt] = mfma16(kf, qf[hv], S[kt]);
      }
      if (kt % 4 == 3) __builtin_amdgcn_sched_barrier(0);   // bounded key fragments in flight
    }
    if (kc + NT * 16 > m) {
#pragma unroll
      for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
          if (kc + kt * 16 + 4 * g + ii >= m) S[kt][ii] = -INFINITY;
    }
    float mloc = S[0][0];
#pragma unroll
    for (int kt = 0; kt < NT; ++kt)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) mloc = fmaxf(mloc, S[kt][ii]);
    mloc = query_max(mloc);
    if (__any((mloc - m_s) * c > 8.f)) {
      const float m_new = fmaxf(m_s, mloc);
      const float alpha = __builtin_amdgcn_exp2f((m_s - m_new) * c);
      m_s = m_new;
#pragma unroll
      for (int u = 0; u <= NO; ++u) O[u] *= alpha;
    }
    const float nm = -m_s * c;
    bf16x8 P[NT / 2];
#pragma unroll
    for (int kt = 0; kt < NT; ++kt)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii)
        P[kt >> 1][(kt & 1) * 4 + ii] = (bf16)__builtin_amdgcn_exp2f(fmaf(S[kt][ii], c, nm));
#pragma unroll
    for (int pp = 0; pp + 1 < NT / 2; pp += 2) {
      bf16x8 vf[HV][4];
#pragma unroll
      for (int hv = 0; hv < HV; ++hv) vt_frags2(Vh[hv], SC * 4 + pp, vl, vf[hv]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int hv = 0; hv < HV; ++hv) {
          O[2 * hv] = mfma16(vf[hv][2 * u], P[pp + u], O[2 * hv]);
          O[2 * hv + 1] = mfma16(vf[hv][2 * u + 1], P[pp + u], O[2 * hv + 1]);
        }
        O[NO] = mfma16(ones, P[pp + u], O[NO]);
      }
    }
    if constexpr ((NT / 2) % 2 == 1) {
      bf16x8 vf[HV][2];
#pragma unroll
      for (int hv = 0; hv < HV; ++hv) vt_frags1(Vh[hv], SC * 4 + NT / 2 - 1, vl, vf[hv]);
#pragma unroll
      for (int hv = 0; hv < HV; ++hv) {
        O[2 * hv] = mfma16(vf[hv][0], P[NT / 2 - 1], O[2 * hv]);
        O[2 * hv + 1] = mfma16(vf[hv][1], P[NT / 2 - 1], O[2 * hv + 1]);
      }
      O[NO] = mfma16(ones, P[NT / 2 - 1], O[NO]);
    }
  };
  auto run_sc = [&](auto sc_c) {
    constexpr int SC = decltype(sc_c)::value;
    const int rem = m - SC * 128;
    if (rem <= 0) return;
    if (rem > 96) super_chunk(sc_c, std::integral_constant<int, 8>{});
    else if (rem > 64) super_chunk(sc_c, std::integral_constant<int, 6>{});
    else if (rem > 32) super_chunk(sc_c, std::integral_constant<int, 4>{});
    else super_chunk(sc_c, std::integral_constant<int, 2>{});
  };
  run_sc(std::integral_constant<int, 0>{});
  run_sc(std::integral_constant<int, 1>{});
  if constexpr (NMAX > 256) {
    run_sc(std::integral_constant<int, 2>{});
    run_sc(std::integral_constant<int, 3>{});
  }
  if (qvalid) {
    const float inv = 1.f / O[NO][0];
    bf16* orow = p.o + (qbase + jw) * p.ld_o + h * D;
#pragma unroll
    for (int dt = 0; dt < NO; ++dt) {
      bf16x4 ov;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) ov[ii] = (bf16)(O[dt][ii] * inv);
      *reinterpret_cast<bf16x4*>(orow + dt * 16 + 4 * g) = ov;
    }
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
  int64_t ld_bias, ld_bias_head;
  float scale;
  float* o;
  int64_t ld_o;
  const int32_t* work;
  const int32_t* cu_seqlens;
  const int32_t* cu_pairs;
  const int32_t* cu_kv;  // axis 2: key / value offsets (= cu_seqlens for self-attention)
  int64_t ld_q;          // row stride of q (ld_qkv is that of k and v)
  const float* gate;     // NULL, or o = sigmoid(gate) * attention
  int64_t ld_gate;
};

// Exact two-pass softmax per query in fp32: one thread per query.  On axis 2
// the keys of sample i are rows cu_kv[i] .. cu_kv[i+1]; a query with no keys
// gets the empty sum, 0.
template <int D>
__global__ void __launch_bounds__(256) attention_f32_kernel(AttnF32Args p) {
  Seg sg;
  if (!segment_of(p, sg)) return;
  const int h = blockIdx.y;
  int n = sg.n;                                   // keys
  int64_t kbase = sg.base;
  if (p.axis == 2) {
    kbase = p.cu_kv[sg.sample];
    n = p.cu_kv[sg.sample + 1] - (int)kbase;
  }
  for (int qi = sg.q_begin + (int)threadIdx.x; qi < sg.q_end; qi += 256) {
    const int64_t qrow = sg.base + (int64_t)qi * sg.step;
    if (n == 0) {
#pragma unroll
      for (int d = 0; d < D; ++d) p.o[qrow * p.ld_o + h * D + d] = 0.f;
      continue;
    }
    float qv[D];
#pragma unroll
    for (int d = 0; d < D; ++d) qv[d] = p.q[qrow * p.ld_q + h * D + d];
    const float* brow = p.bias ? p.bias + (int64_t)h * p.ld_bias_head + (sg.cu + (p.axis == 0 ? (int64_t)qi * n : qi)) * p.ld_bias
                               : nullptr;
    auto logit = [&](int key) {
      const int64_t krow = kbase + (int64_t)key * sg.step;
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) s = fmaf(qv[d], p.k[krow * p.ld_qkv + h * D + d], s);
      s *= p.scale;
      if (brow) s += brow[(p.axis == 0 ? (int64_t)key : (int64_t)key * n) * p.ld_bias];
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
      const int64_t krow = kbase + (int64_t)key * sg.step;
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] = fmaf(e, p.v[krow * p.ld_qkv + h * D + d], acc[d]);
    }
#pragma unroll
    for (int d = 0; d < D; ++d) {
      float val = acc[d] / sum;
      if (p.gate) val /= 1.f + expf(-p.gate[qrow * p.ld_gate + h * D + d]);
      p.o[qrow * p.ld_o + h * D + d] = val;
    }
  }
}

}  // namespace

// ---------------------------------------------------------------- allocation-free scratch
// Scratch of nt_pair_row_attention_noalloc: one array per device, resolved to
// its device address once per device on first use.  Host code never passes
// the array's name to a kernel, only the resolved address.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

hipError_t noalloc_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[64] = {nullptr};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

size_t attention_workspace_bytes(const nt_layout& L, int axis, int H, int D, nt_dtype dtype, bool has_bias) {
  // only the d = 32 pair kernel (N <= 512) reads the bias through an image
  if (!has_bias || dtype != NT_BF16 || D != 32 || axis == 2 || L.max_len > kAttnLongLen) return 0;
  return (size_t)H * (size_t)L.bias_tiles_total() * 512;
}

namespace {
// 1-D attention on bf16 rows, head_dim 32 or 64: queries by Lq's offsets,
// keys and values by cu_kv (device) whose longest segment is kv_max_len
// (<= kAttnLongLen).
hipError_t launch_seq_attention(const nt_layout& Lq, const int32_t* cu_kv, int kv_max_len, int H, int D,
                                const void* q, int64_t ld_q, const void* k, const void* v, int64_t ld_kv,
                                float scale, void* o, int64_t ld_o, hipStream_t s) {
  if (Lq.sattn_items() == 0) return hipSuccess;
  if (D != 32 && D != 64) return hipErrorInvalidValue;
  const bool shortk = kv_max_len <= kAttnShortLen;
  const int nmax = shortk ? kAttnShortLen : kAttnLongLen;
  SeqAttnArgs a{(const bf16*)q, ld_q, (const bf16*)k, (const bf16*)v, ld_kv, scale * kLog2e, (bf16*)o, ld_o,
                Lq.d_sattn_work, Lq.d_cu_seqlens, cu_kv, H};
  const size_t smem = sizeof(bf16) * 2 * (size_t)(D / 32) * (size_t)nmax * 32;
  const dim3 grid((unsigned)(Lq.sattn_items() * H)), block(512);
  const void* fn = D == 64 ? (shortk ? (const void*)attention_seq_kernel<kAttnShortLen, 64>
                                     : (const void*)attention_seq_kernel<kAttnLongLen, 64>)
                           : (shortk ? (const void*)attention_seq_kernel<kAttnShortLen, 32>
                                     : (const void*)attention_seq_kernel<kAttnLongLen, 32>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e != hipSuccess) return e;
  if (D == 64) {
    if (shortk) attention_seq_kernel<kAttnShortLen, 64><<<grid, block, smem, s>>>(a);
    else attention_seq_kernel<kAttnLongLen, 64><<<grid, block, smem, s>>>(a);
  } else {
    if (shortk) attention_seq_kernel<kAttnShortLen, 32><<<grid, block, smem, s>>>(a);
    else attention_seq_kernel<kAttnLongLen, 32><<<grid, block, smem, s>>>(a);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_cross_attention(const nt_layout& Lq, const nt_layout& Lkv, int H, int D, const void* q,
                                  int64_t ld_q, const void* k, const void* v, int64_t ld_kv, float scale, void* o,
                                  int64_t ld_o, nt_dtype dtype, hipStream_t s) {
  if (Lq.sum_n == 0) return hipSuccess;
  if (dtype == NT_BF16) {
    if (Lkv.max_len > kAttnLongLen) return hipErrorInvalidValue;
    return launch_seq_attention(Lq, Lkv.d_cu_seqlens, Lkv.max_len, H, D, q, ld_q, k, v, ld_kv, scale, o, ld_o, s);
  }
  // fp32: the exact kernel, one workgroup per (sample, query block)
  if (Lq.seq_items() == 0) return hipSuccess;
  AttnF32Args a{2, H, (const float*)q, (const float*)k, (const float*)v, ld_kv, nullptr, 1, 1, scale, (float*)o,
                ld_o, Lq.d_seq_work, Lq.d_cu_seqlens, Lq.d_cu_pairs, Lkv.d_cu_seqlens, ld_q, nullptr, 0};
  const dim3 grid((unsigned)Lq.seq_items(), (unsigned)H), block(256);
  switch (D) {
    case 8: attention_f32_kernel<8><<<grid, block, 0, s>>>(a); break;
    case 16: attention_f32_kernel<16><<<grid, block, 0, s>>>(a); break;
    case 32: attention_f32_kernel<32><<<grid, block, 0, s>>>(a); break;
    case 64: attention_f32_kernel<64><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(const nt_layout& L, int axis, int H, int D, const void* q, const void* k,
                            const void* v, int64_t ld_qkv, const void* bias, int64_t ld_bias, int64_t ld_bias_head,
                            float scale, void* o, int64_t ld_o, nt_dtype dtype, void* workspace, hipStream_t s,
                            const void* gate, int64_t ld_gate) {
  const int32_t* work = axis == 2 ? L.d_seq_work : L.d_attn_work;
  const int64_t items = axis == 2 ? L.seq_items() : L.attn_items();
  if (items == 0) return hipSuccess;
  const dim3 grid((unsigned)items, (unsigned)H), block(256);
  if (dtype == NT_F32) {
    AttnF32Args a{axis, H, (const float*)q, (const float*)k, (const float*)v, ld_qkv, (const float*)bias,
                  ld_bias, ld_bias_head, scale, (float*)o, ld_o, work, L.d_cu_seqlens, L.d_cu_pairs,
                  L.d_cu_seqlens, ld_qkv, (const float*)gate, ld_gate};
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
  if (axis == 2 && L.max_len <= kAttnLongLen)
    return launch_seq_attention(L, L.d_cu_seqlens, L.max_len, H, D, q, ld_qkv, k, v, ld_qkv, scale, o, ld_o, s);
  if (D == 32 && axis != 2 && L.max_len <= kAttnLongLen) {
    if (L.pattn_items() == 0) return hipSuccess;
    const int nmax = L.max_len <= kAttnShortLen ? kAttnShortLen : kAttnLongLen;
    const int64_t tiles = L.bias_tiles_total();
    const uint2* img = nullptr;
    if (bias && tiles > 0) {
      // the caller's workspace receives the bias image
      BiasImgArgs b{axis, L.batch, (const bf16*)bias, ld_bias, ld_bias_head, 1.f / scale, (uint2*)workspace, tiles,
                    L.d_bias_tiles, L.d_cu_seqlens, L.d_cu_pairs};
      bias_image_kernel<<<dim3((unsigned)((tiles + 3) / 4), (unsigned)H), dim3(256), 0, s>>>(b);
      img = (const uint2*)workspace;
    }
    PairAttnArgs a{axis, (const bf16*)q, (const bf16*)k, (const bf16*)v, ld_qkv, (const bf16*)bias, ld_bias,
                   ld_bias_head, scale * kLog2e, (bf16*)o, ld_o, L.d_pattn_work, L.d_cu_seqlens, L.d_cu_pairs, H,
                   img, tiles * 64, L.d_bias_tiles, L.batch, L.sum_n, (const bf16*)gate, ld_gate};
    const size_t smem = sizeof(bf16) * 4 * (size_t)nmax * 32;
    const dim3 grid((unsigned)(L.pattn_items() * H));
    // the key-split instance also holds the hand-over of the upper key halves
    const size_t smem_ks = sizeof(bf16) * 4 * (size_t)kAttnLongLen * 32 + kAttnHandBytes;
    // gated: split rows add 8 gate slots past the hand-over, unsplit rows
    // use 16 slots from its start
    const size_t smem_ksg = sizeof(bf16) * 4 * (size_t)kAttnLongLen * 32 +
                            std::max<size_t>(kAttnHandBytes + kAttnGateBytes / 2, kAttnGateBytes);
    if (gate) {
      // gated output (axes 0 and 1): the GATE instances of the same kernels
      if (nmax == kAttnShortLen) {
        const int per_xcd = std::max(H, compute_units() / kXcds / H * H);
        const dim3 gridp((unsigned)(per_xcd * kXcds));
        hipFuncSetAttribute((const void*)attention_pair_kernel<kAttnShortLen, 16, true, true>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        attention_pair_kernel<kAttnShortLen, 16, true, true><<<gridp, dim3(1024), smem, s>>>(a);
      } else {
        hipFuncSetAttribute((const void*)attention_pair_kernel<kAttnLongLen, 16, false, true, true>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem_ksg);
        attention_pair_kernel<kAttnLongLen, 16, false, true, true><<<grid, dim3(1024), smem_ksg, s>>>(a);
      }
    } else if (axis == 3) {
      // single attention with pair bias: one row per sample, the 8-wave
      // instance over the 1-D attention's (sample, 128-query block) items
      if (L.sattn_items() == 0) return hipSuccess;
      a.work = L.d_sattn_work;
      const size_t smem3 = sizeof(bf16) * 4 * (size_t)kAttnLongLen * 32;
      hipFuncSetAttribute((const void*)attention_pair_kernel<kAttnLongLen, 8, false>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem3);
      attention_pair_kernel<kAttnLongLen, 8, false><<<dim3((unsigned)(L.sattn_items() * H)), dim3(512), smem3, s>>>(a);
    } else if (nmax == kAttnShortLen) {
      // persistent: one workgroup of 16 waves per CU (all queries of a row);
      // per XCD a multiple of H workgroups, at least H, so every head gets an
      // equal share of each XCD's rows
      const int per_xcd = std::max(H, compute_units() / kXcds / H * H);
      const dim3 gridp((unsigned)(per_xcd * kXcds));
      hipFuncSetAttribute((const void*)attention_pair_kernel<kAttnShortLen, 16, true>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      attention_pair_kernel<kAttnShortLen, 16, true><<<gridp, dim3(1024), smem, s>>>(a);
    } else {
      hipFuncSetAttribute((const void*)attention_pair_kernel<kAttnLongLen, 16, false, false, true>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem_ks);
      attention_pair_kernel<kAttnLongLen, 16, false, false, true><<<grid, dim3(1024), smem_ks, s>>>(a);
    }
    return hipGetLastError();
  }
  const int vstride = (npad + 127) / 128 * 128 + 4;
  AttnArgs a{axis, H, (const bf16*)q, (const bf16*)k, (const bf16*)v, ld_qkv, (const bf16*)bias, ld_bias,
             ld_bias_head, scale * kLog2e, (bf16*)o, ld_o, work, L.d_cu_seqlens, L.d_cu_pairs, vstride,
             (const bf16*)gate, ld_gate};
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
