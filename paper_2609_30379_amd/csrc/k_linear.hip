// LayerNorm + Linear on packed rows (Sec. 3.3: V' = V W^T + b, with the
// normalisation acting on each row's feature tail).  Rows are independent, so
// every launch covers the whole ragged batch as one dense [R, K] x [K, N].
//
// bf16 path: matrix cores (v_mfma_f32_16x16x32_bf16), computed transposed as
// D^T = W X^T so that each lane ends up owning four consecutive output
// channels of one row, which the fused epilogues (bias, residual, GELU,
// channel-major tails) consume without a shuffle.
#include <algorithm>

#include "nt_device.h"
#include "nt_internal.h"

namespace nt {
namespace {

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int kSmallRows = 8192;    // row counts taken by the one-wave-per-block kernel
constexpr int SK = BK + 8;          // LDS row stride (bf16): 80 bytes, keeps b128 reads spread

struct LinArgs {
  int rows, K, N, n_main;
  const void* x;
  int64_t ldx;
  const float* gamma;
  const float* beta;
  float eps;
  const bf16* w;
  const float* bias;
  const bf16* res;
  int64_t ld_res;
  bf16* y;
  int64_t ldy;
  bf16* y_tail;
  int64_t ld_tail;
  int tail_mode;
  const int32_t* row_splits2;
  const int32_t* row_sample;
  const int32_t* cu_seqlens;
  const int32_t* cu_pad;
  int sum_n;
  int mblocks, nblocks;
  const int32_t* blk_prow;    // first pair row of every kLinRows-cell block
  const int32_t* cu_pairs;    // sample tables of the streaming kernel's pair-tiled tails
  int batch;
  int wc, ntiles;             // streaming kernel: waves along the columns, 64-row tiles
  int stage_out;              // streaming kernel: write the output tile back through LDS
  // pair-broadcast rows (wave kernel): row cell(i, a, b) is u[eta_i + a] + v[eta_i + b]
  const bf16* bc_u;
  const bf16* bc_v;
  int64_t ld_bc_u, ld_bc_v;
  const int32_t* bc_cu_tiles; // per sample: broadcast tiles (16 cells of one pair row) before it
  int bc_ntiles;              // all broadcast tiles
  const bf16* gate;           // NT_EPI_GATED_RESIDUAL: gate logits [rows, n_main], row stride ld_gate
  int64_t ld_gate;
};

// 1 / (1 + e^-v): the gate of the gated epilogues
__device__ __forceinline__ float sigmoid_gate(float v) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-v * 1.4426950408889634f));
}

// Position of the pair cell (a, b) of sample i in its pair-tiled operand plane:
// row a, column b, or row b, column a for the transposed (incoming) operand.
__device__ __forceinline__ int32_t tiled_cell_pos(int32_t P, int n, int a, int b, bool transposed) {
  const int nkt = (n + 31) >> 5;
  return P + (transposed ? tiled_offset(b, a, nkt) : tiled_offset(a, b, nkt));
}

// Pair-tiled position of packed pair row m (cell (i, a, b)): pair row by
// binary search over the level-2 row splits.
__device__ __forceinline__ int32_t pair_tiled_pos(const LinArgs& p, int m) {
  int lo = 0, hi = p.sum_n - 1;               // largest eta with row_splits2[eta] <= m
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.row_splits2[mid] <= m) lo = mid; else hi = mid - 1;
  }
  const int i = p.row_sample[lo];
  const int n = p.cu_seqlens[i + 1] - p.cu_seqlens[i];
  return tiled_cell_pos(p.cu_pad[i], n, lo - p.cu_seqlens[i], m - p.row_splits2[lo], p.tail_mode == kTailPairTiledT);
}

__device__ __forceinline__ float gelu_erf(float v) { return 0.5f * v * (1.f + erff(v * 0.70710678118654752f)); }

// Raw (unnormalised) global data of one k-step, held in registers while the
// previous step computes.
template <typename XT> struct XStage;
template <> struct XStage<bf16> {
  using T = uint4;
  uint4 d[2];
  static __device__ __forceinline__ uint4 zero() { return make_uint4(0, 0, 0, 0); }
  static __device__ __forceinline__ void unpack(const uint4& t, float* o) {
    const uint32_t w4[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[2 * j] = __uint_as_float(w4[j] << 16);
      o[2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
    }
  }
};
template <> struct XStage<float> {
  using T = float4;
  float4 d[4];
  static __device__ __forceinline__ float4 zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  static __device__ __forceinline__ void unpack(const float4& t, float* o) { o[0] = t.x; o[1] = t.y; o[2] = t.z; o[3] = t.w; }
};

template <typename XT, int EPI>
__global__ void __launch_bounds__(256) linear_mfma_kernel(LinArgs p) {
  __shared__ __attribute__((aligned(16))) bf16 Xs[BM * SK];
  __shared__ __attribute__((aligned(16))) bf16 Ws[BN * SK];
  __shared__ float s_mean[BM], s_rstd[BM];

  // XCD-aware tile order: the n-blocks of one row block run back to back on
  // the same XCD (workgroups are dispatched round-robin over 8 XCDs), so the
  // row block is fetched into one L2 once.
  const int id = blockIdx.x;
  const int xcd = id % kXcds, kq = id / kXcds;
  const int nb = kq % p.nblocks;
  const int mb = (kq / p.nblocks) * kXcds + xcd;
  if (mb >= p.mblocks) return;
  const int m0 = mb * BM, n0 = nb * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const XT* x = static_cast<const XT*>(p.x);
  constexpr int VX = Vec<XT>::N;

  // ---- LayerNorm statistics: 16 lanes per row, two passes, fp32 ----------
  if (p.gamma) {
    for (int rr = tid >> 4; rr < BM; rr += 16) {
      const int m = m0 + rr;
      float mean = 0.f, rstd = 0.f;
      if (m < p.rows) {
        const XT* row = x + (int64_t)m * p.ldx;
        float s = 0.f;
        for (int k = l16 * VX; k < p.K; k += 16 * VX) {
          Vec<XT> t; t.load(row + k);
#pragma unroll
          for (int j = 0; j < VX; ++j) s += t.v[j];
        }
        mean = group_sum<16>(s) / (float)p.K;
        float q = 0.f;
        for (int k = l16 * VX; k < p.K; k += 16 * VX) {
          Vec<XT> t; t.load(row + k);
#pragma unroll
          for (int j = 0; j < VX; ++j) { const float d = t.v[j] - mean; q += d * d; }
        }
        rstd = rsqrtf(group_sum<16>(q) / (float)p.K + p.eps);
      }
      if (l16 == 0) { s_mean[rr] = mean; s_rstd[rr] = rstd; }
    }
  }

  // ---- staging: thread t owns row t/2 and 16 consecutive k ----------------
  const int srow = tid >> 1, skh = (tid & 1) * 16;
  const int xm = m0 + srow, wn = n0 + srow;
  XStage<XT> xs;
  uint4 wsr[2];
  auto load_step = [&](int k0) {
#pragma unroll
    for (int c = 0; c < 16 / VX; ++c) {
      const int k = k0 + skh + c * VX;
      if (xm < p.rows && k < p.K) {
        if constexpr (VX == 8) xs.d[c] = *reinterpret_cast<const uint4*>(x + (int64_t)xm * p.ldx + k);
        else xs.d[c] = *reinterpret_cast<const float4*>(x + (int64_t)xm * p.ldx + k);
      } else {
        if constexpr (VX == 8) xs.d[c] = make_uint4(0, 0, 0, 0);
        else xs.d[c] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int k = k0 + skh + c * 8;
      wsr[c] = (wn < p.N && k < p.K) ? *reinterpret_cast<const uint4*>(p.w + (int64_t)wn * p.K + k)
                                     : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_step = [&](int k0) {
    float v[16];
    if constexpr (VX == 8) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const uint32_t w4[4] = {xs.d[c].x, xs.d[c].y, xs.d[c].z, xs.d[c].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[c * 8 + 2 * j] = __uint_as_float(w4[j] << 16);
          v[c * 8 + 2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
        }
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        v[4 * c] = xs.d[c].x; v[4 * c + 1] = xs.d[c].y; v[4 * c + 2] = xs.d[c].z; v[4 * c + 3] = xs.d[c].w;
      }
    }
    if (p.gamma) {
      const float mu = s_mean[srow], rs = s_rstd[srow];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int k = k0 + skh + 4 * c;
        if (k < p.K) {
          const float4 ga = *reinterpret_cast<const float4*>(p.gamma + k);
          const float4 be = p.beta ? *reinterpret_cast<const float4*>(p.beta + k) : make_float4(0.f, 0.f, 0.f, 0.f);
          v[4 * c + 0] = (v[4 * c + 0] - mu) * rs * ga.x + be.x;
          v[4 * c + 1] = (v[4 * c + 1] - mu) * rs * ga.y + be.y;
          v[4 * c + 2] = (v[4 * c + 2] - mu) * rs * ga.z + be.z;
          v[4 * c + 3] = (v[4 * c + 3] - mu) * rs * ga.w + be.w;
        } else {
          v[4 * c] = v[4 * c + 1] = v[4 * c + 2] = v[4 * c + 3] = 0.f;
        }
      }
      if (xm >= p.rows) {
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = 0.f;
      }
    }
    bf16x8 lo, hi;
#pragma unroll
    for (int j = 0; j < 8; ++j) { lo[j] = (bf16)v[j]; hi[j] = (bf16)v[8 + j]; }
    *reinterpret_cast<bf16x8*>(&Xs[srow * SK + skh]) = lo;
    *reinterpret_cast<bf16x8*>(&Xs[srow * SK + skh + 8]) = hi;
    *reinterpret_cast<uint4*>(&Ws[srow * SK + skh]) = wsr[0];
    *reinterpret_cast<uint4*>(&Ws[srow * SK + skh + 8]) = wsr[1];
  };

  const int wn_off = (wave >> 1) * 64, wm_off = (wave & 1) * 64;
  const bool wave_active = n0 + wn_off < p.N;
  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  __syncthreads();                 // statistics visible
  load_step(0);
  store_step(0);
  __syncthreads();
  for (int k0 = 0; k0 < p.K; k0 += BK) {
    const bool more = k0 + BK < p.K;
    if (more) load_step(k0 + BK);
    if (wave_active) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        af[t] = *reinterpret_cast<const bf16x8*>(&Ws[(wn_off + t * 16 + l16) * SK + g * 8]);
        bfr[t] = *reinterpret_cast<const bf16x8*>(&Xs[(wm_off + t * 16 + l16) * SK + g * 8]);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = mfma16(af[a], bfr[b], acc[a][b]);
    }
    __syncthreads();
    if (more) {
      store_step(k0 + BK);
      __syncthreads();
    }
  }
  if (!wave_active) return;

  // ---- epilogue: lane owns channels n..n+3 of row m for every (a, b) tile --
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int m = m0 + wm_off + b * 16 + l16;
    if (m >= p.rows) continue;
    int64_t tpos = m;
    if (p.y_tail && p.tail_mode != kTailChannelMajor && n0 + BN > p.n_main) tpos = pair_tiled_pos(p, m);
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int n = n0 + wn_off + a * 16 + g * 4;
      if (n >= p.N) continue;
      float r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        r[i] = acc[a][b][i] + ((p.bias && n + i < p.N) ? p.bias[n + i] : 0.f);
        if constexpr (EPI == NT_EPI_GELU) r[i] = gelu_erf(r[i]);
      }
      if (n + 4 <= p.n_main) {
        if constexpr (EPI == NT_EPI_GATED_RESIDUAL) {
#pragma unroll
          for (int i = 0; i < 4; ++i) r[i] *= sigmoid_gate((float)p.gate[(int64_t)m * p.ld_gate + n + i]);
        }
        if constexpr (EPI == NT_EPI_RESIDUAL || EPI == NT_EPI_GATED_RESIDUAL) {
          const uint2 rr = *reinterpret_cast<const uint2*>(p.res + (int64_t)m * p.ld_res + n);
          r[0] += __uint_as_float(rr.x << 16); r[1] += __uint_as_float(rr.x & 0xffff0000u);
          r[2] += __uint_as_float(rr.y << 16); r[3] += __uint_as_float(rr.y & 0xffff0000u);
        }
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (bf16)r[i];
        *reinterpret_cast<bf16x4*>(p.y + (int64_t)m * p.ldy + n) = o;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int nn = n + i;
          if (nn >= p.N) break;
          if (nn < p.n_main) {
            float v = r[i];
            if constexpr (EPI == NT_EPI_GATED_RESIDUAL) v *= sigmoid_gate((float)p.gate[(int64_t)m * p.ld_gate + nn]);
            if constexpr (EPI == NT_EPI_RESIDUAL || EPI == NT_EPI_GATED_RESIDUAL) v += (float)p.res[(int64_t)m * p.ld_res + nn];
            p.y[(int64_t)m * p.ldy + nn] = (bf16)v;
          } else {
            p.y_tail[(int64_t)(nn - p.n_main) * p.ld_tail + tpos] = (bf16)r[i];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------- K-resident
// For the pair path (K <= 256) one workgroup owns a 128-row tile and all
// output columns: the whole normalised tile and one 128-column weight block
// sit in LDS after a single global round trip, LayerNorm statistics come from
// registers (two threads per row), and the next weight block is prefetched
// into registers while the current one runs on the matrix cores.  Rows of a
// pair-level input are cells; their pair-tiled tail offsets come from the
// per-pair-row tables (first pair row of the tile from blk_prow, the tile's
// row splits cached in LDS).
// LDS row stride (elements) for 16-byte fragment reads of a K-wide bf16 tile:
// conflict-free when the stride is 8 (mod 64) dwords, i.e. 16 (mod 128) elements.
template <int K> constexpr int frag_stride() { return K + ((16 - K % 128) + 128) % 128; }

template <typename XT, int EPI, int K>
__global__ void __launch_bounds__(256) linear_res_kernel(LinArgs p) {
  constexpr int SKR = frag_stride<K>();
  constexpr int VX = Vec<XT>::N;
  constexpr int HALF = K / 2;
  constexpr int NV = HALF / VX;               // x vectors per thread
  constexpr int WV = K / 16;                  // weight vectors per thread per block
  __shared__ __attribute__((aligned(16))) bf16 Xs[BM * SKR];
  __shared__ __attribute__((aligned(16))) bf16 Ws[BN * SKR];
  __shared__ int32_t rs[BM + 1];
  const int mb = blockIdx.x;
  const int m0 = mb * BM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const XT* x = static_cast<const XT*>(p.x);

  // ---- issue every global load of the tile and the first weight block ----
  const int r = tid >> 1, hh = tid & 1, xm = m0 + r;
  using XV = typename XStage<XT>::T;
  XV xr[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    if (xm < p.rows) xr[v] = *reinterpret_cast<const XV*>(x + (int64_t)xm * p.ldx + hh * HALF + v * VX);
    else xr[v] = XStage<XT>::zero();
  }
  uint4 wr[WV];
  auto load_w = [&](int n0) {
#pragma unroll
    for (int j = 0; j < WV; ++j) {
      const int c = tid + 256 * j, wrow = c / (K / 8), wcol = (c % (K / 8)) * 8;
      wr[j] = (n0 + wrow < p.N) ? *reinterpret_cast<const uint4*>(p.w + (int64_t)(n0 + wrow) * K + wcol)
                                : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_w = [&]() {
#pragma unroll
    for (int j = 0; j < WV; ++j) {
      const int c = tid + 256 * j, wrow = c / (K / 8), wcol = (c % (K / 8)) * 8;
      *reinterpret_cast<uint4*>(&Ws[wrow * SKR + wcol]) = wr[j];
    }
  };
  load_w(0);
  const bool tiled_tail = p.y_tail && p.tail_mode != kTailChannelMajor;
  int eta0 = 0;
  if (tiled_tail) {
    eta0 = p.blk_prow[mb];
    for (int j = tid; j <= BM; j += 256) rs[j] = p.row_splits2[min(eta0 + j, p.sum_n)];
  }

  // ---- LayerNorm from the raw registers, normalised bf16 tile into LDS ----
  float mean = 0.f, rstd = 1.f;
  if (p.gamma) {
    float s = 0.f;
#pragma unroll
    for (int vv = 0; vv < NV; ++vv) {
      float t[VX];
      XStage<XT>::unpack(xr[vv], t);
#pragma unroll
      for (int e = 0; e < VX; ++e) s += t[e];
    }
    s += __shfl_xor(s, 1, 64);
    mean = s / (float)K;
    float q = 0.f;
#pragma unroll
    for (int vv = 0; vv < NV; ++vv) {
      float t[VX];
      XStage<XT>::unpack(xr[vv], t);
#pragma unroll
      for (int e = 0; e < VX; ++e) { const float d = t[e] - mean; q += d * d; }
    }
    q += __shfl_xor(q, 1, 64);
    rstd = xm < p.rows ? rsqrtf(q / (float)K + p.eps) : 0.f;
  }
#pragma unroll
  for (int j = 0; j < HALF; j += 8) {
    float t[8];
    XStage<XT>::unpack(xr[j / VX], t);
    if constexpr (VX == 4) XStage<XT>::unpack(xr[j / VX + 1], t + 4);
    if (p.gamma) {
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        const float4 ga = *reinterpret_cast<const float4*>(p.gamma + hh * HALF + j + e);
        const float4 be = p.beta ? *reinterpret_cast<const float4*>(p.beta + hh * HALF + j + e)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
        t[e] = (t[e] - mean) * rstd * ga.x + be.x;
        t[e + 1] = (t[e + 1] - mean) * rstd * ga.y + be.y;
        t[e + 2] = (t[e + 2] - mean) * rstd * ga.z + be.z;
        t[e + 3] = (t[e + 3] - mean) * rstd * ga.w + be.w;
      }
      if (xm >= p.rows) {
#pragma unroll
        for (int e = 0; e < 8; ++e) t[e] = 0.f;
      }
    }
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (bf16)t[e];
    *reinterpret_cast<bf16x8*>(&Xs[r * SKR + hh * HALF + j]) = o;
  }
  store_w();
  __syncthreads();

  // pair-tiled offsets of the lane's four rows
  const int wn_off = (wave >> 1) * 64, wm_off = (wave & 1) * 64;
  int32_t tpos[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int m = m0 + wm_off + b * 16 + l16;
    tpos[b] = m;
    if (tiled_tail && m < p.rows) {
      int lo = 0, hi = min(BM, p.sum_n - eta0) - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (rs[mid] <= m) lo = mid; else hi = mid - 1;
      }
      const int eta = eta0 + lo, i = p.row_sample[eta];
      tpos[b] = tiled_cell_pos(p.cu_pad[i], p.cu_seqlens[i + 1] - p.cu_seqlens[i], eta - p.cu_seqlens[i], m - rs[lo],
                               p.tail_mode == kTailPairTiledT);
    }
  }

  for (int n0 = 0; n0 < p.N; n0 += BN) {
    const bool more = n0 + BN < p.N;
    if (more) load_w(n0 + BN);
    f32x4 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bool wave_active = n0 + wn_off < p.N;
    if (wave_active) {
#pragma unroll
      for (int kk = 0; kk < K / 32; ++kk) {
        bf16x8 af[4], bfr[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          af[t] = *reinterpret_cast<const bf16x8*>(&Ws[(wn_off + t * 16 + l16) * SKR + kk * 32 + g * 8]);
          bfr[t] = *reinterpret_cast<const bf16x8*>(&Xs[(wm_off + t * 16 + l16) * SKR + kk * 32 + g * 8]);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = mfma16(af[a], bfr[b], acc[a][b]);
      }
      // epilogue: lane owns channels n..n+3 of row m for every (a, b) tile
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int m = m0 + wm_off + b * 16 + l16;
        if (m >= p.rows) continue;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int n = n0 + wn_off + a * 16 + g * 4;
          if (n >= p.N) continue;
          float rr[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            rr[i] = acc[a][b][i] + ((p.bias && n + i < p.N) ? p.bias[n + i] : 0.f);
            if constexpr (EPI == NT_EPI_GELU) rr[i] = gelu_erf(rr[i]);
          }
          if (n + 4 <= p.n_main) {
            if constexpr (EPI == NT_EPI_RESIDUAL) {
              const uint2 q2 = *reinterpret_cast<const uint2*>(p.res + (int64_t)m * p.ld_res + n);
              rr[0] += __uint_as_float(q2.x << 16); rr[1] += __uint_as_float(q2.x & 0xffff0000u);
              rr[2] += __uint_as_float(q2.y << 16); rr[3] += __uint_as_float(q2.y & 0xffff0000u);
            }
            bf16x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = (bf16)rr[i];
            *reinterpret_cast<bf16x4*>(p.y + (int64_t)m * p.ldy + n) = o;
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int nn = n + i;
              if (nn >= p.N) break;
              if (nn < p.n_main) {
                float val = rr[i];
                if constexpr (EPI == NT_EPI_RESIDUAL) val += (float)p.res[(int64_t)m * p.ld_res + nn];
                p.y[(int64_t)m * p.ldy + nn] = (bf16)val;
              } else {
                p.y_tail[(int64_t)(nn - p.n_main) * p.ld_tail + tpos[b]] = (bf16)rr[i];
              }
            }
          }
        }
      }
    }
    if (more) {
      __syncthreads();
      store_w();
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- small row counts
// Projections over few rows (the single track: one row per token) are pure
// latency: a handful of large tiles would each walk the whole K loop alone.
// Here a workgroup of four waves owns a 16-row x 64-column output block and
// splits K between its waves (wave w takes k-steps w, w + 4, ...): each wave
// issues the loads of all its k-steps at once, so the block costs about one
// memory round trip instead of one per k-step; the partial products meet in
// LDS and wave w finishes column tile w.  No LayerNorm and no tail columns
// (those take the other paths).
constexpr int kSmallWaves = 4;
constexpr int kSmallSteps = 4;       // k-steps per wave loaded at once (K <= 512 in one round)

template <typename XT, int EPI>
__global__ void __launch_bounds__(64 * kSmallWaves) linear_small_kernel(LinArgs p) {
  __shared__ f32x4 part[kSmallWaves][4][64];
  const int lane = threadIdx.x & 63, l16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int m0 = blockIdx.x * 16, n0 = blockIdx.y * 64;
  const XT* x = static_cast<const XT*>(p.x);
  const int m = m0 + l16;
  const bool mrow = m < p.rows;
  const int nks = p.K / 32;
  auto load_step = [&](int k0, bf16x8 (&wa)[4], bf16x8& xb) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int n = n0 + t * 16 + l16;
      wa[t] = n < p.N ? *reinterpret_cast<const bf16x8*>(p.w + (int64_t)n * p.K + k0 + g * 8) : bf16x8{};
    }
    if constexpr (Vec<XT>::N == 8) {
      xb = mrow ? *reinterpret_cast<const bf16x8*>(x + (int64_t)m * p.ldx + k0 + g * 8) : bf16x8{};
    } else {
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
      if (mrow) {
        a = *reinterpret_cast<const float4*>(x + (int64_t)m * p.ldx + k0 + g * 8);
        b = *reinterpret_cast<const float4*>(x + (int64_t)m * p.ldx + k0 + g * 8 + 4);
      }
      xb = bf16x8{(bf16)a.x, (bf16)a.y, (bf16)a.z, (bf16)a.w, (bf16)b.x, (bf16)b.y, (bf16)b.z, (bf16)b.w};
    }
  };
  f32x4 acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s0 = wave; s0 < nks; s0 += kSmallWaves * kSmallSteps) {
    bf16x8 wa[kSmallSteps][4], xb[kSmallSteps];
#pragma unroll
    for (int j = 0; j < kSmallSteps; ++j)
      if (s0 + kSmallWaves * j < nks) load_step((s0 + kSmallWaves * j) * 32, wa[j], xb[j]);
#pragma unroll
    for (int j = 0; j < kSmallSteps; ++j)
      if (s0 + kSmallWaves * j < nks) {
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma16(wa[j][t], xb[j], acc[t]);
      }
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) part[wave][t][lane] = acc[t];
  __syncthreads();
  // column tile t = wave: the four partial products in wave order
  f32x4 r4 = part[0][wave][lane];
#pragma unroll
  for (int w = 1; w < kSmallWaves; ++w) r4 += part[w][wave][lane];
  if (!mrow) return;
  const int n = n0 + wave * 16 + 4 * g;            // lane owns channels n..n+3 of row m
  if (n >= p.N) return;
  float r[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    r[i] = r4[i] + ((p.bias && n + i < p.N) ? p.bias[n + i] : 0.f);
    if constexpr (EPI == NT_EPI_GELU) r[i] = gelu_erf(r[i]);
  }
  if (n + 4 <= p.N) {
    if constexpr (EPI == NT_EPI_RESIDUAL) {
      const uint2 q2 = *reinterpret_cast<const uint2*>(p.res + (int64_t)m * p.ld_res + n);
      r[0] += __uint_as_float(q2.x << 16); r[1] += __uint_as_float(q2.x & 0xffff0000u);
      r[2] += __uint_as_float(q2.y << 16); r[3] += __uint_as_float(q2.y & 0xffff0000u);
    }
    bf16x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = (bf16)r[i];
    *reinterpret_cast<bf16x4*>(p.y + (int64_t)m * p.ldy + n) = o;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (n + i >= p.N) break;
      float v = r[i];
      if constexpr (EPI == NT_EPI_RESIDUAL) v += (float)p.res[(int64_t)m * p.ld_res + n + i];
      p.y[(int64_t)m * p.ldy + n + i] = (bf16)v;
    }
  }
}

// ---------------------------------------------------------------- streaming
// Persistent projection for K in {64, 128} and up to 512 output columns (the
// pair path).  The product is HBM-bound, so the kernel is organised around
// keeping loads in flight and stores coalesced: every workgroup stays
// resident and walks 64-row tiles; the weights of each wave's output columns
// live in registers for the whole launch; while one tile is on the matrix
// cores the next tile's rows are already loading into registers, and the
// normalised tiles alternate between two LDS buffers.  The eight waves split
// a tile as (row groups) x (column groups): a wave owns column tiles
// wcol + wc*t and 16-row subtiles u with u % (8/wc) == wrow.
// The finished tile (bias, activation; fp32 when a residual follows) is
// staged in LDS and written back row-contiguously, 16 bytes per lane, with
// the residual read the same way: a lane's own fragment would otherwise
// scatter every store over 16 rows.
constexpr int kStreamRows = 64;
constexpr int kStreamThreads = 512;
constexpr int kStreamMaxSamples = kPairTiledMaxSamples;   // sample tables cached in LDS for pair-tiled tails

// Pair-tiled position of packed pair cell m (Eq. coordinate inverted with the
// sample tables): sample i by binary search over the pair offsets, then
// (a, b) = divmod(m - o_i, N_i).
__device__ __forceinline__ int32_t tiled_pos_lds(const int32_t* cp, const int32_t* len, const int32_t* pad,
                                                 int batch, int m, bool transposed) {
  int lo = 0, hi = batch - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cp[mid] <= m) lo = mid; else hi = mid - 1;
  }
  const int n = len[lo], local = m - cp[lo];
  int a = (int)((float)local / (float)n);
  int b = local - a * n;
  if (b < 0) { --a; b += n; } else if (b >= n) { ++a; b -= n; }
  return tiled_cell_pos(pad[lo], n, a, b, transposed);
}

// LDS row stride (elements) of the staged output tile.
__host__ __device__ constexpr int stage_stride(int n_main, bool f32) { return n_main + (f32 ? 4 : 8); }

template <typename XT, int EPI, int K, int NTW>
__global__ void __launch_bounds__(kStreamThreads, 2) linear_stream_kernel(LinArgs p) {
  constexpr int TR = kStreamRows;
  constexpr int SKR = frag_stride<K>();
  constexpr int KT = K / 32;
  constexpr int TPR = kStreamThreads / TR;        // staging threads per row
  constexpr int EPT = K / TPR;                    // elements per staging thread
  constexpr int VX = Vec<XT>::N;
  constexpr int NV = EPT / VX;                    // 16-byte loads per staging thread
  constexpr bool RES = EPI == NT_EPI_RESIDUAL;
  constexpr int OCH = RES ? 4 : 2 * NTW;          // output 16-byte chunks per thread per tile, at most
  using XV = typename XStage<XT>::T;
  __shared__ __attribute__((aligned(16))) bf16 Xs[2][TR * SKR];
  __shared__ int32_t s_cp[kStreamMaxSamples + 1], s_len[kStreamMaxSamples], s_pad[kStreamMaxSamples];
  __shared__ __attribute__((aligned(16))) float s_bias[32 * 16];          // bias of all output columns
  __shared__ __attribute__((aligned(16))) float s_gamma[K], s_beta[K];     // LayerNorm affine
  extern __shared__ __attribute__((aligned(16))) unsigned char ys_raw[];   // staged output tile

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int wc = p.wc, wr_n = 8 / wc, wcol = wave % wc, wrow = wave / wc;
  const int nt16 = (p.N + 15) >> 4;
  const XT* x = static_cast<const XT*>(p.x);
  const bool tiled_tail = p.y_tail && p.tail_mode != kTailChannelMajor;
  const bool transposed = p.tail_mode == kTailPairTiledT;
  const bool stage = p.stage_out;                 // n_main % 8 == 0, 16-byte aligned rows
  const int NS = stage_stride(p.n_main, RES);
  const int c8n = p.n_main / 8;                   // 16-byte chunks per output row
  const int G = (int)gridDim.x;
  if ((int)blockIdx.x >= p.ntiles) return;
  auto ysf = [&](int) { return reinterpret_cast<float*>(ys_raw); };
  auto ysb = [&](int) { return reinterpret_cast<bf16*>(ys_raw); };
  auto tile_of = [&](int i) { return (int)blockIdx.x + i * G; };

  // ---- input rows: a ring of PF register slots, loads issued PF tiles ahead
  constexpr int PF = NTW == 2 ? 3 : 1;
  const int srow = tid / TPR, spart = tid % TPR;
  const XT* xthread = x + (int64_t)srow * p.ldx + spart * EPT;   // row srow of tile 0
  const int64_t xtile = (int64_t)TR * p.ldx;
  XV xr[PF][NV];
  auto load_x = [&](int t, XV (&dst)[NV]) {
    const bool ok = t < p.ntiles && t * TR + srow < p.rows;
    const XT* src = xthread + t * xtile;
#pragma unroll
    for (int v = 0; v < NV; ++v) dst[v] = ok ? *reinterpret_cast<const XV*>(src + v * VX) : XStage<XT>::zero();
  };
  // write-back chunks of this thread: (row, 8 columns), fixed for every tile
  int wb_row[OCH], wb_col[OCH];
#pragma unroll
  for (int c = 0; c < OCH; ++c) {
    const int ch = tid + kStreamThreads * c;
    wb_row[c] = (stage && ch < TR * c8n) ? ch / c8n : TR;       // TR: no chunk
    wb_col[c] = (stage && ch < TR * c8n) ? (ch % c8n) * 8 : 0;
  }
  // residual chunks of the staged write-back, loaded a tile ahead of it
  uint4 rres[RES ? OCH : 1];
  auto load_res = [&](int t) {
    if constexpr (RES) {
      const bf16* rtile = p.res + (int64_t)t * TR * p.ld_res;
#pragma unroll
      for (int c = 0; c < OCH; ++c) {
        const bool ok = stage && t < p.ntiles && wb_row[c] < TR && t * TR + wb_row[c] < p.rows;
        rres[c] = ok ? *reinterpret_cast<const uint4*>(rtile + wb_row[c] * p.ld_res + wb_col[c]) : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };
#pragma unroll
  for (int d = 0; d < PF; ++d) load_x(tile_of(d), xr[d]);
  load_res(tile_of(0));

  // ---- resident weights of the wave's column tiles; bias and affine in LDS
  bf16x8 wf[NTW][KT];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    const int ct = wcol + wc * j, n = ct * 16 + l16;
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      if (ct < nt16 && n < p.N) wf[j][kk] = *reinterpret_cast<const bf16x8*>(p.w + (int64_t)n * K + kk * 32 + g * 8);
      else wf[j][kk] = bf16x8{};
    }
  }
  for (int j = tid; j < 32 * 16; j += kStreamThreads) s_bias[j] = (p.bias && j < p.N) ? p.bias[j] : 0.f;
  for (int j = tid; j < K; j += kStreamThreads) {
    s_gamma[j] = p.gamma ? p.gamma[j] : 1.f;
    s_beta[j] = p.beta ? p.beta[j] : 0.f;
  }
  if (tiled_tail) {
    for (int j = tid; j <= p.batch; j += kStreamThreads) s_cp[j] = p.cu_pairs[j];
    for (int j = tid; j < p.batch; j += kStreamThreads) {
      s_len[j] = p.cu_seqlens[j + 1] - p.cu_seqlens[j];
      s_pad[j] = p.cu_pad[j];
    }
  }
  __syncthreads();                                // tables visible before the first tile

  // ---- stage 1: LayerNorm of tile i's rows into Xs[i & 1] ------------------
  auto ln_stage = [&](int i, XV (&cur)[NV]) {
    const int tile = tile_of(i);
    bf16* xs = Xs[i & 1];
    float v[EPT];
#pragma unroll
    for (int vv = 0; vv < NV; ++vv) XStage<XT>::unpack(cur[vv], v + vv * VX);
    const bool valid = tile * TR + srow < p.rows;
    if (p.gamma) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < EPT; ++e) s += v[e];
      const float mean = group_sum<TPR>(s) / (float)K;
      float q = 0.f;
#pragma unroll
      for (int e = 0; e < EPT; ++e) { const float d = v[e] - mean; q += d * d; }
      const float rstd = valid ? rsqrtf(group_sum<TPR>(q) / (float)K + p.eps) : 0.f;
#pragma unroll
      for (int e = 0; e < EPT; e += 4) {
        const float4 ga = *reinterpret_cast<const float4*>(&s_gamma[spart * EPT + e]);
        const float4 be = *reinterpret_cast<const float4*>(&s_beta[spart * EPT + e]);
        v[e] = valid ? (v[e] - mean) * rstd * ga.x + be.x : 0.f;
        v[e + 1] = valid ? (v[e + 1] - mean) * rstd * ga.y + be.y : 0.f;
        v[e + 2] = valid ? (v[e + 2] - mean) * rstd * ga.z + be.z : 0.f;
        v[e + 3] = valid ? (v[e + 3] - mean) * rstd * ga.w + be.w : 0.f;
      }
    }
#pragma unroll
    for (int e = 0; e < EPT; e += 8) {
      bf16x8 o;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (bf16)v[e + j];
      *reinterpret_cast<bf16x8*>(&xs[srow * SKR + spart * EPT + e]) = o;
    }
    load_x(tile_of(i + PF), cur);                 // the slot is free again
  };

  // ---- stage 2: the wave's subtiles of tile i into Ys[i & 1] ---------------
  auto compute_stage = [&](int i) {
    const int tile = tile_of(i);
    const bf16* xs = Xs[i & 1];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (u % wr_n != wrow) continue;
      bf16x8 xf[KT];
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) xf[kk] = *reinterpret_cast<const bf16x8*>(&xs[(u * 16 + l16) * SKR + kk * 32 + g * 8]);
      f32x4 acc[NTW];
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (wcol + wc * j < nt16) {
#pragma unroll
          for (int kk = 0; kk < KT; ++kk) acc[j] = mfma16(wf[j][kk], xf[kk], acc[j]);
        }
      }
      const int rl = u * 16 + l16, m = tile * TR + rl;
      if (m >= p.rows) continue;
      int32_t tpos = m;
      if (tiled_tail) tpos = tiled_pos_lds(s_cp, s_len, s_pad, p.batch, m, transposed);
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int n = (wcol + wc * j) * 16 + 4 * g;
        if (n >= p.N) continue;
        const float4 bq = *reinterpret_cast<const float4*>(&s_bias[n]);
        float r[4] = {acc[j][0] + bq.x, acc[j][1] + bq.y, acc[j][2] + bq.z, acc[j][3] + bq.w};
        if constexpr (EPI == NT_EPI_GELU) {
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) r[ii] = gelu_erf(r[ii]);
        }
        if (stage && n + 4 <= p.n_main) {
          if constexpr (RES) *reinterpret_cast<float4*>(&ysf(i & 1)[rl * NS + n]) = make_float4(r[0], r[1], r[2], r[3]);
          else {
            bf16x4 o;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) o[ii] = (bf16)r[ii];
            *reinterpret_cast<bf16x4*>(&ysb(i & 1)[rl * NS + n]) = o;
          }
        } else if (n + 4 <= p.n_main) {
          if constexpr (RES) {
            const uint2 q2 = *reinterpret_cast<const uint2*>(p.res + (int64_t)m * p.ld_res + n);
            r[0] += __uint_as_float(q2.x << 16); r[1] += __uint_as_float(q2.x & 0xffff0000u);
            r[2] += __uint_as_float(q2.y << 16); r[3] += __uint_as_float(q2.y & 0xffff0000u);
          }
          bf16x4 o;
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) o[ii] = (bf16)r[ii];
          *reinterpret_cast<bf16x4*>(p.y + (int64_t)m * p.ldy + n) = o;
        } else {
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) {
            const int nn = n + ii;
            if (nn >= p.N) break;
            if (nn < p.n_main) {
              float val = r[ii];
              if constexpr (RES) val += (float)p.res[(int64_t)m * p.ld_res + nn];
              p.y[(int64_t)m * p.ldy + nn] = (bf16)val;
            } else {
              p.y_tail[(int64_t)(nn - p.n_main) * p.ld_tail + tpos] = (bf16)r[ii];
            }
          }
        }
      }
    }
  };

  // ---- stage 3: staged write-back of tile i, 16 contiguous bytes per lane --
  auto wb_stage = [&](int i) {
    const int tile = tile_of(i);
    bf16* ytile = p.y + (int64_t)tile * TR * p.ldy;
#pragma unroll
    for (int c = 0; c < OCH; ++c) {
      const int row = wb_row[c], col = wb_col[c];
      if (row >= TR || tile * TR + row >= p.rows) continue;
      bf16x8 o;
      if constexpr (RES) {
        const float* ys = ysf(i & 1);
        const float4 a0 = *reinterpret_cast<const float4*>(&ys[row * NS + col]);
        const float4 a1 = *reinterpret_cast<const float4*>(&ys[row * NS + col + 4]);
        const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        float rv[8];
        XStage<bf16>::unpack(rres[c], rv);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (bf16)(av[e] + rv[e]);
      } else {
        o = *reinterpret_cast<const bf16x8*>(&ysb(i & 1)[row * NS + col]);
      }
      *reinterpret_cast<bf16x8*>(ytile + row * p.ldy + col) = o;
    }
    load_res(tile_of(i + 1));
  };

  // ---- per tile: normalise (and prefetch) | barrier | matrix cores into the
  // staged tile | barrier | coalesced write-back
  int n_my = 0;
  while (tile_of(n_my) < p.ntiles) ++n_my;
  auto body = [&](int i, XV (&cur)[NV]) {
    ln_stage(i, cur);
    __syncthreads();
    compute_stage(i);
    if (stage) {
      __syncthreads();
      wb_stage(i);
    }
  };
  for (int i = 0; i < n_my;) {
    body(i++, xr[0]);
    if constexpr (PF > 1) { if (i < n_my) body(i++, xr[1]); }
    if constexpr (PF > 2) { if (i < n_my) body(i++, xr[2]); }
  }
}

// ---------------------------------------------------------------- wave-streamed
// Projection for bf16 rows, K in {64, 128}, a row-major main output and an
// optional channel-major tail, with no workgroup barrier after set-up: the
// weights of all output columns sit in LDS as matrix-core fragment images
// (copied once per workgroup), and every wave streams its own 16-row tiles
// -- rows loaded straight into B-fragment order one tile ahead,
// LayerNorm in registers (a row's K values are spread over the four lanes
// l16 + 16 g, two lane swaps per statistic), the products over groups of 8
// column tiles, and a write-back through a wave-private LDS stage so that
// global stores are row-contiguous 16-byte pieces.  Waves of one CU thus
// never wait for each other; per tile a wave reads the weights from LDS once
// per 16 rows.
constexpr int kWaveThreads = 512;
constexpr int kWaveGroup = 8;                     // column tiles per product group (128 columns)
// Outputs of one column group (G = 1) and the tail tiles are written without
// a loop of run-time trip count: such a loop that stores makes the compiler
// wait for every load in flight (the next tile's rows) before entering it.
// Wider outputs (G > 1) keep the group loop and that wait.
constexpr int kWaveMaxGroups = 4;                 // main columns up to 512
constexpr int kWaveMaxTail = 2;                   // channel-major tail up to 32 channels

// residual epilogues stage fp32 values; the others bf16.  Row strides of
// 132 floats and 136 bf16 put rows 4 banks apart (mod 64): the 8-byte writes
// of 16 rows x 2 lane groups and the 16-byte write-back reads of a row both
// fall on distinct banks
template <int EPI> constexpr bool wave_res() { return EPI == NT_EPI_RESIDUAL || EPI == NT_EPI_GATED_RESIDUAL; }
template <int EPI> constexpr int wave_stage_stride() { return wave_res<EPI>() ? 132 : 136; }
template <int EPI> constexpr int wave_stage_bytes() {
  return 16 * wave_stage_stride<EPI>() * (wave_res<EPI>() ? 4 : 2);
}
template <int K, int EPI> size_t wave_smem_bytes(int nt16) {
  return (size_t)nt16 * (K / 32) * 1024 + (size_t)nt16 * 16 * 4 + 2 * (size_t)K * 4 +
         (size_t)(kWaveThreads / 64) * wave_stage_bytes<EPI>();
}

// With BC the rows are not read from x: row m = cell(i, a, b) of a pair layout
// is the pair broadcast u[eta_i + a] + v[eta_i + b] (fp32 sum rounded to bf16,
// exactly what the broadcast op stores), built as the tile is loaded.  A tile
// is then 16 cells of one pair row (the last of a row masked), so u is one
// row per tile and v rows follow the lane; each wave takes a contiguous range
// of tiles and walks it with wave-uniform (sample, pair row, column tile)
// counters.  (A per-lane cursor that wraps across pair rows makes the
// compiler copy the prefetched rows out of their load registers, which waits
// for the loads and defeats the prefetch.)
template <int EPI, int K, bool BC, int G>
__global__ void __launch_bounds__(kWaveThreads, 1) linear_wave_kernel(LinArgs p) {
  constexpr bool GATE = EPI == NT_EPI_GATED_RESIDUAL;  // residual + sigmoid(gate) * product
  constexpr bool RES = wave_res<EPI>();
  static_assert(!BC || !RES, "the broadcast rows use the residual buffers");
  constexpr int KT = K / 32;
  constexpr int SS = wave_stage_stride<EPI>();
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  const int nt16 = (p.N + 15) >> 4;
  bf16* Wimg = reinterpret_cast<bf16*>(smem_raw);                         // [nt16][KT] fragment images
  float* s_bias = reinterpret_cast<float*>(smem_raw + (size_t)nt16 * KT * 1024);
  float* s_gamma = s_bias + nt16 * 16;
  float* s_beta = s_gamma + K;
  unsigned char* stage_base = reinterpret_cast<unsigned char*>(s_beta + K);
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  const bf16* x = static_cast<const bf16*>(p.x);

  // ---- set-up: weight images (rows past N repeat row N-1; their channels
  // are never stored), bias, LayerNorm affine
  for (int im = wave; im < nt16 * KT; im += kWaveThreads / 64) {
    const int ct = im / KT, kk = im % KT;
    const int n = min(ct * 16 + l16, p.N - 1);
    const bf16* src = p.w + (int64_t)n * K + kk * 32 + g * 8;
    __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(Wimg + im * 512), 16, 0, 0);
  }
  for (int j = tid; j < nt16 * 16; j += kWaveThreads) s_bias[j] = (p.bias && j < p.N) ? p.bias[j] : 0.f;
  for (int j = tid; j < K; j += kWaveThreads) {
    s_gamma[j] = p.gamma ? p.gamma[j] : 1.f;
    s_beta[j] = p.beta ? p.beta[j] : 0.f;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const int ntile = (p.rows + 15) >> 4;
  const int wid = (int)blockIdx.x * (kWaveThreads / 64) + wave;
  const int nw = (int)gridDim.x * (kWaveThreads / 64);
  unsigned char* stage = stage_base + (size_t)wave * wave_stage_bytes<EPI>();
  const int c8n = p.n_main / 8;                   // 16-byte chunks per output row

  // broadcast walk (uniform across the wave): sample w_i with N_i = w_n,
  // first single row w_vb and first pair cell w_cup; pair row w_a, column
  // tile w_ct.  Sample tables are read only when the walk enters a sample.
  int w_i = 0, w_n = 1, w_vb = 0, w_cup = 0, w_a = 0, w_ct = 0;
  auto bc_sample = [&](int i) {
    w_i = i;
    w_vb = __builtin_amdgcn_readfirstlane(p.cu_seqlens[i]);
    w_n = __builtin_amdgcn_readfirstlane(p.cu_seqlens[i + 1]) - w_vb;
    w_cup = __builtin_amdgcn_readfirstlane(p.cu_pairs[i]);
  };
  auto bc_start = [&](int t) {
    int lo = 0, hi = p.batch;                   // bc_cu_tiles[lo] <= t < bc_cu_tiles[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.bc_cu_tiles[mid] <= t) lo = mid;
      else hi = mid;
    }
    lo = __builtin_amdgcn_readfirstlane(lo);
    bc_sample(lo);
    const int loc = t - __builtin_amdgcn_readfirstlane(p.bc_cu_tiles[lo]), ctn = (w_n + 15) >> 4;
    w_a = loc / ctn;
    w_ct = loc - w_a * ctn;
  };
  auto bc_advance = [&]() {                     // to the next tile (stays on the last one at the end)
    if (++w_ct * 16 >= w_n) {
      w_ct = 0;
      if (++w_a == w_n) {
        w_a = 0;
        int i = w_i + 1;
        while (i < p.batch && p.cu_seqlens[i + 1] == p.cu_seqlens[i]) ++i;
        if (i < p.batch) bc_sample(__builtin_amdgcn_readfirstlane(i));
        else { w_a = w_n - 1; w_ct = (w_n - 1) >> 4; }
      }
    }
  };

  // rows of tile t in B-fragment order: lane (l16, g) holds row 16t + l16,
  // k = 32 kk + 8 g .. +7; residual rows in write-back order (4 chunks a lane);
  // broadcast sources: u in xr, v in rr (the walk is at the tile).  m0 and nv:
  // the tile's first output row and its rows
  auto load_tile = [&](int t, uint4 (&xr)[KT], uint4 (&rr)[4], uint4 (&gr)[4], int64_t& m0, int& nv) {
    if constexpr (BC) {
      static_assert(KT <= 4, "v rows fit the residual buffers");
      const bf16* su = p.bc_u + (int64_t)(w_vb + w_a) * p.ld_bc_u + g * 8;
      const bf16* sv = p.bc_v + (int64_t)(w_vb + min(w_ct * 16 + l16, w_n - 1)) * p.ld_bc_v + g * 8;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        xr[kk] = *reinterpret_cast<const uint4*>(su + kk * 32);
        rr[kk] = *reinterpret_cast<const uint4*>(sv + kk * 32);
      }
      m0 = (int64_t)w_cup + (int64_t)w_a * w_n + w_ct * 16;
      nv = min(16, w_n - w_ct * 16);
      bc_advance();
      return;
    }
    m0 = (int64_t)t * 16;
    nv = min(16, p.rows - t * 16);
    // unconditional loads from rows clamped to the last one (rows past the
    // end are masked by the LayerNorm or never stored): a load under a lane
    // predicate would write zeros into registers that may still be awaiting
    // an earlier load, and the compiler then waits for every load in flight
    const int m = min(t * 16 + l16, p.rows - 1);
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) xr[kk] = *reinterpret_cast<const uint4*>(x + (int64_t)m * p.ldx + kk * 32 + g * 8);
    if constexpr (RES) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = q * 4 + (lane >> 4), cc = max(min(lane & 15, c8n - 1), 0), mm = min(t * 16 + row, p.rows - 1);
        rr[q] = *reinterpret_cast<const uint4*>(p.res + (int64_t)mm * p.ld_res + cc * 8);
        if constexpr (GATE) gr[q] = *reinterpret_cast<const uint4*>(p.gate + (int64_t)mm * p.ld_gate + cc * 8);
      }
    }
  };

  auto process = [&](int64_t m0, int nv, const uint4 (&xr_in)[KT], const uint4 (&rr)[4], const uint4 (&gr)[4]) {
    const int64_t m = m0 + l16;
    const bool mv = l16 < nv;
    uint4 xr[KT];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) xr[kk] = xr_in[kk];
    if constexpr (BC) {
      // the broadcast cell, rounded to bf16 as the broadcast op stores it
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        float a[8], b[8];
        XStage<bf16>::unpack(xr_in[kk], a);
        XStage<bf16>::unpack(rr[kk], b);
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (bf16)(a[e] + b[e]);
        xr[kk] = __builtin_bit_cast(uint4, o);
      }
    }
    // ---- LayerNorm (or plain conversion) into B fragments
    bf16x8 xb[KT];
    if (p.gamma) {
      // affine first: its LDS reads overlap the statistics
      float4 ga[KT][2], be[KT][2];
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int k0 = kk * 32 + g * 8;
        ga[kk][0] = *reinterpret_cast<const float4*>(&s_gamma[k0]);
        ga[kk][1] = *reinterpret_cast<const float4*>(&s_gamma[k0 + 4]);
        be[kk][0] = *reinterpret_cast<const float4*>(&s_beta[k0]);
        be[kk][1] = *reinterpret_cast<const float4*>(&s_beta[k0 + 4]);
      }
      float v[KT][8];
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) XStage<bf16>::unpack(xr[kk], v[kk]);
      float s = 0.f;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk)
#pragma unroll
        for (int e = 0; e < 8; ++e) s += v[kk][e];
      const float mean = sum_over_kgroups(s) / (float)K;
      float q = 0.f;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk)
#pragma unroll
        for (int e = 0; e < 8; ++e) { const float d = v[kk][e] - mean; q += d * d; }
      const float rstd = rsqrtf(sum_over_kgroups(q) / (float)K + p.eps);
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const float gg[8] = {ga[kk][0].x, ga[kk][0].y, ga[kk][0].z, ga[kk][0].w, ga[kk][1].x, ga[kk][1].y, ga[kk][1].z, ga[kk][1].w};
        const float bb[8] = {be[kk][0].x, be[kk][0].y, be[kk][0].z, be[kk][0].w, be[kk][1].x, be[kk][1].y, be[kk][1].z, be[kk][1].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) xb[kk][e] = (bf16)(mv ? (v[kk][e] - mean) * rstd * gg[e] + bb[e] : 0.f);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) xb[kk] = __builtin_bit_cast(bf16x8, xr[kk]);
    }
    // ---- main columns, group by group of 8 column tiles
    const int nmt = (p.n_main + 15) >> 4;
    auto group = [&](int cg) __attribute__((always_inline)) {
      f32x4 acc[kWaveGroup];
#pragma unroll
      for (int j = 0; j < kWaveGroup; ++j) {
        const int ct = cg * kWaveGroup + j;
        if (ct >= nmt) break;
        acc[j] = *reinterpret_cast<const f32x4*>(&s_bias[ct * 16 + 4 * g]);
#pragma unroll
        for (int kk = 0; kk < KT; ++kk)
          acc[j] = mfma16(*reinterpret_cast<const bf16x8*>(&Wimg[(ct * KT + kk) * 512 + lane * 8]), xb[kk], acc[j]);
        if (j & 1) __builtin_amdgcn_sched_barrier(0);   // two column tiles of weight fragments in flight
      }
      // acc[j][i]: channel 16 ct + 4g + i of row m, staged
#pragma unroll
      for (int j = 0; j < kWaveGroup; ++j) {
        const int ct = cg * kWaveGroup + j;
        if (ct >= nmt) break;
        const int n = ct * 16 + 4 * g;
        if (n >= p.n_main) continue;              // n_main % 8 == 0: all four are main channels
        float r[4] = {acc[j][0], acc[j][1], acc[j][2], acc[j][3]};
        if constexpr (EPI == NT_EPI_GELU) {
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) r[ii] = gelu_erf(r[ii]);
        }
        if constexpr (RES) *reinterpret_cast<float4*>(stage + (size_t)(l16 * SS + j * 16 + 4 * g) * 4) = make_float4(r[0], r[1], r[2], r[3]);
        else {
          bf16x4 o;
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) o[ii] = (bf16)r[ii];
          *reinterpret_cast<bf16x4*>(stage + (size_t)(l16 * SS + j * 16 + 4 * g) * 2) = o;
        }
      }
      // write-back of the group's main columns: lane L, pass q -> row
      // 4q + L/16, 8 columns from 8 (L % 16); four rows per store instruction
      const int cc = lane & 15, col = cg * 128 + cc * 8;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = q * 4 + (lane >> 4);
        const int64_t mm = m0 + row;
        if (col >= p.n_main || row >= nv) continue;
        bf16x8 o;
        if constexpr (RES) {
          const float* sf = reinterpret_cast<const float*>(stage) + row * SS + cc * 8;
          const float4 a0 = *reinterpret_cast<const float4*>(sf), a1 = *reinterpret_cast<const float4*>(sf + 4);
          const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
          float rv[8];
          XStage<bf16>::unpack(rr[q], rv);
          if constexpr (GATE) {
            float gv[8];
            XStage<bf16>::unpack(gr[q], gv);
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (bf16)(av[e] * sigmoid_gate(gv[e]) + rv[e]);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (bf16)(av[e] + rv[e]);
          }
        } else {
          o = *reinterpret_cast<const bf16x8*>(stage + (size_t)(row * SS + cc * 8) * 2);
        }
        // Non-temporal: measured on the pair block, streaming these outputs
        // past the caches leaves the memory-side cache to the next kernels
        // (row attention 158 -> 146 us; the projections themselves unchanged).
        store_nt(p.y + mm * p.ldy + col, o);
      }
    };
    if constexpr (G == 1) group(0);
    else
      for (int cg = 0; cg * kWaveGroup < nmt; ++cg) group(cg);
    // ---- tail columns (channel-major planes), column tile by column tile
    if (p.y_tail) {
#pragma unroll
      for (int jt = 0; jt < kWaveMaxTail; ++jt) {
        const int ct = (p.n_main >> 4) + jt;
        if (ct >= nt16) break;
        f32x4 acc = *reinterpret_cast<const f32x4*>(&s_bias[ct * 16 + 4 * g]);
#pragma unroll
        for (int kk = 0; kk < KT; ++kk)
          acc = mfma16(*reinterpret_cast<const bf16x8*>(&Wimg[(ct * KT + kk) * 512 + lane * 8]), xb[kk], acc);
        if (!mv) continue;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int nn = ct * 16 + 4 * g + ii;
          float r = acc[ii];
          if constexpr (EPI == NT_EPI_GELU) r = gelu_erf(r);
          if (nn >= p.n_main && nn < p.N) p.y_tail[(int64_t)(nn - p.n_main) * p.ld_tail + m] = (bf16)r;
        }
      }
    }
  };

  // tiles: strided over the waves, or with BC a contiguous range per wave
  const int nT = BC ? p.bc_ntiles : ntile;
  const int t0 = BC ? (int)((int64_t)nT * wid / nw) : wid;
  const int t1 = BC ? (int)((int64_t)nT * (wid + 1) / nw) : ntile;
  const int ts = BC ? 1 : nw;
  if (t0 >= t1) return;                         // (no barrier follows)
  if constexpr (BC) bc_start(t0);
  // Two register slots, each step issuing the next tile's loads before it
  // processes the current one: the compiler's wait counts treat loads
  // carried around a loop as just issued, so a tile consumed in the step
  // after its loads would wait for everything in flight; loads issued in the
  // same step before the first use stay outstanding.  Past the end the
  // loads repeat valid rows and are never used.
  uint4 xa[KT], ra[4], ga[4], xb[KT], rb[4], gb[4];
  int64_t ma, mb;
  int na, nb;
  load_tile(t0, xa, ra, ga, ma, na);
  for (int t = t0; t < t1; t += 2 * ts) {
    load_tile(t + ts, xb, rb, gb, mb, nb);
    process(ma, na, xa, ra, ga);
    if (t + ts >= t1) break;
    load_tile(t + 2 * ts, xa, ra, ga, ma, na);
    process(mb, nb, xb, rb, gb);
  }
}

// ---------------------------------------------------------------- tiled output
// Projection whose every output column goes to a pair-tiled plane (the
// triangle operands).  A workgroup tile is one 128-element chunk of the
// planes: rows r = 0..15 and k = 8*gk .. 8*gk+7 of fragment tile (rt, kt) of
// one sample, i.e. 128 cells gathered from 16 pair rows (8 consecutive cells
// each; transposed: 8 pair rows, 16 cells each).  Tile rows are ordered
// kk*16 + r, so the wave's 16-row subtile kk holds k-offset kk for all 16 r
// and after the 8 subtiles each lane holds the 8 consecutive k of its row r
// for every channel it owns: one 16-byte store per channel, and the 16 lanes
// of a channel write 256 contiguous bytes.  Chunk t of the planes is tile t,
// so tiles run over [0, sum_pad/128) and padding cells get bias-only values.
// GLU (K = 128, N = 512 product columns, 256 outputs): the weight rows are
// [a_p; a_g; b_p; b_g] of 128 each, and output channel c of part q (a or b)
// is sigmoid(g) * p of product columns 256 q + c and 256 q + 128 + c.  With
// wave w owning column tiles w + 8 j, j = 0..3, a wave holds both columns of
// every output it writes (j = 0, 1 for a; 2, 3 for b), so the gate is applied
// in registers and only the gated operands are stored.
constexpr int kTiledRows = 128;

template <int K, int NTW, bool GLU = false>
__global__ void __launch_bounds__(kStreamThreads, 1) linear_tiled_kernel(LinArgs p) {
  static_assert(!GLU || (K == 128 && NTW == 4), "the gated-operand instance takes 4 x 128 product columns");
  constexpr int TR = kTiledRows;
  constexpr int SKR = frag_stride<K>();
  constexpr int KT = K / 32;
  constexpr int TPR = kStreamThreads / TR;        // 4 staging threads per row
  constexpr int EPT = K / TPR;
  constexpr int NV = EPT / 8;
  __shared__ __attribute__((aligned(16))) bf16 Xs[2][TR * SKR];
  __shared__ int32_t s_pad[kStreamMaxSamples + 1], s_cp[kStreamMaxSamples], s_len[kStreamMaxSamples];
  __shared__ __attribute__((aligned(16))) float s_gamma[K], s_beta[K];     // LayerNorm affine

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int nt16 = (p.N + 15) >> 4;
  const bf16* x = static_cast<const bf16*>(p.x);
  const bool transposed = p.tail_mode == kTailPairTiledT;
  int tile = blockIdx.x;
  if (tile >= p.ntiles) return;
  for (int j = tid; j <= p.batch; j += kStreamThreads) s_pad[j] = p.cu_pad[j];
  for (int j = tid; j < p.batch; j += kStreamThreads) {
    s_cp[j] = p.cu_pairs[j];
    s_len[j] = p.cu_seqlens[j + 1] - p.cu_seqlens[j];
  }
  for (int j = tid; j < K; j += kStreamThreads) {
    s_gamma[j] = p.gamma ? p.gamma[j] : 1.f;
    s_beta[j] = p.beta ? p.beta[j] : 0.f;
  }
  __syncthreads();

  // packed row of tile row `row` of tile t, or -1 for a padding cell
  auto cell_row = [&](int t, int row) -> int {
    const int e = t * TR;
    int lo = 0, hi = p.batch - 1;                 // sample whose plane holds chunk t
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_pad[mid] <= e) lo = mid; else hi = mid - 1;
    }
    const int n = s_len[lo], nkt = (n + 31) >> 5;
    const int tl = (e - s_pad[lo]) / TR;          // chunk index inside the plane
    const int gk = tl & 3, kt = (tl >> 2) % nkt, rt = (tl >> 2) / nkt;
    const int rr = 16 * rt + (row & 15), kk = 32 * kt + 8 * gk + (row >> 4);
    const int a = transposed ? kk : rr, b = transposed ? rr : kk;
    return (a < n && b < n) ? s_cp[lo] + a * n + b : -1;
  };

  const int srow = tid / TPR, spart = tid % TPR;
  // a tile row's input: padding cells load row 0 and are zeroed when staged
  // (a load under a lane predicate would zero registers that may await an
  // earlier load, and the compiler then waits for every load in flight)
  auto load_x = [&](int t, uint4 (&xr)[NV], bool& valid) {
    const int m = cell_row(t, srow);
    valid = m >= 0;
    const int64_t mm = valid ? m : 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) xr[v] = *reinterpret_cast<const uint4*>(x + mm * p.ldx + spart * EPT + v * 8);
  };

  bf16x8 wf[NTW][KT];
  float bv[NTW][4];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    const int ct = wave + 8 * j, n = ct * 16 + l16;
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      if (ct < nt16 && n < p.N) wf[j][kk] = *reinterpret_cast<const bf16x8*>(p.w + (int64_t)n * K + kk * 32 + g * 8);
      else wf[j][kk] = bf16x8{};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int nb = ct * 16 + 4 * g + i;
      bv[j][i] = (p.bias && nb < p.N) ? p.bias[nb] : 0.f;
    }
  }

  // Each step issues the next tile's loads before it stages the current
  // one (two register sets): loads carried around a loop are treated by the
  // compiler as just issued, so consuming them first would wait for
  // everything in flight.  The barrier after staging waits for the LDS writes
  // only (__syncthreads would also wait for the loads just issued).
  uint4 xa[NV], xb[NV];
  bool va, vb;
  load_x(tile, xa, va);
  auto step = [&](int it, uint4 (&cur)[NV], bool vcur, uint4 (&nxt)[NV], bool& vnxt) __attribute__((always_inline)) {
    const int next = tile + (int)gridDim.x;
    load_x(next < p.ntiles ? next : tile, nxt, vnxt);   // unconditional: see above (unused past the end)
    bf16* xs = Xs[it & 1];
    {
      float v[EPT];
#pragma unroll
      for (int vv = 0; vv < NV; ++vv) XStage<bf16>::unpack(cur[vv], v + vv * 8);
      if (!vcur) {
#pragma unroll
        for (int e = 0; e < EPT; ++e) v[e] = 0.f;
      }
      if (p.gamma) {                              // padding cells (zero rows) normalise to beta
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < EPT; ++e) s += v[e];
        const float mean = group_sum<TPR>(s) / (float)K;
        float q = 0.f;
#pragma unroll
        for (int e = 0; e < EPT; ++e) { const float d = v[e] - mean; q += d * d; }
        const float rstd = rsqrtf(group_sum<TPR>(q) / (float)K + p.eps);
#pragma unroll
        for (int e = 0; e < EPT; e += 4) {
          const float4 ga = *reinterpret_cast<const float4*>(&s_gamma[spart * EPT + e]);
          const float4 be = *reinterpret_cast<const float4*>(&s_beta[spart * EPT + e]);
          v[e] = (v[e] - mean) * rstd * ga.x + be.x;
          v[e + 1] = (v[e + 1] - mean) * rstd * ga.y + be.y;
          v[e + 2] = (v[e + 2] - mean) * rstd * ga.z + be.z;
          v[e + 3] = (v[e + 3] - mean) * rstd * ga.w + be.w;
        }
      }
#pragma unroll
      for (int e = 0; e < EPT; e += 8) {
        bf16x8 o;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = (bf16)v[e + j];
        *reinterpret_cast<bf16x8*>(&xs[srow * SKR + spart * EPT + e]) = o;
      }
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);          // lgkmcnt(0): this thread's LDS writes done
    __builtin_amdgcn_s_barrier();

    // 8 subtiles (k-offsets); lane (r = l16, g) collects k-offsets 0..7 of
    // channels 4g..4g+3 of each owned column tile
    constexpr int NH = GLU ? NTW / 2 : NTW;       // output column tiles held
    bf16x8 hold[NH][4];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      bf16x8 xf[KT];
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) xf[kk] = *reinterpret_cast<const bf16x8*>(&xs[(u * 16 + l16) * SKR + kk * 32 + g * 8]);
      if constexpr (GLU) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          f32x4 ap = f32x4{0.f, 0.f, 0.f, 0.f}, ag = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < KT; ++kk) {
            ap = mfma16(wf[2 * q][kk], xf[kk], ap);
            ag = mfma16(wf[2 * q + 1][kk], xf[kk], ag);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i)
            hold[q][i][u] = (bf16)((ap[i] + bv[2 * q][i]) * sigmoid_gate(ag[i] + bv[2 * q + 1][i]));
        }
      } else {
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
          if (wave + 8 * j < nt16) {
#pragma unroll
            for (int kk = 0; kk < KT; ++kk) acc = mfma16(wf[j][kk], xf[kk], acc);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) hold[j][i][u] = (bf16)(acc[i] + bv[j][i]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NH; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // GLU: output channel 128 q + 16 wave + 4 g + i of the two gated operands
        const int c = GLU ? j * 128 + wave * 16 + 4 * g + i : (wave + 8 * j) * 16 + 4 * g + i;
        if (GLU || c < p.N)
          *reinterpret_cast<bf16x8*>(p.y_tail + (int64_t)c * p.ld_tail + (int64_t)tile * TR + 8 * l16) = hold[j][i];
      }
    tile = next;
  };
  for (int it = 0; tile < p.ntiles; it += 2) {
    step(it, xa, va, xb, vb);
    if (tile >= p.ntiles) break;
    step(it + 1, xb, vb, xa, va);
  }
}

// ---------------------------------------------------------------- SwiGLU
// Pre-normalised SwiGLU transition (Eq. running-block, second line):
//   y = res + (silu(LN(x) Wg^T + bg) * (LN(x) Wu^T + bu)) Wd^T + bd.
// One workgroup owns 64*MT rows; each wave keeps its normalised rows as
// matrix-core B fragments in registers, walks the hidden width in chunks of
// 32, and feeds the gated hidden chunk straight from the first product's
// accumulators into the second product (same lane layout), so the hidden
// activations never leave registers.
struct SwiArgs {
  int rows, K, F, N;
  const bf16* x;
  int64_t ldx;
  const float* gamma;
  const float* beta;
  float eps;
  const bf16* w;       // [2F, K]: gate rows then up rows
  const float* bias;   // [2F] or NULL
  const bf16* w2;      // [N, F]
  const float* bias2;  // [N] or NULL
  const bf16* res;
  int64_t ld_res;
  bf16* y;
  int64_t ldy;
};

template <int MT, int K, int N>
__global__ void __launch_bounds__(256) swiglu_kernel(SwiArgs p) {
  constexpr int RW = 4 * MT * 16;                 // rows per workgroup
  constexpr int KMAX = K, NMAX = N;
  constexpr int SD = 36;                          // down-projection chunk: 8-byte reads, 2 (mod 4) dwords
  constexpr int SKW = frag_stride<K>(), SKX = frag_stride<K>();   // 16-byte fragment rows
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int m0 = blockIdx.x * RW;

  // ---- prologue: LayerNorm of the workgroup's rows into LDS --------------
  // 16 lanes per row; every load of the workgroup's rows is issued first.
  bf16* Xn = smem;                                 // [RW][SKX]
  constexpr int KC = (K + 127) / 128;              // 16-byte vectors per lane per row
  uint4 raw[RW / 16][KC];
#pragma unroll
  for (int it = 0; it < RW / 16; ++it) {
    const int m = m0 + (tid >> 4) + 16 * it;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (l16 + 16 * c) * 8;
      raw[it][c] = (m < p.rows && k < K) ? *reinterpret_cast<const uint4*>(p.x + (int64_t)m * p.ldx + k)
                                         : make_uint4(0, 0, 0, 0);
    }
  }
#pragma unroll
  for (int it = 0; it < RW / 16; ++it) {
    const int rr = (tid >> 4) + 16 * it;
    const int m = m0 + rr;
    float v[2][8];
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      if (c < KC) {
        XStage<bf16>::unpack(raw[it][c], v[c]);
#pragma unroll
        for (int j = 0; j < 8; ++j) s += v[c][j];
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[c][j] = 0.f;
      }
    }
    const float mean = group_sum<16>(s) / (float)K;
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int k = (l16 + 16 * c) * 8;
      if (k < K) {
#pragma unroll
        for (int j = 0; j < 8; ++j) { const float d = v[c][j] - mean; q += d * d; }
      }
    }
    const float rstd = rsqrtf(group_sum<16>(q) / (float)K + p.eps);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int k = (l16 + 16 * c) * 8;
      if (k < K) {
        bf16x8 o;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          float t = (v[c][j] - mean) * rstd;
          if (p.gamma) t = t * p.gamma[k + j] + (p.beta ? p.beta[k + j] : 0.f);
          o[j] = (bf16)(m < p.rows ? t : 0.f);
        }
        *reinterpret_cast<bf16x8*>(&Xn[rr * SKX + k]) = o;
      }
    }
  }
  __syncthreads();
  constexpr int KT = K / 32;
  bf16x8 xf[MT][KMAX / 32];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int kk = 0; kk < KMAX / 32; ++kk)
      if (kk < KT) xf[mt][kk] = *reinterpret_cast<const bf16x8*>(&Xn[(wave * MT * 16 + mt * 16 + l16) * SKX + kk * 32 + g * 8]);
  __syncthreads();                                 // Xn is reused for weight chunks

  bf16* Wg = smem;                                 // [32][SKW]
  bf16* Wu = smem + 32 * SKW;                      // [32][SKW]
  bf16* Wd = smem + 64 * SKW;                      // [N][SD]
  constexpr int NT = N / 16;
  f32x4 accY[NMAX / 16][MT];
#pragma unroll
  for (int a = 0; a < NMAX / 16; ++a)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) accY[a][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // staging assignment: gate/up chunks = 64 rows x K/8 vectors, down chunk = N rows x 4 vectors
  constexpr int gu_vecs = 64 * (K / 8), d_vecs = N * 4;
  for (int f0 = 0; f0 < p.F; f0 += 32) {
    for (int t = tid; t < gu_vecs; t += 256) {
      const int r = t / (K / 8), kc = (t % (K / 8)) * 8;
      const int wrow = r < 32 ? f0 + r : p.F + f0 + (r - 32);
      const uint4 d = *reinterpret_cast<const uint4*>(p.w + (int64_t)wrow * K + kc);
      *reinterpret_cast<uint4*>(&smem[r * SKW + kc]) = d;
    }
    for (int t = tid; t < d_vecs; t += 256) {
      const int n = t >> 2, fc = (t & 3) * 8;
      const uint4 d = *reinterpret_cast<const uint4*>(p.w2 + (int64_t)n * p.F + f0 + fc);
      *reinterpret_cast<uint2*>(&Wd[n * SD + fc]) = make_uint2(d.x, d.y);     // rows are 8-byte aligned
      *reinterpret_cast<uint2*>(&Wd[n * SD + fc + 4]) = make_uint2(d.z, d.w);
    }
    __syncthreads();

    f32x4 accG[2][MT], accU[2][MT];
#pragma unroll
    for (int ft = 0; ft < 2; ++ft)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) { accG[ft][mt] = f32x4{0.f, 0.f, 0.f, 0.f}; accU[ft][mt] = accG[ft][mt]; }
#pragma unroll
    for (int kk = 0; kk < KMAX / 32; ++kk) {
      if (kk >= KT) break;
#pragma unroll
      for (int ft = 0; ft < 2; ++ft) {
        const bf16x8 ag = *reinterpret_cast<const bf16x8*>(&Wg[(ft * 16 + l16) * SKW + kk * 32 + g * 8]);
        const bf16x8 au = *reinterpret_cast<const bf16x8*>(&Wu[(ft * 16 + l16) * SKW + kk * 32 + g * 8]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          accG[ft][mt] = mfma16(ag, xf[mt][kk], accG[ft][mt]);
          accU[ft][mt] = mfma16(au, xf[mt][kk], accU[ft][mt]);
        }
      }
    }
    // gated hidden chunk, in the B-operand layout of the second product:
    // element j < 4 is hidden f0 + 4g + j, element j >= 4 is f0 + 16 + 4g + (j-4)
    float bgv[8], buv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int f = f0 + (j < 4 ? 4 * g + j : 16 + 4 * g + (j - 4));
      bgv[j] = p.bias ? p.bias[f] : 0.f;
      buv[j] = p.bias ? p.bias[p.F + f] : 0.f;
    }
    bf16x8 hv[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int ft = j >> 2, i = j & 3;
        const float gv = accG[ft][mt][i] + bgv[j];
        const float uv = accU[ft][mt][i] + buv[j];
        hv[mt][j] = (bf16)(gv / (1.f + __expf(-gv)) * uv);
      }
#pragma unroll
    for (int a = 0; a < NMAX / 16; ++a) {
      if (a >= NT) break;
      const bf16x4 lo = *reinterpret_cast<const bf16x4*>(&Wd[(a * 16 + l16) * SD + 4 * g]);
      const bf16x4 hi = *reinterpret_cast<const bf16x4*>(&Wd[(a * 16 + l16) * SD + 16 + 4 * g]);
      const bf16x8 ad = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) accY[a][mt] = mfma16(ad, hv[mt], accY[a][mt]);
    }
    __syncthreads();
  }

  // ---- epilogue: residual + bias, lane owns channels n..n+3 of row m ------
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = m0 + wave * MT * 16 + mt * 16 + l16;
    if (m >= p.rows) continue;
#pragma unroll
    for (int a = 0; a < NMAX / 16; ++a) {
      if (a >= NT) break;
      const int n = a * 16 + 4 * g;
      const uint2 rr = *reinterpret_cast<const uint2*>(p.res + (int64_t)m * p.ld_res + n);
      const float rv[4] = {__uint_as_float(rr.x << 16), __uint_as_float(rr.x & 0xffff0000u),
                           __uint_as_float(rr.y << 16), __uint_as_float(rr.y & 0xffff0000u)};
      bf16x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (bf16)(accY[a][mt][i] + (p.bias2 ? p.bias2[n + i] : 0.f) + rv[i]);
      *reinterpret_cast<bf16x4*>(p.y + (int64_t)m * p.ldy + n) = o;
    }
  }
}

// ---------------------------------------------------------------- fp32 path
// Plain fp32 FMA path (used by the fp32 workloads): RB rows per workgroup, one
// wave normalises each row into LDS, then threads compute output channels.
constexpr int RB = 4;

struct F32Args {
  int rows, K, N, n_main, F, epi;
  const float* x;
  int64_t ldx;
  const float* gamma;
  const float* beta;
  float eps;
  const float* w;
  const float* bias;
  const float* w2;
  const float* bias2;
  const float* res;
  int64_t ld_res;
  float* y;
  int64_t ldy;
  float* y_tail;
  int64_t ld_tail;
  LinArgs pair;         // only the pair-tiled tail fields are used
  const float* gate;    // NT_EPI_GATED_RESIDUAL
  int64_t ld_gate;
};

__global__ void __launch_bounds__(256) linear_f32_kernel(F32Args p) {
  extern __shared__ float fsm[];
  float* xs = fsm;                      // [RB][K]
  float* hs = fsm + RB * p.K;           // [RB][F] (SwiGLU only)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.x * RB;
  {
    const int r = wave, m = m0 + r;
    if (m < p.rows) {
      const float* row = p.x + (int64_t)m * p.ldx;
      float mean = 0.f, rstd = 1.f;
      if (p.gamma) {
        float s = 0.f;
        for (int k = lane; k < p.K; k += 64) s += row[k];
        mean = group_sum<64>(s) / (float)p.K;
        float q = 0.f;
        for (int k = lane; k < p.K; k += 64) { const float d = row[k] - mean; q += d * d; }
        rstd = 1.f / sqrtf(group_sum<64>(q) / (float)p.K + p.eps);
      }
      for (int k = lane; k < p.K; k += 64)
        xs[r * p.K + k] = p.gamma ? (row[k] - mean) * rstd * p.gamma[k] + (p.beta ? p.beta[k] : 0.f) : row[k];
    }
  }
  __syncthreads();
  if (p.epi == NT_EPI_SWIGLU_RESIDUAL) {
    for (int idx = tid; idx < RB * p.F; idx += 256) {
      const int r = idx / p.F, f = idx % p.F;
      if (m0 + r >= p.rows) continue;
      float gsum = p.bias ? p.bias[f] : 0.f, usum = p.bias ? p.bias[p.F + f] : 0.f;
      const float* wg = p.w + (int64_t)f * p.K;
      const float* wu = p.w + (int64_t)(p.F + f) * p.K;
      for (int k = 0; k < p.K; ++k) { gsum = fmaf(xs[r * p.K + k], wg[k], gsum); usum = fmaf(xs[r * p.K + k], wu[k], usum); }
      hs[r * p.F + f] = gsum / (1.f + expf(-gsum)) * usum;
    }
    __syncthreads();
    for (int idx = tid; idx < RB * p.N; idx += 256) {
      const int r = idx / p.N, n = idx % p.N, m = m0 + r;
      if (m >= p.rows) continue;
      float s = p.bias2 ? p.bias2[n] : 0.f;
      const float* wd = p.w2 + (int64_t)n * p.F;
      for (int f = 0; f < p.F; ++f) s = fmaf(hs[r * p.F + f], wd[f], s);
      p.y[(int64_t)m * p.ldy + n] = p.res[(int64_t)m * p.ld_res + n] + s;
    }
    return;
  }
  for (int idx = tid; idx < RB * p.N; idx += 256) {
    const int r = idx / p.N, n = idx % p.N, m = m0 + r;
    if (m >= p.rows) continue;
    float s = p.bias ? p.bias[n] : 0.f;
    const float* wr = p.w + (int64_t)n * p.K;
    for (int k = 0; k < p.K; ++k) s = fmaf(xs[r * p.K + k], wr[k], s);
    if (p.epi == NT_EPI_GELU) s = 0.5f * s * (1.f + erff(s * 0.70710678118654752f));
    if (n < p.n_main) {
      if (p.epi == NT_EPI_GATED_RESIDUAL) s /= 1.f + expf(-p.gate[(int64_t)m * p.ld_gate + n]);
      if (p.epi == NT_EPI_RESIDUAL || p.epi == NT_EPI_GATED_RESIDUAL) s += p.res[(int64_t)m * p.ld_res + n];
      p.y[(int64_t)m * p.ldy + n] = s;
    } else {
      const int64_t pos = p.pair.tail_mode == kTailChannelMajor ? (int64_t)m : pair_tiled_pos(p.pair, m);
      p.y_tail[(int64_t)(n - p.n_main) * p.ld_tail + pos] = s;
    }
  }
}


// One resident workgroup per slot: grid = min(tiles, resident workgroups per
// CU x CUs); every workgroup walks tiles blockIdx.x + j * gridDim.x.
template <typename XT, int EPI, int K, int NTW>
void launch_stream(const LinArgs& p, hipStream_t s) {
  const size_t smem = p.stage_out ? (size_t)kStreamRows * stage_stride(p.n_main, EPI == NT_EPI_RESIDUAL) *
                                        (EPI == NT_EPI_RESIDUAL ? 4 : 2)
                                  : 0;
  auto kern = linear_stream_kernel<XT, EPI, K, NTW>;
  (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kStreamThreads, smem) != hipSuccess || nb < 1) nb = 1;
  const int grid = std::min(p.ntiles, nb * compute_units());
  kern<<<dim3((unsigned)grid), dim3(kStreamThreads), smem, s>>>(p);
}

template <int EPI, int K, bool BC, int G>
void launch_wave_g(const LinArgs& p, hipStream_t s) {
  const int nt16 = (p.N + 15) / 16;
  const size_t smem = wave_smem_bytes<K, EPI>(nt16);
  auto kern = linear_wave_kernel<EPI, K, BC, G>;
  (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  const int ntile = (p.rows + 15) / 16;
  const int grid = std::min((ntile + kWaveThreads / 64 - 1) / (kWaveThreads / 64), compute_units());
  kern<<<dim3((unsigned)grid), dim3(kWaveThreads), smem, s>>>(p);
}

// instance by main column groups: one (up to 128 columns) or up to four
template <int EPI, int K, bool BC = false>
void launch_wave(const LinArgs& p, hipStream_t s) {
  if (p.n_main <= 16 * kWaveGroup) launch_wave_g<EPI, K, BC, 1>(p, s);
  else if constexpr (!wave_res<EPI>()) launch_wave_g<EPI, K, BC, kWaveMaxGroups>(p, s);
}

template <int K, bool GLU = false>
void launch_tiled(const LinArgs& p, hipStream_t s) {
  constexpr int NTW = GLU ? 4 : 2;
  static int per_cu = 0;
  if (per_cu == 0) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, linear_tiled_kernel<K, NTW, GLU>, kStreamThreads, 0) !=
            hipSuccess || nb < 1)
      nb = 1;
    per_cu = nb;
  }
  const int grid = std::min(p.ntiles, per_cu * compute_units());
  if (grid > 0) linear_tiled_kernel<K, NTW, GLU><<<dim3((unsigned)grid), dim3(kStreamThreads), 0, s>>>(p);
}

}  // namespace

// Compute units of the current device (cached per device).
int compute_units() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

namespace {

// The transition kernel serves a bf16 SwiGLU whose residual is x itself.
bool uses_transition(const nt_linear_args& a) {
  if (a.dtype != NT_BF16 || a.epilogue != NT_EPI_SWIGLU_RESIDUAL || a.bcast_u) return false;
  const bool res_is_x = !a.residual || (a.residual == a.x && a.ld_residual == a.ldx);
  return res_is_x && transition_supported(a.c_in, a.c_out, a.hidden);
}

// The large-K product: bf16 rows and weights, no tail, whole 16-byte rows.
bool uses_gemm(const nt_linear_args& a) {
  if (a.dtype != NT_BF16 || a.bcast_u || a.epilogue == NT_EPI_SWIGLU_RESIDUAL) return false;
  return a.x_dtype == NT_BF16 && a.n_tail == 0 && a.c_in >= 384 && a.c_in % 32 == 0 && a.c_out % 8 == 0 &&
         a.ldx % 8 == 0 && a.ldy % 8 == 0 && (a.epilogue != NT_EPI_RESIDUAL || a.ld_residual % 8 == 0) &&
         (a.epilogue == NT_EPI_NONE || a.epilogue == NT_EPI_GELU || a.epilogue == NT_EPI_RESIDUAL) &&
         gemm_fits(a.c_in) && a.c_in <= 4096;
}

}  // namespace

size_t linear_workspace_bytes(const nt_linear_args& a) {
  if (uses_transition(a)) return transition_image_bytes(a.c_in, a.hidden);
  if (uses_gemm(a) && a.ln_gamma)     // LN(x) rows written once, then read by the product
    return (size_t)a.rows * (size_t)a.c_in * sizeof(bf16);
  return 0;
}

hipError_t launch_linear(const LinearPlan& plan, hipStream_t s) {
  const nt_linear_args& a = *plan.a;
  const int rows = (int)a.rows;
  if (rows == 0) return hipSuccess;
  LinArgs p{};
  p.rows = rows; p.K = a.c_in; p.N = a.c_out; p.n_main = a.c_out - a.n_tail;
  p.x = a.x; p.ldx = a.ldx; p.gamma = a.ln_gamma; p.beta = a.ln_beta; p.eps = a.ln_eps;
  p.w = (const bf16*)a.w; p.bias = a.bias;
  p.res = (const bf16*)a.residual; p.ld_res = a.ld_residual;
  p.y = (bf16*)a.y; p.ldy = a.ldy;
  p.y_tail = (bf16*)a.y_tail; p.ld_tail = a.ld_tail; p.tail_mode = plan.tail_mode;
  if (plan.layout && plan.layout->has_device) {
    p.row_splits2 = plan.layout->d_row_splits2; p.row_sample = plan.layout->d_row_sample;
    p.cu_seqlens = plan.layout->d_cu_seqlens; p.cu_pad = plan.layout->d_cu_pad;
    p.sum_n = (int)plan.layout->sum_n;
    p.blk_prow = plan.layout->d_blk_prow;
  }
  if (a.n_tail == 0) p.y_tail = nullptr;
  p.gate = (const bf16*)a.gate; p.ld_gate = a.ld_gate;

  if (a.bcast_u) {
    // pair-broadcast rows: the wave-streamed kernel builds them from u and v
    const int nt16 = (a.c_out + 15) / 16;
    const size_t smem = a.c_in == 64 ? wave_smem_bytes<64, NT_EPI_NONE>(nt16) : wave_smem_bytes<128, NT_EPI_NONE>(nt16);
    if (smem > 150 * 1024) return hipErrorInvalidValue;
    p.bc_u = (const bf16*)a.bcast_u; p.bc_v = (const bf16*)a.bcast_v;
    p.ld_bc_u = a.ld_bcast_u; p.ld_bc_v = a.ld_bcast_v;
    p.bc_cu_tiles = plan.layout->d_bc_cu_tiles;
    p.bc_ntiles = plan.layout->bc_cu_tiles.back();
    p.cu_seqlens = plan.layout->d_cu_seqlens;
    p.cu_pairs = plan.layout->d_cu_pairs;
    p.batch = plan.layout->batch;
    p.ldx = a.c_in;
#define NT_WB(EPI) do { if (a.c_in == 64) launch_wave<EPI, 64, true>(p, s); else launch_wave<EPI, 128, true>(p, s); } while (0)
    if (a.epilogue == NT_EPI_GELU) NT_WB(NT_EPI_GELU);
    else NT_WB(NT_EPI_NONE);
#undef NT_WB
    return hipGetLastError();
  }

  if (a.dtype == NT_F32) {
    F32Args f{};
    f.rows = rows; f.K = a.c_in; f.N = a.c_out; f.n_main = p.n_main; f.F = a.hidden; f.epi = a.epilogue;
    f.x = (const float*)a.x; f.ldx = a.ldx; f.gamma = a.ln_gamma; f.beta = a.ln_beta; f.eps = a.ln_eps;
    f.w = (const float*)a.w; f.bias = a.bias; f.w2 = (const float*)a.w2; f.bias2 = a.bias2;
    f.res = a.residual ? (const float*)a.residual : (const float*)a.x;
    f.ld_res = a.residual ? a.ld_residual : a.ldx;
    f.y = (float*)a.y; f.ldy = a.ldy; f.y_tail = (float*)a.y_tail; f.ld_tail = a.ld_tail; f.pair = p;
    f.gate = (const float*)a.gate; f.ld_gate = a.ld_gate;
    const size_t smem = sizeof(float) * RB * ((size_t)a.c_in + (a.epilogue == NT_EPI_SWIGLU_RESIDUAL ? a.hidden : 0));
    linear_f32_kernel<<<dim3((rows + RB - 1) / RB), dim3(256), smem, s>>>(f);
    return hipGetLastError();
  }

  if (a.epilogue == NT_EPI_SWIGLU_RESIDUAL) {
    SwiArgs w{};
    w.rows = rows; w.K = a.c_in; w.F = a.hidden; w.N = a.c_out;
    w.x = (const bf16*)a.x; w.ldx = a.ldx; w.gamma = a.ln_gamma; w.beta = a.ln_beta; w.eps = a.ln_eps;
    w.w = (const bf16*)a.w; w.bias = a.bias; w.w2 = (const bf16*)a.w2; w.bias2 = a.bias2;
    w.res = a.residual ? (const bf16*)a.residual : (const bf16*)a.x;
    w.ld_res = a.residual ? a.ld_residual : a.ldx;
    w.y = (bf16*)a.y; w.ldy = a.ldy;
    if (uses_transition(a)) {
      TransArgs t{};
      t.rows = rows; t.K = a.c_in; t.F = a.hidden;
      t.x = w.x; t.ldx = w.ldx; t.gamma = w.gamma; t.beta = w.beta; t.eps = w.eps;
      t.w = w.w; t.bias = w.bias; t.w2 = w.w2; t.bias2 = w.bias2;
      t.y = w.y; t.ldy = w.ldy;
      return launch_transition(t, a.workspace, s);
    }
    constexpr int MT = 2;
    const int rw = 4 * MT * 16;
    const int sk = a.c_in + ((16 - a.c_in % 128) + 128) % 128;
    const size_t xn = (size_t)rw * sk;
    const size_t wc = (size_t)64 * sk + (size_t)a.c_out * 36;
    const size_t smem = sizeof(bf16) * (xn > wc ? xn : wc);
    const dim3 grid((rows + rw - 1) / rw);
    if (a.c_in == 64 && a.c_out == 64) swiglu_kernel<MT, 64, 64><<<grid, dim3(256), smem, s>>>(w);
    else if (a.c_in == 128 && a.c_out == 128) swiglu_kernel<MT, 128, 128><<<grid, dim3(256), smem, s>>>(w);
    else if (a.c_in == 256 && a.c_out == 256) swiglu_kernel<MT, 256, 256><<<grid, dim3(256), smem, s>>>(w);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }

  p.mblocks = (rows + BM - 1) / BM;
  p.nblocks = (a.c_out + BN - 1) / BN;
  const bool xf = a.x_dtype == NT_F32;

  if (a.epilogue == NT_EPI_SIGMOID_GLU) {
    // gated operands straight into pair-tiled planes (checked by the caller:
    // bf16, K = 128, hidden = 128, 256 outputs, all pair-tiled)
    p.N = 2 * a.c_out;                            // product columns
    p.n_main = 0;
    p.cu_pairs = plan.layout->d_cu_pairs;
    p.batch = plan.layout->batch;
    p.ntiles = (int)(plan.layout->sum_pad / kTiledRows);
    launch_tiled<128, true>(p, s);
    return hipGetLastError();
  }
  if (a.epilogue == NT_EPI_GATED_RESIDUAL) {
    // the wave-streamed kernel for bf16 rows of 64 or 128 features and at
    // most 128 outputs, else the generic tile kernel
    const int nt16 = (a.c_out + 15) / 16;
    const size_t smem = a.c_in == 64 ? wave_smem_bytes<64, NT_EPI_GATED_RESIDUAL>(nt16)
                                     : wave_smem_bytes<128, NT_EPI_GATED_RESIDUAL>(nt16);
    if (!xf && a.n_tail == 0 && (a.c_in == 64 || a.c_in == 128) && p.n_main % 8 == 0 && p.n_main <= 128 &&
        a.ldx % 8 == 0 && p.ldy % 8 == 0 && a.ld_residual % 8 == 0 && a.ld_gate % 8 == 0 && smem <= 150 * 1024) {
      if (a.c_in == 64) launch_wave<NT_EPI_GATED_RESIDUAL, 64>(p, s);
      else launch_wave<NT_EPI_GATED_RESIDUAL, 128>(p, s);
      return hipGetLastError();
    }
    const unsigned grid = (unsigned)(((p.mblocks + kXcds - 1) / kXcds) * kXcds * p.nblocks);
    if (xf) linear_mfma_kernel<float, NT_EPI_GATED_RESIDUAL><<<dim3(grid), dim3(256), 0, s>>>(p);
    else linear_mfma_kernel<bf16, NT_EPI_GATED_RESIDUAL><<<dim3(grid), dim3(256), 0, s>>>(p);
    return hipGetLastError();
  }

  const bool tiled = p.y_tail && p.tail_mode != kTailChannelMajor;
  if (!a.ln_gamma && a.n_tail == 0 && a.c_in % 32 == 0 && rows <= kSmallRows) {
    const dim3 g1((unsigned)((rows + 15) / 16), (unsigned)((a.c_out + 63) / 64)), b1(64 * kSmallWaves);
#define NT_SM(XT, EPI) linear_small_kernel<XT, EPI><<<g1, b1, 0, s>>>(p)
#define NT_SM_X(EPI) do { if (xf) NT_SM(float, EPI); else NT_SM(bf16, EPI); } while (0)
    switch (a.epilogue) {
      case NT_EPI_NONE: NT_SM_X(NT_EPI_NONE); break;
      case NT_EPI_RESIDUAL: NT_SM_X(NT_EPI_RESIDUAL); break;
      case NT_EPI_GELU: NT_SM_X(NT_EPI_GELU); break;
      default: return hipErrorInvalidValue;
    }
#undef NT_SM_X
#undef NT_SM
    return hipGetLastError();
  }
  if (tiled && p.n_main == 0 && !xf && a.epilogue == NT_EPI_NONE && (a.c_in == 64 || a.c_in == 128) &&
      a.c_out <= 256 && plan.layout && plan.layout->batch <= kStreamMaxSamples) {
    p.cu_pairs = plan.layout->d_cu_pairs;
    p.batch = plan.layout->batch;
    p.ntiles = (int)(plan.layout->sum_pad / kTiledRows);
    if (a.c_in == 64) launch_tiled<64>(p, s);
    else launch_tiled<128>(p, s);
    return hipGetLastError();
  }
  {
    // wave-streamed kernel: bf16 rows, a row-major main output (whole 16-byte
    // chunks) and at most a channel-major tail, weights within the LDS budget
    const bool res = a.epilogue == NT_EPI_RESIDUAL;
    const int nt16 = (a.c_out + 15) / 16;
    const size_t smem = a.c_in == 64 ? (res ? wave_smem_bytes<64, NT_EPI_RESIDUAL>(nt16) : wave_smem_bytes<64, NT_EPI_NONE>(nt16))
                                     : (res ? wave_smem_bytes<128, NT_EPI_RESIDUAL>(nt16) : wave_smem_bytes<128, NT_EPI_NONE>(nt16));
    const int main_groups = (p.n_main + 16 * kWaveGroup - 1) / (16 * kWaveGroup);
    const int tail_tiles = nt16 - p.n_main / 16;
    if (!xf && !tiled && (a.c_in == 64 || a.c_in == 128) && p.n_main % 8 == 0 && a.ldx % 8 == 0 &&
        p.ldy % 8 == 0 && (!res || (p.n_main <= 128 && a.ld_residual % 8 == 0)) && smem <= 150 * 1024 &&
        main_groups <= kWaveMaxGroups && tail_tiles <= kWaveMaxTail &&
        (a.epilogue == NT_EPI_NONE || a.epilogue == NT_EPI_GELU || res)) {
#define NT_WV(EPI) do { if (a.c_in == 64) launch_wave<EPI, 64>(p, s); else launch_wave<EPI, 128>(p, s); } while (0)
      if (res) NT_WV(NT_EPI_RESIDUAL);
      else if (a.epilogue == NT_EPI_GELU) NT_WV(NT_EPI_GELU);
      else NT_WV(NT_EPI_NONE);
#undef NT_WV
      return hipGetLastError();
    }
  }
  if ((a.c_in == 64 || a.c_in == 128) && a.c_out <= 512 &&
      (!tiled || (plan.layout && plan.layout->batch <= kStreamMaxSamples))) {
    if (tiled) { p.cu_pairs = plan.layout->d_cu_pairs; p.batch = plan.layout->batch; }
    const int nt16 = (a.c_out + 15) / 16;
    const int ntw = nt16 <= 16 ? 2 : 4;
    int wc = 2;
    while (wc < 8 && wc * ntw < nt16) wc *= 2;
    p.wc = wc;
    p.ntiles = (rows + kStreamRows - 1) / kStreamRows;
    // staged write-back: whole 16-byte chunks per row, within the LDS budget
    const bool res = a.epilogue == NT_EPI_RESIDUAL;
    const size_t stage_bytes = (size_t)kStreamRows * stage_stride(p.n_main, res) * (res ? 4 : 2);
    p.stage_out = p.n_main > 0 && p.n_main % 8 == 0 && p.ldy % 8 == 0 && (!res || a.ld_residual % 8 == 0) &&
                  p.n_main <= (res ? 256 : 32 * ntw * 8) && stage_bytes <= 108 * 1024;
#define NT_ST(XT, EPI, KK, W) launch_stream<XT, EPI, KK, W>(p, s)
#define NT_ST_W(XT, EPI, KK) do { if (ntw == 2) NT_ST(XT, EPI, KK, 2); else NT_ST(XT, EPI, KK, 4); } while (0)
#define NT_ST_K(XT, EPI) do { if (a.c_in == 64) NT_ST_W(XT, EPI, 64); else NT_ST_W(XT, EPI, 128); } while (0)
#define NT_ST_X(EPI) do { if (xf) NT_ST_K(float, EPI); else NT_ST_K(bf16, EPI); } while (0)
    switch (a.epilogue) {
      case NT_EPI_NONE: NT_ST_X(NT_EPI_NONE); break;
      case NT_EPI_RESIDUAL: NT_ST_X(NT_EPI_RESIDUAL); break;
      case NT_EPI_GELU: NT_ST_X(NT_EPI_GELU); break;
      default: return hipErrorInvalidValue;
    }
#undef NT_ST_X
#undef NT_ST_K
#undef NT_ST_W
#undef NT_ST
    return hipGetLastError();
  }
  if (uses_gemm(a)) {
    GemmArgs g{};
    g.rows = rows; g.K = a.c_in; g.N = a.c_out;
    g.x = (const bf16*)a.x; g.ldx = a.ldx; g.gamma = a.ln_gamma; g.beta = a.ln_beta; g.eps = a.ln_eps;
    g.ln_ws = (bf16*)a.workspace;
    g.w = (const bf16*)a.w; g.bias = a.bias; g.res = (const bf16*)a.residual; g.ld_res = a.ld_residual;
    g.y = (bf16*)a.y; g.ldy = a.ldy; g.epi = a.epilogue;
    return launch_gemm(g, s);
  }
  if (a.c_in == 64 || a.c_in == 128 || a.c_in == 256) {
    const dim3 g1((unsigned)p.mblocks), b1(256);
#define NT_RES(XT, EPI, KK) linear_res_kernel<XT, EPI, KK><<<g1, b1, 0, s>>>(p)
#define NT_RES_K(XT, EPI) \
    do { if (a.c_in == 64) NT_RES(XT, EPI, 64); else if (a.c_in == 128) NT_RES(XT, EPI, 128); else NT_RES(XT, EPI, 256); } while (0)
#define NT_RES_X(EPI) do { if (xf) NT_RES_K(float, EPI); else NT_RES_K(bf16, EPI); } while (0)
    switch (a.epilogue) {
      case NT_EPI_NONE: NT_RES_X(NT_EPI_NONE); break;
      case NT_EPI_RESIDUAL: NT_RES_X(NT_EPI_RESIDUAL); break;
      case NT_EPI_GELU: NT_RES_X(NT_EPI_GELU); break;
      default: return hipErrorInvalidValue;
    }
#undef NT_RES_X
#undef NT_RES_K
#undef NT_RES
    return hipGetLastError();
  }
  const unsigned grid = (unsigned)(((p.mblocks + kXcds - 1) / kXcds) * kXcds * p.nblocks);
  const bool xf32 = a.x_dtype == NT_F32;
#define NT_LAUNCH_LIN(XT, EPI) linear_mfma_kernel<XT, EPI><<<dim3(grid), dim3(256), 0, s>>>(p)
  switch (a.epilogue) {
    case NT_EPI_NONE: if (xf32) NT_LAUNCH_LIN(float, NT_EPI_NONE); else NT_LAUNCH_LIN(bf16, NT_EPI_NONE); break;
    case NT_EPI_RESIDUAL: if (xf32) NT_LAUNCH_LIN(float, NT_EPI_RESIDUAL); else NT_LAUNCH_LIN(bf16, NT_EPI_RESIDUAL); break;
    case NT_EPI_GELU: if (xf32) NT_LAUNCH_LIN(float, NT_EPI_GELU); else NT_LAUNCH_LIN(bf16, NT_EPI_GELU); break;
    default: return hipErrorInvalidValue;
  }
#undef NT_LAUNCH_LIN
  return hipGetLastError();
}

}  // namespace nt
