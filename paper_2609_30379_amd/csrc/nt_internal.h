// Host-side internals shared by the C ABI, the layout planner and the kernel
// launchers.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "nt.h"

namespace nt {

constexpr int kXcds = 8;          // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr int kTriTile = 64;      // triangle output tile: 64 x 64 cells
constexpr int kSeqQBlock = 64;    // 1-D attention: queries per workgroup
constexpr int kLinRows = 128;     // rows per projection workgroup (pair-row table granularity)
constexpr int kAttnQB = 128;      // pair attention (head_dim 32): queries per workgroup (8 waves x 16)
constexpr int kAttnRG = 16;       // pair attention (head_dim 32): pair rows per workgroup
constexpr int kAttnShortLen = 256;  // its instance with two workgroups per CU: longest sample
constexpr int kAttnLongLen = 512;   // its instance with one workgroup per CU: longest sample

// Samples whose tables the pair-tiled projection kernels cache in LDS.
constexpr int kPairTiledMaxSamples = 1024;

// Attention limits imposed by staging a whole key segment in LDS.
constexpr int kAttnMaxLenD32 = 1024;
constexpr int kAttnMaxLenD64 = 512;

}  // namespace nt

// Opaque layout object (see nt.h).  Host arrays are the canonical copies;
// device mirrors live in one allocation.
struct nt_layout {
  int32_t batch = 0;
  int32_t max_len = 0;
  int64_t sum_n = 0, sum_n2 = 0, sum_n3 = 0;
  int64_t sum_pad = 0;             // sum_i round_up(N_i,16) * round_up(N_i,32): pair-tiled plane extent
  bool rect = false;               // rectangular pairs N_i x M_i (cols differ from lengths)
  int64_t sum_m = 0;               // sum_i M_i (= sum_n for square pairs)
  std::vector<int32_t> cols;         // [B] M_i
  std::vector<int32_t> cu_cols;      // [B+1] column offsets kappa
  std::vector<int32_t> col_sample;   // [sum M] sample id of every column

  std::vector<int32_t> lengths;      // [B]
  std::vector<int32_t> cu_seqlens;   // [B+1]
  std::vector<int32_t> cu_pairs;     // [B+1]
  std::vector<int32_t> cu_pad;       // [B+1] offsets P_i of the pair-tiled operand planes
  std::vector<int32_t> row_splits2;  // [sum N + 1]
  std::vector<int32_t> row_sample;   // [sum N]
  std::vector<int32_t> attn_work;    // pairs (sample, row); count multiple of 8; (-1,-1) = idle
  std::vector<int32_t> tri_work;     // quads (sample, xt, yt, first item of the sample); count multiple of 8
  std::vector<int32_t> tri_split;    // [9] cost-balanced item ranges of the 8 XCDs
  int32_t tri_xcd_items = 0;         // largest item count of one XCD
  std::vector<int32_t> seq_work;     // pairs (sample, query block); count multiple of 8
  std::vector<int32_t> pattn_work;  // quads (sample, first 16-query tile, row group, tile count)
  std::vector<int32_t> bias_tiles;   // [B+1] prefix of ceil(N_i/16) * round_up(N_i,64)/16: bias image tiles
  std::vector<int32_t> sattn_work;   // 1-D attention: quads (sample, first 16-query tile, 0, tile count)
  std::vector<int32_t> blk_prow;     // [ceil(sum N^2 / kLinRows)] pair row holding cell kLinRows*b
  std::vector<int32_t> bc_cu_tiles;  // [B+1] prefix of N_i * ceil(N_i/16): broadcast tiles (16 cells of one pair row)
  std::vector<int32_t> cu_qblk;      // [B+1] prefix of ceil(N_i/16): 16-query blocks (attention bias gradient)

  bool has_device = false;
  int device = -1;
  void* d_base = nullptr;
  const int32_t* d_lengths = nullptr;
  const int32_t* d_cu_seqlens = nullptr;
  const int32_t* d_cu_pairs = nullptr;
  const int32_t* d_cu_pad = nullptr;
  const int32_t* d_row_splits2 = nullptr;
  const int32_t* d_row_sample = nullptr;
  const int32_t* d_attn_work = nullptr;
  const int32_t* d_tri_work = nullptr;
  const int32_t* d_seq_work = nullptr;
  const int32_t* d_pattn_work = nullptr;
  const int32_t* d_blk_prow = nullptr;
  const int32_t* d_bias_tiles = nullptr;
  const int32_t* d_sattn_work = nullptr;
  const int32_t* d_bc_cu_tiles = nullptr;
  const int32_t* d_cu_qblk = nullptr;
  const int32_t* d_tri_split = nullptr;
  const int32_t* d_cu_cols = nullptr;
  const int32_t* d_col_sample = nullptr;

  int64_t attn_items() const { return (int64_t)attn_work.size() / 2; }
  int64_t tri_items() const { return (int64_t)tri_work.size() / 4; }
  int64_t seq_items() const { return (int64_t)seq_work.size() / 2; }
  int64_t pattn_items() const { return (int64_t)pattn_work.size() / 4; }
  int64_t sattn_items() const { return (int64_t)sattn_work.size() / 4; }
  int64_t bias_tiles_total() const { return bias_tiles.empty() ? 0 : bias_tiles.back(); }
};

namespace nt {

// Large-K bf16 projection (k_gemm.hip): y = epi(LN?(x) W^T + b) for row-major
// x [rows, K], w [N, K], y [rows, N]; K % 32 == 0, N % 8 == 0, 16-byte rows.
struct GemmArgs {
  int rows, K, N;
  const __bf16* x;
  int64_t ldx;
  const float* gamma;    // LayerNorm of x when non-NULL
  const float* beta;
  float eps;
  __bf16* ln_ws;         // with gamma: rows * K bf16 of caller workspace for LN(x)
  const __bf16* w;
  const float* bias;
  const __bf16* res;     // epi == NT_EPI_RESIDUAL
  int64_t ld_res;
  __bf16* y;
  int64_t ldy;
  int epi;               // NT_EPI_NONE, NT_EPI_GELU or NT_EPI_RESIDUAL
  int ntm, ntn;          // tiles (set by the launcher)
};
bool gemm_fits(int K);
// With gamma set, the rows are first normalised into p.ln_ws.
hipError_t launch_gemm(GemmArgs p, hipStream_t s);

// SwiGLU transition with residual (k_transition.hip):
//   y = x + (silu(LN(x) W_g^T + b_g) * (LN(x) W_u^T + b_u)) W_d^T + b_d
// for x, y [rows, K] bf16, w [2F, K] (gate rows, then up rows), w2 [K, F].
constexpr int kTransitionMaxHidden = 768;
struct TransArgs {
  int rows, K, F;
  const __bf16* x;
  int64_t ldx;
  const float* gamma;    // LayerNorm affine (NULL: 1 / 0)
  const float* beta;
  float eps;
  const __bf16* w;
  const float* bias;     // [2F] or NULL
  const __bf16* w2;
  const float* bias2;    // [K] or NULL
  __bf16* y;             // may alias x
  int64_t ldy;
  const __bf16* wimg;    // set by the launcher: weights in consumption order
};
// The residual must be x itself (same rows and stride).
bool transition_supported(int K, int N, int F);
size_t transition_image_bytes(int K, int F);
// wimg_workspace: transition_image_bytes(K, F) bytes of device memory that the
// launch rewrites (weights in consumption order); calls sharing it must be ordered.
hipError_t launch_transition(TransArgs p, void* wimg_workspace, hipStream_t s);
int compute_units();


// Sets the thread-local error message and returns the status.
nt_status fail(nt_status s, const std::string& msg);

// ---- kernel launchers (return hipGetLastError() after the launch) ----------

hipError_t launch_pair_broadcast(const nt_layout& L, int C, const void* u, int64_t ld_u,
                                 const void* v, int64_t ld_v, void* z, int64_t ld_z,
                                 int accumulate, nt_dtype dtype, hipStream_t s);

// y in y_dtype (fp32 for the public reduce; bf16 for gradients handed to a product)
hipError_t launch_segment_reduce(const nt_layout& L, nt_level level, int op, int C,
                                 const void* x, int64_t ld_x, nt_dtype x_dtype,
                                 void* y, int64_t ld_y, hipStream_t s, int accumulate = 0,
                                 nt_dtype y_dtype = NT_F32);

size_t loss_workspace_bytes(const nt_layout& L);
hipError_t launch_weighted_square_loss(const nt_layout& L, nt_level level, int C, const void* x, int64_t ld_x,
                                       nt_dtype dtype, const float* w, float scale, float* loss, void* dx,
                                       int64_t ld_dx, nt_dtype dx_dtype, void* workspace, hipStream_t s);

hipError_t launch_segment_reduce_backward(const nt_layout& L, nt_level level, int op, int C, const float* dy,
                                          int64_t ld_dy, void* dx, int64_t ld_dx, nt_dtype dtype, int accumulate,
                                          hipStream_t s);

// Tail output modes of the projection (columns routed to y_tail).
enum TailMode { kTailChannelMajor = 0, kTailPairTiled = 1, kTailPairTiledT = 2 };

struct LinearPlan {
  const nt_linear_args* a;
  int tail_mode;
  const nt_layout* layout;   // for pair-tiled tail modes
};
// Workspace bytes the call needs (0: none): LN(x) rows of the large-K product
// or the transition's weight image.  Mirrors the kernel choice of launch_linear.
size_t linear_workspace_bytes(const nt_linear_args& a);
// a.workspace must hold linear_workspace_bytes(a) bytes (checked by the caller).
hipError_t launch_linear(const LinearPlan& p, hipStream_t s);

// Allocation-free attention (nt_pair_row_attention_noalloc): its scratch is a
// file-scope device array of this many bytes, one per device.
constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
// Device address of the calling thread's current device's array (looked up
// once per device).
hipError_t noalloc_scratch(void** ptr);

// LayerNorm+Linear backward (k_backward.hip): workspace bytes and launch.
size_t linear_backward_workspace_bytes(const nt_linear_bwd_args& a);
hipError_t launch_linear_backward(const nt_linear_bwd_args& a, void* ws, hipStream_t s);

// Attention backward (k_attention_backward.hip): bf16, head_dim 32, axes 0
// and 1, N_i <= 512.  Workspace: the softmax statistics of every query
// element, attention_backward_workspace_bytes(L, H) bytes.
size_t attention_backward_workspace_bytes(const nt_layout& L, int H);
hipError_t launch_attention_backward(const nt_layout& L, int axis, int H, const void* q, const void* k,
                                     const void* v, int64_t ld_qkv, const void* bias, int64_t ld_bias,
                                     int64_t ld_bias_head, const void* dout,
                                     int64_t ld_dout, float scale, void* dq, void* dk, void* dv, int64_t ld_dqkv,
                                     float* dbias, int64_t ld_dbias, int64_t ld_dbias_head, void* workspace,
                                     hipStream_t s);

// Bias-image bytes of a pair attention call (0: none).
size_t attention_workspace_bytes(const nt_layout& L, int axis, int H, int D, nt_dtype dtype, bool has_bias);
// bias element (cell c, head h) at bias[c * ld_bias + h * ld_bias_head];
// workspace: attention_workspace_bytes(...) bytes.
// gate (axes 0 and 1, or NULL): o = sigmoid(gate) * attention, gate element
// (cell, channel) at gate[cell * ld_gate + channel].
hipError_t launch_attention(const nt_layout& L, int axis, int H, int D,
                            const void* q, const void* k, const void* v, int64_t ld_qkv,
                            const void* bias, int64_t ld_bias, int64_t ld_bias_head, float scale,
                            void* o, int64_t ld_o, nt_dtype dtype, void* workspace, hipStream_t s,
                            const void* gate = nullptr, int64_t ld_gate = 0);

// Cross-attention over singles: queries by Lq's offsets, keys and values by
// Lkv's (same batch); bf16 head_dim 32 / 64 with every key segment at most
// kAttnLongLen long, or fp32 head_dim 8 / 16 / 32 / 64.
hipError_t launch_cross_attention(const nt_layout& Lq, const nt_layout& Lkv, int H, int D, const void* q,
                                  int64_t ld_q, const void* k, const void* v, int64_t ld_kv, float scale, void* o,
                                  int64_t ld_o, nt_dtype dtype, hipStream_t s);

// Workspace bytes of a triangle call: the re-tiled a and b for packed
// operands, 0 for pair-tiled ones.
size_t triangle_workspace_bytes(const nt_layout& L, int C, nt_tri_operands operands, nt_dtype dtype);
// Pair-tiled operands (plane variant matching the direction) are contracted
// directly; packed ones are first re-tiled into the workspace.
hipError_t launch_triangle(const nt_layout& L, int direction, int C, const void* a, const void* b,
                           int64_t ld_ab, nt_tri_operands operands, void* z, int64_t ld_z, nt_dtype dtype,
                           void* workspace, hipStream_t s);
// Gated operands: packed (a, b: [sum N^2, 2C] rows of [projection | gate
// logits], row stride ld_ab, gated while re-tiled into the workspace) or
// already-gated pair-tiled planes; t = triangle(a, b), overwritten.
hipError_t launch_triangle_gated(const nt_layout& L, int direction, int C, const void* a, const void* b,
                                 int64_t ld_ab, nt_tri_operands operands, void* t, int64_t ld_t, nt_dtype dtype,
                                 void* workspace, hipStream_t s);
// Backward of the triangle update on packed operands: da, db (row stride
// ld_dab; either may be NULL) accumulate the gradients; the workspace is
// triangle_workspace_bytes(L, C, NT_TRI_PACKED, dtype).
hipError_t launch_triangle_backward(const nt_layout& L, int direction, int C, const void* a, const void* b,
                                    int64_t ld_ab, const void* dt, int64_t ld_dt, void* da, void* db,
                                    int64_t ld_dab, nt_dtype dtype, void* workspace, hipStream_t s);

// Host-side planner (pure C++; no HIP calls).  Fills every host array of the
// layout from the lengths, or returns an error status.
// cols non-NULL: rectangular pairs N_i x M_i (M_i = cols[i]).
nt_status plan_layout(const int32_t* lengths, int32_t batch, nt_layout* L, const int32_t* cols = nullptr);

}  // namespace nt
