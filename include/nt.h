/*
 * nt.h -- C ABI of the packed multi-ragged pair-state library for MI355X
 * (gfx950).
 *
 * The library computes on packed values plus tensor-backed partitions, the
 * representation of "DanLing NestedTensor: Composable Multi-Ragged Tensors for
 * Deep Learning" (Sec. 3.1): a batch of B individually dense elements is
 * stored as one value buffer whose leading axis concatenates every sample's
 * ragged prefix, with sample offsets o (o_0 = 0, o_{i+1} - o_i = p_i,
 * o_B = T; Appendix A) held on the host and mirrored on the device.
 *
 * Packed layouts used by the calls below (all row-major, elements not bytes):
 *   singles      [sum_i N_i, C]        row eta_i + a         (eta = cu_seqlens)
 *   square pairs [sum_i N_i^2, C]      row o_i + a N_i + b   (Eq. coordinate)
 *   pair-tiled channel-major operands of the triangle update: channel c of
 *                sample i is an N_i x N_i plane (row r, column k) stored from
 *                c*ld + P_i, cut into 16 x 32 tiles (row tiles outer, tile
 *                (r/16, k/32) at ((r/16) nkt_i + k/32) * 512 with
 *                nkt_i = ceil(N_i/32)), element (r,k) inside its tile at
 *                ((k%32)/8 * 16 + r%16) * 8 + k%8 -- the lane order of a
 *                matrix-core fragment, so a wave reads 1 KB contiguously.
 *                A plane spans n16_i n32_i elements (N_i rounded up to 16 and
 *                to 32) and P_i = sum_{j<i} n16_j n32_j; entries outside the
 *                N_i x N_i matrix are padding and never read as data.  Plain
 *                variant: cell (i,a,b) is element (r,k) = (a,b); transposed
 *                variant: (r,k) = (b,a)
 *   pair bias    [sum_i N_i^2, H] with a row stride (cell-major, heads
 *                last), or any other (cell stride, head stride) pair, e.g.
 *                head-major [H][ld] = (1, ld)
 * Row strides ("ld_*") are in elements and let callers address column slices
 * of a wider buffer (e.g. u and v inside one [sum N, 2C] projection).
 *
 * Ownership: every value buffer is a device pointer owned by the caller; op
 * calls never allocate, free or retain memory.  An nt_layout and its device
 * mirrors are owned by the library from nt_from_* until nt_layout_destroy;
 * the caller must not destroy a layout while work that uses it is queued.
 * Workspaces: an op that needs scratch device memory (a bias image, packed
 * operands re-tiled, normalised rows, weights in consumption order) takes it
 * as a caller-provided (workspace, workspace_bytes) pair whose minimum size
 * the matching *_workspace query returns; 0 means the call needs none.  A
 * call that needs a workspace and is given none, or too little, returns
 * NT_ERR_INVALID_ARG without enqueuing anything.  The workspace is scratch for
 * the duration of the call's device work: calls that share one must be
 * stream-ordered.
 *
 * Streams: every op enqueues asynchronously on the caller's HIP stream
 * (NULL = the default stream) and returns without synchronising.  Only
 * nt_from_* copies host->device (stream-ordered) and nt_layout_destroy frees.
 *
 * Errors: every call returns an nt_status; nothing aborts or throws across the
 * ABI.  All argument checks run on the host before any launch; on an error no
 * work is enqueued and nt_last_error() (thread-local, valid until the next
 * call on the same thread) describes it.  Device pointers must be 16-byte
 * aligned and row strides multiples of 8 elements (bf16) or 4 (f32) unless a
 * call says otherwise.
 */
#ifndef NT_H
#define NT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nt_layout nt_layout;          /* opaque, library-owned */

typedef enum {
  NT_OK = 0,
  NT_ERR_INVALID_ARG = -1,     /* null pointer, bad size, misalignment, bad enum */
  NT_ERR_LAYOUT_MISMATCH = -2, /* operands with different logical partitions   */
  NT_ERR_OVERFLOW = -3,        /* a packed extent does not fit int32            */
  NT_ERR_UNSUPPORTED = -4,     /* valid request outside the implemented shapes  */
  NT_ERR_HIP = -5,             /* HIP runtime or launch failure                 */
  NT_ERR_OOM = -6              /* device allocation of layout mirrors failed    */
} nt_status;

typedef enum { NT_F32 = 0, NT_BF16 = 1 } nt_dtype;

typedef enum {
  NT_EPI_NONE = 0,             /* y = LN(x) W^T + b                                  */
  NT_EPI_RESIDUAL = 1,         /* y = residual + LN(x) W^T + b                       */
  NT_EPI_SWIGLU_RESIDUAL = 2,  /* y = residual + (silu(g) * u) W2^T + b2,
                                  [g|u] = LN(x) W^T + b (W stacks W_gate; W_up)       */
  NT_EPI_GELU = 3,             /* y = gelu(LN(x) W^T + b), exact erf form            */
  NT_EPI_GATED_RESIDUAL = 4,   /* y = residual + sigmoid(gate) * (LN(x) W^T + b): the
                                  output gate of the AlphaFold 3 triangle update
                                  cited in Sec. 4.3 (gate: [R, N] logits)             */
  NT_EPI_SIGMOID_GLU = 5       /* gated operands of that update: W has 2N rows in
                                  blocks of 2G (G = hidden), [projection; gate];
                                  y[:, G q + c] = sigmoid(p[:, 2G q + G + c]) *
                                  p[:, 2G q + c] with p = LN(x) W^T + b            */
} nt_epilogue;

typedef enum {
  NT_LEVEL_SINGLES = 0,        /* complete reduction within each sample's rows      */
  NT_LEVEL_PAIRS = 1,          /* over the second pair axis (pair columns b)        */
  NT_LEVEL_PAIRS_FIRST = 2     /* over the first pair axis (pair rows a)            */
} nt_level;

/* Operand layout of the triangle update (nt_triangle_mul). */
typedef enum {
  NT_TRI_PACKED = 0,           /* a, b: packed pair tensors [sum N^2, C], row stride ld_ab */
  NT_TRI_PAIR_TILED = 1,       /* a, b: pair-tiled channel-major planes, channel stride ld_ab */
  NT_TRI_PAIR_TILED_T = 2      /* the transposed pair-tiled variant                        */
} nt_tri_operands;

/* Layout of the columns that nt_layernorm_linear routes to y_tail. */
typedef enum {
  NT_TAIL_CHANNEL_MAJOR = 0,   /* column j of row r at j*ld_tail + r               */
  NT_TAIL_PAIR_TILED = 1,      /* pair-tiled channel-major (needs a pair layout)   */
  NT_TAIL_PAIR_TILED_T = 2     /* transposed pair-tiled channel-major              */
} nt_tail_layout;

enum { NT_LAYOUT_HOST_ONLY = 1u };           /* nt_from_*: no device mirrors */

/* Host arrays a layout exposes through nt_layout_host_array(). */
typedef enum {
  NT_ARR_LENGTHS = 0,          /* N_i, [B]                                      */
  NT_ARR_CU_SEQLENS = 1,       /* single offsets eta, [B+1]                     */
  NT_ARR_CU_PAIRS = 2,         /* square-pair offsets o, [B+1]                  */
  NT_ARR_ROW_SPLITS2 = 3,      /* level-2 pair row splits, [1 + sum N_i]        */
  NT_ARR_ROW_SAMPLE = 4,       /* sample id of every single row, [sum N_i]      */
  NT_ARR_ATTN_WORK = 5,        /* pair-row work map (sample, row) pairs, XCD-ordered */
  NT_ARR_TRI_WORK = 6,         /* triangle tile map (sample, x-tile, y-tile, first tile of the sample) quads */
  NT_ARR_SEQ_WORK = 7,         /* 1-D attention map (sample, query block) pairs */
  NT_ARR_CU_PAD = 8,           /* P_i offsets of pair-tiled operands, [B+1]     */
  NT_ARR_COLS = 9,             /* M_i, [B] (= N_i for square pairs)             */
  NT_ARR_CU_COLS = 10,         /* column offsets kappa, [B+1]                   */
  NT_ARR_TRI_SPLIT = 11        /* triangle tile map cut into 8 XCD ranges, [9]  */
} nt_array;

typedef struct {
  int32_t batch;               /* B                                             */
  int32_t max_len;             /* max_i N_i                                     */
  int64_t sum_n;               /* sum_i N_i    (rows of a single tensor)         */
  int64_t sum_n2;              /* sum_i N_i^2  (rows of a square pair tensor)    */
  int64_t sum_n3;              /* sum_i N_i^3  (work of the pair contractions)   */
  int64_t sum_pad;             /* sum_i n16_i n32_i (channel extent of pair-tiled operands) */
  const int32_t* d_cu_seqlens; /* device mirrors (NULL for host-only layouts)   */
  const int32_t* d_cu_pairs;
  const int32_t* d_row_splits2;
  int64_t sum_m;               /* sum_i M_i (columns; = sum_n for square pairs)  */
  int32_t rect;                /* 1 for rectangular pairs N_i x M_i             */
  const int32_t* d_cu_cols;    /* column offsets kappa (device)                 */
} nt_layout_info_t;

/* ---------------------------------------------------------------- layouts
 * Partitions of a batch of square pair states, built from the per-sample
 * lengths N_i (Sec. 3.1 "Structural metadata"; Fig. "representation"):
 * single offsets eta (cu_seqlens), pair offsets o with p_i = N_i^2, the
 * level-2 row splits o_i + a N_i (1 + sum N_i entries), and the tile-to-sample
 * work maps the kernels launch from, so that no wavefront crosses a sample
 * boundary.  Zero-length samples are allowed (Appendix A: zero-volume
 * elements have coincident offsets).
 *   lengths   host, [batch], each >= 0.            batch >= 1.
 *   flags     0, or NT_LAYOUT_HOST_ONLY to build host arrays only (no device
 *             memory is touched; op calls then reject the layout).
 *   stream    HIP stream for the host->device copies of the mirrors.
 *   out       receives the new layout.
 * Errors: NT_ERR_INVALID_ARG (null, batch < 1, negative length),
 *         NT_ERR_OVERFLOW (sum N_i^2 or sum N_i does not fit int32),
 *         NT_ERR_OOM / NT_ERR_HIP (device mirrors).                          */
nt_status nt_from_lengths(const int32_t* lengths, int32_t batch, uint32_t flags,
                          void* stream, nt_layout** out);

/* Rectangular pairs (Eq. packing with p_i = N_i M_i; Eq. pair-reduction):
 * element i is an N_i x M_i pair state from a row track of N_i singles
 * (offsets eta) and a column track of M_i singles (offsets kappa); cell
 * (i, a, b) is packed row o_i + a M_i + b.  rows = N_i, cols = M_i (host,
 * [batch], each >= 0).  The sum_n2 field of nt_layout_info counts the cells
 * (sum_i N_i M_i).  Broadcast, segment reductions, their backward, and the
 * row-wise ops accept rectangular layouts; attention over pair axes and the
 * triangle update need square pairs (NT_ERR_UNSUPPORTED).
 * Errors: as nt_from_lengths.                                                */
nt_status nt_from_rect_lengths(const int32_t* rows, const int32_t* cols, int32_t batch, uint32_t flags,
                               void* stream, nt_layout** out);

/* Same from single offsets (cu_seqlens, host, [batch+1]); they must satisfy
 * o_0 = 0 and be non-decreasing (Appendix A, "Structural invariants"),
 * otherwise NT_ERR_INVALID_ARG.                                              */
nt_status nt_from_offsets(const int32_t* cu_seqlens, int32_t batch, uint32_t flags,
                          void* stream, nt_layout** out);

/* Frees the layout and its device mirrors (NULL is accepted).  Waits for the
 * device to finish using the mirrors (hipFree semantics).                    */
nt_status nt_layout_destroy(nt_layout* layout);

nt_status nt_layout_info(const nt_layout* layout, nt_layout_info_t* info);

/* Host copy of one metadata array (pointer valid for the layout's lifetime);
 * *count receives the number of int32 entries.                              */
nt_status nt_layout_host_array(const nt_layout* layout, nt_array which,
                               const int32_t** data, int64_t* count);

/* 1 if the two layouts describe the same logical partition (equal length
 * vectors), else 0.  Equal packed totals are not enough: (2,6) and (3,4)
 * pairs both hold twelve rows but are incompatible (Sec. 3.2).              */
int32_t nt_layouts_compatible(const nt_layout* a, const nt_layout* b);

/* ---------------------------------------------------------------- broadcast
 * Pair construction by broadcasting (Eq. running-block, first line; Sec. 3.2
 * "Creating axes through broadcasting"): for every sample i, a < N_i, b < M_i
 *     z[o_i + a M_i + b, c] (+)= u[eta_i + a, c] + v[kappa_i + b, c]
 * (square pairs: M_i = N_i, kappa = eta) computed in fp32 and rounded once to
 * the storage dtype.
 *   C          channels (> 0).
 *   u, v       row singles [sum N, C] and column singles [sum M, C] with row
 *              strides ld_u, ld_v (may alias for square pairs).
 *   z          pairs [sum N^2, C] with row stride ld_z (must not alias u/v).
 *   accumulate 0: z is overwritten; 1: z is read and the sum added to it.
 *   dtype      NT_F32 or NT_BF16 for u, v and z.
 * Errors: NT_ERR_INVALID_ARG.                                                */
nt_status nt_pair_broadcast(const nt_layout* layout, int32_t C,
                            const void* u, int64_t ld_u, const void* v, int64_t ld_v,
                            void* z, int64_t ld_z, int32_t accumulate,
                            nt_dtype dtype, void* stream);

/* ---------------------------------------------------------------- LN + Linear
 * Feature transform on packed rows (Sec. 3.3: V' = V W^T + b, normalisation on
 * each row's feature tail; rows are independent, so one launch covers every
 * sample):  y = epilogue(LN(x; gamma, beta, eps) W^T + b).
 * LayerNorm uses the biased variance with statistics in fp32.  bf16 runs on
 * matrix cores (bf16 operands, fp32 accumulation); f32 runs in fp32 FMA.      */
typedef struct {
  int64_t rows;                /* R >= 0                                         */
  int32_t c_in;                /* K (multiple of 8)                               */
  int32_t c_out;               /* N: output width (for SwiGLU: the residual width) */
  nt_dtype dtype;              /* dtype of W, W2, residual and y                  */
  const void* x;               /* [R, K] row stride ldx                           */
  int64_t ldx;
  nt_dtype x_dtype;            /* x may be f32 when dtype is bf16 (e.g. a reduce output) */
  const float* ln_gamma;       /* [K] or NULL (no LayerNorm); ln_beta NULL = 0    */
  const float* ln_beta;
  float ln_eps;
  const void* w;               /* [N_w, K] row-major; N_w = N, or 2F for SwiGLU    */
  const float* bias;           /* [N_w] or NULL                                   */
  nt_epilogue epilogue;
  int32_t hidden;              /* F for SwiGLU (multiple of 32), else 0           */
  const void* w2;              /* SwiGLU down projection [N, F], else NULL        */
  const float* bias2;          /* [N] or NULL                                     */
  const void* residual;        /* [R, N - n_tail] row stride ld_residual (added to the
                                  main columns only); NULL = x for SwiGLU          */
  int64_t ld_residual;
  void* y;                     /* [R, N - n_tail] row stride ldy (may alias residual) */
  int64_t ldy;
  int32_t n_tail;              /* last n_tail output columns go to y_tail instead */
  void* y_tail;                /* [n_tail][ld_tail], arranged as tail_layout says  */
  int64_t ld_tail;
  nt_tail_layout tail_layout;
  const nt_layout* layout;     /* optional: rows must equal the layout's row count */
  nt_level level;              /*   at this level                               */
  const nt_layout* residual_layout;  /* optional: must be compatible with layout */
  /* Broadcast rows (x NULL, bcast_u and bcast_v set): the rows are the pair
   * broadcast of u and v over `layout` (level NT_LEVEL_PAIRS):
   *     x[o_i + a N_i + b] = u[eta_i + a] + v[eta_i + b]
   * summed in fp32 and rounded to bf16 -- exactly what nt_pair_broadcast
   * stores -- so LN(broadcast) W^T + b is computed without writing or reading
   * the broadcast pair tensor (Eq. running-block, first two lines, fused).
   * bf16 only, c_in in {64, 128}, c_out <= 512 (multiple of 8), epilogue
   * NONE or GELU, no tail, no residual; u, v: [sum N, c_in] with row strides
   * ld_bcast_u, ld_bcast_v (multiples of 8; may alias).                    */
  const void* bcast_u;
  int64_t ld_bcast_u;
  const void* bcast_v;
  int64_t ld_bcast_v;
  /* Caller-provided scratch (see nt_layernorm_linear_workspace); NULL / 0
   * when the call needs none.                                              */
  void* workspace;
  uint64_t workspace_bytes;
  /* NT_EPI_GATED_RESIDUAL: gate logits [R, N] in dtype, row stride ld_gate
   * (>= N, a multiple of 8 for bf16 / 4 for f32, 16-byte aligned); NULL for
   * every other epilogue.  No tail with this epilogue.                     */
  const void* gate;
  int64_t ld_gate;
} nt_linear_args;

/* Workspace (args->workspace, args->workspace_bytes): two kinds of bf16 call
 * need one.  A call with a LayerNorm, bf16 x, K >= 384 (K % 32 == 0,
 * K <= 4096), N % 8 == 0 and no tail first writes LN(x) there (rounded to
 * bf16, as the product consumes it): R * K * 2 bytes.  A SwiGLU transition
 * with K in {64, 128} and F <= 768 first copies its weights there in the
 * order its kernel consumes them: 3 * F * K * 2 bytes.  Every other call needs
 * none.  nt_layernorm_linear_workspace returns the size for a given argument
 * set (it reads only sizes, dtypes and flags, never the pointers).
 * Errors: NT_ERR_INVALID_ARG (also a missing or too small workspace),
 * NT_ERR_LAYOUT_MISMATCH (residual_layout differs
 * from layout, or rows differ from the layout's count), NT_ERR_UNSUPPORTED
 * (NT_EPI_SIGMOID_GLU unless bf16, K == 128, hidden == 128, N == 256 and
 * every output column in a pair-tiled tail (n_tail == N);
 * bf16 SwiGLU unless x is bf16, K == N in {64, 128, 256} and F % 32 == 0;
 * f32 SwiGLU with K > 1024 or F > 4096; n_tail with SwiGLU; a pair-tiled
 * tail without a pair layout), NT_ERR_HIP (also when the workspace cannot be
 * allocated).  ln_gamma/ln_beta must be 16-byte aligned.                     */
nt_status nt_layernorm_linear(const nt_linear_args* args, void* stream);

/* Minimum workspace of nt_layernorm_linear(args) in bytes (0: none).
 * Errors: NT_ERR_INVALID_ARG (NULL).                                        */
nt_status nt_layernorm_linear_workspace(const nt_linear_args* args, uint64_t* bytes);

/* ---------------------------------------------------------------- attention
 * Segmented softmax attention, one launch over the whole batch.
 *   axis 0  row attention with pair bias around the starting node: for sample
 *           i, pair row r, query j, head h
 *             o[cell(r,j),h] = sum_k softmax_k(scale q[cell(r,j),h].k[cell(r,k),h]
 *                                              + bias[h][cell(j,k)]) v[cell(r,k),h]
 *   axis 1  the same around the ending node: axis 0 applied to each sample's
 *           transpose (q, k, v and the bias read at cell(b,a) for (a,b)).
 *   axis 2  1-D variable-length self-attention over the tokens of each sample
 *           (Sec. 3.3 "Attention through packed blocks"); bias must be NULL.
 *   axis 3  single attention with pair bias (the Pairformer's, cited in
 *           Sec. 4.3): over the tokens of each sample, query t, key k,
 *             o[t,h] = sum_k softmax_k(scale q[t,h].k[k,h] + bias[h][cell(t,k)]) v[k,h]
 *           with q, k, v, o token-major (rows = sum N) and the bias read from
 *           the pair state; bf16, d = 32, N_i <= 512 (else NT_ERR_UNSUPPORTED).
 * cell(a,b) = o_i + a N_i + b.  Pair attention follows the Pairformer's
 * triangle attention cited in Sec. 4.3 (reading: no gating, no mask).
 *   heads, head_dim  H and d; d in {8, 16 (f32 only), 32, 64}; H*d <= ld_qkv.
 *   q, k, v  [rows, H*d] with common row stride ld_qkv (may be slices of one
 *            buffer); rows = sum N^2 (axes 0/1) or sum N (axes 2/3).
 *   bias     NULL (axes 0/1/3), or the pair bias: head h of cell c at
 *            bias[c * ld_bias + h * ld_bias_head], i.e. [sum N^2, H] with row
 *            stride ld_bias (>= H) and ld_bias_head = 1; the head-major form
 *            [H][ld] is ld_bias = 1, ld_bias_head = ld (>= sum N^2).  Strides
 *            are positive and in elements.
 *   scale    softmax scale (e.g. 1/sqrt(d)).
 *   o        [rows, H*d] row stride ld_o.
 * Workspace: with a bias, bf16, d = 32 and every N_i <= 512 the call first
 * writes bias/scale (rounded to bf16) in the per-lane order of the attention
 * kernel into the workspace: H * T * 512 bytes with
 * T = sum_i ceil(N_i/16) * ceil(N_i/64) * 4 (nt_pair_row_attention_workspace).
 * Errors: NT_ERR_INVALID_ARG (also a missing or too small workspace),
 * NT_ERR_UNSUPPORTED (d, or N_i beyond the on-chip limit: 1024 for d=32,
 * 512 for d=64), NT_ERR_HIP.                                                 */
nt_status nt_pair_row_attention(const nt_layout* layout, int32_t axis,
                                int32_t heads, int32_t head_dim,
                                const void* q, const void* k, const void* v, int64_t ld_qkv,
                                const void* bias, int64_t ld_bias, int64_t ld_bias_head, float scale,
                                void* o, int64_t ld_o, nt_dtype dtype,
                                void* workspace, uint64_t workspace_bytes, void* stream);

/* Gated pair attention (the AlphaFold 3 form of the triangle attention that
 * Sec. 4.3 cites): nt_pair_row_attention on axis 0 or 1, with the output
 * multiplied by the sigmoid of per-cell, per-channel gate logits:
 *   o[cell, c] = sigmoid(gate[cell, c]) * attention[cell, c],  c < H*d
 * gate: [sum N^2, >= H*d] in dtype, row stride ld_gate (a multiple of 8 for
 * bf16 / 4 for f32, 16-byte aligned); it may be a column slice of the
 * projection that produced q, k and v.  Other arguments, workspace and
 * errors as nt_pair_row_attention (also NT_ERR_INVALID_ARG for axes 2 and 3
 * or a NULL gate).                                                         */
nt_status nt_pair_row_attention_gated(const nt_layout* layout, int32_t axis, int32_t heads, int32_t head_dim,
                                      const void* q, const void* k, const void* v, int64_t ld_qkv,
                                      const void* gate, int64_t ld_gate,
                                      const void* bias, int64_t ld_bias, int64_t ld_bias_head, float scale,
                                      void* o, int64_t ld_o, nt_dtype dtype,
                                      void* workspace, uint64_t workspace_bytes, void* stream);

/* Cross-attention over singles with different query and key lengths (Sec.
 * 3.3 "Attention through packed blocks": the output takes the query
 * structure, so queries and keys may be ragged differently).  Sample i has
 * N_i queries (q_layout) and M_i keys and values (kv_layout); per head h
 *   o[eta_i + t, h] = sum_k softmax_k(scale q[eta_i + t, h].k[kappa_i + k, h]) v[kappa_i + k, h]
 * with eta the query offsets and kappa the key offsets.  A query whose sample
 * has no keys (M_i = 0) gets the empty sum, 0.  Self-attention is
 * nt_pair_row_attention with axis 2 (the same operation with kv = q layout).
 *   q_layout, kv_layout  single-level layouts of one batch (equal batch size,
 *            else NT_ERR_LAYOUT_MISMATCH); only their lengths are used.
 *   q, o     [sum N, H*d], row strides ld_q, ld_o.
 *   k, v     [sum M, H*d], common row stride ld_kv (may be NULL when sum M = 0).
 *   dtype    bf16 (matrix cores, fp32 softmax; head_dim 32 or 64, M_i <= 512)
 *            or f32 (exact two-pass softmax; head_dim 8, 16, 32, 64; M_i <= 4096).
 * No workspace.  Errors: NT_ERR_INVALID_ARG, NT_ERR_LAYOUT_MISMATCH,
 * NT_ERR_UNSUPPORTED (head_dim or key length beyond the limits), NT_ERR_HIP. */
nt_status nt_cross_attention(const nt_layout* q_layout, const nt_layout* kv_layout, int32_t heads, int32_t head_dim,
                             const void* q, int64_t ld_q, const void* k, const void* v, int64_t ld_kv,
                             float scale, void* o, int64_t ld_o, nt_dtype dtype, void* stream);

/* For callers that cannot allocate device memory (code under graph capture,
 * tight serving loops, harnesses that forbid allocation): the same operation
 * and arguments as nt_pair_row_attention without a workspace.  The bias image
 * goes into a scratch array of 16 MiB that the library holds on each device
 * it runs on until the process ends (resolved once per device on the first
 * call there); no call allocates or frees.  A call whose bias image would
 * exceed 16 MiB (H * T * 512 bytes, see above) returns NT_ERR_UNSUPPORTED
 * before any work.  Every call on one device shares that device's array, so
 * calls that overlap in time on one device (different streams, or threads
 * without ordering) race; calls ordered on one stream are safe.
 * Errors: as nt_pair_row_attention, plus NT_ERR_UNSUPPORTED (scratch too
 * small) and NT_ERR_HIP (the array's address cannot be resolved).           */
nt_status nt_pair_row_attention_noalloc(const nt_layout* layout, int32_t axis,
                                        int32_t heads, int32_t head_dim,
                                        const void* q, const void* k, const void* v, int64_t ld_qkv,
                                        const void* bias, int64_t ld_bias, int64_t ld_bias_head, float scale,
                                        void* o, int64_t ld_o, nt_dtype dtype, void* stream);

/* Minimum workspace of nt_pair_row_attention for these arguments, in bytes
 * (0: none); has_bias is 0 or 1.
 * Errors: NT_ERR_INVALID_ARG.                                               */
nt_status nt_pair_row_attention_workspace(const nt_layout* layout, int32_t axis, int32_t heads,
                                          int32_t head_dim, nt_dtype dtype, int32_t has_bias,
                                          uint64_t* bytes);

/* ---------------------------------------------------------------- triangle
 * Triangle multiplicative update, channelwise (Sec. 4.3, after the AlphaFold 3
 * Pairformer; reading: no gates, no output projection), accumulated into z:
 *   direction 0 (outgoing)  z[cell(x,y),c] += sum_k a[cell(x,k),c] b[cell(y,k),c]
 *   direction 1 (incoming)  z[cell(x,y),c] += sum_k a[cell(k,x),c] b[cell(k,y),c]
 * One ragged grouped GEMM over all samples and channels (per sample and
 * channel an N_i x N_i x N_i product); fp32 accumulation, z rounded once.
 *   operands  NT_TRI_PACKED: a, b are packed pair tensors [sum N^2, C] (the
 *             paper's layout, Eq. packing) with row stride ld_ab (>= C); the
 *             call re-tiles them into the workspace, 2 * C * round_up(sum_pad,
 *             8) elements (nt_triangle_mul_workspace), in the variant the
 *             direction needs.
 *             NT_TRI_PAIR_TILED / NT_TRI_PAIR_TILED_T: a, b are already
 *             pair-tiled channel-major planes with channel stride ld_ab
 *             (>= sum_pad, multiple of 8), as nt_layernorm_linear writes them
 *             with NT_TAIL_PAIR_TILED(_T); the plain variant serves direction
 *             0 and the transposed one direction 1 (the incoming update is the
 *             outgoing contraction of the transposes); a variant that does
 *             not match the direction is rejected.  No workspace.
 *   z         channel-last pair state [sum N^2, C] with row stride ld_z.
 * Errors: NT_ERR_INVALID_ARG (C not a multiple of 32 for bf16 or of 4 for f32,
 * operand variant and direction disagree, missing or too small workspace).   */
nt_status nt_triangle_mul(const nt_layout* layout, int32_t direction, int32_t C,
                          const void* a, const void* b, int64_t ld_ab, nt_tri_operands operands,
                          void* z, int64_t ld_z, nt_dtype dtype,
                          void* workspace, uint64_t workspace_bytes, void* stream);

/* Contraction of the gated triangle update (the AlphaFold 3 form of the
 * update that Sec. 4.3 cites): the operands are gated projections,
 *   a = sigmoid(a_g) * a_p,  b = sigmoid(b_g) * b_p   (elementwise, fp32, rounded once)
 * and the contraction t (outgoing / incoming as nt_triangle_mul) is written
 * to t, not added (the gated update normalises t before its own gated
 * residual: nt_layernorm_linear with NT_EPI_GATED_RESIDUAL).
 *   operands  NT_TRI_PACKED: a, b are packed pair rows [sum N^2, >= 2C] with
 *             row stride ld_ab, channels [0, C) the projection and [C, 2C)
 *             the gate logits (a and b may be column slices of one
 *             projection output); they are gated while re-tiled into the
 *             workspace (as nt_triangle_mul with NT_TRI_PACKED).
 *             NT_TRI_PAIR_TILED / NT_TRI_PAIR_TILED_T: a, b are gated
 *             operands already in pair-tiled planes (channel stride ld_ab),
 *             as nt_layernorm_linear with NT_EPI_SIGMOID_GLU writes them; the
 *             variant must match the direction, as for nt_triangle_mul.  No
 *             workspace.
 *   t         [sum N^2, C], row stride ld_t, overwritten.
 * Errors: as nt_triangle_mul.                                               */
nt_status nt_triangle_mul_gated(const nt_layout* layout, int32_t direction, int32_t C,
                                const void* a, const void* b, int64_t ld_ab, nt_tri_operands operands,
                                void* t, int64_t ld_t, nt_dtype dtype,
                                void* workspace, uint64_t workspace_bytes, void* stream);

/* Minimum workspace of nt_triangle_mul in bytes (0: none).
 * Errors: NT_ERR_INVALID_ARG.                                               */
nt_status nt_triangle_mul_workspace(const nt_layout* layout, int32_t C, nt_tri_operands operands,
                                    nt_dtype dtype, uint64_t* bytes);

/* ---------------------------------------------------------------- reduce
 * Reductions that consume a ragged axis, with fp32 accumulation and fp32
 * output, one launch, no atomics (rectangular pairs: cell (a, b) at
 * o_i + a M_i + b, square: M_i = N_i, kappa = eta):
 *   level NT_LEVEL_PAIRS   (pair columns, Eq. pair-reduction)
 *       y[eta_i + a, c] = sum_b x[o_i + a M_i + b, c]     (op 1: / M_i)
 *   level NT_LEVEL_PAIRS_FIRST (the other pair axis; the broadcast's
 *       gradient with respect to its column operand)
 *       y[kappa_i + b, c] = sum_a x[o_i + a M_i + b, c]   (op 1: / N_i)
 *   level NT_LEVEL_SINGLES (complete reduction within each element, Appendix A)
 *       y[i, c] = sum_t x[eta_i + t, c]                    (op 1: / N_i;
 *       an empty sample gives 0 for the sum and NaN for the mean)
 *   op       0 sum, 1 mean.
 *   x        [rows, C] row stride ld_x, dtype x_dtype.   y: fp32, row stride ld_y.
 * Errors: NT_ERR_INVALID_ARG.                                                */
nt_status nt_segment_reduce(const nt_layout* layout, nt_level level, int32_t op, int32_t C,
                            const void* x, int64_t ld_x, nt_dtype x_dtype,
                            float* y, int64_t ld_y, void* stream);

/* ---------------------------------------------------------------- backward
 * Gradients of the calls above for a training step (forward, loss and
 * backward through the packed representation, Sec. 3.4 "Gradients across
 * representations"): every gradient has the packed layout of its value.    */

/* Backward of nt_pair_broadcast (z = u_a + v_b):
 *   du[eta_i + a, c]   (+)= sum_b dz[o_i + a M_i + b, c]
 *   dv[kappa_i + b, c] (+)= sum_a dz[o_i + a M_i + b, c]
 * dz [cells, C] (dtype, row stride ld_dz); du [sum N, C] and dv [sum M, C] in
 * out_dtype (fp32, or bf16 rounded once from the fp32 sums) with row strides
 * ld_du, ld_dv; accumulate 0 overwrites, 1 adds.  Either of du, dv may be
 * NULL (not computed).  fp32 accumulation, no atomics.
 * Errors: NT_ERR_INVALID_ARG.                                                */
nt_status nt_pair_broadcast_backward(const nt_layout* layout, int32_t C, const void* dz, int64_t ld_dz,
                                     nt_dtype dtype, void* du, int64_t ld_du, void* dv, int64_t ld_dv,
                                     nt_dtype out_dtype, int32_t accumulate, void* stream);

/* Sample-weighted squared norm and its gradient, the diagnostic loss of the
 * measured single-pair-single program (App. A, Eq. joint-diagnostic-loss):
 *   loss[i] = scale * weights[i] * sum over sample i's rows r, channels c of x[r, c]^2
 *   dx[r, c] = 2 * scale * weights[i] * x[r, c]          (dx NULL: not written)
 * level NT_LEVEL_SINGLES: rows eta_i .. eta_{i+1}; NT_LEVEL_PAIRS: the pair
 * cells o_i .. o_{i+1}.  weights, loss: device fp32 [B]; x in dtype, dx in
 * dx_dtype.  The per-sample sums are fp32 partials reduced in a fixed order.
 * Workspace: nt_weighted_square_loss_workspace (B * 256 bytes).
 * Errors: NT_ERR_INVALID_ARG.                                                */
nt_status nt_weighted_square_loss(const nt_layout* layout, nt_level level, int32_t C, const void* x, int64_t ld_x,
                                  nt_dtype dtype, const float* weights, float scale, float* loss, void* dx,
                                  int64_t ld_dx, nt_dtype dx_dtype, void* workspace, uint64_t workspace_bytes,
                                  void* stream);
nt_status nt_weighted_square_loss_workspace(const nt_layout* layout, uint64_t* bytes);

/* Backward of nt_segment_reduce: every reduced position receives its group's
 * gradient dy (fp32, the reduce's output layout, row stride ld_dy), divided
 * by N_i for op 1 (mean):
 *   NT_LEVEL_PAIRS        dx[o_i + a M_i + b] (+)= dy[eta_i + a]   (/ M_i)
 *   NT_LEVEL_PAIRS_FIRST  dx[o_i + a M_i + b] (+)= dy[kappa_i + b] (/ N_i)
 *   NT_LEVEL_SINGLES      dx[eta_i + t]       (+)= dy[i]        (/ N_i)
 * dx in dtype with row stride ld_dx; accumulate 0 overwrites, 1 adds.
 * Errors: NT_ERR_INVALID_ARG.                                                */
nt_status nt_segment_reduce_backward(const nt_layout* layout, nt_level level, int32_t op, int32_t C,
                                     const float* dy, int64_t ld_dy, void* dx, int64_t ld_dx, nt_dtype dtype,
                                     int32_t accumulate, void* stream);

/* Backward of nt_triangle_mul on packed operands (a, b: [sum N^2, C], row
 * stride ld_ab), for the cotangent dt of the update t (dt: [sum N^2, C], row
 * stride ld_dt), per sample and channel c:
 *   direction 0  t = a b^T:   da += dt b,     db += dt^T a
 *   direction 1  t = a^T b:   da += b dt^T,   db += a dt
 * (a, b, dt read as each sample's N_i x N_i channel planes).  da and db
 * (row stride ld_dab; either may be NULL) are accumulated in their dtype,
 * fp32 sums rounded once per call.  Workspace: the same as the forward on
 * packed operands (nt_triangle_mul_workspace with NT_TRI_PACKED).
 * Errors: as nt_triangle_mul.                                                */
nt_status nt_triangle_mul_backward(const nt_layout* layout, int32_t direction, int32_t C,
                                   const void* a, const void* b, int64_t ld_ab, const void* dt, int64_t ld_dt,
                                   void* da, void* db, int64_t ld_dab, nt_dtype dtype,
                                   void* workspace, uint64_t workspace_bytes, void* stream);

/* Backward of nt_pair_row_attention on axes 0 and 1 (bf16, head_dim 32,
 * N_i <= 512).  Inputs are the forward's q, k, v (row stride ld_qkv), its
 * bias (as in the forward, or NULL), the output's gradient dout (ld_dout)
 * and the softmax scale; the softmax is recomputed.  Per pair row r and head
 * h, with S = scale q k^T + bias and P = softmax_k(S):
 *   dS = P (dP - rowsum(P dP)), dP = dout v^T,  dq = scale dS k,  dk = scale dS^T q,
 *   dv = P^T dout,  dbias = sum over the pair rows r of dS
 * (axis 1 on each sample's transpose, the bias gradient transposed back).
 * dq, dk, dv: bf16 [sum N^2, H*d] with row stride ld_dqkv, overwritten;
 * dbias: fp32, head h of cell c at dbias[c * ld_dbias + h * ld_dbias_head],
 * overwritten (NULL: not computed).  fp32 arithmetic, no atomics.
 * Workspace: 8 * H * sum N^2 bytes (the softmax statistics of every query),
 * nt_pair_row_attention_backward_workspace.
 * Errors: NT_ERR_INVALID_ARG, NT_ERR_UNSUPPORTED (axis, dtype, head_dim,
 * N_i > 512).                                                                */
nt_status nt_pair_row_attention_backward(const nt_layout* layout, int32_t axis, int32_t heads, int32_t head_dim,
                                         const void* q, const void* k, const void* v, int64_t ld_qkv,
                                         const void* bias, int64_t ld_bias, int64_t ld_bias_head,
                                         const void* dout, int64_t ld_dout, float scale,
                                         void* dq, void* dk, void* dv, int64_t ld_dqkv,
                                         float* dbias, int64_t ld_dbias, int64_t ld_dbias_head,
                                         nt_dtype dtype, void* workspace, uint64_t workspace_bytes, void* stream);
nt_status nt_pair_row_attention_backward_workspace(const nt_layout* layout, int32_t axis, int32_t heads,
                                                   int32_t head_dim, nt_dtype dtype, uint64_t* bytes);

/* Backward of nt_layernorm_linear (rows of a packed tensor, any level):
 *   y = epilogue(LN(x) W^T + b)
 * Given dy = dL/dy it adds the gradients of the weights and writes dx:
 *   NONE / RESIDUAL   p = LN(x) W^T + b, dp = dy (the residual's gradient is
 *                     dy itself; the caller adds it where it belongs)
 *   GELU              dp = dy gelu'(p), p recomputed from x
 *   SWIGLU_RESIDUAL   [g|u] = LN(x) W^T + b recomputed, h = silu(g) u,
 *                     dW2 += dy^T h, db2 += sum dy, dh = dy W2,
 *                     dp = [dh u silu'(g) | dh silu(g)]; with residual_is_x
 *                     (the forward's residual was x) dx also receives dy
 *   dW += dp^T LN(x),  db += sum_rows dp,  d(LN x) = dp W, then through the
 *   LayerNorm: dx = rstd (g - mean(g) - xhat mean(g xhat)), g = d(LN x) gamma,
 *   dgamma += sum_rows d(LN x) xhat,  dbeta += sum_rows d(LN x).
 * bf16 weights and dy; products on matrix cores with fp32 accumulation; the
 * normalised rows and the recomputed hidden are rounded to bf16 as the
 * forward consumed them.  Weight gradients (dw, db, dgamma, dbeta, dw2, db2:
 * fp32, contiguous, NULL = not wanted) are accumulated (overwritten with
 * overwrite_weights); dx (x_dtype or fp32) is overwritten unless accumulate_dx.  Partial sums are reduced in a fixed
 * order: the result is deterministic.  Every pointer, the LayerNorm affine
 * and the bias included, must be 16-byte aligned.                            */
typedef struct {
  int64_t rows;                /* R                                              */
  int32_t c_in;                /* K (multiple of 8, <= 1024)                      */
  int32_t c_out;               /* N: width of y (SwiGLU: the residual width)      */
  const void* x;               /* forward input [R, K], row stride ldx            */
  int64_t ldx;
  nt_dtype x_dtype;            /* bf16 or fp32                                   */
  const float* ln_gamma;       /* [K] or NULL (no LayerNorm)                      */
  const float* ln_beta;        /* [K] or NULL                                    */
  float ln_eps;
  const void* w;               /* bf16 [N_w, K] contiguous, N_w = N or 2F          */
  const float* bias;           /* [N_w] or NULL (needed to recompute GELU / SwiGLU) */
  nt_epilogue epilogue;
  int32_t hidden;              /* F for SwiGLU                                   */
  const void* w2;              /* SwiGLU: bf16 [N, F] contiguous                  */
  int32_t residual_is_x;       /* SwiGLU: the residual was x                      */
  const void* dy;              /* bf16 [R, N], row stride ld_dy                   */
  int64_t ld_dy;
  void* dx;                    /* [R, K] in dx_dtype, row stride ld_dx, or NULL    */
  int64_t ld_dx;
  nt_dtype dx_dtype;
  int32_t accumulate_dx;
  int32_t overwrite_weights;   /* 1: dw .. db2 are overwritten instead of accumulated */
  float* dw;                   /* [N_w, K]  */
  float* db;                   /* [N_w]     */
  float* dgamma;               /* [K]       */
  float* dbeta;                /* [K]       */
  float* dw2;                  /* [N, F]    */
  float* db2;                  /* [N]       */
  void* workspace;             /* nt_layernorm_linear_backward_workspace bytes    */
  uint64_t workspace_bytes;
} nt_linear_bwd_args;

/* Errors: NT_ERR_INVALID_ARG (also a missing or too small workspace),
 * NT_ERR_UNSUPPORTED (fp32 weights, K > 1024, no LayerNorm with a bf16 dx
 * that accumulates), NT_ERR_HIP.                                             */
nt_status nt_layernorm_linear_backward(const nt_linear_bwd_args* args, void* stream);
nt_status nt_layernorm_linear_backward_workspace(const nt_linear_bwd_args* args, uint64_t* bytes);

/* Thread-local description of the last error on this thread. */
const char* nt_last_error(void);

/* Library version string. */
const char* nt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NT_H */
