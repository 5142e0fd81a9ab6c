// C ABI entry points (include/nt.h): argument validation on the host, layout
// lifetime, and dispatch to the kernel launchers.  No entry point throws or
// aborts; op calls neither allocate nor synchronise (scratch memory is the
// caller's workspace, sized by the *_workspace queries).
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "nt_internal.h"

namespace {

thread_local std::string g_last_error;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int vec_elems(nt_dtype t) { return t == NT_BF16 ? 8 : 4; }

bool valid_dtype(nt_dtype t) { return t == NT_F32 || t == NT_BF16; }

nt_status check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return NT_OK;
  return nt::fail(NT_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

nt_status need_device(const nt_layout* L) {
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (!L->has_device) return nt::fail(NT_ERR_INVALID_ARG, "layout was built host-only; it has no device mirrors");
  return NT_OK;
}

nt_status need_square(const nt_layout* L, const char* op) {
  if (L && L->rect) return nt::fail(NT_ERR_UNSUPPORTED, std::string(op) + " needs square pairs (N_i x N_i)");
  return NT_OK;
}

nt_status need_workspace(size_t need, const void* ws, uint64_t bytes, const char* query) {
  if (need == 0) return NT_OK;
  if (!ws || bytes < need)
    return nt::fail(NT_ERR_INVALID_ARG, "this call needs a workspace of " + std::to_string(need) + " bytes (" +
                                            query + "); given " + (ws ? std::to_string(bytes) : std::string("none")));
  if (!aligned16(ws)) return nt::fail(NT_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  return NT_OK;
}

bool same_partition(const nt_layout* a, const nt_layout* b) {
  return a == b || (a && b && a->lengths == b->lengths && a->cols == b->cols);
}

nt_status upload(nt_layout* L, hipStream_t s) {
  struct Part { const std::vector<int32_t>* v; const int32_t** dst; };
  Part parts[] = {
      {&L->lengths, &L->d_lengths},       {&L->cu_seqlens, &L->d_cu_seqlens},
      {&L->cu_pairs, &L->d_cu_pairs},     {&L->cu_pad, &L->d_cu_pad},
      {&L->row_splits2, &L->d_row_splits2}, {&L->row_sample, &L->d_row_sample},
      {&L->attn_work, &L->d_attn_work},   {&L->tri_work, &L->d_tri_work},
      {&L->seq_work, &L->d_seq_work},
      {&L->blk_prow, &L->d_blk_prow},
      {&L->pattn_work, &L->d_pattn_work}, {&L->bias_tiles, &L->d_bias_tiles},
      {&L->sattn_work, &L->d_sattn_work},
      {&L->bc_cu_tiles, &L->d_bc_cu_tiles},
      {&L->cu_qblk, &L->d_cu_qblk},       {&L->tri_split, &L->d_tri_split},
      {&L->cu_cols, &L->d_cu_cols},       {&L->col_sample, &L->d_col_sample},
  };
  size_t total = 0;
  for (auto& p : parts) total += (p.v->size() * sizeof(int32_t) + 255) / 256 * 256;
  std::vector<int32_t> staging(total / sizeof(int32_t), 0);
  if (hipGetDevice(&L->device) != hipSuccess) return nt::fail(NT_ERR_HIP, "hipGetDevice failed");
  hipError_t e = hipMalloc(&L->d_base, total);
  if (e != hipSuccess) {
    L->d_base = nullptr;
    return nt::fail(e == hipErrorOutOfMemory ? NT_ERR_OOM : NT_ERR_HIP,
                    std::string("hipMalloc of layout mirrors: ") + hipGetErrorString(e));
  }
  size_t off = 0;
  for (auto& p : parts) {
    std::memcpy(staging.data() + off / sizeof(int32_t), p.v->data(), p.v->size() * sizeof(int32_t));
    *p.dst = reinterpret_cast<const int32_t*>(static_cast<char*>(L->d_base) + off);
    off += (p.v->size() * sizeof(int32_t) + 255) / 256 * 256;
  }
  e = hipMemcpyAsync(L->d_base, staging.data(), total, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);   // staging is a local buffer
  if (e != hipSuccess) return check_hip(e, "copy of layout mirrors");
  L->has_device = true;
  return NT_OK;
}

nt_status build(const int32_t* lengths, int32_t batch, uint32_t flags, void* stream, nt_layout** out,
                const int32_t* cols = nullptr) {
  if (!out) return nt::fail(NT_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (flags & ~(uint32_t)NT_LAYOUT_HOST_ONLY) return nt::fail(NT_ERR_INVALID_ARG, "unknown flags");
  nt_layout* L = new (std::nothrow) nt_layout();
  if (!L) return nt::fail(NT_ERR_OOM, "host allocation failed");
  nt_status st = nt::plan_layout(lengths, batch, L, cols);
  if (st == NT_OK && !(flags & NT_LAYOUT_HOST_ONLY)) st = upload(L, static_cast<hipStream_t>(stream));
  if (st != NT_OK) {
    nt_layout_destroy(L);
    return st;
  }
  *out = L;
  return NT_OK;
}

}  // namespace

namespace nt {
nt_status fail(nt_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

}  // namespace nt

extern "C" {

const char* nt_last_error(void) { return g_last_error.c_str(); }

const char* nt_version(void) { return "nt-mi355x 0.1 (gfx950)"; }

nt_status nt_from_lengths(const int32_t* lengths, int32_t batch, uint32_t flags, void* stream,
                          nt_layout** out) {
  g_last_error.clear();
  return build(lengths, batch, flags, stream, out);
}

nt_status nt_from_rect_lengths(const int32_t* rows, const int32_t* cols, int32_t batch, uint32_t flags, void* stream,
                               nt_layout** out) {
  g_last_error.clear();
  if (!cols) return nt::fail(NT_ERR_INVALID_ARG, "cols is NULL");
  return build(rows, batch, flags, stream, out, cols);
}

nt_status nt_from_offsets(const int32_t* cu_seqlens, int32_t batch, uint32_t flags, void* stream,
                          nt_layout** out) {
  g_last_error.clear();
  if (!cu_seqlens) return nt::fail(NT_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (batch < 1) return nt::fail(NT_ERR_INVALID_ARG, "batch must be >= 1");
  if (cu_seqlens[0] != 0) return nt::fail(NT_ERR_INVALID_ARG, "offsets must start at 0");
  std::vector<int32_t> lengths(batch);
  for (int32_t i = 0; i < batch; ++i) {
    if (cu_seqlens[i + 1] < cu_seqlens[i])
      return nt::fail(NT_ERR_INVALID_ARG, "offsets must be non-decreasing (sample " + std::to_string(i) + ")");
    lengths[i] = cu_seqlens[i + 1] - cu_seqlens[i];
  }
  return build(lengths.data(), batch, flags, stream, out);
}

nt_status nt_layout_destroy(nt_layout* L) {
  if (!L) return NT_OK;
  nt_status st = NT_OK;
  if (L->d_base) {
    if (hipFree(L->d_base) != hipSuccess) st = nt::fail(NT_ERR_HIP, "hipFree of layout mirrors failed");
  }
  delete L;
  return st;
}

nt_status nt_layout_info(const nt_layout* L, nt_layout_info_t* info) {
  g_last_error.clear();
  if (!L || !info) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  info->batch = L->batch;
  info->max_len = L->max_len;
  info->sum_n = L->sum_n;
  info->sum_n2 = L->sum_n2;
  info->sum_n3 = L->sum_n3;
  info->sum_pad = L->sum_pad;
  info->d_cu_seqlens = L->d_cu_seqlens;
  info->d_cu_pairs = L->d_cu_pairs;
  info->d_row_splits2 = L->d_row_splits2;
  info->sum_m = L->sum_m;
  info->rect = L->rect ? 1 : 0;
  info->d_cu_cols = L->d_cu_cols;
  return NT_OK;
}

nt_status nt_layout_host_array(const nt_layout* L, nt_array which, const int32_t** data, int64_t* count) {
  g_last_error.clear();
  if (!L || !data || !count) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  const std::vector<int32_t>* v = nullptr;
  switch (which) {
    case NT_ARR_LENGTHS: v = &L->lengths; break;
    case NT_ARR_CU_SEQLENS: v = &L->cu_seqlens; break;
    case NT_ARR_CU_PAIRS: v = &L->cu_pairs; break;
    case NT_ARR_ROW_SPLITS2: v = &L->row_splits2; break;
    case NT_ARR_ROW_SAMPLE: v = &L->row_sample; break;
    case NT_ARR_ATTN_WORK: v = &L->attn_work; break;
    case NT_ARR_TRI_WORK: v = &L->tri_work; break;
    case NT_ARR_SEQ_WORK: v = &L->seq_work; break;
    case NT_ARR_CU_PAD: v = &L->cu_pad; break;
    case NT_ARR_COLS: v = &L->cols; break;
    case NT_ARR_CU_COLS: v = &L->cu_cols; break;
    case NT_ARR_TRI_SPLIT: v = &L->tri_split; break;
    default: return nt::fail(NT_ERR_INVALID_ARG, "unknown array id");
  }
  *data = v->data();
  *count = (int64_t)v->size();
  return NT_OK;
}

int32_t nt_layouts_compatible(const nt_layout* a, const nt_layout* b) {
  if (a && b && a != b && (a->rect || b->rect) && a->cols != b->cols) return 0;
  return (a && b && same_partition(a, b)) ? 1 : 0;
}

nt_status nt_pair_broadcast(const nt_layout* L, int32_t C, const void* u, int64_t ld_u, const void* v,
                            int64_t ld_v, void* z, int64_t ld_z, int32_t accumulate, nt_dtype dtype,
                            void* stream) {
  g_last_error.clear();
  if (nt_status st = need_device(L)) return st;
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "dtype must be NT_F32 or NT_BF16");
  if (C <= 0) return nt::fail(NT_ERR_INVALID_ARG, "C must be > 0");
  if (accumulate != 0 && accumulate != 1) return nt::fail(NT_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  const int ve = vec_elems(dtype);
  if (C % ve) return nt::fail(NT_ERR_INVALID_ARG, "C must be a multiple of " + std::to_string(ve));
  if (L->sum_n2 == 0) return NT_OK;
  if (!u || !v || !z) return nt::fail(NT_ERR_INVALID_ARG, "u, v and z must be non-NULL");
  if (!aligned16(u) || !aligned16(v) || !aligned16(z)) return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  if (ld_u < C || ld_v < C || ld_z < C || ld_u % ve || ld_v % ve || ld_z % ve)
    return nt::fail(NT_ERR_INVALID_ARG, "row strides must be >= C and multiples of the vector width");
  return check_hip(nt::launch_pair_broadcast(*L, C, u, ld_u, v, ld_v, z, ld_z, accumulate, dtype,
                                             static_cast<hipStream_t>(stream)),
                   "nt_pair_broadcast launch");
}

nt_status nt_segment_reduce(const nt_layout* L, nt_level level, int32_t op, int32_t C, const void* x,
                            int64_t ld_x, nt_dtype x_dtype, float* y, int64_t ld_y, void* stream) {
  g_last_error.clear();
  if (nt_status st = need_device(L)) return st;
  if (level != NT_LEVEL_SINGLES && level != NT_LEVEL_PAIRS && level != NT_LEVEL_PAIRS_FIRST)
    return nt::fail(NT_ERR_INVALID_ARG, "bad level");
  if (op != 0 && op != 1) return nt::fail(NT_ERR_INVALID_ARG, "op must be 0 (sum) or 1 (mean)");
  if (!valid_dtype(x_dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (C <= 0) return nt::fail(NT_ERR_INVALID_ARG, "C must be > 0");
  const int ve = vec_elems(x_dtype);
  if (C % ve || ld_x % ve || ld_x < C) return nt::fail(NT_ERR_INVALID_ARG, "C and ld_x must be multiples of the vector width, ld_x >= C");
  if (ld_y < C || ld_y % 4) return nt::fail(NT_ERR_INVALID_ARG, "ld_y must be >= C and a multiple of 4");
  const int64_t out_rows = level == NT_LEVEL_PAIRS ? L->sum_n : (level == NT_LEVEL_PAIRS_FIRST ? L->sum_m : L->batch);
  if (out_rows == 0) return NT_OK;
  if (!y) return nt::fail(NT_ERR_INVALID_ARG, "y is NULL");
  if (!x && (level != NT_LEVEL_SINGLES ? L->sum_n2 : L->sum_n) > 0) return nt::fail(NT_ERR_INVALID_ARG, "x is NULL");
  if ((x && !aligned16(x)) || !aligned16(y)) return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  return check_hip(nt::launch_segment_reduce(*L, level, op, C, x, ld_x, x_dtype, y, ld_y,
                                             static_cast<hipStream_t>(stream)),
                   "nt_segment_reduce launch");
}

nt_status nt_pair_broadcast_backward(const nt_layout* L, int32_t C, const void* dz, int64_t ld_dz, nt_dtype dtype,
                                     void* du, int64_t ld_du, void* dv, int64_t ld_dv, nt_dtype out_dtype,
                                     int32_t accumulate, void* stream) {
  g_last_error.clear();
  if (nt_status st = need_device(L)) return st;
  if (!valid_dtype(dtype) || !valid_dtype(out_dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (C <= 0 || C % vec_elems(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "C must be > 0 and a multiple of the vector width");
  if (accumulate != 0 && accumulate != 1) return nt::fail(NT_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  if (ld_dz < C || ld_dz % vec_elems(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad ld_dz");
  if ((du && ld_du < C) || (dv && ld_dv < C)) return nt::fail(NT_ERR_INVALID_ARG, "ld_du / ld_dv must be >= C");
  if (L->sum_n2 == 0 || (!du && !dv)) return NT_OK;
  if (!dz) return nt::fail(NT_ERR_INVALID_ARG, "dz is NULL");
  if (!aligned16(dz) || (du && (reinterpret_cast<uintptr_t>(du) & 3u)) || (dv && (reinterpret_cast<uintptr_t>(dv) & 3u)))
    return nt::fail(NT_ERR_INVALID_ARG, "misaligned pointer");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (du) {
    if (nt_status st = check_hip(nt::launch_segment_reduce(*L, NT_LEVEL_PAIRS, 0, C, dz, ld_dz, dtype, du, ld_du, s,
                                                           accumulate, out_dtype),
                                 "nt_pair_broadcast_backward launch"))
      return st;
  }
  if (dv) {
    if (nt_status st = check_hip(nt::launch_segment_reduce(*L, NT_LEVEL_PAIRS_FIRST, 0, C, dz, ld_dz, dtype, dv, ld_dv,
                                                           s, accumulate, out_dtype),
                                 "nt_pair_broadcast_backward launch"))
      return st;
  }
  return NT_OK;
}

nt_status nt_weighted_square_loss_workspace(const nt_layout* L, uint64_t* bytes) {
  g_last_error.clear();
  if (!L || !bytes) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  *bytes = nt::loss_workspace_bytes(*L);
  return NT_OK;
}

nt_status nt_weighted_square_loss(const nt_layout* L, nt_level level, int32_t C, const void* x, int64_t ld_x,
                                  nt_dtype dtype, const float* weights, float scale, float* loss, void* dx,
                                  int64_t ld_dx, nt_dtype dx_dtype, void* workspace, uint64_t workspace_bytes,
                                  void* stream) {
  g_last_error.clear();
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (level != NT_LEVEL_SINGLES && level != NT_LEVEL_PAIRS) return nt::fail(NT_ERR_INVALID_ARG, "level must be singles or pairs");
  if (!valid_dtype(dtype) || !valid_dtype(dx_dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  const int ve = vec_elems(dtype);
  if (C <= 0 || C % ve || ld_x < C || ld_x % ve) return nt::fail(NT_ERR_INVALID_ARG, "C and ld_x must be multiples of the vector width, ld_x >= C");
  if (dx && ld_dx < C) return nt::fail(NT_ERR_INVALID_ARG, "ld_dx must be >= C");
  if (!(scale == scale)) return nt::fail(NT_ERR_INVALID_ARG, "scale is NaN");
  if (nt_status st = need_workspace(nt::loss_workspace_bytes(*L), workspace, workspace_bytes,
                                    "nt_weighted_square_loss_workspace"))
    return st;
  if (nt_status st = need_device(L)) return st;
  if (!weights || !loss) return nt::fail(NT_ERR_INVALID_ARG, "weights and loss must be non-NULL");
  if ((L->sum_n > 0 && !x) || (x && !aligned16(x))) return nt::fail(NT_ERR_INVALID_ARG, "x is NULL or misaligned");
  if (dx && (reinterpret_cast<uintptr_t>(dx) & 3u)) return nt::fail(NT_ERR_INVALID_ARG, "dx misaligned");
  return check_hip(nt::launch_weighted_square_loss(*L, level, C, x, ld_x, dtype, weights, scale, loss, dx, ld_dx,
                                                   dx_dtype, workspace, static_cast<hipStream_t>(stream)),
                   "nt_weighted_square_loss launch");
}

nt_status nt_segment_reduce_backward(const nt_layout* L, nt_level level, int32_t op, int32_t C, const float* dy,
                                     int64_t ld_dy, void* dx, int64_t ld_dx, nt_dtype dtype, int32_t accumulate,
                                     void* stream) {
  g_last_error.clear();
  if (nt_status st = need_device(L)) return st;
  if (level != NT_LEVEL_SINGLES && level != NT_LEVEL_PAIRS && level != NT_LEVEL_PAIRS_FIRST)
    return nt::fail(NT_ERR_INVALID_ARG, "bad level");
  if (op != 0 && op != 1) return nt::fail(NT_ERR_INVALID_ARG, "op must be 0 (sum) or 1 (mean)");
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (accumulate != 0 && accumulate != 1) return nt::fail(NT_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  const int ve = vec_elems(dtype);
  if (C <= 0 || C % ve || ld_dx < C || ld_dx % ve) return nt::fail(NT_ERR_INVALID_ARG, "C and ld_dx must be multiples of the vector width, ld_dx >= C");
  if (ld_dy < C) return nt::fail(NT_ERR_INVALID_ARG, "ld_dy must be >= C");
  if (L->sum_n == 0) return NT_OK;
  if (!dy || !dx) return nt::fail(NT_ERR_INVALID_ARG, "dy and dx must be non-NULL");
  if (!aligned16(dx) || (reinterpret_cast<uintptr_t>(dy) & 3u)) return nt::fail(NT_ERR_INVALID_ARG, "misaligned pointer");
  return check_hip(nt::launch_segment_reduce_backward(*L, level, op, C, dy, ld_dy, dx, ld_dx, dtype, accumulate,
                                                      static_cast<hipStream_t>(stream)),
                   "nt_segment_reduce_backward launch");
}

nt_status nt_layernorm_linear(const nt_linear_args* a, void* stream) {
  g_last_error.clear();
  if (!a) return nt::fail(NT_ERR_INVALID_ARG, "args is NULL");
  if (!valid_dtype(a->dtype) || !valid_dtype(a->x_dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (a->dtype == NT_F32 && a->x_dtype != NT_F32) return nt::fail(NT_ERR_INVALID_ARG, "f32 weights need f32 input");
  if (a->rows < 0 || a->c_in <= 0 || a->c_out <= 0) return nt::fail(NT_ERR_INVALID_ARG, "bad sizes");
  if (a->rows > INT32_MAX) return nt::fail(NT_ERR_OVERFLOW, "rows exceed int32");
  if (a->c_in % 8) return nt::fail(NT_ERR_INVALID_ARG, "c_in must be a multiple of 8");
  if (a->epilogue < NT_EPI_NONE || a->epilogue > NT_EPI_SIGMOID_GLU) return nt::fail(NT_ERR_INVALID_ARG, "bad epilogue");
  if (a->ln_beta && !a->ln_gamma) return nt::fail(NT_ERR_INVALID_ARG, "ln_beta without ln_gamma");
  if (a->ln_gamma && !(a->ln_eps >= 0.f)) return nt::fail(NT_ERR_INVALID_ARG, "ln_eps must be >= 0");
  const bool gated = a->epilogue == NT_EPI_GATED_RESIDUAL;
  const bool swiglu = a->epilogue == NT_EPI_SWIGLU_RESIDUAL;
  const int vx = vec_elems(a->x_dtype), vy = vec_elems(a->dtype);
  const bool bcast = a->bcast_u || a->bcast_v;
  if (bcast) {
    if (!a->bcast_u || !a->bcast_v) return nt::fail(NT_ERR_INVALID_ARG, "broadcast rows need both bcast_u and bcast_v");
    if (a->x) return nt::fail(NT_ERR_INVALID_ARG, "x must be NULL with broadcast rows");
    if (!a->layout || a->level != NT_LEVEL_PAIRS) return nt::fail(NT_ERR_INVALID_ARG, "broadcast rows need a pair-level layout");
    if (!a->layout->has_device) return nt::fail(NT_ERR_INVALID_ARG, "broadcast rows need a layout with device mirrors");
    if (nt_status st = need_square(a->layout, "broadcast rows")) return st;
    if (a->dtype != NT_BF16 || a->x_dtype != NT_BF16 || (a->c_in != 64 && a->c_in != 128) || a->c_out > 512 ||
        a->c_out % 8 || (a->epilogue != NT_EPI_NONE && a->epilogue != NT_EPI_GELU) || a->n_tail || a->residual)
      return nt::fail(NT_ERR_UNSUPPORTED, "broadcast rows: bf16, c_in in {64, 128}, c_out <= 512 (multiple of 8), "
                                          "epilogue none or gelu, no tail, no residual");
    if (a->ld_bcast_u < a->c_in || a->ld_bcast_u % 8 || a->ld_bcast_v < a->c_in || a->ld_bcast_v % 8)
      return nt::fail(NT_ERR_INVALID_ARG, "ld_bcast_u/v must be >= c_in and multiples of 8");
    if (!aligned16(a->bcast_u) || !aligned16(a->bcast_v)) return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  } else if (a->ldx < a->c_in || a->ldx % vx) {
    return nt::fail(NT_ERR_INVALID_ARG, "ldx must be >= c_in and a multiple of the vector width");
  }
  if (a->n_tail < 0 || a->n_tail > a->c_out) return nt::fail(NT_ERR_INVALID_ARG, "n_tail out of range");
  if (a->tail_layout < NT_TAIL_CHANNEL_MAJOR || a->tail_layout > NT_TAIL_PAIR_TILED_T)
    return nt::fail(NT_ERR_INVALID_ARG, "bad tail_layout");
  const int n_main = a->c_out - a->n_tail;
  if (a->layout) {
    if (!a->layout->has_device && a->n_tail && a->tail_layout != NT_TAIL_CHANNEL_MAJOR)
      return nt::fail(NT_ERR_INVALID_ARG, "pair-tiled tails need a layout with device mirrors");
    const int64_t expect = a->level == NT_LEVEL_PAIRS ? a->layout->sum_n2 : a->layout->sum_n;
    if (a->level != NT_LEVEL_PAIRS && a->level != NT_LEVEL_SINGLES) return nt::fail(NT_ERR_INVALID_ARG, "bad level");
    if (expect != a->rows) return nt::fail(NT_ERR_LAYOUT_MISMATCH, "rows differ from the layout's row count");
  }
  if (a->residual_layout && !same_partition(a->layout, a->residual_layout))
    return nt::fail(NT_ERR_LAYOUT_MISMATCH, "residual has a different logical partition than x");
  if (a->n_tail && a->tail_layout != NT_TAIL_CHANNEL_MAJOR &&
      (!a->layout || a->level != NT_LEVEL_PAIRS || a->layout->rect))
    return nt::fail(NT_ERR_UNSUPPORTED, "pair-tiled tail output needs a square pair-level layout");
  if (swiglu) {
    if (a->dtype == NT_BF16 && (a->c_in != a->c_out || (a->c_in != 64 && a->c_in != 128 && a->c_in != 256) ||
                                a->hidden <= 0 || a->hidden % 32 || a->x_dtype != NT_BF16))
      return nt::fail(NT_ERR_UNSUPPORTED, "bf16 SwiGLU needs bf16 x, c_in == c_out in {64, 128, 256} and hidden % 32 == 0");
    if (a->dtype == NT_F32 && (a->c_in > 1024 || a->hidden <= 0 || a->hidden > 4096))
      return nt::fail(NT_ERR_UNSUPPORTED, "f32 SwiGLU needs c_in <= 1024 and 0 < hidden <= 4096");
    if (a->n_tail) return nt::fail(NT_ERR_UNSUPPORTED, "SwiGLU has no tail output");
    if (!a->w2) return nt::fail(NT_ERR_INVALID_ARG, "SwiGLU needs w2");
    if (!a->residual && a->c_out != a->c_in) return nt::fail(NT_ERR_INVALID_ARG, "SwiGLU without residual needs c_out == c_in");
    if (!a->residual && a->x_dtype != a->dtype) return nt::fail(NT_ERR_INVALID_ARG, "SwiGLU residual = x needs x in the output dtype");
  }
  if (a->dtype == NT_F32 && !swiglu && a->c_in > 4096) return nt::fail(NT_ERR_UNSUPPORTED, "f32 path needs c_in <= 4096");
  if (a->epilogue == NT_EPI_RESIDUAL && !a->residual) return nt::fail(NT_ERR_INVALID_ARG, "residual epilogue needs residual");
  if (gated && (!a->residual || !a->gate)) return nt::fail(NT_ERR_INVALID_ARG, "gated residual epilogue needs residual and gate");
  if (gated && a->n_tail) return nt::fail(NT_ERR_UNSUPPORTED, "the gated residual epilogue has no tail output");
  if (!gated && a->gate) return nt::fail(NT_ERR_INVALID_ARG, "gate is only read by the gated residual epilogue");
  if (a->epilogue == NT_EPI_SIGMOID_GLU &&
      (a->dtype != NT_BF16 || a->x_dtype != NT_BF16 || a->c_in != 128 || a->hidden != 128 || a->c_out != 256 ||
       a->n_tail != a->c_out || a->tail_layout == NT_TAIL_CHANNEL_MAJOR || bcast || a->residual ||
       !a->layout || a->layout->batch > nt::kPairTiledMaxSamples))
    return nt::fail(NT_ERR_UNSUPPORTED, "the sigmoid GLU epilogue supports bf16, c_in = hidden = 128 and 256 outputs, "
                                        "all in a pair-tiled tail");
  if (a->rows == 0) return NT_OK;
  if ((!a->x && !bcast) || !a->w) return nt::fail(NT_ERR_INVALID_ARG, "x and w must be non-NULL");
  if (n_main > 0 && !a->y) return nt::fail(NT_ERR_INVALID_ARG, "y is NULL");
  if (a->n_tail > 0 && !a->y_tail) return nt::fail(NT_ERR_INVALID_ARG, "y_tail is NULL");
  if ((a->ln_gamma && !aligned16(a->ln_gamma)) || (a->ln_beta && !aligned16(a->ln_beta)))
    return nt::fail(NT_ERR_INVALID_ARG, "ln_gamma and ln_beta must be 16-byte aligned");
  if ((a->x && !aligned16(a->x)) || !aligned16(a->w) || (a->y && !aligned16(a->y)) || (a->residual && !aligned16(a->residual)) ||
      (a->w2 && !aligned16(a->w2)) || (a->y_tail && !aligned16(a->y_tail)))
    return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  if (n_main > 0 && (a->ldy < n_main || a->ldy % vy)) return nt::fail(NT_ERR_INVALID_ARG, "ldy must be >= the main width and a multiple of the vector width");
  if (a->residual && (a->ld_residual < n_main || a->ld_residual % vy)) return nt::fail(NT_ERR_INVALID_ARG, "bad ld_residual");
  if (gated && (a->ld_gate < n_main || a->ld_gate % vy || !aligned16(a->gate)))
    return nt::fail(NT_ERR_INVALID_ARG, "gate must be 16-byte aligned with ld_gate >= c_out, a multiple of the vector width");
  if (a->n_tail > 0) {
    const int64_t need = a->tail_layout == NT_TAIL_CHANNEL_MAJOR ? a->rows : a->layout->sum_pad;
    if (a->ld_tail < need) return nt::fail(NT_ERR_INVALID_ARG, "ld_tail is smaller than the tail's row extent");
    if (a->tail_layout != NT_TAIL_CHANNEL_MAJOR && a->ld_tail % 8)
      return nt::fail(NT_ERR_INVALID_ARG, "pair-tiled tails need ld_tail % 8 == 0");
  }
  if (nt_status st = need_workspace(nt::linear_workspace_bytes(*a), a->workspace, a->workspace_bytes,
                                    "nt_layernorm_linear_workspace"))
    return st;
  nt::LinearPlan p{a, a->tail_layout, a->layout};
  return check_hip(nt::launch_linear(p, static_cast<hipStream_t>(stream)), "nt_layernorm_linear launch");
}

nt_status nt_layernorm_linear_workspace(const nt_linear_args* a, uint64_t* bytes) {
  g_last_error.clear();
  if (!a || !bytes) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  *bytes = a->rows > 0 ? (uint64_t)nt::linear_workspace_bytes(*a) : 0;
  return NT_OK;
}

nt_status nt_layernorm_linear_backward_workspace(const nt_linear_bwd_args* a, uint64_t* bytes) {
  g_last_error.clear();
  if (!a || !bytes) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  *bytes = a->rows > 0 && a->c_in > 0 && a->c_out > 0 ? (uint64_t)nt::linear_backward_workspace_bytes(*a) : 0;
  return NT_OK;
}

nt_status nt_layernorm_linear_backward(const nt_linear_bwd_args* a, void* stream) {
  g_last_error.clear();
  if (!a) return nt::fail(NT_ERR_INVALID_ARG, "args is NULL");
  if (a->rows < 0 || a->c_in <= 0 || a->c_out <= 0) return nt::fail(NT_ERR_INVALID_ARG, "bad sizes");
  if (a->rows > INT32_MAX) return nt::fail(NT_ERR_OVERFLOW, "rows exceed int32");
  if (a->c_in % 8 || a->c_in > 1024) return nt::fail(NT_ERR_UNSUPPORTED, "c_in must be a multiple of 8 and <= 1024");
  if (!valid_dtype(a->x_dtype) || !valid_dtype(a->dx_dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  const bool swiglu = a->epilogue == NT_EPI_SWIGLU_RESIDUAL;
  if (a->epilogue < NT_EPI_NONE || a->epilogue > NT_EPI_GELU) return nt::fail(NT_ERR_INVALID_ARG, "bad epilogue");
  if (swiglu && (a->hidden <= 0 || !a->w2)) return nt::fail(NT_ERR_INVALID_ARG, "SwiGLU needs hidden > 0 and w2");
  if (swiglu && a->residual_is_x && (a->c_out != a->c_in || !a->ln_gamma || a->dx_dtype != NT_BF16))
    return nt::fail(NT_ERR_UNSUPPORTED, "SwiGLU with residual x needs c_out == c_in, a LayerNorm and a bf16 dx");
  if (!a->ln_gamma && a->dx && a->dx_dtype == NT_BF16 && a->accumulate_dx)
    return nt::fail(NT_ERR_UNSUPPORTED, "without a LayerNorm a bf16 dx cannot accumulate");
  if (a->ln_beta && !a->ln_gamma) return nt::fail(NT_ERR_INVALID_ARG, "ln_beta without ln_gamma");
  if (a->ldx < a->c_in || a->ld_dy < a->c_out || (a->dx && a->ld_dx < a->c_in))
    return nt::fail(NT_ERR_INVALID_ARG, "row strides too small");
  if (a->x_dtype == NT_F32 && !a->ln_gamma && a->ldx != a->c_in)
    return nt::fail(NT_ERR_UNSUPPORTED, "fp32 x without a LayerNorm must be contiguous");
  if (a->rows == 0) return NT_OK;
  if (!a->x || !a->w || !a->dy) return nt::fail(NT_ERR_INVALID_ARG, "x, w and dy must be non-NULL");
  if (!aligned16(a->x) || !aligned16(a->w) || !aligned16(a->dy) || (a->dx && !aligned16(a->dx)) ||
      (a->w2 && !aligned16(a->w2)) || (a->ln_gamma && !aligned16(a->ln_gamma)) ||
      (a->ln_beta && !aligned16(a->ln_beta)) || (a->bias && !aligned16(a->bias)))
    return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  if (nt_status st = need_workspace(nt::linear_backward_workspace_bytes(*a), a->workspace, a->workspace_bytes,
                                    "nt_layernorm_linear_backward_workspace"))
    return st;
  return check_hip(nt::launch_linear_backward(*a, a->workspace, static_cast<hipStream_t>(stream)),
                   "nt_layernorm_linear_backward launch");
}

namespace {
nt_status pair_row_attention(const nt_layout* L, int32_t axis, int32_t H, int32_t D, const void* q,
                             const void* k, const void* v, int64_t ld_qkv, const void* gate, int64_t ld_gate,
                             const void* bias, int64_t ld_bias, int64_t ld_bias_head, float scale, void* o,
                             int64_t ld_o, nt_dtype dtype, void* workspace, uint64_t workspace_bytes, void* stream) {
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (axis < 0 || axis > 3) return nt::fail(NT_ERR_INVALID_ARG, "axis must be 0, 1, 2 or 3");
  if (axis != 2) if (nt_status st = need_square(L, "pair attention")) return st;
  if (axis == 3 && (dtype != NT_BF16 || D != 32 || L->max_len > nt::kAttnLongLen))
    return nt::fail(NT_ERR_UNSUPPORTED, "single attention with pair bias supports bf16, head_dim 32, N_i <= " +
                                            std::to_string(nt::kAttnLongLen));
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (H <= 0 || D <= 0) return nt::fail(NT_ERR_INVALID_ARG, "heads and head_dim must be > 0");
  if (dtype == NT_BF16 && D != 32 && D != 64) return nt::fail(NT_ERR_UNSUPPORTED, "bf16 attention supports head_dim 32 or 64");
  if (dtype == NT_F32 && D != 8 && D != 16 && D != 32 && D != 64) return nt::fail(NT_ERR_UNSUPPORTED, "f32 attention supports head_dim 8, 16, 32 or 64");
  if (axis == 2 && bias) return nt::fail(NT_ERR_INVALID_ARG, "1-D attention takes no pair bias");
  const int ve = vec_elems(dtype);
  if ((int64_t)H * D > ld_qkv || ld_qkv % ve || (int64_t)H * D > ld_o || ld_o % ve)
    return nt::fail(NT_ERR_INVALID_ARG, "row strides must hold H*head_dim and be multiples of the vector width");
  const int lim = dtype == NT_F32 ? 4096 : (D == 32 ? nt::kAttnMaxLenD32 : nt::kAttnMaxLenD64);
  if (L->max_len > lim) return nt::fail(NT_ERR_UNSUPPORTED, "a sample is longer than the attention limit " + std::to_string(lim));
  const int64_t rows = axis >= 2 ? L->sum_n : L->sum_n2;
  if (bias && (ld_bias <= 0 || ld_bias_head <= 0)) return nt::fail(NT_ERR_INVALID_ARG, "bias strides must be positive");
  if (nt_status st = need_workspace(nt::attention_workspace_bytes(*L, axis, H, D, dtype, bias != nullptr), workspace,
                                    workspace_bytes, "nt_pair_row_attention_workspace"))
    return st;
  if (nt_status st = need_device(L)) return st;
  if (rows == 0) return NT_OK;
  if (!q || !k || !v || !o) return nt::fail(NT_ERR_INVALID_ARG, "q, k, v and o must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
      (bias && (reinterpret_cast<uintptr_t>(bias) & (dtype == NT_BF16 ? 1u : 3u))))
    return nt::fail(NT_ERR_INVALID_ARG, "q, k, v, o must be 16-byte aligned, bias element-aligned");
  if (!(scale == scale)) return nt::fail(NT_ERR_INVALID_ARG, "scale is NaN");
  if (gate && ((int64_t)H * D > ld_gate || ld_gate % ve || !aligned16(gate)))
    return nt::fail(NT_ERR_INVALID_ARG, "gate must be 16-byte aligned with ld_gate >= H*head_dim, a multiple of the vector width");
  return check_hip(nt::launch_attention(*L, axis, H, D, q, k, v, ld_qkv, bias, ld_bias, ld_bias_head, scale, o, ld_o,
                                        dtype, workspace, static_cast<hipStream_t>(stream), gate, ld_gate),
                   "nt_pair_row_attention launch");
}
}  // namespace

nt_status nt_pair_row_attention(const nt_layout* L, int32_t axis, int32_t H, int32_t D, const void* q,
                                const void* k, const void* v, int64_t ld_qkv, const void* bias,
                                int64_t ld_bias, int64_t ld_bias_head, float scale, void* o, int64_t ld_o,
                                nt_dtype dtype, void* workspace, uint64_t workspace_bytes, void* stream) {
  g_last_error.clear();
  return pair_row_attention(L, axis, H, D, q, k, v, ld_qkv, nullptr, 0, bias, ld_bias, ld_bias_head, scale, o, ld_o,
                            dtype, workspace, workspace_bytes, stream);
}

nt_status nt_pair_row_attention_gated(const nt_layout* L, int32_t axis, int32_t H, int32_t D, const void* q,
                                      const void* k, const void* v, int64_t ld_qkv, const void* gate,
                                      int64_t ld_gate, const void* bias, int64_t ld_bias, int64_t ld_bias_head,
                                      float scale, void* o, int64_t ld_o, nt_dtype dtype, void* workspace,
                                      uint64_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (axis != 0 && axis != 1) return nt::fail(NT_ERR_INVALID_ARG, "the gated attention covers axes 0 and 1");
  if (!gate && L && L->sum_n2 > 0) return nt::fail(NT_ERR_INVALID_ARG, "gate is NULL");
  return pair_row_attention(L, axis, H, D, q, k, v, ld_qkv, gate, ld_gate, bias, ld_bias, ld_bias_head, scale, o,
                            ld_o, dtype, workspace, workspace_bytes, stream);
}

nt_status nt_cross_attention(const nt_layout* Lq, const nt_layout* Lkv, int32_t H, int32_t D, const void* q,
                             int64_t ld_q, const void* k, const void* v, int64_t ld_kv, float scale, void* o,
                             int64_t ld_o, nt_dtype dtype, void* stream) {
  g_last_error.clear();
  if (!Lq || !Lkv) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (Lq->batch != Lkv->batch)
    return nt::fail(NT_ERR_LAYOUT_MISMATCH, "query and key layouts hold different batch sizes (" +
                                                std::to_string(Lq->batch) + " vs " + std::to_string(Lkv->batch) + ")");
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (H <= 0 || D <= 0) return nt::fail(NT_ERR_INVALID_ARG, "heads and head_dim must be > 0");
  if (dtype == NT_BF16 && D != 32 && D != 64)
    return nt::fail(NT_ERR_UNSUPPORTED, "bf16 cross-attention supports head_dim 32 or 64");
  if (dtype == NT_F32 && D != 8 && D != 16 && D != 32 && D != 64)
    return nt::fail(NT_ERR_UNSUPPORTED, "f32 cross-attention supports head_dim 8, 16, 32 or 64");
  if (dtype == NT_BF16 && Lkv->max_len > nt::kAttnLongLen)
    return nt::fail(NT_ERR_UNSUPPORTED, "bf16 cross-attention supports at most " + std::to_string(nt::kAttnLongLen) +
                                            " keys per sample");
  if (dtype == NT_F32 && Lkv->max_len > 4096)
    return nt::fail(NT_ERR_UNSUPPORTED, "f32 cross-attention supports at most 4096 keys per sample");
  const int ve = vec_elems(dtype);
  const int64_t c = (int64_t)H * D;
  if (c > ld_q || c > ld_kv || c > ld_o || ld_q % ve || ld_kv % ve || ld_o % ve)
    return nt::fail(NT_ERR_INVALID_ARG, "row strides must hold H*head_dim and be multiples of the vector width");
  if (!(scale == scale)) return nt::fail(NT_ERR_INVALID_ARG, "scale is NaN");
  if (nt_status st = need_device(Lq)) return st;
  if (nt_status st = need_device(Lkv)) return st;
  if (Lq->sum_n == 0) return NT_OK;
  if (!q || !o || (Lkv->sum_n > 0 && (!k || !v))) return nt::fail(NT_ERR_INVALID_ARG, "q, k, v and o must be non-NULL");
  if (!aligned16(q) || !aligned16(o) || (k && !aligned16(k)) || (v && !aligned16(v)))
    return nt::fail(NT_ERR_INVALID_ARG, "q, k, v, o must be 16-byte aligned");
  return check_hip(nt::launch_cross_attention(*Lq, *Lkv, H, D, q, ld_q, k, v, ld_kv, scale, o, ld_o, dtype,
                                              static_cast<hipStream_t>(stream)),
                   "nt_cross_attention launch");
}

nt_status nt_pair_row_attention_backward_workspace(const nt_layout* L, int32_t axis, int32_t H, int32_t D,
                                                   nt_dtype dtype, uint64_t* bytes) {
  g_last_error.clear();
  if (!L || !bytes) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  if (axis < 0 || axis > 1 || H <= 0 || D <= 0 || !valid_dtype(dtype))
    return nt::fail(NT_ERR_INVALID_ARG, "bad axis, heads, head_dim or dtype");
  *bytes = nt::attention_backward_workspace_bytes(*L, H);
  return NT_OK;
}

nt_status nt_pair_row_attention_backward(const nt_layout* L, int32_t axis, int32_t H, int32_t D, const void* q,
                                         const void* k, const void* v, int64_t ld_qkv, const void* bias,
                                         int64_t ld_bias, int64_t ld_bias_head,
                                         const void* dout, int64_t ld_dout, float scale, void* dq, void* dk, void* dv,
                                         int64_t ld_dqkv, float* dbias, int64_t ld_dbias, int64_t ld_dbias_head,
                                         nt_dtype dtype, void* workspace, uint64_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (nt_status st = need_square(L, "pair attention")) return st;
  if (axis != 0 && axis != 1) return nt::fail(NT_ERR_UNSUPPORTED, "the attention backward covers axes 0 and 1");
  if (dtype != NT_BF16 || D != 32) return nt::fail(NT_ERR_UNSUPPORTED, "the attention backward needs bf16 and head_dim 32");
  if (H <= 0) return nt::fail(NT_ERR_INVALID_ARG, "heads must be > 0");
  if (L->max_len > nt::kAttnLongLen)
    return nt::fail(NT_ERR_UNSUPPORTED, "the attention backward supports N_i <= " + std::to_string(nt::kAttnLongLen));
  if ((int64_t)H * D > ld_qkv || ld_qkv % 8 || (int64_t)H * D > ld_dout ||
      ld_dout % 8 || (int64_t)H * D > ld_dqkv || ld_dqkv % 8)
    return nt::fail(NT_ERR_INVALID_ARG, "row strides must hold H*head_dim and be multiples of 8");
  if (bias && (ld_bias <= 0 || ld_bias_head <= 0)) return nt::fail(NT_ERR_INVALID_ARG, "bias strides must be positive");
  if (dbias && (ld_dbias <= 0 || ld_dbias_head <= 0)) return nt::fail(NT_ERR_INVALID_ARG, "dbias strides must be positive");
  if (!(scale == scale)) return nt::fail(NT_ERR_INVALID_ARG, "scale is NaN");
  if (nt_status st = need_workspace(nt::attention_backward_workspace_bytes(*L, H), workspace, workspace_bytes,
                                    "nt_pair_row_attention_backward_workspace"))
    return st;
  if (nt_status st = need_device(L)) return st;
  if (L->sum_n2 == 0) return NT_OK;
  if (!q || !k || !v || !dout || !dq || !dk || !dv) return nt::fail(NT_ERR_INVALID_ARG, "NULL tensor");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(dq) ||
      !aligned16(dk) || !aligned16(dv) || (bias && (reinterpret_cast<uintptr_t>(bias) & 1u)) ||
      (dbias && (reinterpret_cast<uintptr_t>(dbias) & 3u)))
    return nt::fail(NT_ERR_INVALID_ARG, "misaligned pointer");
  return check_hip(nt::launch_attention_backward(*L, axis, H, q, k, v, ld_qkv, bias, ld_bias, ld_bias_head,
                                                 dout, ld_dout, scale, dq, dk, dv, ld_dqkv, dbias, ld_dbias,
                                                 ld_dbias_head, workspace, static_cast<hipStream_t>(stream)),
                   "nt_pair_row_attention_backward launch");
}

nt_status nt_pair_row_attention_noalloc(const nt_layout* L, int32_t axis, int32_t H, int32_t D, const void* q,
                                        const void* k, const void* v, int64_t ld_qkv, const void* bias,
                                        int64_t ld_bias, int64_t ld_bias_head, float scale, void* o, int64_t ld_o,
                                        nt_dtype dtype, void* stream) {
  g_last_error.clear();
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (axis < 0 || axis > 3 || H <= 0 || D <= 0 || !valid_dtype(dtype))
    return nt::fail(NT_ERR_INVALID_ARG, "bad axis, heads, head_dim or dtype");
  const size_t need = nt::attention_workspace_bytes(*L, axis, H, D, dtype, bias != nullptr);
  if (need > nt::kNoAllocScratchBytes)
    return nt::fail(NT_ERR_UNSUPPORTED, "this call needs " + std::to_string(need) + " bytes of scratch; the "
                                        "allocation-free entry point holds " + std::to_string(nt::kNoAllocScratchBytes) +
                                        " (use nt_pair_row_attention with a workspace)");
  void* ws = nullptr;
  if (need > 0) {
    if (nt_status st = need_device(L)) return st;
    if (nt_status st = check_hip(nt::noalloc_scratch(&ws), "scratch address lookup")) return st;
  }
  return nt_pair_row_attention(L, axis, H, D, q, k, v, ld_qkv, bias, ld_bias, ld_bias_head, scale, o, ld_o, dtype,
                               ws, need, stream);
}

nt_status nt_pair_row_attention_workspace(const nt_layout* L, int32_t axis, int32_t H, int32_t D, nt_dtype dtype,
                                          int32_t has_bias, uint64_t* bytes) {
  g_last_error.clear();
  if (!L || !bytes) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  if (axis < 0 || axis > 3 || H <= 0 || D <= 0 || !valid_dtype(dtype) || (has_bias != 0 && has_bias != 1))
    return nt::fail(NT_ERR_INVALID_ARG, "bad axis, heads, head_dim, dtype or has_bias");
  *bytes = nt::attention_workspace_bytes(*L, axis, H, D, dtype, has_bias != 0);
  return NT_OK;
}

nt_status nt_triangle_mul(const nt_layout* L, int32_t direction, int32_t C, const void* a, const void* b,
                          int64_t ld_ab, nt_tri_operands operands, void* z, int64_t ld_z, nt_dtype dtype,
                          void* workspace, uint64_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (nt_status st = need_square(L, "the triangle update")) return st;
  if (direction != 0 && direction != 1) return nt::fail(NT_ERR_INVALID_ARG, "direction must be 0 or 1");
  if (operands != NT_TRI_PACKED && operands != NT_TRI_PAIR_TILED && operands != NT_TRI_PAIR_TILED_T)
    return nt::fail(NT_ERR_INVALID_ARG, "bad operand layout");
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (C <= 0) return nt::fail(NT_ERR_INVALID_ARG, "C must be > 0");
  if (dtype == NT_BF16 && C % 32) return nt::fail(NT_ERR_INVALID_ARG, "bf16 triangle needs C % 32 == 0");
  const int ve = vec_elems(dtype);
  if (dtype == NT_F32 && C % ve) return nt::fail(NT_ERR_INVALID_ARG, "f32 triangle needs C % 4 == 0");
  if (ld_z < C || ld_z % ve) return nt::fail(NT_ERR_INVALID_ARG, "ld_z must be >= C and a multiple of the vector width");
  if (operands == NT_TRI_PACKED) {
    if (ld_ab < C || ld_ab % ve) return nt::fail(NT_ERR_INVALID_ARG, "packed operands: ld_ab must be >= C and a multiple of the vector width");
  } else {
    if ((operands == NT_TRI_PAIR_TILED) != (direction == 0))
      return nt::fail(NT_ERR_INVALID_ARG, direction == 0
                                              ? "the outgoing update needs the plain pair-tiled variant (NT_TRI_PAIR_TILED)"
                                              : "the incoming update needs the transposed pair-tiled variant (NT_TRI_PAIR_TILED_T)");
    if (ld_ab < L->sum_pad || ld_ab % 8) return nt::fail(NT_ERR_INVALID_ARG, "pair-tiled operands: ld_ab must be >= sum_pad and a multiple of 8");
  }
  if (nt_status st = need_workspace(nt::triangle_workspace_bytes(*L, C, operands, dtype), workspace, workspace_bytes,
                                    "nt_triangle_mul_workspace"))
    return st;
  if (nt_status st = need_device(L)) return st;
  if (L->sum_n2 == 0) return NT_OK;
  if (!a || !b || !z) return nt::fail(NT_ERR_INVALID_ARG, "a, b and z must be non-NULL");
  if (!aligned16(a) || !aligned16(b) || !aligned16(z)) return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  return check_hip(nt::launch_triangle(*L, direction, C, a, b, ld_ab, operands, z, ld_z, dtype, workspace,
                                       static_cast<hipStream_t>(stream)),
                   "nt_triangle_mul launch");
}

nt_status nt_triangle_mul_gated(const nt_layout* L, int32_t direction, int32_t C, const void* a, const void* b,
                                int64_t ld_ab, nt_tri_operands operands, void* t, int64_t ld_t, nt_dtype dtype,
                                void* workspace, uint64_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (nt_status st = need_square(L, "the triangle update")) return st;
  if (direction != 0 && direction != 1) return nt::fail(NT_ERR_INVALID_ARG, "direction must be 0 or 1");
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (C <= 0) return nt::fail(NT_ERR_INVALID_ARG, "C must be > 0");
  if (dtype == NT_BF16 && C % 32) return nt::fail(NT_ERR_INVALID_ARG, "bf16 triangle needs C % 32 == 0");
  const int ve = vec_elems(dtype);
  if (C % ve) return nt::fail(NT_ERR_INVALID_ARG, "C must be a multiple of the vector width");
  if (operands != NT_TRI_PACKED && operands != NT_TRI_PAIR_TILED && operands != NT_TRI_PAIR_TILED_T)
    return nt::fail(NT_ERR_INVALID_ARG, "bad operand layout");
  if (ld_t < C || ld_t % ve) return nt::fail(NT_ERR_INVALID_ARG, "ld_t must be >= C and a multiple of the vector width");
  if (operands == NT_TRI_PACKED) {
    if (ld_ab < 2 * (int64_t)C || ld_ab % ve)
      return nt::fail(NT_ERR_INVALID_ARG, "packed gated operands: ld_ab must be >= 2C and a multiple of the vector width");
  } else {
    if ((operands == NT_TRI_PAIR_TILED) != (direction == 0))
      return nt::fail(NT_ERR_INVALID_ARG, "the pair-tiled operand variant does not match the direction");
    if (ld_ab < L->sum_pad || ld_ab % 8) return nt::fail(NT_ERR_INVALID_ARG, "pair-tiled operands: ld_ab must be >= sum_pad and a multiple of 8");
  }
  if (nt_status st = need_workspace(nt::triangle_workspace_bytes(*L, C, operands, dtype), workspace,
                                    workspace_bytes, "nt_triangle_mul_workspace"))
    return st;
  if (nt_status st = need_device(L)) return st;
  if (L->sum_n2 == 0) return NT_OK;
  if (!a || !b || !t) return nt::fail(NT_ERR_INVALID_ARG, "a, b and t must be non-NULL");
  if (!aligned16(a) || !aligned16(b) || !aligned16(t)) return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  return check_hip(nt::launch_triangle_gated(*L, direction, C, a, b, ld_ab, operands, t, ld_t, dtype, workspace,
                                             static_cast<hipStream_t>(stream)),
                   "nt_triangle_mul_gated launch");
}

nt_status nt_triangle_mul_backward(const nt_layout* L, int32_t direction, int32_t C, const void* a, const void* b,
                                   int64_t ld_ab, const void* dt, int64_t ld_dt, void* da, void* db, int64_t ld_dab,
                                   nt_dtype dtype, void* workspace, uint64_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!L) return nt::fail(NT_ERR_INVALID_ARG, "layout is NULL");
  if (nt_status st = need_square(L, "the triangle update")) return st;
  if (direction != 0 && direction != 1) return nt::fail(NT_ERR_INVALID_ARG, "direction must be 0 or 1");
  if (!valid_dtype(dtype)) return nt::fail(NT_ERR_INVALID_ARG, "bad dtype");
  if (C <= 0) return nt::fail(NT_ERR_INVALID_ARG, "C must be > 0");
  if (dtype == NT_BF16 && C % 32) return nt::fail(NT_ERR_INVALID_ARG, "bf16 triangle needs C % 32 == 0");
  const int ve = vec_elems(dtype);
  if (C % ve) return nt::fail(NT_ERR_INVALID_ARG, "C must be a multiple of the vector width");
  if (ld_ab < C || ld_ab % ve || ld_dt < C || ld_dt % ve || ld_dab < C || ld_dab % ve)
    return nt::fail(NT_ERR_INVALID_ARG, "row strides must be >= C and multiples of the vector width");
  if (nt_status st = need_workspace(nt::triangle_workspace_bytes(*L, C, NT_TRI_PACKED, dtype), workspace,
                                    workspace_bytes, "nt_triangle_mul_workspace"))
    return st;
  if (nt_status st = need_device(L)) return st;
  if (L->sum_n2 == 0 || (!da && !db)) return NT_OK;
  if (!dt || (da && !b) || (db && !a)) return nt::fail(NT_ERR_INVALID_ARG, "missing operand");
  if ((a && !aligned16(a)) || (b && !aligned16(b)) || !aligned16(dt) || (da && !aligned16(da)) || (db && !aligned16(db)))
    return nt::fail(NT_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
  return check_hip(nt::launch_triangle_backward(*L, direction, C, a, b, ld_ab, dt, ld_dt, da, db, ld_dab, dtype,
                                                workspace, static_cast<hipStream_t>(stream)),
                   "nt_triangle_mul_backward launch");
}

nt_status nt_triangle_mul_workspace(const nt_layout* L, int32_t C, nt_tri_operands operands, nt_dtype dtype,
                                    uint64_t* bytes) {
  g_last_error.clear();
  if (!L || !bytes) return nt::fail(NT_ERR_INVALID_ARG, "NULL argument");
  if (C <= 0 || !valid_dtype(dtype) || (operands != NT_TRI_PACKED && operands != NT_TRI_PAIR_TILED &&
                                       operands != NT_TRI_PAIR_TILED_T))
    return nt::fail(NT_ERR_INVALID_ARG, "bad C, dtype or operand layout");
  *bytes = nt::triangle_workspace_bytes(*L, C, operands, dtype);
  return NT_OK;
}

}  // extern "C"
