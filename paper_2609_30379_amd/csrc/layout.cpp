// Layout planner: partitions and tile-to-sample work maps of a batch of square
// pair states (Sec. 3.1 "Structural metadata", Fig. "representation",
// Appendix A "Structural invariants"), built on the host from the per-sample
// lengths.  Pure C++: the same code is exercised by host-only layouts.
#include <algorithm>
#include <array>
#include <climits>
#include <numeric>

#include "nt_internal.h"

namespace nt {
namespace {

// Orders work items for launch so that the item at position p is executed by
// XCD p % 8 (MI355X dispatches workgroups of one launch round-robin over its
// 8 XCDs).  Items of one sample are kept on as few XCDs as possible, so
// per-sample operands (pair bias, triangle rows) are reused from one L2, and
// the summed cost per XCD is balanced.  Idle positions are filled with -1.
template <int W>
std::vector<int32_t> xcd_order(const std::vector<std::array<int32_t, W>>& items,
                               const std::vector<double>& cost, bool largest_first = true) {
  const size_t n = items.size();
  std::vector<size_t> idx(n);
  std::iota(idx.begin(), idx.end(), 0);
  // per-sample totals; items arrive grouped by sample (field 0)
  std::vector<double> sample_cost;
  for (size_t t = 0; t < n; ++t) {
    const int32_t s = items[t][0];
    if ((int32_t)sample_cost.size() <= s) sample_cost.resize(s + 1, 0.0);
    sample_cost[s] += cost[t];
  }
  std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) {
    const double ca = sample_cost[items[a][0]], cb = sample_cost[items[b][0]];
    if (ca != cb) return ca > cb;
    return items[a][0] < items[b][0];
  });
  double total = 0.0;
  for (double c : cost) total += c;
  const double quota = total / kXcds;
  std::array<std::vector<size_t>, kXcds> q;
  std::array<double, kXcds> load{};
  int x = 0;
  for (size_t t : idx) {
    if (x < kXcds - 1 && load[x] >= quota * (1.0 - 1e-12) && load[x] > 0.0) ++x;
    q[x].push_back(t);
    load[x] += cost[t];
  }
  size_t depth = 0;
  for (auto& v : q) {
    if (largest_first) std::stable_sort(v.begin(), v.end(), [&](size_t a, size_t b) { return cost[a] > cost[b]; });
    depth = std::max(depth, v.size());
  }
  std::vector<int32_t> out(depth * kXcds * W, -1);
  for (size_t k = 0; k < depth; ++k)
    for (int xx = 0; xx < kXcds; ++xx)
      if (k < q[xx].size()) {
        const auto& it = items[q[xx][k]];
        for (int f = 0; f < W; ++f) out[(k * kXcds + xx) * W + f] = it[f];
      }
  return out;
}

// Rectangular pairs (N_i x M_i; Eq. packing with p_i = N_i M_i): row offsets
// eta over N_i, column offsets kappa over M_i, cell (i, a, b) at
// o_i + a M_i + b, level-2 splits o_i + a M_i.  The square-only work maps
// (attention, triangle, pair-tiled operands) are left empty: calls that need
// them reject rectangular layouts.
nt_status plan_rect_layout(const int32_t* rows, const int32_t* cols, int32_t batch, nt_layout* L) {
  L->batch = batch;
  L->rect = true;
  L->lengths.assign(rows, rows + batch);
  L->cols.assign(cols, cols + batch);
  L->cu_seqlens.assign(batch + 1, 0);
  L->cu_cols.assign(batch + 1, 0);
  L->cu_pairs.assign(batch + 1, 0);
  L->cu_pad.assign(batch + 1, 0);
  int64_t sn = 0, sm = 0, cells = 0;
  int32_t mx = 0;
  for (int32_t i = 0; i < batch; ++i) {
    const int64_t n = rows[i], m = cols[i];
    if (n < 0 || m < 0) return fail(NT_ERR_INVALID_ARG, "negative length at sample " + std::to_string(i));
    sn += n;
    sm += m;
    cells += n * m;
    if (sn > INT32_MAX || sm > INT32_MAX || cells > INT32_MAX)
      return fail(NT_ERR_OVERFLOW, "packed pair extent exceeds int32 at sample " + std::to_string(i));
    L->cu_seqlens[i + 1] = (int32_t)sn;
    L->cu_cols[i + 1] = (int32_t)sm;
    L->cu_pairs[i + 1] = (int32_t)cells;
    mx = std::max<int32_t>(mx, (int32_t)std::max(n, m));
  }
  L->sum_n = sn;
  L->sum_m = sm;
  L->sum_n2 = cells;
  L->sum_n3 = 0;
  L->sum_pad = 0;
  L->max_len = mx;
  L->row_splits2.assign(sn + 1, 0);
  L->row_sample.assign(sn, 0);
  L->col_sample.assign(sm, 0);
  for (int32_t i = 0; i < batch; ++i) {
    for (int32_t a = 0; a < rows[i]; ++a) {
      const int64_t eta = (int64_t)L->cu_seqlens[i] + a;
      L->row_splits2[eta] = L->cu_pairs[i] + a * cols[i];
      L->row_sample[eta] = i;
    }
    for (int32_t b = 0; b < cols[i]; ++b) L->col_sample[L->cu_cols[i] + b] = i;
  }
  L->row_splits2[sn] = (int32_t)cells;
  return NT_OK;
}

}  // namespace

nt_status plan_layout(const int32_t* lengths, int32_t batch, nt_layout* L, const int32_t* cols) {
  if (!lengths) return fail(NT_ERR_INVALID_ARG, "lengths is NULL");
  if (batch < 1) return fail(NT_ERR_INVALID_ARG, "batch must be >= 1");
  if (cols) return plan_rect_layout(lengths, cols, batch, L);
  L->batch = batch;
  L->lengths.assign(lengths, lengths + batch);
  L->cu_seqlens.assign(batch + 1, 0);
  L->cu_pairs.assign(batch + 1, 0);
  L->cu_pad.assign(batch + 1, 0);
  int64_t sn = 0, sn2 = 0, sn3 = 0, spad = 0;
  int32_t mx = 0;
  for (int32_t i = 0; i < batch; ++i) {
    const int64_t n = lengths[i];
    if (n < 0) return fail(NT_ERR_INVALID_ARG, "negative length at sample " + std::to_string(i));
    sn += n;
    sn2 += n * n;
    sn3 += n * n * n;
    spad += ((n + 15) / 16 * 16) * ((n + 31) / 32 * 32);
    if (sn > INT32_MAX || sn2 > INT32_MAX || spad > INT32_MAX)
      return fail(NT_ERR_OVERFLOW, "packed pair extent exceeds int32 at sample " + std::to_string(i));
    L->cu_seqlens[i + 1] = (int32_t)sn;
    L->cu_pairs[i + 1] = (int32_t)sn2;
    L->cu_pad[i + 1] = (int32_t)spad;
    mx = std::max<int32_t>(mx, (int32_t)n);
  }
  L->sum_n = sn;
  L->sum_n2 = sn2;
  L->sum_n3 = sn3;
  L->sum_pad = spad;
  L->max_len = mx;

  // level-2 row splits: o_i + a N_i for every pair row, then the total
  L->row_splits2.assign(sn + 1, 0);
  L->row_sample.assign(sn, 0);
  for (int32_t i = 0; i < batch; ++i) {
    const int32_t n = lengths[i];
    for (int32_t a = 0; a < n; ++a) {
      const int64_t eta = (int64_t)L->cu_seqlens[i] + a;
      L->row_splits2[eta] = L->cu_pairs[i] + a * n;
      L->row_sample[eta] = i;
    }
  }
  L->row_splits2[sn] = (int32_t)sn2;
  // square pairs: the column partition is the row partition
  L->cols = L->lengths;
  L->cu_cols = L->cu_seqlens;
  L->col_sample = L->row_sample;
  L->sum_m = sn;

  // first pair row of every kLinRows-cell block of the pair tensor (row tiles
  // of the projections that write pair-tiled outputs)
  const int64_t nblk = (sn2 + kLinRows - 1) / kLinRows;
  L->blk_prow.assign(nblk, 0);
  for (int64_t b = 0, eta = 0; b < nblk; ++b) {
    const int64_t m = b * kLinRows;
    while (eta + 1 < sn && L->row_splits2[eta + 1] <= m) ++eta;
    L->blk_prow[b] = (int32_t)eta;
  }

  // broadcast sources of the projections: the rows are walked as tiles of
  // 16 cells of one pair row (ceil(N_i / 16) per pair row, the last one
  // masked); bc_cu_tiles[i] counts the tiles of the samples before i
  {
    L->bc_cu_tiles.assign(batch + 1, 0);
    int64_t t = 0;
    for (int32_t i = 0; i < batch; ++i) {
      t += (int64_t)lengths[i] * ((lengths[i] + 15) / 16);
      if (t > INT32_MAX) return fail(NT_ERR_OVERFLOW, "broadcast tile count exceeds int32 at sample " + std::to_string(i));
      L->bc_cu_tiles[i + 1] = (int32_t)t;
    }
  }

  // 16-query blocks of every sample (bias gradient of the pair attention)
  L->cu_qblk.assign(batch + 1, 0);
  for (int32_t i = 0; i < batch; ++i) L->cu_qblk[i + 1] = L->cu_qblk[i] + (lengths[i] + 15) / 16;

  // pair-row attention: one item per (sample, pair row), cost N_i^2
  {
    std::vector<std::array<int32_t, 2>> items;
    std::vector<double> cost;
    items.reserve(sn);
    for (int32_t i = 0; i < batch; ++i)
      for (int32_t r = 0; r < lengths[i]; ++r) {
        items.push_back({i, r});
        cost.push_back((double)lengths[i] * lengths[i]);
      }
    L->attn_work = xcd_order<2>(items, cost);
  }
  // pair attention: a sample's 16-query tiles are split evenly over
  // ceil(tiles / W) blocks of at most W tiles (items: sample, first tile, row
  // group, tile count), so no block leaves most of its waves idle; generation
  // order is kept in each XCD's queue so the blocks of a row group stay
  // adjacent and share keys and values.  For the 16-wave key-split instance
  // (N <= 512) W is 16 for samples up to 256 long (a wave per query tile) and
  // 8 for longer ones (a wave pair per query tile); the N <= 256 persistent
  // instance needs no list (its workgroups find their rows from the prefix
  // sums).
  auto pair_attn_items = [&](auto W_of) {
    std::vector<std::array<int32_t, 4>> items;
    std::vector<double> cost;
    for (int32_t i = 0; i < batch; ++i) {
      const int32_t n = lengths[i], tiles = (n + 15) / 16, W = W_of(n);
      const int32_t blocks = (tiles + W - 1) / W;
      for (int32_t rg = 0; rg * kAttnRG < n; ++rg)
        for (int32_t b = 0; b < blocks; ++b) {
          const int32_t t0 = b * tiles / blocks, t1 = (b + 1) * tiles / blocks;
          items.push_back({i, t0, rg, t1 - t0});
          cost.push_back((double)std::min(kAttnRG, n - rg * kAttnRG) * std::min(16 * (t1 - t0), n - 16 * t0) * n);
        }
    }
    return xcd_order<4>(items, cost, false);
  };
  L->pattn_work = pair_attn_items([](int32_t n) { return n <= kAttnShortLen ? 16 : 8; });
  // 1-D attention: the same even split of a sample's 16-query tiles over
  // blocks of at most kAttnQB queries, one item per block
  {
    std::vector<std::array<int32_t, 4>> items;
    std::vector<double> cost;
    for (int32_t i = 0; i < batch; ++i) {
      const int32_t n = lengths[i], tiles = (n + 15) / 16;
      const int32_t blocks = (tiles + kAttnQB / 16 - 1) / (kAttnQB / 16);
      for (int32_t b = 0; b < blocks; ++b) {
        const int32_t t0 = b * tiles / blocks, t1 = (b + 1) * tiles / blocks;
        items.push_back({i, t0, 0, t1 - t0});
        cost.push_back((double)std::min(16 * (t1 - t0), n - 16 * t0) * n);
      }
    }
    L->sattn_work = xcd_order<4>(items, cost, true);
  }
  // pair attention bias image: per sample, one 512-byte tile per (16-query
  // tile, 16-key tile) up to the 64-key padded length
  L->bias_tiles.assign(batch + 1, 0);
  for (int32_t i = 0; i < batch; ++i) {
    const int64_t n = lengths[i];
    const int64_t t = L->bias_tiles[i] + (n + 15) / 16 * ((n + 63) / 64 * 4);
    if (t > INT32_MAX) return fail(NT_ERR_OVERFLOW, "bias image extent exceeds int32 at sample " + std::to_string(i));
    L->bias_tiles[i + 1] = (int32_t)t;
  }
  // triangle: one item per (sample, 64x64 output tile), largest samples first,
  // a sample's tiles contiguous and each carrying the index of the sample's
  // first item (the launch walks (sample, channel line group, tile) in this
  // order, one cost-balanced stretch per XCD); the list is padded to a
  // multiple of 8 with idle items.
  {
    std::vector<int32_t> order(batch);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return lengths[a] > lengths[b]; });
    L->tri_work.clear();
    for (int32_t i : order) {
      const int32_t n = lengths[i], nt = (n + kTriTile - 1) / kTriTile;
      const int32_t first = (int32_t)(L->tri_work.size() / 4);
      // bands of two tile rows, walked column by column: eight consecutive
      // tiles (what an XCD holds at once, with the four channel blocks of a
      // z line) read two row blocks of a and four of b
      for (int32_t xb = 0; xb < nt; xb += 2)
        for (int32_t yt = 0; yt < nt; ++yt)
          for (int32_t xt = xb; xt < std::min(xb + 2, nt); ++xt) {
            L->tri_work.push_back(i);
            L->tri_work.push_back(xt);
            L->tri_work.push_back(yt);
            L->tri_work.push_back(first);
          }
    }
    while ((L->tri_work.size() / 4) % kXcds) L->tri_work.insert(L->tri_work.end(), {-1, -1, -1, -1});
    // XCD x takes the items [tri_split[x], tri_split[x + 1]) (times the channel
    // line groups of a call).  A tile costs its sample's 32-wide k-steps plus
    // about two for reading and writing its z block; the cuts balance that
    // cost, since equal item counts would leave the XCD with the largest
    // samples doing most of the work.
    const int64_t nitems = (int64_t)L->tri_work.size() / 4;
    std::vector<double> pre(nitems + 1, 0.0);
    for (int64_t e = 0; e < nitems; ++e) {
      const int32_t i = L->tri_work[4 * e];
      pre[e + 1] = pre[e] + (i < 0 ? 0.0 : (double)((lengths[i] + 31) / 32 + 2));
    }
    L->tri_split.assign(kXcds + 1, 0);
    int64_t e = 0;
    for (int x = 1; x < kXcds; ++x) {
      const double target = pre[nitems] * x / kXcds;
      while (e < nitems && pre[e + 1] <= target) ++e;
      // the cut nearest the target
      if (e < nitems && target - pre[e] > pre[e + 1] - target) ++e;
      L->tri_split[x] = (int32_t)e;
    }
    L->tri_split[kXcds] = (int32_t)nitems;
    int32_t widest = 0;
    for (int x = 0; x < kXcds; ++x) widest = std::max(widest, L->tri_split[x + 1] - L->tri_split[x]);
    L->tri_xcd_items = widest;
  }
  // 1-D attention: one item per (sample, block of kSeqQBlock queries), cost = queries * N_i
  {
    std::vector<std::array<int32_t, 2>> items;
    std::vector<double> cost;
    for (int32_t i = 0; i < batch; ++i) {
      const int32_t n = lengths[i];
      for (int32_t qb = 0; qb * kSeqQBlock < n; ++qb) {
        items.push_back({i, qb});
        cost.push_back((double)std::min(kSeqQBlock, n - qb * kSeqQBlock) * n);
      }
    }
    L->seq_work = xcd_order<2>(items, cost);
  }
  return NT_OK;
}

}  // namespace nt
