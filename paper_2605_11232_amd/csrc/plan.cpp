// Host planner: splits one attention launch into work items.
//
// Rows of a sequence are its (query, head-in-group) pairs for one kv-head, so
// every row of an item reads the same keys and values (grouped-query
// attention).  Sequences with many rows (suffix prefill, prefill chunks) are
// cut into 128-row tile items, each a workgroup of four wavefronts sharing
// key/value tiles through LDS.  Sequences with at most 64 rows (decode: G rows;
// verification: n_q * G rows) become single-wavefront row items of up to 16
// rows whose key range is split so the launch has enough wavefronts in flight
// to stream the cache at HBM bandwidth; the row groups of one key range sit
// next to each other so their loads meet in cache, and split partial results
// are combined by log-sum-exp in a merge pass.  Paper: Section 5.2 (split
// prefills under a batched-token budget, mixed prefill and decode), Section 6,
// Table "playbook" (long prefills blocking short decodes).
//
// Dispatch order: workgroup ids are handed to the eight XCDs round robin, and
// each XCD has its own L2.  Items are queued per XCD by kv-head so that all
// work of one kv-head -- and so the shared prefix blocks of that head, which
// every sequence reads -- stays in one XCD's L2.  Within a queue, items are
// ordered longest first (coarse counting sort) to shorten the tail.
#include <algorithm>
#include <array>
#include <vector>

#include "internal.h"
#include "plan_format.h"

namespace {

constexpr int kXcds = 8;

using Rec = std::array<int32_t, pa::kItemWords>;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// XCD queues a kv-head's work goes to: with fewer heads than XCDs a head is
// spread over kXcds / Hkv queues.
std::vector<int> xcds_of_head(int g, int hkv) {
  std::vector<int> x;
  if (hkv >= kXcds) {
    x.push_back(g % kXcds);
  } else {
    for (int q = 0; q < kXcds; ++q)
      if (q % hkv == g) x.push_back(q);
    if (x.empty()) x.push_back(g % kXcds);
  }
  return x;
}

// Indices of `cost` ordered longest first by a stable counting sort on 256
// coarse buckets (relative to the largest cost): O(n), and equal-cost items
// keep their generation order (row groups of one key range stay adjacent).
std::vector<int32_t> order_longest_first(const std::vector<int64_t>& cost) {
  const size_t n = cost.size();
  std::vector<int32_t> out(n);
  if (n == 0) return out;
  int64_t mx = 1;
  for (int64_t c : cost) mx = std::max(mx, c);
  std::vector<int32_t> key(n);
  std::array<int32_t, 257> cnt{};
  for (size_t i = 0; i < n; ++i) {
    key[i] = 255 - static_cast<int32_t>((cost[i] * 255) / mx);  // 0 = longest
    ++cnt[key[i] + 1];
  }
  for (int b = 0; b < 256; ++b) cnt[b + 1] += cnt[b];
  for (size_t i = 0; i < n; ++i) out[cnt[key[i]]++] = static_cast<int32_t>(i);
  return out;
}

// Interleave per-XCD queues of units into dispatch order: unit slot b goes to
// queue b % kXcds while it has units, else to the longest remaining queue.
template <class U>
std::vector<U> interleave(const std::vector<std::vector<U>>& queues) {
  std::vector<U> out;
  std::vector<size_t> pos(queues.size(), 0);
  size_t total = 0;
  for (auto& q : queues) total += q.size();
  out.reserve(total);
  for (size_t b = 0; b < total; ++b) {
    size_t q = b % queues.size();
    if (pos[q] >= queues[q].size()) {
      size_t best = q;
      size_t left = 0;
      for (size_t k = 0; k < queues.size(); ++k)
        if (queues[k].size() - pos[k] > left) left = queues[k].size() - pos[k], best = k;
      q = best;
    }
    out.push_back(queues[q][pos[q]++]);
  }
  return out;
}

}  // namespace

extern "C" int pa_attn_plan(int32_t kind, int32_t n_q, int32_t n_seqs, const int32_t* seq_lens,
                            const int32_t* cu_seqlens_q, int32_t num_q_heads,
                            int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                            int32_t dtype, int32_t num_cus, int32_t* plan,
                            int64_t plan_capacity, pa_plan_info* info) {
  pa::clear_error();
  if (!info || n_seqs < 0 || (n_seqs > 0 && (!seq_lens || !cu_seqlens_q)))
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: NULL or invalid argument");
  if (kind < PA_KIND_PREFILL || kind > PA_KIND_VERIFY)
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: unknown kind %d", kind);
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads)
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: num_q_heads %d must be a positive multiple of "
                    "num_kv_heads %d", num_q_heads, num_kv_heads);
  if (head_dim != 64 && head_dim != 128)
    return pa::fail(PA_ERR_UNSUPPORTED, "pa_attn_plan: head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16)
    return pa::fail(PA_ERR_UNSUPPORTED, "pa_attn_plan: block_size %d (supported: 16)", block_size);
  if (dtype != PA_F32 && dtype != PA_BF16)
    return pa::fail(PA_ERR_UNSUPPORTED, "pa_attn_plan: dtype %d", dtype);
  if (kind == PA_KIND_DECODE) n_q = 1;
  if (kind == PA_KIND_VERIFY && (n_q < 1 || n_q > 8))
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: verify n_q %d outside [1, 8]", n_q);
  if (kind == PA_KIND_PREFILL) n_q = 0;
  if (num_cus <= 0) num_cus = 256;
  const int32_t G = num_q_heads / num_kv_heads;
  if (n_seqs > 0 && cu_seqlens_q[0] != 0)
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: cu_seqlens_q[0] must be 0");
  for (int32_t r = 0; r < n_seqs; ++r) {
    const int32_t n = cu_seqlens_q[r + 1] - cu_seqlens_q[r];
    if (n < 0 || n > seq_lens[r])
      return pa::fail(PA_ERR_ARG, "pa_attn_plan: sequence %d has q_len %d, seq_len %d", r, n,
                      seq_lens[r]);
    if (kind != PA_KIND_PREFILL && n != n_q)
      return pa::fail(PA_ERR_ARG, "pa_attn_plan: sequence %d has q_len %d, plan kind needs %d", r,
                      n, n_q);
  }
  const int32_t total_q = n_seqs > 0 ? cu_seqlens_q[n_seqs] : 0;

  std::vector<std::array<int32_t, pa::kGroupWords>> groups;
  int64_t partial_rows = 0;
  std::vector<Rec> tiles;
  std::vector<std::array<Rec, 4>> quads;

  if (dtype == PA_BF16) {
    // Key-range split of row items: aim for enough single-wave items to keep
    // ~16 wavefronts per CU busy, never below 256 keys per item.
    int64_t row_keys = 0;
    for (int32_t r = 0; r < n_seqs; ++r) {
      const int32_t n = cu_seqlens_q[r + 1] - cu_seqlens_q[r];
      if (n > 0 && n * G <= pa::kRowSeqRows)
        row_keys += int64_t(seq_lens[r]) * num_kv_heads * cdiv(n * G, pa::kRowItemRows);
    }
    const int64_t target_waves = int64_t(num_cus) * 16;
    int64_t chunk = std::max<int64_t>(256, cdiv(row_keys, std::max<int64_t>(1, target_waves)));
    chunk = cdiv(chunk, pa::kKeyStep) * pa::kKeyStep;

    std::vector<std::vector<Rec>> head_tiles(num_kv_heads), head_rows(num_kv_heads);
    std::vector<std::vector<int64_t>> tile_cost(num_kv_heads), row_cost(num_kv_heads);
    {
      // exact per-head item counts, so the lists are allocated once
      int64_t nt = 0, nr = 0;
      for (int32_t r = 0; r < n_seqs; ++r) {
        const int32_t n = cu_seqlens_q[r + 1] - cu_seqlens_q[r];
        if (n == 0) continue;
        if (n * G <= pa::kRowSeqRows)
          nr += cdiv(n * G, pa::kRowItemRows) * std::max<int64_t>(1, cdiv(seq_lens[r], chunk));
        else
          nt += cdiv(int64_t(n) * G, pa::kTileRows);
      }
      for (int32_t g = 0; g < num_kv_heads; ++g) {
        head_tiles[g].reserve(nt);
        tile_cost[g].reserve(nt);
        head_rows[g].reserve(nr);
        row_cost[g].reserve(nr);
      }
    }
    for (int32_t r = 0; r < n_seqs; ++r) {
      const int32_t n = cu_seqlens_q[r + 1] - cu_seqlens_q[r];
      const int32_t L = seq_lens[r];
      if (n == 0) continue;
      const int32_t rows = n * G;
      if (rows <= pa::kRowSeqRows) {
        const int32_t nsplit = static_cast<int32_t>(std::max<int64_t>(1, cdiv(L, chunk)));
        // equal key ranges, multiples of the key step, covering [0, L)
        const int64_t per = cdiv(cdiv(L, nsplit), pa::kKeyStep) * pa::kKeyStep;
        int32_t used = 0;
        while (used < nsplit && int64_t(used) * per < L) ++used;
        const int32_t ngroups = static_cast<int32_t>(cdiv(rows, pa::kRowItemRows));
        for (int32_t g = 0; g < num_kv_heads; ++g) {
          int64_t base[pa::kRowSeqRows / pa::kRowItemRows];
          for (int32_t gi = 0; gi < ngroups; ++gi) {
            const int32_t row0 = gi * pa::kRowItemRows;
            const int32_t nr = std::min(pa::kRowItemRows, rows - row0);
            base[gi] = used > 1 ? partial_rows : -1;
            if (used > 1) {
              groups.push_back({r, g, row0, nr, used, int32_t(partial_rows), 0, 0});
              partial_rows += int64_t(used) * nr;
            }
          }
          // per split, the row groups back to back
          for (int32_t sp = 0; sp < used; ++sp) {
            const int64_t k0 = sp * per, k1 = std::min<int64_t>(L, (sp + 1) * per);
            for (int32_t gi = 0; gi < ngroups; ++gi) {
              const int32_t row0 = gi * pa::kRowItemRows;
              const int32_t nr = std::min(pa::kRowItemRows, rows - row0);
              head_rows[g].push_back({r, g, row0, nr, int32_t(k0), int32_t(k1),
                                      base[gi] < 0 ? -1 : int32_t(base[gi] + int64_t(sp) * nr), 0});
              row_cost[g].push_back(k1 - k0);
            }
          }
        }
      } else {
        const int32_t ntiles = static_cast<int32_t>(cdiv(rows, pa::kTileRows));
        for (int32_t g = 0; g < num_kv_heads; ++g) {
          for (int32_t t = 0; t < ntiles; ++t) {
            const int32_t row0 = t * pa::kTileRows;
            const int32_t nrows = std::min(pa::kTileRows, rows - row0);
            const int32_t last_q = (row0 + nrows - 1) / G;
            const int32_t kv1 = L - n + last_q + 1;
            head_tiles[g].push_back({r, g, row0, nrows, 0, kv1, -1, 0});
            tile_cost[g].push_back(int64_t(kv1) * nrows);
          }
        }
      }
    }
    // Tile items: per head, longest first, dealt round robin to the head's
    // XCD queues (which stay longest first).
    std::vector<std::vector<Rec>> tile_q(kXcds);
    for (int32_t g = 0; g < num_kv_heads; ++g) {
      const auto xs = xcds_of_head(g, num_kv_heads);
      const auto ord = order_longest_first(tile_cost[g]);
      for (size_t i = 0; i < ord.size(); ++i) tile_q[xs[i % xs.size()]].push_back(head_tiles[g][ord[i]]);
    }
    tiles = interleave(tile_q);
    // Row items: per head, longest first, four to a workgroup (padded with
    // empty items) so a workgroup's waves share one kv-head.
    std::vector<std::vector<std::array<Rec, 4>>> quad_q(kXcds);
    const Rec empty = {-1, 0, 0, 0, 0, 0, -1, 0};
    for (int32_t g = 0; g < num_kv_heads; ++g) {
      const auto xs = xcds_of_head(g, num_kv_heads);
      const auto ord = order_longest_first(row_cost[g]);
      size_t quad = 0;
      for (size_t i = 0; i < ord.size(); i += 4, ++quad) {
        std::array<Rec, 4> qd;
        for (size_t k = 0; k < 4; ++k) qd[k] = i + k < ord.size() ? head_rows[g][ord[i + k]] : empty;
        quad_q[xs[quad % xs.size()]].push_back(qd);
      }
    }
    quads = interleave(quad_q);
  }

  const int64_t n_row = int64_t(quads.size()) * 4;
  const int64_t n_groups = int64_t(groups.size());
  const int64_t tile_off = pa::kHeaderWords;
  const int64_t row_off = tile_off + int64_t(tiles.size()) * pa::kItemWords;
  const int64_t group_off = row_off + n_row * pa::kItemWords;
  const int64_t words = group_off + n_groups * pa::kGroupWords;
  const int64_t grid = dtype == PA_F32 ? int64_t(total_q) * num_q_heads
                                       : int64_t(tiles.size()) + int64_t(quads.size());
  if (words >= (int64_t{1} << 31) || grid >= (int64_t{1} << 31) || partial_rows >= (int64_t{1} << 31))
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: launch too large");

  info->kind = kind;
  info->n_q = n_q;
  info->n_tile_items = int32_t(tiles.size());
  info->n_row_items = int32_t(n_row);
  info->n_groups = int32_t(n_groups);
  info->n_merge_rows = 0;
  for (auto& g : groups) info->n_merge_rows += g[pa::G_NROWS];
  info->grid = int32_t(grid);
  info->variant = dtype == PA_F32 ? 0 : 1;
  info->plan_words = words;
  info->workspace_bytes = partial_rows * int64_t(head_dim + 1) * int64_t(sizeof(float));
  if (!plan) return PA_OK;
  if (plan_capacity < words)
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: plan capacity %lld < %lld words",
                    (long long)plan_capacity, (long long)words);
  int32_t* h = plan;
  std::fill(h, h + pa::kHeaderWords, 0);
  h[pa::H_MAGIC] = pa::kPlanMagic;
  h[pa::H_KIND] = kind;
  h[pa::H_N_TILE] = int32_t(tiles.size());
  h[pa::H_N_ROW] = int32_t(n_row);
  h[pa::H_N_GROUPS] = int32_t(n_groups);
  h[pa::H_GRID] = int32_t(grid);
  h[pa::H_HQ] = num_q_heads;
  h[pa::H_HKV] = num_kv_heads;
  h[pa::H_D] = head_dim;
  h[pa::H_N_SEQS] = n_seqs;
  h[pa::H_TOTAL_Q] = total_q;
  h[pa::H_TILE_OFF] = int32_t(tile_off);
  h[pa::H_ROW_OFF] = int32_t(row_off);
  h[pa::H_GROUP_OFF] = int32_t(group_off);
  h[pa::H_PARTIAL_ROWS] = int32_t(partial_rows);
  int32_t* p = plan + tile_off;
  for (auto& it : tiles) p = std::copy(it.begin(), it.end(), p);
  for (auto& q : quads)
    for (auto& it : q) p = std::copy(it.begin(), it.end(), p);
  for (auto& g : groups) p = std::copy(g.begin(), g.end(), p);
  return PA_OK;
}
