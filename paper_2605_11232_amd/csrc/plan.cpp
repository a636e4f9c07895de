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
// are combined by log-sum-exp in a merge pass.  Paper: Section 5.2 (split prefills under a batched-token budget, mixed
// prefill and decode), Section 6, Table "playbook" (long prefills blocking
// short decodes).
//
// Dispatch order: workgroup ids are handed to the eight XCDs round robin, and
// each XCD has its own L2.  Items are queued per XCD by kv-head so that all
// work of one kv-head -- and so the shared prefix blocks of that head, which
// every sequence reads -- stays in one XCD's L2.  Within a queue, items are
// ordered longest first to shorten the tail.
#include <algorithm>
#include <array>
#include <vector>

#include "internal.h"
#include "plan_format.h"

namespace {

constexpr int kXcds = 8;

struct Item {
  std::array<int32_t, pa::kItemWords> w;
  int64_t cost;
};

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

// Interleave per-XCD queues of units into dispatch order: unit slot b goes to
// queue b % kXcds while it has units, else to the longest remaining queue.
template <class U>
std::vector<U> interleave(std::vector<std::vector<U>>& queues) {
  std::vector<U> out;
  std::vector<size_t> pos(queues.size(), 0);
  size_t total = 0;
  for (auto& q : queues) total += q.size();
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

  std::vector<std::vector<Item>> tile_q(kXcds), row_q(kXcds);
  std::vector<std::array<int32_t, pa::kGroupWords>> groups;
  int64_t partial_rows = 0;
  int64_t n_tile = 0, n_row_real = 0;

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

    std::vector<std::vector<std::vector<Item>>> head_rows(num_kv_heads);
    std::vector<std::vector<Item>> head_tiles(num_kv_heads);
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
        for (int32_t g = 0; g < num_kv_heads; ++g) {
          // per split, the row groups back to back
          std::vector<Item> its;
          std::vector<int32_t> base;
          for (int32_t row0 = 0; row0 < rows; row0 += pa::kRowItemRows) {
            const int32_t nr = std::min(pa::kRowItemRows, rows - row0);
            base.push_back(used > 1 ? int32_t(partial_rows) : -1);
            if (used > 1) {
              groups.push_back({r, g, row0, nr, used, int32_t(partial_rows), 0, 0});
              partial_rows += int64_t(used) * nr;
            }
          }
          for (int32_t s = 0; s < used; ++s) {
            const int64_t k0 = s * per, k1 = std::min<int64_t>(L, (s + 1) * per);
            int32_t gi = 0;
            for (int32_t row0 = 0; row0 < rows; row0 += pa::kRowItemRows, ++gi) {
              const int32_t nr = std::min(pa::kRowItemRows, rows - row0);
              Item it{};
              it.w = {r, g, row0, nr, int32_t(k0), int32_t(k1),
                      base[gi] < 0 ? -1 : int32_t(base[gi] + int64_t(s) * nr), 0};
              it.cost = k1 - k0;
              its.push_back(it);
              ++n_row_real;
            }
          }
          head_rows[g].push_back(std::move(its));
        }
      } else {
        const int32_t ntiles = static_cast<int32_t>(cdiv(rows, pa::kTileRows));
        for (int32_t g = 0; g < num_kv_heads; ++g) {
          for (int32_t t = 0; t < ntiles; ++t) {
            const int32_t row0 = t * pa::kTileRows;
            const int32_t nrows = std::min(pa::kTileRows, rows - row0);
            const int32_t last_q = (row0 + nrows - 1) / G;
            const int32_t kv1 = L - n + last_q + 1;
            Item it{};
            it.w = {r, g, row0, nrows, 0, kv1, -1, 0};
            it.cost = int64_t(kv1) * nrows;
            head_tiles[g].push_back(it);
            ++n_tile;
          }
        }
      }
    }
    // Tile items: per-head lists, longest first, dealt to the head's XCD queues.
    for (int32_t g = 0; g < num_kv_heads; ++g) {
      auto& v = head_tiles[g];
      std::stable_sort(v.begin(), v.end(), [](const Item& a, const Item& b) { return a.cost > b.cost; });
      const auto xs = xcds_of_head(g, num_kv_heads);
      for (size_t i = 0; i < v.size(); ++i) tile_q[xs[i % xs.size()]].push_back(v[i]);
    }
    for (auto& q : tile_q)
      std::stable_sort(q.begin(), q.end(), [](const Item& a, const Item& b) { return a.cost > b.cost; });
    // Row items: per head, longest first, packed four to a workgroup (padded
    // with empty items) so a workgroup's waves share one kv-head.
    for (int32_t g = 0; g < num_kv_heads; ++g) {
      std::vector<Item> flat;
      for (auto& its : head_rows[g]) flat.insert(flat.end(), its.begin(), its.end());
      std::stable_sort(flat.begin(), flat.end(), [](const Item& a, const Item& b) { return a.cost > b.cost; });
      const auto xs = xcds_of_head(g, num_kv_heads);
      size_t quad = 0;
      for (size_t i = 0; i < flat.size(); i += 4, ++quad) {
        auto& q = row_q[xs[quad % xs.size()]];
        for (size_t k = 0; k < 4; ++k) {
          if (i + k < flat.size()) {
            q.push_back(flat[i + k]);
          } else {
            Item e{};
            e.w = {-1, 0, 0, 0, 0, 0, -1, 0};
            q.push_back(e);
          }
        }
      }
    }
  }

  // Flatten: tile items one per workgroup; row items as quads.
  std::vector<Item> tiles = interleave(tile_q);
  std::vector<std::array<Item, 4>> quads;
  {
    std::vector<std::vector<std::array<Item, 4>>> qq(kXcds);
    for (int x = 0; x < kXcds; ++x)
      for (size_t i = 0; i < row_q[x].size(); i += 4)
        qq[x].push_back({row_q[x][i], row_q[x][i + 1], row_q[x][i + 2], row_q[x][i + 3]});
    quads = interleave(qq);
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
  (void)n_tile;
  (void)n_row_real;

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
  for (auto& it : tiles) p = std::copy(it.w.begin(), it.w.end(), p);
  for (auto& q : quads)
    for (auto& it : q) p = std::copy(it.w.begin(), it.w.end(), p);
  for (auto& g : groups) p = std::copy(g.begin(), g.end(), p);
  return PA_OK;
}
