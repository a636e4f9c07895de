// Host planner: splits one attention launch into work items.
//
// Rows of a sequence are its (query, head-in-group) pairs for one kv-head, so
// every row of an item reads the same keys and values (grouped-query
// attention).  Sequences with many rows (suffix prefill, prefill chunks) are
// cut into 128-row tile items, each a workgroup of four wavefronts sharing
// key/value tiles through LDS.  Sequences with at most 32 rows (decode: G
// rows; short verification: n_q * G rows) become single-wavefront row items
// whose key range is split so the launch has enough wavefronts in flight to
// stream the cache at HBM bandwidth; sequences with 33..64 rows run their
// split key ranges as tile items.  Split partial results are combined by
// log-sum-exp in a merge pass.
//
// Shared prefixes (cascade): few-row sequences whose block tables start
// with the same blocks read the same prefix keys (Section 2, Automatic Prefix
// Caching; Section 5.3, the same policy prefix across thousands of requests).
// Their attention over the shared keys is computed once, as 128-row MFMA tiles
// of all the group's query rows (every such query sees every shared key), and
// merged with each sequence's private-key part by log-sum-exp: the prefix is
// read from memory once per launch instead of once per sequence.
//
// Paper: Section 5.2 (split
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
#include <climits>
#include <cstdint>
#include <unordered_map>
#include <vector>

#include "internal.h"
#include "plan_format.h"

namespace {

constexpr int kXcds = 8;
constexpr int64_t kRowWavesPerCu = 16;      // row-item split target
constexpr int64_t kPrivateTileKeys = 2048;  // most private keys a few-row tile item covers

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
                            const int32_t* cu_seqlens_q, const int32_t* block_table,
                            int32_t max_blocks_per_seq, int32_t num_q_heads,
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
  if (block_table && max_blocks_per_seq < 1)
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: max_blocks_per_seq %d < 1", max_blocks_per_seq);
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
    if (block_table && cdiv(seq_lens[r], block_size) > max_blocks_per_seq)
      return pa::fail(PA_ERR_ARG, "pa_attn_plan: sequence %d needs more than %d blocks", r,
                      max_blocks_per_seq);
  }
  const int32_t total_q = n_seqs > 0 ? cu_seqlens_q[n_seqs] : 0;

  std::vector<std::array<int32_t, pa::kGroupWords>> groups;
  std::vector<int32_t> members;  // cascade member tables, (sequence, partial base) pairs
  int64_t partial_rows = 0;
  std::vector<Rec> shared, tiles;
  // Row-item workgroups in dispatch order, as (kv-head, index of the group's
  // first item in that head's longest-first order); records are written once,
  // straight into the plan.
  std::vector<std::pair<int32_t, int32_t>> quads;
  std::vector<std::vector<Rec>> head_rows;
  std::vector<std::vector<int32_t>> head_order;

  if (dtype == PA_BF16) {
    auto qlen = [&](int32_t r) { return cu_seqlens_q[r + 1] - cu_seqlens_q[r]; };
    // Sequences with few rows (decode, verification) get split key ranges and
    // may join a cascade group.  Their private keys run on one single-wave
    // row item per key range when it holds all their rows (at most 32), else
    // on tile items, whose four wavefronts share each key tile through LDS.
    auto is_row = [&](int32_t r) { return qlen(r) > 0 && qlen(r) * G <= pa::kRowSeqRows; };
    auto on_tiles = [&](int32_t r) { return qlen(r) * G > pa::kRowItemRows; };

    // Cascade groups: few-row sequences with the same first block and
    // q_len whose leading blocks coincide share those keys; attention over
    // them runs once for all the group's rows.
    std::vector<int32_t> kstart(n_seqs, 0);       // first private key
    std::vector<int32_t> cgroup(n_seqs, -1);      // cascade group of a sequence
    std::vector<std::vector<int32_t>> cg_members;
    std::vector<int32_t> cg_keys, cg_chunks;  // shared keys, key chunks (one merge part each)
    if (block_table) {
      std::unordered_map<int64_t, int32_t> by_key;
      std::vector<std::vector<int32_t>> cand;
      for (int32_t r = 0; r < n_seqs; ++r) {
        if (!is_row(r)) continue;
        const int64_t key = (int64_t(block_table[int64_t(r) * max_blocks_per_seq]) << 8) | qlen(r);
        auto it = by_key.find(key);
        if (it == by_key.end()) {
          by_key.emplace(key, int32_t(cand.size()));
          cand.push_back({r});
        } else {
          cand[it->second].push_back(r);
        }
      }
      for (auto& mem : cand) {
        if (mem.size() < 2) continue;
        const int32_t* b0 = block_table + int64_t(mem[0]) * max_blocks_per_seq;
        int64_t lcp = max_blocks_per_seq;
        int64_t limit = INT64_MAX;
        for (int32_t r : mem) {
          const int32_t* br = block_table + int64_t(r) * max_blocks_per_seq;
          const int64_t nb = std::min<int64_t>(lcp, cdiv(seq_lens[r], block_size));
          int64_t k = 0;
          while (k < nb && br[k] == b0[k]) ++k;
          lcp = k;
          limit = std::min<int64_t>(limit, seq_lens[r] - qlen(r));
        }
        int64_t S = std::min<int64_t>(lcp * block_size, limit);
        S = S / pa::kTileStep * pa::kTileStep;
        if (S < pa::kSharedMinKeys) continue;
        for (int32_t r : mem) {
          kstart[r] = int32_t(S);
          cgroup[r] = int32_t(cg_members.size());
        }
        cg_members.push_back(mem);
        cg_keys.push_back(int32_t(S));
        cg_chunks.push_back(int32_t(cdiv(S, pa::kSharedChunk)));
      }
    }

    // Key-range split of row items (private keys only for cascade members):
    // aim for enough single-wave items to keep kRowWavesPerCu wavefronts per
    // CU busy, never below 256 keys and never above 1024 keys per item.
    int64_t row_keys = 0;
    for (int32_t r = 0; r < n_seqs; ++r)
      if (is_row(r) && !on_tiles(r))
        row_keys += int64_t(seq_lens[r] - kstart[r]) * num_kv_heads;
    const int64_t target_waves = int64_t(num_cus) * kRowWavesPerCu;
    int64_t chunk = std::max<int64_t>(256, cdiv(row_keys, std::max<int64_t>(1, target_waves)));
    chunk = cdiv(chunk, pa::kKeyStep) * pa::kKeyStep;
    // a row item's block ids fit one wavefront (64 lanes): at most 1024 keys
    chunk = std::min<int64_t>(chunk, int64_t(pa::kRowItemBlocks) * block_size);

    std::vector<std::vector<Rec>> head_tiles(num_kv_heads);
    head_rows.assign(num_kv_heads, {});
    std::vector<std::vector<int64_t>> tile_cost(num_kv_heads), row_cost(num_kv_heads);
    // partial base of (cascade group member, kv-head): member_base[r * Hkv + g]
    std::vector<int32_t> member_base(cg_members.empty() ? 0 : size_t(n_seqs) * num_kv_heads, -1);
    {
      // exact per-head item counts, so the lists are allocated once
      int64_t nt = 0, nr = 0;
      for (int32_t r = 0; r < n_seqs; ++r) {
        if (qlen(r) == 0) continue;
        if (is_row(r) && on_tiles(r))
          nt += cdiv(seq_lens[r] - kstart[r], kPrivateTileKeys);
        else if (is_row(r))
          nr += std::max<int64_t>(1, cdiv(seq_lens[r] - kstart[r], chunk));
        else
          nt += cdiv(int64_t(qlen(r)) * G, pa::kTileRows);
      }
      for (int32_t g = 0; g < num_kv_heads; ++g) {
        head_tiles[g].reserve(nt);
        tile_cost[g].reserve(nt);
        head_rows[g].reserve(nr);
        row_cost[g].reserve(nr);
      }
      int64_t ng = 0;  // merge groups, one per kMergeRows rows of a few-row sequence
      for (int32_t r = 0; r < n_seqs; ++r)
        if (is_row(r)) ng += cdiv(qlen(r) * G, pa::kMergeRows);
      groups.reserve(size_t(ng) * num_kv_heads);
    }
    for (int32_t r = 0; r < n_seqs; ++r) {
      const int32_t n = qlen(r);
      const int32_t L = seq_lens[r];
      if (n == 0) continue;
      const int32_t rows = n * G;
      if (is_row(r)) {
        const int32_t k0s = kstart[r];
        const bool tiled = on_tiles(r);
        const int64_t split = tiled ? kPrivateTileKeys : chunk;
        const int64_t kstep = tiled ? pa::kTileStep : pa::kKeyStep;
        const int32_t nsplit = static_cast<int32_t>(std::max<int64_t>(1, cdiv(L - k0s, split)));
        // equal private key ranges, multiples of the key step, covering [k0s, L)
        const int64_t per = cdiv(cdiv(L - k0s, nsplit), kstep) * kstep;
        int32_t used = 0;
        while (used < nsplit && k0s + int64_t(used) * per < L) ++used;
        // parts 0 .. first-1 are the shared prefix's key chunks
        const int32_t first = cgroup[r] >= 0 ? cg_chunks[cgroup[r]] : 0;
        const int32_t parts = used + first;
        const int32_t nmerge = static_cast<int32_t>(cdiv(rows, pa::kMergeRows));
        for (int32_t g = 0; g < num_kv_heads; ++g) {
          int64_t base = -1;
          if (parts > 1) {
            base = partial_rows;
            partial_rows += int64_t(parts) * rows;
            for (int32_t gi = 0; gi < nmerge; ++gi) {
              const int32_t row0 = gi * pa::kMergeRows;
              const int32_t nr = std::min(pa::kMergeRows, rows - row0);
              groups.push_back({r, g, row0, nr, parts, int32_t(base + row0), rows, 0});
            }
            if (first) member_base[size_t(r) * num_kv_heads + g] = int32_t(base);
          }
          // per split, the row pieces back to back
          for (int32_t sp = 0; sp < used; ++sp) {
            const int64_t k0 = k0s + sp * per, k1 = std::min<int64_t>(L, k0s + (sp + 1) * per);
            if (tiled) {
              const int32_t part = base < 0 ? -1 : int32_t(base + int64_t(sp + first) * rows);
              head_tiles[g].push_back({r, g, 0, rows, int32_t(k0), int32_t(k1), part, 0});
              tile_cost[g].push_back((k1 - k0) * rows);
              continue;
            }
            const int32_t part = base < 0 ? -1 : int32_t(base + int64_t(sp + first) * rows);
            head_rows[g].push_back({r, g, 0, rows, int32_t(k0), int32_t(k1), part, 0});
            row_cost[g].push_back(k1 - k0);
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
    // Shared-prefix items: per cascade group and kv-head, a member table and
    // 128-row tiles of the gathered rows over key chunks of the shared keys.
    std::vector<std::vector<Rec>> head_shared(num_kv_heads);
    std::vector<std::vector<int64_t>> shared_cost(num_kv_heads);
    for (size_t cg = 0; cg < cg_members.size(); ++cg) {
      const auto& mem = cg_members[cg];
      const int32_t S = cg_keys[cg];
      const int32_t rpm = qlen(mem[0]) * G;
      const int64_t total_rows = int64_t(rpm) * mem.size();
      const int32_t nch = cg_chunks[cg];
      // chunk boundaries on the tile step; every chunk is non-empty because
      // S / nch >= kSharedChunk / 2 > kTileStep
      auto bound = [&](int64_t c) {
        return c >= nch ? int64_t(S) : (c * S / nch) / pa::kTileStep * pa::kTileStep;
      };
      for (int32_t g = 0; g < num_kv_heads; ++g) {
        for (int32_t ch = 0; ch < nch; ++ch) {
          const int64_t k0 = bound(ch), k1 = bound(ch + 1);
          // member table of this chunk: (sequence, partial row of its row 0)
          const int32_t off = int32_t(members.size());
          for (int32_t r : mem) {
            members.push_back(r);
            members.push_back(member_base[size_t(r) * num_kv_heads + g] + ch * rpm);
          }
          for (int64_t row0 = 0; row0 < total_rows; row0 += pa::kTileRows) {
            const int32_t nrows = int32_t(std::min<int64_t>(pa::kTileRows, total_rows - row0));
            head_shared[g].push_back({off, g, int32_t(row0), nrows, int32_t(k0), int32_t(k1), rpm,
                                      mem[0]});
            shared_cost[g].push_back((k1 - k0) * nrows);
          }
        }
      }
    }
    // Shared and tile items: per head, longest first, dealt round robin to the
    // head's XCD queues (which stay longest first).
    auto deal = [&](std::vector<std::vector<Rec>>& lists, std::vector<std::vector<int64_t>>& costs) {
      std::vector<std::vector<Rec>> q(kXcds);
      for (int32_t g = 0; g < num_kv_heads; ++g) {
        const auto xs = xcds_of_head(g, num_kv_heads);
        const auto ord = order_longest_first(costs[g]);
        for (size_t i = 0; i < ord.size(); ++i) q[xs[i % xs.size()]].push_back(lists[g][ord[i]]);
      }
      return q;
    };
    const auto shared_q = deal(head_shared, shared_cost);
    const auto tile_q = deal(head_tiles, tile_cost);
    // Row items: per head, longest first, four to a workgroup (padded with
    // empty items) so a workgroup's waves share one kv-head.
    std::vector<std::vector<std::pair<int32_t, int32_t>>> quad_q(kXcds);
    head_order.resize(num_kv_heads);
    for (int32_t g = 0; g < num_kv_heads; ++g) {
      const auto xs = xcds_of_head(g, num_kv_heads);
      head_order[g] = order_longest_first(row_cost[g]);
      const int32_t nq = int32_t(cdiv(int64_t(head_order[g].size()), 4));
      for (auto x : xs) quad_q[x].reserve(quad_q[x].size() + size_t(nq) / xs.size() + 1);
      for (int32_t q = 0; q < nq; ++q) quad_q[xs[q % xs.size()]].push_back({g, 4 * q});
    }
    shared = interleave(shared_q);
    tiles = interleave(tile_q);
    quads = interleave(quad_q);
  }

  const int64_t n_row = int64_t(quads.size()) * 4;
  const int64_t n_groups = int64_t(groups.size());
  const int64_t shared_off = pa::kHeaderWords;
  const int64_t tile_off = shared_off + int64_t(shared.size()) * pa::kSharedWords;
  const int64_t row_off = tile_off + int64_t(tiles.size()) * pa::kItemWords;
  const int64_t group_off = row_off + n_row * pa::kItemWords;
  const int64_t member_off = group_off + n_groups * pa::kGroupWords;
  const int64_t words = member_off + int64_t(members.size());
  const int64_t grid = dtype == PA_F32 ? int64_t(total_q) * num_q_heads
                                       : int64_t(shared.size() + tiles.size() + quads.size());
  if (words >= (int64_t{1} << 31) || grid >= (int64_t{1} << 31) || partial_rows >= (int64_t{1} << 31))
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: launch too large");

  info->kind = kind;
  info->n_q = n_q;
  info->n_shared_items = int32_t(shared.size());
  info->n_tile_items = int32_t(tiles.size());
  info->n_row_items = int32_t(n_row);
  info->n_groups = int32_t(n_groups);
  info->n_merge_rows = 0;
  for (auto& g : groups) info->n_merge_rows += g[pa::G_NROWS];
  info->grid = int32_t(grid);
  bool wide = false;
  for (const auto& rows : head_rows)
    for (const auto& it : rows) wide = wide || it[pa::I_NROWS] > 16;
  info->variant = dtype == PA_F32 ? 0 : (pa::kVariantBf16 | (wide ? pa::kVariantWideRows : 0));
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
  h[pa::H_N_SHARED] = int32_t(shared.size());
  h[pa::H_N_TILE] = int32_t(tiles.size());
  h[pa::H_N_ROW] = int32_t(n_row);
  h[pa::H_N_GROUPS] = int32_t(n_groups);
  h[pa::H_GRID] = int32_t(grid);
  h[pa::H_HQ] = num_q_heads;
  h[pa::H_HKV] = num_kv_heads;
  h[pa::H_D] = head_dim;
  h[pa::H_N_SEQS] = n_seqs;
  h[pa::H_TOTAL_Q] = total_q;
  h[pa::H_SHARED_OFF] = int32_t(shared_off);
  h[pa::H_TILE_OFF] = int32_t(tile_off);
  h[pa::H_ROW_OFF] = int32_t(row_off);
  h[pa::H_GROUP_OFF] = int32_t(group_off);
  h[pa::H_MEMBER_OFF] = int32_t(member_off);
  h[pa::H_PARTIAL_ROWS] = int32_t(partial_rows);
  int32_t* p = plan + shared_off;
  for (auto& it : shared) {
    Rec w = it;
    w[pa::S_MEMBERS] += int32_t(member_off);  // absolute word offset of the member table
    p = std::copy(w.begin(), w.end(), p);
  }
  for (auto& it : tiles) p = std::copy(it.begin(), it.end(), p);
  const Rec empty = {-1, 0, 0, 0, 0, 0, -1, 0};
  for (const auto& q : quads) {
    const auto& ord = head_order[q.first];
    for (int32_t k = 0; k < 4; ++k) {
      const size_t i = size_t(q.second) + k;
      const Rec& it = i < ord.size() ? head_rows[q.first][ord[i]] : empty;
      p = std::copy(it.begin(), it.end(), p);
    }
  }
  for (auto& g : groups) p = std::copy(g.begin(), g.end(), p);
  std::copy(members.begin(), members.end(), p);
  return PA_OK;
}
