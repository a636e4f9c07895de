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
// Caching; Section 5.4, the same policy prefix across thousands of requests).
// Their attention over the shared keys is computed once, as 128-row MFMA tiles
// of all the group's query rows (every such query sees every shared key), and
// merged with each sequence's private-key part by log-sum-exp: the prefix is
// read from memory once per launch instead of once per sequence.
//
// Paper: Section 5.2 (split prefills under a batched-token budget, mixed
// prefill and decode), Section 6, Table "playbook" (long prefills blocking
// short decodes).
//
// Dispatch order: workgroup ids are handed to the eight XCDs round robin, and
// each XCD has its own L2.  Items are queued per XCD by kv-head so that all
// work of one kv-head -- and so the shared prefix blocks of that head, which
// every sequence reads -- stays in one XCD's L2.  Within a queue, shared and
// row items are ordered longest first (coarse counting sort) to shorten the
// tail, tile items grouped by sequence (each sequence's keys are re-read from
// L2 by its tiles running together).  The dispatch list is the queues
// interleaved segment by segment: shared items, then tile items with the row
// quads spread evenly among them.  The last full tiles in that order form a
// tail list that wildcard workgroups take at run time from whichever XCD
// gets to them first.
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
constexpr int64_t kRowWavesPerCu = 10;      // row-item split target
constexpr int64_t kPrivateTileKeys = 4160;  // most private keys a few-row tile item covers
constexpr int64_t kMinRowKeys = 256;        // split target floor of row items
constexpr int64_t kTailWorkPct = 10;        // row work given half-length items (per cent)
constexpr int64_t kStealPct = 5;            // tile work in the tail list (per cent)

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

// Tile items grouped by sequence: sequences by their total cost, longest
// first, and each sequence's items longest first.  The items of one sequence
// then run at about the same time on its kv-head's XCDs and share its keys
// in L2.
std::vector<int32_t> order_by_sequence(const std::vector<int64_t>& cost,
                                       const std::vector<std::array<int32_t, 8>>& items) {
  const size_t n = cost.size();
  std::unordered_map<int32_t, int64_t> total;
  for (size_t i = 0; i < n; ++i) total[items[i][0]] += cost[i];
  std::vector<int32_t> out(n);
  for (size_t i = 0; i < n; ++i) out[i] = static_cast<int32_t>(i);
  std::stable_sort(out.begin(), out.end(), [&](int32_t a, int32_t b) {
    const int32_t ra = items[a][0], rb = items[b][0];
    const int64_t ta = total[ra], tb = total[rb];
    if (ta != tb) return ta > tb;
    if (ra != rb) return ra < rb;
    return cost[a] > cost[b];
  });
  return out;
}

// Length of the common prefix of a[0, n) and b[0, n), compared sixteen
// entries at a time (the or-reduction vectorises).
int64_t common_prefix(const int32_t* a, const int32_t* b, int64_t n) {
  int64_t k = 0;
  for (; k + 16 <= n; k += 16) {
    int32_t d = 0;
    for (int i = 0; i < 16; ++i) d |= a[k + i] ^ b[k + i];
    if (d) break;
  }
  while (k < n && a[k] == b[k]) ++k;
  return k;
}

// Append per-XCD queues of units to dispatch list `out`: the unit at dispatch
// position b goes to queue b % kXcds (the XCD that runs workgroup b) while it
// has units, else to the longest remaining queue.
template <class U>
void interleave(std::vector<U>& out, const std::vector<std::vector<U>>& queues) {
  std::vector<size_t> pos(queues.size(), 0);
  size_t total = 0;
  for (auto& q : queues) total += q.size();
  out.reserve(out.size() + total);
  for (size_t b = 0, slot = out.size() % queues.size(); b < total;
       ++b, slot = slot + 1 == queues.size() ? 0 : slot + 1) {
    size_t q = slot;
    if (pos[q] >= queues[q].size()) {
      size_t best = q;
      size_t left = 0;
      for (size_t k = 0; k < queues.size(); ++k)
        if (queues[k].size() - pos[k] > left) left = queues[k].size() - pos[k], best = k;
      q = best;
    }
    out.push_back(queues[q][pos[q]++]);
  }
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

  // Items are generated once, as templates for kv-head 0: every kv-head has
  // the same items, with its own kvh and its own block of partial rows (head
  // g's partial rows are g * head_partial plus the template's).  Dispatch
  // lists hold (kv-head, template index) pairs; records are stamped when the
  // plan is written.
  using Grp = std::array<int32_t, pa::kGroupWords>;
  using Ref = std::pair<int32_t, int32_t>;
  std::vector<Rec> t_shared, t_tiles, t_rows;
  std::vector<Grp> t_groups;
  std::vector<int32_t> t_members;  // head 0's member tables: (sequence, partial base) pairs
  std::vector<Rec> sorted_rows;    // row templates, longest first, padded to whole quads
  int64_t head_partial = 0;
  // dispatch list: (kv-head, template index) per workgroup; template indices
  // run over the shared, tile and row templates in that order (a row
  // workgroup names the first of its four row templates)
  std::vector<Ref> dispatch;
  // per XCD queue, the tile items wildcard workgroups take at run time
  std::array<std::vector<Ref>, pa::kXcdQueues> tail;
  int64_t n_shared_wg = 0, n_tile_wg = 0, n_quads = 0;

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
    // them runs once for all the group's rows.  Candidates are found by
    // sorting (first block, q_len, sequence) keys.
    std::vector<int32_t> kstart(n_seqs, 0);   // first private key
    std::vector<int32_t> cgroup(n_seqs, -1);  // cascade group of a sequence
    std::vector<int32_t> cg_seqs;             // members of all groups, group by group
    std::vector<int32_t> cg_begin{0};         // group c's members start at cg_seqs[cg_begin[c]]
    std::vector<int32_t> cg_keys, cg_chunks;  // shared keys, key chunks (one merge part each)
    if (block_table) {
      std::vector<std::pair<int64_t, int32_t>> cand;
      cand.reserve(n_seqs);
      for (int32_t r = 0; r < n_seqs; ++r)
        if (is_row(r))
          cand.push_back({(int64_t(block_table[int64_t(r) * max_blocks_per_seq]) << 8) | qlen(r), r});
      std::sort(cand.begin(), cand.end());
      cg_seqs.reserve(cand.size());
      for (size_t i = 0, j = 0; i < cand.size(); i = j) {
        for (j = i + 1; j < cand.size() && cand[j].first == cand[i].first;) ++j;
        if (j - i < 2) continue;
        const int32_t* b0 = block_table + int64_t(cand[i].second) * max_blocks_per_seq;
        int64_t lcp = max_blocks_per_seq;
        int64_t limit = INT64_MAX;
        for (size_t m = i; m < j; ++m) {
          const int32_t r = cand[m].second;
          const int32_t* br = block_table + int64_t(r) * max_blocks_per_seq;
          const int64_t nb = std::min<int64_t>(lcp, cdiv(seq_lens[r], block_size));
          lcp = common_prefix(br, b0, nb);
          limit = std::min<int64_t>(limit, seq_lens[r] - qlen(r));
        }
        int64_t S = std::min<int64_t>(lcp * block_size, limit);
        S = S / pa::kTileStep * pa::kTileStep;
        if (S < pa::kSharedMinKeys) continue;
        for (size_t m = i; m < j; ++m) {
          const int32_t r = cand[m].second;
          kstart[r] = int32_t(S);
          cgroup[r] = int32_t(cg_keys.size());
          cg_seqs.push_back(r);
        }
        cg_begin.push_back(int32_t(cg_seqs.size()));
        cg_keys.push_back(int32_t(S));
        cg_chunks.push_back(int32_t(cdiv(S, pa::kSharedChunk)));
      }
    }

    // Key-range split of row items (private keys only for cascade members):
    // aim for enough single-wave items to keep kRowWavesPerCu wavefronts per
    // CU busy, a split target of at least kMinRowKeys and at most 1024 keys
    // per item (halved for the tail below).
    int64_t row_keys = 0;
    for (int32_t r = 0; r < n_seqs; ++r)
      if (is_row(r) && !on_tiles(r))
        row_keys += int64_t(seq_lens[r] - kstart[r]) * num_kv_heads;
    const int64_t target_waves = int64_t(num_cus) * kRowWavesPerCu;
    int64_t chunk = std::max<int64_t>(kMinRowKeys, cdiv(row_keys, std::max<int64_t>(1, target_waves)));
    chunk = cdiv(chunk, pa::kKeyStep) * pa::kKeyStep;
    // a row item's block ids fit one wavefront (64 lanes): at most 1024 keys
    chunk = std::min<int64_t>(chunk, int64_t(pa::kRowItemBlocks) * block_size);
    // The sequences with the fewest private keys, up to kTailWork of the row
    // work, get half-length items: ordered longest first, those run last, so
    // the launch drains sooner.  A sequence keeps at most cdiv(L, kMinRowKeys)
    // private parts (the workspace bound).
    std::vector<int64_t> row_chunk(n_seqs, chunk);
    if (row_keys > 0) {
      std::vector<std::pair<int64_t, int32_t>> by_len;
      for (int32_t r = 0; r < n_seqs; ++r)
        if (is_row(r) && !on_tiles(r)) by_len.push_back({int64_t(seq_lens[r] - kstart[r]), r});
      std::sort(by_len.begin(), by_len.end());
      const int64_t half = std::max<int64_t>(pa::kKeyStep, chunk / 2 / pa::kKeyStep * pa::kKeyStep);
      int64_t acc = 0;
      for (const auto& [len, r] : by_len) {
        acc += len * num_kv_heads;
        if (acc > row_keys * kTailWorkPct / 100) break;
        if (cdiv(len, half) <= cdiv(seq_lens[r], kMinRowKeys)) row_chunk[r] = half;
      }
    }

    std::vector<int64_t> tile_cost, row_cost, shared_cost;
    // head-0 partial base of a cascade member's merge group
    std::vector<int32_t> member_base(cg_keys.empty() ? 0 : size_t(n_seqs), -1);
    {
      // exact item counts, so the lists are allocated once
      int64_t nt = 0, nr = 0, ng = 0;
      for (int32_t r = 0; r < n_seqs; ++r) {
        if (qlen(r) == 0) continue;
        if (is_row(r)) ng += cdiv(qlen(r) * G, pa::kMergeRows);
        if (is_row(r) && on_tiles(r))
          nt += cdiv(seq_lens[r] - kstart[r], kPrivateTileKeys);
        else if (is_row(r))
          nr += std::max<int64_t>(1, cdiv(seq_lens[r] - kstart[r], row_chunk[r]));
        else
          nt += cdiv(int64_t(qlen(r)) * G, pa::kTileRows);
      }
      t_tiles.reserve(nt);
      tile_cost.reserve(nt);
      t_rows.reserve(nr);
      row_cost.reserve(nr);
      t_groups.reserve(ng);
    }
    for (int32_t r = 0; r < n_seqs; ++r) {
      const int32_t n = qlen(r);
      const int32_t L = seq_lens[r];
      if (n == 0) continue;
      const int32_t rows = n * G;
      if (is_row(r)) {
        const int32_t k0s = kstart[r];
        const bool tiled = on_tiles(r);
        const int64_t split = tiled ? kPrivateTileKeys : row_chunk[r];
        const int64_t kstep = tiled ? pa::kTileStep : pa::kKeyStep;
        const int32_t nsplit = static_cast<int32_t>(std::max<int64_t>(1, cdiv(L - k0s, split)));
        // equal private key ranges, multiples of the key step, covering [k0s, L)
        const int64_t per = cdiv(cdiv(L - k0s, nsplit), kstep) * kstep;
        int32_t used = 0;
        while (used < nsplit && k0s + int64_t(used) * per < L) ++used;
        // parts 0 .. first-1 are the shared prefix's key chunks
        const int32_t first = cgroup[r] >= 0 ? cg_chunks[cgroup[r]] : 0;
        const int32_t parts = used + first;
        int64_t base = -1;
        if (parts > 1) {
          base = head_partial;
          head_partial += int64_t(parts) * rows;
          for (int32_t row0 = 0; row0 < rows; row0 += pa::kMergeRows) {
            const int32_t nr = std::min(pa::kMergeRows, rows - row0);
            t_groups.push_back({r, 0, row0, nr, parts, int32_t(base + row0), rows, 0});
          }
          if (first) member_base[r] = int32_t(base);
        }
        // per split, the row pieces back to back
        for (int32_t sp = 0; sp < used; ++sp) {
          const int64_t k0 = k0s + sp * per, k1 = std::min<int64_t>(L, k0s + (sp + 1) * per);
          const int32_t part = base < 0 ? -1 : int32_t(base + int64_t(sp + first) * rows);
          if (tiled) {
            t_tiles.push_back({r, 0, 0, rows, int32_t(k0), int32_t(k1), part, pa::kItemStream});
            tile_cost.push_back((k1 - k0) * rows);
          } else {
            t_rows.push_back({r, 0, 0, rows, int32_t(k0), int32_t(k1), part, 0});
            row_cost.push_back(k1 - k0);
          }
        }
      } else {
        for (int32_t row0 = 0; row0 < rows; row0 += pa::kTileRows) {
          const int32_t nrows = std::min(pa::kTileRows, rows - row0);
          const int32_t last_q = (row0 + nrows - 1) / G;
          const int32_t kv1 = L - n + last_q + 1;
          t_tiles.push_back({r, 0, row0, nrows, 0, kv1, -1, 0});
          tile_cost.push_back(int64_t(kv1) * nrows);
        }
      }
    }
    // Shared-prefix items: per cascade group, a member table and 128-row
    // tiles of the gathered rows over key chunks of the shared keys.
    for (size_t cg = 0; cg < cg_keys.size(); ++cg) {
      const int32_t* mem = cg_seqs.data() + cg_begin[cg];
      const int32_t nmem = cg_begin[cg + 1] - cg_begin[cg];
      const int32_t S = cg_keys[cg];
      const int32_t rpm = qlen(mem[0]) * G;
      const int64_t total_rows = int64_t(rpm) * nmem;
      const int32_t nch = cg_chunks[cg];
      // chunk boundaries on the tile step; every chunk is non-empty because
      // S / nch >= kSharedChunk / 2 > kTileStep
      auto bound = [&](int64_t c) {
        return c >= nch ? int64_t(S) : (c * S / nch) / pa::kTileStep * pa::kTileStep;
      };
      for (int32_t ch = 0; ch < nch; ++ch) {
        const int64_t k0 = bound(ch), k1 = bound(ch + 1);
        // member table of this chunk: (sequence, partial row of its row 0)
        const int32_t off = int32_t(t_members.size());
        for (int32_t m = 0; m < nmem; ++m) {
          t_members.push_back(mem[m]);
          t_members.push_back(member_base[mem[m]] + ch * rpm);
        }
        for (int64_t row0 = 0; row0 < total_rows; row0 += pa::kTileRows) {
          const int32_t nrows = int32_t(std::min<int64_t>(pa::kTileRows, total_rows - row0));
          t_shared.push_back({off, 0, int32_t(row0), nrows, int32_t(k0), int32_t(k1), rpm, mem[0]});
          shared_cost.push_back((k1 - k0) * nrows);
        }
      }
    }
    // Shared and tile items: per head, in the order above, dealt round robin
    // to the head's XCD queues.
    std::vector<std::vector<int>> xs_of(num_kv_heads);
    for (int32_t g = 0; g < num_kv_heads; ++g) xs_of[g] = xcds_of_head(g, num_kv_heads);
    // With by_seq (tile items grouped by sequence), a head spread over
    // several XCDs gets each sequence's items on one XCD, the least loaded so
    // far, so the sequence's keys are fetched into one L2; a sequence costing
    // more than half an XCD's share is still dealt round robin.
    auto deal = [&](const std::vector<int64_t>& costs, const std::vector<Rec>* by_seq) {
      const auto ord = by_seq ? order_by_sequence(costs, *by_seq) : order_longest_first(costs);
      std::vector<std::vector<Ref>> q(kXcds);
      for (auto& x : q) x.reserve(ord.size() * num_kv_heads / kXcds + ord.size());
      int64_t total = 0;
      for (int64_t c : costs) total += c;
      std::array<int64_t, kXcds> load{};
      for (int32_t g = 0; g < num_kv_heads; ++g) {
        const auto& xs = xs_of[g];
        size_t x = 0;
        for (size_t i = 0; i < ord.size();) {
          size_t e = i + 1;  // the run of items of one sequence
          int64_t run = costs[ord[i]];
          if (by_seq && xs.size() > 1) {
            while (e < ord.size() && (*by_seq)[ord[e]][pa::I_SEQ] == (*by_seq)[ord[i]][pa::I_SEQ])
              run += costs[ord[e++]];
          }
          if (e - i > 1 && 2 * run * int64_t(xs.size()) <= total) {
            size_t best = 0;
            for (size_t k = 1; k < xs.size(); ++k)
              if (load[xs[k]] < load[xs[best]]) best = k;
            for (; i < e; ++i) q[xs[best]].push_back({g, ord[i]});
            load[xs[best]] += run;
          } else {
            for (; i < e; ++i, x = x + 1 == xs.size() ? 0 : x + 1) {
              q[xs[x]].push_back({g, ord[i]});
              load[xs[x]] += costs[ord[i]];
            }
          }
        }
      }
      return q;
    };
    auto shift = [](std::vector<std::vector<Ref>>& q, int32_t by) {
      for (auto& x : q)
        for (auto& r : x) r.second += by;
    };
    auto shared_q = deal(shared_cost, nullptr);
#ifndef PA_TILE_ORDER
#define PA_TILE_ORDER 1
#endif
    auto tile_q = deal(tile_cost, PA_TILE_ORDER ? &t_tiles : nullptr);
    shift(tile_q, int32_t(t_shared.size()));
    // Row items: per head, longest first, four to a workgroup (padded with
    // empty items) so a workgroup's waves share one kv-head.
    {
      const auto ord = order_longest_first(row_cost);
      sorted_rows.reserve(cdiv(int64_t(ord.size()), 4) * 4);
      for (int32_t i : ord) sorted_rows.push_back(t_rows[i]);
      while (sorted_rows.size() % 4) sorted_rows.push_back({-1, 0, 0, 0, 0, 0, -1, 0});
    }
    const int32_t nq = int32_t(sorted_rows.size() / 4);
    const int32_t row_base = int32_t(t_shared.size() + t_tiles.size());
    std::vector<std::vector<Ref>> quad_q(kXcds);
    for (auto& x : quad_q) x.reserve(size_t(nq) * num_kv_heads / kXcds + nq);
    for (int32_t g = 0; g < num_kv_heads; ++g) {
      const auto& xs = xs_of[g];
      for (size_t q = 0, x = 0; q < size_t(nq); ++q, x = x + 1 == xs.size() ? 0 : x + 1)
        quad_q[xs[x]].push_back({g, row_base + int32_t(4 * q)});
    }
    for (const auto& x : shared_q) n_shared_wg += int64_t(x.size());
    for (const auto& x : tile_q) n_tile_wg += int64_t(x.size());
    n_quads = int64_t(nq) * num_kv_heads;
    // Dispatch order: shared-prefix items first (the longest items, each a
    // cascade chunk over all its group's rows), then the tile items with the
    // row quads among them.
    {
      // Row quads (memory-bound) are spread evenly through each XCD's tile
      // items (matrix-bound) instead of following them, so a mixed launch
      // streams its decode rows while the tiles keep the matrix cores busy.
      std::vector<std::vector<Ref>> body(kXcds);
      for (int x = 0; x < kXcds; ++x) {
        const auto& t = tile_q[x];
        const auto& rq = quad_q[x];
        const size_t nt = t.size(), nr = rq.size();
        body[x].reserve(nt + nr);
        for (size_t it = 0, ir = 0; it < nt || ir < nr;) {
          // a quad goes next while the quads are not ahead of the tiles
          if (ir < nr && (it >= nt || ir * nt <= it * nr)) body[x].push_back(rq[ir++]);
          else body[x].push_back(t[it++]);
        }
      }
      dispatch.reserve(size_t(n_shared_wg + n_tile_wg + n_quads));
      interleave(dispatch, shared_q);
      interleave(dispatch, body);
    }
    // Tail stealing: the XCDs run at slightly different speeds (equal work
    // ends up to ~7 % apart), which no static order can know.  The last
    // plain full-tile items in dispatch order, kStealPct of the tile work,
    // move to the tail list of their XCD queue, in dispatch order, and their
    // dispatch slots become wildcards that take tail items until none is
    // left anywhere: XCDs that run ahead take over the others' last items.
    static_assert(pa::kXcdQueues == kXcds, "one tail list per XCD queue");
    if (kStealPct > 0) {
      const int32_t t_lo = int32_t(t_shared.size()), t_hi = t_lo + int32_t(t_tiles.size());
      auto stealable = [&](const Ref& r) {
        if (r.second < t_lo || r.second >= t_hi) return false;
        const Rec& t = t_tiles[r.second - t_lo];
        return t[pa::I_NROWS] > pa::kTileRows - 32 && t[pa::I_FLAGS] == 0;
      };
      int64_t total = 0;
      for (const auto& r : dispatch)
        if (stealable(r)) total += tile_cost[r.second - t_lo];
      const int64_t budget = total * kStealPct / 100;
      int64_t acc = 0;
      for (size_t b = dispatch.size(); b-- > 0 && acc < budget;) {
        if (!stealable(dispatch[b])) continue;
        acc += tile_cost[dispatch[b].second - t_lo];
        tail[b % kXcds].push_back(dispatch[b]);
        dispatch[b] = {0, pa::kWildcard};
      }
      // the walk ran backwards: each list back in dispatch order (a
      // sequence's tiles together, the longest sequences first)
      for (auto& l : tail) std::reverse(l.begin(), l.end());
    }
  }

  const int64_t partial_rows = head_partial * num_kv_heads;
  const int64_t n_row = n_quads * 4;
  const int64_t n_groups = int64_t(t_groups.size()) * num_kv_heads;
  const int64_t head_members = int64_t(t_members.size());
  const int64_t grid = dtype == PA_F32 ? int64_t(total_q) * num_q_heads
                                       : int64_t(dispatch.size());
  // layout: header, dispatch list, tail table and lists, counters,
  // templates (shared, tile, row, group), member table
  const int64_t dispatch_off = pa::kHeaderWords;
  int64_t n_tail = 0;
  for (const auto& l : tail) n_tail += int64_t(l.size());
  const int64_t tail_off = dispatch_off + (dtype == PA_F32 ? 0 : grid);
  const int64_t ctr_off = tail_off + (n_tail ? 2 * pa::kXcdQueues + n_tail : 0);
  const int64_t shared_off = ctr_off + (n_tail ? pa::kCounterBlockWords : 0);
  const int64_t tile_off = shared_off + int64_t(t_shared.size()) * pa::kSharedWords;
  const int64_t row_off = tile_off + int64_t(t_tiles.size()) * pa::kItemWords;
  const int64_t group_off = row_off + int64_t(sorted_rows.size()) * pa::kItemWords;
  const int64_t member_off = group_off + int64_t(t_groups.size()) * pa::kGroupWords;
  const int64_t words = member_off + head_members;
  if (dtype == PA_BF16 &&
      (num_kv_heads >= (1 << (31 - pa::kDispatchHeadShift)) ||
       t_shared.size() + t_tiles.size() + sorted_rows.size() >= size_t(pa::kWildcard)))
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: launch too large");
  if (words >= (int64_t{1} << 31) || grid >= (int64_t{1} << 31) || partial_rows >= (int64_t{1} << 31))
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: launch too large");

  info->kind = kind;
  info->n_q = n_q;
  info->n_shared_items = int32_t(n_shared_wg);
  info->n_tile_items = int32_t(n_tile_wg);
  info->n_row_items = int32_t(n_row);
  info->n_groups = int32_t(n_groups);
  info->n_merge_rows = 0;
  for (const auto& g : t_groups) info->n_merge_rows += int64_t(g[pa::G_NROWS]) * num_kv_heads;
  info->grid = int32_t(grid);
  bool wide = false;
  for (const auto& it : t_rows) wide = wide || it[pa::I_NROWS] > 16;
  info->variant = dtype == PA_F32 ? 0
                                  : (pa::kVariantBf16 | (wide ? pa::kVariantWideRows : 0) |
                                     (n_tail ? pa::kVariantTail : 0));
  info->plan_words = words;
  info->workspace_bytes = partial_rows * int64_t(head_dim + 1) * int64_t(sizeof(float));
  info->n_seqs = n_seqs;
  info->total_q = total_q;
  info->num_q_heads = num_q_heads;
  info->num_kv_heads = num_kv_heads;
  info->head_dim = head_dim;
  info->dtype = dtype;
  info->partial_rows = partial_rows;
  if (!plan) return PA_OK;
  if (plan_capacity < words)
    return pa::fail(PA_ERR_ARG, "pa_attn_plan: plan capacity %lld < %lld words",
                    (long long)plan_capacity, (long long)words);
  int32_t* h = plan;
  std::fill(h, h + pa::kHeaderWords, 0);
  h[pa::H_MAGIC] = pa::kPlanMagic;
  h[pa::H_KIND] = kind;
  h[pa::H_N_SHARED] = int32_t(n_shared_wg);
  h[pa::H_N_TILE] = int32_t(n_tile_wg);
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
  h[pa::H_DISPATCH_OFF] = int32_t(dispatch_off);
  h[pa::H_HEAD_PARTIAL] = int32_t(head_partial);
  h[pa::H_N_SHARED_TMPL] = int32_t(t_shared.size());
  h[pa::H_N_TILE_TMPL] = int32_t(t_tiles.size());
  h[pa::H_N_ROW_TMPL] = int32_t(sorted_rows.size());
  h[pa::H_N_GROUP_TMPL] = int32_t(t_groups.size());
  h[pa::H_TAIL_OFF] = int32_t(tail_off);
  h[pa::H_N_TAIL] = int32_t(n_tail);
  h[pa::H_N_WILD] = int32_t(n_tail);  // one wildcard per tail item
  h[pa::H_CTR_OFF] = int32_t(ctr_off);
  if (dtype == PA_BF16) {
    int32_t* p = plan + dispatch_off;
    auto word = [](const Ref& r) { return (r.first << pa::kDispatchHeadShift) | r.second; };
    for (const auto& r : dispatch) *p++ = word(r);
    if (n_tail) {
      // tail table (list offsets, then lengths), the lists, zeroed counters
      int32_t* tab = p;
      p += 2 * pa::kXcdQueues;
      for (int q = 0; q < pa::kXcdQueues; ++q) {
        tab[q] = int32_t(p - plan);
        tab[pa::kXcdQueues + q] = int32_t(tail[q].size());
        for (const auto& r : tail[q]) *p++ = word(r);
      }
      std::fill(p, p + pa::kCounterBlockWords, 0);
    }
    p = plan + shared_off;
    for (const auto& t : t_shared) {
      std::copy(t.begin(), t.end(), p);
      p[pa::S_MEMBERS] = int32_t(member_off + t[pa::S_MEMBERS]);  // absolute word offset
      p += pa::kSharedWords;
    }
    for (const auto& t : t_tiles) p = std::copy(t.begin(), t.end(), p);
    for (const auto& t : sorted_rows) p = std::copy(t.begin(), t.end(), p);
    for (const auto& t : t_groups) p = std::copy(t.begin(), t.end(), p);
    p = std::copy(t_members.begin(), t_members.end(), p);
  }
  return PA_OK;
}

// Workspace bound.  A sequence with split keys writes one partial row per
// (query row, part); its parts are its private key ranges (at least
// kMinRowKeys keys each, kPrivateTileKeys for tile-run private parts) plus
// its shared prefix's key chunks (at least kSharedChunk / 2 keys each, and
// never more than cdiv(shared keys, kSharedChunk)).  Both counts grow with
// the key count, so a sequence of at most L keys has at most
// cdiv(L, kMinRowKeys) + cdiv(L, kSharedChunk) parts (no shared chunk when
// L <= kSharedMinKeys), and a query token has num_q_heads rows.
namespace {
int workspace_bound(const char* fn, int32_t total_q, int32_t num_q_heads, int32_t head_dim,
                    int32_t max_seq_len, size_t* bytes) {
  pa::clear_error();
  if (!bytes || total_q < 0 || num_q_heads < 0 || max_seq_len < 0)
    return pa::fail(PA_ERR_ARG, "%s: NULL or negative argument", fn);
  if (head_dim != 64 && head_dim != 128)
    return pa::fail(PA_ERR_UNSUPPORTED, "%s: head_dim %d (supported: 64, 128)", fn, head_dim);
  // a shared prefix needs kSharedMinKeys keys and leaves at least one private key
  const int64_t shared_parts =
      max_seq_len > pa::kSharedMinKeys ? cdiv(max_seq_len, pa::kSharedChunk) : 0;
  const int64_t parts = cdiv(max_seq_len, kMinRowKeys) + shared_parts;
  // a sequence with a single part writes no partial rows
  const int64_t rows = parts > 1 ? int64_t(total_q) * num_q_heads * parts : 0;
  *bytes = size_t(rows) * size_t(head_dim + 1) * sizeof(float);
  return PA_OK;
}
}  // namespace

extern "C" int pa_attn_workspace_size(int32_t total_q, int32_t num_q_heads, int32_t head_dim,
                                      int32_t max_seq_len, size_t* bytes) {
  return workspace_bound("pa_attn_workspace_size", total_q, num_q_heads, head_dim, max_seq_len,
                         bytes);
}

extern "C" int pa_attn_decode_workspace_size(int32_t n_seqs, int32_t num_q_heads,
                                             int32_t head_dim, int32_t max_seq_len,
                                             size_t* bytes) {
  return workspace_bound("pa_attn_decode_workspace_size", n_seqs, num_q_heads, head_dim,
                         max_seq_len, bytes);
}
