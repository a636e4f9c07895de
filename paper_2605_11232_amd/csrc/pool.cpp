// Host block manager: prefix-hit lookup, block allocation, block tables and
// slot mapping for a paged KV cache whose leading blocks are shared prefixes.
//
// Paper: Section 2 (PagedAttention's block-granular KV layout addressed through
// a per-request block table; Automatic Prefix Caching reuses the KV blocks of
// matching prefixes), Section 3 (shared policy prefixes are not recomputed),
// Section 5.4 (prefixes identical across thousands of requests).
//
// A cached block is identified by (predecessor block, its block_size tokens).
// Because a block is cached only when its predecessor is cached, that pair
// stands for the whole token prefix up to the block, so a match on it is a
// match on the full prefix.  The hash only narrows candidates (open
// addressing, linear probing): every hit is confirmed by comparing the
// predecessor id and the stored tokens, so hash collisions cannot produce a
// false hit.
//
// Eviction (optional, least recently used): a cached block that no live
// sequence holds is idle.  Because a sequence holds every block of its own
// chain, the blocks continuing an idle block are idle too, so idle blocks
// without cached successors (leaves) can always be evicted first; each
// release stamps the blocks that became idle, tail first, and the leaf with
// the oldest stamp goes first.  An evicted block leaves the index before its
// id is reused, so (predecessor, tokens) keys never refer to stale content.
#include <algorithm>
#include <cstring>
#include <deque>
#include <new>
#include <set>
#include <unordered_map>
#include <vector>

#include "internal.h"

struct pa_pool {
  int32_t num_blocks = 0;
  int32_t bs = 0;
  std::deque<int32_t> free_list;
  std::vector<int32_t> ref;          // live sequences holding each block
  std::vector<uint8_t> cached;       // block is in the prefix index
  std::vector<int32_t> pred;         // cached block's predecessor (-1: first block)
  std::vector<int32_t> content;      // cached block's tokens, [num_blocks][bs]
  // Open-addressing index of cached blocks: slot_hash 0 = empty, otherwise the
  // (never zero) key hash; slot_block the cached block.  Capacity is a power
  // of two >= 2 * num_blocks, so the load factor stays <= 1/2.
  std::vector<uint64_t> slot_hash;
  std::vector<int32_t> slot_block;
  uint64_t slot_mask = 0;

  // eviction state
  bool evict = false;
  std::vector<int32_t> n_succ;     // cached blocks whose predecessor is this block
  std::vector<uint64_t> stamp;     // release stamp of an idle cached block
  uint64_t clock = 0;
  int64_t n_cached = 0, n_idle = 0, n_evicted = 0;
  std::set<std::pair<uint64_t, int32_t>> leaves;  // idle cached blocks without successors

  struct Seq {
    std::vector<int32_t> tokens;
    std::vector<int32_t> blocks;
    int32_t n_cached_run = 0;  // leading blocks of this sequence that are in the index
  };
  std::unordered_map<int64_t, Seq> seqs;

  static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

  uint64_t key_hash(int32_t p, const int32_t* t) const {
    // two tokens per 64-bit mixing round
    uint64_t h = 0x9E3779B97F4A7C15ull ^ static_cast<uint32_t>(p);
    int32_t i = 0;
    for (; i + 1 < bs; i += 2) {
      const uint64_t w = static_cast<uint32_t>(t[i]) | (uint64_t(static_cast<uint32_t>(t[i + 1])) << 32);
      h = (h ^ w) * 0xFF51AFD7ED558CCDull;
      h ^= h >> 32;
    }
    if (i < bs) h = ((h ^ static_cast<uint32_t>(t[i])) * 0xC4CEB9FE1A85EC53ull) ^ (h >> 29);
    h ^= h >> 29;
    return h | 1;  // never 0 (the empty-slot marker)
  }

  // Cached block whose predecessor is p and whose tokens are t[0..bs), or -1.
  int32_t find(int32_t p, const int32_t* t) const {
    const uint64_t h = key_hash(p, t);
    for (uint64_t i = h & slot_mask;; i = (i + 1) & slot_mask) {
      const uint64_t sh = slot_hash[i];
      if (sh == 0) return -1;
      if (sh != h) continue;
      const int32_t b = slot_block[i];
      if (pred[b] == p &&
          std::memcmp(&content[static_cast<size_t>(b) * bs], t, sizeof(int32_t) * bs) == 0)
        return b;
    }
  }

  void insert(uint64_t h, int32_t b) {
    uint64_t i = h & slot_mask;
    while (slot_hash[i] != 0) i = (i + 1) & slot_mask;
    slot_hash[i] = h;
    slot_block[i] = b;
  }

  // Remove cached block b from the index (backward-shift deletion keeps every
  // remaining key reachable from its home slot without tombstones).
  void erase(int32_t b) {
    const uint64_t h = key_hash(pred[b], &content[static_cast<size_t>(b) * bs]);
    uint64_t i = h & slot_mask;
    while (!(slot_hash[i] == h && slot_block[i] == b)) i = (i + 1) & slot_mask;
    for (uint64_t j = (i + 1) & slot_mask; slot_hash[j] != 0; j = (j + 1) & slot_mask) {
      const uint64_t home = slot_hash[j] & slot_mask;
      const bool movable = i <= j ? (home <= i || home > j) : (home <= i && home > j);
      if (movable) {
        slot_hash[i] = slot_hash[j];
        slot_block[i] = slot_block[j];
        i = j;
      }
    }
    slot_hash[i] = 0;
    slot_block[i] = -1;
  }

  // A cached block's holder count went 1 -> 0 (idle) or 0 -> 1 (reused).
  void make_idle(int32_t b) {
    stamp[b] = ++clock;
    ++n_idle;
    if (n_succ[b] == 0) leaves.insert({stamp[b], b});
  }
  void reuse(int32_t b) {
    --n_idle;
    leaves.erase({stamp[b], b});
  }

  // Blocks an allocation can obtain: the free list, plus idle cached blocks
  // other than `held_idle` ones about to be reused when eviction is on.
  int64_t obtainable(int64_t held_idle) const {
    return static_cast<int64_t>(free_list.size()) + (evict ? n_idle - held_idle : 0);
  }

  // Next block for an allocation: the free list's front, else the least
  // recently released idle leaf (callers check obtainable() first).
  int32_t take() {
    if (!free_list.empty()) {
      const int32_t b = free_list.front();
      free_list.pop_front();
      return b;
    }
    const auto it = leaves.begin();
    const int32_t b = it->second;
    leaves.erase(it);
    erase(b);
    cached[b] = 0;
    --n_cached;
    --n_idle;
    ++n_evicted;
    const int32_t p = pred[b];
    pred[b] = -1;
    if (p >= 0 && --n_succ[p] == 0 && cached[p] && ref[p] == 0) leaves.insert({stamp[p], p});
    return b;
  }

  // Cache the sequence's full blocks after its cached run, in logical order,
  // while the chain is unbroken and each prefix is new.
  void cache_run(Seq& s) {
    int32_t j = s.n_cached_run;
    const int64_t L = static_cast<int64_t>(s.tokens.size());
    while (static_cast<int64_t>(j + 1) * bs <= L) {
      const int32_t p = j ? s.blocks[j - 1] : -1;
      const int32_t* t = &s.tokens[static_cast<size_t>(j) * bs];
      if (find(p, t) >= 0) break;
      const int32_t b = s.blocks[j];
      cached[b] = 1;
      ++n_cached;
      pred[b] = p;
      if (p >= 0) ++n_succ[p];
      std::memcpy(&content[static_cast<size_t>(b) * bs], t, sizeof(int32_t) * bs);
      insert(key_hash(p, t), b);
      ++j;
    }
    s.n_cached_run = j;
  }
};

namespace pa {
int32_t pool_block_size(const pa_pool* pool) { return pool->bs; }
}  // namespace pa

extern "C" {

int pa_pool_create(int32_t num_blocks, int32_t block_size, const int32_t* free_order,
                   pa_pool** out) {
  pa::clear_error();
  if (!out || !free_order) return pa::fail(PA_ERR_ARG, "pa_pool_create: NULL argument");
  *out = nullptr;
  if (num_blocks <= 0 || block_size <= 0)
    return pa::fail(PA_ERR_ARG, "pa_pool_create: num_blocks %d and block_size %d must be positive",
                    num_blocks, block_size);
  if (static_cast<int64_t>(num_blocks) * block_size >= (int64_t{1} << 31))
    return pa::fail(PA_ERR_ARG, "pa_pool_create: num_blocks * block_size must be < 2^31");
  std::vector<uint8_t> seen(num_blocks, 0);
  for (int32_t i = 0; i < num_blocks; ++i) {
    const int32_t b = free_order[i];
    if (b < 0 || b >= num_blocks || seen[b])
      return pa::fail(PA_ERR_ARG, "pa_pool_create: free_order is not a permutation (entry %d = %d)",
                      i, b);
    seen[b] = 1;
  }
  pa_pool* p = new (std::nothrow) pa_pool();
  if (!p) return pa::fail(PA_ERR_ARG, "pa_pool_create: out of host memory");
  p->num_blocks = num_blocks;
  p->bs = block_size;
  p->free_list.assign(free_order, free_order + num_blocks);
  p->ref.assign(num_blocks, 0);
  p->cached.assign(num_blocks, 0);
  p->pred.assign(num_blocks, -1);
  p->content.assign(static_cast<size_t>(num_blocks) * block_size, 0);
  p->n_succ.assign(num_blocks, 0);
  p->stamp.assign(num_blocks, 0);
  uint64_t cap = 16;
  while (cap < 2 * static_cast<uint64_t>(num_blocks)) cap <<= 1;
  p->slot_hash.assign(cap, 0);
  p->slot_block.assign(cap, -1);
  p->slot_mask = cap - 1;
  *out = p;
  return PA_OK;
}

void pa_pool_destroy(pa_pool* pool) { delete pool; }

int pa_seq_add(pa_pool* pool, int64_t seq_id, const int32_t* tokens, int32_t n_tokens,
               int32_t* n_cached_out) {
  pa::clear_error();
  if (!pool || !tokens) return pa::fail(PA_ERR_ARG, "pa_seq_add: NULL argument");
  if (n_tokens < 1) return pa::fail(PA_ERR_ARG, "pa_seq_add: n_tokens %d < 1", n_tokens);
  if (pool->seqs.count(seq_id))
    return pa::fail(PA_ERR_ARG, "pa_seq_add: sequence %lld already exists", (long long)seq_id);
  const int32_t bs = pool->bs;
  std::vector<int32_t> hits;
  int32_t prev = -1;
  while (static_cast<int64_t>(hits.size() + 1) * bs <= n_tokens - 1) {
    const int32_t b = pool->find(prev, tokens + hits.size() * bs);
    if (b < 0) break;
    hits.push_back(b);
    prev = b;
  }
  const int64_t need = pa_pool::cdiv(n_tokens, bs) - static_cast<int64_t>(hits.size());
  int64_t idle_hits = 0;
  for (int32_t b : hits) idle_hits += pool->ref[b] == 0;
  if (need > pool->obtainable(idle_hits))
    return pa::fail(PA_ERR_NO_BLOCKS, "pa_seq_add: need %lld blocks, %lld obtainable",
                    (long long)need, (long long)pool->obtainable(idle_hits));
  pa_pool::Seq s;
  s.tokens.assign(tokens, tokens + n_tokens);
  s.blocks = hits;
  s.n_cached_run = static_cast<int32_t>(hits.size());
  for (int32_t b : hits)
    if (pool->ref[b]++ == 0) pool->reuse(b);
  for (int64_t i = 0; i < need; ++i) {
    const int32_t b = pool->take();
    pool->ref[b] = 1;
    s.blocks.push_back(b);
  }
  pool->cache_run(s);
  pool->seqs.emplace(seq_id, std::move(s));
  if (n_cached_out) *n_cached_out = static_cast<int32_t>(hits.size()) * bs;
  return PA_OK;
}

int pa_seq_extend(pa_pool* pool, int64_t seq_id, const int32_t* tokens, int32_t n_tokens) {
  pa::clear_error();
  if (!pool || (n_tokens > 0 && !tokens)) return pa::fail(PA_ERR_ARG, "pa_seq_extend: NULL argument");
  if (n_tokens < 0) return pa::fail(PA_ERR_ARG, "pa_seq_extend: n_tokens %d < 0", n_tokens);
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end())
    return pa::fail(PA_ERR_UNKNOWN_SEQ, "pa_seq_extend: unknown sequence %lld", (long long)seq_id);
  pa_pool::Seq& s = it->second;
  const int64_t new_len = static_cast<int64_t>(s.tokens.size()) + n_tokens;
  if (new_len >= (int64_t{1} << 31))
    return pa::fail(PA_ERR_ARG, "pa_seq_extend: sequence length overflows int32");
  const int64_t need = pa_pool::cdiv(new_len, pool->bs) - static_cast<int64_t>(s.blocks.size());
  if (need > pool->obtainable(0))
    return pa::fail(PA_ERR_NO_BLOCKS, "pa_seq_extend: need %lld blocks, %lld obtainable",
                    (long long)need, (long long)pool->obtainable(0));
  for (int64_t i = 0; i < need; ++i) {
    const int32_t b = pool->take();
    pool->ref[b] = 1;
    s.blocks.push_back(b);
  }
  s.tokens.insert(s.tokens.end(), tokens, tokens + n_tokens);
  return PA_OK;
}

int pa_seq_truncate(pa_pool* pool, int64_t seq_id, int32_t new_len) {
  pa::clear_error();
  if (!pool) return pa::fail(PA_ERR_ARG, "pa_seq_truncate: NULL pool");
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end())
    return pa::fail(PA_ERR_UNKNOWN_SEQ, "pa_seq_truncate: unknown sequence %lld", (long long)seq_id);
  pa_pool::Seq& s = it->second;
  const int64_t L = static_cast<int64_t>(s.tokens.size());
  const int64_t floor_len = static_cast<int64_t>(s.n_cached_run) * pool->bs;
  if (new_len < 1 || new_len > L || new_len < floor_len)
    return pa::fail(PA_ERR_ARG, "pa_seq_truncate: new_len %d outside [%lld, %lld]", new_len,
                    (long long)std::max<int64_t>(1, floor_len), (long long)L);
  const size_t keep = static_cast<size_t>(pa_pool::cdiv(new_len, pool->bs));
  for (size_t j = s.blocks.size(); j-- > keep;) {
    const int32_t b = s.blocks[j];
    --pool->ref[b];
    pool->free_list.push_front(b);
  }
  s.blocks.resize(keep);
  s.tokens.resize(static_cast<size_t>(new_len));
  return PA_OK;
}

int pa_seq_free(pa_pool* pool, int64_t seq_id) {
  pa::clear_error();
  if (!pool) return pa::fail(PA_ERR_ARG, "pa_seq_free: NULL pool");
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end())
    return pa::fail(PA_ERR_UNKNOWN_SEQ, "pa_seq_free: unknown sequence %lld", (long long)seq_id);
  pa_pool::Seq& s = it->second;
  pool->cache_run(s);
  for (int32_t b : s.blocks) {
    if (--pool->ref[b] == 0 && !pool->cached[b]) pool->free_list.push_back(b);
  }
  // blocks that became idle are stamped tail first
  for (size_t j = s.blocks.size(); j-- > 0;) {
    const int32_t b = s.blocks[j];
    if (pool->ref[b] == 0 && pool->cached[b]) pool->make_idle(b);
  }
  pool->seqs.erase(it);
  return PA_OK;
}

}  // extern "C"

namespace {
template <class F>
int batch(const char* fn, int32_t n, const int64_t* seq_ids, int32_t* n_done, F&& op) {
  if (n_done) *n_done = 0;
  if (n < 0 || (n > 0 && !seq_ids)) return pa::fail(PA_ERR_ARG, "%s: invalid batch", fn);
  for (int32_t i = 0; i < n; ++i) {
    const int rc = op(i);
    if (rc != PA_OK) return rc;
    if (n_done) *n_done = i + 1;
  }
  return PA_OK;
}

bool offsets_ok(int32_t n, const int32_t* off, const int32_t* tokens) {
  if (n == 0) return true;
  if (!off || off[0] != 0) return false;
  for (int32_t i = 0; i < n; ++i)
    if (off[i + 1] < off[i]) return false;
  return off[n] == 0 || tokens != nullptr;
}
}  // namespace

extern "C" {

int pa_seqs_add(pa_pool* pool, int32_t n, const int64_t* seq_ids, const int32_t* token_offsets,
                const int32_t* tokens, int32_t* n_cached_out, int32_t* n_done) {
  if (!offsets_ok(n, token_offsets, tokens))
    return pa::fail(PA_ERR_ARG, "pa_seqs_add: invalid token offsets");
  return batch("pa_seqs_add", n, seq_ids, n_done, [&](int32_t i) {
    return pa_seq_add(pool, seq_ids[i], tokens + token_offsets[i],
                      token_offsets[i + 1] - token_offsets[i],
                      n_cached_out ? n_cached_out + i : nullptr);
  });
}

int pa_seqs_extend(pa_pool* pool, int32_t n, const int64_t* seq_ids,
                   const int32_t* token_offsets, const int32_t* tokens, int32_t* n_done) {
  if (!offsets_ok(n, token_offsets, tokens))
    return pa::fail(PA_ERR_ARG, "pa_seqs_extend: invalid token offsets");
  return batch("pa_seqs_extend", n, seq_ids, n_done, [&](int32_t i) {
    return pa_seq_extend(pool, seq_ids[i], tokens + token_offsets[i],
                         token_offsets[i + 1] - token_offsets[i]);
  });
}

int pa_seqs_truncate(pa_pool* pool, int32_t n, const int64_t* seq_ids, const int32_t* new_lens,
                     int32_t* n_done) {
  if (n > 0 && !new_lens) return pa::fail(PA_ERR_ARG, "pa_seqs_truncate: NULL new_lens");
  return batch("pa_seqs_truncate", n, seq_ids, n_done,
               [&](int32_t i) { return pa_seq_truncate(pool, seq_ids[i], new_lens[i]); });
}

int pa_seqs_free(pa_pool* pool, int32_t n, const int64_t* seq_ids, int32_t* n_done) {
  return batch("pa_seqs_free", n, seq_ids, n_done,
               [&](int32_t i) { return pa_seq_free(pool, seq_ids[i]); });
}

int pa_pool_apply(pa_pool* pool, int32_t n, const int32_t* ops, const int64_t* seq_ids,
                  const int32_t* token_offsets, const int32_t* tokens, const int32_t* new_lens,
                  int32_t* n_cached_out, int32_t* n_done) {
  if (n > 0 && (!ops || !token_offsets))
    return pa::fail(PA_ERR_ARG, "pa_pool_apply: NULL ops or token offsets");
  if (!offsets_ok(n, token_offsets, tokens))
    return pa::fail(PA_ERR_ARG, "pa_pool_apply: invalid token offsets");
  return batch("pa_pool_apply", n, seq_ids, n_done, [&](int32_t i) {
    const int32_t* t = tokens ? tokens + token_offsets[i] : nullptr;
    const int32_t cnt = token_offsets[i + 1] - token_offsets[i];
    if (n_cached_out) n_cached_out[i] = 0;
    switch (ops[i]) {
      case PA_OP_ADD:
        return pa_seq_add(pool, seq_ids[i], t, cnt, n_cached_out ? n_cached_out + i : nullptr);
      case PA_OP_EXTEND:
        return pa_seq_extend(pool, seq_ids[i], t, cnt);
      case PA_OP_TRUNCATE:
        if (!new_lens) return pa::fail(PA_ERR_ARG, "pa_pool_apply: NULL new_lens");
        return pa_seq_truncate(pool, seq_ids[i], new_lens[i]);
      case PA_OP_FREE:
        return pa_seq_free(pool, seq_ids[i]);
      default:
        return pa::fail(PA_ERR_ARG, "pa_pool_apply: unknown operation %d", ops[i]);
    }
  });
}

int pa_seq_len(const pa_pool* pool, int64_t seq_id, int32_t* len_out) {
  pa::clear_error();
  if (!pool || !len_out) return pa::fail(PA_ERR_ARG, "pa_seq_len: NULL argument");
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end())
    return pa::fail(PA_ERR_UNKNOWN_SEQ, "pa_seq_len: unknown sequence %lld", (long long)seq_id);
  *len_out = static_cast<int32_t>(it->second.tokens.size());
  return PA_OK;
}

int pa_seq_blocks(const pa_pool* pool, int64_t seq_id, int32_t* out, int32_t capacity,
                  int32_t* n_out) {
  pa::clear_error();
  if (!pool || !n_out || (capacity > 0 && !out))
    return pa::fail(PA_ERR_ARG, "pa_seq_blocks: NULL argument");
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end())
    return pa::fail(PA_ERR_UNKNOWN_SEQ, "pa_seq_blocks: unknown sequence %lld", (long long)seq_id);
  const auto& b = it->second.blocks;
  *n_out = static_cast<int32_t>(b.size());
  if (static_cast<int64_t>(b.size()) > capacity)
    return pa::fail(PA_ERR_ARG, "pa_seq_blocks: capacity %d < %zu", capacity, b.size());
  std::copy(b.begin(), b.end(), out);
  return PA_OK;
}

int pa_pool_set_eviction(pa_pool* pool, int32_t enabled) {
  pa::clear_error();
  if (!pool) return pa::fail(PA_ERR_ARG, "pa_pool_set_eviction: NULL pool");
  pool->evict = enabled != 0;
  return PA_OK;
}

int pa_pool_get_stats(const pa_pool* pool, pa_pool_stats* out) {
  pa::clear_error();
  if (!pool || !out) return pa::fail(PA_ERR_ARG, "pa_pool_get_stats: NULL argument");
  pa_pool_stats st{};
  st.num_blocks = pool->num_blocks;
  st.free_blocks = static_cast<int64_t>(pool->free_list.size());
  st.cached_blocks = pool->n_cached;
  st.idle_cached_blocks = pool->n_idle;
  st.evictions = pool->n_evicted;
  st.live_seqs = static_cast<int64_t>(pool->seqs.size());
  for (const auto& kv : pool->seqs) {
    st.live_tokens += static_cast<int64_t>(kv.second.tokens.size());
    st.logical_blocks += static_cast<int64_t>(kv.second.blocks.size());
  }
  for (int32_t b = 0; b < pool->num_blocks; ++b) st.physical_blocks += pool->ref[b] > 0;
  *out = st;
  return PA_OK;
}

int pa_pool_kv_waste(const pa_pool* pool, int32_t max_seq_len, pa_kv_waste* out) {
  pa::clear_error();
  if (!pool || !out) return pa::fail(PA_ERR_ARG, "pa_pool_kv_waste: NULL argument");
  pa_pool_stats st;
  int rc = pa_pool_get_stats(pool, &st);
  if (rc) return rc;
  int64_t longest = 0;
  for (const auto& kv : pool->seqs)
    longest = std::max<int64_t>(longest, static_cast<int64_t>(kv.second.tokens.size()));
  if (max_seq_len < longest)
    return pa::fail(PA_ERR_ARG, "pa_pool_kv_waste: max_seq_len %d below the longest live sequence %lld",
                    max_seq_len, (long long)longest);
  pa_kv_waste w{};
  w.tokens = st.live_tokens;
  w.paged_slots = st.logical_blocks * pool->bs;
  w.physical_slots = st.physical_blocks * pool->bs;
  w.contiguous_slots = st.live_seqs * static_cast<int64_t>(max_seq_len);
  w.paged_waste = w.paged_slots ? 1.0 - double(w.tokens) / double(w.paged_slots) : 0.0;
  w.contiguous_waste =
      w.contiguous_slots ? 1.0 - double(w.tokens) / double(w.contiguous_slots) : 0.0;
  w.sharing_factor = w.physical_slots ? double(w.paged_slots) / double(w.physical_slots) : 1.0;
  *out = w;
  return PA_OK;
}

int pa_pool_free_list(const pa_pool* pool, int32_t* out, int32_t capacity, int32_t* n_out) {
  pa::clear_error();
  if (!pool || !n_out || (capacity > 0 && !out))
    return pa::fail(PA_ERR_ARG, "pa_pool_free_list: NULL argument");
  *n_out = static_cast<int32_t>(pool->free_list.size());
  if (static_cast<int64_t>(pool->free_list.size()) > capacity)
    return pa::fail(PA_ERR_ARG, "pa_pool_free_list: capacity %d < %zu", capacity,
                    pool->free_list.size());
  std::copy(pool->free_list.begin(), pool->free_list.end(), out);
  return PA_OK;
}

int pa_build_metadata(const pa_pool* pool, int32_t n_seqs, const int64_t* seq_ids,
                      const int32_t* q_lens, int32_t max_blocks_per_seq, int32_t* block_table,
                      int32_t* seq_lens, int32_t* cu_seqlens_q, int32_t* slot_mapping,
                      int64_t slot_capacity) {
  pa::clear_error();
  if (!pool || n_seqs < 0 || max_blocks_per_seq < 1 || !cu_seqlens_q ||
      (n_seqs > 0 && (!seq_ids || !q_lens || !block_table || !seq_lens)))
    return pa::fail(PA_ERR_ARG, "pa_build_metadata: NULL or invalid argument");
  const int32_t bs = pool->bs;
  // validate everything before writing anything
  std::vector<const pa_pool::Seq*> seqs(n_seqs);
  std::unordered_map<int64_t, int32_t> seen;
  int64_t total = 0;
  for (int32_t r = 0; r < n_seqs; ++r) {
    auto it = pool->seqs.find(seq_ids[r]);
    if (it == pool->seqs.end())
      return pa::fail(PA_ERR_UNKNOWN_SEQ, "pa_build_metadata: unknown sequence %lld",
                      (long long)seq_ids[r]);
    if (!seen.emplace(seq_ids[r], r).second)
      return pa::fail(PA_ERR_ARG, "pa_build_metadata: sequence %lld appears twice",
                      (long long)seq_ids[r]);
    const pa_pool::Seq& s = it->second;
    const int64_t L = static_cast<int64_t>(s.tokens.size());
    if (q_lens[r] < 0 || q_lens[r] > L)
      return pa::fail(PA_ERR_ARG, "pa_build_metadata: q_len %d outside [0, %lld] for row %d",
                      q_lens[r], (long long)L, r);
    if (static_cast<int64_t>(s.blocks.size()) > max_blocks_per_seq)
      return pa::fail(PA_ERR_ARG, "pa_build_metadata: sequence needs %zu blocks > max %d",
                      s.blocks.size(), max_blocks_per_seq);
    total += q_lens[r];
    seqs[r] = &s;
  }
  if (total >= (int64_t{1} << 31))
    return pa::fail(PA_ERR_ARG, "pa_build_metadata: total query tokens overflow int32");
  if (total > slot_capacity || (total > 0 && !slot_mapping))
    return pa::fail(PA_ERR_ARG, "pa_build_metadata: slot_capacity %lld < %lld",
                    (long long)slot_capacity, (long long)total);
  int64_t k = 0;
  cu_seqlens_q[0] = 0;
  for (int32_t r = 0; r < n_seqs; ++r) {
    const pa_pool::Seq& s = *seqs[r];
    const int32_t L = static_cast<int32_t>(s.tokens.size());
    int32_t* row = block_table + static_cast<int64_t>(r) * max_blocks_per_seq;
    std::fill(row, row + max_blocks_per_seq, -1);
    std::copy(s.blocks.begin(), s.blocks.end(), row);
    seq_lens[r] = L;
    cu_seqlens_q[r + 1] = cu_seqlens_q[r] + q_lens[r];
    for (int32_t t = L - q_lens[r]; t < L; ++t) slot_mapping[k++] = s.blocks[t / bs] * bs + t % bs;
  }
  return PA_OK;
}

}  // extern "C"
