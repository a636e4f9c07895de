// Adapter-first, length-bucketed batch forming for a request that carries
// prompts for several adapters of one base model (paper: Section 5.6,
// "Multi-Adapter and Length-Aware Batching"; Table "casec_adapter").  Each
// item is (adapter id, prompt length, original index); items are grouped by
// adapter, each adapter group is split into length buckets, every bucket is
// one batch, and results are restored to the original order.
//
// Readings where the paper leaves the choice open: adapter groups run in the
// order of their first item; buckets run from short to long; inside a bucket
// items keep their original order; bucket k holds the lengths below
// bounds[k] that no earlier bucket holds, the last bucket the rest.
#include <algorithm>
#include <unordered_map>
#include <vector>

#include "internal.h"

extern "C" int pa_form_batches(int32_t n, const int32_t* adapter_ids, const int32_t* prompt_lens,
                               int32_t n_bounds, const int32_t* bucket_bounds, int32_t* order,
                               int32_t* position, int32_t* batch_offsets, int32_t* batch_adapter,
                               int32_t* batch_bucket, int32_t* n_batches) {
  pa::clear_error();
  if (n < 0 || n_bounds < 0 || !n_batches || !batch_offsets ||
      (n > 0 && (!adapter_ids || !prompt_lens || !order || !position || !batch_adapter ||
                 !batch_bucket)) ||
      (n_bounds > 0 && !bucket_bounds))
    return pa::fail(PA_ERR_ARG, "pa_form_batches: NULL or negative argument");
  for (int32_t k = 1; k < n_bounds; ++k)
    if (bucket_bounds[k] <= bucket_bounds[k - 1])
      return pa::fail(PA_ERR_ARG, "pa_form_batches: bucket bounds must be strictly ascending");
  for (int32_t i = 0; i < n; ++i)
    if (prompt_lens[i] < 0)
      return pa::fail(PA_ERR_ARG, "pa_form_batches: prompt %d has negative length", i);

  // adapter group by first appearance, then (group, bucket) keys
  std::unordered_map<int32_t, int32_t> group_of;
  std::vector<int32_t> group_adapter;
  const int32_t nb = n_bounds + 1;
  std::vector<int64_t> key(n);
  for (int32_t i = 0; i < n; ++i) {
    auto it = group_of.find(adapter_ids[i]);
    int32_t g;
    if (it == group_of.end()) {
      g = static_cast<int32_t>(group_adapter.size());
      group_of.emplace(adapter_ids[i], g);
      group_adapter.push_back(adapter_ids[i]);
    } else {
      g = it->second;
    }
    const int32_t b = static_cast<int32_t>(
        std::upper_bound(bucket_bounds, bucket_bounds + n_bounds, prompt_lens[i]) - bucket_bounds);
    key[i] = int64_t(g) * nb + b;
  }
  // stable counting sort by key
  const int64_t nkeys = int64_t(group_adapter.size()) * nb;
  std::vector<int32_t> count(static_cast<size_t>(nkeys) + 1, 0);
  for (int32_t i = 0; i < n; ++i) ++count[static_cast<size_t>(key[i]) + 1];
  for (int64_t k = 0; k < nkeys; ++k) count[k + 1] += count[k];
  std::vector<int32_t> start(count.begin(), count.end() - 1);
  for (int32_t i = 0; i < n; ++i) order[start[static_cast<size_t>(key[i])]++] = i;
  for (int32_t p = 0; p < n; ++p) position[order[p]] = p;
  // batches = runs of equal key
  int32_t nbat = 0;
  batch_offsets[0] = 0;
  for (int32_t p = 0; p < n; ++p) {
    if (p > 0 && key[order[p]] == key[order[p - 1]]) continue;
    if (p > 0) batch_offsets[nbat] = p;
    const int64_t k = key[order[p]];
    batch_adapter[nbat] = group_adapter[static_cast<size_t>(k / nb)];
    batch_bucket[nbat] = static_cast<int32_t>(k % nb);
    ++nbat;
  }
  batch_offsets[nbat] = n;
  *n_batches = nbat;
  return PA_OK;
}
