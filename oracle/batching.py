"""Adapter-first, length-bucketed batch forming (test infrastructure only).

Follows the dispatch procedure of the paper's Section 5.6 ("Multi-Adapter and
Length-Aware Batching"): each prompt of a request is taken as (adapter id,
prompt length, original index); prompts are grouped by adapter, each adapter
group is sub-bucketed by length range, every bucket is executed as one batch,
and the results are put back into the original order.  Readings where the
paper leaves the choice open: adapter groups in order of first appearance,
buckets from short to long, original order inside a bucket, bucket k = the
lengths below bounds[k] that no earlier bucket takes (the last bucket takes
the rest).
"""
from __future__ import annotations


def bucket_of(length: int, bounds) -> int:
    for k, b in enumerate(bounds):
        if length < b:
            return k
    return len(bounds)


def form_batches(adapter_ids, prompt_lens, bounds):
    """Return (order, position, batches); batches = [(adapter, bucket, [indices])]."""
    bounds = list(bounds)
    if any(b1 <= b0 for b0, b1 in zip(bounds, bounds[1:])):
        raise ValueError("bucket bounds must be strictly ascending")
    groups = {}                      # adapter -> {bucket: [original indices]}
    for i, (a, ln) in enumerate(zip(adapter_ids, prompt_lens)):
        if ln < 0:
            raise ValueError("negative prompt length")
        groups.setdefault(a, {}).setdefault(bucket_of(ln, bounds), []).append(i)
    batches = []
    for a, buckets in groups.items():          # dicts keep first-appearance order
        for k in sorted(buckets):
            batches.append((a, k, buckets[k]))
    order = [i for _, _, idx in batches for i in idx]
    position = [0] * len(order)
    for p, i in enumerate(order):
        position[i] = p
    return order, position, batches
