"""CPU oracle for prefix-cached paged attention -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import anything from this package.  The product path (the HIP library and its
Python binding) never calls it, and this package imports nothing from the
product package: it depends on numpy alone.

Contents
--------
``apc``        Prefix-cache bookkeeping written with a trie of Python dicts keyed by
               block token tuples: prefix-hit lookup, block allocation from a
               caller-ordered free list, block tables, slot mapping and varlen
               metadata (paper: Section 2 on PagedAttention's block-granular,
               virtual-memory-like KV layout and on Automatic Prefix Caching
               reusing the KV blocks of matching prefixes; Section 3, shared
               policy prefixes are not recomputed; Section 5.4).
``attention``  float64 causal softmax(q k^T / sqrt(D)) v over each request's
               logical token sequence, rebuilt from its block table, plus the
               oracle's own paged KV store (the same definition of the cache
               layout as the library documents, implemented independently).
``brute``      Pure-Python loops over tiny inputs, no numpy, used to pin the
               vectorised float64 code.

Every function is pinned by the CPU tests (``tests/test_oracle_*.py``) against
closed forms, brute force, a library routine (torch's
``scaled_dot_product_attention`` in float64) and invariants; none is "parity
unpinned".
"""
