/*
 * pa.h -- C ABI of libpa: prefix-cached paged attention for AMD MI355X (gfx950).
 *
 * The library serves requests whose prompts share long, identical prefixes
 * (policy text, taxonomies, output schemas) followed by short per-case
 * evidence and a short structured output (paper: Introduction; Section 3,
 * workload phenotypes).  KV memory is held in fixed-size blocks addressed
 * through a per-request block table (Section 2, PagedAttention), and blocks
 * holding a matching prefix are reused instead of recomputed (Section 2,
 * Automatic Prefix Caching; Section 3: shared policy prefixes should not be
 * recomputed; Section 5.4).  Attention runs for suffix prefill (per-case
 * evidence against the cached prefix plus its own causal context), decode,
 * and speculative verification of draft tokens (Section 2 and Section 5.3,
 * EAGLE-style speculative decoding), including chunked-prefill chunks mixed
 * with decode tokens in one launch (Section 5.2: split prefills under a
 * batched-token budget; Section 6, Table "playbook": long prefills blocking
 * short decodes).
 *
 * Conventions
 *  - Every function returns a pa_status (0 on success, negative on error);
 *    pa_last_error() returns a message for the calling thread's last error.
 *  - Host functions take host pointers.  Device functions take device
 *    pointers owned by the caller and enqueue work on the caller's
 *    hipStream_t (passed as void*; NULL = the default stream) without
 *    synchronising.  The library allocates no device memory.
 *  - Arguments are checked on the host before anything is launched; a failed
 *    check launches nothing.  Pool operations that fail leave the pool
 *    unchanged.
 *  - Cache layout (both tensors contiguous, element type = dtype):
 *      k_cache[num_blocks][num_kv_heads][head_dim/32][block_size][32]
 *      v_cache[num_blocks][num_kv_heads][head_dim][block_size]
 *    A token's slot is block * block_size + offset.  Key dim d of the token
 *    at offset o is k_cache[block][h][d/32][pos(o)][d%32], where pos(o) is o
 *    with bits 2 and 3 swapped: each 32-dim group of a block is 1 KB (bf16,
 *    head_dim 128) that attention reads contiguously, eight keys of a decode
 *    tile at a time.  Values are transposed per block so that the PV product
 *    reads keys contiguously.
 *  - Query/output layout: q[total_q][num_q_heads][head_dim] packed by
 *    sequence (sequence r owns rows cu_seqlens_q[r] .. cu_seqlens_q[r+1]-1,
 *    which are its LAST q_len positions); out has q's layout and dtype;
 *    lse[total_q][num_q_heads] is float32 natural-log log-sum-exp of the
 *    scaled scores, or NULL.
 *  - Query head h reads kv-head h / (num_q_heads / num_kv_heads).
 *  - A query at logical position a sees keys 0..a (causal, bottom-right).
 *  - Supported: block_size 16, head_dim 64 or 128, num_q_heads a multiple of
 *    num_kv_heads; dtype PA_BF16 (MFMA path, float32 accumulation) or PA_F32
 *    (float32 VALU path).  Integers are int32; num_blocks * block_size must
 *    be below 2^31.
 *  - Not thread-safe per pool; device calls on one stream are ordered.
 */
#ifndef PA_H_
#define PA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PA_OK = 0,
  PA_ERR_ARG = -1,          /* invalid argument / inconsistent sizes            */
  PA_ERR_UNSUPPORTED = -2,  /* valid but not implemented (head_dim, dtype, ...) */
  PA_ERR_NO_BLOCKS = -3,    /* the free list cannot satisfy an allocation       */
  PA_ERR_UNKNOWN_SEQ = -4,  /* no live sequence with that id                    */
  PA_ERR_LAUNCH = -5        /* the HIP runtime rejected a launch                */
} pa_status;

typedef enum { PA_F32 = 0, PA_BF16 = 1 } pa_dtype;

/* Message describing the calling thread's most recent error ("" if none). */
const char* pa_last_error(void);
/* ABI version of this header (increments on incompatible changes). */
int32_t pa_abi_version(void);

/* ------------------------------------------------------------------------ *
 * Host block manager: prefix-hit lookup, block allocation, block tables,    *
 * slot mapping (paper: Section 2, PagedAttention block tables and APC).     *
 * ------------------------------------------------------------------------ */

typedef struct pa_pool pa_pool; /* opaque, host memory owned by the library */

/* Create a pool of num_blocks blocks of block_size tokens.  free_order is a
 * permutation of 0..num_blocks-1 giving the order in which blocks are handed
 * out (copied; the caller keeps ownership).  *out receives the pool. */
int pa_pool_create(int32_t num_blocks, int32_t block_size, const int32_t* free_order,
                   pa_pool** out);
void pa_pool_destroy(pa_pool* pool);

/* Admit sequence seq_id with its n_tokens prompt tokens.  Full blocks are
 * matched against cached blocks from the start: block j is reused when the
 * whole token prefix up to and including it equals a cached one; the walk
 * stops at the first miss and never covers the last token (at most
 * (n_tokens-1)/block_size blocks are reused).  The remaining blocks are taken
 * from the front of the free list; the prompt's full blocks are then cached
 * (each only if the block before it is cached and its prefix is new).
 * *n_cached_out (may be NULL) receives the number of reused tokens.
 * Errors: PA_ERR_ARG (duplicate id, n_tokens < 1, NULL tokens),
 * PA_ERR_NO_BLOCKS (pool unchanged). */
int pa_seq_add(pa_pool* pool, int64_t seq_id, const int32_t* tokens, int32_t n_tokens,
               int32_t* n_cached_out);

/* Append n_tokens tokens (decode, draft or later prefill-chunk tokens).  New
 * blocks come from the front of the free list; nothing is cached until the
 * sequence is freed.  Errors: PA_ERR_UNKNOWN_SEQ, PA_ERR_ARG, PA_ERR_NO_BLOCKS. */
int pa_seq_extend(pa_pool* pool, int64_t seq_id, const int32_t* tokens, int32_t n_tokens);

/* Roll sequence seq_id back to new_len tokens (rejected drafts, a chunk to
 * redo).  Blocks no longer needed return to the FRONT of the free list, so
 * extend followed by truncate restores the pool exactly.  new_len must be at
 * least the number of tokens in the sequence's leading cached blocks.
 * Errors: PA_ERR_UNKNOWN_SEQ, PA_ERR_ARG. */
int pa_seq_truncate(pa_pool* pool, int64_t seq_id, int32_t new_len);

/* Release a finished sequence.  Its full blocks are cached first (same rule as
 * at admission); cached blocks stay resident with no owner (idle) until
 * evicted; uncached blocks return to the back of the free list.
 * Errors: PA_ERR_UNKNOWN_SEQ. */
int pa_seq_free(pa_pool* pool, int64_t seq_id);

/* Least-recently-used eviction of idle cached blocks (paper: Section 2, APC
 * keeps reusable prefix blocks resident; Section 5.4, a prefix identical
 * across many requests stays hot).  Off by default: an admission or extension
 * needing more blocks than the free list holds then fails with
 * PA_ERR_NO_BLOCKS.  On: the free list is used first, then idle cached blocks
 * (held by no live sequence) are evicted one at a time, always a block that
 * no other cached block continues, the one released longest ago first
 * (blocks released by one pa_seq_free count as released last block first).
 * An evicted block leaves the prefix cache and goes to the request; a later
 * request with that prefix recomputes it.  The failure check counts idle
 * blocks, so a failing request still leaves the pool unchanged. */
int pa_pool_set_eviction(pa_pool* pool, int32_t enabled);

/* Occupancy counters of a pool. */
typedef struct {
  int64_t num_blocks;
  int64_t free_blocks;        /* on the free list */
  int64_t cached_blocks;      /* in the prefix cache, held or idle */
  int64_t idle_cached_blocks; /* cached and held by no live sequence */
  int64_t evictions;          /* cached blocks evicted since creation */
  int64_t live_seqs;
  int64_t live_tokens;        /* sum of live sequence lengths */
  int64_t logical_blocks;     /* sum of live block-table lengths */
  int64_t physical_blocks;    /* distinct blocks held by live sequences */
} pa_pool_stats;
int pa_pool_get_stats(const pa_pool* pool, pa_pool_stats* out);

/* KV memory accounting of the live sequences (paper: Section 2, paged KV
 * memory against contiguous per-request reservations, Table "playbook"):
 * slots allocated in blocks versus reserving max_seq_len contiguous slots per
 * request.  Paged waste per sequence is below block_size / length; shared
 * prefix blocks count once in physical_slots.  Errors: PA_ERR_ARG when
 * max_seq_len is below the longest live sequence. */
typedef struct {
  int64_t tokens;           /* sum of live sequence lengths */
  int64_t paged_slots;      /* block_size x sum of block-table lengths */
  int64_t physical_slots;   /* block_size x distinct blocks held */
  int64_t contiguous_slots; /* live sequences x max_seq_len */
  double paged_waste;       /* 1 - tokens / paged_slots (0 with no sequences) */
  double contiguous_waste;  /* 1 - tokens / contiguous_slots */
  double sharing_factor;    /* paged_slots / physical_slots (1 with no sequences) */
} pa_kv_waste;
int pa_pool_kv_waste(const pa_pool* pool, int32_t max_seq_len, pa_kv_waste* out);

/* Batched forms for a serving step: n operations applied in order, exactly as
 * n calls of the single-sequence function would (sequence i owns tokens
 * token_offsets[i] .. token_offsets[i+1]-1 of the concatenated `tokens`).
 * They stop at the first failing operation, which leaves the pool as it was
 * before that operation; *n_done (may be NULL) receives the number of
 * operations applied.  n_cached_out (may be NULL) receives n entries. */
int pa_seqs_add(pa_pool* pool, int32_t n, const int64_t* seq_ids, const int32_t* token_offsets,
                const int32_t* tokens, int32_t* n_cached_out, int32_t* n_done);
int pa_seqs_extend(pa_pool* pool, int32_t n, const int64_t* seq_ids,
                   const int32_t* token_offsets, const int32_t* tokens, int32_t* n_done);
int pa_seqs_truncate(pa_pool* pool, int32_t n, const int64_t* seq_ids, const int32_t* new_lens,
                     int32_t* n_done);
int pa_seqs_free(pa_pool* pool, int32_t n, const int64_t* seq_ids, int32_t* n_done);

/* A serving step's pool operations of mixed kinds in one call: operation i
 * applies ops[i] to seq_ids[i] exactly as the single-sequence function would;
 * PA_OP_ADD / PA_OP_EXTEND take tokens token_offsets[i] .. token_offsets[i+1]-1
 * (token_offsets has n+1 entries; other kinds own an empty range),
 * PA_OP_TRUNCATE takes new_lens[i] (new_lens may be NULL if there is none),
 * PA_OP_FREE takes nothing.  n_cached_out[i] (may be NULL) receives the
 * reused-token count of an admission, 0 otherwise.  Stops at the first
 * failing operation (pool as before that operation); *n_done (may be NULL)
 * receives the number applied. */
typedef enum { PA_OP_ADD = 0, PA_OP_EXTEND = 1, PA_OP_TRUNCATE = 2, PA_OP_FREE = 3 } pa_op;
int pa_pool_apply(pa_pool* pool, int32_t n, const int32_t* ops, const int64_t* seq_ids,
                  const int32_t* token_offsets, const int32_t* tokens, const int32_t* new_lens,
                  int32_t* n_cached_out, int32_t* n_done);

/* Current length of a live sequence.  Errors: PA_ERR_UNKNOWN_SEQ. */
int pa_seq_len(const pa_pool* pool, int64_t seq_id, int32_t* len_out);

/* Copy the physical blocks of a live sequence (logical order) into out
 * (capacity entries); *n_out receives the count.  Errors: PA_ERR_UNKNOWN_SEQ,
 * PA_ERR_ARG (capacity too small). */
int pa_seq_blocks(const pa_pool* pool, int64_t seq_id, int32_t* out, int32_t capacity,
                  int32_t* n_out);

/* Copy the free list (front first) into out; *n_out receives its length. */
int pa_pool_free_list(const pa_pool* pool, int32_t* out, int32_t capacity, int32_t* n_out);

/* Build the varlen metadata of one launch over n_seqs live sequences (batch
 * order = seq_ids order; an id may appear once).  q_lens[r] in [0, len_r]
 * query tokens are the sequence's last q_lens[r] positions.  Outputs (host,
 * caller-owned):
 *   block_table[n_seqs][max_blocks_per_seq]  physical block ids, padded -1
 *   seq_lens[n_seqs]                         sequence lengths (keys visible)
 *   cu_seqlens_q[n_seqs+1]                   exclusive prefix sum of q_lens
 *   slot_mapping[sum q_lens]                 slot of every query token
 * slot_capacity is the length of slot_mapping.  Errors: PA_ERR_ARG
 * (q_len out of range, a sequence needing more than max_blocks_per_seq blocks,
 * repeated id, capacity too small), PA_ERR_UNKNOWN_SEQ. */
int pa_build_metadata(const pa_pool* pool, int32_t n_seqs, const int64_t* seq_ids,
                      const int32_t* q_lens, int32_t max_blocks_per_seq, int32_t* block_table,
                      int32_t* seq_lens, int32_t* cu_seqlens_q, int32_t* slot_mapping,
                      int64_t slot_capacity);

/* Adapter-first, length-bucketed batch forming (paper: Section 5.6,
 * "Multi-Adapter and Length-Aware Batching", and Table "casec_adapter"): item
 * i is (adapter_ids[i], prompt_lens[i], i).  Items are grouped by adapter
 * (groups in the order of their first item) and each group is split into
 * length buckets by the strictly ascending upper bounds bucket_bounds[0 ..
 * n_bounds): bucket k holds lengths below bucket_bounds[k] that no earlier
 * bucket holds, bucket n_bounds the rest.  Every non-empty (adapter, bucket)
 * is one batch; batches run adapter group by adapter group, short buckets
 * first, items in original order inside a batch.  Outputs (host,
 * caller-owned):
 *   order[n]            original index of the item at execution position p
 *   position[n]         execution position of original item i (restores the
 *                       original order: result i = executed result position[i])
 *   batch_offsets[n+1]  batch b is order[batch_offsets[b] .. batch_offsets[b+1])
 *   batch_adapter[n]    adapter of batch b
 *   batch_bucket[n]     length bucket of batch b (0 = shortest)
 *   *n_batches          number of batches (<= n)
 * Errors: PA_ERR_ARG (NULL or negative argument, negative length, bounds not
 * strictly ascending). */
int pa_form_batches(int32_t n, const int32_t* adapter_ids, const int32_t* prompt_lens,
                    int32_t n_bounds, const int32_t* bucket_bounds, int32_t* order,
                    int32_t* position, int32_t* batch_offsets, int32_t* batch_adapter,
                    int32_t* batch_bucket, int32_t* n_batches);

/* ------------------------------------------------------------------------ *
 * Launch plan (host).                                                        *
 * ------------------------------------------------------------------------ */

typedef enum { PA_KIND_PREFILL = 0, PA_KIND_DECODE = 1, PA_KIND_VERIFY = 2 } pa_kind;

typedef struct pa_plan_info {
  int32_t kind;            /* pa_kind the plan was built for                      */
  int32_t n_q;             /* query tokens per sequence (decode 1, verify n_q)    */
  int32_t n_shared_items;  /* shared-prefix (cascade) items, one workgroup each   */
  int32_t n_tile_items;    /* 128-row work items (one workgroup each)             */
  int32_t n_row_items;     /* <=32-row work items (one wavefront each)            */
  int32_t n_groups;        /* split groups the merge step combines                */
  int32_t n_merge_rows;    /* (token, head) rows produced by the merge step       */
  int32_t grid;            /* workgroups of the attention launch                  */
  int32_t variant;         /* kernel instantiation (internal)                     */
  int32_t reserved;
  int64_t plan_words;      /* int32 words of the plan array                       */
  int64_t workspace_bytes; /* device scratch the attention call needs             */
  /* The launch shape the plan was built for; the attention calls reject a
   * call whose arguments differ. */
  int32_t n_seqs;
  int32_t total_q;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t dtype;
  int64_t partial_rows;    /* float32 partial rows in the workspace               */
} pa_plan_info;

/* Split one attention launch into work items from HOST copies of seq_lens,
 * cu_seqlens_q and (optionally) block_table[n_seqs][max_blocks_per_seq], as
 * produced by pa_build_metadata.  With a block table, sequences of at most
 * 64 query rows per kv-head (decode, verification) whose tables start with
 * the same blocks form shared-prefix groups: their attention over the shared
 * keys is computed once for all their rows and merged with each sequence's
 * private part by log-sum-exp (pass NULL to disable).  With plan == NULL only
 * *info is filled (size query).  Otherwise the int32 plan (plan_capacity
 * words, host memory) is written; the caller copies it to device memory and
 * passes the device copy and *info to the attention call.  If plan_capacity
 * is too small the call fails with PA_ERR_ARG and *info holds the size.
 * kind PA_KIND_DECODE requires every q_len == 1, PA_KIND_VERIFY every q_len ==
 * n_q (1..8); PA_KIND_PREFILL takes any q_len >= 0 (prefill chunks and decode
 * tokens may be mixed).  num_cus = compute units to fill (0: 256).
 * Errors: PA_ERR_ARG, PA_ERR_UNSUPPORTED. */
int pa_attn_plan(int32_t kind, int32_t n_q, int32_t n_seqs, const int32_t* seq_lens,
                 const int32_t* cu_seqlens_q, const int32_t* block_table,
                 int32_t max_blocks_per_seq, int32_t num_q_heads, int32_t num_kv_heads,
                 int32_t head_dim, int32_t block_size, int32_t dtype, int32_t num_cus,
                 int32_t* plan, int64_t plan_capacity, pa_plan_info* info);

/* Upper bound on the split-K workspace (float32 partial outputs and their
 * log-sum-exps, merged by the attention call) of any plan pa_attn_plan builds
 * for a launch of total_q query tokens whose sequences are at most
 * max_seq_len keys long, at num_q_heads query heads and head_dim (paper:
 * Section 5.3, decode of short structured outputs, where long key ranges are
 * split across wavefronts to stream the cache).  Lets a caller size one
 * workspace before any plan exists; a plan's own need, info->workspace_bytes,
 * is never larger.  Host only, allocates nothing.  *bytes receives the bound.
 * Errors: PA_ERR_ARG (negative size, NULL bytes), PA_ERR_UNSUPPORTED
 * (head_dim). */
int pa_attn_workspace_size(int32_t total_q, int32_t num_q_heads, int32_t head_dim,
                           int32_t max_seq_len, size_t* bytes);

/* The same bound for a decode launch of n_seqs sequences (one query token
 * each): pa_attn_workspace_size(n_seqs, ...). */
int pa_attn_decode_workspace_size(int32_t n_seqs, int32_t num_q_heads, int32_t head_dim,
                                  int32_t max_seq_len, size_t* bytes);

/* The host side of one serving step's launch in one call (paper: Section 2,
 * block tables and Automatic Prefix Caching; Section 5.2, one batched launch
 * per step): exactly
 *   pa_pool_apply(pool, n_ops, ops, op_seq_ids, op_token_offsets, op_tokens,
 *                 op_new_lens, op_n_cached, NULL)          (skipped if n_ops == 0)
 *   pa_build_metadata(pool, n_seqs, seq_ids, q_lens, max_blocks_per_seq,
 *                     block_table, seq_lens, cu_seqlens_q, slot_mapping,
 *                     slot_capacity)
 *   pa_attn_plan(kind, n_q, n_seqs, seq_lens, cu_seqlens_q,
 *                shared_prefix ? block_table : NULL, max_blocks_per_seq,
 *                num_q_heads, num_kv_heads, head_dim, <the pool's block size>,
 *                dtype, num_cus, plan, plan_capacity, info)
 * with the arguments, layouts, ownership (all host, caller-owned) and error
 * behaviour of those three functions.  It stops at the first failing step
 * and returns its code: pool operations already applied stay applied (as
 * pa_pool_apply documents); outputs of later steps are not written. */
int pa_prepare_launch(pa_pool* pool, int32_t n_ops, const int32_t* ops,
                      const int64_t* op_seq_ids, const int32_t* op_token_offsets,
                      const int32_t* op_tokens, const int32_t* op_new_lens, int32_t* op_n_cached,
                      int32_t n_seqs, const int64_t* seq_ids, const int32_t* q_lens,
                      int32_t max_blocks_per_seq, int32_t* block_table, int32_t* seq_lens,
                      int32_t* cu_seqlens_q, int32_t* slot_mapping, int64_t slot_capacity,
                      int32_t kind, int32_t n_q, int32_t num_q_heads, int32_t num_kv_heads,
                      int32_t head_dim, int32_t dtype, int32_t num_cus, int32_t shared_prefix,
                      int32_t* plan, int64_t plan_capacity, pa_plan_info* info);

/* ------------------------------------------------------------------------ *
 * Device operations.                                                         *
 * ------------------------------------------------------------------------ */

/* Store the keys/values of n_tokens new tokens into their cache slots (paper:
 * Section 2, PagedAttention keeps a request's KV in blocks addressed through
 * its block table; a token's KV is written once and then reused by every
 * later step and, for cached prefix blocks, by every request that hits them):
 * k_cache[s/bs][h][d/32][pos(s%bs)][d%32] = k_new[i][h][d] and
 * v_cache[s/bs][h][d][s%bs] = v_new[i][h][d] for s = slot_mapping[i] (the
 * cache layout above).
 * k_new, v_new: [n_tokens][num_kv_heads][head_dim] (dtype).  A slot outside
 * [0, num_blocks*block_size) skips its token (use -1 for padding).  All
 * pointers are caller-owned device memory; asynchronous on stream; allocates
 * nothing.  Bit-exact copy.  Errors: PA_ERR_ARG (NULL pointer with tokens to
 * store, negative n_tokens, bad sizes), PA_ERR_UNSUPPORTED (head_dim,
 * block_size, dtype), PA_ERR_LAUNCH. */
int pa_kv_append(const void* k_new, const void* v_new, const int32_t* slot_mapping,
                 int32_t n_tokens, void* k_cache, void* v_cache, int32_t num_blocks,
                 int32_t num_kv_heads, int32_t head_dim, int32_t block_size, int32_t dtype,
                 void* stream);

/* Upload of a launch's host-built metadata and plan (paper: Section 5.2, one
 * batched launch per serving step): copies bytes (a multiple of 4) from src,
 * page-locked host memory the device can read (e.g. from hipHostMalloc), to
 * dst, device memory, by a kernel on the stream, which reads the host buffer
 * over the bus (no copy-engine start-up).  The caller must not modify src
 * until the copy has completed on the stream (e.g. an event recorded after
 * this call).  Errors (checked before anything is launched): PA_ERR_ARG (size
 * not a multiple of 4, misaligned or NULL pointers, either end of the source
 * range not pinned host memory the device can address, or of the destination
 * range not device memory); PA_ERR_LAUNCH. */
int pa_stage_upload(void* dst, const void* src, int64_t bytes, void* stream);

/* Paged attention over a prefix-shared KV cache (paper: Section 2,
 * PagedAttention's block tables and Automatic Prefix Caching; Section 3,
 * cached shared policy prefixes give the result of recomputing them, so
 * serving a suffix against cached prefix blocks is exact attention over the
 * whole logical sequence).  pa_attn_prefill serves suffix prefill of per-case
 * evidence against the cached prefix and, with a plan mixing prefill chunks
 * and decode tokens, the mixed launch (Section 5.2, split prefills under a
 * batched-token budget; Section 6, Table "playbook": long prefills blocking
 * short decodes).
 * For sequence r, q-head h and its query i at logical position
 * a = seq_lens[r] - q_len_r + i:
 *   out = sum_{t<=a} softmax_t(scale * q . k_t) v_t,   k_t, v_t from kv-head
 *   h / G of the block table row r,
 *   lse = log sum_{t<=a} exp(scale * q . k_t).
 * Device inputs: q, caches, block_table[n_seqs][max_blocks_per_seq],
 * seq_lens[n_seqs], cu_seqlens_q[n_seqs+1] (the same values the plan was built
 * from), plan (device copy of pa_attn_plan's output) with its *info (the
 * block table must be the one the plan's shared-prefix groups were found in),
 * workspace of at least info->workspace_bytes bytes (any contents) or NULL if
 * that is 0.  Block ids must lie in [0, num_blocks); out-of-range ids are
 * clamped so no access leaves the cache (results are then undefined).
 * Every pointer is caller-owned device memory (info: host); the call
 * allocates nothing, writes only out, lse, the workspace and two counter
 * words of the plan's header, which its work-stealing workgroups count on
 * (device-scope atomics) and which it leaves zero, as pa_attn_plan wrote
 * them, so one device plan serves any number of calls ordered on a stream
 * (calls sharing one device plan must not overlap in time), and is
 * asynchronous on stream.  The three entry points differ only in the plan
 * kind they accept.
 * Errors (checked before anything is launched): PA_ERR_ARG (NULL pointer with
 * work to do, a plan of another kind, n_seqs / total_q / num_q_heads /
 * num_kv_heads / head_dim / dtype other than the plan's info records, a
 * workspace smaller than info->workspace_bytes), PA_ERR_UNSUPPORTED (head_dim,
 * block_size, dtype), PA_ERR_LAUNCH (the runtime rejected the launch). */
int pa_attn_prefill(const void* q, const void* k_cache, const void* v_cache, int32_t num_blocks,
                    const int32_t* block_table, int32_t max_blocks_per_seq,
                    const int32_t* seq_lens, const int32_t* cu_seqlens_q, int32_t n_seqs,
                    int32_t total_q, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                    int32_t block_size, float scale, int32_t dtype, int32_t* plan,
                    const pa_plan_info* info, void* workspace, size_t workspace_bytes,
                    void* out, float* lse, void* stream);

/* Decode: one query token per sequence (plan kind PA_KIND_DECODE); paper:
 * Section 5.3 (short structured outputs, decode-time control) and Section 3,
 * Table "phenotype" (long input, short JSON output).  Arguments, layouts,
 * ownership and errors as pa_attn_prefill. */
int pa_attn_decode(const void* q, const void* k_cache, const void* v_cache, int32_t num_blocks,
                   const int32_t* block_table, int32_t max_blocks_per_seq,
                   const int32_t* seq_lens, const int32_t* cu_seqlens_q, int32_t n_seqs,
                   int32_t total_q, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                   int32_t block_size, float scale, int32_t dtype, int32_t* plan,
                   const pa_plan_info* info, void* workspace, size_t workspace_bytes,
                   void* out, float* lse, void* stream);

/* Speculative verification: n_q = info->n_q query tokens per sequence (the
 * draft tokens and the bonus position), causal among themselves (plan kind
 * PA_KIND_VERIFY); paper: Section 5.3 and Table "caseb" (EAGLE-style
 * speculative decoding, whose target-model pass scores every draft token
 * against the cached context at once), Section 2 (speculative decoding).
 * Arguments, layouts, ownership and errors as pa_attn_prefill. */
int pa_attn_verify(const void* q, const void* k_cache, const void* v_cache, int32_t num_blocks,
                   const int32_t* block_table, int32_t max_blocks_per_seq,
                   const int32_t* seq_lens, const int32_t* cu_seqlens_q, int32_t n_seqs,
                   int32_t total_q, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                   int32_t block_size, float scale, int32_t dtype, int32_t* plan,
                   const pa_plan_info* info, void* workspace, size_t workspace_bytes,
                   void* out, float* lse, void* stream);

/* Decode for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops that must not call hipMalloc, harnesses that
 * forbid it): exactly pa_attn_decode with the same arguments minus the
 * workspace.  The split-K partial results go to a device array the library
 * owns, PA_NOALLOC_WORKSPACE_BYTES bytes on each GPU it runs on, set up on
 * the first call on that GPU (the calling thread's current device, which must
 * be the stream's) and held until the process ends; the call allocates
 * nothing.  Every call on one GPU shares that array and it keeps the last
 * call's contents (nothing in it needs to start at zero): calls ordered on
 * one stream are safe, calls that overlap in time on one GPU (other streams,
 * other threads) race.
 * Errors: those of pa_attn_decode, plus PA_ERR_ARG when the plan's
 * info->workspace_bytes exceeds PA_NOALLOC_WORKSPACE_BYTES (use
 * pa_attn_decode with a workspace of that size instead), PA_ERR_LAUNCH when
 * the array's device address cannot be obtained. */
#define PA_NOALLOC_WORKSPACE_BYTES ((size_t)32 << 20)
int pa_attn_decode_noalloc(const void* q, const void* k_cache, const void* v_cache,
                           int32_t num_blocks, const int32_t* block_table,
                           int32_t max_blocks_per_seq, const int32_t* seq_lens,
                           const int32_t* cu_seqlens_q, int32_t n_seqs, int32_t total_q,
                           int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                           int32_t block_size, float scale, int32_t dtype, int32_t* plan,
                           const pa_plan_info* info, void* out, float* lse, void* stream);

/* Timing hook, for callers that time attention calls on the device
 * (benchmarks, profilers) without event packets between kernels: the next
 * pa_attn_* call on this thread attaches start_event to the dispatch of its
 * first kernel (recorded when that kernel starts) and stop_event to the
 * dispatch of its last (recorded when it ends), through hipExtLaunchKernel,
 * instead of separate event records, each of which idles the device for a
 * few microseconds between back-to-back kernels.  Either may be NULL.  The
 * events are hipEvent_t handles the caller created (with timing, for
 * hipEventElapsedTime), passed as void*, and stay the caller's.  That call
 * consumes the setting, also when it fails; later calls attach nothing
 * until it is set again.  A call that launches no kernel records both
 * events on its stream.  Errors: none. */
int pa_set_launch_events(void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif

#endif /* PA_H_ */
