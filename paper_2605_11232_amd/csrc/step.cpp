// The host side of one serving step's attention launch in a single call:
// the step's pool operations (admissions with prefix-cache lookup, extends,
// rollbacks, releases), the launch metadata and the launch plan, written
// straight into caller-owned (typically pinned) buffers.  Paper: Section 2
// (block tables, Automatic Prefix Caching) and Section 5.2 (each step batches
// its requests into one launch under a token budget).  The call composes
// pa_pool_apply, pa_build_metadata and pa_attn_plan; it exists so a driver
// crosses the C boundary once per step instead of three times.
#include "internal.h"

extern "C" int pa_prepare_launch(pa_pool* pool, int32_t n_ops, const int32_t* ops,
                                 const int64_t* op_seq_ids, const int32_t* op_token_offsets,
                                 const int32_t* op_tokens, const int32_t* op_new_lens,
                                 int32_t* op_n_cached, int32_t n_seqs, const int64_t* seq_ids,
                                 const int32_t* q_lens, int32_t max_blocks_per_seq,
                                 int32_t* block_table, int32_t* seq_lens, int32_t* cu_seqlens_q,
                                 int32_t* slot_mapping, int64_t slot_capacity, int32_t kind,
                                 int32_t n_q, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t dtype, int32_t num_cus,
                                 int32_t shared_prefix, int32_t* plan, int64_t plan_capacity,
                                 pa_plan_info* info) {
  pa::clear_error();
  if (!pool) return pa::fail(PA_ERR_ARG, "pa_prepare_launch: NULL pool");
  if (n_ops < 0) return pa::fail(PA_ERR_ARG, "pa_prepare_launch: n_ops %d < 0", n_ops);
  if (n_ops > 0) {
    const int rc = pa_pool_apply(pool, n_ops, ops, op_seq_ids, op_token_offsets, op_tokens,
                                 op_new_lens, op_n_cached, nullptr);
    if (rc != PA_OK) return rc;
  }
  int rc = pa_build_metadata(pool, n_seqs, seq_ids, q_lens, max_blocks_per_seq, block_table,
                             seq_lens, cu_seqlens_q, slot_mapping, slot_capacity);
  if (rc != PA_OK) return rc;
  return pa_attn_plan(kind, n_q, n_seqs, seq_lens, cu_seqlens_q,
                      shared_prefix ? block_table : nullptr, max_blocks_per_seq, num_q_heads,
                      num_kv_heads, head_dim, pa::pool_block_size(pool), dtype, num_cus, plan,
                      plan_capacity, info);
}
