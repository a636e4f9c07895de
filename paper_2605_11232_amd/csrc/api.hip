// C-ABI device entry points: argument validation on the host, then launches
// on the caller's stream.  See include/pa.h for the contract of each call.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"
#include "plan_format.h"

namespace pa {
namespace dev {
int launch_attn_bf16(const void* q, const void* kc, const void* vc, int32_t num_blocks,
                     const int32_t* bt, int32_t max_blocks, const int32_t* seq_lens,
                     const int32_t* cu_q, int32_t hq, int32_t hkv, int32_t d, float scale,
                     const int32_t* plan, int32_t grid, int32_t n_tile, int32_t n_groups,
                     bool wide_rows, bool tail, int64_t partial_rows, void* ws, void* out,
                     float* lse, hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop);
int launch_attn_f32(const void* q, const void* kc, const void* vc, int32_t num_blocks,
                    const int32_t* bt, int32_t max_blocks, const int32_t* seq_lens,
                    const int32_t* cu_q, int32_t n_seqs, int32_t total_q, int32_t hq, int32_t hkv,
                    int32_t d, float scale, void* out, float* lse, hipStream_t stream,
                    hipEvent_t ev_start, hipEvent_t ev_stop);
int launch_kv_append(const void* kn, const void* vn, const int32_t* slots, int32_t n, void* kc,
                     void* vc, int32_t nb, int32_t hkv, int32_t d, int32_t dtype,
                     hipStream_t stream);
int launch_stage_upload(const void* src, void* dst, int64_t n_dwords, hipStream_t stream);
}  // namespace dev

namespace {

// Timing events for the next attention call on this thread
// (pa_set_launch_events); each call takes them and clears them.
thread_local hipEvent_t t_ev_start = nullptr, t_ev_stop = nullptr;

int check_shape(const char* fn, int32_t num_blocks, int32_t num_kv_heads, int32_t head_dim,
                int32_t block_size, int32_t dtype) {
  if (num_blocks <= 0 || num_kv_heads <= 0)
    return fail(PA_ERR_ARG, "%s: num_blocks %d and num_kv_heads %d must be positive", fn,
                num_blocks, num_kv_heads);
  if (int64_t(num_blocks) * block_size >= (int64_t{1} << 31))
    return fail(PA_ERR_ARG, "%s: num_blocks * block_size must be < 2^31", fn);
  if (head_dim != 64 && head_dim != 128)
    return fail(PA_ERR_UNSUPPORTED, "%s: head_dim %d (supported: 64, 128)", fn, head_dim);
  if (block_size != 16)
    return fail(PA_ERR_UNSUPPORTED, "%s: block_size %d (supported: 16)", fn, block_size);
  if (dtype != PA_F32 && dtype != PA_BF16)
    return fail(PA_ERR_UNSUPPORTED, "%s: dtype %d (supported: PA_F32, PA_BF16)", fn, dtype);
  return PA_OK;
}

// Split-K workspace of pa_attn_decode_noalloc: one array per GPU, in the
// code object's device memory.  Its name is a host-side stand-in; kernels
// get the device address each GPU reports for it.
static __device__ __align__(256) unsigned char scratch[PA_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of `scratch` on the calling thread's current device, looked
// up once per device.
int scratch_address(const char* fn, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return fail(PA_ERR_LAUNCH, "%s: hipGetDevice: %s", fn, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(PA_ERR_UNSUPPORTED, "%s: device %d (at most %d devices)", fn, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(PA_ERR_LAUNCH, "%s: hipGetSymbolAddress: %s", fn, hipGetErrorString(e));
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return PA_OK;
}

int attn_common(const char* fn, int32_t want_kind, const void* q, const void* k_cache,
                const void* v_cache, int32_t num_blocks, const int32_t* block_table,
                int32_t max_blocks_per_seq, const int32_t* seq_lens, const int32_t* cu_seqlens_q,
                int32_t n_seqs, int32_t total_q, int32_t num_q_heads, int32_t num_kv_heads,
                int32_t head_dim, int32_t block_size, float scale, int32_t dtype,
                const int32_t* plan, const pa_plan_info* info, void* workspace,
                size_t workspace_bytes, void* out, float* lse, void* stream,
                bool noalloc = false) {
  clear_error();
  const hipEvent_t ev_start = t_ev_start, ev_stop = t_ev_stop;
  t_ev_start = t_ev_stop = nullptr;
  int rc = check_shape(fn, num_blocks, num_kv_heads, head_dim, block_size, dtype);
  if (rc) return rc;
  if (num_q_heads <= 0 || num_q_heads % num_kv_heads)
    return fail(PA_ERR_ARG, "%s: num_q_heads %d must be a positive multiple of num_kv_heads %d",
                fn, num_q_heads, num_kv_heads);
  if (n_seqs < 0 || total_q < 0 || max_blocks_per_seq < 1)
    return fail(PA_ERR_ARG, "%s: negative size or max_blocks_per_seq < 1", fn);
  if (!(scale > 0.f) || scale == __builtin_huge_valf())
    return fail(PA_ERR_ARG, "%s: scale must be positive and finite", fn);
  if (!info) return fail(PA_ERR_ARG, "%s: NULL plan info", fn);
  if (info->kind != want_kind)
    return fail(PA_ERR_ARG, "%s: plan was built for kind %d, this call needs kind %d", fn,
                info->kind, want_kind);
  // the plan's items index sequences, heads and rows of the launch it was
  // built for: any other shape could send them past the caller's buffers
  if (info->n_seqs != n_seqs || info->total_q != total_q || info->num_q_heads != num_q_heads ||
      info->num_kv_heads != num_kv_heads || info->head_dim != head_dim || info->dtype != dtype)
    return fail(PA_ERR_ARG,
                "%s: plan was built for n_seqs %d, total_q %d, heads %d/%d, head_dim %d, "
                "dtype %d; this call has n_seqs %d, total_q %d, heads %d/%d, head_dim %d, "
                "dtype %d", fn, info->n_seqs, info->total_q, info->num_q_heads,
                info->num_kv_heads, info->head_dim, info->dtype, n_seqs, total_q, num_q_heads,
                num_kv_heads, head_dim, dtype);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (total_q == 0 || n_seqs == 0) {
    // nothing to launch: the events still mark this point of the stream
    for (hipEvent_t ev : {ev_start, ev_stop}) {
      const hipError_t e = ev ? hipEventRecord(ev, st) : hipSuccess;
      if (e != hipSuccess)
        return fail(PA_ERR_LAUNCH, "%s: hipEventRecord: %s", fn, hipGetErrorString(e));
    }
    return PA_OK;
  }
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !cu_seqlens_q || !out)
    return fail(PA_ERR_ARG, "%s: NULL device pointer", fn);
  if (dtype == PA_F32) {
    rc = dev::launch_attn_f32(q, k_cache, v_cache, num_blocks, block_table, max_blocks_per_seq,
                              seq_lens, cu_seqlens_q, n_seqs, total_q, num_q_heads, num_kv_heads,
                              head_dim, scale, out, lse, st, ev_start, ev_stop);
  } else {
    if (!plan) return fail(PA_ERR_ARG, "%s: NULL plan", fn);
    if ((info->variant & ~(kVariantWideRows | kVariantTail)) != kVariantBf16 || info->grid < 0 ||
        info->n_groups < 0 ||
        info->n_tile_items < 0 || info->n_shared_items < 0 ||
        int64_t(info->n_tile_items) + info->n_shared_items > info->grid ||
        info->partial_rows < 0 ||
        info->workspace_bytes != info->partial_rows * int64_t(head_dim + 1) * 4)
      return fail(PA_ERR_ARG, "%s: corrupt plan info", fn);
    if (noalloc) {
      // the workspace is the library's per-device array
      if (static_cast<uint64_t>(info->workspace_bytes) > PA_NOALLOC_WORKSPACE_BYTES)
        return fail(PA_ERR_ARG, "%s: the plan needs %lld bytes of workspace, more than the "
                    "%zu bytes this call holds per device; call pa_attn_decode with a "
                    "workspace of that size", fn, (long long)info->workspace_bytes,
                    (size_t)PA_NOALLOC_WORKSPACE_BYTES);
      workspace = nullptr;
      workspace_bytes = 0;
      if (info->workspace_bytes > 0) {
        rc = scratch_address(fn, &workspace);
        if (rc) return rc;
        workspace_bytes = PA_NOALLOC_WORKSPACE_BYTES;
      }
    }
    if (static_cast<int64_t>(workspace_bytes) < info->workspace_bytes ||
        (info->workspace_bytes > 0 && !workspace))
      return fail(PA_ERR_ARG, "%s: workspace of %zu bytes, plan needs %lld", fn, workspace_bytes,
                  (long long)info->workspace_bytes);
    const int64_t partial_rows = info->partial_rows;
    rc = dev::launch_attn_bf16(q, k_cache, v_cache, num_blocks, block_table, max_blocks_per_seq,
                               seq_lens, cu_seqlens_q, num_q_heads, num_kv_heads, head_dim, scale,
                               plan, info->grid, info->n_shared_items + info->n_tile_items,
                               info->n_groups, (info->variant & kVariantWideRows) != 0,
                               (info->variant & kVariantTail) != 0,
                               partial_rows,
                               workspace, out, lse, st, ev_start, ev_stop);
  }
  if (rc) return fail(PA_ERR_LAUNCH, "%s: %s", fn, hipGetErrorString(static_cast<hipError_t>(rc)));
  return PA_OK;
}

}  // namespace
}  // namespace pa

extern "C" {

int pa_kv_append(const void* k_new, const void* v_new, const int32_t* slot_mapping,
                 int32_t n_tokens, void* k_cache, void* v_cache, int32_t num_blocks,
                 int32_t num_kv_heads, int32_t head_dim, int32_t block_size, int32_t dtype,
                 void* stream) {
  pa::clear_error();
  int rc = pa::check_shape("pa_kv_append", num_blocks, num_kv_heads, head_dim, block_size, dtype);
  if (rc) return rc;
  if (n_tokens < 0) return pa::fail(PA_ERR_ARG, "pa_kv_append: n_tokens %d < 0", n_tokens);
  if (n_tokens == 0) return PA_OK;
  if (!k_new || !v_new || !slot_mapping || !k_cache || !v_cache)
    return pa::fail(PA_ERR_ARG, "pa_kv_append: NULL device pointer");
  rc = pa::dev::launch_kv_append(k_new, v_new, slot_mapping, n_tokens, k_cache, v_cache,
                                 num_blocks, num_kv_heads, head_dim, dtype,
                                 static_cast<hipStream_t>(stream));
  if (rc)
    return pa::fail(PA_ERR_LAUNCH, "pa_kv_append: %s",
                    hipGetErrorString(static_cast<hipError_t>(rc)));
  return PA_OK;
}

// Both ends of [p, p + bytes) must be memory of the given kind that the device
// can address; *dev receives the device address of p.  A failed query leaves
// no HIP error behind.
static bool device_visible(const void* p, int64_t bytes, hipMemoryType want, void** dev) {
  const char* c = static_cast<const char*>(p);
  for (const char* q : {c, c + bytes - 1}) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, q) != hipSuccess) {
      (void)hipGetLastError();
      return false;
    }
    if (at.type != want || at.devicePointer == nullptr) return false;
    if (q == c) *dev = at.devicePointer;
  }
  return true;
}

int pa_stage_upload(void* dst, const void* src, int64_t bytes, void* stream) {
  pa::clear_error();
  if (bytes < 0 || bytes % 4 ||
      (bytes > 0 && (!dst || !src ||
                     ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 3))))
    return pa::fail(PA_ERR_ARG, "pa_stage_upload: bytes %lld must be a multiple of 4 with "
                    "4-byte aligned, non-NULL pointers", (long long)bytes);
  if (bytes == 0) return PA_OK;
  void* src_dev = nullptr;
  void* dst_dev = nullptr;
  if (!device_visible(src, bytes, hipMemoryTypeHost, &src_dev))
    return pa::fail(PA_ERR_ARG, "pa_stage_upload: source is not pinned host memory the device "
                    "can read");
  if (!device_visible(dst, bytes, hipMemoryTypeDevice, &dst_dev))
    return pa::fail(PA_ERR_ARG, "pa_stage_upload: destination is not device memory");
  const int rc =
      pa::dev::launch_stage_upload(src_dev, dst_dev, bytes / 4, static_cast<hipStream_t>(stream));
  if (rc)
    return pa::fail(PA_ERR_LAUNCH, "pa_stage_upload: %s",
                    hipGetErrorString(static_cast<hipError_t>(rc)));
  return PA_OK;
}

#define PA_ATTN_ARGS                                                                            \
  const void *q, const void *k_cache, const void *v_cache, int32_t num_blocks,                  \
      const int32_t *block_table, int32_t max_blocks_per_seq, const int32_t *seq_lens,          \
      const int32_t *cu_seqlens_q, int32_t n_seqs, int32_t total_q, int32_t num_q_heads,        \
      int32_t num_kv_heads, int32_t head_dim, int32_t block_size, float scale, int32_t dtype,   \
      int32_t *plan, const pa_plan_info *info, void *workspace, size_t workspace_bytes,         \
      void *out, float *lse, void *stream
#define PA_ATTN_PASS                                                                            \
  q, k_cache, v_cache, num_blocks, block_table, max_blocks_per_seq, seq_lens, cu_seqlens_q,     \
      n_seqs, total_q, num_q_heads, num_kv_heads, head_dim, block_size, scale, dtype, plan,     \
      info, workspace, workspace_bytes, out, lse, stream

int pa_attn_prefill(PA_ATTN_ARGS) {
  return pa::attn_common("pa_attn_prefill", PA_KIND_PREFILL, PA_ATTN_PASS);
}
int pa_attn_decode(PA_ATTN_ARGS) {
  return pa::attn_common("pa_attn_decode", PA_KIND_DECODE, PA_ATTN_PASS);
}
int pa_attn_verify(PA_ATTN_ARGS) {
  return pa::attn_common("pa_attn_verify", PA_KIND_VERIFY, PA_ATTN_PASS);
}

int pa_attn_decode_noalloc(const void* q, const void* k_cache, const void* v_cache,
                           int32_t num_blocks, const int32_t* block_table,
                           int32_t max_blocks_per_seq, const int32_t* seq_lens,
                           const int32_t* cu_seqlens_q, int32_t n_seqs, int32_t total_q,
                           int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                           int32_t block_size, float scale, int32_t dtype, int32_t* plan,
                           const pa_plan_info* info, void* out, float* lse, void* stream) {
  return pa::attn_common("pa_attn_decode_noalloc", PA_KIND_DECODE, q, k_cache, v_cache,
                         num_blocks, block_table, max_blocks_per_seq, seq_lens, cu_seqlens_q,
                         n_seqs, total_q, num_q_heads, num_kv_heads, head_dim, block_size, scale,
                         dtype, plan, info, nullptr, 0, out, lse, stream, /*noalloc=*/true);
}

int pa_set_launch_events(void* start_event, void* stop_event) {
  pa::clear_error();
  pa::t_ev_start = static_cast<hipEvent_t>(start_event);
  pa::t_ev_stop = static_cast<hipEvent_t>(stop_event);
  return PA_OK;
}

}  // extern "C"
