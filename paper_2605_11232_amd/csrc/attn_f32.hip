// float32 paged attention (VALU): the exact-precision path for float32 caches.
//
// Same definition as the bf16 path (paper: Section 2 PagedAttention / APC;
// Section 3, cached prefixes give the recomputed result): causal softmax over
// keys 0..a of the request's logical sequence, read through its block table.
// One wavefront per (query token, q-head); a 64-key chunk puts one key in each
// lane for the scores, then the lanes switch to owning head dimensions for
// the weighted value sum.  All arithmetic is float32 with fused multiply-adds;
// exp/log are the device library's float32 functions.
#include "device_common.h"

namespace pa {
namespace dev {
namespace {

template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kc, const float* __restrict__ vc,
    const int32_t* __restrict__ bt, int32_t max_blocks, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ cu_q, int32_t n_seqs, int32_t hq, int32_t hkv, int32_t num_blocks,
    float scale, float* __restrict__ out, float* __restrict__ lse) {
  __shared__ float qsh[D];
  const int token = blockIdx.x / hq, h = blockIdx.x % hq;
  const int lane = threadIdx.x;
  // sequence r: the last r with cu_q[r] <= token (empty sequences are skipped)
  int lo = 0, hi = n_seqs;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu_q[mid] <= token) lo = mid; else hi = mid;
  }
  const int r = lo;
  const int L = seq_lens[r];
  const int n = cu_q[r + 1] - cu_q[r];
  const int a = L - n + (token - cu_q[r]);
  const int g = h / (hq / hkv);
  const int32_t* row = bt + (int64_t)r * max_blocks;
  for (int d = lane; d < D; d += 64) qsh[d] = q[((int64_t)token * hq + h) * D + d];
  __syncthreads();

  float od[(D + 63) / 64];
#pragma unroll
  for (int k = 0; k < (D + 63) / 64; ++k) od[k] = 0.f;
  float m = kNegInf, l = 0.f;
  for (int c0 = 0; c0 <= a; c0 += 64) {
    const int key = c0 + lane;
    const bool vis = key <= a;
    float s = kNegInf;
    int blk = 0;
    if (vis) {
      blk = clamp_block(row[min(key / kBlock, max_blocks - 1)], num_blocks);
      // the key's 32-dim runs in the grouped key layout
      const float* kp = kc + ((int64_t)blk * hkv + g) * kBlock * D + key_elem(key % kBlock, 0);
      float dot = 0.f;
#pragma unroll
      for (int gd = 0; gd < D; gd += kKeyGroup)
#pragma unroll 8
        for (int d = 0; d < kKeyGroup; ++d)
          dot = fmaf(qsh[gd + d], kp[gd * kBlock + d], dot);
      s = dot * scale;
    }
    float cm = s;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cm = fmaxf(cm, __shfl_xor(cm, o, 64));
    const float mnew = fmaxf(m, cm);
    const float alpha = m == kNegInf ? 0.f : expf(m - mnew);
    const float p = vis ? expf(s - mnew) : 0.f;
    float ps = p;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ps += __shfl_xor(ps, o, 64);
    l = l * alpha + ps;
    m = mnew;
#pragma unroll
    for (int k = 0; k < (D + 63) / 64; ++k) od[k] *= alpha;
    const int nk = min(64, a + 1 - c0);
    for (int kk = 0; kk < nk; ++kk) {
      const float pk = __shfl(p, kk, 64);
      const int bk = __shfl(blk, kk, 64);
      const int off = (c0 + kk) % kBlock;
      const float* vp = vc + ((int64_t)bk * hkv + g) * D * kBlock + off;
#pragma unroll
      for (int k = 0; k < (D + 63) / 64; ++k) {
        const int d = lane + 64 * k;
        if (d < D) od[k] = fmaf(pk, vp[d * kBlock], od[k]);
      }
    }
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int k = 0; k < (D + 63) / 64; ++k) {
    const int d = lane + 64 * k;
    if (d < D) out[((int64_t)token * hq + h) * D + d] = od[k] * inv;
  }
  if (lse && lane == 0) lse[(int64_t)token * hq + h] = m + logf(l);
}

}  // namespace

int launch_attn_f32(const void* q, const void* kc, const void* vc, int32_t num_blocks,
                    const int32_t* bt, int32_t max_blocks, const int32_t* seq_lens,
                    const int32_t* cu_q, int32_t n_seqs, int32_t total_q, int32_t hq, int32_t hkv,
                    int32_t d, float scale, void* out, float* lse, hipStream_t stream) {
  const int64_t grid = int64_t(total_q) * hq;
  if (grid == 0) return 0;
  if (d == 128)
    hipLaunchKernelGGL(attn_f32_kernel<128>, dim3(grid), dim3(64), 0, stream,
                       static_cast<const float*>(q), static_cast<const float*>(kc),
                       static_cast<const float*>(vc), bt, max_blocks, seq_lens, cu_q, n_seqs, hq,
                       hkv, num_blocks, scale, static_cast<float*>(out), lse);
  else
    hipLaunchKernelGGL(attn_f32_kernel<64>, dim3(grid), dim3(64), 0, stream,
                       static_cast<const float*>(q), static_cast<const float*>(kc),
                       static_cast<const float*>(vc), bt, max_blocks, seq_lens, cu_q, n_seqs, hq,
                       hkv, num_blocks, scale, static_cast<float*>(out), lse);
  return static_cast<int>(hipGetLastError());
}

}  // namespace dev
}  // namespace pa
