// float32 paged attention (VALU): the exact-precision path for float32 caches.
//
// Same definition as the bf16 path (paper: Section 2 PagedAttention / APC;
// Section 3, cached prefixes give the recomputed result): causal softmax over
// keys 0..a of the request's logical sequence, read through its block table.
// One wavefront per (query token, q-head); a 64-key chunk puts one key in each
// lane for the scores (16-byte loads of the key's 32-dim runs, four partial
// sums), then the lanes switch to owning head dimensions for the weighted
// value sum: each lane reads one dimension's 16 offsets of a block as four
// 16-byte loads and takes the probabilities from LDS, keys in order.  All
// arithmetic is float32 with fused multiply-adds; exp/log are the device
// library's float32 functions.
#include <hip/hip_ext.h>

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
  constexpr int DL = D / 64;  // value dimensions per lane
  static_assert(D % 64 == 0, "head_dim 64 or 128");
  __shared__ float qsh[D];
  __shared__ float psh[64];
  __shared__ int bsh[64 / kBlock];
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

  float od[DL];
#pragma unroll
  for (int k = 0; k < DL; ++k) od[k] = 0.f;
  float m = kNegInf, l = 0.f;
  for (int c0 = 0; c0 <= a; c0 += 64) {
    const int key = c0 + lane;
    const bool vis = key <= a;
    // every lane's block id is a clamped table entry, so each address below
    // is inside the cache
    const int blk = clamp_block(row[min(key / kBlock, max_blocks - 1)], num_blocks);
    float s = kNegInf;
    if (vis) {
      // the key's 32-dim runs in the grouped key layout, 32 floats each
      const float* kp = kc + ((int64_t)blk * hkv + g) * kBlock * D + key_elem(key % kBlock, 0);
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int gd = 0; gd < D; gd += kKeyGroup) {
        const f32x4* k4 = reinterpret_cast<const f32x4*>(kp + gd * kBlock);
#pragma unroll
        for (int j = 0; j < kKeyGroup / 4; ++j) {
          const f32x4 kv = k4[j];
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[j % 4] = fmaf(qsh[gd + 4 * j + e], kv[e], acc[j % 4]);
        }
      }
      s = ((acc[0] + acc[1]) + (acc[2] + acc[3])) * scale;
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
    for (int k = 0; k < DL; ++k) od[k] *= alpha;
    psh[lane] = p;
    if (lane % kBlock == 0) bsh[lane / kBlock] = blk;
    __syncthreads();
    // keys c0 .. c0 + nk - 1 are visible; the chunk starts on a block boundary
    const int nk = min(64, a + 1 - c0);
    for (int b = 0; b * kBlock < nk; ++b) {
      const float* vb = vc + ((int64_t)bsh[b] * hkv + g) * D * kBlock;
      const int kb = b * kBlock, nb = min(kBlock, nk - kb);
#pragma unroll
      for (int k = 0; k < DL; ++k) {
        const f32x4* v4 = reinterpret_cast<const f32x4*>(vb + (lane + 64 * k) * kBlock);
        f32x4 vv[kBlock / 4];
#pragma unroll
        for (int j = 0; j < kBlock / 4; ++j) vv[j] = v4[j];
        if (nb == kBlock) {
#pragma unroll
          for (int j = 0; j < kBlock; ++j) od[k] = fmaf(psh[kb + j], vv[j / 4][j % 4], od[k]);
        } else {
          // keys past the last visible one: slots that may never have been written
#pragma unroll
          for (int j = 0; j < kBlock; ++j)
            if (j < nb) od[k] = fmaf(psh[kb + j], vv[j / 4][j % 4], od[k]);
        }
      }
    }
    __syncthreads();  // psh and bsh are rewritten by the next chunk
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int k = 0; k < DL; ++k) out[((int64_t)token * hq + h) * D + lane + 64 * k] = od[k] * inv;
  if (lse && lane == 0) lse[(int64_t)token * hq + h] = m + logf(l);
}

}  // namespace

int launch_attn_f32(const void* q, const void* kc, const void* vc, int32_t num_blocks,
                    const int32_t* bt, int32_t max_blocks, const int32_t* seq_lens,
                    const int32_t* cu_q, int32_t n_seqs, int32_t total_q, int32_t hq, int32_t hkv,
                    int32_t d, float scale, void* out, float* lse, hipStream_t stream,
                    hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int64_t grid = int64_t(total_q) * hq;
  if (grid == 0) {
    // nothing launched: the events still mark this point of the stream
    for (hipEvent_t ev : {ev_start, ev_stop}) {
      const hipError_t e = ev ? hipEventRecord(ev, stream) : hipSuccess;
      if (e != hipSuccess) return static_cast<int>(e);
    }
    return 0;
  }
  // the caller's timing events ride on the dispatch (no event packets)
  if (d == 128)
    hipExtLaunchKernelGGL(attn_f32_kernel<128>, dim3(grid), dim3(64), 0, stream, ev_start, ev_stop,
                          0, static_cast<const float*>(q), static_cast<const float*>(kc),
                          static_cast<const float*>(vc), bt, max_blocks, seq_lens, cu_q, n_seqs,
                          hq, hkv, num_blocks, scale, static_cast<float*>(out), lse);
  else
    hipExtLaunchKernelGGL(attn_f32_kernel<64>, dim3(grid), dim3(64), 0, stream, ev_start, ev_stop,
                          0, static_cast<const float*>(q), static_cast<const float*>(kc),
                          static_cast<const float*>(vc), bt, max_blocks, seq_lens, cu_q, n_seqs,
                          hq, hkv, num_blocks, scale, static_cast<float*>(out), lse);
  return static_cast<int>(hipGetLastError());
}

}  // namespace dev
}  // namespace pa
